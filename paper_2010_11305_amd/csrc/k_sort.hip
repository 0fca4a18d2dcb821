// Sort and de-duplication of one step's lookups (the paper's Sec. 5.1: sort the
// row indices of the mini-batch, merge the gradients of each row).
//
//   k_expand       lookups -> (set-major row key, gradient-row index), position order
//   radix passes   stable LSD radix sort, 8-bit digits, wave-ballot ranking, one kernel
//                  per pass with decoupled look-back
//   scans          3-phase exclusive prefix sums (u32 / u64)
//   k_uniq_*       unique-row and touched-set lists (first occurrence of each row / set)
#include "embc_device.h"
#include "embc_dispatch.h"
#include "embc_sort.h"

namespace embc {

constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanThreads * kScanItems;
constexpr int kRadixThreads = 256;
constexpr int kRadixItems = 16;
constexpr int kRadixTile = kRadixThreads * kRadixItems;
constexpr int kRadixWaves = kRadixThreads / 64;

size_t scan_partial_words(int64_t n) { return (size_t)((n + kScanTile - 1) / kScanTile + 64); }

// ---- block-wide exclusive scan of one value per thread (256 threads) -------------------
template <typename T>
__device__ __forceinline__ T block_exclusive_scan(T v, T* lds4, T& total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  T x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const T y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) lds4[wv] = x;
  __syncthreads();
  T pre = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < kScanThreads / 64; ++w) {
    const T s = lds4[w];
    if (w < wv) pre += s;
    total += s;
  }
  __syncthreads();
  return pre + x - v;
}

// ---- 3-phase exclusive scan ---------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kScanThreads) void k_scan_reduce(const T* __restrict__ in, int64_t n,
                                                              const unsigned long long* dev_n, T* part) {
  __shared__ T lds4[4];
  if (dev_n) n = min(n, (int64_t)*dev_n);
  if ((int64_t)blockIdx.x * kScanTile >= n) return;  // a tile past the values (whole block)
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  T s = 0;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i)
    if (base + i < n) s += in[base + i];
  T tot;
  block_exclusive_scan<T>(s, lds4, tot);
  if (threadIdx.x == 0) part[blockIdx.x] = tot;
}

// Exclusive scan of in[0, nb) into out (which may be in) by one block of kScanThreads,
// kTopItems consecutive values per thread and round; *total_out = the sum.
constexpr int kTopItems = 16;
template <typename T>
__device__ __forceinline__ void scan_one_block(const T* in, T* out, int64_t nb, T* total_out) {
  __shared__ T lds4[4];
  T carry = 0;
  for (int64_t b0 = 0; b0 < nb; b0 += (int64_t)kScanThreads * kTopItems) {
    const int64_t base = b0 + (int64_t)threadIdx.x * kTopItems;
    T v[kTopItems];
    T s = 0;
#pragma unroll
    for (int q = 0; q < kTopItems; ++q) {
      v[q] = base + q < nb ? in[base + q] : (T)0;
      s += v[q];
    }
    T tot;
    T run = carry + block_exclusive_scan<T>(s, lds4, tot);
#pragma unroll
    for (int q = 0; q < kTopItems; ++q) {
      if (base + q < nb) out[base + q] = run;
      run += v[q];
    }
    carry += tot;
  }
  if (threadIdx.x == 0 && total_out) *total_out = carry;
}

// The tiles past the device-side count (dev_n) hold no values: only the first
// ceil(min(n, dev_n) / kScanTile) partials are scanned.
template <typename T>
__global__ __launch_bounds__(kScanThreads) void k_scan_top(T* part, int64_t nb, int64_t n,
                                                           const unsigned long long* dev_n, T* total_out) {
  if (dev_n) nb = min(nb, (min(n, (int64_t)*dev_n) + kScanTile - 1) / kScanTile);
  scan_one_block<T>(part, part, nb, total_out);
}

// A short array (tens of thousands of values) in one launch.
template <typename T>
__global__ __launch_bounds__(kScanThreads) void k_scan_one(const T* in, T* out, int64_t n, T* total_out) {
  scan_one_block<T>(in, out, n, total_out);
}

template <typename T>
__global__ __launch_bounds__(kScanThreads) void k_scan_down(const T* __restrict__ in, T* __restrict__ out, int64_t n,
                                                            const unsigned long long* dev_n, const T* part) {
  __shared__ T lds4[4];
  if (dev_n) n = min(n, (int64_t)*dev_n);
  if ((int64_t)blockIdx.x * kScanTile >= n) return;  // a tile past the values (whole block)
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  T v[kScanItems];
  T s = 0;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    v[i] = base + i < n ? in[base + i] : (T)0;
    s += v[i];
  }
  T tot;
  T run = block_exclusive_scan<T>(s, lds4, tot) + part[blockIdx.x];
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    if (base + i < n) out[base + i] = run;
    run += v[i];
  }
}

template <typename T>
hipError_t scan_exclusive(const T* in, T* out, int64_t n, const unsigned long long* dev_n, T* part, T* total,
                          hipStream_t s) {
  if (n <= 0) {
    if (total) k_scan_top<T><<<1, kScanThreads, 0, s>>>(part, 0, 0, nullptr, total);
    return hipGetLastError();
  }
  const int64_t nb = (n + kScanTile - 1) / kScanTile;
  k_scan_reduce<T><<<(unsigned)nb, kScanThreads, 0, s>>>(in, n, dev_n, part);
  k_scan_top<T><<<1, kScanThreads, 0, s>>>(part, nb, n, dev_n, total);
  k_scan_down<T><<<(unsigned)nb, kScanThreads, 0, s>>>(in, out, n, dev_n, part);
  return hipGetLastError();
}

// kScanItems consecutive values of a and b from element base (0 past n); whole runs are
// read 16 bytes at a time (the arrays are 16-byte aligned and base is a multiple of 8).
__device__ __forceinline__ void load_pair_items(const uint32_t* a, const uint32_t* b, int64_t n, int64_t base,
                                                uint32_t (&va)[kScanItems], uint32_t (&vb)[kScanItems]) {
  static_assert(kScanItems % 4 == 0, "runs of 16 bytes");
  if (base + kScanItems <= n) {
#pragma unroll
    for (int i = 0; i < kScanItems; i += 4) {
      const uint4 x = *reinterpret_cast<const uint4*>(a + base + i);
      const uint4 y = *reinterpret_cast<const uint4*>(b + base + i);
      va[i] = x.x; va[i + 1] = x.y; va[i + 2] = x.z; va[i + 3] = x.w;
      vb[i] = y.x; vb[i + 1] = y.y; vb[i + 2] = y.z; vb[i + 3] = y.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
      va[i] = base + i < n ? a[base + i] : 0u;
      vb[i] = base + i < n ? b[base + i] : 0u;
    }
  }
}

// Exclusive scans of two u32 arrays at once (a + b * 2^32 as one u64 value per element:
// the prefix sums of a stay below 2^32), written to out_a and out_b (which may be a and
// b); *total = the two totals packed the same way.
__global__ __launch_bounds__(kScanThreads) void k_scan2_reduce(const uint32_t* __restrict__ a,
                                                               const uint32_t* __restrict__ b, int64_t n,
                                                               const unsigned long long* dev_n,
                                                               unsigned long long* part) {
  __shared__ unsigned long long lds4[4];
  if (dev_n) n = min(n, (int64_t)*dev_n);
  if ((int64_t)blockIdx.x * kScanTile >= n) return;
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  uint32_t va[kScanItems], vb[kScanItems];
  load_pair_items(a, b, n, base, va, vb);
  unsigned long long s = 0;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) s += (unsigned long long)va[i] | ((unsigned long long)vb[i] << 32);
  unsigned long long tot;
  block_exclusive_scan<unsigned long long>(s, lds4, tot);
  if (threadIdx.x == 0) part[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kScanThreads) void k_scan2_down(const uint32_t* a, const uint32_t* b, uint32_t* out_a,
                                                             uint32_t* out_b, int64_t n,
                                                             const unsigned long long* dev_n,
                                                             const unsigned long long* part) {
  __shared__ unsigned long long lds4[4];
  if (dev_n) n = min(n, (int64_t)*dev_n);
  if ((int64_t)blockIdx.x * kScanTile >= n) return;
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  uint32_t va[kScanItems], vb[kScanItems];
  load_pair_items(a, b, n, base, va, vb);
  unsigned long long s = 0;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) s += (unsigned long long)va[i] | ((unsigned long long)vb[i] << 32);
  unsigned long long tot;
  unsigned long long run = block_exclusive_scan<unsigned long long>(s, lds4, tot) + part[blockIdx.x];
  // the exclusive prefixes replace the values in place (va, vb)
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    const unsigned long long v = (unsigned long long)va[i] | ((unsigned long long)vb[i] << 32);
    va[i] = (uint32_t)run;
    vb[i] = (uint32_t)(run >> 32);
    run += v;
  }
  if (base + kScanItems <= n) {
#pragma unroll
    for (int i = 0; i < kScanItems; i += 4) {
      *reinterpret_cast<uint4*>(out_a + base + i) = make_uint4(va[i], va[i + 1], va[i + 2], va[i + 3]);
      *reinterpret_cast<uint4*>(out_b + base + i) = make_uint4(vb[i], vb[i + 1], vb[i + 2], vb[i + 3]);
    }
  } else {
#pragma unroll
    for (int i = 0; i < kScanItems; ++i)
      if (base + i < n) {
        out_a[base + i] = va[i];
        out_b[base + i] = vb[i];
      }
  }
}

hipError_t scan_exclusive_pair(const uint32_t* a, const uint32_t* b, uint32_t* out_a, uint32_t* out_b, int64_t n,
                               const unsigned long long* dev_n, unsigned long long* part,
                               unsigned long long* total, hipStream_t s) {
  if (n <= 0) {
    k_scan_top<unsigned long long><<<1, kScanThreads, 0, s>>>(part, 0, 0, nullptr, total);
    return hipGetLastError();
  }
  const int64_t nb = (n + kScanTile - 1) / kScanTile;
  k_scan2_reduce<<<(unsigned)nb, kScanThreads, 0, s>>>(a, b, n, dev_n, part);
  k_scan_top<unsigned long long><<<1, kScanThreads, 0, s>>>(part, nb, n, dev_n, total);
  k_scan2_down<<<(unsigned)nb, kScanThreads, 0, s>>>(a, b, out_a, out_b, n, dev_n, part);
  return hipGetLastError();
}

template hipError_t scan_exclusive<uint32_t>(const uint32_t*, uint32_t*, int64_t, const unsigned long long*,
                                             uint32_t*, uint32_t*, hipStream_t);
template hipError_t scan_exclusive<unsigned long long>(const unsigned long long*, unsigned long long*, int64_t,
                                                       const unsigned long long*, unsigned long long*,
                                                       unsigned long long*, hipStream_t);

// ---- LSD radix sort of (key, value) pairs -----------------------------------------------
// Lanes whose 8-bit digits are equal, among the `valid` lanes of the wave.
__device__ __forceinline__ uint64_t match_digit(uint32_t d, bool valid) {
  uint64_t m = __ballot(valid);
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    // keep the lanes whose bit b equals this lane's: bit b sign-extended, XNOR the ballot
    const uint32_t s = (uint32_t)((int32_t)(d << (31 - b)) >> 31);
    const uint64_t bb = __ballot(s != 0);
    m &= ~(bb ^ (((uint64_t)s << 32) | s));
  }
  return m;
}

// Stable LSD radix sort, one kernel per 8-bit digit pass, after the Onesweep method
// (Adinets and Merrill, "Onesweep: A Faster Least Significant Digit Radix Sort for
// GPUs", 2022): one histogram pass for every digit, then per digit pass a single
// sweep in which each tile finds its output offsets by decoupled look-back (Merrill
// and Garland, "Single-pass Parallel Prefix Scan with Decoupled Look-back", 2016):
//   k_sort_hist   global histograms of every pass's digit in one read of the keys
//   k_sort_scan   their exclusive prefix sums: where each digit's run starts
//   k_sort_pass   per tile of kRadixTile pairs (tiles taken in launch order from an
//                 atomic ticket): rank the tile's digits, publish the per-digit tile
//                 counts, find the tile's offset inside each digit's run by looking
//                 back over the published counts of the preceding tiles (decoupled
//                 look-back), then scatter through LDS in digit runs.
// A status word per (tile, digit) holds a 2-bit state and a 30-bit count: not yet
// published, the tile's own count, or the inclusive count up to and including the
// tile.  Tiles are numbered in the order their workgroups start, so every tile a
// look-back waits for is already running; the wait is bounded all the same (after
// kSortSpinLimit polls the step is flagged as failed and the tile goes on).
//
// Segmented mode.  The lookups arrive grouped by table (bag t*B + b belongs to table
// t), so the keys of table t fill the positions [P_t, P_t+1) and every valid key there
// lies in table t's key range.  Sorting each segment by the local key (key minus the
// table's key base) gives the global order in fewer passes when every table's key
// range is far smaller than the sum of them (100 tables of 5M rows: 3 passes instead
// of 4).  Tiles never straddle a segment (each segment starts a new tile), a look-back
// ends at the segment's first tile, and digit runs start at P_t.  The per-table digit
// counts are taken by the expansion (k_expand) as it forms the keys, so this mode has
// no histogram pass of its own.  A skipped lookup
// (kKeyInvalid) takes digit 255 in every pass, above every valid local key, so it ends
// its table's segment; when there is any, one more stable pass (digit 1 for a skipped
// key, 0 for the others) moves them behind every valid key, and the pairs are copied
// back so that the result stays in the same buffer.
constexpr uint32_t kStAgg = 1u << 30;
constexpr uint32_t kStPre = 2u << 30;
constexpr uint32_t kStCount = (1u << 30) - 1;
constexpr uint32_t kSortSpinLimit = 1u << 20;

size_t sort_status_words(int64_t n, int T) {
  return 256 * (size_t)((n + kRadixTile - 1) / kRadixTile + T + 1);
}
size_t sort_seg_words(int T) { return 2 * (size_t)T * kMaxPasses * 256 + 2 * (size_t)(T + 1) + 64; }

__device__ __forceinline__ uint32_t status_load(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void status_store(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Segment of tile `tile` (< tbase[T]): the largest t with tbase[t] <= tile.  Empty
// segments share their successor's first tile and are never returned.
__device__ __forceinline__ int seg_of_tile(const uint32_t* tbase, int T, uint32_t tile) {
  int lo = 0, hi = T;  // tbase[lo] <= tile < tbase[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (tbase[mid] <= tile) lo = mid; else hi = mid;
  }
  return lo;
}

// Digit of a key in a pass of the segmented mode: the local key's, or 255 when skipped.
__device__ __forceinline__ uint32_t seg_digit(uint32_t key, uint32_t kb, int shift) {
  return key == kKeyInvalid ? 255u : ((key - kb) >> shift) & 255u;
}

// ghist [kMaxPasses][256] and the pass tickets must be zero on entry (k_sort_begin).
// Also clears the status words of the first pass.
__global__ __launch_bounds__(256) void k_sort_hist(const uint32_t* __restrict__ keys, int64_t n, int passes,
                                                   uint32_t* __restrict__ ghist, uint32_t* __restrict__ status,
                                                   int64_t status_words) {
  __shared__ uint32_t h[kRadixWaves][kMaxPasses][256];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < kRadixWaves * kMaxPasses * 256; i += 256) (&h[0][0][0])[i] = 0;
  __syncthreads();
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  // whole waves iterate together (the tail lanes count nothing), so that the lanes
  // sharing lane 0's digit are counted with one atomic: high digits of keys that
  // are nearly sorted would otherwise all hit one LDS word
  for (int64_t i0 = (int64_t)blockIdx.x * blockDim.x + wv * 64; i0 < n; i0 += stride) {
    const int64_t i = i0 + lane;
    const bool valid = i < n;
    const uint32_t k = valid ? keys[i] : 0u;
    for (int p = 0; p < passes; ++p) {
      const uint32_t d = (k >> (8 * p)) & 255u;
      const uint32_t d0 = __builtin_amdgcn_readfirstlane(d);  // all lanes active: lane 0's
      const uint64_t same = __ballot(valid && d == d0);
      if (lane == 0) atomicAdd(&h[wv][p][d0], (uint32_t)__popcll(same));
      if (valid && d != d0) atomicAdd(&h[wv][p][d], 1u);
    }
  }
  __syncthreads();
  for (int p = 0; p < passes; ++p) {
    uint32_t c = 0;
#pragma unroll
    for (int w = 0; w < kRadixWaves; ++w) c += h[w][p][threadIdx.x];
    if (c) atomicAdd(&ghist[p * 256 + threadIdx.x], c);
  }
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < status_words; i += stride) status[i] = 0;
}

__global__ void k_sort_begin(uint32_t* __restrict__ ghist, uint32_t* __restrict__ tickets) {
  for (int i = threadIdx.x; i < kMaxPasses * 256; i += blockDim.x) ghist[i] = 0;
  if (threadIdx.x < kMaxPasses) tickets[threadIdx.x] = 0;
}

// gbase[p][d] = number of keys whose pass-p digit is below d.
__global__ __launch_bounds__(256) void k_sort_scan(const uint32_t* __restrict__ ghist, uint32_t* __restrict__ gbase,
                                                   int passes) {
  __shared__ uint32_t lds4[4];
  for (int p = 0; p < passes; ++p) {
    uint32_t tot;
    gbase[p * 256 + threadIdx.x] = block_exclusive_scan<uint32_t>(ghist[p * 256 + threadIdx.x], lds4, tot);
  }
}

// Segment starts P_t (t = 0..T; P_0 = 0 and P_T = n, so positions outside every bag,
// which hold skipped keys, join the first or the last segment) and the first tile of
// each segment (tbase[T] = number of tiles), by block 0, which also zeroes the digit
// counts and tickets (as k_sort_begin does).  With malformed offsets every key is skipped
// and the whole stream is one segment.  The grid clears the per-table histograms.
__global__ __launch_bounds__(256) void k_seg_setup(const int32_t* __restrict__ off, int32_t B, int T, int64_t n,
                                                   const unsigned long long* __restrict__ ctr, SegSort sg,
                                                   uint32_t* __restrict__ ghist, uint32_t* __restrict__ tickets) {
  __shared__ uint32_t lds4[4];
  const int64_t hw = (int64_t)T * kMaxPasses * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < hw; i += (int64_t)gridDim.x * 256) sg.hist[i] = 0;
  if (blockIdx.x != 0) return;
  for (int i = threadIdx.x; i < kMaxPasses * 256; i += blockDim.x) ghist[i] = 0;
  if (threadIdx.x < kMaxPasses) tickets[threadIdx.x] = 0;
  const bool bad = ctr[kCBadOffsets] != 0;
  const auto start = [&](int t) -> int64_t {
    if (t <= 0) return 0;
    if (t >= T || bad) return n;
    return min<int64_t>(max<int64_t>(off[(int64_t)t * B], 0), n);
  };
  uint32_t run = 0;
  for (int t0 = 0; t0 <= T; t0 += 256) {
    const int t = t0 + (int)threadIdx.x;
    uint32_t tiles = 0;
    int64_t p = 0;
    if (t <= T) {
      p = start(t);
      if (t < T) tiles = (uint32_t)((start(t + 1) - p + kRadixTile - 1) / kRadixTile);
    }
    uint32_t tot;
    const uint32_t ex = block_exclusive_scan<uint32_t>(tiles, lds4, tot);
    if (t <= T) {
      sg.pos[t] = (uint32_t)p;
      sg.tbase[t] = run + ex;
    }
    run += tot;
  }
}

// base[t][p][d] = P_t + number of table t's keys whose pass-p digit is below d (one
// block per table); block 0 also writes the bases of the pass that moves skipped keys
// last: valid keys from 0, skipped ones from n - n_skipped.
__global__ __launch_bounds__(256) void k_seg_scan(SegSort sg, int passes, int64_t n,
                                                  const uint32_t* __restrict__ n_skipped,
                                                  uint32_t* __restrict__ skip_base) {
  __shared__ uint32_t lds4[4];
  const int t = blockIdx.x;
  for (int p = 0; p < passes; ++p) {
    const int64_t i = ((int64_t)t * kMaxPasses + p) * 256 + threadIdx.x;
    uint32_t tot;
    sg.base[i] = sg.pos[t] + block_exclusive_scan<uint32_t>(sg.hist[i], lds4, tot);
  }
  if (t == 0 && threadIdx.x < 2) skip_base[threadIdx.x] = threadIdx.x == 0 ? 0u : (uint32_t)(n - n_skipped[0]);
}

// One radix pass.  kModeSeg: tiles of the segmented mode (sg, pass), digits of the local
// key.  Otherwise tiles of the whole stream, with the key's digit at `shift`
// (kModeWhole) or 1 for a skipped key and 0 for the others (kModeSkipped); a non-null
// only_if skips the pass (and the copy below) unless *only_if.
// Without LOOP, a workgroup handles the one tile its ticket names (grid = tiles: a new
// workgroup's loads overlap the scatter of a finishing one).  With LOOP the grid is at
// most what the device holds at once and every workgroup takes tiles from the ticket
// until none is left (the pass that only runs when some key was skipped: when none
// was, it ends after one read of the flag per workgroup).  Either way a look-back only
// waits on tiles whose workgroups took their ticket earlier and are running.
constexpr int kModeWhole = 0, kModeSeg = 1, kModeSkipped = 2;

template <int MODE, bool LOOP>
__global__ __launch_bounds__(kRadixThreads) void k_sort_pass(const uint32_t* __restrict__ kin,
                                                             const uint32_t* __restrict__ vin,
                                                             uint32_t* __restrict__ kout, uint32_t* __restrict__ vout,
                                                             int64_t n, int shift, const uint32_t* __restrict__ gbase,
                                                             uint32_t* __restrict__ status, uint32_t* __restrict__ ticket,
                                                             uint32_t* __restrict__ next_status,
                                                             int64_t status_words, int32_t* __restrict__ err,
                                                             SegSort sg, const int64_t* __restrict__ key_base, int T,
                                                             int pass, const uint32_t* __restrict__ only_if) {
  __shared__ uint32_t wcnt[kRadixWaves][256];
  __shared__ uint32_t dpre[256];
  __shared__ uint32_t goff[256];
  __shared__ uint32_t skey[kRadixTile];
  __shared__ uint32_t sval[kRadixTile];
  __shared__ uint32_t lds4[4];
  __shared__ uint32_t tile_s;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  constexpr bool SEG = MODE == kModeSeg;
  const int64_t ntiles = SEG ? (int64_t)sg.tbase[T]
                             : (only_if == nullptr || *only_if != 0) ? (n + kRadixTile - 1) / kRadixTile : 0;
  for (;;) {
    for (int i = threadIdx.x; i < kRadixWaves * 256; i += kRadixThreads) (&wcnt[0][0])[i] = 0;
    if (threadIdx.x == 0) tile_s = ntiles > 0 ? atomicAdd(ticket, 1u) : 0xFFFFFFFFu;
    __syncthreads();
    const int64_t tile = tile_s;
    if (tile >= ntiles) break;  // block-uniform
    // the tile's table and position range
    int t = 0;
    int64_t tfirst = 0, lo = tile * kRadixTile, hi = min<int64_t>(n, lo + kRadixTile);
    uint32_t kb = 0;
    if (SEG) {
      t = seg_of_tile(sg.tbase, T, (uint32_t)tile);
      tfirst = sg.tbase[t];
      lo = sg.pos[t] + (tile - tfirst) * kRadixTile;
      hi = min<int64_t>(sg.pos[t + 1], lo + kRadixTile);
      kb = (uint32_t)key_base[t];
    }
    const auto digit = [&](uint32_t key) -> uint32_t {
      if constexpr (MODE == kModeSeg) return seg_digit(key, kb, shift);
      else if constexpr (MODE == kModeSkipped) return key == kKeyInvalid ? 1u : 0u;
      else return (key >> shift) & 255u;
    };
    const int64_t base = lo + (int64_t)wv * 64 * kRadixItems;
    uint32_t k[kRadixItems], v[kRadixItems], rank[kRadixItems];
#pragma unroll
    for (int i = 0; i < kRadixItems; ++i) {
      const int64_t p = base + i * 64 + lane;
      const bool valid = p < hi;
      k[i] = valid ? kin[p] : 0xFFFFFFFFu;
      v[i] = valid ? vin[p] : 0u;
    }
#pragma unroll
    for (int i = 0; i < kRadixItems; ++i) {
      const int64_t p = base + i * 64 + lane;
      const bool valid = p < hi;
      const uint32_t d = digit(k[i]);
      const uint64_t peers = match_digit(d, valid);
      const uint32_t before = (uint32_t)__popcll(peers & lanemask_lt());
      // the first lane of each digit adds the digit's lanes to the wave's count and
      // hands the old count to the others; a wave's LDS operations complete in issue
      // order, so each item sees the counts of the items before it, and the 16
      // atomics of a thread are in flight together
      uint32_t old = 0;
      if (valid && before == 0) old = atomicAdd(&wcnt[wv][d], (uint32_t)__popcll(peers));
      const int first = valid ? (int)__builtin_ctzll(peers) : lane;
      rank[i] = __shfl(old, first) + before;
    }
    __syncthreads();
    {
      const int d = threadIdx.x;
      uint32_t run = 0;
#pragma unroll
      for (int w = 0; w < kRadixWaves; ++w) {
        const uint32_t c = wcnt[w][d];
        wcnt[w][d] = run;
        run += c;
      }
      uint32_t* st = status + tile * 256 + d;
      uint32_t excl = 0;
      if (tile == tfirst) {
        status_store(st, kStPre | run);
      } else {
        status_store(st, kStAgg | run);
        int64_t j = tile - 1;
        uint32_t polls = 0;
        for (;;) {
          const uint32_t w = status_load(status + j * 256 + d);
          const uint32_t state = w & ~kStCount;
          if (state == 0) {
            if (++polls > kSortSpinLimit) {
              atomicOr(err, kErrSort);
              break;
            }
            __builtin_amdgcn_s_sleep(1);
            continue;
          }
          excl += w & kStCount;
          if (state == kStPre || j == tfirst) break;
          --j;
        }
        status_store(st, kStPre | (excl + run));
      }
      uint32_t tot;
      dpre[d] = block_exclusive_scan<uint32_t>(run, lds4, tot);
      goff[d] = (SEG ? sg.base[((int64_t)t * kMaxPasses + pass) * 256 + d] : gbase[d]) + excl;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kRadixItems; ++i) {
      const int64_t p = base + i * 64 + lane;
      if (p < hi) {
        const uint32_t d = digit(k[i]);
        const uint32_t pos = dpre[d] + wcnt[wv][d] + rank[i];
        skey[pos] = k[i];
        sval[pos] = v[i];
      }
    }
    __syncthreads();
    const int cnt = (int)(hi - lo);
    for (int j = threadIdx.x; j < cnt; j += kRadixThreads) {
      const uint32_t key = skey[j];
      const uint32_t d = digit(key);
      const uint32_t g = goff[d] + (uint32_t)j - dpre[d];
      if ((int64_t)g < n) {  // always, unless a look-back gave up
        kout[g] = key;
        vout[g] = sval[j];
      }
    }
    if constexpr (!LOOP) break;
    __syncthreads();  // LDS is reused by the next tile
  }
  // the other status buffer (the previous pass's, finished) is cleared for the next pass
  if (next_status) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < status_words; i += stride) next_status[i] = 0;
  }
}

// (src) -> (dst) pairs when *only_if is non-zero.
__global__ __launch_bounds__(256) void k_copy_pairs(const uint32_t* __restrict__ ks, const uint32_t* __restrict__ vs,
                                                    uint32_t* __restrict__ kd, uint32_t* __restrict__ vd, int64_t n,
                                                    const uint32_t* __restrict__ only_if) {
  if (*only_if == 0) return;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    kd[i] = ks[i];
    vd[i] = vs[i];
  }
}

// workgroups of a pass that loops over `tiles` tiles: no more than the device holds at once
template <int MODE>
unsigned pass_grid(int64_t tiles) {
  const int64_t r = resident_grid(reinterpret_cast<const void*>(k_sort_pass<MODE, true>), kRadixThreads);
  return (unsigned)std::max<int64_t>(1, std::min<int64_t>(tiles, r));
}

hipError_t sort_pairs(uint32_t* kA, uint32_t* vA, uint32_t* kB, uint32_t* vB, int64_t n, int passes,
                      const SortScratch& ss, int32_t* err, int* in_B, hipStream_t s) {
  *in_B = 0;
  if (n <= 0) return hipSuccess;
  if (passes < 1 || passes > kMaxPasses || n > (int64_t)kStCount) return hipErrorInvalidValue;
  const int64_t nb = (n + kRadixTile - 1) / kRadixTile;
  const int64_t sw = 256 * nb;
  k_sort_begin<<<1, 256, 0, s>>>(ss.ghist, ss.tickets);
  k_sort_hist<<<grid_for(n, 2048), 256, 0, s>>>(kA, n, passes, ss.ghist, ss.status[0], sw);
  k_sort_scan<<<1, 256, 0, s>>>(ss.ghist, ss.gbase, passes);
  for (int pass = 0; pass < passes; ++pass) {
    const uint32_t* ki = *in_B ? kB : kA;
    const uint32_t* vi = *in_B ? vB : vA;
    uint32_t* ko = *in_B ? kA : kB;
    uint32_t* vo = *in_B ? vA : vB;
    uint32_t* next = pass + 1 < passes ? ss.status[(pass + 1) & 1] : nullptr;
    k_sort_pass<kModeWhole, false><<<(unsigned)nb, kRadixThreads, 0, s>>>(ki, vi, ko, vo, n, 8 * pass, ss.gbase + 256 * pass,
                                                              ss.status[pass & 1], ss.tickets + pass, next, sw, err,
                                                              SegSort{}, nullptr, 0, pass, nullptr);
    *in_B = !*in_B;
  }
  return hipGetLastError();
}

hipError_t seg_begin(int64_t n, int passes, const int32_t* off, int32_t B, int T, const int64_t* key_base,
                     const unsigned long long* ctr, const SortScratch& ss, const SegSort& sg, ExpandHist* eh,
                     hipStream_t s) {
  if (n <= 0 || passes < 1 || passes >= kMaxPasses || n > (int64_t)kStCount || T < 1) return hipErrorInvalidValue;
  const int64_t hw = (int64_t)T * kMaxPasses * 256;
  k_seg_setup<<<(unsigned)std::min<int64_t>(64, (hw + 1023) / 1024), 256, 0, s>>>(off, B, T, n, ctr, sg, ss.ghist,
                                                                                 ss.tickets);
  eh->hist = sg.hist;
  eh->key_base = key_base;
  eh->n_skipped = ss.ghist;
  eh->status = ss.status[0];
  eh->status_words = 256 * ((n + kRadixTile - 1) / kRadixTile + T);
  eh->passes = passes;
  return hipGetLastError();
}

hipError_t sort_pairs_segmented(uint32_t* kA, uint32_t* vA, uint32_t* kB, uint32_t* vB, int64_t n, int passes,
                                const int32_t* off, int32_t B, int T, const int64_t* key_base,
                                const unsigned long long* ctr, const SortScratch& ss, const SegSort& sg, int32_t* err,
                                int* in_B, hipStream_t s) {
  *in_B = 0;
  if (n <= 0) return hipSuccess;
  if (passes < 1 || passes >= kMaxPasses || n > (int64_t)kStCount || T < 1) return hipErrorInvalidValue;
  const int64_t nb_max = (n + kRadixTile - 1) / kRadixTile + T;  // every segment adds at most one partial tile
  const int64_t sw = 256 * nb_max;
  uint32_t* n_skipped = ss.ghist;  // zeroed by k_seg_setup
  uint32_t* skip_base = ss.gbase;
  k_seg_scan<<<(unsigned)T, 256, 0, s>>>(sg, passes, n, n_skipped, skip_base);
  for (int pass = 0; pass < passes; ++pass) {
    const uint32_t* ki = *in_B ? kB : kA;
    const uint32_t* vi = *in_B ? vB : vA;
    uint32_t* ko = *in_B ? kA : kB;
    uint32_t* vo = *in_B ? vA : vB;
    // the last segmented pass clears the status words of the pass for skipped keys
    uint32_t* next = ss.status[(pass + 1) & 1];
    k_sort_pass<kModeSeg, false><<<(unsigned)nb_max, kRadixThreads, 0, s>>>(ki, vi, ko, vo, n, 8 * pass, nullptr,
                                                                 ss.status[pass & 1], ss.tickets + pass, next, sw,
                                                                 err, sg, key_base, T, pass, nullptr);
    *in_B = !*in_B;
  }
  // skipped keys behind every valid key, then back into the same buffer; both kernels
  // return at once when there is none
  uint32_t* kr = *in_B ? kB : kA;
  uint32_t* vr = *in_B ? vB : vA;
  uint32_t* ko = *in_B ? kA : kB;
  uint32_t* vo = *in_B ? vA : vB;
  const uint32_t* any_skipped = n_skipped;
  const int64_t nb = (n + kRadixTile - 1) / kRadixTile;
  k_sort_pass<kModeSkipped, true><<<pass_grid<kModeSkipped>(nb), kRadixThreads, 0, s>>>(kr, vr, ko, vo, n, 0, skip_base,
                                                            ss.status[passes & 1], ss.tickets + passes, nullptr,
                                                            256 * nb, err, SegSort{}, nullptr, 0, 0, any_skipped);
  k_copy_pairs<<<grid_for(n, 2048), 256, 0, s>>>(ko, vo, kr, vr, n, any_skipped);
  return hipGetLastError();
}

// ---- lookups -> sort pairs ----------------------------------------------------------------
// One wave per 64 consecutive bags (global bag = t*B + b); each position of those
// bags finds its bag by a binary search over the 64 lane-held bag starts.
// key: set-major row key (kKeyInvalid for an out-of-range row); value: the bag b
// within its table (its gradient row in grad_out [B][T][d] is b*T + t).
// With SEG (the per-table sort mode) the expansion also does the counting of that mode,
// from the keys it forms rather than from a second read of them: per table, the digit
// counts of every pass of the local key (255 in every digit for a skipped key), the
// number of skipped keys, and the cleared status words of the first pass.  A
// workgroup gathers the counts of its first bag's table in LDS and adds them once; a
// key of another table (a workgroup across a table boundary) is added directly.
// Positions outside every bag belong to the first table's segment (before the first
// bag) or the last one's (after the last bag), as the segment starts place them.
template <bool SEG>
__global__ __launch_bounds__(256) void k_expand(Dev dv, const int32_t* __restrict__ idx, int64_t L,
                                                const int32_t* __restrict__ off, int32_t B, DivConst byB,
                                                uint32_t* __restrict__ keys, uint32_t* __restrict__ vals,
                                                int64_t nbag_waves, int64_t bag_blocks,
                                                const unsigned long long* __restrict__ ctr, ExpandHist eh) {
  __shared__ uint32_t h[SEG ? kMaxPasses * 256 : 1];
  __shared__ uint32_t skipped_s;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t nbags = (int64_t)dv.T * B;
  if constexpr (SEG) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < eh.status_words; i += stride)
      eh.status[i] = 0;
  }
  if (ctr[kCBadOffsets]) {
    // offsets failed validation: every lookup of the step is skipped (and the whole
    // stream is the first table's segment)
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < L; p += stride)
      keys[p] = kKeyInvalid, vals[p] = 0;
    if constexpr (SEG) {
      if (blockIdx.x == 0 && threadIdx.x == 0 && L > 0) {
        for (int p = 0; p < eh.passes; ++p) atomicAdd(&eh.hist[p * 256 + 255], (uint32_t)L);
        atomicAdd(eh.n_skipped, (uint32_t)L);
      }
    }
    return;
  }
  if ((int64_t)blockIdx.x >= bag_blocks) {
    // positions outside every bag: [0, off[0]) and [off[nbags], L)
    const int64_t head = min<int64_t>(max<int64_t>(off[0], 0), L);
    const int64_t tail = min<int64_t>(max<int64_t>(off[nbags], head), L);
    const int64_t tid = ((int64_t)blockIdx.x - bag_blocks) * blockDim.x + threadIdx.x;
    const int64_t stride = ((int64_t)gridDim.x - bag_blocks) * blockDim.x;
    for (int64_t p = tid; p < head; p += stride) keys[p] = kKeyInvalid, vals[p] = 0;
    for (int64_t p = tail + tid; p < L; p += stride) keys[p] = kKeyInvalid, vals[p] = 0;
    if constexpr (SEG) {
      if (tid == 0 && head + (L - tail) > 0) {
        const int64_t last = (int64_t)(dv.T - 1) * kMaxPasses * 256;
        for (int p = 0; p < eh.passes; ++p) {
          if (head) atomicAdd(&eh.hist[p * 256 + 255], (uint32_t)head);
          if (L - tail) atomicAdd(&eh.hist[last + p * 256 + 255], (uint32_t)(L - tail));
        }
        atomicAdd(eh.n_skipped, (uint32_t)(head + (L - tail)));
      }
    }
    return;
  }
  // the table whose counts this workgroup gathers in LDS: that of its first bag
  const int t_wg = (int)div_by((uint32_t)((int64_t)blockIdx.x * 256), byB);
  uint32_t kb_wg = 0;
  if constexpr (SEG) {
    kb_wg = (uint32_t)eh.key_base[t_wg];
    for (int i = threadIdx.x; i < kMaxPasses * 256; i += 256) h[i] = 0;
    if (threadIdx.x == 0) skipped_s = 0;
    __syncthreads();
  }
  uint32_t n_skip = 0;
  const int64_t bw = (int64_t)blockIdx.x * 4 + wv;
  if (bw < nbag_waves) {
    const int64_t bag0 = bw * 64;
    const int64_t mybag = bag0 + lane;
    const int64_t lastbag = min<int64_t>(bag0 + 64, nbags);
    int64_t st = L;
    if (mybag < nbags) st = min<int64_t>(max<int64_t>(off[mybag], 0), L);
    const int64_t P0 = min<int64_t>(max<int64_t>(off[bag0], 0), L);
    const int64_t P1 = min<int64_t>(max<int64_t>(off[lastbag], P0), L);
    uint32_t n_ok = 0, n_bad = 0;
    // global bags are below 2^32 (checked when the handle is created): their table by
    // one high multiply; the descriptor of the wave's first table is loaded once
    const int t_run = (int)div_by((uint32_t)bag0, byB);
    const TableDesc td_run = dv.desc[t_run];
    const auto handle = [&](int64_t p, int32_t r, int j) {
      const uint32_t bag = (uint32_t)(bag0 + j);
      const int t = (int)div_by(bag, byB);
      const int b = (int)(bag - (uint32_t)t * (uint32_t)B);
      const TableDesc td = t == t_run ? td_run : dv.desc[t];
      uint32_t key = kKeyInvalid;
      if (r >= 0 && (int64_t)r < td.N) {
        if (td.n_sets > 0) {
          const uint32_t q = div_by((uint32_t)r, td.by_sets);
          const uint32_t set = (uint32_t)r - q * (uint32_t)td.n_sets;
          key = (uint32_t)(td.key_base + (int64_t)set * td.Q + q);
        } else {
          key = (uint32_t)(td.key_base + r);
        }
        if (t == t_run) ++n_ok; else atomicAdd(&dv.stats[(int64_t)t * kNStat + kStBwdLookups], 1ull);
      } else {
        if (t == t_run) ++n_bad; else atomicAdd(&dv.stats[(int64_t)t * kNStat + kStInvalidBwd], 1ull);
        atomicOr(dv.err, kErrIndex);
      }
      keys[p] = key;
      vals[p] = (uint32_t)b;
      if constexpr (SEG) {
        n_skip += key == kKeyInvalid;
        if (t == t_wg) {
          for (int q = 0; q < eh.passes; ++q) atomicAdd(&h[q * 256 + seg_digit(key, kb_wg, 8 * q)], 1u);
        } else {
          const uint32_t kb = (uint32_t)eh.key_base[t];
          uint32_t* ht = eh.hist + (int64_t)t * kMaxPasses * 256;
          for (int q = 0; q < eh.passes; ++q) atomicAdd(&ht[q * 256 + seg_digit(key, kb, 8 * q)], 1u);
        }
      }
    };
    // two runs of 64 positions at a time: their index loads and bag searches interleave
    for (int64_t pc = P0; pc < P1; pc += 128) {
      const int64_t pA = pc + lane, pB = pc + 64 + lane;
      const bool inA = pA < P1, inB = pB < P1;
      const int32_t rA = inA ? idx[pA] : 0;
      const int32_t rB = inB ? idx[pB] : 0;
      int jA = 0, jB = 0;
#pragma unroll
      for (int step = 32; step >= 1; step >>= 1) {
        const int64_t sA = __shfl(st, jA + step);
        const int64_t sB = __shfl(st, jB + step);
        if (jA + step < 64 && sA <= pA) jA += step;
        if (jB + step < 64 && sB <= pB) jB += step;
      }
      if (inA) handle(pA, rA, jA);
      if (inB) handle(pB, rB, jB);
    }
    // lookups of the wave's first table: one atomic per wave
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      n_ok += __shfl_xor(n_ok, o);
      n_bad += __shfl_xor(n_bad, o);
    }
    if (lane == 0 && n_ok) atomicAdd(&dv.stats[(int64_t)t_run * kNStat + kStBwdLookups], (unsigned long long)n_ok);
    if (lane == 0 && n_bad) atomicAdd(&dv.stats[(int64_t)t_run * kNStat + kStInvalidBwd], (unsigned long long)n_bad);
  }
  if constexpr (SEG) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) n_skip += __shfl_xor(n_skip, o);
    if (lane == 0 && n_skip) atomicAdd(&skipped_s, n_skip);
    __syncthreads();
    uint32_t* ht = eh.hist + (int64_t)t_wg * kMaxPasses * 256;
    for (int i = threadIdx.x; i < eh.passes * 256; i += 256) {
      const uint32_t c = h[i];
      if (c) atomicAdd(&ht[i], c);
    }
    if (threadIdx.x == 0 && skipped_s) atomicAdd(eh.n_skipped, skipped_s);
  }
}

__global__ __launch_bounds__(256) void k_check_offsets(Dev dv, const int32_t* __restrict__ off, int64_t nbags,
                                                       int64_t L, unsigned long long* __restrict__ ctr) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nbags; i += stride) {
    const int64_t a = off[i], b = off[i + 1];
    if (a < 0 || b < a || b > L) {
      ctr[kCBadOffsets] = 1;
      atomicOr(dv.err, kErrOffsets);
    }
  }
}

hipError_t launch_expand(const Dev& dv, const int32_t* idx, int64_t L, const int32_t* off, int32_t B, uint32_t* keys,
                         uint32_t* vals, unsigned long long* ctr, const ExpandHist* eh, hipStream_t s) {
  const int64_t nbags = (int64_t)dv.T * B;
  const int64_t nbag_waves = (nbags + 63) / 64;
  const int64_t bag_blocks = (nbag_waves + 3) / 4;
  const int64_t tail_blocks = 16;
  const DivConst byB = div_const(B > 0 ? (uint32_t)B : 1u);  // no bag when B = 0
  const unsigned grid = (unsigned)(bag_blocks + tail_blocks);
  if (eh) {
    k_expand<true><<<grid, 256, 0, s>>>(dv, idx, L, off, B, byB, keys, vals, nbag_waves, bag_blocks, ctr, *eh);
  } else {
    k_expand<false><<<grid, 256, 0, s>>>(dv, idx, L, off, B, byB, keys, vals, nbag_waves, bag_blocks, ctr,
                                         ExpandHist{});
  }
  return hipGetLastError();
}

// ---- unique rows and touched sets ---------------------------------------------------------
// A row start is a valid key that differs from its predecessor in the sorted stream; a
// set start is a row start of a cached table whose (table, set) differs from the
// predecessor's.  Two passes over tiles of kUqTile keys (kUqPer consecutive keys per
// thread): k_uniq_count writes each tile's counts packed as (sets << 32 | rows); after
// their exclusive scan, k_uniq_write writes every start at its tile's offset plus its
// rank inside the tile: the key and first occurrence of each unique row, and the first
// unique row of each touched set.
constexpr int kUqPer = 16;
constexpr int kUqTile = 256 * kUqPer;

size_t uniq_tile_words(int64_t n) { return (size_t)((n + kUqTile - 1) / kUqTile + 1); }

// Table of the keys seen by one thread, with the key range and set stride of that table.
struct TabCursor {
  int t = -1;
  int64_t kb = 0, kb_next = 0;
  DivConst byQ;
  bool cached = false;
  __device__ void load(const Dev& dv) {
    kb = dv.key_base[t];
    kb_next = dv.key_base[t + 1];
    const TableDesc& td = dv.desc[t];
    byQ = td.by_Q;
    cached = td.n_sets > 0;
  }
  // position on the table of a valid key (keys only increase after the first call)
  __device__ void seek(const Dev& dv, uint32_t key) {
    if (t < 0) {
      t = table_of_key(dv.key_base, dv.T, key);
      load(dv);
    }
    while ((int64_t)key >= kb_next) {
      ++t;
      load(dv);
    }
  }
  __device__ uint32_t set_of(uint32_t key) const { return div_by((uint32_t)((int64_t)key - kb), byQ); }
};

// Walks the thread's keys; calls on_start(i, key, is_set_start, table) for every row start.
// Returns the index of the first invalid key if it lies in the thread's range, else -1.
template <typename F>
__device__ __forceinline__ int64_t walk_starts(const Dev& dv, const uint32_t* __restrict__ sk, int64_t n,
                                               int64_t i0, const uint32_t (&k)[kUqPer], F&& on_start) {
  uint32_t prev = i0 > 0 ? sk[i0 - 1] : kKeyInvalid;
  TabCursor cur;
  int pt = -1;        // table of prev (valid prev only)
  uint32_t pset = 0;  // set of prev (cached table only)
  if (prev != kKeyInvalid) {
    cur.seek(dv, prev);
    pt = cur.t;
    if (cur.cached) pset = cur.set_of(prev);
  }
  int64_t first_invalid = -1;
#pragma unroll
  for (int j = 0; j < kUqPer; ++j) {
    const int64_t i = i0 + j;
    if (i < n) {
      const uint32_t key = k[j];
      if (key == kKeyInvalid) {
        if (prev != kKeyInvalid || i == 0) first_invalid = i;
      } else if (i == 0 || key != prev) {
        cur.seek(dv, key);
        bool new_set = false;
        if (cur.cached) {
          const uint32_t st = cur.set_of(key);
          new_set = pt != cur.t || st != pset || i == 0;
          pset = st;
        }
        pt = cur.t;
        on_start(i, key, new_set, cur.t);
      }
      prev = key;
    }
  }
  return first_invalid;
}

__device__ __forceinline__ void load_tile_keys(const uint32_t* __restrict__ sk, int64_t n, int64_t i0,
                                               uint32_t (&k)[kUqPer]) {
  if (i0 + kUqPer <= n) {
    const uint4* p = reinterpret_cast<const uint4*>(sk + i0);
#pragma unroll
    for (int j = 0; j < kUqPer / 4; ++j) {
      const uint4 v = p[j];
      k[4 * j] = v.x; k[4 * j + 1] = v.y; k[4 * j + 2] = v.z; k[4 * j + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int j = 0; j < kUqPer; ++j) k[j] = i0 + j < n ? sk[i0 + j] : kKeyInvalid;
  }
}

__global__ __launch_bounds__(256) void k_uniq_count(Dev dv, const uint32_t* __restrict__ sk, int64_t n,
                                                    unsigned long long* __restrict__ tile_cnt,
                                                    unsigned long long* __restrict__ thread_pre,
                                                    unsigned long long* __restrict__ ctr) {
  __shared__ unsigned long long lds4[4];
  const int64_t i0 = (int64_t)blockIdx.x * kUqTile + (int64_t)threadIdx.x * kUqPer;
  uint32_t k[kUqPer];
  load_tile_keys(sk, n, i0, k);
  unsigned long long c = 0;
  const int64_t fi = walk_starts(dv, sk, n, i0, k, [&](int64_t, uint32_t, bool ns, int) {
    c += 1ull + (ns ? (1ull << 32) : 0ull);
  });
  if (fi >= 0) ctr[kCValid] = (unsigned long long)fi;
  unsigned long long tot;
  thread_pre[(int64_t)blockIdx.x * 256 + threadIdx.x] = block_exclusive_scan<unsigned long long>(c, lds4, tot);
  if (threadIdx.x == 0) tile_cnt[blockIdx.x] = tot;
}

__global__ __launch_bounds__(256) void k_uniq_write(Dev dv, const uint32_t* __restrict__ sk, int64_t n,
                                                    const unsigned long long* __restrict__ tile_pre,
                                                    const unsigned long long* __restrict__ thread_pre,
                                                    uint32_t* __restrict__ uk, uint32_t* __restrict__ seg,
                                                    uint32_t* __restrict__ set_first, int32_t* __restrict__ utab,
                                                    unsigned long long* __restrict__ ctr) {
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    const unsigned long long tot = ctr[kCScanTotal];
    const uint32_t nu = (uint32_t)(tot & 0xFFFFFFFFull), ns = (uint32_t)(tot >> 32);
    ctr[kCUnique] = nu;
    ctr[kCSets] = ns;
    seg[nu] = (uint32_t)ctr[kCValid];
    set_first[ns] = nu;
  }
  const int64_t i0 = (int64_t)blockIdx.x * kUqTile + (int64_t)threadIdx.x * kUqPer;
  uint32_t k[kUqPer];
  load_tile_keys(sk, n, i0, k);
  // the thread's offset: its tile's, plus its own inside the tile (both from k_uniq_count)
  const unsigned long long base = thread_pre[(int64_t)blockIdx.x * 256 + threadIdx.x] + tile_pre[blockIdx.x];
  uint32_t u = (uint32_t)(base & 0xFFFFFFFFull), st = (uint32_t)(base >> 32);
  walk_starts(dv, sk, n, i0, k, [&](int64_t i, uint32_t key, bool ns, int t) {
    uk[u] = key;
    seg[u] = (uint32_t)i;
    utab[u] = t;
    if (ns) set_first[st++] = u;
    ++u;
  });
}

hipError_t launch_unique(const Dev& dv, const uint32_t* sk, int64_t n, unsigned long long* tile_cnt,
                         unsigned long long* tile_pre, unsigned long long* thread_pre, uint32_t* uk, uint32_t* seg,
                         uint32_t* set_first, int32_t* utab, unsigned long long* ctr,
                         hipStream_t s) {
  const int64_t tiles = (n + kUqTile - 1) / kUqTile;
  if (tiles > 0) k_uniq_count<<<(unsigned)tiles, 256, 0, s>>>(dv, sk, n, tile_cnt, thread_pre, ctr);
  k_scan_one<unsigned long long><<<1, kScanThreads, 0, s>>>(tile_cnt, tile_pre, tiles, ctr + kCScanTotal);
  k_uniq_write<<<(unsigned)(tiles > 0 ? tiles : 1), 256, 0, s>>>(dv, sk, n, tile_pre, thread_pre, uk, seg,
                                                                 set_first, utab, ctr);
  return hipGetLastError();
}

}  // namespace embc
