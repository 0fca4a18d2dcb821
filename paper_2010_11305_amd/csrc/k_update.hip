// Backward + sparse update of one step (Sec. 3 update operator, Alg. 2, Sec. 5.1 de-dup).
//
// After the sort (k_sort.hip) the lookups are grouped by row, the rows by set:
//   k_probe     per unique row: residency (slot or miss), LRU stamp / LFU count update
//   k_partials  chunk sums (64 lookups each) of the merged gradient of rows with 65..512 lookups
//   k_policy    per touched set, a group of G >= assoc lanes (one lane per way; 64/G sets
//               per wave): which missed rows enter the cache and which resident each of
//               them displaces (decisions only)
//   k_block_partials  per (table, bag block): the block's gradient rows staged in LDS
//               once, the block sums of every row with > 512 lookups; k_block_fold
//               folds them per row (chunk sums are folded by the kernel that uses them)
//   k_evict     per insert that displaces a resident: the resident's FP32 row (updated
//               first if it was itself updated this step, LFU) is quantized into T
//   k_update    per unique row: merged gradient, fetch, optimizer, then the cache way
//               (hit or insert) or quantization into T (bypass); it runs after k_evict,
//               so every displaced row has been read before an insert overwrites its way
// The row kernels split tables over the XCDs (XcdSplit) so that each L2 serves one table.
#include "embc_device.h"
#include "embc_dispatch.h"
#include "embc_sort.h"

namespace embc {

constexpr int32_t kActDone = 4;  // row fully handled by k_policy

constexpr int kUnroll = 2;  // independent row loads in flight per row group
constexpr int64_t kSpreadBelow = 1 << 21;  // lookups per step below which SPREAD kernels run

__global__ void k_bwd_begin(Dev dv, unsigned long long* ctr, int64_t L) {
  for (int i = threadIdx.x; i < dv.T; i += blockDim.x) {
    for (int f = kStBwdLookups; f <= kStHitEvictions; ++f) dv.stats[(int64_t)i * kNStat + f] = 0;
    dv.stats[(int64_t)i * kNStat + kStInvalidBwd] = 0;
  }
  if (threadIdx.x == 0) {
    for (int c = 0; c < kNCounters; ++c) ctr[c] = 0;
    ctr[kCValid] = (unsigned long long)L;
  }
}

// LFU decay: every count halved, unless the step's offsets were rejected (such a call
// changes no state).
__global__ __launch_bounds__(256) void k_decay(int32_t* __restrict__ cnt, int64_t n,
                                               const unsigned long long* __restrict__ ctr) {
  if (ctr[kCBadOffsets]) return;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) cnt[i] >>= 1;
}

// ---- probe ---------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_probe(Dev dv, Work w, uint32_t step) {
  const int64_t nU = (int64_t)w.ctr[kCUnique];
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t base = (int64_t)blockIdx.x * blockDim.x; base < nU; base += stride) {
    const int64_t u = base + threadIdx.x;
    const bool act = u < nU;
    int t = 0;
    int32_t slot = -1;
    if (act) {
      const uint32_t key = w.uniq_key[u];
      t = w.utab[u];  // written with the key by k_uniq_write
      const TableDesc td = dv.desc[t];
      const int64_t local = (int64_t)key - td.key_base;
      int64_t r = local;
      if (td.n_sets > 0) {
        const uint32_t sq = div_by((uint32_t)local, td.by_Q);  // local = set * Q + q
        r = (int64_t)((uint32_t)local - sq * (uint32_t)td.Q) * td.n_sets + sq;
      }
      const int64_t grow = td.row_base + r;
      const uint32_t count = w.seg[u + 1] - w.seg[u];
      slot = probe_slot(dv, td, (int32_t)r);
      w.urow[u] = (int32_t)grow;
      w.uslot[u] = slot;
      w.uact[u] = slot >= 0 ? kActHitStay : kActBypass;
      // chunks of kSumChunk lookups for 64 < count <= kBlockAbove; bag blocks above
      const bool big = count > kBlockAbove;
      w.nch[u] = count > (uint32_t)kSumChunk && !big ? (count + kSumChunk - 1) / kSumChunk : 0u;
      w.ubig[u] = big ? 1u : 0u;
      if (dv.policy == 0) {
        if (slot >= 0) dv.ts[slot] = (int32_t)step;
      } else {
        const int64_t c = (int64_t)dv.cnt[grow] + count;
        const int32_t cn = c > 0x7FFFFFFF ? 0x7FFFFFFF : (int32_t)c;
        dv.cnt[grow] = cn;
        // a missed row's rank among the candidates of its set: count, then lower row first
        w.ukey[u] = slot >= 0 ? 0ull : ((unsigned long long)(uint32_t)cn << 32) | (uint32_t)~(uint32_t)grow;
      }
    }
  }
}

// ---- merged gradient ----------------------------------------------------------------------
// R9 order: a row's lookups in position order; up to kSumChunk of them summed left to
// right (seeded with the first); up to kBlockAbove in chunks of kSumChunk consecutive
// lookups (k_partials), the chunk sums folded left to right; more by bag blocks of
// NB = kBlockFloats/d bags (k_block_partials), the non-empty block sums folded left
// to right.  The sort's value of a lookup is its bag b within the table.

// Gradient rows of table t: grad_out is [B][T][d], so bag b's row is row b*T + t (an
// index below 2^32: B*T < 2^32 is checked when the handle is created).
template <int D>
struct GradRows {
  const float* grad;
  uint32_t T, t;
  __device__ const float* row(uint32_t b) const { return grad + (int64_t)(b * T + t) * D; }
};

template <int D>
__device__ __forceinline__ GradRows<D> grad_rows(const float* grad, int t, int T) {
  return GradRows<D>{grad, (uint32_t)T, (uint32_t)t};
}

// Left-to-right sum of the gradient rows of occurrences [i0, i1) of the sorted
// stream (i0 < i1), seeded with the first.  Lane j of the group preloads the bag of
// occurrence j of each run of LPR occurrences (for the first run the caller may pass
// them in, myv0); U rows are loaded before they are added in order.
// Rows narrower than 16 lanes (d < 128) hold kRun/LPR bags per lane, so that a run (one
// load of bags) covers kRun occurrences whatever the width, with kSmallUnroll rows in
// flight; the order of the additions is the same.
constexpr int kRun = 16;
constexpr int kSmallUnroll = 8;

template <int D>
__device__ __forceinline__ void sum_occ(const uint32_t* __restrict__ sval, int64_t i0, int64_t i1, GradRows<D> gr,
                                        int g, float (&acc)[8], uint32_t myv0 = 0u, bool have0 = false) {
  constexpr int LPR = Geo<D>::LPR, CPL = 8, U = kUnroll;
  if constexpr (LPR < kRun) {
    constexpr int BPL = kRun / LPR, US = kSmallUnroll;
    bool first = true;
    for (int64_t ic = i0; ic < i1; ic += kRun) {
      const int n = (int)min<int64_t>(kRun, i1 - ic);
      // occurrence j of the run: bag myv[j / LPR] of lane j % LPR
      uint32_t myv[BPL];
#pragma unroll
      for (int b = 0; b < BPL; ++b) {
        const int64_t i = ic + b * LPR + g;
        myv[b] = (b == 0 && have0 && ic == i0) ? myv0 : (i < i1 ? sval[i] : 0u);
      }
#pragma unroll
      for (int j0 = 0; j0 < kRun; j0 += US) {
        if (j0 >= n) break;
        float x[US][CPL];
#pragma unroll
        for (int q = 0; q < US; ++q) {
          const int j = j0 + q;
          if (j < n) load_row<D>(gr.row(__shfl(myv[j / LPR], j % LPR, LPR)), g, x[q]);
        }
#pragma unroll
        for (int q = 0; q < US; ++q) {
          if (j0 + q >= n) break;
          if (first) {
#pragma unroll
            for (int k = 0; k < CPL; ++k) acc[k] = x[q][k];
            first = false;
          } else {
#pragma unroll
            for (int k = 0; k < CPL; ++k) acc[k] = acc[k] + x[q][k];
          }
        }
      }
    }
    return;
  }
  bool first = true;
  for (int64_t ic = i0; ic < i1; ic += LPR) {
    const int n = (int)min<int64_t>(LPR, i1 - ic);
    // the first run's values may have been loaded by the caller (have0)
    const uint32_t myv = (have0 && ic == i0) ? myv0 : (g < n ? sval[ic + g] : 0u);
    int j = 0;
    if (first) {
      load_row<D>(gr.row(__shfl(myv, 0, LPR)), g, acc);
      first = false;
      j = 1;
    }
    for (; j + U <= n; j += U) {
      float x[U][CPL];
#pragma unroll
      for (int q = 0; q < U; ++q) load_row<D>(gr.row(__shfl(myv, j + q, LPR)), g, x[q]);
#pragma unroll
      for (int q = 0; q < U; ++q)
#pragma unroll
        for (int k = 0; k < CPL; ++k) acc[k] = acc[k] + x[q][k];
    }
    for (; j < n; ++j) {
      float x[CPL];
      load_row<D>(gr.row(__shfl(myv, j, LPR)), g, x);
#pragma unroll
      for (int k = 0; k < CPL; ++k) acc[k] = acc[k] + x[k];
    }
  }
}

constexpr int kChunkUnroll = 4;  // gradient rows in flight per row group in a chunk sum

// Sum of one chunk (occurrences [i0, i1) of the sorted stream, 0 < i1 - i0 <= 64),
// left to right, seeded with the first.  The bags of the next LPR occurrences are
// loaded while the current ones are summed, U gradient rows are in flight at a
// time, and a row listed more than once in one bag (adjacent occurrences with the
// same bag) adds the row already in registers instead of loading it again (same
// operands, same sums).
template <int D>
__device__ __forceinline__ void chunk_sum(const uint32_t* __restrict__ sval, int64_t i0, int64_t i1, GradRows<D> gr,
                                          int g, float (&acc)[8]) {
  constexpr int LPR = Geo<D>::LPR, CPL = 8, U = kChunkUnroll;
  // the sum starts from -0, the identity of IEEE addition: adding the first term gives
  // exactly that term, as in the seeded left-to-right sum (the chunk is not empty)
#pragma unroll
  for (int k = 0; k < CPL; ++k) acc[k] = -0.0f;
  if constexpr (LPR < kRun) {
    // narrow rows: runs of kRun occurrences (kRun/LPR bags per lane), kSmallUnroll rows
    // in flight, the next run's bags loaded while one is summed
    constexpr int BPL = kRun / LPR, US = kSmallUnroll;
    uint32_t vn[BPL];
#pragma unroll
    for (int b = 0; b < BPL; ++b) vn[b] = i0 + b * LPR + g < i1 ? sval[i0 + b * LPR + g] : 0u;
    for (int64_t ic = i0; ic < i1; ic += kRun) {
      const int n = (int)min<int64_t>(kRun, i1 - ic);
      uint32_t myv[BPL];
#pragma unroll
      for (int b = 0; b < BPL; ++b) {
        myv[b] = vn[b];
        const int64_t i = ic + kRun + b * LPR + g;
        vn[b] = i < i1 ? sval[i] : 0u;
      }
#pragma unroll
      for (int j0 = 0; j0 < kRun; j0 += US) {
        if (j0 >= n) break;
        float x[US][CPL];
#pragma unroll
        for (int q = 0; q < US; ++q) {
          const int j = j0 + q;
          if (j < n) load_row<D>(gr.row(__shfl(myv[j / LPR], j % LPR, LPR)), g, x[q]);
        }
#pragma unroll
        for (int q = 0; q < US; ++q) {
          if (j0 + q >= n) break;
#pragma unroll
          for (int k = 0; k < CPL; ++k) acc[k] = acc[k] + x[q][k];
        }
      }
    }
    return;
  }
  uint32_t pv = 0xFFFFFFFFu;  // bag of the last occurrence added (none yet)
  float last[CPL];
#pragma unroll
  for (int k = 0; k < CPL; ++k) last[k] = 0.0f;
  uint32_t vnext = i0 + g < i1 ? sval[i0 + g] : 0u;
  for (int64_t ic = i0; ic < i1; ic += LPR) {
    const int n = (int)min<int64_t>(LPR, i1 - ic);
    const uint32_t myv = vnext;
    vnext = ic + LPR + g < i1 ? sval[ic + LPR + g] : 0u;
    for (int j = 0; j < n; j += U) {
      uint32_t v[U];
      bool fresh[U];
      float x[U][CPL];
#pragma unroll
      for (int q = 0; q < U; ++q) {
        v[q] = __shfl(myv, j + q, LPR);
        fresh[q] = j + q < n && v[q] != (q == 0 ? pv : v[q - 1]);
        if (fresh[q]) load_row<D>(gr.row(v[q]), g, x[q]);
      }
#pragma unroll
      for (int q = 0; q < U; ++q) {
        if (j + q < n) {
          if (!fresh[q]) {
#pragma unroll
            for (int k = 0; k < CPL; ++k) x[q][k] = last[k];
          }
#pragma unroll
          for (int k = 0; k < CPL; ++k) acc[k] = acc[k] + x[q][k];
#pragma unroll
          for (int k = 0; k < CPL; ++k) last[k] = x[q][k];
          pv = v[q];
        }
      }
    }
  }
}

// Left-to-right fold of the n >= 1 chunk sums of one row, rows c0 .. c0+n-1 of
// `partial` (acc = p0, then acc + p1, ...), U rows loaded before they are added.
template <int D>
__device__ __forceinline__ void fold_chunks(const float* __restrict__ partial, int64_t c0, uint32_t n, int g,
                                            float (&acc)[8]) {
  constexpr int U = kUnroll;
  load_row<D>(partial + c0 * D, g, acc);
  uint32_t j = 1;
  for (; j + U <= n; j += U) {
    float x[U][8];
#pragma unroll
    for (int q = 0; q < U; ++q) load_row<D>(partial + (c0 + j + q) * D, g, x[q]);
#pragma unroll
    for (int q = 0; q < U; ++q)
#pragma unroll
      for (int k = 0; k < 8; ++k) acc[k] = acc[k] + x[q][k];
  }
  for (; j < n; ++j) {
    float x[8];
    load_row<D>(partial + (c0 + j) * D, g, x);
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] = acc[k] + x[k];
  }
}

// Left-to-right fold of the non-empty block sums of big row h (blocks 0 .. nblk-1),
// seeded with the first; U blocks (bounds and sums) are loaded at a time (the fold is
// one chain of loads per row over few rows: 16 at a time, not 4, takes it from 149 to
// 92 us on the stress workload's 512 blocks).  The sum slot of an empty block holds no
// value and is not added.
template <int D>
__device__ __forceinline__ void fold_blocks(const Work& w, int64_t h, int nblk, int g, float (&acc)[8]) {
  constexpr int U = 16;
  const uint32_t* bb = w.bbound + h * (int64_t)bound_stride(w.max_nblk);
  const float* bp = w.bpart + h * (int64_t)w.max_nblk * D;
  bool first = true;
  uint32_t prev = bb[0];
  for (int k0 = 0; k0 < nblk; k0 += U) {
    uint32_t nx[U];
    float x[U][8];
#pragma unroll
    for (int q = 0; q < U; ++q) {
      const int k = min(k0 + q, nblk - 1);
      nx[q] = bb[(k + 1) * kStages];
      load_row<D>(bp + (int64_t)k * D, g, x[q]);
    }
#pragma unroll
    for (int q = 0; q < U; ++q) {
      if (k0 + q < nblk && nx[q] > prev) {
        if (first) {
#pragma unroll
          for (int k = 0; k < 8; ++k) acc[k] = x[q][k];
          first = false;
        } else {
#pragma unroll
          for (int k = 0; k < 8; ++k) acc[k] = acc[k] + x[q][k];
        }
      }
      if (k0 + q < nblk) prev = nx[q];
    }
  }
}

// Fold of the block sums of every big row (one row group per row), left in the
// row's first block slot.
template <int D>
__global__ __launch_bounds__(256) void k_block_fold(Work w, int nblk) {
  constexpr int LPR = Geo<D>::LPR, GPB = 256 / LPR;
  const int g = threadIdx.x & (LPR - 1);
  const int64_t nbig = (int64_t)w.ctr[kCBig];
  for (int64_t h = (int64_t)blockIdx.x * GPB + threadIdx.x / LPR; h < nbig; h += (int64_t)gridDim.x * GPB) {
    float acc[8];
    fold_blocks<D>(w, h, nblk, g, acc);
    store_row<D>(w.bpart + h * (int64_t)w.max_nblk * D, g, acc);
  }
}

// Merged gradient of unique row u (occurrences [s0, s1) of the sorted stream).
template <int D>
__device__ __forceinline__ void merged_grad(const Work& w, const uint32_t* __restrict__ sval, GradRows<D> gr,
                                            int64_t u, int g, float (&acc)[8]) {
  const uint32_t s0 = w.seg[u], s1 = w.seg[u + 1];
  if (s1 - s0 > kBlockAbove) load_row<D>(w.bpart + (int64_t)w.ubig[u] * w.max_nblk * D, g, acc);
  else if (w.nch[u] > 0) fold_chunks<D>(w.partial, w.chunk_base[u], w.nch[u], g, acc);
  else sum_occ<D>(sval, s0, s1, gr, g, acc);
}

// bbound[h][j] = first occurrence of big row h whose bag lies in stage j (the j-th run
// of NB/kStages bags) or after (j = 0 .. kStages*nblk; the last = the end of its
// occurrences): one thread per (row, stage) binary-searches the row's occurrences,
// whose bags ascend.  Bag block k is stages kStages*k .. kStages*k + kStages - 1.
__global__ __launch_bounds__(256) void k_block_bounds(Work w, const uint32_t* __restrict__ sval, int stage_shift,
                                                      int nblk) {
  const int64_t nbig = (int64_t)w.ctr[kCBig];
  const int ns = kStages * nblk;
  const int64_t n = nbig * (ns + 1);
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += stride) {
    const int64_t h = e / (ns + 1);
    const int j = (int)(e - h * (ns + 1));
    const int64_t u = w.big_rows[h];
    uint32_t a = w.seg[u], b = w.seg[u + 1];  // first occurrence with bag >= j*NS lies in [a, b]
    if (j < ns) {
      const uint32_t key = (uint32_t)j << stage_shift;
      while (a < b) {
        const uint32_t m = a + (b - a) / 2;
        if (sval[m] < key) a = m + 1; else b = m;
      }
    } else {
      a = b;
    }
    w.bbound[h * (int64_t)bound_stride(w.max_nblk) + j] = a;
  }
}

// Block sums of the big rows: per (table t, bag block k), the gradient rows of the
// block's NB bags are staged in LDS a stage of NB/kStages bags (64 KiB) at a time, so
// that two workgroups share a CU (while one waits on a long sum the other works); one
// group of GL = min(64, d) lanes per big row of t with occurrences in the stage (CL =
// d/GL columns per lane; rows taken longest first) adds them left to right to the
// row's block sum, which starts from -0 (the identity of IEEE addition) in the block's
// first stage with occurrences and is carried between stages in the row's block slot.
// The bags of 4*GL occurrences are loaded at a time (4 per lane) and U staged rows are
// read at a time.  Tables split over the XCDs; a workgroup takes every units-th
// (segment, block) pair of its XCD.
constexpr int kBlockThreads = 512;

template <int D>
__global__ __launch_bounds__(kBlockThreads) void k_block_partials(Dev dv, Work w, const uint32_t* __restrict__ sval,
                                                                  const float* __restrict__ grad, int32_t B,
                                                                  int nblk) {
  // the gradient sums run beside the eviction on the second stream and decide when the
  // row update can start: their waves issue first where they share a SIMD
  __builtin_amdgcn_s_setprio(3);
  constexpr int NB = kBlockFloats / D;
  constexpr int NS = NB / kStages;  // bags per stage
  constexpr int SF = kBlockFloats / kStages;  // floats per stage
  constexpr int GL = D < 64 ? D : 64;  // lanes per row group
  constexpr int CL = D / GL;           // columns per lane (1, 2 or 4)
  constexpr int U = 8;
  constexpr int PER = SF / 4 / kBlockThreads;  // float4 staged per thread
  __shared__ float4 stage[SF / 4];
  __shared__ uint32_t lrow[kBlockThreads], lr0[kBlockThreads], lr1[kBlockThreads], cnt_s[4];
  const float* sf = reinterpret_cast<const float*>(stage);
  const int l = threadIdx.x & (GL - 1);
  const XcdSplit xs(dv.T, true);
  const int64_t stride_b = bound_stride(w.max_nblk);
  // (segment, block) pairs of this XCD: segment xs.xcd + kXcds*i holds blocks
  // [klo, khi) of its table, at most kcap of them
  const int64_t kcap = (nblk + xs.parts - 1) / xs.parts;
  const int64_t nseg_x = (xs.segments(dv.T) - xs.xcd + kXcds - 1) / kXcds;
  for (int64_t job = xs.unit; job < nseg_x * kcap; job += xs.units) {
    const int seg = xs.xcd + kXcds * (int)(job / kcap);
    const int t = seg / xs.parts;
    const int64_t h0 = w.ubig[w.tab_first[t]], h1 = w.ubig[w.tab_first[t + 1]];
    if (h0 == h1) continue;
    int64_t klo, khi;
    part_range(0, nblk, seg % xs.parts, xs.parts, klo, khi);
    const int64_t k = klo + job % kcap;
    if (k >= khi) continue;
    for (int hs = 0; hs < kStages; ++hs) {
      const int64_t js = k * kStages + hs;  // stage index
      const int64_t bag0 = js * NS;
      if (bag0 >= B) break;
      const int nrows = (int)min<int64_t>(NS, (int64_t)B - bag0);
      __syncthreads();  // the previous stage's sums are done with `stage`
      {
        float4 v[PER];
#pragma unroll
        for (int q = 0; q < PER; ++q) {
          const int i = q * kBlockThreads + threadIdx.x;
          const int r = min(i / (D / 4), nrows - 1);  // rows past the last bag re-read it (not used)
          v[q] = reinterpret_cast<const float4*>(grad + ((bag0 + r) * dv.T + t) * D)[i % (D / 4)];
        }
#pragma unroll
        for (int q = 0; q < PER; ++q) stage[q * kBlockThreads + threadIdx.x] = v[q];
      }
      __syncthreads();
      // the table's big rows, kBlockThreads at a time: their ranges in this stage are
      // listed in LDS with the rows of more than 4*GL occurrences first, and the row
      // groups take list entries in order (the longest sums start first)
      for (int64_t hc = h0; hc < h1; hc += kBlockThreads) {
        const int nr = (int)min<int64_t>(kBlockThreads, h1 - hc);
        if (threadIdx.x == 0) {
          cnt_s[0] = 0;  // rows with more than 4*GL occurrences in the stage
          cnt_s[1] = 0;  // list positions taken by those rows
          cnt_s[2] = 0;  // list positions taken by the others (after them)
          cnt_s[3] = 0;  // next list entry for a row group
        }
        __syncthreads();
        uint32_t r0 = 0, r1 = 0;
        bool heavy = false, carry = false;
        if ((int)threadIdx.x < nr) {
          const uint32_t* bb = w.bbound + (hc + threadIdx.x) * stride_b;
          r0 = bb[js];
          r1 = bb[js + 1];
          carry = bb[k * kStages] < r0;  // occurrences in an earlier stage of the block
          heavy = r1 - r0 > 4u * GL;
          if (heavy) atomicAdd(&cnt_s[0], 1u);
        }
        __syncthreads();
        if ((int)threadIdx.x < nr) {
          const uint32_t pos = heavy ? atomicAdd(&cnt_s[1], 1u) : cnt_s[0] + atomicAdd(&cnt_s[2], 1u);
          lrow[pos] = (uint32_t)threadIdx.x | (carry ? 0x80000000u : 0u);
          lr0[pos] = r0;
          lr1[pos] = r1;
        }
        __syncthreads();
        for (;;) {
          uint32_t e = 0;
          if (l == 0) e = atomicAdd(&cnt_s[3], 1u);
          e = __shfl(e, 0, GL);
          if ((int)e >= nr) break;
          const uint32_t le = lrow[e];
          const int64_t h = hc + (le & 0x7FFFFFFFu);
          const uint32_t i0 = lr0[e], i1 = lr1[e];
          if (i0 >= i1) continue;
          // the block sum goes on from the earlier stages' terms, or starts from -0,
          // the identity of IEEE addition: adding the first term gives exactly that term
          float* o = w.bpart + (h * (int64_t)w.max_nblk + k) * D + l * CL;
          float acc[CL];
#pragma unroll
          for (int c = 0; c < CL; ++c) acc[c] = (le >> 31) ? o[c] : -0.0f;
          // runs of 4*GL occurrences: lane l holds the bags (relative to the block) of
          // occurrences 4l .. 4l+3 of the run; occurrence j of the run is component j%4
          // of lane j/4.  Every occurrence in [i0, i1) lies in the block; indices past
          // i1 re-read the last one (a bag of the block, not added).
          uint32_t rnext[4];  // the next run's bags, loaded one run ahead
#pragma unroll
          for (int c = 0; c < 4; ++c) rnext[c] = sval[min(i0 + 4 * l + c, i1 - 1)];
          for (uint32_t ic = i0; ic < i1; ic += 4 * GL) {
            const int n = min(4 * GL, (int)(i1 - ic));
            uint32_t rv[4];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
              rv[c] = rnext[c] - (uint32_t)bag0;
              rnext[c] = sval[min(ic + 4 * GL + 4 * l + c, i1 - 1)];
            }
            const auto batch = [&](int j, int m) {  // occurrences j .. j+m-1 of the run, m <= U
              float x[U][CL];
#pragma unroll
              for (int q = 0; q < U; ++q) {
                // U is a multiple of 4 and j of U: the component is static
                uint32_t v;
                if constexpr (GL == 64) v = __builtin_amdgcn_readlane(rv[q % 4], (j + q) / 4);
                else v = __shfl(rv[q % 4], (j + q) / 4, GL);
                const float* r = sf + (size_t)v * D + l * CL;
#pragma unroll
                for (int c = 0; c < CL; ++c) x[q][c] = r[c];
              }
#pragma unroll
              for (int q = 0; q < U; ++q)
                if (q < m)
#pragma unroll
                  for (int c = 0; c < CL; ++c) acc[c] = acc[c] + x[q][c];
            };
            int j = 0;
            for (; j + U <= n; j += U) batch(j, U);  // full batches: no per-term test
            if (j < n) batch(j, n - j);
          }
#pragma unroll
          for (int c = 0; c < CL; ++c) o[c] = acc[c];
        }
        __syncthreads();  // every group is done with the list (and its sums) before it is rebuilt
      }
    }
  }
}

// [lo, hi) of the unique rows of table t (rows are sorted table-major).
__device__ __forceinline__ void table_rows(const Work& w, int t, int64_t& lo, int64_t& hi) {
  lo = w.tab_first[t];
  hi = w.tab_first[t + 1];
}

// tab_first[t] = first unique row of table t (>= t), tab_first[T] = number of unique rows.
// Also the statistics that follow from those ranges: the unique rows of each table, and,
// for a table without a cache, its bypasses (every row).  (Unique hits are counted by
// k_policy, inserts and the other bypasses too.)
// The first unique row with table >= t (rows are sorted table-major), searched by a whole
// wave: each round, lane l tests the l-th of 64 points spread over the remaining range,
// which shrinks 64-fold (4 dependent loads for 5M unique rows instead of 23 for a binary
// search).  Wave-uniform; every lane returns the result.
__device__ __forceinline__ int64_t first_row_of_table_wave(const Work& w, int64_t nU, int t) {
  const int lane = threadIdx.x & 63;
  int64_t a = 0, b = nU;  // the row lies in [a, b] (b: there is none)
  while (a < b) {
    const int64_t step = (b - a + 63) / 64;
    const int64_t m = a + (int64_t)lane * step;
    const uint64_t ge = __ballot(m >= b || w.utab[m] >= t);
    const int f = ge ? (int)__builtin_ctzll(ge) : 64;  // first probe at or past the row
    if (f == 0) break;  // the row is a
    const int64_t prev = a + (int64_t)(f - 1) * step;
    if (f < 64) b = min<int64_t>(b, a + (int64_t)f * step);
    a = prev + 1;
  }
  return a;
}

// One wave per table boundary t = 0 .. T.
__global__ __launch_bounds__(256) void k_tab_first(Dev dv, Work w, int T) {
  const int64_t nU = (int64_t)w.ctr[kCUnique];
  const int t = (int)(((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6);
  if (t > T) return;  // whole waves
  const int64_t lo = first_row_of_table_wave(w, nU, t);
  const int64_t hi = t < T ? first_row_of_table_wave(w, nU, t + 1) : nU;
  if ((threadIdx.x & 63) != 0) return;
  w.tab_first[t] = (int32_t)lo;
  if (t < T) {
    const int64_t n = hi - lo;
    unsigned long long* st = dv.stats + (int64_t)t * kNStat;
    st[kStUnique] = (unsigned long long)n;
    if (dv.desc[t].n_sets == 0) st[kStBypasses] = (unsigned long long)n;
  }
}

// chunk_span[c] = occurrences [x, y) of the sorted stream that chunk c sums, and
// big_rows[h] = the unique row of big row h (ubig holds the big rows' prefix count).
// Also, after the paired scan of the chunk counts and big-row flags, the chunk total and
// the big-row total, the latter also as ubig[nU] (read by the kernels after this one).
__global__ __launch_bounds__(256) void k_chunk_spans(Work w) {
  const int64_t nU = (int64_t)w.ctr[kCUnique];
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    const unsigned long long tot = w.ctr[kCScanTotal];
    w.ctr[kCChunks] = tot & 0xFFFFFFFFull;
    w.ctr[kCBig] = tot >> 32;
    w.ubig[nU] = (uint32_t)(tot >> 32);
  }
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < nU; u += stride) {
    const uint32_t n = w.nch[u];
    const uint32_t s0 = w.seg[u], s1 = w.seg[u + 1];
    if (s1 - s0 > kBlockAbove) w.big_rows[w.ubig[u]] = (int32_t)u;
    if (n == 0) continue;
    const int64_t c0 = w.chunk_base[u];
    for (uint32_t j = 0; j < n; ++j) {
      const uint32_t a = s0 + j * (uint32_t)kSumChunk;
      w.chunk_span[c0 + j] = make_uint2(a, min(a + (uint32_t)kSumChunk, s1));
    }
  }
}

template <int D, bool SPREAD>
__global__ __launch_bounds__(256) void k_partials(Dev dv, Work w, const uint32_t* __restrict__ sval,
                                                  const float* __restrict__ grad) {
  // the gradient sums run beside the eviction on the second stream and decide when the
  // row update can start: their waves issue first where they share a SIMD
  __builtin_amdgcn_s_setprio(3);
  constexpr int LPR = Geo<D>::LPR;
  constexpr int GPB = 256 / LPR;
  const int g = threadIdx.x & (LPR - 1);
  const int64_t nC = (int64_t)w.ctr[kCChunks];
  const int64_t nU = (int64_t)w.ctr[kCUnique];
  if (nC == 0) return;
  const XcdSplit xs(dv.T);
  const int64_t gx0 = xs.unit * GPB + threadIdx.x / LPR, gstride = xs.units * GPB;
  int64_t carry = 0;
  for (int seg = xs.xcd; seg < xs.segments(dv.T); seg += kXcds) {
    const int t = seg / xs.parts;
    int64_t ulo, uhi;
    table_rows(w, t, ulo, uhi);
    const int64_t clo_t = ulo < nU ? (int64_t)w.chunk_base[ulo] : nC;
    const int64_t chi_t = uhi < nU ? (int64_t)w.chunk_base[uhi] : nC;
    int64_t clo, chi;
    part_range(clo_t, chi_t, seg % xs.parts, xs.parts, clo, chi);
    const int64_t gx = SPREAD ? spread_start(gx0, gstride, chi - clo, carry) : gx0;
    if (clo + gx >= chi) continue;
    const GradRows gr = grad_rows<D>(grad, t, dv.T);
    // the next chunk's span is loaded one chunk ahead (clamped index, unconditional load)
    uint2 next = w.chunk_span[clo + gx];
    for (int64_t c = clo + gx; c < chi; c += gstride) {
      const uint2 sp = next;
      next = w.chunk_span[min<int64_t>(c + gstride, chi - 1)];
      float acc[8];
      chunk_sum<D>(sval, sp.x, sp.y, gr, g, acc);
      store_row<D>(w.partial + c * D, g, acc);
    }
  }
}

// ---- optimizer (FP32) -----------------------------------------------------------------------
// SGD: x = fma(-lr, g, x).  Row-wise Adagrad: S = halving-tree sum of g_j^2
// (a[j] += a[j + h] for h = D/2, ..., 1, the pairs of columns taken across or inside
// the lanes as the row layout places them), G += S * (1/D), r = lr / (sqrt(G) + eps),
// x = fma(-r, g, x).
template <int D>
__device__ __forceinline__ void apply_optimizer(const Dev& dv, float (&x)[8], const float (&gr)[8], float* acc,
                                                int g, float G_old) {
  constexpr int LPR = Geo<D>::LPR;
  if (dv.optimizer == 0) {
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = __builtin_fmaf(-dv.lr, gr[i], x[i]);
    return;
  }
  // the halving tree over the row's squares, in the lanes' column layout
  float a[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = gr[i] * gr[i];
  if constexpr (kSplit<D>) {
    // h = D/2 pairs element i with i + 4 of the same lane; h = D/4 .. 4 pairs lanes
    // g and g ^ (h/4); h = 2, 1 are inside the lane
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = a[i] + a[i + 4];
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = butterfly<LPR>(a[i], [](float p, float q) { return p + q; });
#pragma unroll
    for (int h = 2; h >= 1; h >>= 1)
#pragma unroll
      for (int i = 0; i < h; ++i) a[i] = a[i] + a[i + h];
  } else {
    // h = D/2 .. 8 pairs lanes g and g ^ (h/8); h = 4, 2, 1 are inside the lane
#pragma unroll
    for (int i = 0; i < 8; ++i) a[i] = butterfly<LPR>(a[i], [](float p, float q) { return p + q; });
#pragma unroll
    for (int h = 4; h >= 1; h >>= 1)
#pragma unroll
      for (int i = 0; i < h; ++i) a[i] = a[i] + a[i + h];
  }
  const float Gn = G_old + a[0] * (1.0f / (float)D);
  if (g == 0) *acc = Gn;
  const float rate = dv.lr / (__builtin_sqrtf(Gn) + dv.eps);
#pragma unroll
  for (int i = 0; i < 8; ++i) x[i] = __builtin_fmaf(-rate, gr[i], x[i]);
}

// A row's Adagrad accumulator: in the slot array while the row is cached, in its record
// otherwise (it moves with the row on an insert and an eviction).
__device__ __forceinline__ float load_G(const Dev& dv, const float* acc) {
  return dv.optimizer ? *acc : 0.0f;
}

// ---- replacement decision, one wave per touched set ------------------------------------------
struct PolicyLds {
  int32_t hitu[64];       // unique row that hit way w this step, or -1
  int32_t cand_u[64];     // candidates by rank
  long long cand_pv[64];
  int32_t vic_way[64];    // victims by rank
  long long vic_pv[64];
};

// Statistics of the sets a wave handles, accumulated while the table does not change.
struct PolicyStats {
  int t = -1;
  uint32_t ins = 0, byp = 0, ev = 0, em = 0, he = 0, hits = 0;
  __device__ void flush(unsigned long long* stats) {
    if (t < 0) return;
    unsigned long long* s = stats + (int64_t)t * kNStat;
    if (hits) atomicAdd(s + kStUniqueHits, (unsigned long long)hits);
    if (ins) atomicAdd(s + kStInserts, (unsigned long long)ins);
    if (byp) atomicAdd(s + kStBypasses, (unsigned long long)byp);
    if (ev) atomicAdd(s + kStEvictions, (unsigned long long)ev);
    if (em) atomicAdd(s + kStEmptyFills, (unsigned long long)em);
    if (he) atomicAdd(s + kStHitEvictions, (unsigned long long)he);
    ins = byp = ev = em = he = hits = 0;
  }
};

// G lanes per set (G >= assoc): a wave decides 64/G sets at once, each group of G
// lanes on its own run of consecutive sets.  Every cross-lane step (ballot, shuffle,
// LDS slot) stays inside the group, and every branch below is uniform over a group.
template <int G>
__global__ __launch_bounds__(256) void k_policy(Dev dv, Work w, uint32_t step) {
  __shared__ PolicyLds lds_all[4];
  PolicyLds& L = lds_all[threadIdx.x >> 6];
  constexpr int NG = 64 / G;
  const int lane = threadIdx.x & 63;
  const int gb = lane & ~(G - 1);  // the group's first lane
  const int l = lane & (G - 1);    // lane within the group
  const uint64_t gmask = G == 64 ? ~0ull : (((1ull << G) - 1) << gb);
  const uint64_t below = lanemask_lt() & gmask;
  const int A = dv.assoc;
  const bool lru = dv.policy == 0;
  const int64_t nS = (int64_t)w.ctr[kCSets];
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  // contiguous runs of sets per group, so that the table (and its statistics) rarely changes
  const int64_t ngroups = nwaves * NG, grp = wave0 * NG + lane / G;
  const int64_t per = (nS + ngroups - 1) / ngroups;
  const int64_t k0 = grp * per, k1 = min<int64_t>(k0 + per, nS);
  PolicyStats ps;  // meaningful in the group's lane 0
  for (int64_t k = k0; k < k1; ++k) {
    const int64_t u0 = w.set_first[k], u1 = w.set_first[k + 1];
    const int t = w.utab[u0];
    const TableDesc td = dv.desc[t];
    const int64_t r0 = (int64_t)w.urow[u0] - td.row_base;
    const int64_t sbase = td.slot_base + (r0 % td.n_sets) * A;

    if (t != ps.t) {
      if (l == 0) ps.flush(dv.stats);
      ps.t = t;
    }
    // residents that hit this step, and the number of missed rows
    L.hitu[lane] = -1;
    __builtin_amdgcn_wave_barrier();
    int64_t M = 0, H = 0;
    for (int64_t c = u0; c < u1; c += G) {
      const int64_t u = c + l;
      bool miss = false, hit = false;
      if (u < u1) {
        const int32_t sl = w.uslot[u];
        if (sl >= 0) {
          L.hitu[gb + (sl - sbase)] = (int32_t)u;
          hit = true;
        } else {
          miss = true;
        }
      }
      M += __popcll(__ballot(miss) & gmask);
      H += __popcll(__ballot(hit) & gmask);
    }
    __builtin_amdgcn_wave_barrier();
    if (l == 0) ps.hits += (uint32_t)H;
    if (M == 0) continue;

    // ways, their tags and priorities (empty = lowest)
    int32_t tg = -1;
    long long vpv = LLONG_MAX;
    if (l < A) {
      tg = dv.tag[sbase + l];
      vpv = tg < 0 ? LLONG_MIN : (lru ? (long long)dv.ts[sbase + l] : (long long)dv.cnt[td.row_base + tg]);
    }
    // lane k < n_ins: the k-th insert (unique row my_u) takes way my_way, displacing my_old
    // (-1 if the way was empty); my_hu is my_old's unique row if it was updated this step
    int my_way = 0;
    int32_t my_u = -1, my_old = -1, my_hu = -1;
    int n_ins = 0;

    if (A == 1 && lru) {
      // direct-mapped LRU: no priority test; the largest missed row ends in the way
      int64_t win = -1;
      for (int64_t c = u0; c < u1; c += G) {
        const int64_t u = c + l;
        const bool miss = u < u1 && w.uslot[u] < 0;
        const uint64_t m = __ballot(miss) & gmask;
        if (m) win = c + (63 - __clzll((unsigned long long)m)) - gb;
      }
      n_ins = 1;
      my_u = (int32_t)win;
      my_old = __shfl(tg, gb);
      my_hu = my_old >= 0 ? L.hitu[gb] : -1;
    } else {
      // victims ranked by (priority asc, way asc); every lane of the group runs the shuffles
      int vr = 0;
      for (int j = 0; j < A; ++j) {
        const long long pj = __shfl(vpv, gb + j);
        vr += (pj < vpv || (pj == vpv && j < l)) ? 1 : 0;
      }
      if (l < A) {
        L.vic_way[gb + vr] = l;
        L.vic_pv[gb + vr] = vpv;
      }
      // candidates ranked by (priority desc, row asc); only ranks < A matter
      int64_t K = M < A ? M : A;
      if (lru) {
        int64_t seen = 0;
        for (int64_t c = u0; c < u1 && seen < K; c += G) {
          const int64_t u = c + l;
          const bool miss = u < u1 && w.uslot[u] < 0;
          const uint64_t m = __ballot(miss) & gmask;
          const int64_t rank = seen + __popcll(m & below);
          if (miss && rank < K) {
            L.cand_u[gb + rank] = (int32_t)u;
            L.cand_pv[gb + rank] = (long long)step;
          }
          seen += __popcll(m);
        }
      } else {
        // the candidates in rank order, found one at a time as the largest key below the
        // previous one (keys are unique: they hold the row), for as long as the k-th
        // candidate beats the k-th victim; the first that does not ends the inserts
        __builtin_amdgcn_wave_barrier();
        unsigned long long prev = ~0ull;
        int64_t taken = 0;
        for (int64_t r = 0; r < K; ++r) {
          unsigned long long best = 0;
          int32_t bu = -1;
          for (int64_t c = u0 + l; c < u1; c += G) {
            const unsigned long long k = w.ukey[c];
            if (k < prev && k > best) {
              best = k;
              bu = (int32_t)c;
            }
          }
#pragma unroll
          for (int o = G / 2; o >= 1; o >>= 1) {
            const unsigned long long ob = __shfl_xor(best, o, G);
            const int32_t ou = __shfl_xor(bu, o, G);
            if (ob > best) {
              best = ob;
              bu = ou;
            }
          }
          const long long cpv = (long long)(best >> 32);
          if (best == 0 || !(cpv > L.vic_pv[gb + r])) break;
          if (l == 0) {
            L.cand_u[gb + r] = bu;
            L.cand_pv[gb + r] = cpv;
          }
          prev = best;
          taken = r + 1;
        }
        K = taken;  // every listed candidate beats its victim
      }
      __builtin_amdgcn_wave_barrier();
      // the k-th candidate takes the k-th victim while strictly higher; stop at the first failure
      const bool ok = l < K && L.cand_pv[gb + l] > L.vic_pv[gb + l];
      const uint64_t fail = __ballot(l < K && !ok) & gmask;
      n_ins = fail ? __ffsll((unsigned long long)fail) - 1 - gb : (int)K;
      my_way = l < n_ins ? L.vic_way[gb + l] : 0;
      my_old = __shfl(tg, gb + my_way);
      my_u = l < n_ins ? L.cand_u[gb + l] : -1;
      my_hu = (l < n_ins && my_old >= 0) ? L.hitu[gb + my_way] : -1;
      __builtin_amdgcn_wave_barrier();
    }
    if (l < n_ins) {
      w.uact[my_u] = kActInsert;
      w.udest[my_u] = (int32_t)(sbase + my_way);
      w.uvic_row[my_u] = my_old;
      w.uvic_u[my_u] = my_hu;
      if (my_hu >= 0) w.uact[my_hu] = kActDone;  // handled by the row that displaces it
    }
    const uint32_t n_valid = (uint32_t)__popcll(__ballot(l < n_ins && my_old >= 0) & gmask);
    const uint32_t n_hitev = (uint32_t)__popcll(__ballot(l < n_ins && my_hu >= 0) & gmask);
    if (l == 0 && n_hitev) atomicAdd(&w.ctr[kCHitEv], (unsigned long long)n_hitev);
    if (l == 0) {
      ps.ins += (uint32_t)n_ins;
      ps.byp += (uint32_t)(M - n_ins);
      ps.ev += n_valid;
      ps.em += (uint32_t)n_ins - n_valid;
      ps.he += n_hitev;
    }
  }
  if (l == 0) ps.flush(dv.stats);
}

// ---- displaced residents -> T -----------------------------------------------------------------
// UPDATED = false: residents not updated this step (their FP32 way is quantized as it
// is; no merged gradient needed, so this runs beside the gradient sums);
// UPDATED = true: residents updated this step and then displaced (LFU or direct-mapped;
// their merged gradient is applied first), after the gradient sums.
template <int D, int BITS, bool SB16, bool UPDATED>
__global__ __launch_bounds__(256) void k_evict(Dev dv, Work w, const uint32_t* __restrict__ sval,
                                               const float* __restrict__ grad, uint32_t step) {
  if (UPDATED && w.ctr[kCHitEv] == 0) return;
  constexpr int LPR = Geo<D>::LPR;
  constexpr int GPW = 64 / LPR;  // row groups per wave
  const int lane = threadIdx.x & 63;
  const int g = lane & (LPR - 1), grp = lane / LPR;
  const bool sr = dv.rounding != 0;
  const XcdSplit xs(dv.T, true);
  // each wave takes windows of 64 consecutive unique rows: one coalesced load of each
  // row's decision, a ballot of the rows that displace a resident, then those rows
  // GPW at a time (one per row group), so no group idles on rows without a victim
  const int64_t wv = xs.unit * (blockDim.x / 64) + threadIdx.x / 64, wstride = xs.units * (blockDim.x / 64);
  for (int seg = xs.xcd; seg < xs.segments(dv.T); seg += kXcds) {
    const int t = seg / xs.parts;
    int64_t tlo, thi, lo, hi;
    table_rows(w, t, tlo, thi);
    part_range(tlo, thi, seg % xs.parts, xs.parts, lo, hi);
    const TableDesc td = dv.desc[t];
    if (td.n_sets == 0) continue;
    for (int64_t w0 = lo + wv * 64; w0 < hi; w0 += wstride * 64) {
      const int64_t u = w0 + lane;
      int32_t dst = 0, vrow = -1, vu = -1;
      bool take = false;
      if (u < hi) {
        const int32_t act = w.uact[u];
        dst = w.udest[u];
        vrow = w.uvic_row[u];
        vu = w.uvic_u[u];
        take = act == kActInsert && vrow >= 0 && (vu >= 0) == UPDATED;
      }
      uint64_t mask = __ballot(take);
      while (mask) {
        // the grp-th set bit of mask is this group's row (none when fewer remain)
        uint64_t m = mask;
        for (int k = 0; k < grp && m; ++k) m &= m - 1;
        const int src = m ? __builtin_ctzll(m) : 0;
        const bool mine = m != 0;
        for (int k = 0; k < GPW && mask; ++k) mask &= mask - 1;
        const int32_t e_dst = __shfl(dst, src), e_vrow = __shfl(vrow, src), e_vu = __shfl(vu, src);
        if (!mine) continue;
        const int64_t vgrow = td.row_base + e_vrow;
        uint8_t* vrec = rec_of<D, BITS, SB16>(dv, vgrow);
        float xv[8];
        load_row_nt<D>(dv.crow + (int64_t)e_dst * D, g, xv);
        // the displaced row's accumulator leaves the slot for its record (before the
        // insert that takes the slot writes its own there)
        float* acc = dv.optimizer ? acc_of<D, BITS, SB16>(dv, vgrow, vrec) : nullptr;
        if (UPDATED) {
          // the displaced resident was updated this step (LFU): its new value goes to T
          const float Gv = dv.optimizer ? dv.acc_slot[e_dst] : 0.0f;
          float gv[8];
          merged_grad<D>(w, sval, grad_rows<D>(grad, t, dv.T), e_vu, g, gv);
          apply_optimizer<D>(dv, xv, gv, acc, g, Gv);
        } else if (dv.optimizer && g == 0) {
          *acc = dv.acc_slot[e_dst];
        }
        quantize_store<D, BITS, SB16>(xv, g, vrec, sr, dv.seed, step, (uint32_t)t, (uint32_t)e_vrow);
      }
    }
  }
}

// ---- per unique row: optimizer and write-back ------------------------------------------------
// The inputs of k_update for unique row u, packed into one 16-byte word once the
// replacement decisions are final (one load per row instead of eight):
//   x = global row;  y = cache slot (a hit: its way; an insert: the way it takes);
//   z = the bag of its one occurrence if the row has one lookup, else its first
//       occurrence in the sorted stream;  w = lookups | kind << 30 (lookups < 2^30).
// A row with one lookup (most rows) then loads its gradient row together with its
// own row and accumulator, one dependent load fewer.
constexpr uint32_t kKindHit = 0, kKindInsert = 1, kKindBypass = 2, kKindDone = 3;
constexpr uint32_t kLookupMask = (1u << 30) - 1;

__global__ __launch_bounds__(256) void k_pack_meta(Work w, const uint32_t* __restrict__ sval) {
  const int64_t nU = (int64_t)w.ctr[kCUnique];
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < nU; u += stride) {
    const int32_t act = w.uact[u];
    const uint32_t s0 = w.seg[u], n = w.seg[u + 1] - s0;
    const uint32_t kind = act == kActHitStay ? kKindHit
                          : act == kActInsert ? kKindInsert
                          : act == kActBypass ? kKindBypass
                                              : kKindDone;
    const int32_t cs = kind == kKindHit ? w.uslot[u] : kind == kKindInsert ? w.udest[u] : -1;
    const uint32_t z = n == 1 ? sval[s0] : s0;
    w.umeta[u] = make_uint4((uint32_t)w.urow[u], (uint32_t)cs, z, n | (kind << 30));
  }
}

// SPREAD: small steps (few rows per table), whose segments spread over all row groups
// (spread_start); large steps keep the plain assignment, which needs fewer registers.
// At d >= 128 the kernel is held to 96 VGPRs (5 waves per SIMD), spilling a few: with
// 97-102 VGPRs (4 waves) the 128-column INT2 and FP16 tables took 1950 and 1916 us
// (1767, 1765 held); INT4 and the 256-column INT8 table are unchanged by it.
template <int D, int BITS, bool SB16, bool SPREAD>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(kSplit<D> ? 5 : 1)))
void k_update(Dev dv, Work w, const uint32_t* __restrict__ sval, const float* __restrict__ grad, uint32_t step) {
  constexpr int LPR = Geo<D>::LPR;
  constexpr int GPB = 256 / LPR;
  const int g = threadIdx.x & (LPR - 1);
  const bool sr = dv.rounding != 0;
  const XcdSplit xs(dv.T, true);
  const int64_t gx0 = xs.unit * GPB + threadIdx.x / LPR, gstride = xs.units * GPB;
  int64_t carry = 0;
  for (int seg = xs.xcd; seg < xs.segments(dv.T); seg += kXcds) {
    const int t = seg / xs.parts;
    int64_t tlo, thi, lo, hi;
    table_rows(w, t, tlo, thi);
    part_range(tlo, thi, seg % xs.parts, xs.parts, lo, hi);
    const TableDesc td = dv.desc[t];
    const GradRows gtab = grad_rows<D>(grad, t, dv.T);
    const int64_t gx = SPREAD ? spread_start(gx0, gstride, hi - lo, carry) : gx0;
    if (lo + gx >= hi) continue;
    uint4 next = w.umeta[lo + gx];
    for (int64_t u = lo + gx; u < hi; u += gstride) {
      const uint4 m = next;
      // the next row's inputs are in flight while this row is handled (the index is
      // clamped so that the load is unconditional; the last one is not used)
      next = w.umeta[min<int64_t>(u + gstride, hi - 1)];
      const uint32_t kind = m.w >> 30, n = m.w & kLookupMask;
      if (kind == kKindDone) continue;
      const int64_t grow = m.x;
      uint8_t* rec = rec_of<D, BITS, SB16>(dv, grow);
      const bool hit = kind == kKindHit;
      // the accumulator: in the slot of a hit, in the record of a miss; an insert takes it
      // to the slot it fills, a bypass leaves it in the record
      float* acc = nullptr;
      float* acc_out = nullptr;
      if (dv.optimizer) {
        acc = hit ? dv.acc_slot + (int32_t)m.y : acc_of<D, BITS, SB16>(dv, grow, rec);
        acc_out = kind == kKindBypass ? acc : dv.acc_slot + (int32_t)m.y;
      }
      const bool big = n > kBlockAbove;
      // first level of loads: the row, its accumulator, and the gradient row (one
      // lookup) or the first occurrence values (2 to kSumChunk lookups)
      float x[8], gr[8];
      // both loads unconditional (a row with more lookups re-reads bag 0's gradient
      // row; the position index is clamped into the row's occurrences, or 0)
      load_row<D>(gtab.row(n == 1 ? m.z : 0u), g, gr);
      const uint32_t myv0 = sval[n == 1 ? 0u : m.z + min<uint32_t>((uint32_t)g, n - 1)];
      CodeWords<BITS> cw;
      SbWords<SB16> sbw;
      if (hit) {
        load_row_nt<D>(dv.crow + (int64_t)(int32_t)m.y * D, g, x);
      } else {
        if constexpr (kSplit<D>) cw = load_split_code_words<D, BITS, true>(rec, g);
        else cw = load_code_words<BITS, true>(rec, g);
        sbw = load_sb_words<D, BITS, SB16>(rec);
      }
      // the accumulator is loaded by lane 0 alone and passed to the group by a lane move
      // (every lane loading it: 1865 us against 1767); the pointers are formed here (formed
      // where the accumulator is stored instead: 1866 us)
      float G_old = g == 0 ? load_G(dv, acc) : 0.0f;
      if (big) load_row<D>(w.bpart + (int64_t)w.ubig[u] * w.max_nblk * D, g, gr);
      else if (n > (uint32_t)kSumChunk)
        fold_chunks<D>(w.partial, w.chunk_base[u], (n + kSumChunk - 1) / kSumChunk, g, gr);
      else if (n > 1) sum_occ<D>(sval, m.z, m.z + n, gtab, g, gr, myv0, true);
      if (!hit) {
        float sc, bi;
        decode_sb<SB16>(sbw, sc, bi);
        dequant8<BITS>(cw, sc, bi, x);
      }
      G_old = __shfl(G_old, 0, LPR);
      apply_optimizer<D>(dv, x, gr, acc_out, g, G_old);
      if (hit || kind == kKindInsert) {
        const int64_t cs = (int32_t)m.y;
        store_row_nt<D>(dv.crow + cs * D, g, x);
        if (!hit && g == 0) {
          dv.tag[cs] = (int32_t)(grow - td.row_base);
          if (dv.policy == 0) dv.ts[cs] = (int32_t)step;
        }
      } else {
        quantize_store<D, BITS, SB16>(x, g, rec, sr, dv.seed, step, (uint32_t)t, (uint32_t)(grow - td.row_base));
      }
    }
  }
}

// ---- one training step ----------------------------------------------------------------------
hipError_t launch_backward(const Dev& d, const Work& w, const int32_t* idx, int64_t L, const int32_t* off, int32_t B,
                           const float* grad, uint64_t step64, int key_bits, int seg_passes, bool decay,
                           const hipEvent_t* update_events, const SideStream& side, hipStream_t s) {
  const uint32_t step = (uint32_t)step64;
  k_bwd_begin<<<1, 256, 0, s>>>(d, w.ctr, L);
  // offsets first: a rejected call must not reach the decay either
  const int64_t nbags = (int64_t)d.T * B;
  k_check_offsets<<<grid_for(nbags, 2048), 256, 0, s>>>(d, off, nbags, L, w.ctr);
  if (decay && d.cnt) k_decay<<<grid_for(d.total_rows), 256, 0, s>>>(d.cnt, d.total_rows, w.ctr);
  const int passes = (key_bits + 7) / 8;
  int in_B = 0;
  const SortScratch ss{w.sort_small, w.sort_small + kMaxPasses * 256, w.sort_small + 2 * kMaxPasses * 256,
                       {w.sort_status[0], w.sort_status[1]}};
  hipError_t e;
  if (seg_passes > 0 && seg_passes < passes && L > 0) {
    // per-table sort: the expansion also counts the digits
    const size_t TT = (size_t)d.T * kMaxPasses * 256;
    const SegSort sg{w.sort_seg, w.sort_seg + (d.T + 1), w.sort_seg + 2 * (d.T + 1), w.sort_seg + 2 * (d.T + 1) + TT};
    ExpandHist eh;
    e = seg_begin(L, seg_passes, off, B, d.T, d.key_base, w.ctr, ss, sg, &eh, s);
    if (e == hipSuccess) e = launch_expand(d, idx, L, off, B, w.keysA, w.valsA, w.ctr, &eh, s);
    if (e == hipSuccess)
      e = sort_pairs_segmented(w.keysA, w.valsA, w.keysB, w.valsB, L, seg_passes, off, B, d.T, d.key_base, w.ctr,
                               ss, sg, d.err, &in_B, s);
  } else {
    e = launch_expand(d, idx, L, off, B, w.keysA, w.valsA, w.ctr, nullptr, s);
    if (e == hipSuccess) e = sort_pairs(w.keysA, w.valsA, w.keysB, w.valsB, L, passes, ss, d.err, &in_B, s);
  }
  if (e != hipSuccess) return e;
  const uint32_t* sk = in_B ? w.keysB : w.keysA;
  const uint32_t* sv = in_B ? w.valsB : w.valsA;
  e = launch_unique(d, sk, L, w.tile_cnt, w.tile_pre, w.thread_pre, w.uniq_key, w.seg, w.set_first, w.utab,
                    w.ctr, s);
  if (e != hipSuccess) return e;
  const auto grid = [](auto kernel) { return resident_grid(reinterpret_cast<const void*>(kernel)); };
  k_probe<<<grid(k_probe), 256, 0, s>>>(d, w, step);
  k_tab_first<<<(unsigned)((64 * (int64_t)(d.T + 1) + 255) / 256), 256, 0, s>>>(d, w, d.T);
  e = scan_exclusive_pair(w.nch, w.ubig, w.chunk_base, w.ubig, L, w.ctr + kCUnique, w.part, w.ctr + kCScanTotal, s);
  if (e != hipSuccess) return e;
  k_chunk_spans<<<grid(k_chunk_spans), 256, 0, s>>>(w);
  // bag blocks of NB = kBlockFloats/d bags (a power of two) for the big rows
  const int nb_shift = __builtin_ctz((unsigned)(kBlockFloats / d.dim));
  const int stage_shift = nb_shift - __builtin_ctz((unsigned)kStages);
  const int nblk = (int)(((int64_t)B + (kBlockFloats / d.dim) - 1) / (kBlockFloats / d.dim));
  // a small step spreads its tables' rows over all row groups (a larger one has more rows
  // per table than groups anyway, and keeps the kernels with fewer registers)
  const bool spread = L < kSpreadBelow;
  if (nblk > w.max_nblk) return hipErrorInvalidValue;
  if (nblk > 0) k_block_bounds<<<grid(k_block_bounds), 256, 0, s>>>(w, sv, stage_shift, nblk);
  return dispatch_row(d.dim, d.bits, d.sb16, [&]<int D, int BITS, bool SB16>() -> hipError_t {
    // replacement decisions and the write-back of residents displaced without an update
    // on the side stream, the merged gradients on `s`; joined before the updates (the
    // packing of the row update's inputs on the side stream, after the decisions: the
    // block sums beside the eviction 1111 -> 1434 us)
    const bool cached = d.total_slots > 0;
    if (cached) {
      hipError_t e2 = hipEventRecord(side.fork, s);
      if (e2 == hipSuccess) e2 = hipStreamWaitEvent(side.s, side.fork, 0);
      if (e2 != hipSuccess) return e2;
      if (d.assoc <= 16) k_policy<16><<<grid(k_policy<16>), 256, 0, side.s>>>(d, w, step);
      else if (d.assoc <= 32) k_policy<32><<<grid(k_policy<32>), 256, 0, side.s>>>(d, w, step);
      else k_policy<64><<<grid(k_policy<64>), 256, 0, side.s>>>(d, w, step);
      k_evict<D, BITS, SB16, false><<<grid(k_evict<D, BITS, SB16, false>), 256, 0, side.s>>>(d, w, sv, grad, step);
      e2 = hipEventRecord(side.join, side.s);
      if (e2 != hipSuccess) return e2;
    }
    if (spread) k_partials<D, true><<<grid(k_partials<D, true>), 256, 0, s>>>(d, w, sv, grad);
    else k_partials<D, false><<<grid(k_partials<D, false>), 256, 0, s>>>(d, w, sv, grad);
    if (nblk > 0) {
      k_block_partials<D><<<resident_grid(reinterpret_cast<const void*>(k_block_partials<D>), kBlockThreads),
                            kBlockThreads, 0, s>>>(d, w, sv, grad, B, nblk);
      k_block_fold<D><<<grid(k_block_fold<D>), 256, 0, s>>>(w, nblk);
    }
    if (cached) {
      const hipError_t e2 = hipStreamWaitEvent(s, side.join, 0);
      if (e2 != hipSuccess) return e2;
      // a resident hit this step is displaced only under LFU or in a direct-mapped LRU
      // cache (under LRU a hit takes the step's stamp, which no candidate exceeds)
      if (d.policy != 0 || d.assoc == 1)
        k_evict<D, BITS, SB16, true><<<grid(k_evict<D, BITS, SB16, true>), 256, 0, s>>>(d, w, sv, grad, step);
    }
    k_pack_meta<<<grid(k_pack_meta), 256, 0, s>>>(w, sv);
    if (update_events) {
      const hipError_t e2 = hipEventRecord(update_events[0], s);
      if (e2 != hipSuccess) return e2;
    }
    if (spread) k_update<D, BITS, SB16, true><<<grid(k_update<D, BITS, SB16, true>), 256, 0, s>>>(d, w, sv, grad, step);
    else k_update<D, BITS, SB16, false><<<grid(k_update<D, BITS, SB16, false>), 256, 0, s>>>(d, w, sv, grad, step);
    if (update_events) {
      const hipError_t e2 = hipEventRecord(update_events[1], s);
      if (e2 != hipSuccess) return e2;
    }
    return hipGetLastError();
  });
}

}  // namespace embc
