// Backward + sparse update of one step (Sec. 3 update operator, Alg. 2, Sec. 5.1 de-dup).
//
// After the sort (k_sort.hip) the lookups are grouped by row, the rows by set:
//   k_probe     per unique row: residency (slot or miss), LRU stamp / LFU count update
//   k_partials  chunk sums (64 lookups each) of the merged gradient of rows with > 64 lookups
//   k_policy    per touched set, one wave (one lane per way): which missed rows enter the
//               cache and which resident each of them displaces (decisions only)
//   k_hot_fold  per row with > kFoldDirect chunk sums, one workgroup: its chunk sums folded
//               left to right through LDS; the result replaces the row's first chunk sum
//               (rows with fewer chunks are folded by the kernel that consumes them)
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

// Per-table counts of the active lanes (tables may differ across lanes): one atomic
// for the lanes sharing the first active lane's table, one per lane for the others.
// Must be called by all 64 lanes.
__device__ __forceinline__ void wave_stat_add(unsigned long long* stats, int t, int field, uint32_t v, bool active) {
  const uint64_t act = __ballot(active && v != 0);
  if (!act) return;
  const int leader = __ffsll((unsigned long long)act) - 1;
  const int t0 = __shfl(t, leader);
  const bool same = active && t == t0;
  uint32_t s = same ? v : 0u;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o);
  const int lane = threadIdx.x & 63;
  if (lane == leader && s) atomicAdd(&stats[(int64_t)t0 * kNStat + field], (unsigned long long)s);
  if (active && !same && v) atomicAdd(&stats[(int64_t)t * kNStat + field], (unsigned long long)v);
}

__global__ void k_chunks_total(unsigned long long* ctr) { ctr[kCChunks] = ctr[kCScanTotal] & 0xFFFFFFFFull; }

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

// LFU decay: every count halved.
__global__ __launch_bounds__(256) void k_decay(int32_t* __restrict__ cnt, int64_t n) {
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
    bool nocache = false;
    if (act) {
      const uint32_t key = w.uniq_key[u];
      t = table_of_key(dv.key_base, dv.T, key);
      const TableDesc td = dv.desc[t];
      const int64_t local = (int64_t)key - td.key_base;
      int64_t r = local;
      if (td.n_sets > 0) r = (local % td.Q) * td.n_sets + local / td.Q;
      nocache = td.n_sets == 0;
      const int64_t grow = td.row_base + r;
      const uint32_t count = w.seg[u + 1] - w.seg[u];
      slot = probe_slot(dv, td, (int32_t)r);
      w.urow[u] = (int32_t)grow;
      w.utab[u] = t;
      w.uslot[u] = slot;
      w.uact[u] = slot >= 0 ? kActHitStay : kActBypass;
      w.nch[u] = count > (uint32_t)kSumChunk ? (count + kSumChunk - 1) / kSumChunk : 0u;
      if (dv.policy == 0) {
        if (slot >= 0) dv.ts[slot] = (int32_t)step;
      } else {
        const int64_t c = (int64_t)dv.cnt[grow] + count;
        dv.cnt[grow] = c > 0x7FFFFFFF ? 0x7FFFFFFF : (int32_t)c;
      }
    }
    wave_stat_add(dv.stats, t, kStUnique, 1u, act);
    wave_stat_add(dv.stats, t, kStUniqueHits, slot >= 0 ? 1u : 0u, act);
    wave_stat_add(dv.stats, t, kStBypasses, nocache ? 1u : 0u, act);
  }
}

// ---- merged gradient ----------------------------------------------------------------------
// Left-to-right FP32 sum of the gradient rows of occurrences [i0, i1) of the sorted
// stream (i0 < i1), seeded with the first.  Lane j of the group preloads the row
// index of occurrence j of each chunk of LPR occurrences (for the first chunk the
// caller may pass them in, myv0); U rows are loaded before they are added in order.
template <int D>
__device__ __forceinline__ void sum_occ(const uint32_t* __restrict__ sval, int64_t i0, int64_t i1,
                                        const float* __restrict__ grad, int g, float (&acc)[8],
                                        uint32_t myv0 = 0u, bool have0 = false) {
  constexpr int LPR = Geo<D>::LPR, CPL = 8, U = kUnroll;
  bool first = true;
  for (int64_t ic = i0; ic < i1; ic += LPR) {
    const int n = (int)min<int64_t>(LPR, i1 - ic);
    // the first chunk's values may have been loaded by the caller (have0)
    const uint32_t myv = (have0 && ic == i0) ? myv0 : (g < n ? sval[ic + g] : 0u);
    int j = 0;
    if (first) {
      load_frow8(grad + (int64_t)__shfl(myv, 0, LPR) * D, g, acc);
      first = false;
      j = 1;
    }
    for (; j + U <= n; j += U) {
      float x[U][CPL];
#pragma unroll
      for (int q = 0; q < U; ++q) load_frow8(grad + (int64_t)__shfl(myv, j + q, LPR) * D, g, x[q]);
#pragma unroll
      for (int q = 0; q < U; ++q)
#pragma unroll
        for (int k = 0; k < CPL; ++k) acc[k] = acc[k] + x[q][k];
    }
    for (; j < n; ++j) {
      float x[CPL];
      load_frow8(grad + (int64_t)__shfl(myv, j, LPR) * D, g, x);
#pragma unroll
      for (int k = 0; k < CPL; ++k) acc[k] = acc[k] + x[k];
    }
  }
}

constexpr int kChunkUnroll = 4;  // gradient rows in flight per row group in a chunk sum

// Sum of one chunk (occurrences [i0, i1) of the sorted stream, 0 < i1 - i0 <= 64),
// left to right, seeded with the first.  The occurrence values of the next LPR
// occurrences are loaded while the current ones are summed, U gradient rows are in
// flight at a time, and a row listed more than once in one bag (adjacent occurrences
// with the same gradient row) adds the row already in registers instead of loading it
// again (same operands, same sums).
template <int D>
__device__ __forceinline__ void chunk_sum(const uint32_t* __restrict__ sval, int64_t i0, int64_t i1,
                                          const float* __restrict__ grad, int g, float (&acc)[8]) {
  constexpr int LPR = Geo<D>::LPR, CPL = 8, U = kChunkUnroll;
  bool first = true;
  uint32_t pv = 0xFFFFFFFFu;  // gradient row of the last occurrence added (none yet)
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
        if (fresh[q]) load_frow8(grad + (int64_t)v[q] * D, g, x[q]);
      }
#pragma unroll
      for (int q = 0; q < U; ++q) {
        if (j + q < n) {
          if (!fresh[q]) {
#pragma unroll
            for (int k = 0; k < CPL; ++k) x[q][k] = last[k];
          }
          if (first) {
#pragma unroll
            for (int k = 0; k < CPL; ++k) acc[k] = x[q][k];
            first = false;
          } else {
#pragma unroll
            for (int k = 0; k < CPL; ++k) acc[k] = acc[k] + x[q][k];
          }
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
  load_frow8(partial + c0 * D, g, acc);
  uint32_t j = 1;
  for (; j + U <= n; j += U) {
    float x[U][8];
#pragma unroll
    for (int q = 0; q < U; ++q) load_frow8(partial + (c0 + j + q) * D, g, x[q]);
#pragma unroll
    for (int q = 0; q < U; ++q)
#pragma unroll
      for (int k = 0; k < 8; ++k) acc[k] = acc[k] + x[q][k];
  }
  for (; j < n; ++j) {
    float x[8];
    load_frow8(partial + (c0 + j) * D, g, x);
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] = acc[k] + x[k];
  }
}

// Merged gradient of unique row u from its lookups (<= 64), its chunk sums (<=
// kFoldDirect of them) or the fold of its chunk sums left by k_hot_fold in its
// first chunk slot.
template <int D>
__device__ __forceinline__ void merged_grad(const Work& w, const uint32_t* __restrict__ sval,
                                            const float* __restrict__ grad, int64_t u, int g, float (&acc)[8]) {
  const uint32_t n = w.nch[u];
  if (n == 0) sum_occ<D>(sval, w.seg[u], w.seg[u + 1], grad, g, acc);
  else if (n <= kFoldDirect) fold_chunks<D>(w.partial, w.chunk_base[u], n, g, acc);
  else load_frow8(w.partial + (int64_t)w.chunk_base[u] * D, g, acc);
}

// Fold of the chunk sums of each row with more than kFoldDirect of them: acc = p0 +
// p1 + ... left to right, per column, into the row's first chunk slot.  One workgroup
// per row (from the list k_chunk_spans builds): all threads stage R chunk sums in LDS,
// load the next R into registers, and one thread per column folds the staged ones.
template <int D>
__global__ __launch_bounds__(256) void k_hot_fold(Work w) {
  constexpr int R = 8192 / D < 256 ? 8192 / D : 256;  // chunk rows per LDS round (32 KiB)
  constexpr int PER = R * D / 4 / 256;                 // float4 per thread and round
  __shared__ float4 stage[R * D / 4];
  const int64_t nl = (int64_t)w.ctr[kCLongRows];
  const int tid = threadIdx.x;
  for (int64_t h = blockIdx.x; h < nl; h += gridDim.x) {
    const int64_t u = w.long_rows[h];
    const int64_t c0 = w.chunk_base[u];
    const int64_t nch = w.nch[u];
    const float4* src = reinterpret_cast<const float4*>(w.partial + c0 * D);
    const int64_t n4 = nch * (D / 4);
    // loads past the row's last chunk sum re-read its last element (kept branch-free,
    // so that all PER loads are in flight together); those staged values are not folded
    float nxt[PER][4];
    const auto fetch = [&](int64_t first) {
#pragma unroll
      for (int k = 0; k < PER; ++k) {
        const float4 v = src[min<int64_t>(first + tid + k * 256, n4 - 1)];
        nxt[k][0] = v.x; nxt[k][1] = v.y; nxt[k][2] = v.z; nxt[k][3] = v.w;
      }
    };
    fetch(0);
    float acc = 0.0f;
    for (int64_t r0 = 0; r0 < nch; r0 += R) {
      const int rn = (int)min<int64_t>(R, nch - r0);
      __syncthreads();  // the previous round's fold is done with `stage`
#pragma unroll
      for (int k = 0; k < PER; ++k) stage[tid + k * 256] = make_float4(nxt[k][0], nxt[k][1], nxt[k][2], nxt[k][3]);
      __syncthreads();
      fetch((r0 + R) * (D / 4));
      if (tid < D) {
        const float* st = reinterpret_cast<const float*>(stage) + tid;
        int r = 0;
        if (r0 == 0) {
          acc = st[0];
          r = 1;
        }
        for (; r + 8 <= rn; r += 8) {
          float v[8];
#pragma unroll
          for (int k = 0; k < 8; ++k) v[k] = st[(r + k) * D];
#pragma unroll
          for (int k = 0; k < 8; ++k) acc = acc + v[k];
        }
        for (; r < rn; ++r) acc = acc + st[r * D];
      }
    }
    if (tid < D) w.partial[c0 * D + tid] = acc;
  }
}

// [lo, hi) of the unique rows of table t (rows are sorted table-major).
__device__ __forceinline__ void table_rows(const Work& w, int t, int64_t& lo, int64_t& hi) {
  lo = w.tab_first[t];
  hi = w.tab_first[t + 1];
}

// tab_first[t] = first unique row of table t (>= t), tab_first[T] = number of unique rows.
__global__ void k_tab_first(Work w, int T) {
  const int64_t nU = (int64_t)w.ctr[kCUnique];
  for (int t = blockIdx.x * blockDim.x + threadIdx.x; t <= T; t += gridDim.x * blockDim.x) {
    int64_t a = 0, b = nU;
    while (a < b) {
      const int64_t m = (a + b) >> 1;
      if (w.utab[m] < t) a = m + 1; else b = m;
    }
    w.tab_first[t] = (int32_t)a;
  }
}

// chunk_span[c] = occurrences [x, y) of the sorted stream that chunk c sums; rows with
// more than kFoldDirect chunks are listed for k_hot_fold (in any order).
__global__ __launch_bounds__(256) void k_chunk_spans(Work w) {
  const int64_t nU = (int64_t)w.ctr[kCUnique];
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < nU; u += stride) {
    const uint32_t n = w.nch[u];
    if (n == 0) continue;
    const int64_t c0 = w.chunk_base[u];
    const uint32_t s0 = w.seg[u], s1 = w.seg[u + 1];
    for (uint32_t j = 0; j < n; ++j) {
      const uint32_t a = s0 + j * (uint32_t)kSumChunk;
      w.chunk_span[c0 + j] = make_uint2(a, min(a + (uint32_t)kSumChunk, s1));
    }
    if (n > kFoldDirect) w.long_rows[atomicAdd(&w.ctr[kCLongRows], 1ull)] = (int32_t)u;
  }
}

template <int D>
__global__ __launch_bounds__(256) void k_partials(Dev dv, Work w, const uint32_t* __restrict__ sval,
                                                  const float* __restrict__ grad) {
  constexpr int LPR = Geo<D>::LPR;
  constexpr int GPB = 256 / LPR;
  const int g = threadIdx.x & (LPR - 1);
  const int64_t nC = (int64_t)w.ctr[kCChunks];
  const int64_t nU = (int64_t)w.ctr[kCUnique];
  if (nC == 0) return;
  const XcdSplit xs(dv.T);
  const int64_t gx = xs.unit * GPB + threadIdx.x / LPR, gstride = xs.units * GPB;
  for (int seg = xs.xcd; seg < xs.segments(dv.T); seg += kXcds) {
    const int t = seg / xs.parts;
    int64_t ulo, uhi;
    table_rows(w, t, ulo, uhi);
    const int64_t clo_t = ulo < nU ? (int64_t)w.chunk_base[ulo] : nC;
    const int64_t chi_t = uhi < nU ? (int64_t)w.chunk_base[uhi] : nC;
    int64_t clo, chi;
    part_range(clo_t, chi_t, seg % xs.parts, xs.parts, clo, chi);
    if (clo + gx >= chi) continue;
    // the next chunk's span is loaded one chunk ahead (clamped index, unconditional load)
    uint2 next = w.chunk_span[clo + gx];
    for (int64_t c = clo + gx; c < chi; c += gstride) {
      const uint2 sp = next;
      next = w.chunk_span[min<int64_t>(c + gstride, chi - 1)];
      float acc[8];
      chunk_sum<D>(sval, sp.x, sp.y, grad, g, acc);
      store_frow8(w.partial + c * D, g, acc);
    }
  }
}

// ---- optimizer (FP32) -----------------------------------------------------------------------
// SGD: x = fma(-lr, g, x).  Row-wise Adagrad: S = halving-tree sum of g_j^2
// (a[j] += a[j + h] for h = D/2, ..., 1: across lanes g ^ (h/8) while h >= 8, then
// inside the lane), G += S * (1/D), r = lr / (sqrt(G) + eps), x = fma(-r, g, x).
template <int D>
__device__ __forceinline__ void apply_optimizer(const Dev& dv, float (&x)[8], const float (&gr)[8], int64_t grow,
                                                int g, float G_old) {
  constexpr int LPR = Geo<D>::LPR;
  if (dv.optimizer == 0) {
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = __builtin_fmaf(-dv.lr, gr[i], x[i]);
    return;
  }
  float a[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = gr[i] * gr[i];
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = butterfly<LPR>(a[i], [](float p, float q) { return p + q; });
#pragma unroll
  for (int h = 4; h >= 1; h >>= 1)
#pragma unroll
    for (int i = 0; i < h; ++i) a[i] = a[i] + a[i + h];
  const float Gn = G_old + a[0] * (1.0f / (float)D);
  if (g == 0) dv.G[grow] = Gn;
  const float rate = dv.lr / (__builtin_sqrtf(Gn) + dv.eps);
#pragma unroll
  for (int i = 0; i < 8; ++i) x[i] = __builtin_fmaf(-rate, gr[i], x[i]);
}

__device__ __forceinline__ float load_G(const Dev& dv, int64_t grow) { return dv.optimizer ? dv.G[grow] : 0.0f; }

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
  uint32_t ins = 0, byp = 0, ev = 0, em = 0, he = 0;
  __device__ void flush(unsigned long long* stats) {
    if (t < 0) return;
    unsigned long long* s = stats + (int64_t)t * kNStat;
    if (ins) atomicAdd(s + kStInserts, (unsigned long long)ins);
    if (byp) atomicAdd(s + kStBypasses, (unsigned long long)byp);
    if (ev) atomicAdd(s + kStEvictions, (unsigned long long)ev);
    if (em) atomicAdd(s + kStEmptyFills, (unsigned long long)em);
    if (he) atomicAdd(s + kStHitEvictions, (unsigned long long)he);
    ins = byp = ev = em = he = 0;
  }
};

__global__ __launch_bounds__(256) void k_policy(Dev dv, Work w, uint32_t step) {
  __shared__ PolicyLds lds_all[4];
  PolicyLds& L = lds_all[threadIdx.x >> 6];
  const int lane = threadIdx.x & 63;
  const int A = dv.assoc;
  const bool lru = dv.policy == 0;
  const int64_t nS = (int64_t)w.ctr[kCSets];
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  // contiguous runs of sets per wave, so that the table (and its statistics) rarely changes
  const int64_t per = (nS + nwaves - 1) / nwaves;
  const int64_t k0 = wave0 * per, k1 = min<int64_t>(k0 + per, nS);
  PolicyStats ps;  // meaningful in lane 0
  for (int64_t k = k0; k < k1; ++k) {
    const int64_t u0 = w.set_first[k], u1 = w.set_first[k + 1];
    const int t = w.utab[u0];
    const TableDesc td = dv.desc[t];
    const int64_t r0 = (int64_t)w.urow[u0] - td.row_base;
    const int64_t sbase = td.slot_base + (r0 % td.n_sets) * A;

    // residents that hit this step, and the number of missed rows
    L.hitu[lane] = -1;
    __builtin_amdgcn_wave_barrier();
    int64_t M = 0;
    for (int64_t c = u0; c < u1; c += 64) {
      const int64_t u = c + lane;
      bool miss = false;
      if (u < u1) {
        const int32_t sl = w.uslot[u];
        if (sl >= 0) L.hitu[sl - sbase] = (int32_t)u;
        else miss = true;
      }
      M += __popcll(__ballot(miss));
    }
    __builtin_amdgcn_wave_barrier();
    if (M == 0) continue;
    if (t != ps.t) {
      if (lane == 0) ps.flush(dv.stats);
      ps.t = t;
    }

    // ways, their tags and priorities (empty = lowest)
    int32_t tg = -1;
    long long vpv = LLONG_MAX;
    if (lane < A) {
      tg = dv.tag[sbase + lane];
      vpv = tg < 0 ? LLONG_MIN : (lru ? (long long)dv.ts[sbase + lane] : (long long)dv.cnt[td.row_base + tg]);
    }
    // lane k < n_ins: the k-th insert (unique row my_u) takes way my_way, displacing my_old
    // (-1 if the way was empty); my_hu is my_old's unique row if it was updated this step
    int my_way = 0;
    int32_t my_u = -1, my_old = -1, my_hu = -1;
    int n_ins = 0;

    if (A == 1 && lru) {
      // direct-mapped LRU: no priority test; the largest missed row ends in the way
      int64_t win = -1;
      for (int64_t c = u0; c < u1; c += 64) {
        const int64_t u = c + lane;
        const bool miss = u < u1 && w.uslot[u] < 0;
        const uint64_t m = __ballot(miss);
        if (m) win = c + 63 - __clzll((unsigned long long)m);
      }
      n_ins = 1;
      my_u = (int32_t)win;
      my_old = __shfl(tg, 0);
      my_hu = my_old >= 0 ? L.hitu[0] : -1;
    } else {
      // victims ranked by (priority asc, way asc); every lane runs the shuffles
      int vr = 0;
      for (int j = 0; j < A; ++j) {
        const long long pj = __shfl(vpv, j);
        vr += (pj < vpv || (pj == vpv && j < lane)) ? 1 : 0;
      }
      if (lane < A) {
        L.vic_way[vr] = lane;
        L.vic_pv[vr] = vpv;
      }
      // candidates ranked by (priority desc, row asc); only ranks < A matter
      const int64_t K = M < A ? M : A;
      if (lru) {
        int64_t seen = 0;
        for (int64_t c = u0; c < u1 && seen < K; c += 64) {
          const int64_t u = c + lane;
          const bool miss = u < u1 && w.uslot[u] < 0;
          const uint64_t m = __ballot(miss);
          const int64_t rank = seen + __popcll(m & lanemask_lt());
          if (miss && rank < K) {
            L.cand_u[rank] = (int32_t)u;
            L.cand_pv[rank] = (long long)step;
          }
          seen += __popcll(m);
        }
      } else {
        for (int64_t c = u0; c < u1; c += 64) {
          const int64_t u = c + lane;
          const bool miss = u < u1 && w.uslot[u] < 0;
          const long long mypv = miss ? (long long)dv.cnt[w.urow[u]] : 0;
          const int32_t myrow = u < u1 ? w.urow[u] : 0;
          int64_t rank = 0;
          for (int64_t c2 = u0; c2 < u1; c2 += 64) {
            const int64_t u2 = c2 + lane;
            const bool miss2 = u2 < u1 && w.uslot[u2] < 0;
            const long long pv2 = miss2 ? (long long)dv.cnt[w.urow[u2]] : 0;
            const int32_t row2 = u2 < u1 ? w.urow[u2] : 0;
            for (int j = 0; j < 64; ++j) {
              const long long pj = __shfl(pv2, j);
              const int32_t rj = __shfl(row2, j);
              const int mj = __shfl((int)miss2, j);
              if (mj && (pj > mypv || (pj == mypv && rj < myrow))) ++rank;
            }
          }
          if (miss && rank < K) {
            L.cand_u[rank] = (int32_t)u;
            L.cand_pv[rank] = mypv;
          }
        }
      }
      __builtin_amdgcn_wave_barrier();
      // the k-th candidate takes the k-th victim while strictly higher; stop at the first failure
      const bool ok = lane < K && L.cand_pv[lane] > L.vic_pv[lane];
      const uint64_t fail = __ballot(lane < K && !ok);
      n_ins = fail ? __ffsll((unsigned long long)fail) - 1 : (int)K;
      my_way = lane < n_ins ? L.vic_way[lane] : 0;
      my_old = __shfl(tg, my_way);
      my_u = lane < n_ins ? L.cand_u[lane] : -1;
      my_hu = (lane < n_ins && my_old >= 0) ? L.hitu[my_way] : -1;
      __builtin_amdgcn_wave_barrier();
    }
    if (lane < n_ins) {
      w.uact[my_u] = kActInsert;
      w.udest[my_u] = (int32_t)(sbase + my_way);
      w.uvic_row[my_u] = my_old;
      w.uvic_u[my_u] = my_hu;
      if (my_hu >= 0) w.uact[my_hu] = kActDone;  // handled by the row that displaces it
    }
    const uint32_t n_valid = (uint32_t)__popcll(__ballot(lane < n_ins && my_old >= 0));
    const uint32_t n_hitev = (uint32_t)__popcll(__ballot(lane < n_ins && my_hu >= 0));
    if (lane == 0) {
      ps.ins += (uint32_t)n_ins;
      ps.byp += (uint32_t)(M - n_ins);
      ps.ev += n_valid;
      ps.em += (uint32_t)n_ins - n_valid;
      ps.he += n_hitev;
    }
  }
  if (lane == 0) ps.flush(dv.stats);
}

// ---- displaced residents -> T -----------------------------------------------------------------
template <int D, int BITS, bool SB16>
__global__ __launch_bounds__(256) void k_evict(Dev dv, Work w, const uint32_t* __restrict__ sval,
                                               const float* __restrict__ grad, uint32_t step) {
  constexpr int LPR = Geo<D>::LPR;
  constexpr int GPB = 256 / LPR;
  constexpr int RB = Rec<D, BITS, SB16>::BYTES;
  const int g = threadIdx.x & (LPR - 1);
  const int64_t nU = (int64_t)w.ctr[kCUnique];
  const bool sr = dv.rounding != 0;
  const XcdSplit xs(dv.T);
  const int64_t gx = xs.unit * GPB + threadIdx.x / LPR, gstride = xs.units * GPB;
  for (int seg = xs.xcd; seg < xs.segments(dv.T); seg += kXcds) {
    const int t = seg / xs.parts;
    int64_t tlo, thi, lo, hi;
    table_rows(w, t, tlo, thi);
    part_range(tlo, thi, seg % xs.parts, xs.parts, lo, hi);
    const TableDesc td = dv.desc[t];
    for (int64_t u = lo + gx; u < hi; u += gstride) {
      const int32_t act = w.uact[u];
      const int32_t dst = w.udest[u];
      const int32_t vrow = w.uvic_row[u];
      const int32_t vu = w.uvic_u[u];
      if (act != kActInsert || vrow < 0) continue;
      const int64_t vgrow = td.row_base + vrow;
      float xv[8];
      load_frow8(dv.crow + (int64_t)dst * D, g, xv);
      if (vu >= 0) {
        // the displaced resident was updated this step (LFU): its new value goes to T
        const float Gv = load_G(dv, vgrow);
        float gv[8];
        merged_grad<D>(w, sval, grad, vu, g, gv);
        apply_optimizer<D>(dv, xv, gv, vgrow, g, Gv);
      }
      quantize_store<D, BITS, SB16>(xv, g, dv.rec + vgrow * RB, sr, dv.seed, step, (uint32_t)t, (uint32_t)vrow);
    }
  }
}

// ---- per unique row: optimizer and write-back ------------------------------------------------
// Per-row inputs of k_update, loaded one row ahead of their use.
struct RowMeta {
  int32_t act, grow, slot, dst;
  uint32_t nch, s0, s1, cb;
};

__device__ __forceinline__ RowMeta load_meta(const Work& w, int64_t u) {
  RowMeta m;
  m.act = w.uact[u];
  m.grow = w.urow[u];
  m.slot = w.uslot[u];
  m.dst = w.udest[u];
  m.nch = w.nch[u];
  m.s0 = w.seg[u];
  m.s1 = w.seg[u + 1];
  m.cb = w.chunk_base[u];
  return m;
}

template <int D, int BITS, bool SB16>
__global__ __launch_bounds__(256) void k_update(Dev dv, Work w, const uint32_t* __restrict__ sval,
                                                const float* __restrict__ grad, uint32_t step) {
  constexpr int LPR = Geo<D>::LPR;
  constexpr int GPB = 256 / LPR;
  constexpr int RB = Rec<D, BITS, SB16>::BYTES;
  const int g = threadIdx.x & (LPR - 1);
  const bool sr = dv.rounding != 0;
  const XcdSplit xs(dv.T);
  const int64_t gx = xs.unit * GPB + threadIdx.x / LPR, gstride = xs.units * GPB;
  for (int seg = xs.xcd; seg < xs.segments(dv.T); seg += kXcds) {
    const int t = seg / xs.parts;
    int64_t tlo, thi, lo, hi;
    table_rows(w, t, tlo, thi);
    part_range(tlo, thi, seg % xs.parts, xs.parts, lo, hi);
    const TableDesc td = dv.desc[t];
    if (lo + gx >= hi) continue;
    RowMeta next = load_meta(w, lo + gx);
    for (int64_t u = lo + gx; u < hi; u += gstride) {
      const RowMeta m = next;
      // the next row's metadata is in flight while this row is handled (the index is
      // clamped so that the loads are unconditional; the last one is not used)
      next = load_meta(w, min<int64_t>(u + gstride, hi - 1));
      if (m.act == kActDone) continue;
      const int64_t grow = m.grow;
      uint8_t* rec = dv.rec + grow * RB;
      const bool hit = m.act == kActHitStay;
      // first level of loads: the first occurrence values, the row, its accumulator
      const uint32_t n0 = m.nch == 0 ? min<uint32_t>((uint32_t)LPR, m.s1 - m.s0) : 0u;
      const uint32_t myv0 = (uint32_t)g < n0 ? sval[m.s0 + g] : 0u;
      float x[8], gr[8];
      CodeWords<BITS> cw;
      SbWords<SB16> sbw;
      if (hit) {
        load_frow8(dv.crow + (int64_t)m.slot * D, g, x);
      } else {
        cw = load_code_words<BITS>(rec, g);
        sbw = load_sb_words<D, BITS, SB16>(rec);
      }
      const float G_old = load_G(dv, grow);
      if (m.nch == 0) sum_occ<D>(sval, m.s0, m.s1, grad, g, gr, myv0, true);
      else if (m.nch <= kFoldDirect) fold_chunks<D>(w.partial, m.cb, m.nch, g, gr);
      else load_frow8(w.partial + (int64_t)m.cb * D, g, gr);
      if (!hit) {
        float sc, bi;
        decode_sb<SB16>(sbw, sc, bi);
        dequant8<BITS>(cw, sc, bi, x);
      }
      apply_optimizer<D>(dv, x, gr, grow, g, G_old);
      if (hit) {
        store_frow8(dv.crow + (int64_t)m.slot * D, g, x);
      } else if (m.act == kActInsert) {
        store_frow8(dv.crow + (int64_t)m.dst * D, g, x);
        if (g == 0) {
          dv.tag[m.dst] = (int32_t)(grow - td.row_base);
          if (dv.policy == 0) dv.ts[m.dst] = (int32_t)step;
        }
      } else {
        quantize_store<D, BITS, SB16>(x, g, rec, sr, dv.seed, step, (uint32_t)t, (uint32_t)(grow - td.row_base));
      }
    }
  }
}

// ---- one training step ----------------------------------------------------------------------
hipError_t launch_backward(const Dev& d, const Work& w, const int32_t* idx, int64_t L, const int32_t* off, int32_t B,
                           const float* grad, uint64_t step64, int key_bits, bool decay,
                           const hipEvent_t* update_events, hipStream_t s) {
  const uint32_t step = (uint32_t)step64;
  k_bwd_begin<<<1, 256, 0, s>>>(d, w.ctr, L);
  if (decay && d.cnt) k_decay<<<grid_for(d.total_rows), 256, 0, s>>>(d.cnt, d.total_rows);
  hipError_t e = launch_expand(d, idx, L, off, B, w.keysA, w.valsA, w.ctr, s);
  if (e != hipSuccess) return e;
  const int passes = (key_bits + 7) / 8;
  int in_B = 0;
  const SortScratch ss{w.sort_small, w.sort_small + kMaxPasses * 256, w.sort_small + 2 * kMaxPasses * 256,
                       {w.sort_status[0], w.sort_status[1]}};
  e = sort_pairs(w.keysA, w.valsA, w.keysB, w.valsB, L, passes, ss, d.err, &in_B, s);
  if (e != hipSuccess) return e;
  const uint32_t* sk = in_B ? w.keysB : w.keysA;
  const uint32_t* sv = in_B ? w.valsB : w.valsA;
  e = launch_unique(d, sk, L, w.tile_cnt, w.tile_pre, w.part, w.uniq_key, w.seg, w.set_first, w.ctr, s);
  if (e != hipSuccess) return e;
  const auto grid = [](auto kernel) { return resident_grid(reinterpret_cast<const void*>(kernel)); };
  k_probe<<<grid(k_probe), 256, 0, s>>>(d, w, step);
  k_tab_first<<<1, 256, 0, s>>>(w, d.T);
  e = scan_exclusive<uint32_t>(w.nch, w.chunk_base, L, w.ctr + kCUnique, reinterpret_cast<uint32_t*>(w.part),
                               reinterpret_cast<uint32_t*>(w.ctr + kCScanTotal), s);
  if (e != hipSuccess) return e;
  k_chunks_total<<<1, 1, 0, s>>>(w.ctr);
  k_chunk_spans<<<grid(k_chunk_spans), 256, 0, s>>>(w);
  return dispatch_row(d.dim, d.bits, d.sb16, [&]<int D, int BITS, bool SB16>() -> hipError_t {
    k_partials<D><<<grid(k_partials<D>), 256, 0, s>>>(d, w, sv, grad);
    k_hot_fold<D><<<grid(k_hot_fold<D>), 256, 0, s>>>(w);
    if (d.total_slots > 0) {
      k_policy<<<grid(k_policy), 256, 0, s>>>(d, w, step);
      k_evict<D, BITS, SB16><<<grid(k_evict<D, BITS, SB16>), 256, 0, s>>>(d, w, sv, grad, step);
    }
    if (update_events) {
      const hipError_t e2 = hipEventRecord(update_events[0], s);
      if (e2 != hipSuccess) return e2;
    }
    k_update<D, BITS, SB16><<<grid(k_update<D, BITS, SB16>), 256, 0, s>>>(d, w, sv, grad, step);
    if (update_events) {
      const hipError_t e2 = hipEventRecord(update_events[1], s);
      if (e2 != hipSuccess) return e2;
    }
    return hipGetLastError();
  });
}

}  // namespace embc
