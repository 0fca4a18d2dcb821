// Backward + sparse update of one step (Sec. 3 update operator, Alg. 2, Sec. 5.1 de-dup).
//
// After the sort (k_sort.hip) the lookups are grouped by row, the rows by set:
//   k_probe        per unique row: residency (slot or miss), LRU stamp / LFU count update
//   k_policy       per touched set (one wave, one lane per way): which missed rows
//                  enter the cache, which residents leave
//   k_partials     chunk sums of the merged gradient of rows with > 64 lookups
//   k_update_main  per unique row not inserted, and per displaced resident: merged
//                  gradient, fetch, optimizer, write to the cache way or quantize into T
//   k_update_ins   per inserted row: same, written into its new way (after every
//                  displaced resident has been read)
#include "embc_device.h"
#include "embc_dispatch.h"
#include "embc_sort.h"

namespace embc {

constexpr int kGrid = 2048;  // blocks of the grid-stride kernels (8 per CU)

// Sum `v` over the active lanes of the wave, per table: one atomic for the lanes
// that share the first active lane's table, one per lane for the others.
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

// Wave-aggregated append to a list: returns this lane's position (valid where `want`).
__device__ __forceinline__ uint32_t wave_append(unsigned long long* counter, bool want) {
  const uint64_t m = __ballot(want);
  if (!m) return 0;
  const int leader = __ffsll((unsigned long long)m) - 1;
  const int lane = threadIdx.x & 63;
  unsigned long long base = 0;
  if (lane == leader) base = atomicAdd(counter, (unsigned long long)__popcll(m));
  base = __shfl(base, leader);
  return (uint32_t)(base + __popcll(m & lanemask_lt()));
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
      w.udest[u] = slot;
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

// ---- replacement decision, one wave per touched set ------------------------------------------
struct PolicyLds {
  int32_t hitu[64];       // unique row that hit way w this step, or -1
  int32_t cand_u[64];     // candidates by rank
  long long cand_pv[64];
  int32_t vic_way[64];    // victims by rank
  long long vic_pv[64];
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
  for (int64_t k = wave0; k < nS; k += nwaves) {
    const int64_t u0 = w.set_first[k], u1 = w.set_first[k + 1];
    const int t = w.utab[u0];
    const TableDesc td = dv.desc[t];
    const int64_t r0 = (int64_t)w.urow[u0] - td.row_base;
    const int64_t set = r0 % td.n_sets;
    const int64_t sbase = td.slot_base + set * A;

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

    // ways, their tags and priorities (empty = lowest)
    int32_t tg = -1;
    long long vpv = LLONG_MAX;
    if (lane < A) {
      tg = dv.tag[sbase + lane];
      vpv = tg < 0 ? LLONG_MIN : (lru ? (long long)dv.ts[sbase + lane] : (long long)dv.cnt[td.row_base + tg]);
    }
    // per-lane contributions to the statistics
    uint32_t s_ins = 0, s_byp = 0, s_ev = 0, s_em = 0, s_he = 0;

    if (A == 1 && lru) {
      // direct-mapped LRU: no priority test; the largest missed row ends in the way
      int64_t win = -1;
      for (int64_t c = u0; c < u1; c += 64) {
        const int64_t u = c + lane;
        const bool miss = u < u1 && w.uslot[u] < 0;
        const uint64_t m = __ballot(miss);
        if (m) win = c + 63 - __clzll((unsigned long long)m);
      }
      const int32_t old = __shfl(tg, 0);
      const int32_t hu = L.hitu[0];
      const bool push_victim = lane == 0 && old >= 0 && hu < 0;
      if (lane == 0) {
        w.uact[win] = kActInsert;
        w.udest[win] = (int32_t)sbase;
        if (old >= 0 && hu >= 0) w.uact[hu] = kActHitEvict;
      }
      const uint32_t ip = wave_append(w.ctr + kCInserts, lane == 0);
      if (lane == 0) w.ins_list[ip] = (int32_t)win;
      const uint32_t vp = wave_append(w.ctr + kCVictims, push_victim);
      if (push_victim) {
        w.vic_slot[vp] = (int32_t)sbase;
        w.vic_row[vp] = (int32_t)(td.row_base + old);
        w.vic_tab[vp] = t;
      }
      if (lane == 0) {
        s_ins = 1;
        s_byp = (uint32_t)(M - 1);
        s_ev = old >= 0;
        s_em = old < 0;
        s_he = old >= 0 && hu >= 0;
      }
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
      const int m = fail ? __ffsll((unsigned long long)fail) - 1 : (int)K;
      bool push_victim = false;
      int32_t vslot = 0, vrow = 0, cu = -1;
      const int way = lane < m ? L.vic_way[lane] : 0;
      const int32_t old = __shfl(tg, way);  // tag of the way this lane's candidate takes
      if (lane < m) {
        cu = L.cand_u[lane];
        const int32_t slot = (int32_t)(sbase + way);
        w.uact[cu] = kActInsert;
        w.udest[cu] = slot;
        s_ins = 1;
        if (old < 0) {
          s_em = 1;
        } else {
          s_ev = 1;
          const int32_t hu = L.hitu[way];
          if (hu >= 0) {
            w.uact[hu] = kActHitEvict;
            s_he = 1;
          } else {
            push_victim = true;
            vslot = slot;
            vrow = (int32_t)(td.row_base + old);
          }
        }
      }
      const uint32_t ip = wave_append(w.ctr + kCInserts, lane < m);
      if (lane < m) w.ins_list[ip] = cu;
      const uint32_t vp = wave_append(w.ctr + kCVictims, push_victim);
      if (push_victim) {
        w.vic_slot[vp] = vslot;
        w.vic_row[vp] = vrow;
        w.vic_tab[vp] = t;
      }
      if (lane == 0) s_byp = (uint32_t)(M - m);
      __builtin_amdgcn_wave_barrier();
    }
    wave_stat_add(dv.stats, t, kStInserts, s_ins, true);
    wave_stat_add(dv.stats, t, kStBypasses, s_byp, true);
    wave_stat_add(dv.stats, t, kStEvictions, s_ev, true);
    wave_stat_add(dv.stats, t, kStEmptyFills, s_em, true);
    wave_stat_add(dv.stats, t, kStHitEvictions, s_he, true);
  }
}

// ---- merged gradient ----------------------------------------------------------------------
// Left-to-right FP32 sum of the gradient rows of occurrences [i0, i1) of the sorted
// stream, starting from the first term.  Lane j of the group preloads the row
// index of occurrence j of each chunk of LPR occurrences.
template <int D>
__device__ __forceinline__ void sum_occ(const uint32_t* __restrict__ sval, int64_t i0, int64_t i1,
                                        const float* __restrict__ grad, int g, float (&acc)[Geo<D>::CPL]) {
  constexpr int LPR = Geo<D>::LPR, CPL = Geo<D>::CPL;
  bool first = true;
  for (int64_t ic = i0; ic < i1; ic += LPR) {
    const int n = (int)min<int64_t>(LPR, i1 - ic);
    const uint32_t myv = g < n ? sval[ic + g] : 0u;
    for (int j = 0; j < n; ++j) {
      const uint32_t gv = __shfl(myv, j, LPR);
      float x[CPL];
      load_frow<D>(grad + (int64_t)gv * D, g, x);
      if (first) {
#pragma unroll
        for (int k = 0; k < CPL; ++k) acc[k] = x[k];
        first = false;
      } else {
#pragma unroll
        for (int k = 0; k < CPL; ++k) acc[k] = acc[k] + x[k];
      }
    }
  }
}

template <int D>
__device__ __forceinline__ void merged_grad(const Work& w, const uint32_t* __restrict__ sval,
                                            const float* __restrict__ grad, int64_t u, int g,
                                            float (&acc)[Geo<D>::CPL]) {
  const uint32_t nch = w.nch[u];
  if (nch == 0) {
    sum_occ<D>(sval, w.seg[u], w.seg[u + 1], grad, g, acc);
  } else {
    const int64_t c0 = w.chunk_base[u];
    load_frow<D>(w.partial + c0 * D, g, acc);
    for (uint32_t c = 1; c < nch; ++c) {
      float x[Geo<D>::CPL];
      load_frow<D>(w.partial + (c0 + c) * D, g, x);
#pragma unroll
      for (int k = 0; k < Geo<D>::CPL; ++k) acc[k] = acc[k] + x[k];
    }
  }
}

template <int D>
__global__ __launch_bounds__(256) void k_partials(Work w, const uint32_t* __restrict__ sval,
                                                  const float* __restrict__ grad) {
  constexpr int LPR = Geo<D>::LPR, CPL = Geo<D>::CPL;
  const int g = threadIdx.x & (LPR - 1);
  const int64_t nC = (int64_t)w.ctr[kCChunks];
  const int64_t nU = (int64_t)w.ctr[kCUnique];
  const int64_t ngroups = (int64_t)gridDim.x * blockDim.x / LPR;
  for (int64_t c = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / LPR; c < nC; c += ngroups) {
    // unique row owning chunk c: the largest u with chunk_base[u] <= c
    int64_t lo = 0, hi = nU;
    while (hi - lo > 1) {
      const int64_t mid = (lo + hi) >> 1;
      if ((int64_t)w.chunk_base[mid] <= c) lo = mid; else hi = mid;
    }
    const int64_t u = lo;
    const int64_t j = c - (int64_t)w.chunk_base[u];
    const int64_t i0 = (int64_t)w.seg[u] + j * kSumChunk;
    const int64_t i1 = min<int64_t>(i0 + kSumChunk, (int64_t)w.seg[u + 1]);
    float acc[CPL];
    sum_occ<D>(sval, i0, i1, grad, g, acc);
    store_frow<D>(w.partial + c * D, g, acc);
  }
}

// ---- optimizer (FP32) -----------------------------------------------------------------------
// SGD: x = fma(-lr, g, x).  Row-wise Adagrad: S = halving-tree sum of g_j^2
// (a[j] += a[j + h] for h = D/2, ..., 1), G += S * (1/D), r = lr / (sqrt(G) + eps),
// x = fma(-r, g, x).
template <int D>
__device__ __forceinline__ void apply_optimizer(const Dev& dv, float (&x)[Geo<D>::CPL], const float (&gr)[Geo<D>::CPL],
                                                int64_t grow, int g) {
  constexpr int LPR = Geo<D>::LPR, CPL = Geo<D>::CPL;
  if (dv.optimizer == 0) {
#pragma unroll
    for (int k = 0; k < CPL; ++k) x[k] = __builtin_fmaf(-dv.lr, gr[k], x[k]);
    return;
  }
  float a[CPL];
#pragma unroll
  for (int k = 0; k < CPL; ++k) a[k] = gr[k] * gr[k];
#pragma unroll
  for (int h = CPL / 2; h >= 1; h >>= 1)
#pragma unroll
    for (int k = 0; k < h; ++k) a[k] = a[k] + a[k + h];
  float S = a[0];
#pragma unroll
  for (int o = LPR / 2; o >= 1; o >>= 1) S = S + __shfl_xor(S, o, LPR);
  const float Gn = dv.G[grow] + S * (1.0f / (float)D);
  if (g == 0) dv.G[grow] = Gn;
  const float rate = dv.lr / (__builtin_sqrtf(Gn) + dv.eps);
#pragma unroll
  for (int k = 0; k < CPL; ++k) x[k] = __builtin_fmaf(-rate, gr[k], x[k]);
}

// ---- write-back of updated rows and displaced residents -------------------------------------
template <int D, int BITS, bool SB16>
__global__ __launch_bounds__(256) void k_update_main(Dev dv, Work w, const uint32_t* __restrict__ sval,
                                                     const float* __restrict__ grad, uint32_t step) {
  constexpr int LPR = Geo<D>::LPR, CPL = Geo<D>::CPL;
  constexpr int RB = Rec<D, BITS, SB16>::BYTES;
  const int g = threadIdx.x & (LPR - 1);
  const int64_t nU = (int64_t)w.ctr[kCUnique];
  const int64_t nV = (int64_t)w.ctr[kCVictims];
  const int64_t ngroups = (int64_t)gridDim.x * blockDim.x / LPR;
  const bool sr = dv.rounding != 0;
  for (int64_t it = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / LPR; it < nU + nV; it += ngroups) {
    float x[CPL];
    if (it < nU) {
      const int64_t u = it;
      const int32_t act = w.uact[u];
      if (act == kActInsert) continue;
      const int64_t grow = w.urow[u];
      const int t = w.utab[u];
      float gr[CPL];
      merged_grad<D>(w, sval, grad, u, g, gr);
      uint8_t* rec = dv.rec + grow * RB;
      const int32_t slot = w.uslot[u];
      if (act == kActBypass) dequant_row<D, BITS, SB16>(rec, g, x);
      else load_frow<D>(dv.crow + (int64_t)slot * D, g, x);
      apply_optimizer<D>(dv, x, gr, grow, g);
      if (act == kActHitStay) {
        store_frow<D>(dv.crow + (int64_t)slot * D, g, x);
      } else {
        const uint32_t r = (uint32_t)(grow - dv.desc[t].row_base);
        quantize_store<D, BITS, SB16>(x, g, rec, sr, dv.seed, step, (uint32_t)t, r);
      }
    } else {
      const int64_t v = it - nU;
      const int32_t slot = w.vic_slot[v];
      const int64_t grow = w.vic_row[v];
      const int t = w.vic_tab[v];
      load_frow<D>(dv.crow + (int64_t)slot * D, g, x);
      const uint32_t r = (uint32_t)(grow - dv.desc[t].row_base);
      quantize_store<D, BITS, SB16>(x, g, dv.rec + grow * RB, sr, dv.seed, step, (uint32_t)t, r);
    }
  }
}

template <int D, int BITS, bool SB16>
__global__ __launch_bounds__(256) void k_update_ins(Dev dv, Work w, const uint32_t* __restrict__ sval,
                                                    const float* __restrict__ grad, uint32_t step) {
  constexpr int LPR = Geo<D>::LPR, CPL = Geo<D>::CPL;
  constexpr int RB = Rec<D, BITS, SB16>::BYTES;
  const int g = threadIdx.x & (LPR - 1);
  const int64_t nI = (int64_t)w.ctr[kCInserts];
  const int64_t ngroups = (int64_t)gridDim.x * blockDim.x / LPR;
  for (int64_t it = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / LPR; it < nI; it += ngroups) {
    const int64_t u = w.ins_list[it];
    const int64_t grow = w.urow[u];
    const int t = w.utab[u];
    const int32_t dst = w.udest[u];
    float gr[CPL], x[CPL];
    merged_grad<D>(w, sval, grad, u, g, gr);
    dequant_row<D, BITS, SB16>(dv.rec + grow * RB, g, x);
    apply_optimizer<D>(dv, x, gr, grow, g);
    store_frow<D>(dv.crow + (int64_t)dst * D, g, x);
    if (g == 0) {
      dv.tag[dst] = (int32_t)(grow - dv.desc[t].row_base);
      if (dv.policy == 0) dv.ts[dst] = (int32_t)step;
    }
  }
}

// ---- one training step ----------------------------------------------------------------------
hipError_t launch_backward(const Dev& d, const Work& w, const int32_t* idx, int64_t L, const int32_t* off, int32_t B,
                           const float* grad, uint64_t step64, int key_bits, bool decay, hipStream_t s) {
  const uint32_t step = (uint32_t)step64;
  k_bwd_begin<<<1, 256, 0, s>>>(d, w.ctr, L);
  if (decay && d.cnt) k_decay<<<grid_for(d.total_rows), 256, 0, s>>>(d.cnt, d.total_rows);
  hipError_t e = launch_expand(d, idx, L, off, B, w.keysA, w.valsA, w.ctr, s);
  if (e != hipSuccess) return e;
  const int passes = (key_bits + 7) / 8;
  int in_B = 0;
  e = sort_pairs(w.keysA, w.valsA, w.keysB, w.valsB, L, passes, w.hist, reinterpret_cast<uint32_t*>(w.part), &in_B, s);
  if (e != hipSuccess) return e;
  const uint32_t* sk = in_B ? w.keysB : w.keysA;
  const uint32_t* sv = in_B ? w.valsB : w.valsA;
  e = launch_unique(d, sk, L, w.flag, w.pre, w.part, w.uniq_key, w.seg, w.set_first, w.ctr, s);
  if (e != hipSuccess) return e;
  k_probe<<<kGrid, 256, 0, s>>>(d, w, step);
  e = scan_exclusive<uint32_t>(w.nch, w.chunk_base, L, w.ctr + kCUnique, reinterpret_cast<uint32_t*>(w.part),
                               reinterpret_cast<uint32_t*>(w.ctr + kCScanTotal), s);
  if (e != hipSuccess) return e;
  k_chunks_total<<<1, 1, 0, s>>>(w.ctr);
  if (d.total_slots > 0) k_policy<<<kGrid, 256, 0, s>>>(d, w, step);
  return dispatch_row(d.dim, d.bits, d.sb16, [&]<int D, int BITS, bool SB16>() -> hipError_t {
    k_partials<D><<<kGrid, 256, 0, s>>>(w, sv, grad);
    k_update_main<D, BITS, SB16><<<kGrid, 256, 0, s>>>(d, w, sv, grad, step);
    k_update_ins<D, BITS, SB16><<<kGrid, 256, 0, s>>>(d, w, sv, grad, step);
    return hipGetLastError();
  });
}

}  // namespace embc
