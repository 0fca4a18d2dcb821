// State reset, uniform initialisation, and the forward pass:
// pooled[b][t] = sum over the bag of fetch(T_t, C_t, i) (Sec. 3 fetch operator).
#include "embc_device.h"
#include "embc_dispatch.h"

namespace embc {

__global__ __launch_bounds__(256) void k_fill_u32(uint32_t* __restrict__ p, uint32_t v, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}

hipError_t launch_fill_u32(uint32_t* p, uint32_t v, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  k_fill_u32<<<grid_for(n), 256, 0, s>>>(p, v, n);
  return hipGetLastError();
}

hipError_t launch_reset_state(const Dev& d, hipStream_t s) {
  hipError_t e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.rec), 0u, d.total_rows * d.rec_bytes / 4, s);
  if (e == hipSuccess) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.crow), 0u, d.total_slots * d.dim, s);
  if (e == hipSuccess) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.tag), 0xFFFFFFFFu, d.total_slots, s);
  if (e == hipSuccess && d.ts) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.ts), 0xFFFFFFFFu, d.total_slots, s);
  if (e == hipSuccess && d.cnt) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.cnt), 0u, d.total_rows, s);
  if (e == hipSuccess && d.G) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.G), 0u, d.total_rows, s);
  if (e == hipSuccess) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.stats), 0u, (int64_t)d.T * kNStat * 2, s);
  if (e == hipSuccess) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.err), 0u, 1, s);
  return e;
}

// Table owning global row `grow` (binary search over row_base).
__device__ __forceinline__ int table_of_row(const Dev& dv, int64_t grow) {
  int lo = 0, hi = dv.T;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (grow >= dv.desc[mid].row_base) lo = mid; else hi = mid;
  }
  return lo;
}

// x_j = u*(hi-lo) + lo (fused), u = Philox uniform keyed (init_seed; j/4, row, table, 0xFFFFFFFF),
// then nearest-even quantization of the row.
template <int D, int BITS, bool SB16>
__global__ __launch_bounds__(256) void k_init_uniform(Dev dv, float lo, float hi, uint64_t init_seed) {
  constexpr int LPR = Geo<D>::LPR, CPL = Geo<D>::CPL;
  constexpr int RB = Rec<D, BITS, SB16>::BYTES;
  const int g = threadIdx.x & (LPR - 1);
  const int64_t ngroups = (int64_t)gridDim.x * blockDim.x / LPR;
  const float width = hi - lo;
  for (int64_t grow = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / LPR; grow < dv.total_rows;
       grow += ngroups) {
    const int t = table_of_row(dv, grow);
    const uint32_t r = (uint32_t)(grow - dv.desc[t].row_base);
    float x[CPL];
#pragma unroll
    for (int k = 0; k < CPL; ++k)
      x[k] = __builtin_fmaf(sr_uniform(init_seed, 0xFFFFFFFFu, (uint32_t)t, r, (uint32_t)(g + LPR * k)), width, lo);
    quantize_store<D, BITS, SB16>(x, g, dv.rec + grow * RB, false, 0, 0, 0, 0);
  }
}

hipError_t launch_init_uniform(const Dev& d, float lo, float hi, uint64_t init_seed, hipStream_t s) {
  hipError_t e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.tag), 0xFFFFFFFFu, d.total_slots, s);
  if (e == hipSuccess && d.ts) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.ts), 0xFFFFFFFFu, d.total_slots, s);
  if (e == hipSuccess) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.crow), 0u, d.total_slots * d.dim, s);
  if (e == hipSuccess && d.cnt) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.cnt), 0u, d.total_rows, s);
  if (e == hipSuccess && d.G) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.G), 0u, d.total_rows, s);
  if (e != hipSuccess) return e;
  return dispatch_row(d.dim, d.bits, d.sb16, [&]<int D, int BITS, bool SB16>() -> hipError_t {
    const int64_t threads = d.total_rows * Geo<D>::LPR;
    k_init_uniform<D, BITS, SB16><<<grid_for(threads, 16384), 256, 0, s>>>(d, lo, hi, init_seed);
    return hipGetLastError();
  });
}

// ---- forward --------------------------------------------------------------------------
// One group of LPR lanes per bag, `bpg` consecutive bags per group.  For each
// chunk of up to LPR positions, lane j loads index j and probes its set; then
// the rows are gathered one after the other (each lane its columns) and summed
// left to right.  A bag with no valid lookup gives +0.
template <int D, int BITS, bool SB16>
__global__ __launch_bounds__(256) void k_forward(Dev dv, const int32_t* __restrict__ idx, int64_t L,
                                                 const int32_t* __restrict__ off, int32_t B, float* __restrict__ out,
                                                 int bpg) {
  constexpr int LPR = Geo<D>::LPR, CPL = Geo<D>::CPL;
  constexpr int RB = Rec<D, BITS, SB16>::BYTES;
  const int g = threadIdx.x & (LPR - 1);
  const int64_t grp = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / LPR;
  const int64_t nbags = (int64_t)dv.T * B;
  int64_t bag = grp * bpg;
  const int64_t bag_end = min<int64_t>(bag + bpg, nbags);
  int cur_t = -1;
  uint32_t c_valid = 0, c_hit = 0, c_bad = 0;
  auto flush = [&]() {
#pragma unroll
    for (int o = LPR / 2; o >= 1; o >>= 1) {
      c_valid += __shfl_xor(c_valid, o, LPR);
      c_hit += __shfl_xor(c_hit, o, LPR);
      c_bad += __shfl_xor(c_bad, o, LPR);
    }
    if (g == 0 && cur_t >= 0) {
      unsigned long long* st = dv.stats + (int64_t)cur_t * kNStat;
      if (c_valid) atomicAdd(st + kStLookups, (unsigned long long)c_valid);
      if (c_hit) atomicAdd(st + kStHitLookups, (unsigned long long)c_hit);
      if (c_bad) {
        atomicAdd(st + kStInvalidFwd, (unsigned long long)c_bad);
        atomicOr(dv.err, kErrIndex);
      }
    }
    c_valid = c_hit = c_bad = 0;
  };
  for (; bag < bag_end; ++bag) {
    const int t = (int)(bag / B);
    if (t != cur_t) {
      flush();
      cur_t = t;
    }
    const int b = (int)(bag - (int64_t)t * B);
    const TableDesc td = dv.desc[t];
    int64_t p0 = off[bag], p1 = off[bag + 1];
    p0 = p0 < 0 ? 0 : p0;
    p1 = p1 > L ? L : p1;
    float acc[CPL];
#pragma unroll
    for (int k = 0; k < CPL; ++k) acc[k] = 0.0f;
    bool first = true;
    for (int64_t pc = p0; pc < p1; pc += LPR) {
      const int n = (int)min<int64_t>(LPR, p1 - pc);
      int32_t r = 0, slot = -1, ok = 0;
      if (g < n) {
        r = idx[pc + g];
        ok = (r >= 0 && (int64_t)r < td.N);
        if (ok) {
          slot = probe_slot(dv, td, r);
          ++c_valid;
          c_hit += slot >= 0;
        } else {
          ++c_bad;
        }
      }
      for (int j = 0; j < n; ++j) {
        if (!__shfl(ok, j, LPR)) continue;
        const int32_t rj = __shfl(r, j, LPR);
        const int32_t sj = __shfl(slot, j, LPR);
        float v[CPL];
        if (sj >= 0) {
          load_frow<D>(dv.crow + (int64_t)sj * D, g, v);
        } else {
          dequant_row<D, BITS, SB16>(dv.rec + (td.row_base + rj) * RB, g, v);
        }
        if (first) {
#pragma unroll
          for (int k = 0; k < CPL; ++k) acc[k] = v[k];
          first = false;
        } else {
#pragma unroll
          for (int k = 0; k < CPL; ++k) acc[k] = acc[k] + v[k];
        }
      }
    }
    store_frow<D>(out + ((int64_t)b * dv.T + t) * D, g, acc);
  }
  flush();
}

__global__ void k_zero_stats(Dev dv, int first, int last) {
  for (int i = threadIdx.x; i < dv.T * kNStat; i += blockDim.x) {
    const int f = i % kNStat;
    if (f >= first && f <= last) dv.stats[i] = 0;
  }
}

__global__ void k_zero_fwd_stats(Dev dv) {
  for (int i = threadIdx.x; i < dv.T; i += blockDim.x) {
    dv.stats[(int64_t)i * kNStat + kStLookups] = 0;
    dv.stats[(int64_t)i * kNStat + kStHitLookups] = 0;
    dv.stats[(int64_t)i * kNStat + kStInvalidFwd] = 0;
  }
}

hipError_t launch_forward(const Dev& d, const int32_t* idx, int64_t L, const int32_t* off, int32_t B, float* out,
                          hipStream_t s) {
  k_zero_fwd_stats<<<1, 256, 0, s>>>(d);
  const int64_t nbags = (int64_t)d.T * B;
  if (nbags == 0) return hipGetLastError();
  return dispatch_row(d.dim, d.bits, d.sb16, [&]<int D, int BITS, bool SB16>() -> hipError_t {
    const int bpg = 4;
    const int64_t groups = (nbags + bpg - 1) / bpg;
    const int64_t threads = groups * Geo<D>::LPR;
    k_forward<D, BITS, SB16><<<(unsigned)((threads + 255) / 256), 256, 0, s>>>(d, idx, L, off, B, out, bpg);
    return hipGetLastError();
  });
}

}  // namespace embc
