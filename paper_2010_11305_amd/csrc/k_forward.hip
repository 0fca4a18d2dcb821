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
  constexpr int LPR = Geo<D>::LPR;
  constexpr int RB = Rec<D, BITS, SB16>::BYTES;
  const int g = threadIdx.x & (LPR - 1);
  const int64_t ngroups = (int64_t)gridDim.x * blockDim.x / LPR;
  const float width = hi - lo;
  for (int64_t grow = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / LPR; grow < dv.total_rows;
       grow += ngroups) {
    const int t = table_of_row(dv, grow);
    const uint32_t r = (uint32_t)(grow - dv.desc[t].row_base);
    float u[8], x[8];
    uniforms8(init_seed, 0xFFFFFFFFu, (uint32_t)t, r, g, u);
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = __builtin_fmaf(u[i], width, lo);
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
// One group of LPR lanes per bag (64/LPR bags per wave at once); tables are split
// over the XCDs (XcdSplit), and the groups of an XCD share the bags of its current
// table.  For each chunk of up to LPR positions, lane j loads index j and probes its
// set.  The rows are then fetched FU at a time -- all FU loads (FP32 cache row, or
// codes and scale/bias) issued before any is used -- and summed left to right.  A
// bag with no valid lookup gives +0.
constexpr int kFwdUnroll = 4;

template <int D, int BITS, bool SB16>
__global__ __launch_bounds__(256) void k_forward(Dev dv, const int32_t* __restrict__ idx, int64_t L,
                                                 const int32_t* __restrict__ off, int32_t B, float* __restrict__ out) {
  constexpr int LPR = Geo<D>::LPR, FU = kFwdUnroll;
  constexpr int GPB = 256 / LPR;
  constexpr int RB = Rec<D, BITS, SB16>::BYTES;
  const int g = threadIdx.x & (LPR - 1);
  const XcdSplit xs(dv.T);
  const int64_t gx = xs.unit * GPB + threadIdx.x / LPR, gstride = xs.units * GPB;
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
  for (int seg = xs.xcd; seg < xs.segments(dv.T); seg += kXcds) {
   const int t = seg / xs.parts;
   int64_t blo, bhi;
   part_range(0, B, seg % xs.parts, xs.parts, blo, bhi);
   if (t != cur_t) {
     flush();
     cur_t = t;
   }
   const TableDesc td = dv.desc[t];
   for (int64_t b = blo + gx; b < bhi; b += gstride) {
    const int64_t bag = (int64_t)t * B + b;
    const uint8_t* rec0 = dv.rec + td.row_base * RB;
    int64_t p0 = off[bag], p1 = off[bag + 1];
    p0 = p0 < 0 ? 0 : p0;
    p1 = p1 > L ? L : p1;
    float acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.0f;
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
      for (int j = 0; j < n; j += FU) {
        float raw[FU][8];
        CodeWords<BITS> cw[FU];
        float sq[FU], bq[FU];
        int kind[FU];  // 0 skip, 1 cache row, 2 low-precision row
#pragma unroll
        for (int q = 0; q < FU; ++q) {
          const int okq = __shfl(ok, j + q, LPR);
          const int32_t rq = __shfl(r, j + q, LPR);
          const int32_t sl = __shfl(slot, j + q, LPR);
          kind[q] = (j + q < n && okq) ? (sl >= 0 ? 1 : 2) : 0;
          if (kind[q] == 1) {
            load_frow8(dv.crow + (int64_t)sl * D, g, raw[q]);
          } else if (kind[q] == 2) {
            const uint8_t* rec = rec0 + (int64_t)rq * RB;
            cw[q] = load_code_words<BITS>(rec, g);
            load_sb<D, BITS, SB16>(rec, sq[q], bq[q]);
          }
        }
#pragma unroll
        for (int q = 0; q < FU; ++q) {
          if (kind[q] == 0) continue;
          if (kind[q] == 2) dequant8<BITS>(cw[q], sq[q], bq[q], raw[q]);
          if (first) {
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[i] = raw[q][i];
            first = false;
          } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[i] = acc[i] + raw[q][i];
          }
        }
      }
    }
    store_frow8(out + ((int64_t)b * dv.T + t) * D, g, acc);
   }
  }
  flush();
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
    // whole multiples of 8 workgroups (one per XCD), at most 8 per CU
    const int64_t wgs = (nbags * Geo<D>::LPR + 255) / 256;
    int64_t blocks = (wgs + 7) / 8 * 8;
    blocks = blocks < 8 ? 8 : (blocks > 2048 ? 2048 : blocks);
    const unsigned grid = (unsigned)blocks;
    k_forward<D, BITS, SB16><<<grid, 256, 0, s>>>(d, idx, L, off, B, out);
    return hipGetLastError();
  });
}

}  // namespace embc
