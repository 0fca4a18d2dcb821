// Device-side building blocks of libembcache (gfx950, wave64).
//
// Lane layout of one embedding row of width D: a row is handled by a group of
// LPR = min(D, 64) consecutive lanes; lane g of the group holds the CPL = D/LPR
// columns g, g + LPR, g + 2*LPR, ...  Column pairs (j, j + D/2) of the
// halving-tree sum therefore sit in the same lane while D > 64 and in lanes
// g, g ^ (D/2) below, and consecutive columns (2m, 2m+1) of an INT4 byte sit
// in neighbouring lanes.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "embc_internal.h"

namespace embc {

template <int D>
struct Geo {
  static constexpr int LPR = D < 64 ? D : 64;  // lanes per row
  static constexpr int CPL = D / LPR;          // columns per lane
  static constexpr int GPW = 64 / LPR;         // row groups per wave
};

template <int D, int BITS, bool SB16>
struct Rec {
  static constexpr int CODE_BYTES = D * BITS / 8;
  static constexpr int BYTES = CODE_BYTES + (SB16 ? 4 : 8);
};

// ---- Philox4x32-10 (Salmon et al., SC'11): 10 rounds, Weyl key schedule -------------
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int i = 0; i < 10; ++i) {
    const uint32_t a = c.x, b = c.z;
    const uint32_t hi0 = __umulhi(0xD2511F53u, a), lo0 = 0xD2511F53u * a;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, b), lo1 = 0xCD9E8D57u * b;
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

// Uniform in [0,1) with 24 bits for element (table, row, col) at `step`:
// counter (col/4, row, table, step), key (seed lo, seed hi), word col%4.
__device__ __forceinline__ float sr_uniform(uint64_t seed, uint32_t step, uint32_t table, uint32_t row,
                                            uint32_t col) {
  const uint4 o = philox4x32_10(make_uint4(col >> 2, row, table, step), (uint32_t)seed, (uint32_t)(seed >> 32));
  const uint32_t q = col & 3u;
  const uint32_t w = q == 0 ? o.x : (q == 1 ? o.y : (q == 2 ? o.z : o.w));
  return (float)(w >> 8) * 5.9604644775390625e-08f;  // 2^-24
}

__device__ __forceinline__ float f16_round(float x) { return __half2float(__float2half(x)); }

template <int D, int BITS, bool SB16>
__device__ __forceinline__ void load_sb(const uint8_t* rec, float& s, float& b) {
  constexpr int CB = Rec<D, BITS, SB16>::CODE_BYTES;
  if constexpr (SB16) {
    const uint32_t w = *reinterpret_cast<const uint32_t*>(rec + CB);
    s = __half2float(__ushort_as_half((unsigned short)(w & 0xFFFFu)));
    b = __half2float(__ushort_as_half((unsigned short)(w >> 16)));
  } else {
    const float2 v = *reinterpret_cast<const float2*>(rec + CB);
    s = v.x;
    b = v.y;
  }
}

template <int BITS>
__device__ __forceinline__ uint32_t load_code(const uint8_t* rec, int col) {
  if constexpr (BITS == 8) {
    return rec[col];
  } else {
    const uint32_t byte = rec[col >> 1];
    return (byte >> ((col & 1) * 4)) & 15u;
  }
}

// fetch() of a non-resident row: q*s + b with one rounding (Alg. 1 dequantization).
template <int D, int BITS, bool SB16>
__device__ __forceinline__ void dequant_row(const uint8_t* rec, int g, float (&x)[Geo<D>::CPL]) {
  float s, b;
  load_sb<D, BITS, SB16>(rec, s, b);
#pragma unroll
  for (int k = 0; k < Geo<D>::CPL; ++k)
    x[k] = __builtin_fmaf((float)load_code<BITS>(rec, g + Geo<D>::LPR * k), s, b);
}

template <int D>
__device__ __forceinline__ void load_frow(const float* row, int g, float (&x)[Geo<D>::CPL]) {
#pragma unroll
  for (int k = 0; k < Geo<D>::CPL; ++k) x[k] = row[g + Geo<D>::LPR * k];
}

template <int D>
__device__ __forceinline__ void store_frow(float* row, int g, const float (&x)[Geo<D>::CPL]) {
#pragma unroll
  for (int k = 0; k < Geo<D>::CPL; ++k) row[g + Geo<D>::LPR * k] = x[k];
}

// Down-conversion of one FP32 row into its low-precision record (Alg. 1 with the
// Sec. 3 rounding knob).  b = min, s = (max - min)/(2^BITS - 1) (FP32, correctly
// rounded; then rounded to FP16 when SB16); codes q = round((x - b)/s) clamped to
// [0, 2^BITS - 1], all zero when s == 0.  A -0 extreme is taken as +0.
template <int D, int BITS, bool SB16>
__device__ __forceinline__ void quantize_store(const float (&x)[Geo<D>::CPL], int g, uint8_t* rec, bool sr,
                                               uint64_t seed, uint32_t step, uint32_t table, uint32_t row) {
  constexpr int LPR = Geo<D>::LPR, CPL = Geo<D>::CPL;
  constexpr int CB = Rec<D, BITS, SB16>::CODE_BYTES;
  constexpr float K = (float)((1 << BITS) - 1);
  float mn = x[0], mx = x[0];
#pragma unroll
  for (int k = 1; k < CPL; ++k) {
    mn = fminf(mn, x[k]);
    mx = fmaxf(mx, x[k]);
  }
#pragma unroll
  for (int o = LPR / 2; o >= 1; o >>= 1) {
    mn = fminf(mn, __shfl_xor(mn, o, LPR));
    mx = fmaxf(mx, __shfl_xor(mx, o, LPR));
  }
  mn = mn + 0.0f;
  mx = mx + 0.0f;
  float s = (mx - mn) / K;
  float b = mn;
  if constexpr (SB16) {
    s = f16_round(s);
    b = f16_round(b);
  }
#pragma unroll
  for (int k = 0; k < CPL; ++k) {
    const int col = g + LPR * k;
    float qf = 0.0f;
    if (s != 0.0f) {
      const float v = (x[k] - b) / s;
      if (sr) {
        const float f = floorf(v);
        const float u = sr_uniform(seed, step, table, row, (uint32_t)col);
        qf = (u < v - f) ? f + 1.0f : f;
      } else {
        qf = rintf(v);
      }
      qf = qf < 0.0f ? 0.0f : qf;
      qf = qf > K ? K : qf;
    }
    const uint32_t q = (uint32_t)qf;
    if constexpr (BITS == 8) {
      rec[col] = (uint8_t)q;
    } else {
      const uint32_t hi = (uint32_t)__shfl_xor((int)q, 1, LPR);
      if ((g & 1) == 0) rec[col >> 1] = (uint8_t)(q | (hi << 4));
    }
  }
  if (g == 0) {
    if constexpr (SB16) {
      const uint32_t w = (uint32_t)__half_as_ushort(__float2half(s)) | ((uint32_t)__half_as_ushort(__float2half(b)) << 16);
      *reinterpret_cast<uint32_t*>(rec + CB) = w;
    } else {
      *reinterpret_cast<float2*>(rec + CB) = make_float2(s, b);
    }
  }
}

// Table of a sort key (binary search over key_base[0..T]).
__device__ __forceinline__ int table_of_key(const int64_t* key_base, int T, uint32_t key) {
  int lo = 0, hi = T;  // key_base[lo] <= key < key_base[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if ((int64_t)key >= key_base[mid]) lo = mid; else hi = mid;
  }
  return lo;
}

// Global slot of table-local row r if resident, else -1 (the set's tags are
// compared with int4 loads when assoc is a multiple of 4).
__device__ __forceinline__ int32_t probe_slot(const Dev& dv, const TableDesc& td, int32_t r) {
  if (td.n_sets == 0) return -1;
  const int64_t set = (int64_t)((uint32_t)r % (uint32_t)td.n_sets);
  const int64_t base = td.slot_base + set * dv.assoc;
  const int32_t* tg = dv.tag + base;
  if ((dv.assoc & 3) == 0) {
    for (int w = 0; w < dv.assoc; w += 4) {
      const int4 v = *reinterpret_cast<const int4*>(tg + w);
      if (v.x == r) return (int32_t)(base + w);
      if (v.y == r) return (int32_t)(base + w + 1);
      if (v.z == r) return (int32_t)(base + w + 2);
      if (v.w == r) return (int32_t)(base + w + 3);
    }
  } else {
    for (int w = 0; w < dv.assoc; ++w)
      if (tg[w] == r) return (int32_t)(base + w);
  }
  return -1;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int lane = threadIdx.x & 63;
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

}  // namespace embc
