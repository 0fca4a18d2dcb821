// Device-side building blocks of libembcache (gfx950, wave64).
//
// Lane layout of one embedding row of width D: a row is handled by a group of
// LPR = D/8 consecutive lanes (2..32), and lane g of the group holds 8 of its
// columns as elements 0..7: below d = 128 the contiguous columns [8g, 8g+8); from
// d = 128 on the split columns [4g, 4g+4) and [D/2+4g, D/2+4g+4) (kSplit), so that
// each 16-byte load or store of an FP32 row covers D/2 contiguous floats across the
// group (whole 128-byte lines), where 8 contiguous columns per lane touch every line
// of the row at half use in both.  An FP32 row is two 16-byte loads per lane, the
// 8 stochastic-rounding uniforms of a lane are the 8 words of two Philox blocks, and
// a wave works on 64/LPR rows at once.  The low-precision codes are stored with 8
// contiguous columns per lane-sized word (INT4: one dword, INT8: two, INT2: a
// half-word, FP16 elements: four dwords) and moved between the lanes of a group when
// the row is split.  The halving-tree sum pairs columns (j, j + h): contiguous
// lanes g and g ^ (h/8) while h >= 8, then inside a lane; split, inside a lane for
// h = D/2, then lanes g and g ^ (h/4) while h >= 4, then inside a lane.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <type_traits>
#include <stdint.h>

#include "embc_internal.h"

namespace embc {

template <int D>
struct Geo {
  static constexpr int CPL = 8;        // columns per lane (their layout: kSplit)
  static constexpr int LPR = D / CPL;  // lanes per row
  static constexpr int GPW = 64 / LPR; // rows per wave
};

template <int D>
constexpr bool kSplit = D >= 128;

// A row record of the low-precision table: the codes (BITS 8, 4, 2) followed by the
// row's (scale, bias), FP16 pair or FP32 pair; or, for BITS 16, the row's binary16
// elements alone.  Under row-wise Adagrad the row's FP32 accumulator follows at byte
// BYTES, and the record is padded to a multiple of ALIGN (the alignment BYTES has, at
// most 16), so that every record keeps the alignment of its code words.  The stride
// is Dev::rec_bytes.
template <int D, int BITS, bool SB16>
struct Rec {
  static constexpr int CODE_BYTES = D * BITS / 8;
  static constexpr int BYTES = CODE_BYTES + (BITS == 16 ? 0 : SB16 ? 4 : 8);
  static constexpr int ALIGN = (BYTES & -BYTES) < 16 ? (BYTES & -BYTES) : 16;
};

// Record of global row grow.
template <int D, int BITS, bool SB16>
__device__ __forceinline__ uint8_t* rec_of(const Dev& dv, int64_t grow) {
  return static_cast<uint8_t*>(__builtin_assume_aligned(dv.rec + grow * dv.rec_bytes, Rec<D, BITS, SB16>::ALIGN));
}

// The row-wise Adagrad accumulator of uncached row grow (record rec): inside the record,
// or in the per-row array when the records have no room for it.
template <int D, int BITS, bool SB16>
__device__ __forceinline__ float* acc_of(const Dev& dv, int64_t grow, uint8_t* rec) {
  return dv.acc_rows ? dv.acc_rows + grow : reinterpret_cast<float*>(rec + Rec<D, BITS, SB16>::BYTES);
}

// ---- lane exchange inside a row group ---------------------------------------------------
// x of lane (lane ^ M), for M < LPR.  Masks 1..8 stay inside a 16-lane DPP row and use
// DPP moves (quad permutations and row mirrors compose to every xor below 16):
//   ^1, ^2 = quad_perm [1,0,3,2], [2,3,0,1];  ^4 = half-row mirror (^7) after quad
//   reverse (^3);  ^8 = row mirror (^15) after half-row mirror (^7).
// Mask 16 (32-lane groups) goes through the LDS crossbar.
template <int M>
__device__ __forceinline__ float xor_lane(float x) {
  const int v = __float_as_int(x);
  if constexpr (M == 1) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false));
  } else if constexpr (M == 2) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false));
  } else if constexpr (M == 4) {
    const int r = __builtin_amdgcn_mov_dpp(v, 0x1B, 0xF, 0xF, false);
    return __int_as_float(__builtin_amdgcn_mov_dpp(r, 0x141, 0xF, 0xF, false));
  } else if constexpr (M == 8) {
    const int r = __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, false);
    return __int_as_float(__builtin_amdgcn_mov_dpp(r, 0x140, 0xF, 0xF, false));
  } else {
    static_assert(M == 16, "lane groups are at most 32 lanes");
    return __shfl_xor(x, 16, 32);
  }
}

// Applies op(x, xor_lane<M>(x)) for M = LPR/2, ..., 1 (a butterfly over the row group).
template <int LPR, typename Op>
__device__ __forceinline__ float butterfly(float x, Op op) {
  if constexpr (LPR > 16) x = op(x, xor_lane<16>(x));
  if constexpr (LPR > 8) x = op(x, xor_lane<8>(x));
  if constexpr (LPR > 4) x = op(x, xor_lane<4>(x));
  if constexpr (LPR > 2) x = op(x, xor_lane<2>(x));
  if constexpr (LPR > 1) x = op(x, xor_lane<1>(x));
  return x;
}

// ---- Philox4x32-10 (Salmon et al., SC'11): 10 rounds, Weyl key schedule -------------
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int i = 0; i < 10; ++i) {
    // one 32x32 -> 64-bit product per multiplier (a single v_mad_u64_u32 each)
    const uint64_t p0 = (uint64_t)0xD2511F53u * c.x, p1 = (uint64_t)0xCD9E8D57u * c.z;
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

__device__ __forceinline__ float u24(uint32_t w) { return (float)(w >> 8) * 5.9604644775390625e-08f; }  // 2^-24

// The 8 uniforms of lane g's columns of (table, row) at `step`: column j uses word j%4
// of the block with counter (j/4, row, table, step) and key (seed lo, seed hi).
template <int D>
__device__ __forceinline__ void uniforms_row(uint64_t seed, uint32_t step, uint32_t table, uint32_t row, int g,
                                             float (&u)[8]) {
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  const uint32_t c0 = kSplit<D> ? (uint32_t)g : 2u * g, c1 = kSplit<D> ? (uint32_t)(D / 8 + g) : 2u * g + 1u;
  const uint4 a = philox4x32_10(make_uint4(c0, row, table, step), k0, k1);
  const uint4 b = philox4x32_10(make_uint4(c1, row, table, step), k0, k1);
  u[0] = u24(a.x); u[1] = u24(a.y); u[2] = u24(a.z); u[3] = u24(a.w);
  u[4] = u24(b.x); u[5] = u24(b.y); u[6] = u24(b.z); u[7] = u24(b.w);
}

// The compiler may fuse an FP32 multiply-add with a following conversion to FP16
// (v_fma_mix*), rounding once instead of twice; the empty asm keeps the FP32 value
// as an operand of its own so that the conversion rounds that value.
__device__ __forceinline__ float as_f32_value(float x) {
  asm volatile("" : "+v"(x));
  return x;
}

__device__ __forceinline__ float f16_round(float x) { return __half2float(__float2half(as_f32_value(x))); }

// Scale and bias words of a record, loaded raw so that a caller can issue further loads
// before it converts them (decode_sb).
template <bool SB16>
struct SbWords {
  uint32_t w[SB16 ? 1 : 2];
};

template <int D, int BITS, bool SB16>
__device__ __forceinline__ SbWords<SB16> load_sb_words(const uint8_t* rec) {
  constexpr int CB = Rec<D, BITS, SB16>::CODE_BYTES;
  SbWords<SB16> r;
  if constexpr (BITS == 16) {  // an FP16 table has no (s, b)
    r.w[0] = 0u;
    if constexpr (!SB16) r.w[1] = 0u;
    return r;
  }
  const uint32_t* p = reinterpret_cast<const uint32_t*>(rec + CB);
  r.w[0] = p[0];
  if constexpr (!SB16) r.w[1] = p[1];
  return r;
}

template <bool SB16>
__device__ __forceinline__ void decode_sb(const SbWords<SB16>& r, float& s, float& b) {
  if constexpr (SB16) {
    s = __half2float(__ushort_as_half((unsigned short)(r.w[0] & 0xFFFFu)));
    b = __half2float(__ushort_as_half((unsigned short)(r.w[0] >> 16)));
  } else {
    s = __uint_as_float(r.w[0]);
    b = __uint_as_float(r.w[1]);
  }
}


// Raw code words of lane g: INT2 one half-word (column 8g+i in bits 2i..2i+1), INT4
// one dword (column 8g+i in nibble i), INT8 two dwords (column 8g+i in byte i), FP16
// four dwords (column 8g+i in half i%2 of dword i/2).
template <int BITS>
struct CodeWords {
  static constexpr int N = BITS == 16 ? 4 : BITS == 8 ? 2 : 1;  // dwords per lane
  uint32_t w[N];
};

template <int BITS, bool NT = false>
__device__ __forceinline__ CodeWords<BITS> load_code_words(const uint8_t* rec, int g) {
  CodeWords<BITS> c;
  if constexpr (BITS == 2) {
    const uint16_t* p = reinterpret_cast<const uint16_t*>(rec) + g;
    if constexpr (NT) c.w[0] = __builtin_nontemporal_load(p);
    else c.w[0] = p[0];
  } else {
    const uint32_t* p = reinterpret_cast<const uint32_t*>(rec) + g * CodeWords<BITS>::N;
#pragma unroll
    for (int i = 0; i < CodeWords<BITS>::N; ++i) {
      if constexpr (NT) c.w[i] = __builtin_nontemporal_load(p + i);
      else c.w[i] = p[i];
    }
  }
  return c;
}

// The raw words of a record that lane g needs: its code words (as load_code_words
// returns them) and the record's (scale, bias) words, unpacked by rec_words_unpack once
// they are needed (so that further loads can be issued first).  INT8: one load per lane
// that reads the dwords from the first of its own code words on, one or two (the
// (scale, bias) words) more than it needs, so that the last lane of the group reads the
// (scale, bias) that follow the codes and the other lanes take them from it; every
// dword read lies inside the record's codes and (scale, bias), and each read is dword
// aligned (one vector load of 3 or 4 dwords).  That is done for INT8 rows of d >= 128
// (the gather of 256-column rows: 0.46 -> 0.44 ms); INT4 and INT2 load the codes and
// the (scale, bias) apart (the widened load was slower there: 128-column INT4 rows
// 1.84 -> 1.90 ms), and so do narrower INT8 rows.  FP16: the code words.
template <int N>
struct alignas(4) DWords {
  uint32_t w[N];
};

template <int D, int BITS, bool SB16>
struct RecRaw {
  static constexpr bool kOneLoad = BITS == 8 && kSplit<D>;
  static constexpr int SBW = SB16 ? 1 : 2;  // (scale, bias) dwords
  DWords<kOneLoad ? 2 + SBW : 1> v;         // INT8: code words, then (scale, bias) words
  CodeWords<BITS> c;                        // the others
  SbWords<SB16> sb;
};

template <int D, int BITS, bool SB16>
__device__ __forceinline__ RecRaw<D, BITS, SB16> load_rec_raw(const uint8_t* rec, int g) {
  using R = RecRaw<D, BITS, SB16>;
  R r;
  if constexpr (R::kOneLoad) {
    r.v = *reinterpret_cast<const DWords<2 + R::SBW>*>(rec + 8 * g);
  } else {
    r.c = load_code_words<BITS>(rec, g);
    if constexpr (BITS != 16) r.sb = load_sb_words<D, BITS, SB16>(rec);
  }
  return r;
}

// Every lane of the group must take part.
template <int D, int BITS, bool SB16>
__device__ __forceinline__ void rec_words_unpack(const RecRaw<D, BITS, SB16>& r, CodeWords<BITS>& c,
                                                 SbWords<SB16>& sb) {
  using R = RecRaw<D, BITS, SB16>;
  if constexpr (R::kOneLoad) {
    constexpr int LPR = Geo<D>::LPR;
    c.w[0] = r.v.w[0];
    c.w[1] = r.v.w[1];
#pragma unroll
    for (int i = 0; i < R::SBW; ++i) sb.w[i] = __shfl(r.v.w[2 + i], LPR - 1, LPR);
  } else {
    c = r.c;
    sb = r.sb;
  }
}

// Stores lane g's code words of 8 contiguous columns (the layout of load_code_words;
// w1 only for INT8), nontemporal: a record is written once per step.
template <int BITS>
__device__ __forceinline__ void store_code_words(uint8_t* rec, int g, uint32_t w0, uint32_t w1) {
  if constexpr (BITS == 2) {
    __builtin_nontemporal_store((uint16_t)w0, reinterpret_cast<uint16_t*>(rec) + g);
  } else {
    uint32_t* p = reinterpret_cast<uint32_t*>(rec) + g * (BITS == 8 ? 2 : 1);
    __builtin_nontemporal_store(w0, p);
    if constexpr (BITS == 8) __builtin_nontemporal_store(w1, p + 1);
  }
}

// The codes of lane g's split columns, from the words of load_code_words (8 contiguous
// columns per lane) moved between the group's lanes and packed as those are (element i
// is column 4g+i for i < 4, D/2+4g+i-4 after): lane g's columns are half g%2 of lanes
// g/2 and LPR/2 + g/2.  Every lane of the group must take part.
template <int D, int BITS>
__device__ __forceinline__ CodeWords<BITS> split_code_words(const CodeWords<BITS>& c8, int g) {
  constexpr int LPR = Geo<D>::LPR;
  const int s0 = g >> 1, s1 = LPR / 2 + (g >> 1), h = g & 1;
  CodeWords<BITS> c;
  if constexpr (BITS == 2 || BITS == 4) {
    constexpr int HB = 4 * BITS;  // bits of 4 columns
    const uint32_t m = (1u << HB) - 1u;
    const uint32_t a = (__shfl(c8.w[0], s0, LPR) >> (HB * h)) & m;
    const uint32_t b = (__shfl(c8.w[0], s1, LPR) >> (HB * h)) & m;
    c.w[0] = a | (b << HB);
  } else if constexpr (BITS == 8) {
    const uint32_t a0 = __shfl(c8.w[0], s0, LPR), a1 = __shfl(c8.w[1], s0, LPR);
    const uint32_t b0 = __shfl(c8.w[0], s1, LPR), b1 = __shfl(c8.w[1], s1, LPR);
    c.w[0] = h ? a1 : a0;
    c.w[1] = h ? b1 : b0;
  } else {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint32_t a0 = __shfl(c8.w[i], s0, LPR), a1 = __shfl(c8.w[2 + i], s0, LPR);
      const uint32_t b0 = __shfl(c8.w[i], s1, LPR), b1 = __shfl(c8.w[2 + i], s1, LPR);
      c.w[i] = h ? a1 : a0;
      c.w[2 + i] = h ? b1 : b0;
    }
  }
  return c;
}

// The codes of lane g's split columns loaded in place, packed as split_code_words packs
// them: INT2/INT4 the 4 columns [4g, 4g+4) are byte/half-word g and [D/2+4g, D/2+4g+4)
// byte/half-word D/8+g (a | b << 4*BITS); INT8 dwords g and D/8+g; FP16 dwords 2g, 2g+1
// and D/4+2g, D/4+2g+1.
template <int D, int BITS, bool NT = false>
__device__ __forceinline__ CodeWords<BITS> load_split_code_words(const uint8_t* rec, int g) {
  const auto ld = [](const auto* p) {
    if constexpr (NT) return (uint32_t)__builtin_nontemporal_load(p);
    else return (uint32_t)p[0];
  };
  CodeWords<BITS> c;
  if constexpr (BITS == 2 || BITS == 4) {
    using W = std::conditional_t<BITS == 2, uint8_t, uint16_t>;
    const W* p = reinterpret_cast<const W*>(rec);
    c.w[0] = ld(p + g) | (ld(p + D / 8 + g) << (4 * BITS));
  } else if constexpr (BITS == 8) {
    const uint32_t* p = reinterpret_cast<const uint32_t*>(rec);
    c.w[0] = ld(p + g);
    c.w[1] = ld(p + D / 8 + g);
  } else {
    const uint32_t* p = reinterpret_cast<const uint32_t*>(rec);
    c.w[0] = ld(p + 2 * g);
    c.w[1] = ld(p + 2 * g + 1);
    c.w[2] = ld(p + D / 4 + 2 * g);
    c.w[3] = ld(p + D / 4 + 2 * g + 1);
  }
  return c;
}

// Stores lane g's split codes (packed as load_split_code_words returns them) in place,
// nontemporal.
template <int D, int BITS>
__device__ __forceinline__ void store_split_code_words(uint8_t* rec, int g, const CodeWords<BITS>& c) {
  if constexpr (BITS == 2 || BITS == 4) {
    using W = std::conditional_t<BITS == 2, uint8_t, uint16_t>;
    constexpr int HB = 4 * BITS;
    W* p = reinterpret_cast<W*>(rec);
    __builtin_nontemporal_store((W)(c.w[0] & ((1u << HB) - 1u)), p + g);
    __builtin_nontemporal_store((W)(c.w[0] >> HB), p + D / 8 + g);
  } else if constexpr (BITS == 8) {
    uint32_t* p = reinterpret_cast<uint32_t*>(rec);
    __builtin_nontemporal_store(c.w[0], p + g);
    __builtin_nontemporal_store(c.w[1], p + D / 8 + g);
  } else {
    uint32_t* p = reinterpret_cast<uint32_t*>(rec);
    __builtin_nontemporal_store(c.w[0], p + 2 * g);
    __builtin_nontemporal_store(c.w[1], p + 2 * g + 1);
    __builtin_nontemporal_store(c.w[2], p + D / 4 + 2 * g);
    __builtin_nontemporal_store(c.w[3], p + D / 4 + 2 * g + 1);
  }
}

// The codes of lane g's columns in the row layout of width D (element i in the slot
// of column 8g+i of load_code_words).  Every lane of the group must take part.
template <int D, int BITS>
__device__ __forceinline__ CodeWords<BITS> row_code_words(const CodeWords<BITS>& c8, int g) {
  if constexpr (kSplit<D>) return split_code_words<D, BITS>(c8, g);
  else return c8;
}

template <int BITS>
__device__ __forceinline__ uint32_t code_of(const CodeWords<BITS>& c, int i) {
  if constexpr (BITS == 8) return (c.w[i >> 2] >> (8 * (i & 3))) & 0xFFu;
  else if constexpr (BITS == 4) return (c.w[0] >> (4 * i)) & 0xFu;
  else return (c.w[0] >> (2 * i)) & 0x3u;
}

// Up-conversion of lane g's 8 elements: q*s + b with one rounding (Alg. 1), or the
// exact widening of binary16 elements (s, b unused).
template <int BITS>
__device__ __forceinline__ void dequant8(const CodeWords<BITS>& c, float s, float b, float (&x)[8]) {
  if constexpr (BITS == 16) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
      x[i] = __half2float(__ushort_as_half((unsigned short)(c.w[i >> 1] >> (16 * (i & 1)))));
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = __builtin_fmaf((float)code_of<BITS>(c, i), s, b);
  }
}

// Nontemporal forms for data touched once per kernel (a row fetched and written back,
// a pooled output): the hint keeps such lines from displacing, in L2, the lines that
// other lanes still read (gradient rows, hot cache rows).
typedef float f4v __attribute__((ext_vector_type(4)));

// Lane g's 8 elements of an FP32 row in the row layout of width D: the 16-byte words
// (g, g + D/8) when split, (2g, 2g + 1) otherwise.
template <int D>
__device__ __forceinline__ void load_row(const float* row, int g, float (&x)[8]) {
  const float4* p = reinterpret_cast<const float4*>(row);
  const int i0 = kSplit<D> ? g : 2 * g, i1 = kSplit<D> ? D / 8 + g : 2 * g + 1;
  const float4 a = p[i0], b = p[i1];
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}

template <int D>
__device__ __forceinline__ void load_row_nt(const float* row, int g, float (&x)[8]) {
  const f4v* p = reinterpret_cast<const f4v*>(row);
  const int i0 = kSplit<D> ? g : 2 * g, i1 = kSplit<D> ? D / 8 + g : 2 * g + 1;
  const f4v a = __builtin_nontemporal_load(p + i0), b = __builtin_nontemporal_load(p + i1);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}

template <int D>
__device__ __forceinline__ void store_row(float* row, int g, const float (&x)[8]) {
  float4* p = reinterpret_cast<float4*>(row);
  const int i0 = kSplit<D> ? g : 2 * g, i1 = kSplit<D> ? D / 8 + g : 2 * g + 1;
  p[i0] = make_float4(x[0], x[1], x[2], x[3]);
  p[i1] = make_float4(x[4], x[5], x[6], x[7]);
}

template <int D>
__device__ __forceinline__ void store_row_nt(float* row, int g, const float (&x)[8]) {
  f4v* p = reinterpret_cast<f4v*>(row);
  const int i0 = kSplit<D> ? g : 2 * g, i1 = kSplit<D> ? D / 8 + g : 2 * g + 1;
  __builtin_nontemporal_store(f4v{x[0], x[1], x[2], x[3]}, p + i0);
  __builtin_nontemporal_store(f4v{x[4], x[5], x[6], x[7]}, p + i1);
}

// The binary16 value next to h in increasing (up) or decreasing order, h finite:
// magnitudes are ordered like their bit patterns, the sign flips the direction, and
// both zeros step to the smallest subnormal of the direction.
__device__ __forceinline__ uint32_t f16_next(uint32_t h, bool up) {
  const uint32_t sign = h & 0x8000u, mag = h & 0x7FFFu;
  if (mag == 0) return up ? 0x0001u : 0x8001u;
  return sign | (((sign == 0) == up) ? mag + 1u : mag - 1u);
}

// Down-conversion of x into binary16 bits (Sec. 3 "Rounding" with FP16 as the low
// precision): nearest even (IEEE, overflow to infinity), or stochastic between the
// consecutive finite values x- <= x <= x+, taking x+ when u < (x - x-)/(x+ - x-)
// (exact: neighbours differ by a power of two); beyond 65504 stochastic rounding
// saturates; a representable x or a NaN is kept.
__device__ __forceinline__ uint32_t f16_bits_round(float x, bool sr, float u) {
  x = as_f32_value(x);
  const uint32_t h = (uint32_t)__half_as_ushort(__float2half_rn(x));
  if (!sr || x != x) return h;
  if (x > 65504.0f) return 0x7BFFu;
  if (x < -65504.0f) return 0xFBFFu;
  const float y = __half2float(__ushort_as_half((unsigned short)h));
  if (y == x) return h;
  const uint32_t lo_h = y < x ? h : f16_next(h, false), hi_h = y < x ? f16_next(h, true) : h;
  const float lo = __half2float(__ushort_as_half((unsigned short)lo_h));
  const float hi = __half2float(__ushort_as_half((unsigned short)hi_h));
  return (u < (x - lo) / (hi - lo)) ? hi_h : lo_h;
}

// Down-conversion of one FP32 row into its low-precision record (Alg. 1 with the
// Sec. 3 rounding knob).  Integer codes: b = min, s = (max - min)/(2^BITS - 1)
// (FP32, correctly rounded; then rounded to FP16 when SB16); codes
// q = round((x - b)/s) clamped to [0, 2^BITS - 1], all zero when s == 0; a -0
// extreme is taken as +0.  FP16 table: each element by f16_bits_round.  A record is
// written once per step (nontemporal stores).  x holds lane g's columns in the row
// layout of width D, and a split row's codes are stored in place.  Every lane of the
// group must take part (the row's minimum and maximum).
template <int D, int BITS, bool SB16>
__device__ __forceinline__ void quantize_store(const float (&x)[8], int g, uint8_t* rec, bool sr, uint64_t seed,
                                               uint32_t step, uint32_t table, uint32_t row) {
  if constexpr (BITS == 16) {
    float u[8];
    if (sr) uniforms_row<D>(seed, step, table, row, g, u);
    uint32_t h2[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t lo = f16_bits_round(x[2 * i], sr, sr ? u[2 * i] : 0.0f);
      const uint32_t hi = f16_bits_round(x[2 * i + 1], sr, sr ? u[2 * i + 1] : 0.0f);
      h2[i] = lo | (hi << 16);
    }
    if constexpr (kSplit<D>) {
      store_split_code_words<D, 16>(rec, g, CodeWords<16>{{h2[0], h2[1], h2[2], h2[3]}});
    } else {
      uint32_t* p = reinterpret_cast<uint32_t*>(rec);
#pragma unroll
      for (int i = 0; i < 4; ++i) __builtin_nontemporal_store(h2[i], p + 4 * g + i);
    }
    return;
  }
  constexpr int LPR = Geo<D>::LPR;
  constexpr int CB = Rec<D, BITS, SB16>::CODE_BYTES;
  constexpr float K = (float)((1 << BITS) - 1);
  float mn = x[0], mx = x[0];
#pragma unroll
  for (int i = 1; i < 8; ++i) {
    mn = fminf(mn, x[i]);
    mx = fmaxf(mx, x[i]);
  }
  mn = butterfly<LPR>(mn, [](float a, float b) { return fminf(a, b); });
  mx = butterfly<LPR>(mx, [](float a, float b) { return fmaxf(a, b); });
  mn = mn + 0.0f;
  mx = mx + 0.0f;
  float s = (mx - mn) / K;
  float b = mn;
  if constexpr (SB16) {
    s = f16_round(s);
    b = f16_round(b);
  }
  float u[8];
  if (sr && s != 0.0f) uniforms_row<D>(seed, step, table, row, g, u);
  uint32_t w0 = 0, w1 = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float qf = 0.0f;
    if (s != 0.0f) {
      const float v = (x[i] - b) / s;
      if (sr) {
        const float f = floorf(v);
        qf = (u[i] < v - f) ? f + 1.0f : f;
      } else {
        qf = rintf(v);
      }
      qf = qf < 0.0f ? 0.0f : qf;
      qf = qf > K ? K : qf;
    }
    const uint32_t q = (uint32_t)qf;
    if constexpr (BITS == 8) {
      if (i < 4) w0 |= q << (8 * i);
      else w1 |= q << (8 * (i - 4));
    } else {
      w0 |= q << (BITS * i);
    }
  }
  if constexpr (kSplit<D>) {
    CodeWords<BITS> c;
    c.w[0] = w0;
    if constexpr (BITS == 8) c.w[1] = w1;
    store_split_code_words<D, BITS>(rec, g, c);
  } else {
    store_code_words<BITS>(rec, g, w0, w1);
  }
  if (g == 0) {
    uint32_t* ps = reinterpret_cast<uint32_t*>(rec + CB);
    if constexpr (SB16) {
      ps[0] = (uint32_t)__half_as_ushort(__float2half(s)) | ((uint32_t)__half_as_ushort(__float2half(b)) << 16);
    } else {
      ps[0] = __float_as_uint(s);
      ps[1] = __float_as_uint(b);
    }
  }
}

// n / d and n % d for a DivConst (exact for every 32-bit n).
__device__ __forceinline__ uint32_t div_by(uint32_t n, const DivConst& c) {
  const uint32_t t = __umulhi(c.m, n);
  return (t + ((n - t) >> c.s1)) >> c.s2;
}
__device__ __forceinline__ uint32_t mod_by(uint32_t n, const DivConst& c) { return n - div_by(n, c) * c.d; }

// Table of a sort key (binary search over key_base[0..T]).
__device__ __forceinline__ int table_of_key(const int64_t* key_base, int T, uint32_t key) {
  int lo = 0, hi = T;  // key_base[lo] <= key < key_base[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if ((int64_t)key >= key_base[mid]) lo = mid; else hi = mid;
  }
  return lo;
}

// Global slot of table-local row r if resident, else -1.  All of the set's tags are
// loaded before any is compared (16 bytes at a time when assoc is a multiple of 4), so a
// probe waits for one round of loads rather than one per 16 bytes.
template <int A>
__device__ __forceinline__ int32_t probe_set(const int32_t* __restrict__ tg, int32_t r) {
  int32_t v[A];
  if constexpr (A % 4 == 0) {
#pragma unroll
    for (int w = 0; w < A; w += 4) {
      const int4 q = *reinterpret_cast<const int4*>(tg + w);
      v[w] = q.x; v[w + 1] = q.y; v[w + 2] = q.z; v[w + 3] = q.w;
    }
  } else {
#pragma unroll
    for (int w = 0; w < A; ++w) v[w] = tg[w];
  }
  int32_t found = -1;
#pragma unroll
  for (int w = 0; w < A; ++w) found = v[w] == r ? w : found;
  return found;
}

__device__ __forceinline__ int32_t probe_slot(const Dev& dv, const TableDesc& td, int32_t r) {
  if (td.n_sets == 0) return -1;
  const int64_t set = (int64_t)mod_by((uint32_t)r, td.by_sets);
  const int64_t base = td.slot_base + set * dv.assoc;
  const int32_t* tg = dv.tag + base;
  int32_t w = -1;
  switch (dv.assoc) {
    case 1: w = probe_set<1>(tg, r); break;
    case 2: w = probe_set<2>(tg, r); break;
    case 4: w = probe_set<4>(tg, r); break;
    case 8: w = probe_set<8>(tg, r); break;
    case 16: w = probe_set<16>(tg, r); break;
    case 32: w = probe_set<32>(tg, r); break;
    default: w = probe_set<64>(tg, r); break;
  }
  return w >= 0 ? (int32_t)(base + w) : -1;
}

// XCD-aware work split.  Workgroups are dispatched round-robin over the 8 XCDs
// (workgroup i on XCD i % 8), each with its own L2.  Work is cut into T*P segments
// (table t, part p; P parts per table so that there are at least 8 segments) and
// XCD x takes segments x, x+8, ...; inside an XCD, its workgroups share a segment.
// Every segment sees the same L2, so a table's hot cache rows, tags and gradient
// rows are fetched into one L2 instead of eight.  With `even`, P makes T*P a
// multiple of 8, so every XCD gets the same number of segments (e.g. 100 tables:
// 2 parts, 25 segments per XCD instead of 13 or 12 tables); kernels whose reads
// are mostly private to a row take that, those that share a table's lines across
// rows (tags, gradient rows) keep one part per table.
constexpr int kXcds = 8;

struct XcdSplit {
  int xcd;          // this workgroup's XCD
  int64_t unit;     // this workgroup's index among the XCD's workgroups
  int64_t units;    // workgroups per XCD
  int parts;        // parts per table
  __device__ XcdSplit(int T, bool even = false) {
    xcd = blockIdx.x % kXcds;
    unit = blockIdx.x / kXcds;
    units = gridDim.x / kXcds;
    if (even) parts = kXcds / min(T & -T, kXcds);
    else parts = T >= kXcds ? 1 : (kXcds + T - 1) / T;
  }
  __device__ int segments(int T) const { return T * parts; }
};

// Row groups over the segments an XCD handles in turn: a segment with at least as many
// items as there are groups starts at group 0 (consecutive groups take consecutive
// items), but a smaller one starts where the previous small segments left off, so that
// small segments (small tables) spread over all groups instead of all landing on the
// first ones, one after another.  Returns the group's first item offset in the segment
// (>= n when it has none) and advances `carry` past the segment.
// (carry stays below gstride; gx < gstride; 32-bit, no division, so that the per-lane cost
// is one compare and a subtract)
__device__ __forceinline__ int64_t spread_start(int64_t gx, int64_t gstride, int64_t n, int64_t& carry) {
  if (n >= gstride) return gx;
  const int32_t c = (int32_t)carry, gs = (int32_t)gstride;
  int32_t s = (int32_t)gx + gs - c;
  if (s >= gs) s -= gs;
  carry += n;
  if (carry >= gstride) carry -= gstride;
  return s;
}

// [lo, hi) of `part` out of `parts` equal slices of [a, b).
__device__ __forceinline__ void part_range(int64_t a, int64_t b, int part, int parts, int64_t& lo, int64_t& hi) {
  const int64_t n = b - a;
  lo = a + n * part / parts;
  hi = a + n * (part + 1) / parts;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int lane = threadIdx.x & 63;
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

}  // namespace embc
