// State reset, uniform initialisation, and the forward pass:
// pooled[b][t] = sum over the bag of fetch(T_t, C_t, i) (Sec. 3 fetch operator).
#include <map>
#include <mutex>
#include <type_traits>

#include "emb_cache.h"
#include "embc_device.h"
#include "embc_dispatch.h"
#include "embc_sort.h"

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
  if (e == hipSuccess && d.acc_slot) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.acc_slot), 0u, d.total_slots, s);
  if (e == hipSuccess && d.acc_rows) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.acc_rows), 0u, d.total_rows, s);
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
// then nearest-even quantization of the row; its Adagrad accumulator (if any) to 0.
template <int D, int BITS, bool SB16>
__global__ __launch_bounds__(256) void k_init_uniform(Dev dv, float lo, float hi, uint64_t init_seed) {
  constexpr int LPR = Geo<D>::LPR;
  const int g = threadIdx.x & (LPR - 1);
  const int64_t ngroups = (int64_t)gridDim.x * blockDim.x / LPR;
  const float width = hi - lo;
  for (int64_t grow = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / LPR; grow < dv.total_rows;
       grow += ngroups) {
    const int t = table_of_row(dv, grow);
    const uint32_t r = (uint32_t)(grow - dv.desc[t].row_base);
    float u[8], x[8];
    uniforms_row<D>(init_seed, 0xFFFFFFFFu, (uint32_t)t, r, g, u);
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = __builtin_fmaf(u[i], width, lo);
    uint8_t* rec = rec_of<D, BITS, SB16>(dv, grow);
    quantize_store<D, BITS, SB16>(x, g, rec, false, 0, 0, 0, 0);
    if (dv.optimizer && g == 0) *acc_of<D, BITS, SB16>(dv, grow, rec) = 0.0f;
  }
}

// Row-wise Adagrad: the accumulators of the rows cached in slots [s0, s0 + n) of the table
// whose rows start at row_base, moved from the slots to the records (to_rec) or back.
__global__ __launch_bounds__(256) void k_move_acc(Dev dv, int64_t s0, int64_t n, int64_t row_base, bool to_rec) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const int32_t r = dv.tag[s0 + i];
    if (r < 0) continue;
    float* a = dv.acc_rows ? dv.acc_rows + row_base + r
                           : reinterpret_cast<float*>(dv.rec + (row_base + r) * dv.rec_bytes + dv.acc_offset);
    if (to_rec) *a = dv.acc_slot[s0 + i];
    else dv.acc_slot[s0 + i] = *a;
  }
}

hipError_t launch_move_acc(const Dev& d, int64_t slot0, int64_t slots, int64_t row_base, bool to_rec, hipStream_t s) {
  if (!d.acc_slot || slots <= 0) return hipSuccess;
  k_move_acc<<<grid_for(slots), 256, 0, s>>>(d, slot0, slots, row_base, to_rec);
  return hipGetLastError();
}

hipError_t launch_init_uniform(const Dev& d, float lo, float hi, uint64_t init_seed, hipStream_t s) {
  hipError_t e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.tag), 0xFFFFFFFFu, d.total_slots, s);
  if (e == hipSuccess && d.ts) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.ts), 0xFFFFFFFFu, d.total_slots, s);
  if (e == hipSuccess) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.crow), 0u, d.total_slots * d.dim, s);
  if (e == hipSuccess && d.cnt) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.cnt), 0u, d.total_rows, s);
  if (e == hipSuccess && d.acc_slot) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.acc_slot), 0u, d.total_slots, s);
  if (e == hipSuccess && d.acc_rows) e = launch_fill_u32(reinterpret_cast<uint32_t*>(d.acc_rows), 0u, d.total_rows, s);
  if (e != hipSuccess) return e;
  return dispatch_row(d.dim, d.bits, d.sb16, [&]<int D, int BITS, bool SB16>() -> hipError_t {
    const int64_t threads = d.total_rows * Geo<D>::LPR;
    k_init_uniform<D, BITS, SB16><<<grid_for(threads, 16384), 256, 0, s>>>(d, lo, hi, init_seed);
    return hipGetLastError();
  });
}

// ---- forward --------------------------------------------------------------------------
// Two passes.  k_fwd_probe: one lane per lookup up to 8 ways, 2 lanes for 16 or 32, 4 for 64
// (tables split over the XCDs), checks the row, probes its set, and write a code: the cache slot (hit), -2-row (miss) or
// -1 (skipped).  k_fwd_gather: one group of LPR
// lanes per bag (64/LPR bags per wave), tables split over the XCDs; lane j reads the
// code of position j of each chunk of LPR positions, the rows are fetched FU at a time
// (all FU loads issued before any is used) and summed left to right.  A bag with no
// valid lookup gives +0.
constexpr int kFwdUnroll = 2;

// Lookups in flight per lane group of the probe (PU).  On a large step 6 (96 tags per
// lane, 2 waves per SIMD) is faster than 4 at 4 waves (355 -> 332 us on the industrial
// workload; 8: 334 us, 12: 531 us); a step of few lookups wants the waves instead.
constexpr int kProbeUnroll = 6, kProbeUnrollSmall = 4;
constexpr int64_t kProbeSmallBelow = 1 << 21;  // lookups per call

// QL = assoc/W lanes share one lookup (W = assoc up to 8 ways, 8 at 16 ways, 16 beyond),
// each comparing W of the set's tags loaded 16 bytes at a time; every lane group keeps
// PU lookups in flight (all index loads, then all tag loads).  At 16 ways two lanes of 8
// tags are faster than one of 16 (industrial probe 331 -> 303 us: a wave's tag loads
// then touch 32 sets' lines each instead of 64), four of 4 slower (439 us); at 32 ways four
// lanes of 8 are slower than two of 16 (stress workload 86 -> 127 us).
template <int W, int PU>
__global__ __launch_bounds__(256) void k_fwd_probe(Dev dv, const int32_t* __restrict__ idx, int64_t L,
                                                   const int32_t* __restrict__ off, int32_t B,
                                                   int32_t* __restrict__ src) {
  const XcdSplit xs(dv.T);
  const int64_t tid = xs.unit * blockDim.x + threadIdx.x, stride = xs.units * blockDim.x;
  if (blockIdx.x == 0) {
    // positions outside every bag are skipped
    const int64_t first = min<int64_t>(max<int64_t>(off[0], 0), L);
    const int64_t last = min<int64_t>(max<int64_t>(off[(int64_t)dv.T * B], first), L);
    for (int64_t p = threadIdx.x; p < first; p += blockDim.x) src[p] = -1;
    for (int64_t p = last + threadIdx.x; p < L; p += blockDim.x) src[p] = -1;
  }
  const int A = dv.assoc;
  const int QL = A / W;  // 1 up to 16 ways, 2 or 4 for 32 or 64
  const int sub = threadIdx.x % QL;
  const int64_t ptid = tid / QL, pstride = stride / QL;
  for (int seg = xs.xcd; seg < xs.segments(dv.T); seg += kXcds) {
    const int t = seg / xs.parts;
    const TableDesc td = dv.desc[t];
    const int64_t a = min<int64_t>(max<int64_t>(off[(int64_t)t * B], 0), L);
    const int64_t b = min<int64_t>(max<int64_t>(off[(int64_t)(t + 1) * B], a), L);
    int64_t lo, hi;
    part_range(a, b, seg % xs.parts, xs.parts, lo, hi);
    const int32_t* tags = dv.tag + td.slot_base + sub * W;
    uint32_t ok = 0, hit = 0, bad = 0;
    // the index loads run one iteration ahead of the tag loads, and every load is
    // unconditional (a position past hi re-reads position lo, an invalid row probes
    // set 0), so an iteration's tags are waited for with the next indices in flight
    int32_t rn[PU];
    if (lo + ptid < hi) {
#pragma unroll
      for (int q = 0; q < PU; ++q) {
        const int64_t p = lo + ptid + q * pstride;
        rn[q] = idx[p < hi ? p : lo];
      }
    }
    for (int64_t p0 = lo + ptid; p0 < hi; p0 += pstride * PU) {
      int32_t r[PU], found[PU];
      bool valid[PU];
      int32_t tw[PU][W];
#pragma unroll
      for (int q = 0; q < PU; ++q) {
        r[q] = rn[q];
        valid[q] = p0 + q * pstride < hi && r[q] >= 0 && (int64_t)r[q] < td.N;
        found[q] = -1;
      }
      if (td.n_sets > 0) {
#pragma unroll
        for (int q = 0; q < PU; ++q) {
          const int64_t set = valid[q] ? (int64_t)mod_by((uint32_t)r[q], td.by_sets) : 0;
          const int32_t* tg = tags + set * A;
          if constexpr (W % 4 == 0) {
#pragma unroll
            for (int k = 0; k < W; k += 4) {
              const int4 v = *reinterpret_cast<const int4*>(tg + k);
              tw[q][k] = v.x; tw[q][k + 1] = v.y; tw[q][k + 2] = v.z; tw[q][k + 3] = v.w;
            }
          } else if constexpr (W == 2) {
            const int2 v = *reinterpret_cast<const int2*>(tg);
            tw[q][0] = v.x; tw[q][1] = v.y;
          } else {
            tw[q][0] = tg[0];
          }
        }
      }
      // the next iteration's indices
      {
        const int64_t pn = p0 + pstride * PU;
#pragma unroll
        for (int q = 0; q < PU; ++q) {
          const int64_t p = pn + q * pstride;
          rn[q] = idx[p < hi ? p : lo];
        }
      }
      if (td.n_sets > 0) {
#pragma unroll
        for (int q = 0; q < PU; ++q) {
          const int64_t set = valid[q] ? (int64_t)mod_by((uint32_t)r[q], td.by_sets) : 0;
#pragma unroll
          for (int k = 0; k < W; ++k)
            if (valid[q] && tw[q][k] == r[q]) found[q] = (int32_t)(td.slot_base + set * A + sub * W + k);
        }
      }
#pragma unroll
      for (int q = 0; q < PU; ++q) {
        for (int o = 1; o < QL; o <<= 1) found[q] = max(found[q], __shfl_xor(found[q], o, QL));
        const int64_t p = p0 + q * pstride;
        if (sub == 0 && p < hi) {
          src[p] = valid[q] ? (found[q] >= 0 ? found[q] : -2 - r[q]) : -1;
          ok += valid[q];
          hit += found[q] >= 0;
          bad += !valid[q];
        }
      }
    }
    // statistics of the segment: one atomic per wave and counter
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      ok += __shfl_xor(ok, o);
      hit += __shfl_xor(hit, o);
      bad += __shfl_xor(bad, o);
    }
    if ((threadIdx.x & 63) == 0) {
      unsigned long long* st = dv.stats + (int64_t)t * kNStat;
      if (ok) atomicAdd(st + kStLookups, (unsigned long long)ok);
      if (hit) atomicAdd(st + kStHitLookups, (unsigned long long)hit);
      if (bad) {
        atomicAdd(st + kStInvalidFwd, (unsigned long long)bad);
        atomicOr(dv.err, kErrIndex);
      }
    }
  }
}

template <int D, int BITS, bool SB16>
__global__ __launch_bounds__(256) void k_fwd_gather(Dev dv, const int32_t* __restrict__ src, int64_t L,
                                                    const int32_t* __restrict__ off, int32_t B,
                                                    float* __restrict__ out) {
  constexpr int LPR = Geo<D>::LPR, FU = kFwdUnroll;
  constexpr int GPB = 256 / LPR;
  const int64_t RB = dv.rec_bytes;
  const int g = threadIdx.x & (LPR - 1);
  const XcdSplit xs(dv.T);
  const int64_t gx = xs.unit * GPB + threadIdx.x / LPR, gstride = xs.units * GPB;
  for (int seg = xs.xcd; seg < xs.segments(dv.T); seg += kXcds) {
    const int t = seg / xs.parts;
    int64_t blo, bhi;
    part_range(0, B, seg % xs.parts, xs.parts, blo, bhi);
    const TableDesc td = dv.desc[t];
    const uint8_t* rec0 = dv.rec + td.row_base * RB;
    // codes outside this table's slots and rows are skipped (only malformed offsets
    // produce them); slots, rows and positions are below 2^31 (32-bit arithmetic)
    const int32_t slot_lo = (int32_t)td.slot_base, slot_hi = (int32_t)(td.slot_base + td.n_sets * dv.assoc);
    const int32_t nrows = (int32_t)td.N;
    if (blo + gx >= bhi) continue;
    // the offsets of the group's next bag are loaded one bag ahead, the codes of the
    // next LPR positions one chunk ahead (indices clamped so that the loads are
    // unconditional; a clamped load is not used)
    const int32_t* offt = off + (int64_t)t * B;
    int64_t o0 = offt[blo + gx], o1 = offt[blo + gx + 1];
    for (int64_t b = blo + gx; b < bhi; b += gstride) {
      const int64_t p0 = o0 < 0 ? 0 : o0;
      const int64_t p1 = o1 > L ? L : o1;
      const int64_t nb = min<int64_t>(b + gstride, bhi - 1);
      o0 = offt[nb];
      o1 = offt[nb + 1];
      // the sum starts from -0, the identity of IEEE addition (adding the first term
      // gives exactly that term, as in the seeded left-to-right sum); a bag without a
      // valid lookup gives +0
      float acc[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] = -0.0f;
      bool any = false;
      int32_t code_next = p0 + g < p1 ? src[p0 + g] : -1;
      for (int64_t pc = p0; pc < p1; pc += LPR) {
        const int n = (int)min<int64_t>(LPR, p1 - pc);
        const int32_t code = code_next;
        code_next = pc + LPR + g < p1 ? src[pc + LPR + g] : -1;
        for (int j = 0; j < n; j += FU) {
          float raw[FU][8];
          RecRaw<D, BITS, SB16> rr[FU];
          int kind[FU];  // 0 skip, 1 cache row, 2 low-precision row
#pragma unroll
          for (int q = 0; q < FU; ++q) {
            const int32_t cq = __shfl(code, j + q, LPR);
            kind[q] = 0;
            if (j + q < n) {
              if (cq >= slot_lo && cq < slot_hi) kind[q] = 1;
              else if (cq <= -2 && -2 - cq < nrows) kind[q] = 2;
            }
            if (kind[q] == 1) {
              load_row<D>(dv.crow + (int64_t)cq * D, g, raw[q]);
            } else if (kind[q] == 2) {
              const uint8_t* rec = static_cast<const uint8_t*>(
                  __builtin_assume_aligned(rec0 + (int64_t)(-2 - cq) * RB, Rec<D, BITS, SB16>::ALIGN));
              rr[q] = load_rec_raw<D, BITS, SB16>(rec, g);  // unpacked after the loads
            }
          }
#pragma unroll
          for (int q = 0; q < FU; ++q) {
            if (kind[q] == 0) continue;
            if (kind[q] == 2) {
              CodeWords<BITS> cw;
              SbWords<SB16> sbw;
              rec_words_unpack<D, BITS, SB16>(rr[q], cw, sbw);
              float sq, bq;
              decode_sb<SB16>(sbw, sq, bq);
              dequant8<BITS>(row_code_words<D, BITS>(cw, g), sq, bq, raw[q]);
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[i] = acc[i] + raw[q][i];
            any = true;
          }
        }
      }
      if (!any) {
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = 0.0f;
      }
      store_row_nt<D>(out + ((int64_t)b * dv.T + t) * D, g, acc);
    }
  }
}

__global__ void k_zero_fwd_stats(Dev dv) {
  for (int i = threadIdx.x; i < dv.T; i += blockDim.x) {
    dv.stats[(int64_t)i * kNStat + kStLookups] = 0;
    dv.stats[(int64_t)i * kNStat + kStHitLookups] = 0;
    dv.stats[(int64_t)i * kNStat + kStInvalidFwd] = 0;
  }
}

hipError_t launch_forward(const Dev& d, const Work& w, const int32_t* idx, int64_t L, const int32_t* off, int32_t B,
                          float* out, hipStream_t s) {
  k_zero_fwd_stats<<<1, 256, 0, s>>>(d);
  const int64_t nbags = (int64_t)d.T * B;
  if (nbags == 0) return hipGetLastError();
  k_check_offsets<<<grid_for(nbags, 2048), 256, 0, s>>>(d, off, nbags, L, w.ctr);
  if (L > 0) {
    const auto probe = [&](auto kernel) {
      kernel<<<resident_grid(reinterpret_cast<const void*>(kernel)), 256, 0, s>>>(d, idx, L, off, B, w.fwd_src);
    };
    const auto probe_w = [&](auto pu) {
      constexpr int PU = decltype(pu)::value;
      // tags per lane: the whole set up to 8 ways, 8 of 16 (two lanes per lookup), 16 beyond
      switch (d.assoc <= 8 ? d.assoc : d.assoc == 16 ? 8 : 16) {
        case 1: probe(k_fwd_probe<1, PU>); return hipSuccess;
        case 2: probe(k_fwd_probe<2, PU>); return hipSuccess;
        case 4: probe(k_fwd_probe<4, PU>); return hipSuccess;
        case 8: probe(k_fwd_probe<8, PU>); return hipSuccess;
        case 16: probe(k_fwd_probe<16, PU>); return hipSuccess;
        default: return hipErrorInvalidValue;
      }
    };
    const hipError_t e = L < kProbeSmallBelow ? probe_w(std::integral_constant<int, kProbeUnrollSmall>{})
                                              : probe_w(std::integral_constant<int, kProbeUnroll>{});
    if (e != hipSuccess) return e;
  }
  return dispatch_row(d.dim, d.bits, d.sb16, [&]<int D, int BITS, bool SB16>() -> hipError_t {
    // whole multiples of 8 workgroups (one per XCD), at most the resident count
    const int64_t wgs = (nbags * Geo<D>::LPR + 255) / 256;
    const int64_t cap = resident_grid(reinterpret_cast<const void*>(k_fwd_gather<D, BITS, SB16>));
    int64_t blocks = (wgs + 7) / 8 * 8;
    blocks = blocks < 8 ? 8 : (blocks > cap ? cap : blocks);
    k_fwd_gather<D, BITS, SB16><<<(unsigned)blocks, 256, 0, s>>>(d, w.fwd_src, L, off, B, out);
    return hipGetLastError();
  });
}

// ---- forward without a workspace ---------------------------------------------------------
// For callers that cannot allocate: the forward's per-call temporaries (the counter words
// written by the offset check, then one code per lookup) live in `scratch`, a static
// device array that every GPU the library runs on holds until the process ends.  Host
// code never passes the array's name to a kernel (on the host it is only a stand-in): it
// passes the device address that hipGetSymbolAddress returns for the current device,
// looked up once per device.
constexpr size_t kNoAllocHeader = 256;
static_assert(EMB_NOALLOC_MAX_INDICES == (EMB_NOALLOC_SCRATCH_BYTES - kNoAllocHeader) / 4, "scratch layout");
static_assert(kNCounters * sizeof(unsigned long long) <= kNoAllocHeader, "counter words");
static __device__ __align__(256) uint8_t scratch[EMB_NOALLOC_SCRATCH_BYTES];

hipError_t noalloc_scratch(uint8_t** out) {
  static std::mutex mu;
  static std::map<int, uint8_t*> addr;  // device -> address of its copy of `scratch`
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  const auto it = addr.find(dev);
  if (it != addr.end()) {
    *out = it->second;
    return hipSuccess;
  }
  void* p = nullptr;
  e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess || p == nullptr) return e != hipSuccess ? e : hipErrorInvalidSymbol;
  addr[dev] = static_cast<uint8_t*>(p);
  *out = static_cast<uint8_t*>(p);
  return hipSuccess;
}

hipError_t launch_forward_noalloc(const Dev& d, uint8_t* scratch_dev, const int32_t* idx, int64_t L,
                                  const int32_t* off, int32_t B, float* out, hipStream_t s) {
  if (scratch_dev == nullptr || L < 0 || L > EMB_NOALLOC_MAX_INDICES) return hipErrorInvalidValue;
  // the same kernels as launch_forward; nothing in the scratch is read before it is written
  // in the same call (the counter words are only written), so it needs no clearing
  Work w{};
  w.ctr = reinterpret_cast<unsigned long long*>(scratch_dev);
  w.fwd_src = reinterpret_cast<int32_t*>(scratch_dev + kNoAllocHeader);
  w.max_indices = EMB_NOALLOC_MAX_INDICES;
  return launch_forward(d, w, idx, L, off, B, out, s);
}

}  // namespace embc
