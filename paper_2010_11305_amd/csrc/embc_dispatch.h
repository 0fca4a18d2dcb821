// Compile-time specialisation of the row kernels on (dim, bits, FP16 scale/bias).
#pragma once

#include <hip/hip_runtime.h>

namespace embc {

// Calls fn.template operator()<D, BITS, SB16>() for the runtime triple (BITS 16 is an
// FP16 table, which has no scale/bias: SB16 is false).
template <typename Fn>
hipError_t dispatch_row(int dim, int bits, int sb16, Fn&& fn) {
#define EMBC_DISPATCH_DIM(DD)                                                            \
  case DD:                                                                               \
    if (bits == 16) return fn.template operator()<DD, 16, false>();                      \
    if (bits == 8) return sb16 ? fn.template operator()<DD, 8, true>()                   \
                               : fn.template operator()<DD, 8, false>();                 \
    if (bits == 4) return sb16 ? fn.template operator()<DD, 4, true>()                   \
                               : fn.template operator()<DD, 4, false>();                 \
    if (bits == 2) return sb16 ? fn.template operator()<DD, 2, true>()                   \
                               : fn.template operator()<DD, 2, false>();                 \
    return hipErrorInvalidValue;
  switch (dim) {
    EMBC_DISPATCH_DIM(16)
    EMBC_DISPATCH_DIM(32)
    EMBC_DISPATCH_DIM(64)
    EMBC_DISPATCH_DIM(128)
    EMBC_DISPATCH_DIM(256)
    default:
      return hipErrorInvalidValue;
  }
#undef EMBC_DISPATCH_DIM
}

// Blocks of a grid-stride kernel: as many as are resident at once on the current
// device (occupancy x compute units, for `threads` per block and no dynamic LDS),
// rounded down to a multiple of the 8 XCDs.  The whole grid then runs in one round;
// a larger grid would leave its last blocks running alone after the others end.
unsigned resident_grid(const void* kernel, int threads = 256);

inline unsigned grid_for(int64_t threads, int64_t cap = 8192) {
  int64_t b = (threads + 255) / 256;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (unsigned)b;
}

}  // namespace embc
