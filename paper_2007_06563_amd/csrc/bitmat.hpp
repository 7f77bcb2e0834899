// 32x32 bit-matrix transpose in registers, for moving 32 values out of the
// bitsliced (plane) order: before, bit j of a[i] is bit i of value j; after,
// bit i of a[j] is bit i of value j. Plain C++ so that the same code builds
// for the host (tests) and the device.
#pragma once
#include <stdint.h>

#if defined(__HIPCC__)
#define HOBFLOPS_HD __host__ __device__ __forceinline__
#else
#define HOBFLOPS_HD inline
#endif

namespace hobflops {

// Recursive block swap: at block size s the off-diagonal s x s blocks of
// every 2s x 2s block trade places (five rounds, s = 16, 8, 4, 2, 1).
HOBFLOPS_HD void transpose32(uint32_t (&a)[32]) {
  uint32_t m = 0x0000FFFFu;
#pragma unroll
  for (int s = 16; s != 0; s >>= 1, m ^= m << s) {
#pragma unroll
    for (int k = 0; k < 32; k = (k + s + 1) & ~s) {
      // rows k (low half of the pair) and k+s: swap a[k]'s high s-bit fields
      // with a[k+s]'s low ones
      const uint32_t t = ((a[k] >> s) ^ a[k + s]) & m;
      a[k + s] ^= t;
      a[k] ^= t << s;
    }
  }
}

}  // namespace hobflops
