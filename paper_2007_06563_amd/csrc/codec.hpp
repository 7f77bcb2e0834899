// Conversions between float32 and codes of a (wE, wF) format, per value: the
// quantiser of the pack kernel and the decoder of the unpack kernel and of the
// convolution's float32 epilogue.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hobflops {

// float32 bits -> code of (wE, wF): the exact value rounded to nearest even
// with an unbounded exponent, then range checked (no subnormals in the format).
__device__ __forceinline__ uint32_t quantize_bits(uint32_t bits, int wE, int wF) {
  const uint32_t s = bits >> 31;
  const uint32_t ef = (bits >> 23) & 0xFFu;
  const uint32_t fr = bits & 0x7FFFFFu;
  const int sh_x = wF + wE + 1, sh_s = wF + wE;
  if (ef == 0xFFu) return fr ? (3u << sh_x) : ((2u << sh_x) | (s << sh_s));
  if (ef == 0 && fr == 0) return s << sh_s;
  uint32_t M;
  int u;  // value = M * 2^(u - 23) with M in [2^23, 2^24)
  if (ef) {
    M = fr | 0x800000u;
    u = (int)ef - 127;
  } else {
    const int lz = __clz(fr) - 8;  // fr < 2^23
    M = fr << lz;
    u = -126 - lz;
  }
  const int k = 23 - wF;  // dropped bits, 0..22
  uint32_t q = M >> k;
  if (k > 0) {
    const uint32_t rem = M & ((1u << k) - 1u);
    const uint32_t half = 1u << (k - 1);
    if (rem > half || (rem == half && (q & 1u))) q += 1u;
    if (q == (2u << wF)) {
      q >>= 1;
      u += 1;
    }
  }
  const int Eb = u + (1 << (wE - 1)) - 1;
  if (Eb > (1 << wE) - 1) return (2u << sh_x) | (s << sh_s);
  if (Eb < 0) return s << sh_s;
  return (1u << sh_x) | (s << sh_s) | ((uint32_t)Eb << wF) | (q & ((1u << wF) - 1u));
}

// code of (wE, wF) -> float32 bits (exact unless wE = 8 reaches float32's
// subnormal or overflow range, then rounded to nearest even).
__device__ __forceinline__ uint32_t decode_bits(uint32_t code, int wE, int wF) {
  const uint32_t F = code & ((1u << wF) - 1u);
  const int E = (int)((code >> wF) & ((1u << wE) - 1u));
  const uint32_t s = (code >> (wF + wE)) & 1u;
  const uint32_t x = (code >> (wF + wE + 1)) & 3u;
  if (x == 3u) return 0x7FC00000u;
  if (x == 2u) return (s << 31) | 0x7F800000u;
  if (x == 0u) return s << 31;
  const int e = E - ((1 << (wE - 1)) - 1) + 127;  // float32 biased exponent
  if (e >= 255) return (s << 31) | 0x7F800000u;
  if (e >= 1) return (s << 31) | ((uint32_t)e << 23) | (F << (23 - wF));
  // float32 subnormal: value / 2^-149 = (2^wF + F) * 2^(e + 22 - wF)
  const uint32_t M = (1u << wF) | F;
  const int sh = e + 22 - wF;
  uint32_t m;
  if (sh >= 0) {
    m = M << sh;
  } else if (-sh > 24) {
    m = 0;
  } else {
    const int k = -sh;
    m = M >> k;
    const uint32_t rem = M & ((1u << k) - 1u);
    const uint32_t half = 1u << (k - 1);
    if (rem > half || (rem == half && (m & 1u))) m += 1u;
  }
  return (s << 31) | m;
}

}  // namespace hobflops
