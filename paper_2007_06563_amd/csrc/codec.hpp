// Conversions between float32 and codes of a (wE, wF) format, per value: the
// quantiser of the pack kernel and the decoder of the unpack kernel and of the
// convolution's float32 epilogue.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hobflops {

// float32 bits -> code of (wE, wF): the exact value rounded to nearest even
// with an unbounded exponent, then range checked (no subnormals in the format).
// Every case is computed and selected, with no branches, so that the 64 lanes
// of a wave never split (a mix of specials and normals is common).
__device__ __forceinline__ uint32_t quantize_bits(uint32_t bits, int wE, int wF) {
  const uint32_t s = bits >> 31;
  const uint32_t ef = (bits >> 23) & 0xFFu;
  const uint32_t fr = bits & 0x7FFFFFu;
  const int sh_x = wF + wE + 1, sh_s = wF + wE;
  const uint32_t sgn = s << sh_s;
  // significand M in [2^23, 2^24) and exponent u: value = M * 2^(u - 23);
  // a subnormal float32 is normalised by its leading zeros
  const int lz = __clz(fr | 1u) - 8;
  const bool sub = ef == 0u;
  const uint32_t M = sub ? (fr << lz) : (fr | 0x800000u);
  int u = sub ? -126 - lz : (int)ef - 127;
  const int k = 23 - wF;  // dropped bits, 0..22 (none for wF = 23)
  uint32_t q = M >> k;
  const uint32_t rem = M & ((1u << k) - 1u);
  const uint32_t half = k > 0 ? 1u << (k - 1) : 0u;
  q += (k > 0 && (rem > half || (rem == half && (q & 1u)))) ? 1u : 0u;
  const bool carry = q == (2u << wF);  // rounded up into the next binade
  q = carry ? q >> 1 : q;
  u += carry ? 1 : 0;
  const int Eb = u + (1 << (wE - 1)) - 1;
  const uint32_t inf = (2u << sh_x) | sgn;
  uint32_t code = (1u << sh_x) | sgn | ((uint32_t)Eb << wF) | (q & ((1u << wF) - 1u));
  code = Eb > (1 << wE) - 1 ? inf : code;
  code = Eb < 0 || (sub && fr == 0u) ? sgn : code;         // underflow, +-0
  code = ef == 0xFFu ? (fr ? (3u << sh_x) : inf) : code;  // NaN, +-inf
  return code;
}

// The same code as quantize_bits for wE <= 7 and wF <= 22, in fewer
// instructions. Such a format's smallest normal is 2^-63 or larger, so every
// float32 subnormal (and any value the add below might flush) lies below the
// range. For |x| in [2^u, 2^(u+1)), C = 2^(u + 23 - wF) has the ulp
// 2^(u - wF) in its binade and |x| + C stays in that binade, so the float32
// add rounds |x| to wF fraction bits, ties to even (the multiple index of C
// is even), and subtracting C again is exact; a round-up into the next
// binade shows in the result's exponent. The rounded magnitude r, read as
// an integer, orders like the value, so the range tests compare r with the
// bit patterns of the format's smallest normal and of its overflow
// threshold, and (r >> k) rebiased is the code's E and F fields. |x| is
// clamped to 2^100, which every such format overflows, so that C stays
// finite; NaN is tested on the input. The special cases are per-lane selects
// (v_cndmask_b32) of uniform constants, and the sign goes in last, except on
// NaN.
__device__ __forceinline__ uint32_t quantize_narrow(uint32_t bits, int wE, int wF) {
  const uint32_t a = bits & 0x7FFFFFFFu;
  const uint32_t ac = min(a, 0x71800000u);
  const int k = 23 - wF;
  const float C = __uint_as_float((ac & 0x7F800000u) + ((uint32_t)k << 23));
  const uint32_t r = __float_as_uint(__fsub_rn(__fadd_rn(__uint_as_float(ac), C), C));
  const int bias = (1 << (wE - 1)) - 1;
  const int sh_s = wF + wE, sh_x = sh_s + 1;
  const uint32_t base = (uint32_t)(127 - bias) << wF;                // E = 0 in r >> k
  const uint32_t lo = base << k;                                    // smallest normal
  const uint32_t hi = lo + (1u << (sh_s + k));                      // first overflowing value
  // (1 << sh_x) | t for the fields t = (r >> k) - base of a value in range
  uint32_t code = (r >> k) + ((1u << sh_x) - base);
  code = r < lo ? 0u : code;                                        // +-0
  code = r >= hi ? (2u << sh_x) : code;                             // +-inf
  code |= (bits >> (31 - sh_s)) & (1u << sh_s);                     // the sign
  return a > 0x7F800000u ? (3u << sh_x) : code;                     // NaN
}

// code of (wE, wF) -> float32 bits for wE <= 7, where every value of the
// format is a normal float32 (the result is exact): exponent E + 127 - bias,
// fraction F << (23 - wF), +-0, +-inf, and NaN as 0x7FC00000, all selected
// with masks of the exception bits, without branches.
__device__ __forceinline__ uint32_t decode_narrow(uint32_t code, int wE, int wF) {
  const int sh_s = wF + wE;
  // the normal value: E and F shifted by 23 - wF land on float32's exponent
  // and fraction fields, and one add rebiases the exponent (it stays below 255)
  const uint32_t v = (__builtin_amdgcn_ubfe(code, 0, sh_s) << (23 - wF)) +
                     ((uint32_t)(127 - ((1 << (wE - 1)) - 1)) << 23);
  const uint32_t sbit = (code >> sh_s) << 31;
  const uint32_t x0 = (uint32_t)__builtin_amdgcn_sbfe((int)code, sh_s + 1, 1);  // all ones if set
  const uint32_t x1 = (uint32_t)__builtin_amdgcn_sbfe((int)code, sh_s + 2, 1);
  const uint32_t lo = x0 & v;                                    // x1 = 0: normal or zero
  const uint32_t hi = 0x7F800000u | (x0 & 0x00400000u);          // x1 = 1: inf or NaN
  const uint32_t mag = __builtin_amdgcn_bitop3_b32(x1, hi, lo, 0xCA);
  // the sign, except on NaN: s & ~(x0 & x1) (bitop3 of (s, x0, x1))
  return mag | __builtin_amdgcn_bitop3_b32(sbit, x0, x1, 0x70);
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
