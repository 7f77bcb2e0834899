// Pack (float32 or code -> PL32 bit-planes) and unpack (PL32 -> code or
// float32) kernels. HBM-bound: a pack reads 4 bytes and writes NB/8 bytes per
// value, an unpack the reverse.
//
// Pack: each lane quantises one value; a wave holds two 32-value groups
// (lanes 0-31 and 32-63), and NB ballots turn the wave's codes into the NB
// plane words of both groups at once (the bit transpose of the paper's
// bitslice layout, Sec. 3.2). Lane b then stores plane b of the first group and
// lane 32+b plane b of the second, so a wave's stores are 2*NB consecutive words.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pack.hpp"

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

__global__ __launch_bounds__(256) void pack_kernel(const void* __restrict__ src, int kind,
                                                   int64_t len, int G, int wE, int wF, int NB,
                                                   uint32_t* __restrict__ planes,
                                                   int64_t ngroups) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t q = wave * 2 + (lane >> 5);
  const int j = lane & 31;
  const uint32_t nbmask = NB >= 32 ? 0xFFFFFFFFu : ((1u << NB) - 1u);
  uint32_t code = 0;
  if (q < ngroups) {
    const int64_t r = q / G;
    const int64_t col = (int64_t)(q - r * G) * 32 + j;
    if (col < len) {
      const int64_t i = r * len + col;
      if (kind == 0)
        code = quantize_bits(((const uint32_t*)src)[i], wE, wF);
      else
        code = ((const uint32_t*)src)[i] & nbmask;
    }
  }
  uint32_t mine = 0;
  for (int b = 0; b < NB; ++b) {
    const uint64_t m = __ballot((code >> b) & 1u);
    const uint32_t half = (lane >> 5) ? (uint32_t)(m >> 32) : (uint32_t)m;
    mine = (j == b) ? half : mine;
  }
  if (q < ngroups && j < NB) planes[q * NB + j] = mine;
}

__global__ __launch_bounds__(256) void unpack_kernel(const uint32_t* __restrict__ planes,
                                                     int kind, int64_t len, int G, int wE,
                                                     int wF, int NB, void* __restrict__ dst,
                                                     int64_t ngroups) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t q = wave * 2 + (lane >> 5);
  const int j = lane & 31;
  if (q >= ngroups) return;
  const int64_t r = q / G;
  const int64_t col = (int64_t)(q - r * G) * 32 + j;
  if (col >= len) return;
  const uint32_t* p = planes + q * NB;
  uint32_t code = 0;
  for (int b = 0; b < NB; ++b) code |= ((p[b] >> j) & 1u) << b;
  const int64_t i = r * len + col;
  if (kind == 0)
    ((uint32_t*)dst)[i] = decode_bits(code, wE, wF);
  else
    ((uint32_t*)dst)[i] = code;
}

hipError_t launch_pack(const void* src, int kind, int64_t rows, int64_t len, int wE, int wF,
                       uint32_t* planes, hipStream_t stream) {
  const int NB = 3 + wE + wF;
  const int64_t G = (len + 31) / 32;
  const int64_t ngroups = rows * G;
  const int64_t waves = (ngroups + 1) / 2;
  const int64_t blocks = (waves + 3) / 4;
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(pack_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, src, kind, len,
                     (int)G, wE, wF, NB, planes, ngroups);
  return hipGetLastError();
}

hipError_t launch_unpack(const uint32_t* planes, int64_t rows, int64_t len, int wE, int wF,
                         int kind, void* dst, hipStream_t stream) {
  const int NB = 3 + wE + wF;
  const int64_t G = (len + 31) / 32;
  const int64_t ngroups = rows * G;
  const int64_t waves = (ngroups + 1) / 2;
  const int64_t blocks = (waves + 3) / 4;
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(unpack_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, planes, kind,
                     len, (int)G, wE, wF, NB, dst, ngroups);
  return hipGetLastError();
}

}  // namespace hobflops
