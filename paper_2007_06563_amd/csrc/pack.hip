// Pack (float32 or code -> PL32 bit-planes) and unpack (PL32 -> code or
// float32) kernels. HBM-bound: a pack reads 4 bytes and writes NB/8 bytes per
// value, an unpack the reverse.
//
// Pack: each lane quantises one value per pass; a pass holds two 32-value
// groups (lanes 0-31 and 32-63), and NB ballots turn the wave's codes into the
// NB plane words of both groups at once (the bit transpose of the paper's
// bitslice layout, Sec. 3.2). Lane b then stores plane b of the first group and
// lane 32+b plane b of the second, so a pass's stores are 2*NB consecutive
// words. Unpack: lane j gathers bit j of the NB plane words of its group.
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

// Groups of 32 values a wave handles: two per pass (lanes 0-31, 32-63), kU
// passes whose loads are all issued before any value is quantised, so a wave
// keeps kU loads per lane in flight. NB (planes per value) is a template
// argument, so the plane loops unroll and their loads issue together.
constexpr int kU = 4;

// Row and column of group q: 32-bit arithmetic when the group count allows.
template <bool kWide>
__device__ __forceinline__ void group_rc(int64_t q, int G, int64_t& r, int64_t& c) {
  if (kWide) {
    r = q / G;
    c = q - r * G;
  } else {
    const uint32_t q32 = (uint32_t)q, r32 = q32 / (uint32_t)G;
    r = r32;
    c = q32 - r32 * (uint32_t)G;
  }
}

template <int NB, bool kWide>
__global__ __launch_bounds__(256) void pack_kernel(const void* __restrict__ src, int kind,
                                                   int64_t len, int G, int wE, int wF,
                                                   uint32_t* __restrict__ planes,
                                                   int64_t ngroups) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int j = lane & 31;
  constexpr uint32_t nbmask = NB >= 32 ? 0xFFFFFFFFu : ((1u << (NB & 31)) - 1u);
  uint32_t raw[kU];
  bool have[kU];
#pragma unroll
  for (int u = 0; u < kU; ++u) {  // group q = (wave * kU + u) * 2 + half
    const int64_t q = (wave * kU + u) * 2 + (lane >> 5);
    have[u] = false;
    raw[u] = 0;
    if (q < ngroups) {
      int64_t r, g;
      group_rc<kWide>(q, G, r, g);
      const int64_t col = g * 32 + j;
      if (col < len) {
        raw[u] = ((const uint32_t*)src)[r * len + col];
        have[u] = true;
      }
    }
  }
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int64_t q = (wave * kU + u) * 2 + (lane >> 5);
    const uint32_t code =
        have[u] ? (kind == 0 ? quantize_bits(raw[u], wE, wF) : (raw[u] & nbmask)) : 0u;
    uint32_t mine = 0;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const uint64_t m = __ballot((code >> b) & 1u);
      const uint32_t half = (lane >> 5) ? (uint32_t)(m >> 32) : (uint32_t)m;
      mine = (j == b) ? half : mine;
    }
    if (q < ngroups && j < NB) planes[q * NB + j] = mine;
  }
}

template <int NB, bool kWide>
__global__ __launch_bounds__(256) void unpack_kernel(const uint32_t* __restrict__ planes,
                                                     int kind, int64_t len, int G, int wE,
                                                     int wF, void* __restrict__ dst,
                                                     int64_t ngroups) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int j = lane & 31;
  uint32_t w[kU][NB];
#pragma unroll
  for (int u = 0; u < kU; ++u) {  // every plane word of the lane's kU groups first
    const int64_t q = (wave * kU + u) * 2 + (lane >> 5);
    const uint32_t* p = planes + (q < ngroups ? q : 0) * NB;
#pragma unroll
    for (int b = 0; b < NB; ++b) w[u][b] = p[b];
  }
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int64_t q = (wave * kU + u) * 2 + (lane >> 5);
    if (q >= ngroups) continue;
    int64_t r, g;
    group_rc<kWide>(q, G, r, g);
    const int64_t col = g * 32 + j;
    if (col >= len) continue;
    uint32_t code = 0;
#pragma unroll
    for (int b = 0; b < NB; ++b) code |= ((w[u][b] >> j) & 1u) << b;
    const int64_t i = r * len + col;
    ((uint32_t*)dst)[i] = kind == 0 ? decode_bits(code, wE, wF) : code;
  }
}

namespace {

// NB = 3 + wE + wF runs from 6 to 32.
template <template <int, bool> class K, int NB = 6>
struct nb_dispatch {
  template <class F>
  static hipError_t run(int nb, F&& f) {
    if (nb == NB) return f(K<NB, false>{}, K<NB, true>{});
    return nb_dispatch<K, NB + 1>::run(nb, f);
  }
};
template <template <int, bool> class K>
struct nb_dispatch<K, 33> {
  template <class F>
  static hipError_t run(int, F&&) {
    return hipErrorInvalidValue;
  }
};

template <int NB, bool W>
struct PackK {
  static constexpr auto fn = pack_kernel<NB, W>;
};
template <int NB, bool W>
struct UnpackK {
  static constexpr auto fn = unpack_kernel<NB, W>;
};

}  // namespace

hipError_t launch_pack(const void* src, int kind, int64_t rows, int64_t len, int wE, int wF,
                       uint32_t* planes, hipStream_t stream) {
  const int NB = 3 + wE + wF;
  const int64_t G = (len + 31) / 32;
  const int64_t ngroups = rows * G;
  const int64_t waves = (ngroups + 2 * kU - 1) / (2 * kU);
  const int64_t blocks = (waves + 3) / 4;
  if (blocks == 0) return hipSuccess;
  const bool wide = ngroups + 2 * kU >= ((int64_t)1 << 31);
  return nb_dispatch<PackK>::run(NB, [&](auto narrow_k, auto wide_k) {
    if (wide)
      hipLaunchKernelGGL(decltype(wide_k)::fn, dim3((unsigned)blocks), dim3(256), 0, stream, src,
                         kind, len, (int)G, wE, wF, planes, ngroups);
    else
      hipLaunchKernelGGL(decltype(narrow_k)::fn, dim3((unsigned)blocks), dim3(256), 0, stream, src,
                         kind, len, (int)G, wE, wF, planes, ngroups);
    return hipGetLastError();
  });
}

hipError_t launch_unpack(const uint32_t* planes, int64_t rows, int64_t len, int wE, int wF,
                         int kind, void* dst, hipStream_t stream) {
  const int NB = 3 + wE + wF;
  const int64_t G = (len + 31) / 32;
  const int64_t ngroups = rows * G;
  const int64_t waves = (ngroups + 2 * kU - 1) / (2 * kU);
  const int64_t blocks = (waves + 3) / 4;
  if (blocks == 0) return hipSuccess;
  const bool wide = ngroups + 2 * kU >= ((int64_t)1 << 31);
  return nb_dispatch<UnpackK>::run(NB, [&](auto narrow_k, auto wide_k) {
    if (wide)
      hipLaunchKernelGGL(decltype(wide_k)::fn, dim3((unsigned)blocks), dim3(256), 0, stream,
                         planes, kind, len, (int)G, wE, wF, dst, ngroups);
    else
      hipLaunchKernelGGL(decltype(narrow_k)::fn, dim3((unsigned)blocks), dim3(256), 0, stream,
                         planes, kind, len, (int)G, wE, wF, dst, ngroups);
    return hipGetLastError();
  });
}

}  // namespace hobflops
