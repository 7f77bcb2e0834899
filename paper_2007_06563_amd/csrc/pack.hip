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

#include "codec.hpp"
#include "pack.hpp"

namespace hobflops {

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
