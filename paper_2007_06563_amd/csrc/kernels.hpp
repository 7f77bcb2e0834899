// Bitsliced HOBFLOPS kernels for gfx950 (templates over a generated variant).
//
// Plane layout (PL32): a packed tensor with logical shape [R][L], packed
// along L, is stored as uint32 words[R][ceil(L/32)][NB]; bit j of
// words[r][g][b] is bit b of the code at (r, 32g + j). Padding lanes hold
// code 0 (+0). This is the bitslice-parallel layout of the paper (Sec. 3.2,
// "many values transformed" figure) with 32-lane words.
//
// A Variant type supplies the generated netlists:
//   static constexpr int NIN, NACC, NOUT;     planes per value
//   static __device__ void mac(uint32_t (&acc)[NACC], const uint32_t (&w)[NIN],
//                              const uint32_t (&x)[NIN]);        acc = acc + w*x
//   static __device__ void epi(const uint32_t (&acc)[NACC], uint32_t (&out)[NOUT]);
// or, for the element-wise kernel,
//   static __device__ void muladd(const uint32_t (&a)[NIN], const uint32_t (&b)[NIN],
//                                 const uint32_t (&c)[NIN], uint32_t (&r)[NACC]);
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hobflops {

struct ConvParams {
  int N, H, W, C, M, KH, KW, stride, pad;
  int OH, OW;
  int CG;  // ceil(C / 32): channel words per IFM position
  int MT;  // ceil(M / 32): kernel words (m-tiles) per weight row / OFM position
  int P;   // N * OH * OW output positions
};

constexpr int kConvBlock = 256;  // four wave64s, one SIMD each

// MCMK convolution (paper Sec. 3.4). One lane owns one output position and
// one m-tile of 32 kernels, so every VALU bitwise instruction of the MAC
// netlist performs 32 MACs. A wave covers 64 consecutive positions of one
// m-tile: the 32-kernel weight word of a tap is the same for the whole wave
// (uniform, loaded once per wave), while each lane broadcasts its own IFM
// value's bits into all-zero / all-one words (the paper broadcasts the IFM
// channel value across the kernel lanes). For every output the accumulator
// planes stay in VGPRs and the taps are taken in the fixed order
// ky, kx, c; a padding tap contributes x = +0.
template <class V>
__global__ __launch_bounds__(kConvBlock) void conv2d_kernel(const uint32_t* __restrict__ ifm,
                                                            const uint32_t* __restrict__ w,
                                                            uint32_t* __restrict__ ofm,
                                                            ConvParams p) {
  constexpr int NIN = V::NIN, NACC = V::NACC, NOUT = V::NOUT;
  const int mt = blockIdx.y;
  const int pos = blockIdx.x * kConvBlock + threadIdx.x;
  const bool active = pos < p.P;
  const int q = active ? pos : 0;
  const int ox = q % p.OW;
  const int oy = (q / p.OW) % p.OH;
  const int n = q / (p.OW * p.OH);

  uint32_t acc[NACC];
#pragma unroll
  for (int b = 0; b < NACC; ++b) acc[b] = 0u;  // +0

  const size_t wrow = (size_t)p.MT * NIN;  // words between consecutive weight rows
  for (int ky = 0; ky < p.KH; ++ky) {
    const int iy = oy * p.stride + ky - p.pad;
    for (int kx = 0; kx < p.KW; ++kx) {
      const int ix = ox * p.stride + kx - p.pad;
      const bool valid = active && iy >= 0 && iy < p.H && ix >= 0 && ix < p.W;
      const uint32_t* ip = ifm + ((((size_t)n * p.H + (valid ? iy : 0)) * p.W + (valid ? ix : 0)) *
                                  p.CG) * NIN;
      const uint32_t* wp = w + (size_t)((ky * p.KW + kx) * p.C) * wrow + (size_t)mt * NIN;
      for (int cg = 0; cg < p.CG; ++cg) {
        uint32_t xw[NIN];
#pragma unroll
        for (int b = 0; b < NIN; ++b) xw[b] = valid ? ip[cg * NIN + b] : 0u;
        const int nc = min(32, p.C - 32 * cg);
        const uint32_t* wc = wp + (size_t)(32 * cg) * wrow;
#pragma unroll 2
        for (int c = 0; c < nc; ++c) {
          uint32_t x[NIN], wv[NIN];
#pragma unroll
          for (int b = 0; b < NIN; ++b) {
            x[b] = (uint32_t)__builtin_amdgcn_sbfe((int)xw[b], c, 1);  // bit c -> 0 / ~0
            wv[b] = wc[(size_t)c * wrow + b];
          }
          V::mac(acc, wv, x);
        }
      }
    }
  }
  if (!active) return;
  uint32_t out[NOUT];
  V::epi(acc, out);
  uint32_t* op = ofm + ((size_t)pos * p.MT + mt) * NOUT;
#pragma unroll
  for (int b = 0; b < NOUT; ++b) op[b] = out[b];
}

// Element-wise r = a*b + c (multiply rounded, then add rounded) on flat PL32
// tensors: one lane owns one word group, i.e. 32 independent triples.
template <class V>
__global__ __launch_bounds__(256) void muladd_kernel(const uint32_t* __restrict__ a,
                                                     const uint32_t* __restrict__ b,
                                                     const uint32_t* __restrict__ c,
                                                     uint32_t* __restrict__ r, int64_t groups) {
  constexpr int NIN = V::NIN, NACC = V::NACC;
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= groups) return;
  uint32_t av[NIN], bv[NIN], cv[NIN], rv[NACC];
#pragma unroll
  for (int i = 0; i < NIN; ++i) {
    av[i] = a[g * NIN + i];
    bv[i] = b[g * NIN + i];
    cv[i] = c[g * NIN + i];
  }
  V::muladd(av, bv, cv, rv);
#pragma unroll
  for (int i = 0; i < NACC; ++i) r[g * NACC + i] = rv[i];
}

}  // namespace hobflops
