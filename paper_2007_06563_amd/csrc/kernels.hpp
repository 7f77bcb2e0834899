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
// netlist performs 32 MACs. A workgroup's four waves cover 256 consecutive
// positions of one m-tile: the 32-kernel weight word of a tap is the same for
// all of them, while each lane broadcasts its own IFM value's bits into
// all-zero / all-one words (the paper broadcasts the IFM channel value across
// the kernel lanes). For every output the accumulator planes stay in VGPRs and
// the taps are taken in the fixed order ky, kx, c; a padding tap contributes
// x = +0.
//
// Work is walked in chunks (ky, kx, 32-channel word). With one wave per SIMD
// nothing hides memory latency, so operands are fetched one step ahead:
//  - the weight rows of the next chunk (at most 32 rows of NIN words, one
//    per channel) are loaded from HBM into registers while the current chunk
//    runs, then written to the other half of a double-buffered LDS tile
//    shared by the workgroup; each MAC reads its row with 16-byte LDS loads
//    (one address for the whole wave: a broadcast), prefetched one row ahead;
//  - each lane's IFM channel word of the next chunk is loaded while the
//    current chunk's channels are processed.
// Prefetch addresses are clamped into the buffers, so no load is out of
// bounds, and every lane of the workgroup takes part in the staging.
template <class V>
__global__ __launch_bounds__(kConvBlock) void conv2d_kernel(const uint32_t* __restrict__ ifm,
                                                            const uint32_t* __restrict__ w,
                                                            uint32_t* __restrict__ ofm,
                                                            ConvParams p) {
  constexpr int NIN = V::NIN, NACC = V::NACC, NOUT = V::NOUT;
  constexpr int NINP = (NIN + 3) & ~3;  // LDS row stride: rows start 16-byte aligned
  constexpr int kRows = 32;             // weight rows per chunk (one channel word)
  constexpr int kStage = (kRows * NIN + kConvBlock - 1) / kConvBlock;
  __shared__ uint4 wtile[2][kRows * NINP / 4];

  const int tid = threadIdx.x;
  const int mt = blockIdx.y;
  const int pos = blockIdx.x * kConvBlock + tid;
  const bool active = pos < p.P;
  const int q = active ? pos : 0;
  const int ox = q % p.OW;
  const int oy = (q / p.OW) % p.OH;
  const int n = q / (p.OW * p.OH);
  const int iy0 = oy * p.stride - p.pad, ix0 = ox * p.stride - p.pad;
  const uint32_t* img = ifm + (size_t)n * p.H * p.W * p.CG * NIN;
  const size_t wrow = (size_t)p.MT * NIN;  // words between consecutive weight rows
  const uint32_t* wm = w + (size_t)mt * NIN;

  // IFM words of chunk (ky, kx, cg) for this lane, zero for a padding tap.
  auto load_ifm = [&](int ky, int kx, int cg, uint32_t(&xw)[NIN]) {
    const int iy = iy0 + ky, ix = ix0 + kx;
    const bool valid = active && iy >= 0 && iy < p.H && ix >= 0 && ix < p.W;
    const uint32_t* ip =
        img + (((size_t)(valid ? iy : 0) * p.W + (valid ? ix : 0)) * p.CG + cg) * NIN;
#pragma unroll
    for (int b = 0; b < NIN; ++b) {
      const uint32_t t = ip[b];
      xw[b] = valid ? t : 0u;
    }
  };
  // This thread's share of the weight rows r0 .. r0+nc-1 (HBM -> registers).
  uint32_t stage[kStage];
  auto fetch_w = [&](int r0, int nc) {
#pragma unroll
    for (int s = 0; s < kStage; ++s) {
      const int i = tid + s * kConvBlock;
      const int row = i / NIN, b = i - (i / NIN) * NIN;
      const int r = (row < nc && i < kRows * NIN) ? r0 + row : r0;
      stage[s] = wm[(size_t)r * wrow + (row < nc ? b : 0)];
    }
  };
  auto store_w = [&](int buf) {
    uint32_t* t = reinterpret_cast<uint32_t*>(wtile[buf]);
#pragma unroll
    for (int s = 0; s < kStage; ++s) {
      const int i = tid + s * kConvBlock;
      if (i < kRows * NIN) t[(i / NIN) * NINP + (i - (i / NIN) * NIN)] = stage[s];
    }
  };
  auto read_row = [&](int buf, int c, uint32_t(&wv)[NIN]) {
    const uint32_t* t = reinterpret_cast<const uint32_t*>(wtile[buf]) + c * NINP;
#pragma unroll
    for (int b = 0; b < NIN; ++b) wv[b] = t[b];
  };

  uint32_t acc[NACC];
#pragma unroll
  for (int b = 0; b < NACC; ++b) acc[b] = 0u;  // +0

  uint32_t xn[NIN];
  fetch_w(0, min(kRows, p.C));
  load_ifm(0, 0, 0, xn);
  store_w(0);
  __syncthreads();

  int ky = 0, kx = 0, cg = 0;
  const int nchunks = p.KH * p.KW * p.CG;
  for (int ch = 0; ch < nchunks; ++ch) {
    const int buf = ch & 1;
    const int nc = min(kRows, p.C - kRows * cg);
    int cg2 = cg + 1, kx2 = kx, ky2 = ky;
    if (cg2 == p.CG) {
      cg2 = 0;
      if (++kx2 == p.KW) {
        kx2 = 0;
        if (++ky2 == p.KH) ky2 = 0;  // past the end: refetch chunk 0, unused
      }
    }
    uint32_t xw[NIN];
#pragma unroll
    for (int b = 0; b < NIN; ++b) xw[b] = xn[b];
    fetch_w((ky2 * p.KW + kx2) * p.C + kRows * cg2, min(kRows, p.C - kRows * cg2));
    load_ifm(ky2, kx2, cg2, xn);

    // Two rows in flight, ping-pong: the next row's LDS loads are issued
    // before the current MAC, and a scheduling barrier keeps them there (the
    // scheduler would otherwise sink them next to their use).
    auto mac_step = [&](const uint32_t(&wv)[NIN], int c) {
      uint32_t x[NIN];
#pragma unroll
      for (int b = 0; b < NIN; ++b)
        x[b] = (uint32_t)__builtin_amdgcn_sbfe((int)xw[b], c, 1);  // bit c -> 0 / ~0
      V::mac(acc, wv, x);
    };
    uint32_t wa[NIN], wb[NIN];
    read_row(buf, 0, wa);
    int c = 0;
    for (; c + 2 <= nc; c += 2) {
      read_row(buf, c + 1, wb);
      __builtin_amdgcn_sched_barrier(0);
      mac_step(wa, c);
      read_row(buf, c + 2 < nc ? c + 2 : c + 1, wa);
      __builtin_amdgcn_sched_barrier(0);
      mac_step(wb, c + 1);
    }
    if (c < nc) mac_step(wa, c);
    store_w(buf ^ 1);
    __syncthreads();
    cg = cg2;
    kx = kx2;
    ky = ky2;
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
