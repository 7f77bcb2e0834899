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
//   static constexpr int wE, wF_OUT;          the output format
//   static __device__ void mac(uint32_t (&acc)[NACC], const uint32_t (&w)[NIN],
//                              const uint32_t (&x)[NIN]);        acc = acc + w*x
//   static __device__ void epi(const uint32_t (&acc)[NACC], uint32_t (&out)[NOUT]);
// or, for the element-wise kernel,
//   static __device__ void muladd(const uint32_t (&a)[NIN], const uint32_t (&b)[NIN],
//                                 const uint32_t (&c)[NIN], uint32_t (&r)[NACC]);
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bitmat.hpp"
#include "codec.hpp"

namespace hobflops {

typedef __attribute__((address_space(3))) uint32_t lds_u32;

struct ConvParams {
  int N, H, W, C, M, KH, KW, stride, pad;
  int OH, OW;
  int CG;  // ceil(C / 32): channel words per IFM position
  int MT;  // ceil(M / 32): kernel words (m-tiles) per weight row / OFM position
  int P;   // N * OH * OW output positions
  int ofm_kind;  // kOfmPlanes, kOfmF32 or kOfmCode
  int ofm_vec;   // ofm is 16-byte aligned (value rows may be stored 16 bytes at a time)
  // Split kernel: every wait of a wave for its partner's counter polls at most
  // spin_cap times (a sleep of 64 clocks each); a wait that ends there without
  // the counter adds 1 to *wait_fail (the launch's results are then invalid).
  uint32_t spin_cap;
  uint32_t* wait_fail;
};

// Global average pooling: N images, HW positions each, CG channel words per
// position; `scale` is the code of 1/HW in the accumulator format.
struct PoolParams {
  int N, HW, CG;
  uint32_t scale;
};

// What the convolution writes (hobflops_conv_desc.ofm_kind): PL32 planes, or
// per value, row-major [P][M], float32 values or uint32 codes.
constexpr int kOfmPlanes = 0, kOfmF32 = 1, kOfmCode = 2;

// float32 bit-planes of the 32 values whose (wE, wF) code planes are `c`
// (F, E, s, x0, x1 from plane 0 up), for wE <= 7, where every value of the
// format is a normal float32: exponent E + 127 - bias, fraction F << (23 - wF),
// specials as hobflops_unpack writes them (NaN 0x7FC00000).
template <int wE, int wF>
__device__ __forceinline__ void float_planes(const uint32_t* c, uint32_t (&f)[32]) {
  static_assert(wE <= 7 && wF <= 23, "every value a normal float32");
  const uint32_t s = c[wF + wE], x0 = c[wF + wE + 1], x1 = c[wF + wE + 2];
  const uint32_t norm = x0 & ~x1, nan = x0 & x1;
#pragma unroll
  for (int b = 0; b < 32; ++b) f[b] = 0u;
#pragma unroll
  for (int i = 0; i < wF; ++i) f[23 - wF + i] = norm & c[i];
  f[22] |= nan;
  constexpr uint32_t add = 127u - ((1u << (wE - 1)) - 1u);
  uint32_t carry = 0u;
#pragma unroll
  for (int i = 0; i < 8; ++i) {  // exponent E + add, bitsliced ripple
    const uint32_t e = i < wE ? c[wF + i] : 0u;
    const uint32_t k = ((add >> i) & 1u) ? ~0u : 0u;
    f[23 + i] = (norm & (e ^ k ^ carry)) | x1;
    carry = (e & k) | (carry & (e ^ k));
  }
  f[31] = s & ~nan;
}

// The epilogue's store of one lane's output word group: 32 values of one
// position, kernels 32*mt .. 32*mt+31, as NOUT plane words or, moved out of
// plane order with one bit-matrix transpose, as codes or float32 values (the
// decode done on the planes first), 16 bytes per store where the row allows.
template <int NOUT, int wE, int wF>
__device__ __forceinline__ void store_ofm(const uint32_t (&out)[NOUT], uint32_t* __restrict__ ofm,
                                          int pos, int mt, const ConvParams& p) {
  if (p.ofm_kind == kOfmPlanes) {
    uint32_t* op = ofm + ((size_t)pos * p.MT + mt) * NOUT;
#pragma unroll
    for (int b = 0; b < NOUT; ++b) op[b] = out[b];
    return;
  }
  uint32_t v[32];
  if (p.ofm_kind == kOfmF32 && wE <= 7) {
    float_planes<(wE <= 7 ? wE : 7), wF>(out, v);
    transpose32(v);
  } else {
#pragma unroll
    for (int b = 0; b < 32; ++b) v[b] = b < NOUT ? out[b] : 0u;
    transpose32(v);
    if (p.ofm_kind == kOfmF32) {
#pragma unroll
      for (int j = 0; j < 32; ++j) v[j] = decode_bits(v[j], wE, wF);
    }
  }
  const int m0 = mt * 32;
  const int nm = min(32, p.M - m0);
  uint32_t* op = ofm + (size_t)pos * p.M + m0;
  if (nm == 32 && (p.M & 3) == 0 && p.ofm_vec) {
#pragma unroll
    for (int j = 0; j < 32; j += 4)
      *reinterpret_cast<uint4*>(op + j) = make_uint4(v[j], v[j + 1], v[j + 2], v[j + 3]);
  } else {
#pragma unroll
    for (int j = 0; j < 32; ++j)
      if (j < nm) op[j] = v[j];
  }
}

constexpr int kConvBlock = 256;  // positions per workgroup: four wave64s

// Default bound of every counter wait in the split kernel (sleeps of 64
// clocks): a counter that never arrives ends the wait instead of the kernel
// hanging, and the give-up is counted (ConvParams::wait_fail).
constexpr uint32_t kSpinCap = 1u << 20;

// Kernel shapes of the convolution (hobflops_conv_desc.algo).
constexpr int kAlgoAuto = 0, kAlgoFused = 1, kAlgoSplit = 2, kAlgoSplitCompact = 3;


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

  // Raw IFM words of chunk (ky, kx, cg) for this lane; *valid is false for a
  // padding tap (the words then come from a clamped, in-bounds address and are
  // replaced by zero, i.e. +0, only when the chunk is used, so that the load's
  // latency is not waited for here).
  auto load_ifm = [&](int ky, int kx, int cg, uint32_t(&xw)[NIN], bool* valid) {
    const int iy = iy0 + ky, ix = ix0 + kx;
    *valid = active && iy >= 0 && iy < p.H && ix >= 0 && ix < p.W;
    const uint32_t* ip =
        img + (((size_t)(*valid ? iy : 0) * p.W + (*valid ? ix : 0)) * p.CG + cg) * NIN;
#pragma unroll
    for (int b = 0; b < NIN; ++b) xw[b] = ip[b];
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
  // the two tiles as one array of 2 * kRows rows
  const uint32_t* tile = reinterpret_cast<const uint32_t*>(wtile);
  auto read_row = [&](int row, uint32_t(&wv)[NIN]) {
    const uint32_t* t = tile + row * NINP;
#pragma unroll
    for (int b = 0; b < NIN; ++b) wv[b] = t[b];
  };

  uint32_t acc[NACC];
#pragma unroll
  for (int b = 0; b < NACC; ++b) acc[b] = 0u;  // +0

  // A layer with at most 2 * kRows weight rows per m-tile (a first layer of
  // three channels has 27) keeps all of them in the tile, staged once: no
  // per-chunk staging and no barrier per chunk.
  const int T = p.KH * p.KW * p.C;
  const bool resident = T <= 2 * kRows;
  uint32_t xn[NIN];
  bool xn_valid;
  if (resident) {
    uint32_t* t = reinterpret_cast<uint32_t*>(wtile);
    for (int i = tid; i < T * NIN; i += kConvBlock) {
      const int row = i / NIN, b = i - row * NIN;
      t[row * NINP + b] = wm[(size_t)row * wrow + b];
    }
  } else {
    fetch_w(0, min(kRows, p.C));
    store_w(0);
  }
  load_ifm(0, 0, 0, xn, &xn_valid);
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
    for (int b = 0; b < NIN; ++b) xw[b] = xn_valid ? xn[b] : 0u;
    // the chunk's first row in the tile
    const int r0 = resident ? (ky * p.KW + kx) * p.C + kRows * cg : buf * kRows;
    if (!resident)
      fetch_w((ky2 * p.KW + kx2) * p.C + kRows * cg2, min(kRows, p.C - kRows * cg2));
    load_ifm(ky2, kx2, cg2, xn, &xn_valid);

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
    read_row(r0, wa);
    int c = 0;
    for (; c + 2 <= nc; c += 2) {
      read_row(r0 + c + 1, wb);
      __builtin_amdgcn_sched_barrier(0);
      mac_step(wa, c);
      read_row(r0 + (c + 2 < nc ? c + 2 : c + 1), wa);
      __builtin_amdgcn_sched_barrier(0);
      mac_step(wb, c + 1);
    }
    if (c < nc) mac_step(wa, c);
    if (!resident) {
      store_w(buf ^ 1);
      __syncthreads();
    }
    cg = cg2;
    kx = kx2;
    ky = ky2;
  }
  if (!active) return;
  uint32_t out[NOUT];
  V::epi(acc, out);
  store_ofm<NOUT, V::wE, V::wF_OUT>(out, ofm, pos, mt, p);
}

// MCMK convolution, split shape: multiply and accumulate on different waves.
//
// A wave issues at most one instruction every four clocks, half of what its
// SIMD's VALU can retire, and the chain of adds into one accumulator cannot be
// reordered (the fixed accumulation order), so a launch with about one chain
// wave per SIMD leaves half of the VALU idle. The products w*x do not depend
// on the accumulator, so here each workgroup runs 4 accumulator waves (waves
// 0-3: 64 positions each, one m-tile, accumulator planes in VGPRs, the adder
// netlist only) and 4 multiplier waves (waves 4-7: the same positions; IFM bit
// broadcast and the multiplier netlist). Both netlists run as inline assembly
// whose registers avoid VGPR bank conflicts, so that two waves on a SIMD both
// issue at full rate.
//
// Taps are processed in batches of V::kBatch (even) in the fixed tap order.
// In iteration b, between two workgroup barriers:
//  - accumulator wave i adds the products of batch b (LDS product ring, half b%2);
//  - multiplier wave 4+i computes the products of batch b+1 into half (b+1)%2,
//    reading the batch's weight rows from LDS weight-ring slot (b+1)%3; a tap
//    past the end gets the product -0, which leaves every accumulator value
//    unchanged (x + -0 = x for all x, including both zeros);
//  - the multiplier waves together load the weight rows of batch b+2 from HBM
//    (one word per thread) and store them into weight-ring slot (b+2)%3.
// Each ring slot written in iteration b was last read in iteration b-1 or
// b-2, before a barrier, and is read only after the barrier that ends b.
// Every wave reaches every barrier, so the loop cannot deadlock.
template <class V>
__device__ __forceinline__ void conv2d_split_body(const uint32_t* __restrict__ ifm,
                                                  const uint32_t* __restrict__ w,
                                                  uint32_t* __restrict__ ofm, const ConvParams& p) {
  constexpr int NIN = V::NIN, NACC = V::NACC, NOUT = V::NOUT;
  constexpr int NINP = (NIN + 3) & ~3;    // weight row stride in LDS (16-byte aligned)
  constexpr int NACCP = (NACC + 3) & ~3;  // product entry per lane (16-byte aligned)
  constexpr int K = V::kBatch;
  constexpr int S = V::kSlots;        // product ring depth: batches in flight
  constexpr int kStride = NACCP / 4;  // uint4 per product entry
  static_assert(K % 2 == 0, "the accumulator ping-pong needs an even batch");
  static_assert(S == 2 || S == 3, "ring of two or three batches");
  static_assert(K * NIN <= kConvBlock, "one weight word per multiplier thread");
  static_assert(S * K * 256 * NACCP * 4 <= 144 * 1024, "product ring exceeds the LDS budget");
  static_assert(!V::kPairs || K * NIN <= 64, "pairs: a batch's weights loaded by one wave");
  // [slot][k][wave][kStride][lane]: chunk j of the 64 lanes' entries side by
  // side, so a wave's 16-byte read of one chunk is free of bank conflicts
  __shared__ uint4 pring[S * K * 4 * kStride * 64];
  // weights: shared ring [slot][k][NINP words] (barrier), or one batch per
  // multiplier wave [wave][k][NINP words] (pairs)
  __shared__ uint4 wring[(V::kPairs ? 4 : 3) * K * NINP / 4];
  __shared__ uint32_t flags[4][2];  // pairs: per wave pair, batches made / consumed

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const bool mul_role = wave >= 4;
  const int pw = wave & 3;
  const int mt = blockIdx.y;
  const int pos = blockIdx.x * kConvBlock + pw * 64 + lane;
  const bool active = pos < p.P;
  const int q = active ? pos : 0;
  const int ox = q % p.OW;
  const int oy = (q / p.OW) % p.OH;
  const int n = q / (p.OW * p.OH);
  const int iy0 = oy * p.stride - p.pad, ix0 = ox * p.stride - p.pad;
  const uint32_t* img = ifm + (size_t)n * p.H * p.W * p.CG * NIN;
  const size_t wrow = (size_t)p.MT * NIN;
  const uint32_t* wm = w + (size_t)mt * NIN;
  const int T = p.KH * p.KW * p.C;  // taps per output
  const int nb = (T + K - 1) / K;

  auto entry = [&](int b, int k) {  // batch b lives in ring slot b % S
    // C-style cast: generic pointer into the LDS address space
    return (lds_u32*)(pring + (((size_t)(b % S) * K + k) * 4 + pw) * kStride * 64 + lane);
  };

  // ---- multiplier waves: weight staging (thread t of the 256 loads word t;
  // with pairs, lane t of each multiplier wave, for that wave alone)
  const int mt_tid = V::kPairs ? lane : threadIdx.x - 4 * 64;
  const bool w_lane = mt_tid < K * NIN;  // this thread moves weight word (wk, wbb) of a batch
  const int wk = w_lane ? mt_tid / NIN : 0, wbb = w_lane ? mt_tid - wk * NIN : 0;
  // its LDS word within a weight slot, looked up once: a table read inside the
  // loop would be a memory load, and the wait for it would also wait for the
  // weight and IFM loads issued ahead
  const int w_ofs = wk * NINP + V::kWSlot[wbb];
  uint32_t wstage = 0;
  auto fetch_w = [&](int b) {  // HBM -> register, rows of batch b (clamped)
    // every lane loads (the others a word they do not store): a load under a
    // branch leaves the compiler's wait for it conservative, waiting for all
    wstage = wm[(size_t)min(b * K + wk, T - 1) * wrow + wbb];
  };
  auto store_w = [&](int b) {
    if (w_lane) {
      const int slot = V::kPairs ? pw : b % 3;
      ((lds_u32*)wring)[slot * K * NINP + w_ofs] = wstage;
    }
  };

  // ---- multiplier waves: IFM words of the current and the next chunk. The
  // next chunk's words are loaded into 16-byte register quads, so that the
  // loads land in the registers they are read from a chunk later (loaded into
  // scattered registers, they would be copied, and the copy waits for them).
  constexpr int NQ = (NIN + 3) / 4;
  typedef uint32_t quad_t __attribute__((ext_vector_type(4)));  // stays one 4-register value
  uint32_t xw[NIN];
  quad_t xq[NQ];
  bool xn_valid = false;          // xn is a real tap (else the chunk reads as +0)
  int nky = 0, nkx = 0, ncg = 0;  // coordinates of the chunk held in xn
  int c = 0, nc = 0;              // channel within the current chunk, its size
  auto load_ifm = [&](int ky, int kx, int cg) {  // raw words; masked when used
    const int iy = iy0 + ky, ix = ix0 + kx;
    xn_valid = active && iy >= 0 && iy < p.H && ix >= 0 && ix < p.W;
    const uint32_t* ip =
        img + (((size_t)(xn_valid ? iy : 0) * p.W + (xn_valid ? ix : 0)) * p.CG + cg) * NIN;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      quad_t v = {0u, 0u, 0u, 0u};
      __builtin_memcpy(&v, ip + 4 * q, 4 * min(4, NIN - 4 * q));
      xq[q] = v;
    }
  };
  auto advance = [&]() {  // move to the next (ky, kx, channel-word) chunk
    // the copies are ordered before the next chunk's loads (asm statements
    // keep their order, and loads do not cross the memory clobber): were the
    // loads scheduled first, the old and new words would need separate
    // registers, and the compiler would copy the new ones, waiting for them
#pragma unroll
    for (int bb = 0; bb < NIN; ++bb) {
      uint32_t v;
      asm volatile("v_mov_b32 %0, %1" : "=v"(v) : "v"(xq[bb / 4][bb % 4]));
      xw[bb] = xn_valid ? v : 0u;
    }
    asm volatile("" ::: "memory");
    nc = min(32, p.C - 32 * ncg);
    c = 0;
    if (++ncg == p.CG) {
      ncg = 0;
      if (++nkx == p.KW) {
        nkx = 0;
        if (++nky == p.KH) nky = 0;  // past the end: chunk 0 again, unused
      }
    }
    load_ifm(nky, nkx, ncg);
  };
  auto produce = [&](int b) {
    const int t0 = b * K;
    const int tk = min(K, T - t0);
    const lds_u32* wr = (const lds_u32*)wring + (V::kPairs ? pw : b % 3) * K * NINP;
    if (c == nc) advance();
    if (tk == K && c + K <= nc) {  // whole batch inside one channel word
      V::product_batch(xw, c, wr, entry(b, 0));
      c += K;
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // products visible at the barrier
      return;
    }
#pragma unroll
    for (int k = 0; k < K; ++k) {
      if (k < tk) {
        if (c == nc) advance();
        V::product_step(xw, c, wr + k * NINP, entry(b, k));
        ++c;
      } else {  // tap past the end: product -0 (the sign plane all ones)
        lds_u32* e = entry(b, k);  // word i of this lane's entry at e[(i/4)*256 + i%4]
#pragma unroll
        for (int bb = 0; bb < NACCP; ++bb) e[(bb >> 2) * 256 + (bb & 3)] = 0u;
        const int sg = V::kProdSlot[NACC - 3];
        e[(sg >> 2) * 256 + (sg & 3)] = 0xFFFFFFFFu;
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // products visible at the barrier
  };

  // ---- accumulator waves: planes in register-slot order (V::kAccSlot)
  uint32_t acc[NACCP];
#pragma unroll
  for (int s = 0; s < NACCP; ++s) acc[s] = 0u;  // +0

  // Schedule, one barrier per step i = -(S-1) .. nb-1: the multiplier waves
  // make batch i+S-1 (into ring slot (i+S-1) % S) and stage the weights of
  // batch i+3 (into weight slot i % 3, last read at step i-S+1 < i); the
  // accumulator waves add batch i, complete since the barrier of step i-1,
  // and with a three-slot ring may read batch i+1 (complete since step i-1)
  // before the barrier. Slot i % S is rewritten at step i+1, after the
  // accumulators' last read of it (loads of it still in flight at the
  // barrier are of batch i+1 < i+S only when S = 3, and land in slot
  // (i+1) % 3, which step i+1 does not write).
  // Each role runs its own loop with the same number of barriers (nb + S),
  // so that the multiplier's register use never meets the accumulator's
  // loop-carried planes. The multiplier waves issue at raised priority: their
  // instruction stream stalls on LDS traffic, and without priority the
  // accumulator wave on the same SIMD takes the issue slots it could have
  // filled once the data arrived; the accumulator keeps issuing nearly at its
  // single-wave rate either way.
  if constexpr (V::kPairs) {
    // Pairs: accumulator wave pw and multiplier wave 4+pw hand batches over
    // through flags[pw] (made, consumed); LDS operations of one wave complete
    // in order, so a counter written after a wave's stores (and a wait for
    // them) shows those stores to a reader that reads the counter first. Every
    // wait is bounded by p.spin_cap sleeps; a wave whose wait ends there
    // without its counter counts one give-up in *p.wait_fail.
    // LDS pointers, so that the polls are LDS reads (a generic pointer makes
    // them flat accesses, whose waits also wait for every global load in flight)
    volatile lds_u32* made = (volatile lds_u32*)&flags[pw][0];
    volatile lds_u32* consumed = (volatile lds_u32*)&flags[pw][1];
    uint32_t gave = 0;  // a wait of this wave gave up (wave-uniform)
    if (mul_role) {
      *made = 0u;
      *consumed = 0u;
    }
    __syncthreads();  // counters set before any wave reads them
    if (mul_role) {
      __builtin_amdgcn_s_setprio(3);
      load_ifm(0, 0, 0);
      // This lane's weight word of batches b, b+1, b+2 in three registers,
      // each loaded three batches ahead of its use, so that a miss in this
      // XCD's L2 is covered by three batches of work (the loop is unrolled by
      // three so that no register still being loaded is copied).
      uint32_t wa = 0, wb = 0, wc = 0;
      fetch_w(0);
      wa = wstage;
      fetch_w(1);
      wb = wstage;
      fetch_w(2);
      wc = wstage;
      auto step = [&](int b, uint32_t& wreg) {
        wstage = wreg;
        store_w(b);  // this wave's weights of batch b (read back below, in order)
        fetch_w(b + 3);
        wreg = wstage;
        if (b >= S) {  // slot b % S held batch b-S: wait until it was added
          uint32_t spin = 0;
          while (__builtin_amdgcn_readfirstlane(*consumed) < (uint32_t)(b - S + 1)) {
            if (spin == p.spin_cap) {
              gave = 1u;
              break;
            }
            __builtin_amdgcn_s_sleep(1);
            ++spin;
          }
        }
        produce(b);  // ends with its stores complete
        *made = (uint32_t)(b + 1);
      };
      int b = 0;
      for (; b + 3 <= nb; b += 3) {
        step(b, wa);
        step(b + 1, wb);
        step(b + 2, wc);
      }
      if (b < nb) step(b, wa);
      if (b + 1 < nb) step(b + 1, wb);
      if (gave && lane == 0) atomicAdd(p.wait_fail, 1u);
      return;
    }
    V::accum_loop(acc, entry(0, 0), entry(1, 0), entry(S - 1, 0), (const lds_u32*)&flags[pw][0],
                  nb, p.spin_cap, gave);
    if (gave && lane == 0) atomicAdd(p.wait_fail, 1u);
  } else {
  if (mul_role) {
    __builtin_amdgcn_s_setprio(3);
    load_ifm(0, 0, 0);
#pragma unroll
    for (int j = 0; j <= 3 - S; ++j) {  // weights stored before the first step
      fetch_w(j);
      store_w(j);
    }
    __syncthreads();
    for (int i = 1 - S; i < nb; ++i) {
      fetch_w(i + 3);
      if (i + S - 1 < nb) produce(i + S - 1);
      store_w(i + 3);
      __syncthreads();
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < S; ++j) __syncthreads();
  uint32_t unused;
  V::accum_loop(acc, entry(0, 0), entry(1, 0), entry(S - 1, 0), nullptr, nb, 0u,
                unused);  // nb barriers
  }
  if (!active) return;
  uint32_t planes[NACC], out[NOUT];
#pragma unroll
  for (int bb = 0; bb < NACC; ++bb) planes[bb] = acc[V::kAccSlot[bb]];
  V::epi(planes, out);
  store_ofm<NOUT, V::wE, V::wF_OUT>(out, ofm, pos, mt, p);
}

// The split kernel with one workgroup per CU: one accumulator/multiplier wave
// pair per SIMD, the netlists' registers anywhere up to v255 and up to four
// products per hand-over. For launches with at most one chain wave per SIMD.
template <class V>
__global__ __launch_bounds__(2 * kConvBlock) void conv2d_split_kernel(
    const uint32_t* __restrict__ ifm, const uint32_t* __restrict__ w, uint32_t* __restrict__ ofm,
    ConvParams p) {
  conv2d_split_body<V>(ifm, w, ofm, p);
}

// The compact form: at most 128 VGPRs a wave (the variant's asm blocks end at
// v128) and an LDS ring of two products per hand-over, so that two workgroups
// share a CU and each SIMD runs two wave pairs. For launches with between one
// and two chain waves per SIMD, where the one-workgroup form would need a
// second round of workgroups.
template <class V>
__global__ __launch_bounds__(2 * kConvBlock) __attribute__((amdgpu_waves_per_eu(4)))
void conv2d_split_compact_kernel(const uint32_t* __restrict__ ifm, const uint32_t* __restrict__ w,
                                 uint32_t* __restrict__ ofm, ConvParams p) {
  conv2d_split_body<V>(ifm, w, ofm, p);
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
  // a lane's words are contiguous: moved up to 16 bytes per instruction
  // (a group's NIN words start 4-byte aligned; the loads and stores of a
  // wave still cover its contiguous span together)
  uint32_t av[NIN], bv[NIN], cv[NIN], rv[NACC];
  __builtin_memcpy(av, a + g * NIN, 4 * NIN);
  __builtin_memcpy(bv, b + g * NIN, 4 * NIN);
  __builtin_memcpy(cv, c + g * NIN, 4 * NIN);
  V::muladd(av, bv, cv, rv);
  __builtin_memcpy(r + g * NACC, rv, 4 * NACC);
}

// Global average pooling on PL32 planes (the pooling layer the paper proposes
// for MobileNets' interface between its last convolution and the fully
// connected layer, Sec. 4). One lane is one (image n, channel word cg): 32
// channels, one per bit. acc = +0; for each position i (rows, then columns):
// acc = add(acc, widen(x_i)); then out = scale(acc, s) (a multiply by the code
// of 1/HW, broadcast into planes). in: [N * HW][CG][NIN], out: [N][CG][NOUT].
template <class V>
__global__ __launch_bounds__(256) void avgpool_kernel(const uint32_t* __restrict__ in,
                                                      uint32_t* __restrict__ out, PoolParams p) {
  constexpr int NIN = V::NIN, NACC = V::NACC, NOUT = V::NOUT, DF = NACC - NIN;
  typedef uint32_t quad_t __attribute__((ext_vector_type(4)));
  constexpr int NQ = (NIN + 3) / 4;
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= (int64_t)p.N * p.CG) return;
  const int64_t n = g / p.CG, cg = g - n * p.CG;
  const uint32_t* src = in + ((size_t)n * p.HW * p.CG + cg) * NIN;
  const size_t step = (size_t)p.CG * NIN;
  auto load = [&](quad_t (&q)[NQ], const uint32_t* ptr) {  // NIN words into 4-word vectors
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
      quad_t v = {0u, 0u, 0u, 0u};
      __builtin_memcpy(&v, ptr + 4 * j, 4 * (NIN - 4 * j < 4 ? NIN - 4 * j : 4));
      q[j] = v;
    }
  };
  uint32_t acc[NACC];
#pragma unroll
  for (int b = 0; b < NACC; ++b) acc[b] = 0u;  // +0
  // Positions are requested kAhead ahead of their add, each into the register
  // set its add has just read (the loop is unrolled by kAhead, so no set is
  // copied): with a few waves in the whole launch, one position of lead left
  // most of each load's latency exposed. Requests past the end reload the
  // last position and are not used.
  constexpr int kAhead = 4;
  quad_t buf[kAhead][NQ];
  const size_t last = (size_t)(p.HW - 1) * step;
  auto pos_ptr = [&](int i) { return src + min((size_t)i * step, last); };
#pragma unroll
  for (int k = 0; k < kAhead; ++k) load(buf[k], pos_ptr(k));
  auto add_pos = [&](quad_t (&q)[NQ], int i) {
    // a scheduling barrier per position: the scheduler would otherwise hoist
    // parts of later adds (those on x alone), and their waits would take in
    // the loads requested ahead
    __builtin_amdgcn_sched_barrier(0);
    uint32_t x[NACC];  // widened: fraction planes move up by DF, zeros below
#pragma unroll
    for (int b = 0; b < DF; ++b) x[b] = 0u;
#pragma unroll
    for (int b = 0; b < NIN; ++b) x[DF + b] = q[b / 4][b % 4];
    V::add(acc, x);
    load(q, pos_ptr(i + kAhead));
  };
  int i = 0;
  for (; i + kAhead <= p.HW; i += kAhead) {
#pragma unroll
    for (int k = 0; k < kAhead; ++k) add_pos(buf[k], i + k);
  }
#pragma unroll
  for (int k = 0; k < kAhead - 1; ++k)
    if (i + k < p.HW) add_pos(buf[k], i + k);
  uint32_t sp[NACC], r[NOUT];
#pragma unroll
  for (int b = 0; b < NACC; ++b) sp[b] = ((p.scale >> b) & 1u) ? 0xFFFFFFFFu : 0u;
  V::scale(acc, sp, r);
#pragma unroll
  for (int b = 0; b < NOUT; ++b) out[(size_t)g * NOUT + b] = r[b];
}

}  // namespace hobflops
