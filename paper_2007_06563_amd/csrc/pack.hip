// Pack (float32 or code -> PL32 bit-planes) and unpack (PL32 -> code or
// float32) kernels. HBM-bound: a pack reads 4 bytes and writes NB/8 bytes per
// value, an unpack the reverse.
//
// Pack: each lane quantises one value per pass; a pass holds two 32-value
// groups (lanes 0-31 and 32-63), and a 32 x 32 bit transpose across the lanes
// of each half turns the 32 codes into the plane words of the group (the bit
// transpose of the paper's bitslice layout, Sec. 3.2): lane b then holds plane
// b, and lanes b < NB of both halves store, 2*NB consecutive words a pass.
// Unpack: lanes b < NB load plane b of their group, and the same transpose
// gives lane j the code of value j.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <type_traits>

#include "codec.hpp"
#include "pack.hpp"

namespace hobflops {

typedef __attribute__((address_space(3))) uint32_t lds_word;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));  // one 16-byte access
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;

// Groups of 32 values a wave handles: two per pass (lanes 0-31, 32-63), U
// passes whose loads are all issued before any value is quantised, so a wave
// keeps U loads per lane in flight. NB (planes per value) is a template
// argument, so the plane loops unroll and their loads issue together. Large
// launches take eight passes a wave (more bytes in flight per CU: 13% faster
// on 2^24 values), small ones four (more waves, for latency).
constexpr int kUSmall = 4, kULarge = 8;
constexpr int64_t kLargeGroups = (int64_t)1 << 18;
constexpr int kUMax = kULarge;

// Index of value j of group q in the [rows][len] source, and whether its
// column 32g + j lies inside the row. With len a multiple of 32 the groups tile
// the flat array, and no division is needed (kIdxDense); otherwise row and
// group come from a division by G, in 32-bit arithmetic when the group count
// allows (kIdxNarrow).
constexpr int kIdxNarrow = 0, kIdxWide = 1, kIdxDense = 2;
// Dense, with 16-byte aligned value and plane arrays: a wave moves its values
// and its plane words with 16-byte accesses through LDS (kIdxDenseVec).
constexpr int kIdxDenseVec = 3;

template <int kIdx>
__device__ __forceinline__ int64_t value_index(int64_t q, int j, int G, int64_t len,
                                               bool& in_row) {
  if (kIdx == kIdxDense || kIdx == kIdxDenseVec) {
    in_row = true;
    return q * 32 + j;
  }
  int64_t r, g;
  if (kIdx == kIdxWide) {
    r = q / G;
    g = q - r * G;
  } else {
    const uint32_t q32 = (uint32_t)q, r32 = q32 / (uint32_t)G;
    r = r32;
    g = q32 - r32 * (uint32_t)G;
  }
  const int64_t col = g * 32 + j;
  in_row = col < len;
  return r * len + col;
}

// 32 x 32 bit transpose across each 32-lane half of a wave: lane j returns
// the word whose bit i is bit j of lane i's x. Five stages d = 16, 8, 4, 2, 1
// swap the off-diagonal d x d blocks of lane pairs (j, j ^ d): the lower lane
// takes its partner's bits i (i & d == 0) into positions i + d, the upper one
// its partner's bits i + d into positions i. The stages act on disjoint pairs
// of (lane bit, word bit) coordinates, so they may run in any order.
//
// No stage goes through LDS. The stages d = 8, 4, 2, 1 stay inside 16-lane
// rows: a DPP move brings the partner's word (row rotate by 8, quad
// permutes, and for d = 4 a mirror of each 8 lanes followed by the quad
// permute j ^ 3), then one rotate and one bit select (v_bitop3_b32, truth
// table 0xCA: mask ? r : x) with per-lane rotate amounts and masks set up once
// (row_transpose_setup). The stage d = 16 pairs rows 0-1 and 2-3 of a wave;
// it takes two words a, b at once: v_permlane16_swap_b32 gives every lane of
// row 0 the words of a's lanes j and j + 16 and every lane of row 1 those of
// b's, and two byte permutes form P (low halves) and Q (high halves). After
// it, row 0 (2) of P holds a's result at lanes 0-15 of its half and row 0 (2)
// of Q a's result at lanes 16-31, rows 1 and 3 the same for b ("pair
// layout"); a second swap of P and Q gives back the plain layout.
struct RowT {
  uint32_t rot[4], mask[4];  // stages d = 8, 4, 2, 1
};

__device__ __forceinline__ RowT row_transpose_setup(int j) {
  RowT t;
  constexpr uint32_t kLow[4] = {0x00FF00FFu, 0x0F0F0F0Fu, 0x33333333u, 0x55555555u};
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int d = 8 >> s;
    const bool upper = (j & d) != 0;
    t.rot[s] = upper ? d : 32 - d;               // rotate right: by d, or left by d
    t.mask[s] = upper ? kLow[s] : ~kLow[s];      // the positions taken from the partner
  }
  return t;
}

// The word of lane j ^ (8 >> S) of the same 16-lane row (DPP moves).
template <int S>
__device__ __forceinline__ uint32_t row_xor(uint32_t x) {
  if constexpr (S == 0) {
    return __builtin_amdgcn_mov_dpp(x, 0x128, 0xF, 0xF, false);  // row_ror:8
  } else if constexpr (S == 1) {
    const uint32_t m = __builtin_amdgcn_mov_dpp(x, 0x141, 0xF, 0xF, false);  // j ^ 7
    return __builtin_amdgcn_mov_dpp(m, 0x1B, 0xF, 0xF, false);  // quad_perm [3,2,1,0]: j ^ 3
  } else if constexpr (S == 2) {
    return __builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, false);  // quad_perm [2,3,0,1]
  } else {
    return __builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, false);  // quad_perm [1,0,3,2]
  }
}

// The stages d = 8, 4, 2, 1 on N words.
template <int N>
__device__ __forceinline__ void row_transpose(uint32_t (&x)[N], const RowT& t) {
#define HOBFLOPS_STAGE(S)                                                       \
  {                                                                             \
    uint32_t p[N];                                                              \
    _Pragma("unroll") for (int u = 0; u < N; ++u) p[u] = row_xor<S>(x[u]);      \
    _Pragma("unroll") for (int u = 0; u < N; ++u) {                             \
      const uint32_t r = __builtin_amdgcn_alignbit(p[u], p[u], t.rot[S]);       \
      x[u] = __builtin_amdgcn_bitop3_b32(t.mask[S], r, x[u], 0xCA);             \
    }                                                                           \
  }
  HOBFLOPS_STAGE(0)
  HOBFLOPS_STAGE(1)
  HOBFLOPS_STAGE(2)
  HOBFLOPS_STAGE(3)
#undef HOBFLOPS_STAGE
}

// Exchanges rows 1 and 3 of a with rows 0 and 2 of b.
__device__ __forceinline__ void row_swap(uint32_t& a, uint32_t& b) {
  const auto s = __builtin_amdgcn_permlane16_swap(a, b, false, false);
  a = s[0];
  b = s[1];
}

// Low and high 16-bit halves of two words: lo = lo16(a) | lo16(b) << 16,
// hi = hi16(a) | hi16(b) << 16.
__device__ __forceinline__ uint32_t halves_lo(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x05040100u);
}
__device__ __forceinline__ uint32_t halves_hi(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x07060302u);
}

// The stage d = 16 on words a, b in the plain layout; P and Q in the pair
// layout. kHigh false: the words' high halves are zero and Q (then zero) is
// not formed.
template <bool kHigh>
__device__ __forceinline__ void stage16_to_pairs(uint32_t a, uint32_t b, uint32_t& P,
                                                 uint32_t& Q) {
  row_swap(a, b);
  P = halves_lo(a, b);
  if constexpr (kHigh) Q = halves_hi(a, b);
}

// The stage d = 16 on words a, b given in the pair layout (P: a's lanes 0-15
// in row 0 and b's in row 1, Q: their lanes 16-31; rows 2 and 3 likewise for
// the wave's second half); a and b come out in the plain layout.
__device__ __forceinline__ void stage16_from_pairs(uint32_t P, uint32_t Q, uint32_t& a,
                                                   uint32_t& b) {
  a = halves_lo(P, Q);
  b = halves_hi(P, Q);
  row_swap(a, b);
}

// Whole transpose, plain layout in and out, of U (even) words.
template <int U>
__device__ __forceinline__ void lane_transpose(uint32_t (&x)[U], int j) {
  static_assert(U % 2 == 0, "words go through the d = 16 stage in pairs");
  uint32_t P[U / 2], Q[U / 2];
#pragma unroll
  for (int v = 0; v < U / 2; ++v) stage16_to_pairs<true>(x[2 * v], x[2 * v + 1], P[v], Q[v]);
  const RowT t = row_transpose_setup(j);
  row_transpose(P, t);
  row_transpose(Q, t);
#pragma unroll
  for (int v = 0; v < U / 2; ++v) {
    row_swap(P[v], Q[v]);
    x[2 * v] = P[v];
    x[2 * v + 1] = Q[v];
  }
}

// Group (within the chunk's pass set) of a lane's word of pair v in the pair
// layout: row r of the passes (2v, 2v + 1) holds group
// 2 (2v + (r & 1)) + (r >> 1); the lane's plane is lane & 15 in P, 16 more
// in Q.
__device__ __forceinline__ int pair_group(int v, int lane) {
  const int r = lane >> 4;
  return 4 * v + 2 * (r & 1) + (r >> 1);
}

// A pack launch covers up to kMaxJobs ranges of groups, each of one tensor
// (all in one format): range k holds groups [q0, q1) of its tensor and starts
// at wave wave0 of the launch. A wave finds its range by comparing its index
// with the wave0 of every range (uniform scalar work).
constexpr int kMaxJobs = 8;
struct PackRange {
  const void* src;
  uint32_t* planes;
  int64_t len, q0, q1, wave0;
  int G, kind, idx;  // groups per row, source kind, index mode
};
struct PackLaunch {
  PackRange r[kMaxJobs];
  int count;
};

// Source indices of a wave's U passes: group q = q0 + (local wave * U + u)
// * 2 + half of range R; a lane without a value gets index 0 (loaded, then
// ignored).
template <int kIdx, int U>
__device__ __forceinline__ void value_indices(const PackRange& R, int64_t wave, int lane,
                                              int64_t (&idx)[U], bool (&have)[U]) {
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t q = R.q0 + ((wave - R.wave0) * U + u) * 2 + (lane >> 5);
    bool in_row;
    const int64_t i = value_index<kIdx>(q < R.q1 ? q : R.q0, lane & 31, R.G, R.len, in_row);
    have[u] = q < R.q1 && in_row;
    idx[u] = have[u] ? i : 0;
  }
}

// Decoder of one pass set to float32 bits, or codes kept (uniform branch on
// the destination kind and format).
template <int U>
__device__ __forceinline__ void decode_all(uint32_t (&x)[U], int kind, int wE, int wF) {
  if (kind != 0) return;
  if (wE <= 7) {
#pragma unroll
    for (int u = 0; u < U; ++u) x[u] = decode_narrow(x[u], wE, wF);
  } else {
#pragma unroll
    for (int u = 0; u < U; ++u) x[u] = decode_bits(x[u], wE, wF);
  }
}

// Quantiser of one pass set (uniform branch on the source kind and format).
template <int NB, int U>
__device__ __forceinline__ void quantize_all(uint32_t (&x)[U], const bool (&have)[U], int kind,
                                             int wE, int wF) {
  constexpr uint32_t nbmask = NB >= 32 ? 0xFFFFFFFFu : ((1u << (NB & 31)) - 1u);
  if (kind != 0) {
#pragma unroll
    for (int u = 0; u < U; ++u) x[u] = have[u] ? (x[u] & nbmask) : 0u;
  } else if (wE <= 7 && wF <= 22) {
#pragma unroll
    for (int u = 0; u < U; ++u) x[u] = have[u] ? quantize_narrow(x[u], wE, wF) : 0u;
  } else {
#pragma unroll
    for (int u = 0; u < U; ++u) x[u] = have[u] ? quantize_bits(x[u], wE, wF) : 0u;
  }
}

// Dense ranges with 16-byte aligned arrays (kIdxDenseVec), whole chunks of
// 2U groups (64U values) only: a wave takes chunks_per_wave(U) consecutive chunks
// and keeps the next two chunks' loads in flight while it works on one, so
// that memory stays busy through the quantiser and the transpose. A chunk's
// values come in with 16-byte loads, go through this wave's LDS buffer so
// that each lane takes value j of its half's group per pass, and after the
// transpose the plane words go back through the same buffer and out with
// 16-byte stores. Nothing in the chunk path branches on data, so the waits
// for a load count only the loads before it. A range's last groups that do
// not fill a chunk form a range of their own (the per-value path). LDS
// operations of one wave complete in order, so only the compiler needs to be
// kept from reordering them (wave barriers). Four chunks a wave measured
// faster than two or eight on large launches, for the pack and the unpack
// alike; launches of fewer groups (U = kUSmall, about 1.5 waves a SIMD at
// four chunks on a 1.6 M-value tensor) measured faster at two.
constexpr int kChunksLarge = 4, kChunksSmall = 2;
__host__ __device__ constexpr int chunks_per_wave(int U) {
  return U == kULarge ? kChunksLarge : kChunksSmall;
}

template <int U>
struct ChunkRegs {
  u32x4 v[U / 4];  // one chunk's 16U 16-byte units, U/4 per lane
};

// Requests chunk `chunk` of the range, clamped to the range's last chunk (a
// request past the end loads data that is not used).
template <int U>
__device__ __forceinline__ void pack_load_chunk(const PackRange& R, int64_t chunk, int lane,
                                                ChunkRegs<U>& r) {
  const int64_t last = (R.q1 - R.q0) / (2 * U) - 1;
  const u32x4* src =
      reinterpret_cast<const u32x4*>(R.src) + (R.q0 + min(chunk, last) * 2 * U) * 8;
#pragma unroll
  for (int k = 0; k < U / 4; ++k) r.v[k] = src[lane + 64 * k];
}

template <int NB, int U>
__device__ __forceinline__ void pack_process_chunk(const PackRange& R, int64_t chunk, int lane,
                                                   int wE, int wF, const ChunkRegs<U>& r,
                                                   lds_word* buf) {
  const int64_t qw0 = R.q0 + chunk * 2 * U;
  if (qw0 >= R.q1) return;  // past the range (uniform)
  constexpr int kWords = 2 * U * NB;  // plane words of a chunk
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int k = 0; k < U / 4; ++k) reinterpret_cast<lds_u32x4*>(buf)[lane + 64 * k] = r.v[k];
  __builtin_amdgcn_wave_barrier();
  uint32_t x[U];
  bool have[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    x[u] = buf[64 * u + lane];
    have[u] = true;
  }
  __builtin_amdgcn_wave_barrier();  // every value read before the buffer is rewritten
  quantize_all<NB, U>(x, have, R.kind, wE, wF);
  // the transpose, left in the pair layout: codes of NB <= 16 bits have no
  // high halves, and then the planes 16-31 (Q) are neither formed nor kept
  constexpr bool kHigh = NB > 16;
  uint32_t P[U / 2], Q[U / 2];
#pragma unroll
  for (int v = 0; v < U / 2; ++v) stage16_to_pairs<kHigh>(x[2 * v], x[2 * v + 1], P[v], Q[v]);
  const RowT t = row_transpose_setup(lane & 15);
  row_transpose(P, t);
  if constexpr (kHigh) row_transpose(Q, t);
  const int l = lane & 15;
#pragma unroll
  for (int v = 0; v < U / 2; ++v) {
    const int g = pair_group(v, lane);
    if (l < NB) buf[g * NB + l] = P[v];
    if constexpr (kHigh)
      if (16 + l < NB) buf[g * NB + 16 + l] = Q[v];
  }
  __builtin_amdgcn_wave_barrier();
  u32x4* dst = reinterpret_cast<u32x4*>(R.planes + qw0 * NB);
#pragma unroll
  for (int k = 0; k < (kWords / 4 + 63) / 64; ++k) {
    const int unit = lane + 64 * k;
    if (kWords / 4 % 64 == 0 || unit < kWords / 4)
      dst[unit] = reinterpret_cast<const lds_u32x4*>(buf)[unit];
  }
}

// Eight waves a SIMD (at most 64 VGPRs): the compiler then keeps a few
// values in scratch, and the launch still runs faster than at the six waves
// its free choice of about 76 VGPRs allows.
template <int NB, int U>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(8))) void pack_kernel(
    const PackLaunch L, int wE, int wF) {
  const int lane = threadIdx.x & 63;
  // the wave index as a wave-uniform value, so that the range lookup, the
  // range's fields and the mode branches stay scalar
  const int64_t wave = (int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int j = lane & 31;
  int k = 0;
#pragma unroll
  for (int t = 1; t < kMaxJobs; ++t) k = (t < L.count && wave >= L.r[t].wave0) ? t : k;
  const PackRange& R = L.r[k];
  if (R.idx == kIdxDenseVec) {  // uniform branch
    __shared__ uint32_t stage[4][64 * U > 2 * U * NB ? 64 * U : 2 * U * NB];
    lds_word* buf = (lds_word*)stage[threadIdx.x >> 6];
    constexpr int kChunksPerWave = chunks_per_wave(U);
    const int64_t c0 = (wave - R.wave0) * kChunksPerWave;
    // two register sets, alternating (the loop is unrolled by two so that no
    // set still being loaded is copied)
    ChunkRegs<U> ra, rb;
    pack_load_chunk<U>(R, c0, lane, ra);
    pack_load_chunk<U>(R, c0 + 1, lane, rb);
#pragma unroll
    for (int c = 0; c < kChunksPerWave; c += 2) {
      pack_process_chunk<NB, U>(R, c0 + c, lane, wE, wF, ra, buf);
      if (c + 2 < kChunksPerWave) pack_load_chunk<U>(R, c0 + c + 2, lane, ra);
      pack_process_chunk<NB, U>(R, c0 + c + 1, lane, wE, wF, rb, buf);
      if (c + 3 < kChunksPerWave) pack_load_chunk<U>(R, c0 + c + 3, lane, rb);
    }
    return;
  }
  int64_t idx[U];
  bool have[U];
  if (R.idx == kIdxDense)  // uniform branch
    value_indices<kIdxDense, U>(R, wave, lane, idx, have);
  else if (R.idx == kIdxWide)
    value_indices<kIdxWide, U>(R, wave, lane, idx, have);
  else
    value_indices<kIdxNarrow, U>(R, wave, lane, idx, have);
  // the U loads together, every lane loading, with no branch between them: a
  // load under a branch makes the compiler wait for all loads issued before it
  uint32_t x[U];
#pragma unroll
  for (int u = 0; u < U; ++u) x[u] = ((const uint32_t*)R.src)[idx[u]];
  // one uniform branch for the whole pass set
  quantize_all<NB, U>(x, have, R.kind, wE, wF);
  // lane j of each half now holds plane j of its group
  lane_transpose(x, j);
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t q = R.q0 + ((wave - R.wave0) * U + u) * 2 + (lane >> 5);
    if (q < R.q1 && j < NB) R.planes[q * NB + j] = x[u];
  }
}

// The unpack of dense tensors with 16-byte aligned arrays, whole chunks of 2U
// groups only (the mirror of the pack's; the groups after the last whole
// chunk go to the per-value path): a wave takes chunks_per_wave(U) consecutive
// chunks, with the next two chunks' plane words in flight while it works on
// one. A chunk's words come in with 16-byte loads, go through LDS so that
// each lane takes plane j of its half's group per pass, and after the
// transpose and the decode the 64U values go back through LDS and out with
// 16-byte stores.
template <int NB, int U>
struct PlaneRegs {
  u32x4 v[(2 * U * NB / 4 + 63) / 64];  // one chunk's plane words, 16 bytes a unit
};

template <int NB, int U>
__device__ __forceinline__ void unpack_load_chunk(const uint32_t* __restrict__ planes,
                                                  int64_t nchunks, int64_t chunk, int lane,
                                                  PlaneRegs<NB, U>& r) {
  constexpr int kUnits = 2 * U * NB / 4;
  // clamped: a request past the end loads a chunk that is not used
  const u32x4* src =
      reinterpret_cast<const u32x4*>(planes + min(chunk, nchunks - 1) * 2 * U * NB);
#pragma unroll
  for (int k = 0; k < (kUnits + 63) / 64; ++k) {
    const int unit = lane + 64 * k;
    r.v[k] = src[kUnits % 64 == 0 ? unit : min(unit, kUnits - 1)];
  }
}

template <int NB, int U>
__device__ __forceinline__ void unpack_process_chunk(int64_t nchunks, int64_t chunk, int lane,
                                                     int kind, int wE, int wF,
                                                     const PlaneRegs<NB, U>& r,
                                                     uint32_t* __restrict__ dst, lds_word* buf) {
  constexpr int kUnits = 2 * U * NB / 4;
  if (chunk >= nchunks) return;  // past the end (uniform)
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int k = 0; k < (kUnits + 63) / 64; ++k) {
    const int unit = lane + 64 * k;
    if (kUnits % 64 == 0 || unit < kUnits) reinterpret_cast<lds_u32x4*>(buf)[unit] = r.v[k];
  }
  __builtin_amdgcn_wave_barrier();
  // the plane words come in in the pair layout (planes 16-31 only when NB > 16)
  constexpr bool kHigh = NB > 16;
  const int l = lane & 15;
  uint32_t P[U / 2], Q[U / 2];
#pragma unroll
  for (int v = 0; v < U / 2; ++v) {
    const int g = pair_group(v, lane);
    const uint32_t w = buf[g * NB + min(l, NB - 1)];
    P[v] = l < NB ? w : 0u;
    if constexpr (kHigh) {
      const uint32_t w2 = buf[g * NB + min(16 + l, NB - 1)];
      Q[v] = 16 + l < NB ? w2 : 0u;
    } else {
      Q[v] = 0u;
    }
  }
  __builtin_amdgcn_wave_barrier();  // every word read before the buffer is rewritten
  const RowT t = row_transpose_setup(l);
  row_transpose(P, t);
  if constexpr (kHigh) row_transpose(Q, t);
  uint32_t x[U];
#pragma unroll
  for (int v = 0; v < U / 2; ++v) stage16_from_pairs(P[v], Q[v], x[2 * v], x[2 * v + 1]);
  decode_all<U>(x, kind, wE, wF);
#pragma unroll
  for (int u = 0; u < U; ++u) buf[64 * u + lane] = x[u];
  __builtin_amdgcn_wave_barrier();
  u32x4* d = reinterpret_cast<u32x4*>(dst) + chunk * 16 * U;
#pragma unroll
  for (int k = 0; k < U / 4; ++k) d[lane + 64 * k] = reinterpret_cast<const lds_u32x4*>(buf)[lane + 64 * k];
}

template <int NB, int kIdx, int U>
__global__ __launch_bounds__(256) void unpack_kernel(const uint32_t* __restrict__ planes,
                                                     int kind, int64_t len, int G, int wE,
                                                     int wF, void* __restrict__ dst,
                                                     int64_t ngroups) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int j = lane & 31;
  if constexpr (kIdx == kIdxDenseVec) {  // ngroups is a whole number of chunks here
    __shared__ uint32_t stage[4][64 * U > 2 * U * NB ? 64 * U : 2 * U * NB];
    lds_word* buf = (lds_word*)stage[threadIdx.x >> 6];
    const int64_t nchunks = ngroups / (2 * U);
    constexpr int kChunksPerWave = chunks_per_wave(U);
    const int64_t c0 = __builtin_amdgcn_readfirstlane((int)(wave & 0x7FFFFFFF)) *
                       (int64_t)kChunksPerWave;
    PlaneRegs<NB, U> ra, rb;
    unpack_load_chunk<NB, U>(planes, nchunks, c0, lane, ra);
    unpack_load_chunk<NB, U>(planes, nchunks, c0 + 1, lane, rb);
#pragma unroll
    for (int c = 0; c < kChunksPerWave; c += 2) {
      unpack_process_chunk<NB, U>(nchunks, c0 + c, lane, kind, wE, wF, ra, (uint32_t*)dst, buf);
      if (c + 2 < kChunksPerWave) unpack_load_chunk<NB, U>(planes, nchunks, c0 + c + 2, lane, ra);
      unpack_process_chunk<NB, U>(nchunks, c0 + c + 1, lane, kind, wE, wF, rb, (uint32_t*)dst,
                                  buf);
      if (c + 3 < kChunksPerWave) unpack_load_chunk<NB, U>(planes, nchunks, c0 + c + 3, lane, rb);
    }
    return;
  }
  uint32_t x[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {  // lane j < NB: plane j of its group (clamped load)
    const int64_t q = (wave * U + u) * 2 + (lane >> 5);
    const uint32_t v = planes[(q < ngroups ? q : 0) * NB + min(j, NB - 1)];
    x[u] = j < NB ? v : 0u;
  }
  // the transpose is its own inverse: lane j now holds the code at column 32g + j
  lane_transpose(x, j);
  decode_all<U>(x, kind, wE, wF);
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t q = (wave * U + u) * 2 + (lane >> 5);
    if (q >= ngroups) continue;
    bool in_row;
    const int64_t i = value_index<kIdx>(q, j, G, len, in_row);
    if (!in_row) continue;
    ((uint32_t*)dst)[i] = x[u];
  }
}

namespace {

// NB = 3 + wE + wF runs from 6 to 32; f gets the kernel types of the four
// index modes.
template <template <int, int> class K, int NB = 6>
struct nb_dispatch {
  template <class F>
  static hipError_t run(int nb, F&& f) {
    if (nb == NB)
      return f(K<NB, kIdxNarrow>{}, K<NB, kIdxWide>{}, K<NB, kIdxDense>{}, K<NB, kIdxDenseVec>{});
    return nb_dispatch<K, NB + 1>::run(nb, f);
  }
};
template <template <int, int> class K>
struct nb_dispatch<K, 33> {
  template <class F>
  static hipError_t run(int, F&&) {
    return hipErrorInvalidValue;
  }
};

template <int U, int NB = 6>
struct pack_nb {
  static hipError_t run(int nb, unsigned blocks, hipStream_t stream, const PackLaunch& L, int wE,
                        int wF) {
    if (nb != NB) return pack_nb<U, NB + 1>::run(nb, blocks, stream, L, wE, wF);
    hipLaunchKernelGGL((pack_kernel<NB, U>), dim3(blocks), dim3(256), 0, stream, L, wE, wF);
    return hipGetLastError();
  }
};
template <int U>
struct pack_nb<U, 33> {
  static hipError_t run(int, unsigned, hipStream_t, const PackLaunch&, int, int) {
    return hipErrorInvalidValue;
  }
};

template <int U>
struct UnpackU {
  template <int NB, int M>
  struct K {
    static constexpr auto fn = unpack_kernel<NB, M, U>;
  };
};

}  // namespace

// Index mode of a tensor: dense when the row length is a multiple of 32 (with
// 16-byte accesses when both arrays allow them: vec), else 32-bit division
// when the group count allows.
static int index_mode(int64_t len, int64_t ngroups, bool vec = false) {
  if (len % 32 == 0) return vec ? kIdxDenseVec : kIdxDense;
  return ngroups + 2 * kUMax >= ((int64_t)1 << 31) ? kIdxWide : kIdxNarrow;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// The unpack kernel of the tensor's index mode, U passes a wave.
template <int U, template <int, int> class K, class... Args>
static hipError_t launch_groups(int NB, int64_t len, int64_t ngroups, bool vec,
                                hipStream_t stream, Args... args) {
  const int mode = index_mode(len, ngroups, vec);
  const int64_t chunks = (ngroups + 2 * U - 1) / (2 * U);
  const int64_t waves =
      mode == kIdxDenseVec ? (chunks + chunks_per_wave(U) - 1) / chunks_per_wave(U) : chunks;
  const int64_t blocks = (waves + 3) / 4;
  if (blocks == 0) return hipSuccess;
  return nb_dispatch<K>::run(NB, [&](auto narrow_k, auto wide_k, auto dense_k, auto vec_k) {
    if (mode == kIdxDenseVec)
      hipLaunchKernelGGL(decltype(vec_k)::fn, dim3((unsigned)blocks), dim3(256), 0, stream,
                         args...);
    else if (mode == kIdxDense)
      hipLaunchKernelGGL(decltype(dense_k)::fn, dim3((unsigned)blocks), dim3(256), 0, stream,
                         args...);
    else if (mode == kIdxWide)
      hipLaunchKernelGGL(decltype(wide_k)::fn, dim3((unsigned)blocks), dim3(256), 0, stream,
                         args...);
    else
      hipLaunchKernelGGL(decltype(narrow_k)::fn, dim3((unsigned)blocks), dim3(256), 0, stream,
                         args...);
    return hipGetLastError();
  });
}

hipError_t launch_pack_batch(const PackTensor* t, int count, int wE, int wF, hipStream_t stream) {
  // a range holds at most 2^25 groups and a launch at most 2^22 waves, so
  // that the grid (64 threads a wave) stays far below 2^32 threads
  constexpr int64_t kRangeGroups = (int64_t)1 << 25, kLaunchWaves = (int64_t)1 << 22;
  const int NB = 3 + wE + wF;
  int64_t total = 0;
  for (int n = 0; n < count; ++n) total += t[n].rows * ((t[n].len + 31) / 32);
  const int U = total >= kLargeGroups ? kULarge : kUSmall;
  PackLaunch L{};
  int64_t waves = 0;
  auto flush = [&]() -> hipError_t {
    if (L.count == 0) return hipSuccess;
    const unsigned blocks = (unsigned)((waves + 3) / 4);
    const hipError_t e = U == kULarge
                             ? pack_nb<kULarge>::run(NB, blocks, stream, L, wE, wF)
                             : pack_nb<kUSmall>::run(NB, blocks, stream, L, wE, wF);
    L = PackLaunch{};
    waves = 0;
    return e;
  };
  for (int n = 0; n < count; ++n) {
    const int64_t G = (t[n].len + 31) / 32;
    const int64_t ngroups = t[n].rows * G;
    for (int64_t q0 = 0; q0 < ngroups; q0 += kRangeGroups) {
      const int64_t q1 = std::min(ngroups, q0 + kRangeGroups);
      const int64_t nw = (q1 - q0 + 2 * U - 1) / (2 * U);
      if (L.count == kMaxJobs || waves + nw > kLaunchWaves) {
        const hipError_t e = flush();
        if (e != hipSuccess) return e;
      }
      // 16-byte accesses where the range's values and planes both start
      // 16-byte aligned (a range start is a multiple of 2^25 groups), for its
      // whole chunks of 2U groups; the groups after them, if any, form a range
      // of their own
      const bool vec = aligned16(t[n].src) && aligned16(t[n].planes + q0 * NB);
      const int mode = index_mode(t[n].len, ngroups, vec);
      const int64_t qv = mode == kIdxDenseVec ? q0 + (q1 - q0) / (2 * U) * 2 * U : q0;
      if (qv > q0) {
        L.r[L.count++] = PackRange{t[n].src, t[n].planes, t[n].len, q0, qv, waves, (int)G,
                                   t[n].kind, kIdxDenseVec};
        waves += ((qv - q0) / (2 * U) + chunks_per_wave(U) - 1) / chunks_per_wave(U);
      }
      if (q1 > qv) {
        if (L.count == kMaxJobs) {
          const hipError_t e = flush();
          if (e != hipSuccess) return e;
        }
        L.r[L.count++] = PackRange{t[n].src, t[n].planes, t[n].len, qv, q1, waves, (int)G,
                                   t[n].kind, index_mode(t[n].len, ngroups, false)};
        waves += (q1 - qv + 2 * U - 1) / (2 * U);
      }
    }
  }
  return flush();
}

hipError_t launch_pack(const void* src, int kind, int64_t rows, int64_t len, int wE, int wF,
                       uint32_t* planes, hipStream_t stream) {
  const PackTensor t{src, kind, rows, len, planes};
  return launch_pack_batch(&t, 1, wE, wF, stream);
}

hipError_t launch_unpack(const uint32_t* planes, int64_t rows, int64_t len, int wE, int wF,
                         int kind, void* dst, hipStream_t stream) {
  const int64_t G = (len + 31) / 32;
  const int64_t ngroups = rows * G;
  const int NB = 3 + wE + wF;
  // dense with 16-byte aligned arrays: whole chunks of 2U groups with 16-byte
  // accesses, the groups after them (if any) per value, in a second launch
  const bool vec = len % 32 == 0 && aligned16(planes) && aligned16(dst);
  auto run = [&](auto u_tag) -> hipError_t {
    constexpr int U = decltype(u_tag)::value;
    const int64_t qv = vec ? ngroups / (2 * U) * 2 * U : 0;
    if (qv > 0) {
      const hipError_t e = launch_groups<U, UnpackU<U>::template K>(NB, len, qv, true, stream, planes,
                                                          kind, len, (int)G, wE, wF, dst, qv);
      if (e != hipSuccess) return e;
    }
    if (qv == ngroups) return hipSuccess;
    // the rest: dense groups from qv on (values 32 qv on), or the whole tensor
    return launch_groups<U, UnpackU<U>::template K>(NB, len, ngroups - qv, false, stream,
                                          planes + qv * NB, kind, len, (int)G, wE, wF,
                                          (void*)((uint32_t*)dst + qv * 32), ngroups - qv);
  };
  if (ngroups >= kLargeGroups) return run(std::integral_constant<int, kULarge>{});
  return run(std::integral_constant<int, kUSmall>{});
}

}  // namespace hobflops
