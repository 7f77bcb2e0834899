// Issue-rate probe of the VALU on the device the library runs on (a
// diagnostic for the roofline of the bitsliced kernels, not part of the
// computing path): waves run long straight-line streams of 8-byte
// v_bitop3_b32 and time them with the shader clock (s_memtime) and the
// constant 100 MHz clock (s_memrealtime). It answers what the convolution
// kernels' ceilings depend on: how often one wave can issue a VALU
// instruction, how often a SIMD can when several waves share it, whether
// instructions whose source VGPRs share a bank (register number mod 4) cost
// more, and at what clock the shader runs under this load.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

// One 8-byte instruction: dest, then three sources, all explicit registers.
#define HOBFLOPS_OP(d, a, b, c) "v_bitop3_b32 v" #d ", v" #a ", v" #b ", v" #c " bitop3:0x96\n"
// One 4-byte instruction (VOP2 encoding): dest, then two sources.
#define HOBFLOPS_OP2(d, a, b) "v_xor_b32_e32 v" #d ", v" #a ", v" #b "\n"
// Eight instructions whose sources lie in banks 1, 2 and 3 and whose
// destinations lie in bank 0 (no two sources of an instruction in one bank).
#define HOBFLOPS_BLOCK_FREE                                                          \
  HOBFLOPS_OP(32, 45, 54, 59) HOBFLOPS_OP(36, 49, 58, 63) HOBFLOPS_OP(40, 53, 62, 35) \
  HOBFLOPS_OP(44, 57, 34, 39) HOBFLOPS_OP(48, 61, 38, 43) HOBFLOPS_OP(52, 33, 42, 47) \
  HOBFLOPS_OP(56, 37, 46, 51) HOBFLOPS_OP(60, 41, 50, 55)
// The same with the first two sources of every instruction in bank 1.
#define HOBFLOPS_BLOCK_SHARED                                                        \
  HOBFLOPS_OP(32, 45, 53, 59) HOBFLOPS_OP(36, 49, 57, 63) HOBFLOPS_OP(40, 53, 61, 35) \
  HOBFLOPS_OP(44, 57, 33, 39) HOBFLOPS_OP(48, 61, 37, 43) HOBFLOPS_OP(52, 33, 41, 47) \
  HOBFLOPS_OP(56, 37, 45, 51) HOBFLOPS_OP(60, 41, 49, 55)
// Eight 4-byte instructions, sources in banks 1 and 2, destinations in bank 0.
#define HOBFLOPS_BLOCK_VOP2                                                          \
  HOBFLOPS_OP2(32, 45, 54) HOBFLOPS_OP2(36, 49, 58) HOBFLOPS_OP2(40, 53, 62)          \
  HOBFLOPS_OP2(44, 57, 34) HOBFLOPS_OP2(48, 61, 38) HOBFLOPS_OP2(52, 33, 42)          \
  HOBFLOPS_OP2(56, 37, 46) HOBFLOPS_OP2(60, 41, 50)
// Eight instructions, each reading the previous one's result.
#define HOBFLOPS_BLOCK_CHAIN                                                         \
  HOBFLOPS_OP(32, 45, 54, 60) HOBFLOPS_OP(36, 49, 58, 32) HOBFLOPS_OP(40, 53, 62, 36) \
  HOBFLOPS_OP(44, 57, 34, 40) HOBFLOPS_OP(48, 61, 38, 44) HOBFLOPS_OP(52, 33, 42, 48) \
  HOBFLOPS_OP(56, 37, 46, 52) HOBFLOPS_OP(60, 41, 50, 56)
// Eight instructions, each reading the result of the one two before.
#define HOBFLOPS_BLOCK_DIST2                                                         \
  HOBFLOPS_OP(32, 45, 54, 56) HOBFLOPS_OP(36, 49, 58, 60) HOBFLOPS_OP(40, 53, 62, 32) \
  HOBFLOPS_OP(44, 57, 34, 36) HOBFLOPS_OP(48, 61, 38, 40) HOBFLOPS_OP(52, 33, 42, 44) \
  HOBFLOPS_OP(56, 37, 46, 48) HOBFLOPS_OP(60, 41, 50, 52)
// Eight instructions, each reading the result of the one four before.
#define HOBFLOPS_BLOCK_DIST4                                                         \
  HOBFLOPS_OP(32, 45, 54, 48) HOBFLOPS_OP(36, 49, 58, 52) HOBFLOPS_OP(40, 53, 62, 56) \
  HOBFLOPS_OP(44, 57, 34, 60) HOBFLOPS_OP(48, 61, 38, 32) HOBFLOPS_OP(52, 33, 42, 36) \
  HOBFLOPS_OP(56, 37, 46, 40) HOBFLOPS_OP(60, 41, 50, 44)
// Four 8-byte and four 4-byte instructions, alternating.
#define HOBFLOPS_BLOCK_MIXED                                                         \
  HOBFLOPS_OP(32, 45, 54, 59) HOBFLOPS_OP2(36, 49, 58) HOBFLOPS_OP(40, 53, 62, 35)    \
  HOBFLOPS_OP2(44, 57, 34) HOBFLOPS_OP(48, 61, 38, 43) HOBFLOPS_OP2(52, 33, 42)       \
  HOBFLOPS_OP(56, 37, 46, 51) HOBFLOPS_OP2(60, 41, 50)
// A 4-byte v_xor_b32, seven 8-byte instructions and an s_nop 0: eight
// instructions and 64 bytes, so alignment carries over from group to group.
#define HOBFLOPS_BLOCK_NOP                                                           \
  HOBFLOPS_OP2(32, 45, 54) HOBFLOPS_OP(36, 49, 58, 63) HOBFLOPS_OP(40, 53, 62, 35)    \
  HOBFLOPS_OP(44, 57, 34, 39) HOBFLOPS_OP(48, 61, 38, 43) HOBFLOPS_OP(52, 33, 42, 47) \
  HOBFLOPS_OP(56, 37, 46, 51) HOBFLOPS_OP(60, 41, 50, 55) "s_nop 0\n"
// One 4-byte instruction then seven 8-byte ones: every other group of seven
// starts at an address 4 mod 8.
#define HOBFLOPS_BLOCK_HALF                                                          \
  HOBFLOPS_OP2(32, 45, 54) HOBFLOPS_OP(36, 49, 58, 63) HOBFLOPS_OP(40, 53, 62, 35)    \
  HOBFLOPS_OP(44, 57, 34, 39) HOBFLOPS_OP(48, 61, 38, 43) HOBFLOPS_OP(52, 33, 42, 47) \
  HOBFLOPS_OP(56, 37, 46, 51) HOBFLOPS_OP(60, 41, 50, 55)
#define HOBFLOPS_X16(B) B B B B B B B B B B B B B B B B
#define HOBFLOPS_X128(B) \
  HOBFLOPS_X16(B) HOBFLOPS_X16(B) HOBFLOPS_X16(B) HOBFLOPS_X16(B) \
  HOBFLOPS_X16(B) HOBFLOPS_X16(B) HOBFLOPS_X16(B) HOBFLOPS_X16(B)
#define HOBFLOPS_CLOBBER                                                            \
  "v32", "v33", "v34", "v35", "v36", "v37", "v38", "v39", "v40", "v41", "v42", "v43", \
      "v44", "v45", "v46", "v47", "v48", "v49", "v50", "v51", "v52", "v53", "v54",    \
      "v55", "v56", "v57", "v58", "v59", "v60", "v61", "v62", "v63"

// Instruction streams the probe can run.
enum ProbeKind {
  kFree = 0,     // 8-byte v_bitop3_b32, sources in three banks
  kShared = 1,   // 8-byte, two sources of every instruction in one bank
  kVop2 = 2,     // 4-byte v_xor_b32, sources in two banks
  kLong = 3,     // as kFree, 1024 instructions per loop iteration instead of 128
  kChain = 4,    // as kFree, each instruction depending on the one before
  kMixed = 5,    // 8-byte and 4-byte instructions alternating
  kDist2 = 6,    // as kFree, each instruction depending on the one two before
  kDist4 = 7,    // as kFree, each instruction depending on the one four before
  kAligned = 8,  // as kFree with every 8-byte instruction at an address 0 mod 8
  kHalf = 9,     // groups of one 4-byte and seven 8-byte instructions
  kNop = 10,     // as kHalf plus an s_nop 0 after each group (all aligned)
  kNumKinds = 11
};

__host__ __device__ constexpr int instr_per_iter(int kind) { return kind == kLong ? 1024 : 128; }

// Each wave writes (start, end) shader clocks and (start, end) 100 MHz clocks.
template <int kKind>
__global__ void issue_probe_kernel(uint64_t* __restrict__ stamps, uint32_t* __restrict__ sink,
                                   int iters) {
  const uint32_t seed = threadIdx.x;
  asm volatile(
      "v_mov_b32 v32, %0\n v_mov_b32 v33, %0\n v_mov_b32 v34, %0\n v_mov_b32 v35, %0\n"
      "v_mov_b32 v36, %0\n v_mov_b32 v37, %0\n v_mov_b32 v38, %0\n v_mov_b32 v39, %0\n"
      "v_mov_b32 v40, %0\n v_mov_b32 v41, %0\n v_mov_b32 v42, %0\n v_mov_b32 v43, %0\n"
      "v_mov_b32 v44, %0\n v_mov_b32 v45, %0\n v_mov_b32 v46, %0\n v_mov_b32 v47, %0\n"
      "v_mov_b32 v48, %0\n v_mov_b32 v49, %0\n v_mov_b32 v50, %0\n v_mov_b32 v51, %0\n"
      "v_mov_b32 v52, %0\n v_mov_b32 v53, %0\n v_mov_b32 v54, %0\n v_mov_b32 v55, %0\n"
      "v_mov_b32 v56, %0\n v_mov_b32 v57, %0\n v_mov_b32 v58, %0\n v_mov_b32 v59, %0\n"
      "v_mov_b32 v60, %0\n v_mov_b32 v61, %0\n v_mov_b32 v62, %0\n v_mov_b32 v63, %0\n" ::"v"(seed)
      : HOBFLOPS_CLOBBER);
  const uint64_t t0 = __builtin_amdgcn_s_memtime(), r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < iters; ++it) {
    if constexpr (kKind == kFree)
      asm volatile(HOBFLOPS_X16(HOBFLOPS_BLOCK_FREE)::: HOBFLOPS_CLOBBER);
    else if constexpr (kKind == kShared)
      asm volatile(HOBFLOPS_X16(HOBFLOPS_BLOCK_SHARED)::: HOBFLOPS_CLOBBER);
    else if constexpr (kKind == kVop2)
      asm volatile(HOBFLOPS_X16(HOBFLOPS_BLOCK_VOP2)::: HOBFLOPS_CLOBBER);
    else if constexpr (kKind == kLong)
      asm volatile(HOBFLOPS_X128(HOBFLOPS_BLOCK_FREE)::: HOBFLOPS_CLOBBER);
    else if constexpr (kKind == kChain)
      asm volatile(HOBFLOPS_X16(HOBFLOPS_BLOCK_CHAIN)::: HOBFLOPS_CLOBBER);
    else if constexpr (kKind == kMixed)
      asm volatile(HOBFLOPS_X16(HOBFLOPS_BLOCK_MIXED)::: HOBFLOPS_CLOBBER);
    else if constexpr (kKind == kDist2)
      asm volatile(HOBFLOPS_X16(HOBFLOPS_BLOCK_DIST2)::: HOBFLOPS_CLOBBER);
    else if constexpr (kKind == kDist4)
      asm volatile(HOBFLOPS_X16(HOBFLOPS_BLOCK_DIST4)::: HOBFLOPS_CLOBBER);
    else if constexpr (kKind == kAligned)  // the loop's own instructions take 12 bytes
      asm volatile("s_nop 0\n" HOBFLOPS_X16(HOBFLOPS_BLOCK_FREE)::: HOBFLOPS_CLOBBER);
    else if constexpr (kKind == kHalf)
      asm volatile(HOBFLOPS_X16(HOBFLOPS_BLOCK_HALF)::: HOBFLOPS_CLOBBER);
    else
      asm volatile(HOBFLOPS_X16(HOBFLOPS_BLOCK_NOP)::: HOBFLOPS_CLOBBER);
  }
  const uint64_t t1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
  uint32_t x;
  asm volatile("v_mov_b32 %0, v40" : "=v"(x));
  const int wave = blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6);
  if ((threadIdx.x & 63) == 0) {
    stamps[4 * wave + 0] = t0;
    stamps[4 * wave + 1] = t1;
    stamps[4 * wave + 2] = r0;
    stamps[4 * wave + 3] = r1;
  }
  sink[blockIdx.x * blockDim.x + threadIdx.x] = x;
}

template <int kKind>
void launch_probe(int kind, int blocks, int waves, uint64_t* stamps, uint32_t* sink, int iters) {
  if constexpr (kKind < kNumKinds) {
    if (kind == kKind)
      hipLaunchKernelGGL(issue_probe_kernel<kKind>, dim3(blocks), dim3(64 * waves), 0, 0, stamps,
                         sink, iters);
    else
      launch_probe<kKind + 1>(kind, blocks, waves, stamps, sink, iters);
  }
}

}  // namespace

extern "C" {

// Runs one probe launch on the current device: `blocks` workgroups (one per
// CU when blocks equals the CU count) of `waves` waves each (1..16), every
// wave issuing iters x 128 instructions of the stream `kind`:
//   0  8-byte v_bitop3_b32, the three sources of every instruction in
//      distinct VGPR banks (register number mod 4), results never read
//   1  the same with two sources of every instruction in one bank
//   2  4-byte v_xor_b32 (VOP2 encoding), sources in distinct banks
//   3  as 0 with 1024 instructions between loop branches instead of 128
//   4  as 0, each instruction reading the result of the one before
//   5  8-byte and 4-byte instructions alternating
//   6  as 0, each instruction reading the result of the one two before
//   7  as 0, each instruction reading the result of the one four before
//   8  as 0 with every instruction at an address 0 mod 8 (one s_nop 0 ahead
//      of each 128)
//   9  groups of one 4-byte and seven 8-byte instructions, so that every
//      other group's 8-byte instructions sit at addresses 4 mod 8
//  10  as 9 with an s_nop 0 closing each group: all aligned, one more
//      instruction per group
// Results (averages over the waves):
//   *clk_per_instr  shader clocks per instruction of one wave
//   *simd_interval  shader clocks per instruction of one SIMD: the span of a
//                   workgroup's waves over the instructions each SIMD issued
//                   (waves are spread over a CU's four SIMDs)
//   *ghz            shader clock during the launch (s_memtime over
//                   s_memrealtime at 100 MHz)
// Allocates and frees its own buffers; synchronises the device. Returns 0,
// -1 (bad argument) or the HIP error code.
int hobflops_probe_issue(int blocks, int waves, int kind, int iters, double* clk_per_instr,
                         double* simd_interval, double* ghz) {
  if (blocks < 1 || waves < 1 || waves > 16 || iters < 1 || kind < 0 || kind >= kNumKinds ||
      !clk_per_instr || !simd_interval || !ghz)
    return -1;
  // the same number of instructions for every kind
  const int loops = kind == kLong ? (iters + 7) / 8 : iters;
  const size_t nw = (size_t)blocks * waves;
  uint64_t* stamps = nullptr;
  uint32_t* sink = nullptr;
  hipError_t e = hipMalloc(&stamps, nw * 4 * sizeof(uint64_t));
  if (e == hipSuccess) e = hipMalloc(&sink, nw * 64 * sizeof(uint32_t));
  if (e == hipSuccess) {
    for (int rep = 0; rep < 2 && e == hipSuccess; ++rep) {  // the first launch warms up
      launch_probe<0>(kind, blocks, waves, stamps, sink, loops);
      e = hipGetLastError();
      if (e == hipSuccess) e = hipDeviceSynchronize();
    }
  }
  uint64_t* h = nullptr;
  if (e == hipSuccess) {
    h = new uint64_t[nw * 4];
    e = hipMemcpy(h, stamps, nw * 4 * sizeof(uint64_t), hipMemcpyDeviceToHost);
  }
  if (e == hipSuccess) {
    const double n = (double)loops * instr_per_iter(kind);
    double per_wave = 0.0, span = 0.0, clk = 0.0;
    for (int b = 0; b < blocks; ++b) {
      uint64_t lo = ~0ull, hi = 0;
      for (int w = 0; w < waves; ++w) {
        const uint64_t* s = h + 4 * ((size_t)b * waves + w);
        per_wave += (double)(s[1] - s[0]);
        clk += (double)(s[1] - s[0]) / ((double)(s[3] - s[2]) / 100e6);
        lo = s[0] < lo ? s[0] : lo;
        hi = s[1] > hi ? s[1] : hi;
      }
      span += (double)(hi - lo);
    }
    const int per_simd = (waves + 3) / 4;
    *clk_per_instr = per_wave / (double)nw / n;
    *simd_interval = span / blocks / (n * per_simd);
    *ghz = clk / (double)nw / 1e9;
  }
  delete[] h;
  if (stamps) (void)hipFree(stamps);
  if (sink) (void)hipFree(sink);
  return e == hipSuccess ? 0 : (int)e;
}

}  // extern "C"
