// Table of the generated kernel variants (filled in by the generated
// registry.inc: one entry per format combination the build produced).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.hpp"

namespace hobflops {

typedef hipError_t (*conv_launch_fn)(const uint32_t* ifm, const uint32_t* w, uint32_t* ofm,
                                     const ConvParams& p, int algo, hipStream_t stream);
typedef hipError_t (*muladd_launch_fn)(const uint32_t* a, const uint32_t* b, const uint32_t* c,
                                       uint32_t* r, int64_t groups, hipStream_t stream);

struct ConvVariant {
  int wE, wF_in, wF_acc, wF_out, act;
  int round;      // HOBFLOPS_ROUND_*
  int has_split;  // the split kernel was generated (its netlists fit the registers)
  int has_compact;  // ... and its compact form (two workgroups per CU)
  int mac_ops;    // VALU bitwise instructions of one fused multiply-add step
  int mul_ops;    // ... of the multiplier alone (split kernel, multiplier waves)
  int accum_ops;  // ... of the accumulating adder alone (split kernel, adder waves)
  conv_launch_fn launch;
};

struct MuladdVariant {
  int wE, wF_in, wF_acc;
  int round;  // HOBFLOPS_ROUND_*
  int ops;  // VALU bitwise instructions of one element-wise MAC
  muladd_launch_fn launch;
};

typedef hipError_t (*pool_launch_fn)(const uint32_t* in, uint32_t* out, const PoolParams& p,
                                     hipStream_t stream);

struct PoolVariant {
  int wE, wF_in, wF_acc, wF_out;
  int round;       // HOBFLOPS_ROUND_*
  int accum_ops;   // VALU bitwise instructions of one accumulating add
  int scale_ops;   // ... of the final multiply by the scale
  pool_launch_fn launch;
};

extern const ConvVariant kConvVariants[];
extern const int kNumConvVariants;
extern const MuladdVariant kMuladdVariants[];
extern const int kNumMuladdVariants;
extern const PoolVariant kPoolVariants[];
extern const int kNumPoolVariants;

}  // namespace hobflops
