// Launchers of the pack / unpack kernels (pack.hip).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hobflops {
// one tensor of a batched pack (all of a batch in one format)
struct PackTensor {
  const void* src;
  int kind;
  int64_t rows, len;
  uint32_t* planes;
};
// packs count tensors in ceil(count / 8) launches or more (very large tensors
// are split over several ranges)
hipError_t launch_pack_batch(const PackTensor* t, int count, int wE, int wF, hipStream_t stream);
hipError_t launch_pack(const void* src, int kind, int64_t rows, int64_t len, int wE, int wF,
                       uint32_t* planes, hipStream_t stream);
hipError_t launch_unpack(const uint32_t* planes, int64_t rows, int64_t len, int wE, int wF,
                         int kind, void* dst, hipStream_t stream);
}  // namespace hobflops
