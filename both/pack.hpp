// Launchers of the pack / unpack kernels (pack.hip).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hobflops {
hipError_t launch_pack(const void* src, int kind, int64_t rows, int64_t len, int wE, int wF,
                       uint32_t* planes, hipStream_t stream);
hipError_t launch_unpack(const uint32_t* planes, int64_t rows, int64_t len, int wE, int wF,
                         int kind, void* dst, hipStream_t stream);
}  // namespace hobflops
