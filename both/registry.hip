#include "registry.hpp"
#ifndef __HIP_DEVICE_COMPILE__
namespace hobflops {
hipError_t launch_conv_e5m3_a4_o4(const uint32_t*, const uint32_t*, uint32_t*, const ConvParams&, int, hipStream_t);
const ConvVariant kConvVariants[] = {{5, 3, 4, 4, 0, 236, 78, 156, launch_conv_e5m3_a4_o4}};
const int kNumConvVariants = 1;
const MuladdVariant kMuladdVariants[] = {{5, 3, 4, 241, nullptr}};
const int kNumMuladdVariants = 0;
}
#endif
