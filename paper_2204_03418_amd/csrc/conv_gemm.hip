// Implicit-GEMM continual convolution step on MFMA (groups = 1).
#include "device.hpp"
#include "launch.hpp"

namespace coinf {

hipError_t launch_conv_step_gemm(const ConvGeom&, const ConvLayout&, char*, const StepIO&,
                                 const co_step_plan&, hipStream_t) {
  return hipErrorNotSupported;
}

hipError_t launch_pack_gemm(const ConvGeom&, const ConvLayout&, char*, const void*,
                            hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace coinf
