// Host-only stand-ins for the kernel launchers of sdnn_kernels.hip, linked instead of it
// into the sanitizer build of the host code (a CPU build of sdnn_host.cpp under
// AddressSanitizer and UndefinedBehaviorSanitizer).  That build serves the host-only
// entry points (CSR validation, row orders, packing and its self-check); every call that
// would launch a kernel fails with hipErrorNotSupported, so it surfaces as SDNN_ERR_HIP.
#include <hip/hip_runtime.h>

#include "sdnn_internal.h"

namespace sdnn {

hipError_t launch_spmm(const sdnn_plan_s*, const float*, float*, int32_t, const float*, int,
                       hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_conv3x3(const sdnn_plan_s*, const float*, float*, int32_t, int32_t, int32_t,
                          const float*, int, hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_spmm_split(const sdnn_plan_s*, const float*, float*, int32_t, const float*, int,
                             int, float*, hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_conv3x3_split(const sdnn_plan_s*, const float*, float*, int32_t, int32_t,
                                int32_t, const float*, int, int, float*, hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t tune_spmm(sdnn_plan_s*, const float*, float*, int32_t, hipStream_t, TunedShape*) {
  return hipErrorNotSupported;
}
hipError_t launch_dense(const float*, const float*, float*, int32_t, int32_t, int32_t,
                        const float*, int, hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t scratch_address(int, float**) { return hipErrorNotSupported; }
int split_runs(const sdnn_plan_s*, int32_t, int32_t) { return 1; }
void launch_shape(const sdnn_plan_s* p, int32_t, int32_t* panel_rows, int32_t* waves,
                  int32_t* tile_cols) {
  *panel_rows = p->pk[0].RW;
  *waves = 1;
  *tile_cols = kTileCols;
}

}  // namespace sdnn
