// Kernel launchers of the sanitizer build: no device, so each one reports hipErrorNotSupported.
#include "psattn_launch.h"

namespace psattn {
hipError_t launch_fwd_main(const FwdArgs&, bool, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_fwd_merge(const FwdArgs&, bool, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_bwd_pre(const BwdArgs&, bool, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_bwd_kv(const BwdArgs&, bool, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_bwd_dq(const BwdArgs&, bool, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_bwd_reduce_kv(const BwdArgs&, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_bwd_reduce_dq(const BwdArgs&, bool, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_bwd_zero_pad(const BwdArgs&, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_rope(const PlanView&, int32_t, int32_t, int32_t, float, bool, bool, void*, hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_kv_move(const PlanView&, int32_t, int32_t, bool, const void*, const void*, void*, void*, hipStream_t) {
  return hipErrorNotSupported;
}
}  // namespace psattn
