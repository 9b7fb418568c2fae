// Stand-ins for the kernel launchers (launch.h) in the host-only sanitizer
// build: the driver exercises the host code of api.hip and control.hip, and
// nothing reaches a launcher there except through paths that need a device.
#include <hip/hip_runtime_api.h>

#include "launch.h"

namespace ekv {
hipError_t launch_decode(const DecodeArgs&, int, int, bool, hipStream_t) { return hipErrorNoDevice; }
hipError_t decode_grid(const DecodeArgs&, int, int, bool, int*) { return hipErrorNoDevice; }
hipError_t launch_zero_u32(uint32_t*, size_t, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_demote(const TransitionArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_refine(const TransitionArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_stage(const StageArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_append(const AppendArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_prefill(const PrefillArgs&, int, int, bool, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_validate_batch(const ValidateBatchArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_validate_list(const ValidateListArgs&, hipStream_t) { return hipErrorNoDevice; }
}  // namespace ekv
