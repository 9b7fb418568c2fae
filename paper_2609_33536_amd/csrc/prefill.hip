// Chunked-prefill attention over a mixed-fidelity prefix (paper §3.2).
#include "common.h"
#include "launch.h"

namespace ekv {

hipError_t launch_prefill(const PrefillArgs&, int, int, bool, hipStream_t) { return hipErrorNotSupported; }

}  // namespace ekv
