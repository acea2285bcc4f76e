// Kernel launchers for the host-only build of libsra used by the sanitizer run (built by
// `build.py --sanitize`, never shipped): the scheduler and the C ABI are compiled with
// AddressSanitizer and UndefinedBehaviorSanitizer for the CPU, and every launch reports
// hipErrorNotSupported, so a call that gets past validation fails with SRA_ERR_HIP.
#include "sra_kernels.h"

namespace sra {

hipError_t launch_forward(const FwdArgs&, int, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_delta(const DeltaArgs&, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_dq(const BwdArgs&, int, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_dkv(const BwdArgs&, int, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_fill(const FillArgs&, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_gather(const GatherArgs&, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_scatter(const ScatterArgs&, hipStream_t) { return hipErrorNotSupported; }

}  // namespace sra
