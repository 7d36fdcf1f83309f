// Host-only build of the library (test infrastructure): the engine launcher
// the host builder calls, with no device behind it.
#include <hip/hip_runtime.h>

#include "../../include/simgpu.h"
#include "../../paper_2606_10440_amd/csrc/sim_internal.h"

namespace simgpu {
int launch_engine(const DevNet &, void *) { return hipErrorNoDevice; }
}  // namespace simgpu

// The allocation-free run needs the device array of its own source file.
extern "C" sim_status sim_run_noalloc(sim_ctx *, void *, uint32_t *, uint64_t *, uint64_t *, uint32_t *, uint64_t) {
    return SIM_ERR_DEVICE;
}
