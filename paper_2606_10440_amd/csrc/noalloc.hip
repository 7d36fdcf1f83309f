// Allocation-free run of libsimgpu: sim_run for callers that cannot allocate
// device memory (code under HIP graph capture, tight serving loops, harnesses
// that forbid hipMalloc).  The engines' per-run scratch -- per-scenario
// statuses and processed-cycle counts, and the FIFO rings, per-link scalars
// and request records of the engines that keep them in device memory -- is
// taken from a fixed device array of SIM_NOALLOC_SCRATCH_BYTES instead of the
// context's own block.  The kernels initialise everything they read there,
// so nothing has to be cleared between calls.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/simgpu.h"

namespace simgpu {
sim_status run_on_scratch(sim_ctx *c, void *stream, uint32_t *d_completion, uint64_t *d_tx_lines,
                          uint64_t *d_busy_cycles, uint32_t *d_makespan, uint64_t max_cycles, void *scratch,
                          size_t scratch_bytes);
}

namespace {

// One copy per GPU, held until the process ends.  Its name is only a host
// stand-in: host code uses the device address looked up below.
static __device__ __align__(256) unsigned char scratch[SIM_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_scratch[kMaxDevices];  // device address of scratch on each device, once looked up

}  // namespace

extern "C" sim_status sim_run_noalloc(sim_ctx *ctx, void *hip_stream, uint32_t *d_completion, uint64_t *d_tx_lines,
                                      uint64_t *d_busy_cycles, uint32_t *d_makespan, uint64_t max_cycles) {
    if (!ctx) return SIM_ERR_INVALID_ARG;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return SIM_ERR_DEVICE;
    void *ptr = nullptr;
    {
        std::lock_guard<std::mutex> lock(g_mu);
        if (!g_scratch[dev]) {  // first call on this device, which is current
            void *p = nullptr;
            if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SIM_ERR_DEVICE;
            g_scratch[dev] = p;
        }
        ptr = g_scratch[dev];
    }
    return simgpu::run_on_scratch(ctx, hip_stream, d_completion, d_tx_lines, d_busy_cycles, d_makespan, max_cycles,
                                  ptr, (size_t)SIM_NOALLOC_SCRATCH_BYTES);
}
