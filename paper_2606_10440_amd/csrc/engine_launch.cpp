// Engine dispatch of libsimgpu: one launch per sim_run on the caller's stream.
#include <hip/hip_runtime.h>

#include "sim_internal.h"

namespace simgpu {

int launch_engine(const DevNet &d, void *stream) {
    hipStream_t st = (hipStream_t)stream;
    switch (d.engine) {
    case kEngineB1: return (int)launch_b1_any(d, st);
    case kEngineWave: return (int)launch_wave_any(d, st);
    case kEngineGrid: return (int)launch_grid_any(d, st);
    case kEngineResident: return (int)launch_resident(d, st);
    case kEngineLane:
    case kEngineLaneHbm: return (int)launch_lane_any(d, st);
    default: return (int)launch_workgroup(d, st);
    }
}

}  // namespace simgpu
