// Shared device helpers of libsimgpu's engines: LDS phase fences, the
// injection-stream range cache and the predecessor release test.
#pragma once
#include <hip/hip_runtime.h>

#include "sim_internal.h"

namespace simgpu {
namespace dev {

__device__ __forceinline__ void lds_fence_wave() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void lds_fence_block() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// A stream's current id range and its first PC predecessor descriptors.
template <int PC>
struct RangeReg {
    uint32_t start, len;
    int32_t path, pd0, pd1;
    int32_t pf[PC > 0 ? PC : 1];
    uint32_t pb[PC > 0 ? PC : 1];
};

template <int PC>
__device__ __forceinline__ void load_range(const DevNet &d, int R, RangeReg<PC> &r) {
    r.start = d.r_start[R];
    r.len = d.r_len[R];
    r.path = d.r_path[R];
    r.pd0 = d.r_pd[R];
    r.pd1 = d.r_pd[R + 1];
#pragma unroll
    for (int q = 0; q < PC; q++) {
        const int idx = r.pd0 + q;
        const bool in = idx < r.pd1;
        r.pf[q] = in ? d.pd_flow[idx] : 0;
        r.pb[q] = in ? d.pd_base[idx] : 0;
    }
}

// Line start+o of range r may be injected: every predecessor flow has
// delivered more than base+o lines, or more than base for per-chunk
// dependencies (values as of the start of the cycle).
template <int PC>
__device__ __forceinline__ bool released(const DevNet &d, const RangeReg<PC> &r, uint32_t o, const uint32_t *deliv) {
    bool ok = true;
    // the cached descriptors' counters are read together, without branches
    // (an absent descriptor has flow 0, a valid index, and is ignored)
#pragma unroll
    for (int q = 0; q < PC; q++) {
        const uint32_t v = deliv[r.pf[q]];
        ok = ok & ((r.pd0 + q >= r.pd1) | (v > r.pb[q] + (o & d.pd_omask)));
    }
    for (int idx = r.pd0 + PC; ok && idx < r.pd1; idx++)
        ok = deliv[d.pd_flow[idx]] > d.pd_base[idx] + (o & d.pd_omask);
    return ok;
}

template <bool ONEWAVE>
__device__ __forceinline__ void phase_sync() {
    if (ONEWAVE) lds_fence_wave();
    else lds_fence_block();
}

// ARB is a template parameter: the policy must not be a runtime branch inside
// the divergent ranking loops (an i1 derived from it there was materialised
// as a lane mask that lost bits of lanes leaving the loop early).

}  // namespace dev
}  // namespace simgpu
