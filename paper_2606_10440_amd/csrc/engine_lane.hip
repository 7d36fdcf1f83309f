// ----------------------------------------------------------------------------
// Lane engine.  One workgroup per scenario; lane i owns traffic link i: its
// FIFO ring (LDS, 16-byte entries {line, ready, path index, -}), its head,
// tail, round-robin pointer and counters (registers), the injection stream
// whose first hop is that link (registers), and the arbitration for lines
// entering it.  Cross-lane traffic goes through small LDS mailboxes:
//   requests  a source posts {line, path index, source<<8 | k, port} into
//             the target lane's slots (slot count by LDS atomic);
//   grants    the target writes the grant rank into the source's slot;
//   departs   the source marks granted lines of its longest granted prefix;
//   enter     the target appends the marked lines in grant order.
// Phase boundaries wait on LDS only (s_waitcnt lgkmcnt(0)); completion
// stores to HBM are never waited on.

#include <hip/hip_runtime.h>

#include "engine_common.h"

namespace simgpu {

namespace {

using namespace dev;


// HBMFIFO: the FIFO rings live in HBM instead of LDS (a ring is only ever
// touched by its own lane, so no extra ordering is needed).
template <int BM, bool ONEWAVE, int ARB, bool HBMFIFO>
__global__ void __launch_bounds__(1024) engine_lane(DevNet d) {
    extern __shared__ __align__(16) unsigned char smem[];
    // requests per target ranked in registers (more: ranked from LDS); none
    // for wide links, whose request records already fill the registers
    constexpr int kRankRegs = BM <= 4 ? 8 : 0;
    uint4 *fifo = HBMFIFO ? d.gfifo + (size_t)blockIdx.x * d.fifo_total : reinterpret_cast<uint4 *>(smem);
    int32_t *lpath = reinterpret_cast<int32_t *>(smem + d.o_path);
    uint32_t *deliv = reinterpret_cast<uint32_t *>(smem + d.o_deliv);
    uint32_t *req_cnt = reinterpret_cast<uint32_t *>(smem + d.o_reqcnt);
    uint32_t *reqb = reinterpret_cast<uint32_t *>(smem + d.o_reqb);      // [2*nl]: base, count

    uint4 *req = reinterpret_cast<uint4 *>(smem + d.o_req);
    uint32_t *glist = reinterpret_cast<uint32_t *>(smem + d.o_glist);
    int32_t *grant = reinterpret_cast<int32_t *>(smem + d.o_grant);
    uint32_t *gdep = reinterpret_cast<uint32_t *>(smem + d.o_gdep);
    uint32_t *red = reinterpret_cast<uint32_t *>(smem + d.o_red);

    const int s = blockIdx.x;
    const int i = threadIdx.x;
    const int nthr = blockDim.x;
    const int nl = d.nl;
    const int m = d.m;
    const bool on = i < nl;

    if (d.path_in_lds)
        for (int j = i; j < d.path_len; j += nthr) lpath[j] = d.path_lane[j];
    const int32_t *path = d.path_in_lds ? lpath : d.path_lane;
    for (int j = i; j < d.nflows; j += nthr) deliv[j] = 0;
    for (int j = i; j < nl; j += nthr) {
        req_cnt[j] = 0;
        reqb[2 * j] = (uint32_t)d.ln_req[j];
        reqb[2 * j + 1] = (uint32_t)d.ln_reqcap[j];
    }
    for (int j = i; j < 2 * nl * BM; j += nthr) grant[j] = -1;
    for (int j = i; j < nl * BM; j += nthr) gdep[j] = 0;
    if (i < 16) red[i] = kNever;
    // links without traffic report zero counters
    for (int j = i; j < m; j += nthr)
        if (d.link_lane[j] < 0) {
            d.tx_lines[(size_t)s * m + j] = 0;
            d.busy[(size_t)s * m + j] = 0;
        }

    // lane registers
    int link = 0, b = 0, L = 0, cap = 0, fbase = 0, fmask = 0, rbase = 0, rcap = 0;
    uint32_t P = 1, myport = 0;
    uint32_t head = 0, tail = 0, rr = 0;
    uint64_t tx = 0, busy = 0;
    int R = 0, rend = 0;
    uint32_t o = 0;
    RangeReg<kPredCache> cur{};
    if (on) {
        link = d.ln_link[i];
        const size_t pi = (size_t)s * m + link;
        b = d.bw[pi];
        L = d.lat[pi];
        cap = d.cap[pi];
        P = (uint32_t)d.ln_P[i];
        myport = (uint32_t)d.ln_port[i];
        fbase = d.ln_fifo[i];
        fmask = d.ln_mask[i];
        rbase = d.ln_req[i];
        rcap = d.ln_reqcap[i];
        R = d.ln_srbeg[i];
        rend = d.ln_srend[i];
        if (R < rend) load_range(d, R, cur);
    }
    lds_fence_block();

    uint32_t *comp = d.completion + (size_t)s * d.T;
    uint32_t t = 0;
    uint64_t processed = 0;
    int32_t state = d.T > 0 ? kRunRunning : kRunOk;
    bool overflow = false;
    // a request's arbitration key at this target: its line id, or its
    // round-robin rank (k, port offset from the pointer); ports are < P
    auto req_key = [&](const uint4 &r) -> uint32_t {
        if (ARB == 0) return r.x;
        const uint32_t off = r.w + P - rr;
        return (r.z & 255u) * P + (off >= P ? off - P : off);
    };

    // The first FIFO entries a lane may offer are read at the end of the
    // previous cycle, after its pops and appends, so that their load (from
    // HBM with HBMFIFO) overlaps the time phase instead of opening the next
    // cycle; for narrow links only, whose entries fit the registers.
    constexpr int kPre = BM <= 4 ? BM : 0;
    uint4 pre[kPre > 0 ? kPre : 1];
    auto prefetch = [&]() {
#pragma unroll
        for (int k = 0; k < kPre; k++)
            if (on && k < b && (uint32_t)k < tail - head) pre[k] = fifo[fbase + ((head + k) & fmask)];
    };

    while (state == kRunRunning) {
        // -------------------------------------------------------------- R
        int nf = 0, nsr = 0;
        int32_t ftg[BM];
        uint32_t fxv[BM];
        uint32_t next = kNever;
        if (on) {
            const uint32_t occ = tail - head;
#pragma unroll
            for (int k = 0; k < BM; k++) {
                ftg[k] = 0;
                fxv[k] = 0;
                if (k < b && (uint32_t)k < occ && nf == k) {
                    const uint4 e = kPre > 0 ? pre[k < kPre ? k : 0] : fifo[fbase + ((head + k) & fmask)];
                    if (e.y > t) {
                        next = e.y;
                    } else {
                        const int pp = (int)e.z + 1;
                        const int tg = path[pp];
                        ftg[k] = tg;
                        fxv[k] = e.x;
                        if (tg >= 0) {
                            const uint32_t slot = atomicAdd(&req_cnt[tg], 1u);
                            if (slot < reqb[2 * tg + 1])
                                req[reqb[2 * tg] + slot] =
                                    make_uint4(e.x, (uint32_t)pp, ((uint32_t)(2 * i) << 8) | k, myport);
                            else
                                overflow = true;
                        }
                        nf++;
                    }
                }
            }
            int sR = R;
            uint32_t so = o;
            RangeReg<kPredCache> sr = cur;
#pragma unroll
            for (int k = 0; k < BM; k++) {
                if (k < b && sR < rend && nsr == k) {
                    if (released(d, sr, so, deliv)) {
                        const uint32_t slot = atomicAdd(&req_cnt[i], 1u);
                        if (slot < (uint32_t)rcap)
                            req[rbase + slot] =
                                make_uint4(sr.start + so, (uint32_t)sr.path, ((uint32_t)(2 * i + 1) << 8) | k, P - 1);
                        else
                            overflow = true;
                        nsr++;
                        if (++so == sr.len) {
                            sR++;
                            so = 0;
                            if (sR < rend && k + 1 < b) load_range(d, sR, sr);
                        }
                    }
                }
            }
        }
        phase_sync<ONEWAVE>();
        // -------------------------------------------------------------- G
        int g = 0;
        uint32_t creq = 0;  // this target's request count
        if (on) {
            const uint32_t c = req_cnt[i];
            creq = c;
            if (c) {
                req_cnt[i] = 0;
                if (c > (uint32_t)rcap) overflow = true;
                g = cap - (int)(tail - head);
                if (b < g) g = b;
                if ((int)c < g) g = (int)c;
                if (g > 0 && !overflow && c > (uint32_t)kRankRegs) {
                    // many requests: rank each against all, reading them from LDS
                    for (uint32_t a = 0; a < c; a++) {
                        const uint4 ra = req[rbase + a];
                        const uint32_t ka = req_key(ra);
                        int rank = 0;
                        for (uint32_t q = 0; q < c; q++) rank += req_key(req[rbase + q]) < ka ? 1 : 0;
                        if (rank < g) {
                            grant[(ra.z >> 8) * BM + (ra.z & 255u)] = rank;
                            glist[i * BM + rank] = (uint32_t)rbase + a;
                        }
                    }
                }
                if (g < 0) g = 0;
            }
        }
        if constexpr (kRankRegs > 0) {
            // Up to kRankRegs requests per target: their keys are read once,
            // all together, and ranked in registers; the loops run to the
            // wave's largest request count (wave-uniform bounds, so the
            // register arrays are indexed at compile time).
            const uint32_t cq = (on && g > 0 && !overflow && creq <= (uint32_t)kRankRegs) ? creq : 0u;
            uint32_t cmax = cq;
#pragma unroll
            for (int sh = 32; sh >= 1; sh >>= 1) cmax = max(cmax, (uint32_t)__shfl_xor((int)cmax, sh));
            if (cmax > 0u) {
                uint32_t key[kRankRegs], rz[kRankRegs];
#pragma unroll
                for (int q = 0; q < kRankRegs; q++) {
                    key[q] = 0xFFFFFFFFu;
                    rz[q] = 0u;
                    if ((uint32_t)q < cmax) {
                        const uint4 rq = req[rbase + ((uint32_t)q < cq ? q : 0)];
                        key[q] = (uint32_t)q < cq ? req_key(rq) : 0xFFFFFFFFu;
                        rz[q] = rq.z;
                    }
                }
#pragma unroll
                for (int a = 0; a < kRankRegs; a++) {
                    if ((uint32_t)a < cmax) {
                        int rank = 0;
#pragma unroll
                        for (int q = 0; q < kRankRegs; q++)
                            if ((uint32_t)q < cmax) rank += key[q] < key[a] ? 1 : 0;
                        if (((uint32_t)a < cq) & (rank < g)) {
                            grant[(rz[a] >> 8) * BM + (rz[a] & 255u)] = rank;
                            glist[i * BM + rank] = (uint32_t)rbase + (uint32_t)a;
                        }
                    }
                }
            }
        }
        phase_sync<ONEWAVE>();
        // -------------------------------------------------------------- D
        int dep = 0;
        if (on) {
            bool open = true;
            int depf = 0;
#pragma unroll
            for (int k = 0; k < BM; k++) {
                if (k < nf) {
                    int gr = -2;
                    if (ftg[k] >= 0) {
                        gr = grant[(2 * i) * BM + k];
                        grant[(2 * i) * BM + k] = -1;
                    }
                    if (open && gr != -1) {
                        depf++;
                        if (gr == -2) {
                            comp[fxv[k]] = t + 1;
                            deliv[-ftg[k] - 1] += 1u;
                        } else {
                            gdep[ftg[k] * BM + gr] = 1u;
                        }
                    } else {
                        open = false;
                    }
                }
            }
            head += (uint32_t)depf;
            open = true;
            int deps = 0;
#pragma unroll
            for (int k = 0; k < BM; k++) {
                if (k < nsr) {
                    const int gr = grant[(2 * i + 1) * BM + k];
                    grant[(2 * i + 1) * BM + k] = -1;
                    if (open && gr != -1) {
                        deps++;
                        gdep[i * BM + gr] = 1u;
                    } else {
                        open = false;
                    }
                }
            }
            if (deps) {
                o += (uint32_t)deps;
                while (R < rend && o >= cur.len) {
                    o -= cur.len;
                    R++;
                    if (R < rend) load_range(d, R, cur);
                }
            }
            dep = depf + deps;
        }
        phase_sync<ONEWAVE>();
        // -------------------------------------------------------------- E
        if (on && g > 0) {
            int cnt = 0;
            uint32_t last_port = 0;
            const uint32_t ready = t + (uint32_t)L;
#pragma unroll
            for (int r = 0; r < BM; r++) {
                if (r < g && gdep[i * BM + r]) {
                    gdep[i * BM + r] = 0u;
                    const uint4 rq = req[glist[i * BM + r]];
                    fifo[fbase + (tail & fmask)] = make_uint4(rq.x, ready, rq.y, 0u);
                    tail++;
                    cnt++;
                    last_port = rq.w;
                }
            }
            if (cnt) {
                tx += (uint64_t)cnt;
                busy += 1;
                if (ARB == 1) rr = last_port + 1u == P ? 0u : last_port + 1u;
            }
        }
        // -------------------------------------------------------------- time
        processed++;
        const bool act = on && (tail != head || R < rend);
        bool any_dep, any_act, any_over;
        uint32_t nxt;
        if (ONEWAVE) {
            any_dep = __ballot(dep > 0) != 0;
            any_act = __ballot(act) != 0;
            any_over = __ballot(overflow) != 0;
            nxt = next;
            if (!any_dep) {
#pragma unroll
                for (int sh = 32; sh >= 1; sh >>= 1) {
                    const uint32_t v = (uint32_t)__shfl_xor((int)nxt, sh);
                    nxt = v < nxt ? v : nxt;
                }
            }
        } else {
            // red[4p+0] departures, [4p+1] active, [4p+2] min next, [4p+3] overflow;
            // p alternates so a slot is reset one cycle before it is reused
            const int p = (int)(processed & 1u) * 4;
            const bool wdep = __ballot(dep > 0) != 0, wact = __ballot(act) != 0, wover = __ballot(overflow) != 0;
            if ((i & 63) == 0) {
                if (wdep) red[p] = 1u;
                if (wact) red[p + 1] = 1u;
                if (wover) red[p + 3] = 1u;
            }
            lds_fence_block();
            any_dep = red[p] != kNever;
            any_act = red[p + 1] != kNever;
            any_over = red[p + 3] != kNever;
            nxt = kNever;
            if (!any_dep && any_act && !any_over) {  // only an idle cycle needs the next event time
                uint32_t v = next;
#pragma unroll
                for (int sh = 32; sh >= 1; sh >>= 1) {
                    const uint32_t u = (uint32_t)__shfl_xor((int)v, sh);
                    v = u < v ? u : v;
                }
                if ((i & 63) == 0 && v != kNever) atomicMin(&red[p + 2], v);
                lds_fence_block();
                nxt = red[p + 2];
            }
            const int q = 4 - p;
            if (i < 4) red[q + i] = kNever;
        }
        if (any_over) {
            state = kRunInternal;
        } else if (!any_act) {
            state = kRunOk;
        } else if (any_dep) {
            t = t + 1;
        } else if (nxt == kNever) {
            state = kRunDeadlock;
        } else {
            t = nxt;
        }
        if (state == kRunRunning && (uint64_t)t > d.max_cycles) state = kRunMaxCycles;
        if (state == kRunRunning && processed > d.watchdog) state = kRunWatchdog;
        if (!ONEWAVE) lds_fence_block();
        if constexpr (kPre > 0) prefetch();
    }
    if (on) {
        d.tx_lines[(size_t)s * m + link] = tx;
        d.busy[(size_t)s * m + link] = busy;
    }
    if (i == 0) {
        d.makespan[s] = d.T > 0 ? t + 1 : 0;
        d.status[s] = state;
        d.cycles[s] = processed;
    }
}

template <int BM, bool ONEWAVE, int ARB>
hipError_t launch_lane3(const DevNet &d, hipStream_t st) {
    auto k = d.engine == kEngineLaneHbm ? engine_lane<BM, ONEWAVE, ARB, true> : engine_lane<BM, ONEWAVE, ARB, false>;
    if (d.lds_bytes > 65536)
        (void)hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize, d.lds_bytes);
    hipLaunchKernelGGL(k, dim3((unsigned)d.S), dim3(d.lane_threads), (unsigned)d.lds_bytes, st, d);
    return hipGetLastError();
}

template <int BM>
hipError_t launch_lane(const DevNet &d, hipStream_t st) {
    const bool one = d.lane_threads == 64;
    if (d.arb == 0) return one ? launch_lane3<BM, true, 0>(d, st) : launch_lane3<BM, false, 0>(d, st);
    return one ? launch_lane3<BM, true, 1>(d, st) : launch_lane3<BM, false, 1>(d, st);
}

}  // namespace

hipError_t launch_lane_any(const DevNet &d, hipStream_t st) {
    switch (d.bm) {
    case 1: return launch_lane<1>(d, st);
    case 2: return launch_lane<2>(d, st);
    case 4: return launch_lane<4>(d, st);
    case 8: return launch_lane<8>(d, st);
    case 16: return launch_lane<16>(d, st);
    case 32: return launch_lane<32>(d, st);
    default: return launch_lane<64>(d, st);
    }
}

}  // namespace simgpu
