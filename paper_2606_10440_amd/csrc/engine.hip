// Device engine of libsimgpu: advances every line of every scenario one
// processed cycle at a time.
//
// One workgroup owns one scenario and runs it to completion inside a single
// launch; the four phases of a cycle are separated by workgroup barriers:
//   R  sources (link FIFOs and injection streams) offer up to b lines and
//      post requests to their target links;
//   G  every target link ranks its requests and grants min(b, free, #req);
//   D  every source departs its longest granted prefix; lines leaving their
//      last hop complete (cycle + 1) and bump their flow's delivered count;
//   E  targets append the departing lines in grant order (ready = t + L).
// Then the next cycle is t + 1 if anything departed, otherwise the earliest
// FIFO-head ready time (no such time = deadlock).
//
// Predecessor release uses per-flow delivered counters: lines of one flow
// (same source, destination and hence path) are injected in id order and
// FIFOs never reorder, so a flow delivers its lines in id order and "line
// with flow sequence q has completed" is "delivered > q" at cycle start.
#include <hip/hip_runtime.h>

#include "sim_internal.h"

namespace simgpu {

namespace {

constexpr int kThreads = 256;

__global__ void __launch_bounds__(kThreads) engine_wg(DevNet d) {
    const int s = blockIdx.x;
    const int tid = threadIdx.x;
    const int m = d.m;
    const int bmax = d.bmax;
    const size_t sm = (size_t)s * m;
    const int32_t *__restrict__ bw = d.bw + sm;
    const int32_t *__restrict__ lat = d.lat + sm;
    const int32_t *__restrict__ cap = d.cap + sm;
    const size_t fo = (size_t)s * d.fifo_total;
    uint32_t *fx = d.fifo_x + fo;
    uint32_t *frdy = d.fifo_rdy + fo;
    int32_t *fpp = d.fifo_pp + fo;
    uint32_t *qhead = d.qhead + sm;
    uint32_t *qtail = d.qtail + sm;
    uint32_t *rr = d.rr + sm;
    int32_t *cur_rng = d.cur_rng + (size_t)s * d.ns;
    uint32_t *cur_off = d.cur_off + (size_t)s * d.ns;
    uint32_t *delivered = d.delivered + (size_t)s * d.nflows;
    uint32_t *req_cnt = d.req_cnt + sm;
    uint64_t *req_rec = d.req_rec + (size_t)s * d.req_total;
    const size_t nsrc = (size_t)m + d.ns;
    uint32_t *sreq_x = d.sreq_x + (size_t)s * nsrc * bmax;
    int32_t *sreq_pp = d.sreq_pp + (size_t)s * nsrc * bmax;
    int32_t *sreq_n = d.sreq_n + (size_t)s * nsrc;
    int32_t *grant = d.grant + (size_t)s * nsrc * bmax;
    uint32_t *gcount = d.gcount + sm;
    uint32_t *glist = d.glist + sm * bmax;
    uint8_t *gdep = d.gdep + sm * bmax;
    uint32_t *comp = d.completion + (size_t)s * d.T;
    uint64_t *tx = d.tx_lines + sm;
    uint64_t *busy = d.busy + sm;
    const int32_t *__restrict__ path = d.path_link;

    __shared__ uint32_t sh_t, sh_next, sh_anydep, sh_ndone;
    __shared__ int32_t sh_state;

    for (int l = tid; l < m; l += kThreads) {
        qhead[l] = 0;
        qtail[l] = 0;
        rr[l] = 0;
        req_cnt[l] = 0;
        gcount[l] = 0;
        tx[l] = 0;
        busy[l] = 0;
    }
    for (size_t i = tid; i < (size_t)m * bmax; i += kThreads) gdep[i] = 0;
    for (size_t i = tid; i < nsrc * bmax; i += kThreads) grant[i] = -1;
    for (size_t i = tid; i < nsrc; i += kThreads) sreq_n[i] = 0;
    for (int j = tid; j < d.ns; j += kThreads) {
        cur_rng[j] = d.s_rbeg[j];
        cur_off[j] = 0;
    }
    for (int f = tid; f < d.nflows; f += kThreads) delivered[f] = 0;
    if (tid == 0) {
        sh_t = 0;
        sh_state = d.T > 0 ? kRunRunning : kRunOk;
        sh_next = kNever;
        sh_anydep = 0;
        sh_ndone = 0;
    }
    __syncthreads();

    uint64_t done = 0, processed = 0;  // meaningful in thread 0
    const int nact = d.n_fsrc + d.ns;
    while (sh_state == kRunRunning) {
        const uint32_t t = sh_t;
        // ---------------------------------------------------------------- R
        for (int a = tid; a < nact; a += kThreads) {
            if (a < d.n_fsrc) {
                const int l = d.fsrc_link[a];
                const uint32_t h = qhead[l];
                const uint32_t occ = qtail[l] - h;
                const int b = bw[l];
                const int base = d.fifo_off[l], mask = d.fifo_mask[l];
                int nr = 0;
                for (int k = 0; k < b && (uint32_t)k < occ; k++) {
                    const int e = base + (int)((h + k) & (uint32_t)mask);
                    const uint32_t rdy = frdy[e];
                    if (rdy > t) {
                        atomicMin(&sh_next, rdy);
                        break;
                    }
                    const uint32_t x = fx[e];
                    const int pp = fpp[e] + 1;
                    const int tgt = path[pp];
                    const size_t si = (size_t)l * bmax + k;
                    sreq_x[si] = x;
                    sreq_pp[si] = pp;
                    if (tgt < 0) {
                        grant[si] = -2;  // the sink takes everything
                    } else {
                        const uint32_t P = (uint32_t)d.nports_tail[tgt];
                        const uint32_t key =
                            d.arb == 0 ? x
                                       : (uint32_t)k * P + ((uint32_t)d.port_at_head[l] + P - rr[tgt]) % P;
                        const uint32_t slot = atomicAdd(&req_cnt[tgt], 1u);
                        req_rec[d.req_off[tgt] + slot] = ((uint64_t)key << 32) | ((uint32_t)l << 8) | (uint32_t)k;
                    }
                    nr++;
                }
                sreq_n[l] = nr;
            } else {
                const int j = a - d.n_fsrc;
                const int f = d.s_link[j];
                const int src = m + j;
                int R = cur_rng[j];
                uint32_t o = cur_off[j];
                const int rend = d.s_rend[j];
                const int b = bw[f];
                const uint32_t P = (uint32_t)d.nports_tail[f];
                int nr = 0;
                for (int k = 0; k < b && R < rend; k++) {
                    bool ok = true;
                    for (int q = d.r_pd[R]; q < d.r_pd[R + 1]; q++)
                        if (delivered[d.pd_flow[q]] <= d.pd_base[q] + o) {
                            ok = false;
                            break;
                        }
                    if (!ok) break;
                    const uint32_t x = d.r_start[R] + o;
                    const size_t si = (size_t)src * bmax + k;
                    sreq_x[si] = x;
                    sreq_pp[si] = d.r_path[R];
                    const uint32_t key = d.arb == 0 ? x : (uint32_t)k * P + ((P - 1) + P - rr[f]) % P;
                    const uint32_t slot = atomicAdd(&req_cnt[f], 1u);
                    req_rec[d.req_off[f] + slot] = ((uint64_t)key << 32) | ((uint32_t)src << 8) | (uint32_t)k;
                    nr++;
                    if (++o == d.r_len[R]) {
                        R++;
                        o = 0;
                    }
                }
                sreq_n[src] = nr;
            }
        }
        __syncthreads();
        // ---------------------------------------------------------------- G
        for (int a = tid; a < d.n_fsrc; a += kThreads) {
            const int f = d.fsrc_link[a];
            const uint32_t c = req_cnt[f];
            if (c == 0) continue;
            req_cnt[f] = 0;
            const int occ = (int)(qtail[f] - qhead[f]);
            int g = bw[f];
            if (cap[f] - occ < g) g = cap[f] - occ;
            if ((int)c < g) g = (int)c;
            const uint64_t *rec = req_rec + d.req_off[f];
            for (uint32_t i = 0; i < c; i++) {
                const uint64_t ri = rec[i];
                const uint32_t ki = (uint32_t)(ri >> 32);
                int rank = 0;
                for (uint32_t jj = 0; jj < c; jj++) rank += ((uint32_t)(rec[jj] >> 32) < ki) ? 1 : 0;
                if (rank < g) {
                    const uint32_t sk = (uint32_t)ri;
                    glist[(size_t)f * bmax + rank] = sk;
                    grant[(size_t)(sk >> 8) * bmax + (sk & 255u)] = rank;
                }
            }
            gcount[f] = (uint32_t)(g > 0 ? g : 0);
        }
        __syncthreads();
        // ---------------------------------------------------------------- D
        for (int a = tid; a < nact; a += kThreads) {
            const int src = a < d.n_fsrc ? d.fsrc_link[a] : m + (a - d.n_fsrc);
            const int nr = sreq_n[src];
            if (nr == 0) continue;
            sreq_n[src] = 0;
            int dep = 0, sinks = 0;
            bool open = true;
            for (int k = 0; k < nr; k++) {
                const size_t si = (size_t)src * bmax + k;
                const int gr = grant[si];
                grant[si] = -1;
                if (!open || gr == -1) {
                    open = false;
                    continue;
                }
                dep++;
                const int pv = path[sreq_pp[si]];
                if (gr == -2) {
                    comp[sreq_x[si]] = t + 1;
                    delivered[-pv - 1]++;
                    sinks++;
                } else {
                    gdep[(size_t)pv * bmax + gr] = 1;
                }
            }
            if (dep) {
                sh_anydep = 1;
                if (src < m) {
                    qhead[src] += (uint32_t)dep;
                } else {
                    const int j = src - m;
                    int R = cur_rng[j];
                    uint32_t o = cur_off[j] + (uint32_t)dep;
                    while (R < d.s_rend[j] && o >= d.r_len[R]) {
                        o -= d.r_len[R];
                        R++;
                    }
                    cur_rng[j] = R;
                    cur_off[j] = o;
                }
                if (sinks) atomicAdd(&sh_ndone, (uint32_t)sinks);
            }
        }
        __syncthreads();
        // ---------------------------------------------------------------- E
        for (int a = tid; a < d.n_fsrc; a += kThreads) {
            const int f = d.fsrc_link[a];
            const int g = (int)gcount[f];
            if (g == 0) continue;
            gcount[f] = 0;
            const uint32_t P = (uint32_t)d.nports_tail[f];
            uint32_t tl = qtail[f];
            const int base = d.fifo_off[f], mask = d.fifo_mask[f];
            const uint32_t ready = t + (uint32_t)lat[f];
            int cnt = 0;
            uint32_t last_port = 0;
            for (int r = 0; r < g; r++) {
                const size_t gi = (size_t)f * bmax + r;
                if (!gdep[gi]) continue;
                gdep[gi] = 0;
                const uint32_t sk = glist[gi];
                const int src = (int)(sk >> 8);
                const size_t si = (size_t)src * bmax + (sk & 255u);
                const int e = base + (int)(tl & (uint32_t)mask);
                fx[e] = sreq_x[si];
                frdy[e] = ready;
                fpp[e] = sreq_pp[si];
                tl++;
                cnt++;
                last_port = src < m ? (uint32_t)d.port_at_head[src] : P - 1;
            }
            if (cnt) {
                qtail[f] = tl;
                tx[f] += (uint64_t)cnt;
                busy[f] += 1;
                if (d.arb == 1) rr[f] = (last_port + 1) % P;
            }
        }
        __syncthreads();
        // ---------------------------------------------------------------- time
        if (tid == 0) {
            processed++;
            done += sh_ndone;
            uint32_t nt = t;
            int32_t state = kRunRunning;
            if (done == (uint64_t)d.T) {
                state = kRunOk;
                d.makespan[s] = t + 1;
            } else if (sh_anydep) {
                nt = t + 1;
            } else if (sh_next == kNever) {
                state = kRunDeadlock;
            } else {
                nt = sh_next;
            }
            if (state == kRunRunning && (uint64_t)nt > d.max_cycles) state = kRunMaxCycles;
            if (state == kRunRunning && processed > d.watchdog) state = kRunWatchdog;
            sh_t = nt;
            sh_state = state;
            sh_next = kNever;
            sh_anydep = 0;
            sh_ndone = 0;
        }
        __syncthreads();
    }
    if (tid == 0) {
        if (d.T == 0) d.makespan[s] = 0;
        d.status[s] = sh_state;
        d.cycles[s] = processed;
    }
}

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

__device__ __forceinline__ void lds_fence_wave() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void lds_fence_block() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// A stream's current id range and its first kPredCache predecessor descriptors.
struct RangeReg {
    uint32_t start, len;
    int32_t path, pd0, pd1;
    int32_t pf[kPredCache];
    uint32_t pb[kPredCache];
};

__device__ __forceinline__ void load_range(const DevNet &d, int R, RangeReg &r) {
    r.start = d.r_start[R];
    r.len = d.r_len[R];
    r.path = d.r_path[R];
    r.pd0 = d.r_pd[R];
    r.pd1 = d.r_pd[R + 1];
#pragma unroll
    for (int q = 0; q < kPredCache; q++) {
        const int idx = r.pd0 + q;
        const bool in = idx < r.pd1;
        r.pf[q] = in ? d.pd_flow[idx] : 0;
        r.pb[q] = in ? d.pd_base[idx] : 0;
    }
}

// Line start+o of range r may be injected: every predecessor flow has
// delivered more than base+o lines (values as of the start of the cycle).
__device__ __forceinline__ bool released(const DevNet &d, const RangeReg &r, uint32_t o, const uint32_t *deliv) {
    bool ok = true;
#pragma unroll
    for (int q = 0; q < kPredCache; q++)
        if (r.pd0 + q < r.pd1) ok = ok && deliv[r.pf[q]] > r.pb[q] + o;
    for (int idx = r.pd0 + kPredCache; ok && idx < r.pd1; idx++) ok = deliv[d.pd_flow[idx]] > d.pd_base[idx] + o;
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
template <int BM, bool ONEWAVE, int ARB>
__global__ void __launch_bounds__(1024) engine_lane(DevNet d) {
    extern __shared__ __align__(16) unsigned char smem[];
    uint4 *fifo = reinterpret_cast<uint4 *>(smem);
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
    RangeReg cur{};
    if (on) {
        link = d.fsrc_link[i];
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
                    const uint4 e = fifo[fbase + ((head + k) & fmask)];
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
            RangeReg sr = cur;
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
        if (on) {
            const uint32_t c = req_cnt[i];
            if (c) {
                req_cnt[i] = 0;
                if (c > (uint32_t)rcap) overflow = true;
                g = cap - (int)(tail - head);
                if (b < g) g = b;
                if ((int)c < g) g = (int)c;
                if (g > 0 && !overflow) {
                    if (c == 1) {
                        const uint4 r0 = req[rbase];
                        grant[(r0.z >> 8) * BM + (r0.z & 255u)] = 0;
                        glist[i * BM] = (uint32_t)rbase;
                    } else {
                        for (uint32_t a = 0; a < c; a++) {
                            const uint4 ra = req[rbase + a];
                            const uint32_t ka = ARB == 0 ? ra.x : (ra.z & 255u) * P + (ra.w + P - rr) % P;
                            int rank = 0;
                            for (uint32_t q = 0; q < c; q++) {
                                const uint4 rq = req[rbase + q];
                                const uint32_t kq = ARB == 0 ? rq.x : (rq.z & 255u) * P + (rq.w + P - rr) % P;
                                rank += kq < ka ? 1 : 0;
                            }
                            if (rank < g) {
                                grant[(ra.z >> 8) * BM + (ra.z & 255u)] = rank;
                                glist[i * BM + rank] = (uint32_t)rbase + a;
                            }
                        }
                    }
                }
                if (g < 0) g = 0;
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
                if (ARB == 1) rr = (last_port + 1) % P;
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
            if (dep > 0) red[p] = 1u;
            if (act) red[p + 1] = 1u;
            if (next != kNever) atomicMin(&red[p + 2], next);
            if (overflow) red[p + 3] = 1u;
            lds_fence_block();
            any_dep = red[p] != kNever;
            any_act = red[p + 1] != kNever;
            nxt = red[p + 2];
            any_over = red[p + 3] != kNever;
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
    auto k = engine_lane<BM, ONEWAVE, ARB>;
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

int launch_engine(const DevNet &d, void *stream) {
    hipStream_t st = (hipStream_t)stream;
    if (d.engine == kEngineLane) {
        switch (d.bm) {
        case 1: return (int)launch_lane<1>(d, st);
        case 2: return (int)launch_lane<2>(d, st);
        case 4: return (int)launch_lane<4>(d, st);
        case 8: return (int)launch_lane<8>(d, st);
        case 16: return (int)launch_lane<16>(d, st);
        case 32: return (int)launch_lane<32>(d, st);
        default: return (int)launch_lane<64>(d, st);
        }
    }
    hipLaunchKernelGGL(engine_wg, dim3((unsigned)d.S), dim3(kThreads), 0, st, d);
    return (int)hipGetLastError();
}

}  // namespace simgpu
