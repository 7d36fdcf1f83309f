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
// delivered more than base+o lines (values as of the start of the cycle).
template <int PC>
__device__ __forceinline__ bool released(const DevNet &d, const RangeReg<PC> &r, uint32_t o, const uint32_t *deliv) {
    bool ok = true;
#pragma unroll
    for (int q = 0; q < PC; q++)
        if (r.pd0 + q < r.pd1) ok = ok && deliv[r.pf[q]] > r.pb[q] + o;
    for (int idx = r.pd0 + PC; ok && idx < r.pd1; idx++) ok = deliv[d.pd_flow[idx]] > d.pd_base[idx] + o;
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
// HBMFIFO: the FIFO rings live in HBM instead of LDS (a ring is only ever
// touched by its own lane, so no extra ordering is needed).
template <int BM, bool ONEWAVE, int ARB, bool HBMFIFO>
__global__ void __launch_bounds__(1024) engine_lane(DevNet d) {
    extern __shared__ __align__(16) unsigned char smem[];
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

// ----------------------------------------------------------------------------
// Compact engine for graphs whose every link moves one line per cycle
// (b = 1).  Then a source offers at most one line, a link grants at most one
// and a grant always departs (no void grants), so one exchange decides and
// commits a move; and a link admits at most one line per cycle, so its busy
// cycles equal its admitted lines.  Thread t owns lanes t + q*NT (q < LPT);
// lanes 0..b1_ns-1 start an injection stream and are owned by thread = lane
// as its first lane.  Requests go through one 64-bit LDS word per target:
//   round-robin  the requester ORs in its port bit and posts {line, path
//                index} in its own LDS slot; the winner is the first set bit
//                at or after the pointer, the target copies the winner's post
//                into its ring and marks the post as won;
//   lowest-id    requesters take the atomic minimum of (line << 32 | path
//                index); the target appends the winner and a source departs
//                when the word still holds its line (words are double
//                buffered by cycle parity).
// Rings live in HBM as {line, path index, ready, next hop} and are touched
// only by their own thread; the next hop is looked up once, when the entry is
// appended, and each lane keeps its head entry in registers, fetching the
// next one right after a pop.  Phase boundaries wait on LDS only.
template <int LPT, int ARB, int PC>
__global__ void __launch_bounds__(1024) engine_b1(DevNet d) {
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned long long *word = reinterpret_cast<unsigned long long *>(smem + d.o_word);
    unsigned long long *post = reinterpret_cast<unsigned long long *>(smem + d.o_gnt);
    uint16_t *inl = reinterpret_cast<uint16_t *>(smem + d.o_inl);
    uint32_t *cnt = reinterpret_cast<uint32_t *>(smem + d.o_b1cnt);  // [nl] lines admitted
    uint16_t *lino = reinterpret_cast<uint16_t *>(smem + d.o_b1ino); // [nl] tail node's in-lane offset
    uint32_t *red = reinterpret_cast<uint32_t *>(smem + d.o_b1red);
    const int s = blockIdx.x;
    const int tid = threadIdx.x;
    const int NT = blockDim.x;
    const int nl = d.nl;
    const int m = d.m;
    uint4 *fifo = d.gfifo + (size_t)s * d.fifo_total;
    uint32_t *deliv = d.b1_deliv_lds ? reinterpret_cast<uint32_t *>(smem + d.o_b1deliv)
                                     : (d.gdeliv ? d.gdeliv + (size_t)s * d.nflows : nullptr);
    const int32_t *path = d.path_lane;
    constexpr unsigned long long kNone = ARB == 0 ? ~0ull : 0ull;
    constexpr unsigned long long kWon = ~0ull;
    const int nword = ARB == 0 ? 2 * nl : nl;

    for (int j = tid; j < nword; j += NT) word[j] = kNone;
    if (ARB == 1) {
        for (int j = tid; j < m; j += NT) inl[j] = (uint16_t)d.in_lane[j];
        for (int j = tid; j < nl; j += NT) lino[j] = (uint16_t)d.ln_inoff[j];
    }
    const uint32_t lg = (uint32_t)d.b1_ring_lg;  // every ring has 2^lg entries
    const uint32_t rmask = (1u << lg) - 1u;
    if (PC > 0)
        for (int j = tid; j < d.nflows; j += NT) deliv[j] = 0;
    if (tid < 16) red[tid] = kNever;
    for (int j = tid; j < nl; j += NT) cnt[j] = 0;
    for (int j = tid; j < m; j += NT)
        if (d.link_lane[j] < 0) {
            d.tx_lines[(size_t)s * m + j] = 0;
            d.busy[(size_t)s * m + j] = 0;
        }

    // per-lane registers
    uint32_t head[LPT], tail[LPT];
    uint32_t cx[LPT], cpp[LPT], crdy[LPT];  // cached head entry
    int32_t ctg[LPT];    // cached head entry's next hop (lane, or -(1 + flow) for the sink)
    int32_t ntg[LPT];    // next hop of the last appended entry (load in flight until the next cycle)
    uint32_t st8[LPT];   // rr (bits 0-7) | cache valid (8) | request: sink (9), posted (10) | pending (11)
    uint32_t pa[LPT];    // cap (bits 0-16) | own port (22-27)
    uint32_t pb[LPT];    // P (bits 0-6) | lane has a stream (bit 7) | latency (8-31)
#pragma unroll
    for (int q = 0; q < LPT; q++) {
        head[q] = tail[q] = 0;
        cx[q] = cpp[q] = crdy[q] = 0;
        st8[q] = 0;
        ctg[q] = ntg[q] = 0;
        pa[q] = pb[q] = 0;
        const int lane = tid + q * NT;
        if (lane < nl) {
            const int link = d.ln_link[lane];
            const size_t pi = (size_t)s * m + link;
            pa[q] = (uint32_t)d.cap[pi] | ((uint32_t)d.ln_port[lane] << 22);
            // a lane with a stream has an endpoint tail whose last port is
            // the injection port; no other lane ever sees a request there
            pb[q] = (uint32_t)d.ln_P[lane] | ((uint32_t)d.lat[pi] << 8) |
                    (d.ln_srbeg[lane] != d.ln_srend[lane] ? 128u : 0u);
        }
    }
    int R = 0, rend = 0;
    uint32_t o = 0;
    RangeReg<PC> cur{};
    const bool has_stream = tid < d.b1_ns;
    if (has_stream) {
        R = d.ln_srbeg[tid];
        rend = d.ln_srend[tid];
        if (R < rend) load_range(d, R, cur);
    }
    lds_fence_block();

    uint32_t *comp = d.completion + (size_t)s * d.T;
    uint32_t t = 0;
    uint64_t processed = 0;
    int32_t state = d.T > 0 ? kRunRunning : kRunOk;

    while (state == kRunRunning) {
        const int par = (int)(processed & 1u);
        unsigned long long *wcur = ARB == 0 ? word + (size_t)par * nl : word;
        // -------------------------------------------------------------- R
        uint32_t next = kNever;
#pragma unroll
        for (int q = 0; q < LPT; q++) {
            const int lane = tid + q * NT;
            st8[q] &= 0x9FFu;
            if (st8[q] & 2048u) {
                // complete the entry appended last cycle with its next hop
                const uint32_t last = (tail[q] - 1u) & rmask;
                reinterpret_cast<int32_t *>(fifo + ((size_t)lane << lg) + last)[3] = ntg[q];
                if ((st8[q] & 256u) && head[q] == tail[q] - 1u) ctg[q] = ntg[q];
                st8[q] &= ~2048u;
            }
            if (lane < nl && tail[q] != head[q]) {
                if (!(st8[q] & 256u)) {
                    const uint4 e = fifo[((size_t)lane << lg) + (head[q] & rmask)];
                    cx[q] = e.x;
                    cpp[q] = e.y;
                    crdy[q] = e.z;
                    ctg[q] = (int32_t)e.w;
                    st8[q] |= 256u;
                }
                if (crdy[q] > t) {
                    next = crdy[q] < next ? crdy[q] : next;
                } else {
                    const int tgt = ctg[q];
                    if (tgt < 0) {
                        st8[q] |= 512u;
                    } else {
                        st8[q] |= 1024u;
                        if (ARB == 1) {
                            post[lane] = ((unsigned long long)cx[q] << 32) | (cpp[q] + 1u);
                            atomicOr(&wcur[tgt], 1ull << ((pa[q] >> 22) & 63u));
                        } else {
                            atomicMin(&wcur[tgt], ((unsigned long long)cx[q] << 32) | (cpp[q] + 1u));
                        }
                    }
                }
            }
        }
        bool sreq = false;
        uint32_t sx = 0;
        if (has_stream && R < rend && released(d, cur, o, deliv)) {
            sreq = true;
            sx = cur.start + o;
            if (ARB == 1)
                atomicOr(&wcur[tid], 1ull << ((pb[0] & 127u) - 1u));
            else
                atomicMin(&wcur[tid], ((unsigned long long)sx << 32) | (uint32_t)cur.path);
        }
        lds_fence_block();
        // -------------------------------------------------------------- G
        bool sdep = false;
#pragma unroll
        for (int q = 0; q < LPT; q++) {
            const int lane = tid + q * NT;
            if (lane >= nl) continue;
            if (ARB == 0) word[(size_t)(par ^ 1) * nl + lane] = kNone;  // buffer of the next cycle
            const unsigned long long w = wcur[lane];
            if (w == kNone) continue;
            if (ARB == 1) wcur[lane] = 0ull;
            const uint32_t occ = tail[q] - head[q];
            if (occ >= (pa[q] & 0x1FFFFu)) {
                if (ARB == 0) wcur[lane] = kNone;  // full: nobody moves
                continue;
            }
            const size_t idx = ((size_t)lane << lg) + (tail[q] & rmask);
            const uint32_t ready = t + (pb[q] >> 8);
            uint32_t x, pp;
            if (ARB == 1) {
                const uint32_t P = pb[q] & 127u;
                const uint32_t rrp = st8[q] & 255u;
                const unsigned long long hi = w >> rrp;
                const uint32_t p = hi ? rrp + (uint32_t)__builtin_ctzll(hi) : (uint32_t)__builtin_ctzll(w);
                if ((pb[q] & 128u) && p == P - 1u) {
                    x = sx;  // the injection port: this thread's own stream (lane == tid)
                    pp = (uint32_t)cur.path;
                    sdep = true;
                } else {
                    const int win = inl[(int)lino[lane] + (int)p];
                    const unsigned long long pw = post[win];
                    post[win] = kWon;
                    x = (uint32_t)(pw >> 32);
                    pp = (uint32_t)pw;
                }
                st8[q] = (st8[q] & ~255u) | (p + 1u == P ? 0u : p + 1u);
            } else {
                x = (uint32_t)(w >> 32);
                pp = (uint32_t)w;
            }
            fifo[idx] = make_uint4(x, pp, ready, 0u);
            ntg[q] = path[pp + 1];  // written into the entry at the start of the next cycle
            st8[q] |= 2048u;
            if (occ == 0) {
                cx[q] = x;
                cpp[q] = pp;
                crdy[q] = ready;
                st8[q] |= 256u;
            }
            tail[q]++;
            cnt[lane]++;
        }
        lds_fence_block();
        // -------------------------------------------------------------- D
        int dep = 0;
#pragma unroll
        for (int q = 0; q < LPT; q++) {
            const int lane = tid + q * NT;
            if (lane >= nl) continue;
            bool gone = false;
            if (st8[q] & 512u) {
                comp[cx[q]] = t + 1;
                if (PC > 0) deliv[-ctg[q] - 1] += 1u;
                gone = true;
            } else if (st8[q] & 1024u) {
                gone = ARB == 1 ? post[lane] == kWon : (uint32_t)(wcur[ctg[q]] >> 32) == cx[q];
            }
            if (gone) {
                head[q]++;
                dep++;
                st8[q] &= ~256u;
                // fetch the next head now (used next cycle) unless it is the
                // entry appended this cycle, which is completed next cycle
                if (tail[q] != head[q] && !((st8[q] & 2048u) && head[q] == tail[q] - 1u)) {
                    const uint4 e = fifo[((size_t)lane << lg) + (head[q] & rmask)];
                    cx[q] = e.x;
                    cpp[q] = e.y;
                    crdy[q] = e.z;
                    ctg[q] = (int32_t)e.w;
                    st8[q] |= 256u;
                }
            }
        }
        if (sreq) {
            const bool won = ARB == 1 ? sdep : (uint32_t)(wcur[tid] >> 32) == sx;
            if (won) {
                dep++;
                if (++o >= cur.len) {
                    o = 0;
                    R++;
                    if (R < rend) load_range(d, R, cur);
                }
            }
        }
        // -------------------------------------------------------------- time
        processed++;
        bool act = has_stream && R < rend;
#pragma unroll
        for (int q = 0; q < LPT; q++)
            if (tid + q * NT < nl && tail[q] != head[q]) act = true;
        const int p4 = par * 4;
        const bool wdep = __ballot(dep > 0) != 0, wact = __ballot(act) != 0;
        if ((tid & 63) == 0) {
            if (wdep) red[p4] = 1u;
            if (wact) red[p4 + 1] = 1u;
        }
        lds_fence_block();
        const bool any_dep = red[p4] != kNever;
        const bool any_act = red[p4 + 1] != kNever;
        uint32_t nxt = kNever;
        if (!any_dep && any_act) {  // only an idle cycle needs the next event time
            uint32_t v = next;
#pragma unroll
            for (int sh = 32; sh >= 1; sh >>= 1) {
                const uint32_t u = (uint32_t)__shfl_xor((int)v, sh);
                v = u < v ? u : v;
            }
            if ((tid & 63) == 0 && v != kNever) atomicMin(&red[p4 + 2], v);
            lds_fence_block();
            nxt = red[p4 + 2];
        }
        if (tid < 4) red[(4 - p4) + tid] = kNever;
        if (!any_act) {
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
    }
    lds_fence_block();
#pragma unroll
    for (int q = 0; q < LPT; q++) {
        const int lane = tid + q * NT;
        if (lane < nl) {
            const int link = d.ln_link[lane];
            d.tx_lines[(size_t)s * m + link] = cnt[lane];
            d.busy[(size_t)s * m + link] = cnt[lane];
        }
    }
    if (tid == 0) {
        d.makespan[s] = d.T > 0 ? t + 1 : 0;
        d.status[s] = state;
        d.cycles[s] = processed;
    }
}

template <int ARB>
hipError_t launch_b1(const DevNet &d, hipStream_t st) {
    const int nthr = d.nl > 1024 ? 1024 : ((d.nl + 63) / 64) * 64;
    const int lpt = (d.nl + nthr - 1) / nthr;
    auto go = [&](auto kern) {
        if (d.lds_bytes > 65536)
            (void)hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, d.lds_bytes);
        hipLaunchKernelGGL(kern, dim3((unsigned)d.S), dim3(nthr), (unsigned)d.lds_bytes, st, d);
        return hipGetLastError();
    };
    if (d.has_preds) {
        if (lpt <= 1) return go(engine_b1<1, ARB, kPredCache>);
        if (lpt <= 2) return go(engine_b1<2, ARB, kPredCache>);
        if (lpt <= 4) return go(engine_b1<4, ARB, kPredCache>);
        if (lpt <= 6) return go(engine_b1<6, ARB, kPredCache>);
        return go(engine_b1<8, ARB, kPredCache>);
    }
    if (lpt <= 1) return go(engine_b1<1, ARB, 0>);
    if (lpt <= 2) return go(engine_b1<2, ARB, 0>);
    if (lpt <= 4) return go(engine_b1<4, ARB, 0>);
    if (lpt <= 6) return go(engine_b1<6, ARB, 0>);
    return go(engine_b1<8, ARB, 0>);
}

}  // namespace

int launch_engine(const DevNet &d, void *stream) {
    hipStream_t st = (hipStream_t)stream;
    if (d.engine == kEngineB1) return (int)(d.arb == 0 ? launch_b1<0>(d, st) : launch_b1<1>(d, st));
    if (d.engine == kEngineLane || d.engine == kEngineLaneHbm) {
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
