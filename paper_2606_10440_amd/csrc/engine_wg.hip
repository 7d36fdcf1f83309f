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
// FIFO-head ready time or credit return (no such time = deadlock).
//
// Active sets (ACT): a bitmap in LDS marks the sources that hold anything (a
// link FIFO with entries, waiting or owed a credit; a stream with lines
// left).  Each cycle starts by compacting it into a list, and R and D walk
// that list; R appends each target that receives its first request of the
// cycle to a target list, which G and E walk.  D clears the bit of a source
// it empties, E sets the bit of a link it appends to, so a cycle costs in
// proportion to the busy part of the graph rather than to the whole graph.
// A stream whose next line waits on predecessors sleeps (its bit cleared in
// R) until one of the flows it waits on delivers a line (D sets its bit):
// only a delivery can release a line.
// R also lists every request (target, slot); when the cycle's requests fit
// that list and arbitration is by key alone, G ranks one request per thread
// (its rank = the number of smaller keys at its target) instead of one
// target per thread, which spreads a busy router's many requests.
// Without ACT every phase scans every source or target.
//
// With credit delays a line that leaves a FIFO keeps its slot until the
// credit is back: the entry stays between qcred and qhead with the cycle it
// left in place of its ready time.
//
// Predecessor release uses per-flow delivered counters: lines of one flow
// (same source, destination and hence path) are injected in id order and
// FIFOs never reorder, so a flow delivers its lines in id order and "line
// with flow sequence q has completed" is "delivered > q" at cycle start.
#include <hip/hip_runtime.h>

#include "sim_internal.h"

namespace simgpu {

namespace {

// FIFO heads, requests and grants of one source or target are handled kC at
// a time, so that their memory loads are in flight together.
constexpr int kC = 4;
// Stream offers read kW ranges at a time and their predecessor descriptors
// kE at a time.
constexpr int kW = 4;
constexpr int kE = 8;
constexpr uint32_t kNoSpill = 0xFFFFFFFFu;  // a spill-list entry that holds no chunk

// SM: the per-link and per-stream scalars (queue pointers, request and grant
// counts, round-robin and class pointers, stream cursors) live in LDS, so
// that the every-cycle scans over idle links cost LDS reads; FIFO entries and
// request records stay in HBM.  Otherwise all state is in HBM.
// kThreads: 16 waves per CU in all, so that every scenario's workgroup is
// resident at once when there are at most 1024 (1024 threads up to 256
// scenarios, 512 up to 512, else 256) and each thread keeps up to 128
// registers for the chunked loops below.
// ACT: active sets in LDS, after the scalars (see above).
template <bool SM, bool ACT, int kThreads>
__global__ void __launch_bounds__(kThreads, 4) engine_wg(DevNet d) {
    extern __shared__ __align__(16) uint32_t wg_lds[];
    const int s = blockIdx.x;
    const int tid = threadIdx.x;
    const int m = d.m;
    const int bmax = d.bmax;
    const size_t sm = (size_t)s * m;
    const int32_t *__restrict__ bw = d.bw + sm;
    const int32_t *__restrict__ lat = d.lat + sm;
    const int32_t *__restrict__ cap = d.cap + sm;
    const int32_t *__restrict__ cred = d.credit ? d.credit + sm : nullptr;
    const size_t fo = (size_t)s * d.fifo_total;
    uint32_t *fx = d.fifo_x + fo;
    uint32_t *frdy = d.fifo_rdy + fo;
    int32_t *fpp = d.fifo_pp + fo;
    const bool fair = (d.arb & 2) != 0;
    const uint8_t *lcls = d.line_cls;  // null: every line is data
    const size_t nsrc = (size_t)m + d.ns;
    uint32_t *qhead, *qtail, *qcred, *cptr, *rr, *cur_off, *req_cnt, *gcount;
    int32_t *cur_rng, *sreq_n;
    if constexpr (SM) {
        uint32_t *p = wg_lds;
        qhead = p; p += m;
        qtail = p; p += m;
        qcred = p; p += m;
        cptr = p; p += m;
        rr = p; p += m;
        req_cnt = p; p += m;
        gcount = p; p += m;
        sreq_n = reinterpret_cast<int32_t *>(p); p += nsrc;
        cur_rng = reinterpret_cast<int32_t *>(p); p += d.ns;
        cur_off = p;
    } else {
        qhead = d.qhead + sm;
        qtail = d.qtail + sm;
        qcred = d.qcred + sm;
        cptr = d.cptr + sm;
        rr = d.rr + sm;
        req_cnt = d.req_cnt + sm;
        gcount = d.gcount + sm;
        sreq_n = d.sreq_n + (size_t)s * nsrc;
        cur_rng = d.cur_rng + (size_t)s * d.ns;
        cur_off = d.cur_off + (size_t)s * d.ns;
    }
    uint32_t *delivered = d.delivered + (size_t)s * d.nflows;
    uint64_t *req_rec = d.req_rec + (size_t)s * d.req_total;
    uint32_t *req_aux = d.req_aux ? d.req_aux + (size_t)s * d.req_total : nullptr;
    uint32_t *sreq_x = d.sreq_x + (size_t)s * nsrc * bmax;
    int32_t *sreq_pp = d.sreq_pp + (size_t)s * nsrc * bmax;
    int32_t *grant = d.grant + (size_t)s * nsrc * bmax;
    uint32_t *glist = d.glist + sm * bmax;
    uint8_t *gdep = d.gdep + sm * bmax;
    uint32_t *comp = d.completion + (size_t)s * d.T;
    uint64_t *tx = d.tx_lines + sm;
    uint64_t *busy = d.busy + sm;
    const int32_t *__restrict__ path = d.path_link;

    __shared__ uint32_t sh_t, sh_next, sh_anydep, sh_ndone, sh_nalive, sh_ntgt, sh_nreq, sh_nspill;
    __shared__ int32_t sh_state;
    // active sets: live-source bitmap [nw], live-source list [m + ns], target list [m],
    // request list [wg_rcap] of (target, slot), spill list [wg_scap]
    const int nw = (int)((nsrc + 31) / 32);
    const size_t aoff = SM ? (size_t)d.wg_lds : 0;
    uint32_t *livew = reinterpret_cast<uint32_t *>(reinterpret_cast<unsigned char *>(wg_lds) + aoff);
    int32_t *alist = reinterpret_cast<int32_t *>(livew + nw);
    int32_t *tlist = alist + nsrc;
    uint2 *rlist = reinterpret_cast<uint2 *>(reinterpret_cast<unsigned char *>(wg_lds) +
                                             ((aoff + 4 * ((size_t)nw + nsrc + (size_t)m) + 7) & ~(size_t)7));
    const uint32_t rcap = (uint32_t)d.wg_rcap;
    // spill list [wg_scap]: chunks of long FIFO offers, (link << 8 | first head)
    uint32_t *spill = reinterpret_cast<uint32_t *>(rlist + rcap);
    const uint32_t scap = ACT ? (uint32_t)d.wg_scap : 0u;
    auto post = [&](int tgt, uint32_t slot) {  // a request's place in the active sets
        if (slot == 0u) tlist[atomicAdd(&sh_ntgt, 1u)] = tgt;
        const uint32_t q = atomicAdd(&sh_nreq, 1u);
        if (q < rcap) rlist[q] = make_uint2((uint32_t)tgt, slot);
    };
    auto set_live = [&](int src) { atomicOr(&livew[src >> 5], 1u << (src & 31)); };
    auto clear_live = [&](int src) { atomicAnd(&livew[src >> 5], ~(1u << (src & 31))); };

    for (int l = tid; l < m; l += kThreads) {
        qhead[l] = 0;
        qtail[l] = 0;
        qcred[l] = 0;
        cptr[l] = 0;
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
    if constexpr (ACT)
        for (int j = tid; j < nw; j += kThreads) livew[j] = 0;
    if (tid == 0) {
        sh_t = 0;
        sh_state = d.T > 0 ? kRunRunning : kRunOk;
        sh_next = kNever;
        sh_anydep = 0;
        sh_ndone = 0;
        sh_nalive = 0;
        sh_ntgt = 0;
        sh_nreq = 0;
        sh_nspill = 0;
    }
    __syncthreads();
    if constexpr (ACT) {  // streams with lines are live from the start; links start empty
        for (int j = tid; j < d.ns; j += kThreads)
            if (d.s_rbeg[j] < d.s_rend[j]) set_live(m + j);
        __syncthreads();
    }

    uint64_t done = 0, processed = 0;  // meaningful in thread 0
    const int nact = d.n_fsrc + d.ns;
    while (sh_state == kRunRunning) {
        const uint32_t t = sh_t;
        if constexpr (ACT) {  // the live sources, in no particular order
            for (int j = tid; j < nw; j += kThreads) {
                uint32_t bits = livew[j];
                if (bits == 0u) continue;
                int pos = (int)atomicAdd(&sh_nalive, (uint32_t)__popc(bits));
                while (bits) {
                    alist[pos++] = j * 32 + __ffs(bits) - 1;
                    bits &= bits - 1u;
                }
            }
            __syncthreads();
        }
        const int nsrc_now = ACT ? (int)sh_nalive : nact;
        // ---------------------------------------------------------------- R
        // The ready heads of FIFO link l from head k0 on (below lim), kC of
        // them with their loads in flight together, post their requests;
        // returns how many were ready.  Ready times never decrease along a
        // FIFO, so the ready heads are a prefix and a chunk needs no
        // knowledge of the chunks before it: the first head that is not
        // ready offers the next event, and a later one offers no earlier one.
        auto offer_heads = [&](int l, uint32_t h, int k0, int lim) -> int {
            const int base = d.fifo_off[l], mask = d.fifo_mask[l];
            int e[kC];
            uint32_t rdy[kC];
#pragma unroll
            for (int u = 0; u < kC; u++) {
                e[u] = base + (int)((h + (uint32_t)(k0 + u)) & (uint32_t)mask);
                rdy[u] = k0 + u < lim ? frdy[e[u]] : kNever;
            }
            int nrd = 0;
            bool run = true;
#pragma unroll
            for (int u = 0; u < kC; u++) {
                if (run && k0 + u < lim && rdy[u] > t) atomicMin(&sh_next, rdy[u]);  // first head not ready
                run = run && k0 + u < lim && rdy[u] <= t;
                nrd += run ? 1 : 0;
            }
            uint32_t x[kC];
            int pp[kC], tg[kC];
#pragma unroll
            for (int u = 0; u < kC; u++)
                if (u < nrd) {
                    x[u] = fx[e[u]];
                    pp[u] = fpp[e[u]] + 1;
                }
#pragma unroll
            for (int u = 0; u < kC; u++)
                if (u < nrd) tg[u] = path[pp[u]];
            uint32_t P[kC], rot[kC];
            if (d.arb & 1) {
                const uint32_t ph = (uint32_t)d.port_at_head[l];
#pragma unroll
                for (int u = 0; u < kC; u++)
                    if (u < nrd && tg[u] >= 0) {
                        P[u] = (uint32_t)d.nports_tail[tg[u]];
                        rot[u] = rr[tg[u]];
                    }
#pragma unroll
                for (int u = 0; u < kC; u++)
                    if (u < nrd && tg[u] >= 0) rot[u] = (ph + P[u] - rot[u]) % P[u];
            }
#pragma unroll
            for (int u = 0; u < kC; u++) {
                if (u >= nrd) continue;
                const int k = k0 + u;
                const size_t si = (size_t)l * bmax + k;
                sreq_x[si] = x[u];
                sreq_pp[si] = pp[u];
                if (tg[u] < 0) {
                    grant[si] = -2;  // the sink takes everything
                } else {
                    const uint32_t key = (d.arb & 1) == 0 ? x[u] : (uint32_t)k * P[u] + rot[u];
                    const uint32_t slot = atomicAdd(&req_cnt[tg[u]], 1u);
                    req_rec[d.req_off[tg[u]] + slot] = ((uint64_t)key << 32) | ((uint32_t)l << 8) | (uint32_t)k;
                    if (ACT) post(tg[u], slot);
                }
            }
            return nrd;
        };
        for (int a = tid; a < nsrc_now; a += kThreads) {
            const int sid = ACT ? alist[a] : (a < d.n_fsrc ? d.fsrc_link[a] : m + (a - d.n_fsrc));
            if (sid < m) {
                const int l = sid;
                const uint32_t h = qhead[l];
                const uint32_t occ = qtail[l] - h;
                const int b = bw[l];
                if (cred) {
                    // slots of lines that left at least credit cycles ago are free
                    // again; the next return is an event of the time advance
                    const int base = d.fifo_off[l], mask = d.fifo_mask[l];
                    const uint32_t D = (uint32_t)cred[l];
                    uint32_t qc = qcred[l];
                    while (qc != h && frdy[base + (int)(qc & (uint32_t)mask)] + D <= t) qc++;
                    qcred[l] = qc;
                    if (qc != h) atomicMin(&sh_next, frdy[base + (int)(qc & (uint32_t)mask)] + D);
                    if (ACT && qc == qtail[l]) clear_live(l);  // nothing held: every credit is back
                }
                const int lim = b < (int)occ ? b : (int)occ;
                int nr = lim > 0 ? offer_heads(l, h, 0, lim) : 0;
                if (nr == kC && lim > kC) {
                    // every head of the first chunk is ready: the later chunks go
                    // to the spill list, one per thread after the next barrier
                    // (inline if the list is full)
                    const uint32_t nch = (uint32_t)((lim - 1) / kC);
                    const uint32_t s0 = ACT ? atomicAdd(&sh_nspill, nch) : scap;
                    if (s0 + nch <= scap) {
                        for (uint32_t c = 0; c < nch; c++) spill[s0 + c] = ((uint32_t)l << 8) | (uint32_t)(kC * (c + 1));
                    } else {
                        for (uint32_t c = 0; ACT && s0 + c < scap && c < nch; c++) spill[s0 + c] = kNoSpill;
                        for (int k0 = kC; k0 < lim; k0 += kC) {
                            const int n = offer_heads(l, h, k0, lim);
                            nr += n;
                            if (n < kC) break;
                        }
                    }
                }
                sreq_n[l] = nr;
            } else {
                const int j = sid - m;
                const int f = d.s_link[j];
                const int src = m + j;
                int R = cur_rng[j];
                uint32_t o = cur_off[j];
                const int rend = d.s_rend[j];
                const int b = bw[f];
                const uint32_t P = (uint32_t)d.nports_tail[f];
                if (ACT && R >= rend) clear_live(src);
                // ranges in order, kW at a time (their lengths, first lines,
                // paths and predecessor descriptors read together, then every
                // predecessor count of the window): the lines from o on whose
                // predecessors have all delivered (a prefix), all requested at
                // once from the stream's link
                const uint32_t rot = (d.arb & 1) ? ((P - 1) + P - rr[f]) % P : 0u;
                int nr = 0;
                bool go = R < rend;
                while (go && nr < b) {
                    const int nw = rend - R < kW ? rend - R : kW;
                    uint32_t len[kW], st[kW];
                    int rp[kW], pq[kW + 1];
#pragma unroll
                    for (int u = 0; u < kW; u++)
                        if (u < nw) {
                            len[u] = d.r_len[R + u];
                            st[u] = d.r_start[R + u];
                            rp[u] = d.r_path[R + u];
                            pq[u] = d.r_pd[R + u];
                        }
                    pq[kW] = d.r_pd[R + nw];
#pragma unroll
                    for (int u = 1; u < kW; u++)
                        if (u >= nw) pq[u] = pq[kW];  // empty spans past the window
                    // allowance per range: lines o + i (range 0) or i (later
                    // ranges) with delivered > base + i (per line) or > base
                    uint32_t A[kW];
#pragma unroll
                    for (int u = 0; u < kW; u++) A[u] = 0xFFFFFFFFu;
                    for (int q0 = pq[0]; q0 < pq[kW]; q0 += kE) {
                        int fl[kE];
                        uint32_t bs[kE], dv[kE];
#pragma unroll
                        for (int v = 0; v < kE; v++)
                            if (q0 + v < pq[kW]) {
                                fl[v] = d.pd_flow[q0 + v];
                                bs[v] = d.pd_base[q0 + v];
                            }
#pragma unroll
                        for (int v = 0; v < kE; v++)
                            if (q0 + v < pq[kW]) dv[v] = delivered[fl[v]];
#pragma unroll
                        for (int v = 0; v < kE; v++) {
                            const int q = q0 + v;
                            if (q >= pq[kW]) continue;
                            const uint32_t b0 = bs[v] + (q < pq[1] ? (o & d.pd_omask) : 0u);
                            const uint32_t allow = dv[v] > b0 ? (d.pd_omask ? dv[v] - b0 : 0xFFFFFFFFu) : 0u;
#pragma unroll
                            for (int u = 0; u < kW; u++)
                                if (q >= pq[u] && q < pq[u + 1]) A[u] = A[u] < allow ? A[u] : allow;
                        }
                    }
                    // take the ranges' lines in order
                    const uint32_t o0 = o;
                    uint32_t nu[kW];
                    int cnt = 0;
                    bool stop = false;
#pragma unroll
                    for (int u = 0; u < kW; u++) {
                        nu[u] = 0;
                        if (u >= nw || stop) continue;
                        const uint32_t off = u == 0 ? o0 : 0u;
                        uint32_t n = (uint32_t)(b - nr - cnt) < len[u] - off ? (uint32_t)(b - nr - cnt) : len[u] - off;
                        n = n < A[u] ? n : A[u];
                        nu[u] = n;
                        cnt += (int)n;
                        if (n == 0u || off + n < len[u]) {  // held back by a predecessor or by the bandwidth
                            stop = true;
                            R += u;
                            o = off + n;
                        }
                    }
                    if (!stop) {
                        R += nw;
                        o = 0;
                    }
                    go = !stop && R < rend;
                    if (cnt == 0) {
                        if (ACT && nr == 0) clear_live(src);  // asleep until a flow it waits on delivers
                        break;
                    }
                    const uint32_t slot0 = atomicAdd(&req_cnt[f], (uint32_t)cnt);
                    uint64_t *rec = req_rec + d.req_off[f] + slot0;
                    uint32_t i0 = 0;
#pragma unroll
                    for (int u = 0; u < kW; u++) {
                        const uint32_t x0 = st[u] + (u == 0 ? o0 : 0u);
                        for (uint32_t i = 0; i < nu[u]; i++) {
                            const uint32_t k = (uint32_t)nr + i0 + i;
                            const size_t si = (size_t)src * bmax + k;
                            const uint32_t x = x0 + i;
                            sreq_x[si] = x;
                            sreq_pp[si] = rp[u];
                            const uint32_t key = (d.arb & 1) == 0 ? x : k * P + rot;
                            rec[i0 + i] = ((uint64_t)key << 32) | ((uint32_t)src << 8) | k;
                        }
                        i0 += nu[u];
                    }
                    if (ACT) {
                        if (slot0 == 0u) tlist[atomicAdd(&sh_ntgt, 1u)] = f;
                        const uint32_t q = atomicAdd(&sh_nreq, (uint32_t)cnt);
                        for (uint32_t i = 0; i < (uint32_t)cnt && q + i < rcap; i++)
                            rlist[q + i] = make_uint2((uint32_t)f, slot0 + i);
                    }
                    nr += cnt;
                }
                sreq_n[src] = nr;
            }
        }
        if constexpr (ACT) {
            // the spilled chunks of long FIFO offers
            __syncthreads();
            const uint32_t ns_ = sh_nspill < scap ? sh_nspill : scap;
            for (uint32_t i = (uint32_t)tid; i < ns_; i += kThreads) {
                const uint32_t v = spill[i];
                if (v == kNoSpill) continue;
                const int l = (int)(v >> 8), k0 = (int)(v & 255u);
                const uint32_t h = qhead[l];
                const uint32_t occ = qtail[l] - h;
                const int b = bw[l];
                const int lim = b < (int)occ ? b : (int)occ;
                const int n = offer_heads(l, h, k0, lim);
                if (n) atomicMax(&sreq_n[l], k0 + n);
            }
        }
        __syncthreads();
        // ---------------------------------------------------------------- G
        const int ntgt = ACT ? (int)sh_ntgt : d.n_fsrc;
        const uint32_t nreq = ACT ? sh_nreq : 0u;
        const bool flat = ACT && !fair && nreq <= rcap;  // one request per thread
        if (flat) {
            for (uint32_t q = (uint32_t)tid; q < nreq; q += kThreads) {
                const uint2 rq = rlist[q];
                const int f = (int)rq.x;
                const uint32_t c = req_cnt[f];
                const uint64_t *rec = req_rec + d.req_off[f];
                const uint64_t ri = rec[rq.y];
                const uint32_t ki = (uint32_t)(ri >> 32);
                int rank = 0;
                for (uint32_t jj = 0; jj < c; jj++) rank += ((uint32_t)(rec[jj] >> 32) < ki) ? 1 : 0;
                const int occ = (int)(qtail[f] - (cred ? qcred[f] : qhead[f]));
                int g = bw[f];
                if (cap[f] - occ < g) g = cap[f] - occ;
                if ((int)c < g) g = (int)c;
                if (rank < g) {
                    const uint32_t sk = (uint32_t)ri;
                    glist[(size_t)f * bmax + rank] = sk;
                    grant[(size_t)(sk >> 8) * bmax + (sk & 255u)] = rank;
                }
                if (rq.y == 0u) gcount[f] = (uint32_t)(g > 0 ? g : 0);
            }
        }
        for (int a = tid; a < (flat ? 0 : ntgt); a += kThreads) {
            const int f = ACT ? tlist[a] : d.fsrc_link[a];
            const uint32_t c = req_cnt[f];
            if (c == 0) continue;
            req_cnt[f] = 0;
            const int occ = (int)(qtail[f] - (cred ? qcred[f] : qhead[f]));
            int g = bw[f];
            if (cap[f] - occ < g) g = cap[f] - occ;
            if ((int)c < g) g = (int)c;
            const uint64_t *rec = req_rec + d.req_off[f];
            if (!fair) {
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
            } else {
                // class turns over the sources' heads: each pick takes the lowest
                // key of the class whose turn it is (of either class if none)
                // among requests with no request of the same source ahead of them
                // at this link, and hands the turn to the other class
                uint32_t *aux = req_aux + d.req_off[f];
                auto cls_of = [&](uint32_t sk) -> uint32_t {
                    return lcls ? (uint32_t)lcls[sreq_x[(size_t)(sk >> 8) * bmax + (sk & 255u)]] : 0u;
                };
                for (uint32_t i = 0; i < c; i++) {
                    const uint32_t si = (uint32_t)rec[i];
                    uint32_t ahead = 0;
                    for (uint32_t jj = 0; jj < c; jj++) {
                        const uint32_t sj = (uint32_t)rec[jj];
                        ahead += ((sj >> 8) == (si >> 8) && (sj & 255u) < (si & 255u)) ? 1u : 0u;
                    }
                    aux[i] = ahead;
                }
                uint32_t turn = cptr[f];
                for (int pos = 0; pos < g; pos++) {
                    int best = -1, any = -1;
                    uint32_t kb = 0xFFFFFFFFu, ka = 0xFFFFFFFFu;
                    for (uint32_t i = 0; i < c; i++) {
                        if (aux[i] != 0u) continue;  // picked (all ones) or not yet its source's head
                        const uint32_t ki = (uint32_t)(rec[i] >> 32);
                        if (ki < ka) { ka = ki; any = (int)i; }
                        if (ki < kb && cls_of((uint32_t)rec[i]) == turn) { kb = ki; best = (int)i; }
                    }
                    const int pi = best >= 0 ? best : any;
                    const uint32_t sk = (uint32_t)rec[pi];
                    aux[pi] = 0xFFFFFFFFu;
                    for (uint32_t i = 0; i < c; i++)  // the source's next request moves up
                        if (aux[i] != 0xFFFFFFFFu && ((uint32_t)rec[i] >> 8) == (sk >> 8)) aux[i] -= 1u;
                    glist[(size_t)f * bmax + pos] = sk;
                    grant[(size_t)(sk >> 8) * bmax + (sk & 255u)] = pos;
                    turn = 1u - cls_of(sk);
                }
            }
            gcount[f] = (uint32_t)(g > 0 ? g : 0);
        }
        __syncthreads();
        // ---------------------------------------------------------------- D
        for (int a = tid; a < nsrc_now; a += kThreads) {
            const int src = ACT ? alist[a] : (a < d.n_fsrc ? d.fsrc_link[a] : m + (a - d.n_fsrc));
            const int nr = sreq_n[src];
            if (nr == 0) continue;
            sreq_n[src] = 0;
            // the longest granted prefix departs; every grant slot is reset
            int dep = 0, sinks = 0;
            bool open = true;
            for (int k0 = 0; k0 < nr; k0 += kC) {
                const size_t s0 = (size_t)src * bmax + k0;
                int gr[kC], pv[kC];
                uint32_t xs[kC];
#pragma unroll
                for (int u = 0; u < kC; u++) gr[u] = k0 + u < nr ? grant[s0 + u] : -1;
#pragma unroll
                for (int u = 0; u < kC; u++) {
                    if (k0 + u < nr) grant[s0 + u] = -1;
                    open = open && gr[u] != -1;
                    gr[u] = open ? gr[u] : -1;  // -1: stays
                }
#pragma unroll
                for (int u = 0; u < kC; u++)
                    if (gr[u] != -1) pv[u] = sreq_pp[s0 + u];
#pragma unroll
                for (int u = 0; u < kC; u++)
                    if (gr[u] != -1) pv[u] = path[pv[u]];
#pragma unroll
                for (int u = 0; u < kC; u++)
                    if (gr[u] == -2) xs[u] = sreq_x[s0 + u];
#pragma unroll
                for (int u = 0; u < kC; u++) {
                    if (gr[u] == -1) continue;
                    dep++;
                    if (gr[u] == -2) {
                        comp[xs[u]] = t + 1;
                        atomicAdd(&delivered[-pv[u] - 1], 1u);
                        sinks++;
                        if constexpr (ACT)
                            for (int q = d.fw_ptr[-pv[u] - 1]; q < d.fw_ptr[-pv[u]]; q++) set_live(m + d.fw_str[q]);
                    } else {
                        gdep[(size_t)pv[u] * bmax + gr[u]] = 1;
                    }
                }
                if (!open) {  // the rest stays; reset its grant slots
                    for (int k = k0 + kC; k < nr; k++) grant[(size_t)src * bmax + k] = -1;
                    break;
                }
            }
            if (dep) {
                sh_anydep = 1;
                if (src < m) {
                    if (cred) {  // a left entry keeps its slot until its credit is back
                        const int base = d.fifo_off[src], mask = d.fifo_mask[src];
                        for (int k = 0; k < dep; k++) frdy[base + (int)((qhead[src] + (uint32_t)k) & (uint32_t)mask)] = t;
                    }
                    qhead[src] += (uint32_t)dep;
                    // emptied (left entries that still owe a credit keep it live)
                    if (ACT && !cred && qhead[src] == qtail[src]) clear_live(src);
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
                    if (ACT && R == d.s_rend[j]) clear_live(src);
                }
                if (sinks) atomicAdd(&sh_ndone, (uint32_t)sinks);
            }
        }
        __syncthreads();
        // ---------------------------------------------------------------- E
        for (int a = tid; a < ntgt; a += kThreads) {
            const int f = ACT ? tlist[a] : d.fsrc_link[a];
            if (flat) req_cnt[f] = 0;  // every request of the cycle has been ranked
            const int g = (int)gcount[f];
            if (g == 0) continue;
            gcount[f] = 0;
            const uint32_t P = (uint32_t)d.nports_tail[f];
            uint32_t tl = qtail[f];
            const int base = d.fifo_off[f], mask = d.fifo_mask[f];
            const uint32_t ready = t + (uint32_t)lat[f];
            // the departed grants in rank order, kC at a time
            int cnt = 0, last_src = 0;
            uint32_t last_x = 0;
            for (int r0 = 0; r0 < g; r0 += kC) {
                const size_t g0 = (size_t)f * bmax + r0;
                bool gd[kC];
                uint32_t sk[kC], sx[kC];
                int sp[kC];
#pragma unroll
                for (int u = 0; u < kC; u++) gd[u] = r0 + u < g && gdep[g0 + u] != 0;
#pragma unroll
                for (int u = 0; u < kC; u++)
                    if (gd[u]) {
                        gdep[g0 + u] = 0;
                        sk[u] = glist[g0 + u];
                    }
#pragma unroll
                for (int u = 0; u < kC; u++)
                    if (gd[u]) {
                        const size_t si = (size_t)(sk[u] >> 8) * bmax + (sk[u] & 255u);
                        sx[u] = sreq_x[si];
                        sp[u] = sreq_pp[si];
                    }
#pragma unroll
                for (int u = 0; u < kC; u++) {
                    if (!gd[u]) continue;
                    const int e = base + (int)(tl & (uint32_t)mask);
                    fx[e] = sx[u];
                    frdy[e] = ready;
                    fpp[e] = sp[u];
                    last_x = sx[u];
                    last_src = (int)(sk[u] >> 8);
                    tl++;
                    cnt++;
                }
            }
            if (cnt) {
                if (ACT) set_live(f);
                qtail[f] = tl;
                tx[f] += (uint64_t)cnt;
                busy[f] += 1;
                if (d.arb & 1) {
                    const uint32_t last_port = last_src < m ? (uint32_t)d.port_at_head[last_src] : P - 1;
                    rr[f] = (last_port + 1) % P;
                }
                if (fair) cptr[f] = 1u - (lcls ? (uint32_t)lcls[last_x] : 0u);
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
            sh_nalive = 0;
            sh_ntgt = 0;
            sh_nreq = 0;
            sh_nspill = 0;
        }
        __syncthreads();
    }
    if (tid == 0) {
        if (d.T == 0) d.makespan[s] = 0;
        d.status[s] = sh_state;
        d.cycles[s] = processed;
    }
}

}  // namespace

template <bool ACT, int NT>
hipError_t launch_wg2(const DevNet &d, hipStream_t st) {
    const int lds = d.wg_lds + (ACT ? d.wg_act : 0);
    auto k = d.wg_lds > 0 ? engine_wg<true, ACT, NT> : engine_wg<false, ACT, NT>;
    if (lds > 65536) (void)hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    hipLaunchKernelGGL(k, dim3((unsigned)d.S), dim3(NT), (unsigned)lds, st, d);
    return hipGetLastError();
}

template <int NT>
hipError_t launch_wg(const DevNet &d, hipStream_t st) {
    return d.wg_act > 0 ? launch_wg2<true, NT>(d, st) : launch_wg2<false, NT>(d, st);
}

hipError_t launch_workgroup(const DevNet &d, hipStream_t st) {
    const int per_cu = (d.S + 255) / 256;  // workgroups per CU when all are resident
    if (per_cu <= 1) return launch_wg<1024>(d, st);
    if (per_cu <= 2) return launch_wg<512>(d, st);
    return launch_wg<256>(d, st);
}

}  // namespace simgpu
