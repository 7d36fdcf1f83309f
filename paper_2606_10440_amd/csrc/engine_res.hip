// Device engine of libsimgpu for large graphs batched over many scenarios:
// the workgroup engine's phases with a scenario's per-link state, its link
// parameters and the cycle's requests resident in LDS.
//
// One workgroup owns one scenario and runs it to completion in one launch.
// LDS holds, per link: head and tail positions (with credit delays also the
// credit position) as 16-bit counters over rings of at most 2^15 entries,
// the number of requests received this cycle, bandwidth, capacity, latency,
// the round-robin pointer and input-port count, and this cycle's target-list
// index and grant count; per source: where its block of request records
// starts and how many of them depart; per stream: its cursor, link and last
// range; the active sets (a live-source bitmap and the cycle's source and
// target lists); per target of the cycle: its index segment, its tail at the
// cycle's start and the mask of departing grant ranks; the cycle's request
// records (line, path index, key, target and slot, source, input port,
// grant rank) and the grant step's two index lists.  Records, index entries
// and per-target words past their LDS capacity go to a per-scenario
// overflow area in HBM.  FIFO entries stay in HBM, one 16-byte record
// {line, ready cycle, path index} each.
//
// A cycle, each step ended by a workgroup barrier:
//   A   thread 0 advances the clock past the previous cycle while every
//       thread compacts the live-source bitmap into the source list;
//   R   every listed source reserves a contiguous block of request records
//       and fills it (FIFO links on the first half of the waves, streams on
//       the second).  A FIFO link offers its ready heads (ready times never
//       decrease along a FIFO, so the ready heads are a prefix and each
//       chunk of heads can be tested alone): the first chunk inline, the
//       later ones through a spill list, one chunk per thread after a
//       barrier.  A stream offers its released lines: each window of its
//       next ranges is checked by its own thread (lines released in order
//       from the window's start, and whether all are), and after the
//       barrier the stream adds the windows up to the first one held back,
//       reserves, and writes its records in a second walk;
//   G0  every target that received requests gets a segment of the sorted
//       index list and its grant count g = min(b, free slots, requests);
//   G1  every request drops its record index into its target's segment;
//   G2  every request ranks itself by the keys in its segment (keys are
//       distinct per target) and, with rank r < g, takes grant rank r; one
//       left without a grant cuts its source's departing count to its own
//       index (the source's longest granted prefix departs);
//   D   one request per thread: it departs if its index is below its
//       source's count; a line leaving its last hop completes (cycle + 1)
//       and bumps its flow's delivered count, any other sets its rank's bit
//       in its target's mask; a source's first request moves the source on;
//   E   one request per thread: a departing grant enters its target's FIFO
//       (ready = cycle + L) at the tail the cycle started with plus the
//       number of departing grants ranked before it; per target, the tail,
//       the link counters and the round-robin pointer move on.
// The time advance is the workgroup engine's: the next cycle is t + 1 if
// anything departed, else the earliest FIFO-head ready time or credit
// return, else the scenario has deadlocked.
#include <hip/hip_runtime.h>

#include "sim_internal.h"

namespace simgpu {

namespace {

constexpr int kC = 4;                        // FIFO heads per chunk (loads in flight together)
constexpr int kW = kResWindow;               // stream ranges per window
constexpr int kE = 6;                        // predecessor descriptors per load batch
constexpr uint32_t kNoSpill = 0xFFFFFFFFu;   // spill entry that holds no chunk
// rts (target << 16 | slot) of records that no target ranks
constexpr uint32_t kTsSink = 0xFFFFFFFFu;    // leaves the network: the sink takes it
constexpr uint32_t kTsHole = 0xFFFFFFFEu;    // reserved for a head that was not ready
// rg: grant rank (< 64)
constexpr uint16_t kNoGrant = 0xFFFFu;
constexpr uint16_t kSinkGrant = 0x7FFFu;

// A record field: entries below cap in LDS, the rest in HBM.
template <typename T>
struct Split {
    T *lds;
    T *hbm;  // entry q >= cap at hbm[q - cap]
    uint32_t cap;
    __device__ __forceinline__ T &operator[](uint32_t q) const { return q < cap ? lds[q] : hbm[q - cap]; }
};

// FAIR: class-fair arbitration (control and data lines take turns at a
// link), picked target by target instead of ranked request by request.
template <int ARB, bool CR, bool FAIR, int kThreads>
__global__ void __launch_bounds__(kThreads, 4) engine_res(DevNet d) {
    extern __shared__ __align__(16) unsigned char res_lds[];
    const int s = blockIdx.x;
    const int tid = threadIdx.x;
    const int m = d.m;
    const int ns = d.ns;
    const int nsrc = m + ns;
    const size_t sm = (size_t)s * m;
    const int32_t *__restrict__ path = d.path_link;

    uint16_t *qh = reinterpret_cast<uint16_t *>(res_lds + d.wr_off[0]);
    uint16_t *qt = reinterpret_cast<uint16_t *>(res_lds + d.wr_off[1]);
    uint16_t *qc = reinterpret_cast<uint16_t *>(res_lds + d.wr_off[2]);   // CR
    uint32_t *rqw = reinterpret_cast<uint32_t *>(res_lds + d.wr_off[3]);  // two 16-bit counts per word
    uint16_t *rq = reinterpret_cast<uint16_t *>(rqw);
    uint32_t *kg = reinterpret_cast<uint32_t *>(res_lds + d.wr_off[4]);   // target-list index | g << 24
    uint8_t *bwl = res_lds + d.wr_off[5];
    uint8_t *rrl = res_lds + d.wr_off[6];                                  // ARB == 1
    uint8_t *npl = res_lds + d.wr_off[18];                                 // ARB == 1: input ports at the tail
    uint16_t *sres = reinterpret_cast<uint16_t *>(res_lds + d.wr_off[19]); // stream window checks
    const int nwin = d.wr_nw;                                              // windows per stream
    uint16_t *capl = reinterpret_cast<uint16_t *>(res_lds + d.wr_off[7]);
    uint16_t *latl = reinterpret_cast<uint16_t *>(res_lds + d.wr_off[8]);
    uint16_t *crl = reinterpret_cast<uint16_t *>(res_lds + d.wr_off[9]);  // CR: credit delay
    uint32_t *sqn = reinterpret_cast<uint32_t *>(res_lds + d.wr_off[10]); // first record << 8 | count (departing, after G2)
    int32_t *cur_rng = reinterpret_cast<int32_t *>(res_lds + d.wr_off[11]);
    uint32_t *cur_off = reinterpret_cast<uint32_t *>(res_lds + d.wr_off[12]);
    int32_t *s_lnk = reinterpret_cast<int32_t *>(res_lds + d.wr_off[21]);  // a stream's link
    int32_t *s_end = reinterpret_cast<int32_t *>(res_lds + d.wr_off[22]);  // one past its last range
    uint8_t *cpl = res_lds + d.wr_off[23];  // FAIR: the class whose turn it is at each link
    const uint8_t *__restrict__ lcls = d.line_cls;  // FAIR: 1 control, 0 data (null: all data)
    uint32_t *livew = reinterpret_cast<uint32_t *>(res_lds + d.wr_off[13]);
    uint16_t *alist = reinterpret_cast<uint16_t *>(res_lds + d.wr_off[14]);
    uint16_t *tlist = reinterpret_cast<uint16_t *>(res_lds + d.wr_off[15]);
    uint32_t *spill = reinterpret_cast<uint32_t *>(res_lds + d.wr_off[16]);
    const uint32_t rcap = (uint32_t)d.wr_rcap;
    const uint32_t scap = (uint32_t)d.wr_scap;
    const size_t ov = (size_t)s * d.wr_ovf;
    unsigned char *rb = res_lds + d.wr_off[17];
    const Split<uint32_t> rx{reinterpret_cast<uint32_t *>(rb), d.wr_ox + ov, rcap};
    const Split<int32_t> rpp{reinterpret_cast<int32_t *>(rb + 4 * rcap), d.wr_opp + ov, rcap};
    const Split<uint32_t> rkey{reinterpret_cast<uint32_t *>(rb + 8 * rcap), d.wr_okey + ov, rcap};
    const Split<uint32_t> rts{reinterpret_cast<uint32_t *>(rb + 12 * rcap), d.wr_ots + ov, rcap};
    const Split<uint32_t> sidx{reinterpret_cast<uint32_t *>(rb + 16 * rcap), d.wr_osidx + ov, rcap};
    const Split<uint32_t> gl{reinterpret_cast<uint32_t *>(rb + 20 * rcap), d.wr_ogl + ov, rcap};
    const Split<uint16_t> rport{reinterpret_cast<uint16_t *>(rb + 24 * rcap), d.wr_osrc + ov, rcap};  // ARB == 1
    const Split<uint16_t> rg{reinterpret_cast<uint16_t *>(rb + 26 * rcap), d.wr_og + ov, rcap};
    const Split<uint16_t> rsrc{reinterpret_cast<uint16_t *>(rb + 28 * rcap), d.wr_osrcid + ov, rcap};
    // FAIR: a request's count of requests of its source ahead of it at its target
    const Split<uint16_t> raux{reinterpret_cast<uint16_t *>(rb + 30 * rcap), d.wr_oaux + ov, rcap};
    // per target of the cycle (index in the target list): its segment, its
    // tail at the cycle's start, and the grant ranks that depart
    const uint32_t tcap = (uint32_t)d.wr_tcap;
    const size_t tov = (size_t)s * d.wr_tovf;
    unsigned char *tb = res_lds + d.wr_off[20];
    const Split<unsigned long long> tmask{reinterpret_cast<unsigned long long *>(tb), d.wr_otmask + tov, tcap};
    const Split<uint32_t> tseg{reinterpret_cast<uint32_t *>(tb + 8 * tcap), d.wr_otseg + tov, tcap};
    const Split<uint16_t> tq{reinterpret_cast<uint16_t *>(tb + 12 * tcap), d.wr_otq + tov, tcap};

    uint4 *frec = d.wr_frec + (size_t)s * d.fifo_total;
    uint32_t *delivered = d.delivered + (size_t)s * d.nflows;
    uint32_t *comp = d.completion + (size_t)s * d.T;
    uint64_t *tx = d.tx_lines + sm;
    uint64_t *busy = d.busy + sm;

    __shared__ uint32_t sh_t, sh_next, sh_anydep, sh_ndone, sh_nalive, sh_nalive_s, sh_ntgt, sh_nreq, sh_nspill, sh_koff;
    __shared__ int32_t sh_state;
    const int nw = (nsrc + 31) / 32;
    auto set_live = [&](int src) { atomicOr(&livew[src >> 5], 1u << (src & 31)); };
    auto clear_live = [&](int src) { atomicAnd(&livew[src >> 5], ~(1u << (src & 31))); };
    // n requests to target f: their first slot (16-bit count inside a 32-bit word)
    auto take_slots = [&](int f, uint32_t n) -> uint32_t {
        const uint32_t sh = 16u * (uint32_t)(f & 1);
        return (atomicAdd(&rqw[f >> 1], n << sh) >> sh) & 0xFFFFu;
    };

    for (int l = tid; l < m; l += kThreads) {
        qh[l] = 0;
        qt[l] = 0;
        if (CR) {
            qc[l] = 0;
            crl[l] = (uint16_t)d.credit[sm + l];
        }
        rq[l] = 0;
        kg[l] = 0;
        bwl[l] = (uint8_t)d.bw[sm + l];
        if (ARB == 1) {
            rrl[l] = 0;
            npl[l] = (uint8_t)d.nports_tail[l];
        }
        if (FAIR) cpl[l] = 0;
        capl[l] = (uint16_t)d.cap[sm + l];
        latl[l] = (uint16_t)d.lat[sm + l];
        tx[l] = 0;
        busy[l] = 0;
    }
    for (int i = tid; i < nsrc; i += kThreads) sqn[i] = 0;
    for (int j = tid; j < ns; j += kThreads) {
        cur_rng[j] = d.s_rbeg[j];
        cur_off[j] = 0;
        s_lnk[j] = d.s_link[j];
        s_end[j] = d.s_rend[j];
    }
    for (int f = tid; f < d.nflows; f += kThreads) delivered[f] = 0;
    for (int j = tid; j < nw; j += kThreads) livew[j] = 0;
    if (tid == 0) {
        sh_t = 0;
        sh_state = d.T > 0 ? kRunRunning : kRunOk;
        sh_next = kNever;
        sh_anydep = 0;
        sh_ndone = 0;
        sh_nalive = 0;
        sh_nalive_s = 0;
        sh_ntgt = 0;
        sh_nreq = 0;
        sh_nspill = 0;
        sh_koff = 0;
    }
    __syncthreads();
    for (int j = tid; j < ns; j += kThreads)  // streams with lines are live from the start
        if (d.s_rbeg[j] < d.s_rend[j]) set_live(m + j);
    __syncthreads();

    uint64_t done = 0, processed = 0;  // meaningful in thread 0
    uint32_t t = 0;
    for (bool started = false;; started = true) {
        // ------------------------------------------------------- time and A
        // thread 0 advances the clock past the cycle just processed while
        // every thread compacts the live sources of the next one
        if (tid == 0 && started) {
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
            sh_ntgt = 0;
            sh_nreq = 0;
            sh_nspill = 0;
            sh_koff = 0;
        }
        // one source per thread: live FIFO links from the front of the list,
        // live streams from its back (a slot is a wave-wide count of one per
        // live lane)
        for (int i = tid; i < nsrc; i += kThreads)
            if ((livew[i >> 5] >> (i & 31)) & 1u) {
                if (i < m) alist[atomicAdd(&sh_nalive, 1u)] = (uint16_t)i;
                else alist[nsrc - 1 - (int)atomicAdd(&sh_nalive_s, 1u)] = (uint16_t)i;
            }
        __syncthreads();
        if (sh_state != kRunRunning) break;
        t = sh_t;
        // FIFO links and streams take different code paths: the first half of
        // the workgroup's waves walks the links, the second half the streams
        const int nfl = (int)sh_nalive, nst = (int)sh_nalive_s;
        constexpr int kF = kThreads / 2;
        const bool fside = tid < kF;
        const int a0 = fside ? tid : tid - kF;
        // ---------------------------------------------------------------- R
        // Heads k0 .. k0 + kC - 1 (below lim) of FIFO link l with head
        // position h: their entries, and how many of them are ready (the
        // first that is not offers its ready time as the next event).
        auto load_heads = [&](int l, uint32_t h, int k0, int lim, uint4 *e) -> int {
            const int base = d.fifo_off[l], mask = d.fifo_mask[l];
#pragma unroll
            for (int u = 0; u < kC; u++)
                if (k0 + u < lim) e[u] = frec[base + (int)((h + (uint32_t)(k0 + u)) & (uint32_t)mask)];
            int nrd = 0;
            bool run = true;
#pragma unroll
            for (int u = 0; u < kC; u++) {
                if (run && k0 + u < lim && e[u].y > t) atomicMin(&sh_next, e[u].y);  // first head not ready
                run = run && k0 + u < lim && e[u].y <= t;
                nrd += run ? 1 : 0;
            }
            return nrd;
        };
        // Records q0 + k0 + u of those heads: requests for u < nrd, holes for
        // nrd <= u < nfill.
        auto post_heads = [&](int l, int k0, int nrd, int nfill, const uint4 *e, uint32_t q0) {
            int tg[kC];
#pragma unroll
            for (int u = 0; u < kC; u++)
                if (u < nrd) tg[u] = path[(int)e[u].z + 1];
            uint32_t P[kC];
            if (ARB == 1) {
#pragma unroll
                for (int u = 0; u < kC; u++)
                    if (u < nrd && tg[u] >= 0) P[u] = (uint32_t)npl[tg[u]];
            }
            const uint32_t ph = ARB == 1 ? (uint32_t)d.port_at_head[l] : 0u;
#pragma unroll
            for (int u = 0; u < kC; u++) {
                const int k = k0 + u;
                const uint32_t q = q0 + (uint32_t)k;
                if (u >= nrd) {
                    if (u < nfill) rts[q] = kTsHole;
                    continue;
                }
                rx[q] = e[u].x;
                rsrc[q] = (uint16_t)l;
                if (ARB == 1) rport[q] = (uint16_t)ph;
                if (tg[u] < 0) {  // the sink takes everything
                    rpp[q] = -tg[u] - 1;  // the flow
                    rts[q] = kTsSink;
                    rg[q] = kSinkGrant;
                } else {
                    rpp[q] = (int)e[u].z + 1;
                    uint32_t key;
                    if (ARB == 0) {
                        key = e[u].x;
                    } else {
                        const uint32_t rot = (ph + P[u] - (uint32_t)rrl[tg[u]]) % P[u];
                        key = (uint32_t)k * P[u] + rot;
                    }
                    rkey[q] = key;
                    const uint32_t slot = take_slots(tg[u], 1u);
                    rts[q] = ((uint32_t)tg[u] << 16) | slot;
                    if (slot == 0u) tlist[atomicAdd(&sh_ntgt, 1u)] = (uint16_t)tg[u];
                }
            }
        };
        if (fside) {
            for (int a = a0; a < nfl; a += kF) {
                const int sid = (int)alist[a];
                const int l = sid;
                    const uint32_t h = qh[l];
                    const uint32_t occ = (uint16_t)(qt[l] - h);
                    const int b = bwl[l];
                    if (CR) {
                        // slots of lines that left at least credit cycles ago are free
                        // again; the next return is an event of the time advance
                        const int base = d.fifo_off[l], mask = d.fifo_mask[l];
                        const uint32_t D = crl[l];
                        uint32_t c = qc[l];
                        while ((uint16_t)c != (uint16_t)h && frec[base + (int)(c & (uint32_t)mask)].y + D <= t) c++;
                        qc[l] = (uint16_t)c;
                        if ((uint16_t)c != (uint16_t)h) atomicMin(&sh_next, frec[base + (int)(c & (uint32_t)mask)].y + D);
                        if ((uint16_t)c == qt[l]) clear_live(l);  // nothing held: every credit is back
                    }
                    const int lim = b < (int)occ ? b : (int)occ;
                    if (lim == 0) {
                        sqn[l] = 0;
                        continue;
                    }
                    // the first chunk's readiness decides the reservation: its ready
                    // heads, or (all of it ready) every head up to lim
                    uint4 e[kC];
                    const int nrd0 = load_heads(l, h, 0, lim, e);
                    const bool more = nrd0 == kC && lim > kC;
                    const uint32_t nres = more ? (uint32_t)lim : (uint32_t)nrd0;
                    const uint32_t q0 = nres ? atomicAdd(&sh_nreq, nres) : 0u;
                    post_heads(l, 0, nrd0, nrd0, e, q0);
                    int nr = nrd0;
                    if (more) {
                        const uint32_t nch = (uint32_t)((lim - 1) / kC);
                        const uint32_t s0 = atomicAdd(&sh_nspill, nch);
                        if (s0 + nch <= scap) {
                            for (uint32_t c = 0; c < nch; c++) spill[s0 + c] = ((uint32_t)l << 8) | (uint32_t)(kC * (c + 1));
                        } else {  // the list is full: the later chunks inline
                            for (uint32_t c = 0; s0 + c < scap && c < nch; c++) spill[s0 + c] = kNoSpill;
                            bool open = true;
                            for (int k0 = kC; k0 < lim; k0 += kC) {
                                const int nfill = lim - k0 < kC ? lim - k0 : kC;
                                int n = 0;
                                if (open) {
                                    uint4 e2[kC];
                                    n = load_heads(l, h, k0, lim, e2);
                                    post_heads(l, k0, n, nfill, e2, q0);
                                } else {  // past the first head that is not ready
                                    for (int u = 0; u < nfill; u++) rts[q0 + (uint32_t)(k0 + u)] = kTsHole;
                                }
                                nr += n;
                                open = n == kC;
                            }
                        }
                    }
                    sqn[l] = (q0 << 8) | (uint32_t)nr;
            }
        } else {
            // stream windows: window w of a live stream is its ranges
            // R0 + w kW ... (at most kW, the first from the cursor's offset);
            // each is checked by its own thread: how many lines from its
            // start are released in order (capped at b), and whether all are
            for (int i = a0; i < nst * nwin; i += kThreads - kF) {
                const int a = i / nwin, w = i - a * nwin;
                const int j = (int)alist[nsrc - 1 - a] - m;
                const int f = s_lnk[j];
                const int rend = s_end[j];
                const int b = bwl[f];
                const int Rw = cur_rng[j] + w * kW;
                uint32_t res = 0;
                if (Rw < rend && w * kW < b) {
                    const int nwr = rend - Rw < kW ? rend - Rw : kW;
                    const uint32_t ow = w == 0 ? cur_off[j] : 0u;
                    uint32_t len[kW];
                    int pb[kW], pe[kW];  // descriptor spans (repeated ones shared)
#pragma unroll
                    for (int u = 0; u < kW; u++)
                        if (u < nwr) {
                            len[u] = d.r_len[Rw + u];
                            pb[u] = d.wr_rpb[Rw + u];
                            pe[u] = d.wr_rpe[Rw + u];
                        }
                    int qend = pe[0];  // spans never go back: the window's are [pb[0], qend)
#pragma unroll
                    for (int u = 1; u < kW; u++) {
                        if (u < nwr) qend = pe[u];
                        else pb[u] = pe[u] = qend;
                    }
                    // allowance per range: lines ow + i (first range) or i with
                    // delivered > base + i (per line) or > base (per chunk)
                    uint32_t A[kW];
#pragma unroll
                    for (int u = 0; u < kW; u++) A[u] = 0xFFFFFFFFu;
                    // a window held back at its first line (the usual case) stops
                    // after the batch that holds the first range's descriptors
                    const int qe0 = qend - pb[0] < kE ? qend : pb[0] + kE;
                    for (int q0 = pb[0], qe = qe0; q0 < qend; q0 = qe, qe = qend - qe < kE ? qend : qe + kE) {
                        int fl[kE];
                        uint32_t bs[kE], dv[kE];
#pragma unroll
                        for (int v = 0; v < kE; v++)
                            if (q0 + v < qe) {
                                fl[v] = d.wr_pdf[q0 + v];
                                bs[v] = d.wr_pdb[q0 + v];
                            }
#pragma unroll
                        for (int v = 0; v < kE; v++)
                            if (q0 + v < qe) dv[v] = delivered[fl[v]];
#pragma unroll
                        for (int v = 0; v < kE; v++) {
                            const int q = q0 + v;
                            if (q >= qe) continue;
                            const uint32_t b0 = bs[v] + (ow & d.pd_omask);
                            const uint32_t al0 = dv[v] > b0 ? (d.pd_omask ? dv[v] - b0 : 0xFFFFFFFFu) : 0u;
                            const uint32_t al1 = dv[v] > bs[v] ? (d.pd_omask ? dv[v] - bs[v] : 0xFFFFFFFFu) : 0u;
#pragma unroll
                            for (int u = 0; u < kW; u++) {
                                const uint32_t al = u == 0 ? al0 : al1;
                                if (q >= pb[u] && q < pe[u]) A[u] = A[u] < al ? A[u] : al;
                            }
                        }
                        if (q0 == pb[0] && qe >= pe[0]) {  // the first range is known: taken whole?
                            const uint32_t need = (uint32_t)b < len[0] - ow ? (uint32_t)b : len[0] - ow;
                            if (A[0] < need) break;
                        }
                    }
                    uint32_t cnt = 0;
                    bool whole = true;
#pragma unroll
                    for (int u = 0; u < kW; u++) {
                        if (u >= nwr || !whole || cnt >= (uint32_t)b) continue;
                        const uint32_t off = u == 0 ? ow : 0u;
                        const uint32_t n = len[u] - off < A[u] ? len[u] - off : A[u];
                        cnt += n;
                        if (n == 0u || n < len[u] - off) whole = false;  // held back by a predecessor
                    }
                    res = (cnt < (uint32_t)b ? cnt : (uint32_t)b) | (whole ? 0x8000u : 0u);
                }
                sres[i] = (uint16_t)res;
            }
        }
        __syncthreads();
        if (fside) {  // the spilled chunks of long FIFO offers
            const uint32_t nsp = sh_nspill < scap ? sh_nspill : scap;
            for (uint32_t i = (uint32_t)a0; i < nsp; i += kF) {
                const uint32_t v = spill[i];
                if (v == kNoSpill) continue;
                const int l = (int)(v >> 8), k0 = (int)(v & 255u);
                const uint32_t h = qh[l];
                const uint32_t occ = (uint16_t)(qt[l] - h);
                const int b = bwl[l];
                const int lim = b < (int)occ ? b : (int)occ;
                const uint32_t q0 = sqn[l] >> 8;
                uint4 e[kC];
                const int n = load_heads(l, h, k0, lim, e);
                post_heads(l, k0, n, lim - k0 < kC ? lim - k0 : kC, e, q0);
                if (n) atomicMax(&sqn[l], (q0 << 8) | (uint32_t)(k0 + n));
            }
        } else {  // streams: their windows combined, records reserved and written
            for (int a = a0; a < nst; a += kThreads - kF) {
                const int src = (int)alist[nsrc - 1 - a];
                const int j = src - m;
                const int f = s_lnk[j];
                const int R0 = cur_rng[j];
                const uint32_t o0 = cur_off[j];
                const int rend = s_end[j];
                const int b = bwl[f];
                int cnt = 0;
                for (int w = 0; w < nwin && w * kW < b && R0 + w * kW < rend; w++) {
                    const uint32_t v = sres[a * nwin + w];
                    cnt += (int)(v & 0x7FFFu);
                    if (cnt >= b || (v & 0x8000u) == 0u) break;
                }
                if (cnt > b) cnt = b;
                if (cnt == 0) {
                    clear_live(src);  // done, or asleep until a flow it waits on delivers
                    sqn[src] = 0;
                    continue;
                }
                int R;
                uint32_t o;
                // reserve and write: the same walk takes whole ranges until cnt lines
                const uint32_t q0 = atomicAdd(&sh_nreq, (uint32_t)cnt);
                const uint32_t slot0 = take_slots(f, (uint32_t)cnt);
                if (slot0 == 0u) tlist[atomicAdd(&sh_ntgt, 1u)] = (uint16_t)f;
                uint32_t rot = 0;
                uint32_t P = 1;
                if (ARB == 1) {
                    P = (uint32_t)npl[f];
                    rot = ((P - 1u) + P - (uint32_t)rrl[f]) % P;  // a stream is the link's last port
                }
                R = R0;
                o = o0;
                int k = 0;
                while (k < cnt && R < rend) {
                    const int nwr = rend - R < kW ? rend - R : kW;
                    uint32_t len[kW], st[kW];
                    int rp[kW];
#pragma unroll
                    for (int u = 0; u < kW; u++)
                        if (u < nwr) {
                            len[u] = d.r_len[R + u];
                            st[u] = d.r_start[R + u];
                            rp[u] = d.r_path[R + u];
                        }
#pragma unroll
                    for (int u = 0; u < kW; u++) {
                        if (u >= nwr || k >= cnt) continue;
                        const uint32_t off = u == 0 ? o : 0u;
                        const uint32_t n = (uint32_t)(cnt - k) < len[u] - off ? (uint32_t)(cnt - k) : len[u] - off;
                        for (uint32_t i = 0; i < n; i++) {
                            const uint32_t q = q0 + (uint32_t)k + i;
                            const uint32_t x = st[u] + off + i;
                            rx[q] = x;
                            rsrc[q] = (uint16_t)src;
                            rpp[q] = rp[u];
                            if (ARB == 1) rport[q] = (uint16_t)(P - 1u);
                            rkey[q] = ARB == 0 ? x : ((uint32_t)k + i) * P + rot;
                            rts[q] = ((uint32_t)f << 16) | (slot0 + (uint32_t)k + i);
                        }
                        k += (int)n;
                    }
                    R += nwr;
                    o = 0;
                }
                sqn[src] = (q0 << 8) | (uint32_t)cnt;
            }
        }
        __syncthreads();
        // ---------------------------------------------------------------- G
        const int ntgt = (int)sh_ntgt;
        const uint32_t nreq = sh_nreq;
        for (int a = tid; a < ntgt; a += kThreads) {  // G0: segments and grant counts
            const int f = (int)tlist[a];
            const uint32_t c = rq[f];
            const uint16_t tl = qt[f];
            const int occ = (int)(uint16_t)(tl - (CR ? qc[f] : qh[f]));
            int g = bwl[f];
            if ((int)capl[f] - occ < g) g = (int)capl[f] - occ;
            if ((int)c < g) g = (int)c;
            kg[f] = (uint32_t)a | ((uint32_t)(g > 0 ? g : 0) << 24);
            tseg[a] = atomicAdd(&sh_koff, c);
            tq[a] = tl;
            tmask[a] = 0ull;
        }
        __syncthreads();
        for (uint32_t q = (uint32_t)tid; q < nreq; q += kThreads) {  // G1: indices into the segments
            const uint32_t ts = rts[q];
            if (ts >= kTsHole) continue;
            sidx[tseg[kg[ts >> 16] & 0xFFFFFFu] + (ts & 0xFFFFu)] = q;
        }
        __syncthreads();
        // G2: ranks and grants; a request left without a grant cuts its
        // source's departing prefix there (the count in sqn drops to its index)
        if constexpr (FAIR) {
            // target by target, picks in turn: each takes, among the requests
            // with no request of the same source ahead of them at this link,
            // the lowest key of the class whose turn it is (of either class if
            // none), and hands the turn to the other class
            auto cls_of = [&](uint32_t q) -> uint32_t { return lcls ? (uint32_t)lcls[rx[q]] : 0u; };
            for (int a = tid; a < ntgt; a += kThreads) {
                const int f = (int)tlist[a];
                const uint32_t seg = tseg[a], g = kg[f] >> 24, c = rq[f];
                for (uint32_t i = 0; i < c; i++) {
                    const uint32_t qi = sidx[seg + i];
                    const uint16_t si = rsrc[qi];
                    uint32_t ahead = 0;
                    for (uint32_t jj = 0; jj < c; jj++) {
                        const uint32_t qj = sidx[seg + jj];
                        ahead += (rsrc[qj] == si && qj < qi) ? 1u : 0u;
                    }
                    raux[qi] = (uint16_t)ahead;
                }
                uint32_t turn = cpl[f];
                for (uint32_t pos = 0; pos < g; pos++) {
                    uint32_t best = 0xFFFFFFFFu, any = 0xFFFFFFFFu, kb = 0xFFFFFFFFu, ka = 0xFFFFFFFFu;
                    for (uint32_t i = 0; i < c; i++) {
                        const uint32_t qi = sidx[seg + i];
                        if (raux[qi] != 0u) continue;  // picked, or not yet its source's head
                        const uint32_t ki = rkey[qi];
                        if (ki < ka) {
                            ka = ki;
                            any = qi;
                        }
                        if (ki < kb && cls_of(qi) == turn) {
                            kb = ki;
                            best = qi;
                        }
                    }
                    const uint32_t qp = best != 0xFFFFFFFFu ? best : any;
                    raux[qp] = 0xFFFFu;
                    const uint16_t sp = rsrc[qp];
                    for (uint32_t i = 0; i < c; i++) {  // the source's next request moves up
                        const uint32_t qi = sidx[seg + i];
                        if (raux[qi] != 0xFFFFu && rsrc[qi] == sp) raux[qi] = (uint16_t)(raux[qi] - 1u);
                    }
                    gl[seg + pos] = qp;
                    rg[qp] = (uint16_t)pos;
                    turn = 1u - cls_of(qp);
                }
                for (uint32_t i = 0; i < c; i++) {  // the others get no grant
                    const uint32_t qi = sidx[seg + i];
                    if (raux[qi] == 0xFFFFu) continue;
                    rg[qi] = kNoGrant;
                    const int src = (int)rsrc[qi];
                    const uint32_t q0 = sqn[src] >> 8;
                    atomicMin(&sqn[src], (q0 << 8) | (qi - q0));
                }
            }
        } else
        for (uint32_t q = (uint32_t)tid; q < nreq; q += kThreads) {
            const uint32_t ts = rts[q];
            if (ts >= kTsHole) continue;
            const int f = (int)(ts >> 16);
            const uint32_t v = kg[f];
            const uint32_t seg = tseg[v & 0xFFFFFFu], g = v >> 24;
            const uint32_t c = rq[f];
            const uint32_t ki = rkey[q];
            uint32_t rank = 0;
            for (uint32_t jj = 0; jj < c; jj++) rank += rkey[sidx[seg + jj]] < ki ? 1u : 0u;
            if (rank < g) {
                gl[seg + rank] = q;
                rg[q] = (uint16_t)rank;
            } else {
                rg[q] = kNoGrant;
                const int src = (int)rsrc[q];
                const uint32_t q0 = sqn[src] >> 8;
                atomicMin(&sqn[src], (q0 << 8) | (q - q0));
            }
        }
        __syncthreads();
        // ---------------------------------------------------------------- D
        // one request per thread: those before the first without a grant
        // depart; the first request of a source moves the source on
        for (uint32_t q = (uint32_t)tid; q < nreq; q += kThreads) {
            const uint32_t ts = rts[q];
            if (ts == kTsHole) continue;
            const int src = (int)rsrc[q];
            const uint32_t v = sqn[src];
            const uint32_t q0 = v >> 8, dep = v & 255u, k = q - q0;
            if (k >= dep) continue;
            if (ts == kTsSink) {
                const int fl = rpp[q];
                comp[rx[q]] = t + 1;
                atomicAdd(&delivered[fl], 1u);
                atomicAdd(&sh_ndone, 1u);
                for (int w = d.fw_ptr[fl]; w < d.fw_ptr[fl + 1]; w++) set_live(m + d.fw_str[w]);
            } else {
                atomicOr(&tmask[kg[ts >> 16] & 0xFFFFFFu], 1ull << rg[q]);
            }
            if (k != 0u) continue;
            sh_anydep = 1;
            if (src < m) {
                const uint32_t h = qh[src];
                if (CR) {  // a left entry keeps its slot until its credit is back
                    const int base = d.fifo_off[src], mask = d.fifo_mask[src];
                    for (uint32_t i = 0; i < dep; i++) frec[base + (int)((h + i) & (uint32_t)mask)].y = t;
                }
                const uint16_t nh = (uint16_t)(h + dep);
                qh[src] = nh;
                if (!CR && nh == qt[src]) clear_live(src);  // emptied
            } else {
                const int j = src - m;
                int R = cur_rng[j];
                uint32_t o = cur_off[j] + dep;
                const int rend = s_end[j];
                bool go = R < rend;
                while (go) {  // past the ranges it finished, kW lengths read at a time
                    uint32_t len[kW];
#pragma unroll
                    for (int u = 0; u < kW; u++)
                        if (R + u < rend) len[u] = d.r_len[R + u];
#pragma unroll
                    for (int u = 0; u < kW; u++) {
                        if (!go) continue;
                        if (R < rend && o >= len[u]) {
                            o -= len[u];
                            R++;
                        } else {
                            go = false;
                        }
                    }
                    go = go && R < rend;
                }
                cur_rng[j] = R;
                cur_off[j] = o;
                if (R == rend) clear_live(src);
            }
        }
        __syncthreads();
        // ---------------------------------------------------------------- E
        // one request per thread: a departing grant of rank r enters its
        // target's FIFO at the tail the cycle started with plus the number of
        // departing grants ranked before it
        for (uint32_t q = (uint32_t)tid; q < nreq; q += kThreads) {
            const uint32_t ts = rts[q];
            if (ts >= kTsHole) continue;
            const uint16_t r = rg[q];
            if (r == kNoGrant) continue;
            const int f = (int)(ts >> 16);
            const uint32_t a = kg[f] & 0xFFFFFFu;
            const unsigned long long dm = tmask[a];
            if (((dm >> r) & 1ull) == 0ull) continue;
            const uint32_t pos = (uint32_t)__popcll(dm & ((1ull << r) - 1ull));
            const int base = d.fifo_off[f], mask = d.fifo_mask[f];
            frec[base + (int)(((uint32_t)tq[a] + pos) & (uint32_t)mask)] =
                make_uint4(rx[q], t + (uint32_t)latl[f], (uint32_t)rpp[q], 0u);
        }
        for (int a = tid; a < ntgt; a += kThreads) {  // and per target its tail and counters
            const int f = (int)tlist[a];
            rq[f] = 0;
            const unsigned long long dm = tmask[a];
            if (dm == 0ull) continue;
            const uint32_t cnt = (uint32_t)__popcll(dm);
            set_live(f);
            qt[f] = (uint16_t)(tq[a] + cnt);
            atomicAdd(&tx[f], (unsigned long long)cnt);  // no read back: the counters only grow
            atomicAdd(&busy[f], 1ull);
            if (ARB == 1) {  // past the port of the last line appended
                const uint32_t P = (uint32_t)npl[f];
                const uint32_t lp = rport[gl[tseg[a] + (63u - (uint32_t)__clzll(dm))]];
                rrl[f] = (uint8_t)((lp + 1u) % P);
            }
            if (FAIR) {  // the other class than the last line appended
                const uint32_t ql = gl[tseg[a] + (63u - (uint32_t)__clzll(dm))];
                cpl[f] = (uint8_t)(1u - (lcls ? (uint32_t)lcls[rx[ql]] : 0u));
            }
        }
        __syncthreads();
        if (tid == 0) {  // the compaction counts start over (read into registers above)
            sh_nalive = 0;
            sh_nalive_s = 0;
        }
        __syncthreads();
    }
    if (tid == 0) {
        if (d.T == 0) d.makespan[s] = 0;
        d.status[s] = sh_state;
        d.cycles[s] = processed;
    }
}

template <int ARB, bool CR, bool FAIR, int NT>
hipError_t launch_res3(const DevNet &d, hipStream_t st) {
    auto k = engine_res<ARB, CR, FAIR, NT>;
    if (d.lds_bytes > 65536)
        (void)hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize, d.lds_bytes);
    hipLaunchKernelGGL(k, dim3((unsigned)d.S), dim3(NT), (unsigned)d.lds_bytes, st, d);
    return hipGetLastError();
}

template <int ARB, bool CR, bool FAIR>
hipError_t launch_res2(const DevNet &d, hipStream_t st) {
    if (d.wr_threads >= 1024) return launch_res3<ARB, CR, FAIR, 1024>(d, st);
    if (d.wr_threads >= 512) return launch_res3<ARB, CR, FAIR, 512>(d, st);
    return launch_res3<ARB, CR, FAIR, 256>(d, st);
}

template <int ARB, bool CR>
hipError_t launch_res1(const DevNet &d, hipStream_t st) {
    return (d.arb & 2) ? launch_res2<ARB, CR, true>(d, st) : launch_res2<ARB, CR, false>(d, st);
}

}  // namespace

hipError_t launch_resident(const DevNet &d, hipStream_t st) {
    const bool cr = d.credit != nullptr;
    if (d.arb & 1) return cr ? launch_res1<1, true>(d, st) : launch_res1<1, false>(d, st);
    return cr ? launch_res1<0, true>(d, st) : launch_res1<0, false>(d, st);
}

}  // namespace simgpu
