// Device-wide engine of libsimgpu: one large topology (one scenario) run by
// many workgroups together (a cooperative launch, one workgroup per CU).
//
// The graph's nodes are split over the workgroups.  A workgroup owns, for
// each of its nodes,
//   the target side of the node's out-links: the requests for them, their
//   grants, their append counts, round-robin pointers and counters, and the
//   injection stream of an endpoint (its lines request the stream's first
//   link, an out-link of the endpoint);
//   the source side of the node's in-links: the FIFO heads, whose lines have
//   crossed the link and request their next link -- an out-link of the same
//   node -- or the sink.
// So every request of a cycle is made, ranked, granted and committed inside
// one workgroup, in LDS, exactly as the lane engine does for a whole graph.
// What crosses workgroups:
//   - a FIFO's entries {line, ready, path index}, written by the workgroup of
//     the link's tail when it appends and read by the workgroup of its head
//     (an entry appended at cycle t may leave at t + L >= t + 1);
//   - each FIFO's appended and popped counts, published every processed cycle
//     into the slot of the cycle's parity: the other side reads the slot of
//     the previous cycle, i.e. the values at the start of the current cycle
//     (the model's start-of-cycle snapshot), and never a slot being written;
//   - per-flow delivered counts (predecessor release), kept in LDS by the
//     workgroup where the flow ends and published into two slots tagged with
//     the first cycle they hold for, so a reader picks the newest slot whose
//     tag is not after its cycle;
//   - the next cycle: every workgroup offers t + 1 if any of its lines moved,
//     else its earliest future FIFO-head ready time; the minimum is taken at
//     a grid barrier, one per processed cycle.  The barrier's spin is
//     bounded: past the bound the kernel ends with the watchdog status.
// Every shared word is read and written with device-scope atomic accesses,
// and each workgroup waits for its stores before it arrives at the barrier,
// so the placement of the workgroups on the chip's dies does not matter for
// the result.  Entries a reader uses were written before the barrier that
// precedes its cycle: slot (head + q) is read only if head + q is below the
// appended count of the previous cycle, and the writer only fills slots at
// or beyond that count while the reader's entries stay in the ring (a ring
// holds at least cap entries and the writer respects cap).
#include <hip/hip_runtime.h>

#include "engine_common.h"

namespace simgpu {

namespace {

using namespace dev;

template <typename T>
__device__ __forceinline__ T ld_dev(T *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ void st_dev(T *p, T v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Spins of one barrier wait before the run is declared stuck (each spin is a
// device-scope load, well under a microsecond).
constexpr uint32_t kSpinLimit = 1u << 23;
// FIFO entries per in-link kept in LDS (line, ready, next hop, path index),
// fetched while the workgroup waits at the barrier.
constexpr int kCache = 4;
// A cached entry whose next hop is still to be looked up (in the next poll).
constexpr int32_t kUnresolved = INT32_MIN;
// Predecessor descriptors of a stream's current range kept in LDS (their
// delivered counts are read with the poll); more are read when needed.
constexpr int kPDesc = 2;

// Delivered count of flow f at cycle t from its two tagged slots.
__device__ __forceinline__ uint32_t deliv_at(unsigned long long *slots, int f, uint32_t t) {
    const unsigned long long a = ld_dev(&slots[2 * f]), b = ld_dev(&slots[2 * f + 1]);
    const uint32_t ta = (uint32_t)(a >> 32), tb = (uint32_t)(b >> 32);
    const bool ua = ta <= t, ub = tb <= t;
    if (ua && (!ub || ta >= tb)) return (uint32_t)a;
    return ub ? (uint32_t)b : 0u;
}

__global__ void grid_init(DevNet d) {
    const size_t i0 = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t step = (size_t)gridDim.x * blockDim.x;
    for (size_t j = i0; j < (size_t)4 * d.nl; j += step) d.gd_pub[j] = 0u;
    if (d.gd_tpub)  // tagged counts: no cycle's tag yet
        for (size_t j = i0; j < (size_t)4 * d.nl; j += step) d.gd_tpub[j] = 0xFFFFFFFFull << 32;
    for (size_t j = i0; j < (size_t)2 * d.nflows; j += step) d.gd_dslot[j] = 0ull;
    // [0..5] arrival words of three successive cycles (64 bits each), [6..8]
    // the earliest future ready time offered by workgroups that moved nothing
    if (i0 < 16) d.gd_sync[i0] = (i0 >= 6 && i0 <= 8) ? kNever : 0u;
    if (i0 == 0) {
        d.status[0] = kRunRunning;
        d.makespan[0] = 0;
        d.cycles[0] = 0;
    }
}

// Lines of a stream's current range that may be offered this cycle, from
// offset o on (predecessor release with the delivered counts as of cycle t).
template <bool PREDS>
__device__ __forceinline__ uint32_t stream_allow(const DevNet &d, int pd0, int pd1, uint32_t o, uint32_t t) {
    if (!PREDS) return 0xFFFFFFFFu;
    uint32_t lim = 0xFFFFFFFFu;
    for (int idx = pd0; idx < pd1; idx++) {
        const uint32_t c = deliv_at(d.gd_dslot, d.pd_flow[idx], t), base = d.pd_base[idx];
        if (c <= base) return 0u;  // not even the first line (or, per chunk, none)
        if (d.pd_omask) {          // per line: offsets below c - base
            const uint32_t m = c - base;
            if (m <= o) return 0u;
            lim = lim < m - o ? lim : m - o;
        }
    }
    return lim;
}

template <int ARB, bool PREDS>
__global__ void __launch_bounds__(1024) engine_grid(DevNet d) {
    extern __shared__ __align__(16) unsigned char smem[];
    if (blockIdx.x % (unsigned)d.gd_stride) return;
    const int w = (int)(blockIdx.x / (unsigned)d.gd_stride);
    if (w >= d.gd_nb) return;
    // wave 0 runs the barrier; the other threads own the lanes
    const int tid = threadIdx.x;
    const int lt = tid - 64, NL = (int)blockDim.x - 64;
    const int nl = d.nl, m = d.m, NB = d.gd_nb;
    const int BM = d.bm;
    const int sb = d.gd_sptr[w], ns = d.gd_sptr[w + 1] - sb;  // source sides
    const int tb = d.gd_tptr[w], nt = d.gd_tptr[w + 1] - tb;  // target sides
    const int nmax = ns > nt ? ns : nt;
    const int NS = d.gd_ns_max, NT = d.gd_nt_max;

    // ---- LDS (the host sizes it with the same list)
    size_t off = 0;
    auto carve = [&](size_t bytes) {
        unsigned char *p = smem + off;
        off = (off + bytes + 15) & ~(size_t)15;
        return p;
    };
    uint32_t *s_lane = (uint32_t *)carve(4 * NS), *s_b = (uint32_t *)carve(4 * NS), *s_L = (uint32_t *)carve(4 * NS);
    uint32_t *s_fb = (uint32_t *)carve(4 * NS), *s_fm = (uint32_t *)carve(4 * NS), *s_port = (uint32_t *)carve(4 * NS);
    uint32_t *s_head = (uint32_t *)carve(4 * NS), *s_tkn = (uint32_t *)carve(4 * NS), *s_tkp = (uint32_t *)carve(4 * NS);
    uint32_t *s_nc = (uint32_t *)carve(4 * NS), *s_nf = (uint32_t *)carve(4 * NS);
    uint32_t *s_cx = (uint32_t *)carve(4 * NS * kCache), *s_cr = (uint32_t *)carve(4 * NS * kCache);
    int32_t *s_ct = (int32_t *)carve(4 * NS * kCache);
    uint32_t *s_cp = (uint32_t *)carve(4 * NS * kCache);
    uint32_t *s_fx = (uint32_t *)carve(4 * NS * BM);
    int32_t *s_ftg = (int32_t *)carve(4 * NS * BM), *s_grant = (int32_t *)carve(4 * NS * BM);
    uint32_t *t_lane = (uint32_t *)carve(4 * NT), *t_link = (uint32_t *)carve(4 * NT), *t_b = (uint32_t *)carve(4 * NT);
    uint32_t *t_L = (uint32_t *)carve(4 * NT), *t_cap = (uint32_t *)carve(4 * NT), *t_P = (uint32_t *)carve(4 * NT);
    uint32_t *t_fb = (uint32_t *)carve(4 * NT), *t_fm = (uint32_t *)carve(4 * NT), *t_rqoff = (uint32_t *)carve(4 * NT);
    uint32_t *t_rqcap = (uint32_t *)carve(4 * NT);
    int32_t *t_srend = (int32_t *)carve(4 * NT);
    uint32_t *t_tail = (uint32_t *)carve(4 * NT), *t_khead = (uint32_t *)carve(4 * NT), *t_rr = (uint32_t *)carve(4 * NT);
    uint32_t *t_cnt = (uint32_t *)carve(4 * NT);
    int32_t *t_g = (int32_t *)carve(4 * NT);
    uint32_t *t_nsr = (uint32_t *)carve(4 * NT);
    int32_t *t_R = (int32_t *)carve(4 * NT);
    uint32_t *t_o = (uint32_t *)carve(4 * NT), *t_rs = (uint32_t *)carve(4 * NT), *t_rl = (uint32_t *)carve(4 * NT);
    int32_t *t_rp = (int32_t *)carve(4 * NT), *t_pd0 = (int32_t *)carve(4 * NT), *t_pd1 = (int32_t *)carve(4 * NT);
    int32_t *t_pf = (int32_t *)carve(PREDS ? 4 * NT * kPDesc : 0);
    uint32_t *t_pb = (uint32_t *)carve(PREDS ? 4 * NT * kPDesc : 0);
    uint32_t *t_pc = (uint32_t *)carve(PREDS ? 4 * NT * kPDesc : 0);
    unsigned long long *t_tx = (unsigned long long *)carve(8 * NT);
    unsigned long long *t_busy = (unsigned long long *)carve(8 * NT);
    uint32_t *t_glist = (uint32_t *)carve(4 * NT * BM), *t_gdep = (uint32_t *)carve(4 * NT * BM);
    int32_t *t_sgrant = (int32_t *)carve(4 * NT * BM);
    uint4 *req = (uint4 *)carve(16 * (size_t)d.gd_req_max);
    // delivered counters: one per flow kept here, and a last one for the
    // flows nothing waits on (never published)
    uint32_t *deliv = (uint32_t *)carve(PREDS ? 4 * ((size_t)d.gd_fl_max + 1) : 0);
    int32_t *dflow = (int32_t *)carve(PREDS ? 4 * (size_t)d.gd_fl_max : 0);
    uint32_t *dmark = (uint32_t *)carve(PREDS ? 4 * (size_t)d.gd_fl_max : 0);  // bit 31: newest slot; low bits: changed-at stamp
    uint32_t *dlist = (uint32_t *)carve(PREDS ? 4 * (size_t)d.gd_fl_max : 0);
    uint32_t *red = (uint32_t *)carve(4 * 32);

    // a stream's range: cursor fields and its first predecessor descriptors
    auto set_range = [&](int j, int R) {
        t_rs[j] = d.r_start[R];
        t_rl[j] = d.r_len[R];
        t_rp[j] = d.r_path[R];
        const int pd0 = d.r_pd[R], pd1 = d.r_pd[R + 1];
        t_pd0[j] = pd0;
        t_pd1[j] = pd1;
        if (PREDS)
            for (int q = 0; q < kPDesc; q++)
                if (pd0 + q < pd1) {
                    t_pf[j * kPDesc + q] = d.pd_flow[pd0 + q];
                    t_pb[j * kPDesc + q] = d.pd_base[pd0 + q];
                }
    };
    const int32_t *path = d.gd_path;  // hop lanes -> the target's local index; sink -> -(1 + counter)
    uint32_t *ring = reinterpret_cast<uint32_t *>(d.gfifo);  // 4 words per entry
    uint32_t *comp = d.completion;

    for (int j = lt; j >= 0 && j < ns; j += NL) {
        const int lane = d.gd_slane[sb + j];
        const int link = d.ln_link[lane];
        s_lane[j] = (uint32_t)lane;
        s_b[j] = (uint32_t)d.bw[link];
        s_L[j] = (uint32_t)d.lat[link];
        s_fb[j] = (uint32_t)d.ln_fifo[lane];
        s_fm[j] = (uint32_t)d.ln_mask[lane];
        s_port[j] = (uint32_t)d.ln_port[lane];
        s_head[j] = s_tkn[j] = s_tkp[j] = s_nc[j] = 0;
    }
    for (int j = lt; j >= 0 && j < nt; j += NL) {
        const int lane = d.gd_tlane[tb + j];
        const int link = d.ln_link[lane];
        t_lane[j] = (uint32_t)lane;
        t_link[j] = (uint32_t)link;
        t_b[j] = (uint32_t)d.bw[link];
        t_L[j] = (uint32_t)d.lat[link];
        t_cap[j] = (uint32_t)d.cap[link];
        t_P[j] = (uint32_t)d.ln_P[lane];
        t_fb[j] = (uint32_t)d.ln_fifo[lane];
        t_fm[j] = (uint32_t)d.ln_mask[lane];
        t_rqoff[j] = (uint32_t)d.gd_rqoff[lane];
        t_rqcap[j] = (uint32_t)d.ln_reqcap[lane];
        t_srend[j] = d.ln_srend[lane];
        t_tail[j] = t_rr[j] = t_cnt[j] = 0;
        t_tx[j] = t_busy[j] = 0;
        const int R = d.ln_srbeg[lane];
        t_R[j] = R;
        t_o[j] = 0;
        if (R < t_srend[j]) set_range(j, R);
    }
    for (int j = tid; j < NS * BM; j += blockDim.x) s_grant[j] = -1;
    for (int j = tid; j < NT * BM; j += blockDim.x) {
        t_sgrant[j] = -1;
        t_gdep[j] = 0;
    }
    if (PREDS) {
        for (int j = tid; j <= d.gd_fl_max; j += blockDim.x) deliv[j] = 0;
        const int f0 = d.gd_fptr[w], nf = d.gd_fptr[w + 1] - f0;
        for (int j = tid; j < d.gd_fl_max; j += blockDim.x) {
            dmark[j] = 0;
            dflow[j] = j < nf ? d.gd_fown[f0 + j] : 0;
        }
    }
    if (tid < 32) red[tid] = tid < 16 ? kNever : 0u;
    if (w == 0)
        for (int j = tid; j < m; j += blockDim.x)
            if (d.link_lane[j] < 0) {
                d.tx_lines[j] = 0;
                d.busy[j] = 0;
            }
    __syncthreads();

    uint32_t t = 0, t_prev = 0;
    uint64_t k = 0;
    int32_t state = d.T > 0 ? kRunRunning : kRunOk;
    bool overflow = false;

    while (state == kRunRunning) {
        const int par = (int)(k & 1u);
        uint32_t *tail_prev = d.gd_pub + (size_t)(par ^ 1) * nl;   // appended counts at the start of t
        uint32_t *tail_cur = d.gd_pub + (size_t)par * nl;
        uint32_t *head_prev = d.gd_pub + (size_t)(2 + (par ^ 1)) * nl;  // popped counts at the start of t
        uint32_t *head_cur = d.gd_pub + (size_t)(2 + par) * nl;
        uint32_t next = kNever;
        int dep = 0;
        bool act = false;
        // ------------------------------------------------------------- poll
        // one round of device loads: the appended counts of the in-links and
        // the popped counts of the out-links, as of the start of cycle t
        for (int j = lt; j >= 0 && j < nmax; j += NL) {
            uint32_t a = 0, h = 0;
            int32_t nh[kCache];
            if (j < ns) {
                a = ld_dev(&tail_prev[s_lane[j]]);
                const uint32_t nc = s_nc[j];
#pragma unroll
                for (int q = 0; q < kCache; q++)
                    nh[q] = ((uint32_t)q < nc && s_ct[j * kCache + q] == kUnresolved) ? path[s_cp[j * kCache + q] + 1]
                                                                                     : kUnresolved;
            }
            if (j < nt) h = ld_dev(&head_prev[t_lane[j]]);
            if (PREDS && j < nt && t_R[j] < t_srend[j]) {
                const int npd = t_pd1[j] - t_pd0[j];
#pragma unroll
                for (int q = 0; q < kPDesc; q++)
                    if (q < npd) t_pc[j * kPDesc + q] = deliv_at(d.gd_dslot, t_pf[j * kPDesc + q], t);
            }
            if (j < ns) {
                s_tkp[j] = s_tkn[j];
                s_tkn[j] = a;
#pragma unroll
                for (int q = 0; q < kCache; q++)
                    if (nh[q] != kUnresolved) s_ct[j * kCache + q] = nh[q];
            }
            if (j < nt) t_khead[j] = h;
        }
        // -------------------------------------------------------------- R
        for (int j = lt; j >= 0 && j < ns; j += NL) {
            const uint32_t b = s_b[j], head = s_head[j], tkn = s_tkn[j], tkp = s_tkp[j], nc = s_nc[j];
            const uint32_t avail = tkn - head;
            uint32_t nf = 0;
            for (uint32_t q = 0; q < b && q < avail; q++) {
                uint32_t x, rdy, pp;
                int tg;
                if (q < nc) {  // fetched while waiting at the last barrier
                    x = s_cx[j * kCache + q];
                    rdy = s_cr[j * kCache + q];
                    tg = s_ct[j * kCache + q];
                    pp = s_cp[j * kCache + q];
                } else {
                    if (head + q >= tkp) {  // appended at the last processed cycle
                        rdy = t_prev + s_L[j];
                        if (rdy > t) {
                            next = rdy < next ? rdy : next;
                            break;
                        }
                    }
                    uint32_t *e = ring + 4 * (size_t)(s_fb[j] + ((head + q) & s_fm[j]));
                    x = ld_dev(e);
                    rdy = ld_dev(e + 1);
                    pp = ld_dev(e + 2);
                    tg = path[pp + 1];
                }
                if (rdy > t) {
                    next = rdy < next ? rdy : next;
                    break;
                }
                s_fx[j * BM + q] = x;
                s_ftg[j * BM + q] = tg;
                if (tg >= 0) {
                    const uint32_t slot = atomicAdd(&t_cnt[tg], 1u);
                    if (slot < t_rqcap[tg])
                        req[t_rqoff[tg] + slot] = make_uint4(x, pp + 1, ((uint32_t)(2 * j) << 8) | q, s_port[j]);
                    else
                        overflow = true;
                }
                nf++;
            }
            s_nf[j] = nf;
        }
        for (int j = lt; j >= 0 && j < nt; j += NL) {
            const int rend = t_srend[j];
            int R = t_R[j];
            uint32_t nsr = 0;
            if (R < rend) {
                const uint32_t b = t_b[j], P = t_P[j];
                uint32_t o = t_o[j], start = t_rs[j], len = t_rl[j];
                int rpath = t_rp[j];
                uint32_t allow = 0xFFFFFFFFu;
                if (PREDS) {
                    const int npd = t_pd1[j] - t_pd0[j];
                    if (npd > kPDesc) {
                        allow = stream_allow<PREDS>(d, t_pd0[j], t_pd1[j], o, t);
                    } else {
                        for (int q = 0; q < npd && allow > 0; q++) {
                            const uint32_t c = t_pc[j * kPDesc + q], base = t_pb[j * kPDesc + q];
                            if (c <= base) {
                                allow = 0;
                            } else if (d.pd_omask) {
                                const uint32_t m2 = c - base;
                                allow = m2 <= o ? 0u : (allow < m2 - o ? allow : m2 - o);
                            }
                        }
                    }
                }
                for (uint32_t q = 0; q < b && R < rend && allow > 0; q++) {
                    const uint32_t slot = atomicAdd(&t_cnt[j], 1u);
                    if (slot < t_rqcap[j])
                        req[t_rqoff[j] + slot] = make_uint4(start + o, (uint32_t)rpath, ((uint32_t)(2 * j + 1) << 8) | q,
                                                            P - 1);
                    else
                        overflow = true;
                    nsr++;
                    allow--;
                    if (++o == len) {
                        o = 0;
                        R++;
                        if (R < rend) {
                            start = d.r_start[R];
                            len = d.r_len[R];
                            rpath = d.r_path[R];
                            allow = stream_allow<PREDS>(d, d.r_pd[R], d.r_pd[R + 1], 0, t);
                        }
                    }
                }
            }
            t_nsr[j] = nsr;
        }
        __syncthreads();
        // -------------------------------------------------------------- G
        for (int j = lt; j >= 0 && j < nt; j += NL) {
            const uint32_t c = t_cnt[j];
            int g = 0;
            if (c) {
                t_cnt[j] = 0;
                const uint32_t P = t_P[j], rr = t_rr[j], rq = t_rqoff[j];
                g = (int)t_cap[j] - (int)(t_tail[j] - t_khead[j]);
                if ((int)t_b[j] < g) g = (int)t_b[j];
                if ((int)c < g) g = (int)c;
                if (c > t_rqcap[j]) g = 0;
                auto key = [&](const uint4 &r) -> uint32_t {
                    if (ARB == 0) return r.x;
                    const uint32_t o2 = r.w + P - rr;
                    return (r.z & 255u) * P + (o2 >= P ? o2 - P : o2);
                };
                if (g > 0) {
                    for (uint32_t a = 0; a < c; a++) {
                        const uint4 ra = req[rq + a];
                        const uint32_t ka = key(ra);
                        int rank = 0;
                        for (uint32_t q = 0; q < c; q++) rank += key(req[rq + q]) < ka ? 1 : 0;
                        if (rank < g) {
                            const uint32_t src = ra.z >> 8, kk = ra.z & 255u;
                            if (src & 1u)
                                t_sgrant[(src >> 1) * BM + kk] = rank;
                            else
                                s_grant[(src >> 1) * BM + kk] = rank;
                            t_glist[j * BM + rank] = rq + a;
                        }
                    }
                } else {
                    g = 0;
                }
            }
            t_g[j] = g;
        }
        __syncthreads();
        // -------------------------------------------------------------- D
        for (int j = lt; j >= 0 && j < ns; j += NL) {
            const uint32_t nf = s_nf[j];
            bool open = true;
            uint32_t depf = 0;
            for (uint32_t q = 0; q < nf; q++) {
                const int tg = s_ftg[j * BM + q];
                int gr = -2;
                if (tg >= 0) {
                    gr = s_grant[j * BM + q];
                    s_grant[j * BM + q] = -1;
                }
                if (open && gr != -1) {
                    depf++;
                    if (gr == -2) {
                        const uint32_t x = s_fx[j * BM + q];
                        comp[x] = t + 1;
                        const int fl = -tg - 1;
                        if (PREDS && fl < d.gd_fl_max) {
                            deliv[fl] += 1u;
                            if ((dmark[fl] & 0x7FFFFFFFu) != (uint32_t)(k & 0x7FFFFFFFu) + 1u) {
                                dmark[fl] = (dmark[fl] & 0x80000000u) | ((uint32_t)(k & 0x7FFFFFFFu) + 1u);
                                dlist[atomicAdd(&red[24 + par], 1u)] = (uint32_t)fl;
                            }
                        }
                    } else {
                        t_gdep[tg * BM + gr] = 1u;
                    }
                } else {
                    open = false;
                }
            }
            const uint32_t head = s_head[j] + depf;
            if (depf) {  // the popped entries leave the cache
                const uint32_t nc = s_nc[j];
                const uint32_t keep = nc > depf ? nc - depf : 0u;
                for (uint32_t q = 0; q < keep; q++) {
                    s_cx[j * kCache + q] = s_cx[j * kCache + q + depf];
                    s_cr[j * kCache + q] = s_cr[j * kCache + q + depf];
                    s_ct[j * kCache + q] = s_ct[j * kCache + q + depf];
                    s_cp[j * kCache + q] = s_cp[j * kCache + q + depf];
                }
                s_nc[j] = keep;
                s_head[j] = head;
            }
            st_dev(&head_cur[s_lane[j]], head);
            dep += (int)depf;
            if (head != s_tkn[j]) act = true;  // lines left that were appended before this cycle
        }
        for (int j = lt; j >= 0 && j < nt; j += NL) {
            const uint32_t nsr = t_nsr[j];
            if (nsr) {
                bool open = true;
                uint32_t deps = 0;
                for (uint32_t q = 0; q < nsr; q++) {
                    const int gr = t_sgrant[j * BM + q];
                    t_sgrant[j * BM + q] = -1;
                    if (open && gr != -1) {
                        deps++;
                        t_gdep[j * BM + gr] = 1u;
                    } else {
                        open = false;
                    }
                }
                if (deps) {
                    const int rend = t_srend[j];
                    int R = t_R[j];
                    uint32_t o = t_o[j] + deps;
                    bool moved = false;
                    uint32_t len = t_rl[j];
                    while (R < rend && o >= len) {
                        o -= len;
                        R++;
                        moved = true;
                        if (R < rend) len = d.r_len[R];
                    }
                    if (moved && R < rend) set_range(j, R);
                    t_R[j] = R;
                    t_o[j] = o;
                    dep += (int)deps;
                }
            }
            if (t_R[j] < t_srend[j]) act = true;  // stream lines left
        }
        __syncthreads();
        // -------------------------------------------------------------- E
        for (int j = lt; j >= 0 && j < nt; j += NL) {
            const int g = t_g[j];
            uint32_t tail = t_tail[j];
            if (g > 0) {
                const uint32_t ready = t + t_L[j];
                const uint32_t fb = t_fb[j], fm = t_fm[j];
                int cnt = 0;
                uint32_t last_port = 0;
                for (int r = 0; r < g; r++) {
                    if (t_gdep[j * BM + r]) {
                        t_gdep[j * BM + r] = 0u;
                        const uint4 rq = req[t_glist[j * BM + r]];
                        uint32_t *e = ring + 4 * (size_t)(fb + (tail & fm));
                        st_dev(e, rq.x);
                        st_dev(e + 1, ready);
                        st_dev(e + 2, rq.y);
                        tail++;
                        cnt++;
                        last_port = rq.w;
                    }
                }
                if (cnt) {
                    act = true;  // lines appended this cycle
                    t_tail[j] = tail;
                    t_tx[j] += (unsigned long long)cnt;
                    t_busy[j] += 1ull;
                    if (ARB == 1) {
                        const uint32_t P = t_P[j];
                        t_rr[j] = last_port + 1u == P ? 0u : last_port + 1u;
                    }
                }
            }
            st_dev(&tail_cur[t_lane[j]], tail);
        }
        if (PREDS) {
            // publish the flows that delivered this cycle: the slot not holding
            // the newest value gets (first cycle it holds for << 32 | count)
            const uint32_t nch = red[24 + par];
            for (int q = lt; q >= 0 && q < (int)nch; q += NL) {
                const int fl = (int)dlist[q];
                const int f = dflow[fl];
                const uint32_t mk = dmark[fl];
                const int slot = (mk >> 31) ? 0 : 1;
                st_dev(&d.gd_dslot[2 * f + slot], ((unsigned long long)(t + 1) << 32) | deliv[fl]);
                dmark[fl] = (mk & 0x7FFFFFFFu) | (slot ? 0x80000000u : 0u);
            }
        }
        // -------------------------------------------------------------- time
        // this workgroup's offer: t + 1 if anything moved, else its earliest
        // future FIFO-head ready time
        const int p4 = par * 4;
        {
            const bool wdep = __ballot(dep > 0) != 0, wact = __ballot(act) != 0, wover = __ballot(overflow) != 0;
            uint32_t v = next;
#pragma unroll
            for (int sh = 32; sh >= 1; sh >>= 1) {
                const uint32_t u = (uint32_t)__shfl_xor((int)v, sh);
                v = u < v ? u : v;
            }
            if ((tid & 63) == 0) {
                if (wdep) red[p4] = 1u;
                if (wact) red[p4 + 1] = 1u;
                if (wover) red[p4 + 3] = 1u;
                if (v != kNever) atomicMin(&red[p4 + 2], v);
            }
        }
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this thread's stores are done
        __syncthreads();
        if (tid == 0) {
            // One 64-bit arrival word per cycle (three in rotation):
            // arrivals | movers << 16 | active << 32 | overflowed << 48.  A
            // workgroup that moved nothing first offers its next ready time.
            const bool any_dep = red[p4] != kNever;
            const bool any_act = red[p4 + 1] != kNever;
            const bool any_over = red[p4 + 3] != kNever;
            const int r3 = (int)(k % 3u);
            unsigned long long *word = reinterpret_cast<unsigned long long *>(d.gd_sync) + r3;
            uint32_t *nxtw = d.gd_sync + 6 + r3;
            if (!any_dep && red[p4 + 2] != kNever) {
                __hip_atomic_fetch_min(nxtw, red[p4 + 2], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __builtin_amdgcn_s_waitcnt(0x0F70);  // the offer lands before the arrival
            }
            const unsigned long long mine = 1ull | (any_dep ? 1ull << 16 : 0ull) | (any_act ? 1ull << 32 : 0ull) |
                                            (any_over ? 1ull << 48 : 0ull);
            unsigned long long v = __hip_atomic_fetch_add(word, mine, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + mine;
            uint32_t spins = 0;
            bool stuck = false;
            while ((v & 0xFFFFull) < (unsigned long long)NB) {
                if (++spins > kSpinLimit) {
                    stuck = true;
                    break;
                }
                v = ld_dev(word);
            }
            const bool movers = ((v >> 16) & 0xFFFFull) != 0, active = ((v >> 32) & 0xFFFFull) != 0;
            const bool over = (v >> 48) != 0;
            red[16] = movers ? t + 1 : (active && !over && !stuck ? ld_dev(nxtw) : kNever);
            red[17] = (active ? 1u : 0u) | (over ? 2u : 0u) | (stuck ? 4u : 0u);
            if (w == 0 && !stuck) {  // the words of cycle k + 2 were last read before this barrier
                const int r5 = (int)((k + 2) % 3u);
                st_dev(reinterpret_cast<unsigned long long *>(d.gd_sync) + r5, 0ull);
                st_dev(d.gd_sync + 6 + r5, kNever);
            }
            red[(4 - p4)] = kNever;
            red[(4 - p4) + 1] = kNever;
            red[(4 - p4) + 2] = kNever;
            red[(4 - p4) + 3] = kNever;
            red[24 + (par ^ 1)] = 0u;
        } else {
            // While wave 0 waits: fetch each in-link's next entries (appended
            // before this cycle, so complete and stable) with their next hops.
            for (int j = lt; j >= 0 && j < ns; j += NL) {
                const uint32_t head = s_head[j], tkn = s_tkn[j], nc = s_nc[j];
                uint32_t want = s_b[j] < (uint32_t)kCache ? s_b[j] : (uint32_t)kCache;
                if (want > tkn - head) want = tkn - head;
                if (nc >= want) continue;
                uint32_t ex[kCache], er[kCache], ep[kCache];
#pragma unroll
                for (int q = 0; q < kCache; q++)
                    if ((uint32_t)q >= nc && (uint32_t)q < want) {
                        uint32_t *e = ring + 4 * (size_t)(s_fb[j] + ((head + q) & s_fm[j]));
                        ex[q] = ld_dev(e);
                        er[q] = ld_dev(e + 1);
                        ep[q] = ld_dev(e + 2);
                    }
#pragma unroll
                for (int q = 0; q < kCache; q++)
                    if ((uint32_t)q >= nc && (uint32_t)q < want) {
                        s_cx[j * kCache + q] = ex[q];
                        s_cr[j * kCache + q] = er[q];
                        s_cp[j * kCache + q] = ep[q];
                        s_ct[j * kCache + q] = kUnresolved;
                    }
                s_nc[j] = want;
            }
        }
        __syncthreads();
        const uint32_t nxt = red[16];
        const uint32_t flags = red[17];
        k++;
        if (flags & 4u) {
            state = kRunWatchdog;
        } else if (flags & 2u) {
            state = kRunInternal;
        } else if (!(flags & 1u)) {
            state = kRunOk;
        } else if (nxt == kNever) {
            state = kRunDeadlock;
        } else {
            t_prev = t;
            t = nxt;
        }
        if (state == kRunRunning && (uint64_t)t > d.max_cycles) state = kRunMaxCycles;
        if (state == kRunRunning && k > d.watchdog) state = kRunWatchdog;
        __syncthreads();  // red[16..17] are rewritten next cycle
    }
    for (int j = lt; j >= 0 && j < nt; j += NL) {
        d.tx_lines[t_link[j]] = t_tx[j];
        d.busy[t_link[j]] = t_busy[j];
    }
    if (tid == 0) {
        atomicMax(&d.status[0], state);
        if (w == 0) {
            d.makespan[0] = d.T > 0 ? t + 1 : 0;
            d.cycles[0] = k;
        }
    }
}

// ----------------------------------------------------------------------------
// Grid engine for graphs whose every link moves one line per cycle (b = 1),
// with one source side and one target side per thread, kept in registers.
// Then a FIFO offers at most its head, a link grants at most one request and
// a grant always departs (no void grants), so a cycle needs one exchange of
// LDS words, as in the compact single-workgroup engine:
//   round-robin  the source posts {line, path index} in its own LDS slot and
//                sets its port's bit in the target's word; the target picks
//                the first set bit at or after its pointer, appends the
//                winner and marks the winner's post as won;
//   lowest-id    the source takes the atomic minimum of {line, path index}
//                in the target's word (two words, by cycle parity); the
//                target appends the winner and a source has departed when the
//                word still holds its line.
// The target appends in the grant phase, so a cycle has two LDS phase
// boundaries.  The appended and popped counts cross workgroups as 64-bit
// words tagged with the processed-cycle index (a slot per cycle parity): the
// thread that owns a side waits for the tag of the cycle it needs while wave
// 0 waits at the barrier, so the barrier itself carries no data and nothing
// waits for all stores before arriving.  A count is stored only after the
// entries it covers (the appending thread waits for its entry stores first),
// so an entry below a count read with the right tag is complete.  The head
// entry is fetched, and its next hop looked up, in the same wait.
template <int ARB, bool PREDS>
__global__ void __launch_bounds__(1024) engine_grid1(DevNet d) {
    extern __shared__ __align__(16) unsigned char smem[];
    if (blockIdx.x % (unsigned)d.gd_stride) return;
    const int w = (int)(blockIdx.x / (unsigned)d.gd_stride);
    if (w >= d.gd_nb) return;
    const int tid = threadIdx.x;
    const int j = tid - 64;  // this thread's source side and target side (wave 0 runs the barrier)
    const int nl = d.nl, m = d.m, NB = d.gd_nb;
    const int sb = d.gd_sptr[w], ns = d.gd_sptr[w + 1] - sb;
    const int tb = d.gd_tptr[w], nt = d.gd_tptr[w + 1] - tb;
    const int NT = d.gd_nt_max, NS = d.gd_ns_max;
    const bool hs = j >= 0 && j < ns, ht = j >= 0 && j < nt;

    size_t off = 0;
    auto carve = [&](size_t bytes) {
        unsigned char *p = smem + off;
        off = (off + bytes + 15) & ~(size_t)15;
        return p;
    };
    unsigned long long *word = (unsigned long long *)carve(8 * (size_t)NT * (ARB == 0 ? 2 : 1));
    unsigned long long *post = (unsigned long long *)carve(ARB == 1 ? 8 * (size_t)NS : 0);
    int32_t *inl = (int32_t *)carve(ARB == 1 ? 4 * (size_t)d.gd_inl_max : 0);
    uint32_t *deliv = (uint32_t *)carve(PREDS ? 4 * ((size_t)d.gd_fl_max + 1) : 0);
    int32_t *dflow = (int32_t *)carve(PREDS ? 4 * (size_t)d.gd_fl_max : 0);
    uint32_t *dmark = (uint32_t *)carve(PREDS ? 4 * (size_t)d.gd_fl_max : 0);
    uint32_t *dlist = (uint32_t *)carve(PREDS ? 4 * (size_t)d.gd_fl_max : 0);
    uint32_t *red = (uint32_t *)carve(4 * 32);
    constexpr unsigned long long kNone = ARB == 0 ? ~0ull : 0ull;
    constexpr unsigned long long kWon = ~0ull;

    const int32_t *path = d.gd_path;
    uint32_t *ring = reinterpret_cast<uint32_t *>(d.gfifo);
    uint32_t *comp = d.completion;
    unsigned long long *tpub = d.gd_tpub;  // [parity][tail | head][nl]: (cycle index << 32) | count

    for (int q = tid; q < NT * (ARB == 0 ? 2 : 1); q += blockDim.x) word[q] = kNone;
    if (ARB == 1) {
        const int i0 = d.gd_iptr[w], ni = d.gd_iptr[w + 1] - i0;
        for (int q = tid; q < ni; q += blockDim.x) inl[q] = d.gd_inl[i0 + q];
    }
    if (PREDS) {
        for (int q = tid; q <= d.gd_fl_max; q += blockDim.x) deliv[q] = 0;
        const int f0 = d.gd_fptr[w], nf = d.gd_fptr[w + 1] - f0;
        for (int q = tid; q < d.gd_fl_max; q += blockDim.x) {
            dmark[q] = 0;
            dflow[q] = q < nf ? d.gd_fown[f0 + q] : 0;
        }
    }
    if (tid < 32) red[tid] = tid < 16 ? kNever : 0u;
    if (w == 0)
        for (int q = tid; q < m; q += blockDim.x)
            if (d.link_lane[q] < 0) {
                d.tx_lines[q] = 0;
                d.busy[q] = 0;
            }

    // source side: the in-link's FIFO as seen from its head node
    uint32_t s_lane = 0, s_fb = 0, s_fm = 0, s_L = 0, s_port = 0;
    uint32_t head = 0, tkn = 0, tkp = 0;
    bool cval = false;               // head entry cached
    uint32_t cx = 0, cr = 0, cpp = 0;
    int32_t ct = kUnresolved;        // cached entry's next hop
    if (hs) {
        s_lane = (uint32_t)d.gd_slane[sb + j];
        const int link = d.ln_link[s_lane];
        s_fb = (uint32_t)d.ln_fifo[s_lane];
        s_fm = (uint32_t)d.ln_mask[s_lane];
        s_L = (uint32_t)d.lat[link];
        s_port = (uint32_t)d.ln_port[s_lane];
    }
    // target side: the out-link's arbitration, appends and stream
    uint32_t t_lane = 0, t_link = 0, t_L = 0, t_cap = 0, t_P = 1, t_fb = 0, t_fm = 0, t_toff = 0;
    uint32_t tail = 0, khead = 0, rr = 0;
    unsigned long long tx = 0;
    int R = 0, rend = 0;
    uint32_t o = 0, r_st = 0, r_len = 0;
    int r_path = 0, pd0 = 0, pd1 = 0;
    int32_t pf[kPDesc];
    uint32_t pb[kPDesc];
#pragma unroll
    for (int q = 0; q < kPDesc; q++) pf[q] = 0, pb[q] = 0;
    auto set_range = [&](int Rn) {
        r_st = d.r_start[Rn];
        r_len = d.r_len[Rn];
        r_path = d.r_path[Rn];
        pd0 = d.r_pd[Rn];
        pd1 = d.r_pd[Rn + 1];
        if (PREDS)
#pragma unroll
            for (int q = 0; q < kPDesc; q++)
                if (pd0 + q < pd1) {
                    pf[q] = d.pd_flow[pd0 + q];
                    pb[q] = d.pd_base[pd0 + q];
                }
    };
    if (ht) {
        t_lane = (uint32_t)d.gd_tlane[tb + j];
        t_link = (uint32_t)d.ln_link[t_lane];
        t_L = (uint32_t)d.lat[t_link];
        t_cap = (uint32_t)d.cap[t_link];
        t_P = (uint32_t)d.ln_P[t_lane];
        t_fb = (uint32_t)d.ln_fifo[t_lane];
        t_fm = (uint32_t)d.ln_mask[t_lane];
        t_toff = ARB == 1 ? (uint32_t)d.gd_toff[t_lane] : 0u;
        R = d.ln_srbeg[t_lane];
        rend = d.ln_srend[t_lane];
        if (R < rend) set_range(R);
    }
    __syncthreads();

    uint32_t t = 0, t_prev = 0;
    uint64_t k = 0;
    int32_t state = d.T > 0 ? kRunRunning : kRunOk;

    while (state == kRunRunning) {
        const int par = (int)(k & 1u);
        unsigned long long *wcur = ARB == 0 ? word + (size_t)par * NT : word;
        uint32_t next = kNever;
        int dep = 0;
        bool act = false;
        // -------------------------------------------------------------- R
        bool req_f = false, sink_f = false;  // the head requests a link / the sink
        if (hs && tkn != head) {
            uint32_t x = cx, rdy = cr, pp = cpp;
            int32_t tg = ct;
            bool known = cval;
            if (!cval && head >= tkp) {  // appended at the last processed cycle
                rdy = t_prev + s_L;
                known = rdy > t;         // not ready yet: its contents can wait
            }
            if (!known) {
                uint32_t *e = ring + 4 * (size_t)(s_fb + (head & s_fm));
                cx = x = ld_dev(e);
                cr = rdy = ld_dev(e + 1);
                cpp = pp = ld_dev(e + 2);
                ct = tg = kUnresolved;
                cval = true;
            }
            if (rdy <= t && tg == kUnresolved) ct = tg = path[pp + 1];
            if (rdy > t) {
                next = rdy;
            } else if (tg < 0) {
                sink_f = true;
            } else {
                req_f = true;
                const unsigned long long key = ((unsigned long long)x << 32) | (pp + 1u);
                if (ARB == 1) {
                    post[j] = key;
                    atomicOr(&wcur[tg], 1ull << s_port);
                } else {
                    atomicMin(&wcur[tg], key);
                }
            }
        }
        bool sreq = false;
        if (ht && R < rend) {
            bool ok = true;
            if (PREDS) {
                const int npd = pd1 - pd0;
                if (npd > kPDesc) {
                    ok = stream_allow<PREDS>(d, pd0, pd1, o, t) > 0;
                } else {
#pragma unroll
                    for (int q = 0; q < kPDesc; q++)
                        if (q < npd) ok = ok && deliv_at(d.gd_dslot, pf[q], t) > pb[q] + (o & d.pd_omask);
                }
            }
            if (ok) {
                sreq = true;
                if (ARB == 1)
                    atomicOr(&wcur[j], 1ull << (t_P - 1u));
                else
                    atomicMin(&wcur[j], ((unsigned long long)(r_st + o) << 32) | (uint32_t)r_path);
            }
        }
        __syncthreads();
        // ------------------------------------------------ G (and append)
        bool sdep = false;
        bool appended = false;
        if (ht) {
            if (ARB == 0) word[(size_t)(par ^ 1) * NT + j] = kNone;  // the word of the next cycle
            const unsigned long long wv = wcur[j];
            if (wv != kNone) {
                if (ARB == 1) wcur[j] = 0ull;
                if (tail - khead >= t_cap) {
                    if (ARB == 0) wcur[j] = kNone;  // full: nobody moves
                } else {
                    uint32_t x, pp;
                    if (ARB == 1) {
                        const unsigned long long hi = wv >> rr;
                        const uint32_t p = hi ? rr + (uint32_t)__builtin_ctzll(hi) : (uint32_t)__builtin_ctzll(wv);
                        const int src = inl[t_toff + p];
                        if (src < 0) {  // the injection port: this thread's own stream
                            x = r_st + o;
                            pp = (uint32_t)r_path;
                            sdep = true;
                        } else {
                            const unsigned long long pw = post[src];
                            post[src] = kWon;
                            x = (uint32_t)(pw >> 32);
                            pp = (uint32_t)pw;
                        }
                        rr = p + 1u == t_P ? 0u : p + 1u;
                    } else {
                        x = (uint32_t)(wv >> 32);
                        pp = (uint32_t)wv;
                    }
                    uint32_t *e = ring + 4 * (size_t)(t_fb + (tail & t_fm));
                    st_dev(e, x);
                    st_dev(e + 1, t + t_L);
                    st_dev(e + 2, pp);
                    tail++;
                    tx++;
                    appended = true;
                }
            }
        }
        __syncthreads();
        // -------------------------------------------------------------- D
        if (hs) {
            bool gone = sink_f;
            if (sink_f) {
                comp[cx] = t + 1;
                const int fl = -ct - 1;
                if (PREDS && fl < d.gd_fl_max) {
                    deliv[fl] += 1u;
                    if ((dmark[fl] & 0x7FFFFFFFu) != (uint32_t)(k & 0x7FFFFFFFu) + 1u) {
                        dmark[fl] = (dmark[fl] & 0x80000000u) | ((uint32_t)(k & 0x7FFFFFFFu) + 1u);
                        dlist[atomicAdd(&red[24 + par], 1u)] = (uint32_t)fl;
                    }
                }
            } else if (req_f) {
                gone = ARB == 1 ? post[j] == kWon : (uint32_t)(wcur[ct] >> 32) == cx;
            }
            if (gone) {
                head++;
                cval = false;
                ct = kUnresolved;
                dep++;
            }
            st_dev(&tpub[((size_t)par * 2 + 1) * nl + s_lane], ((unsigned long long)(uint32_t)k << 32) | head);
            if (head != tkn) act = true;
        }
        if (ht) {
            if (sreq && (ARB == 1 ? sdep : (uint32_t)(wcur[j] >> 32) == r_st + o)) {
                dep++;
                if (++o == r_len) {
                    o = 0;
                    R++;
                    if (R < rend) set_range(R);
                }
            }
            if (appended) act = true;
            if (R < rend) act = true;
        }
        if (PREDS) {
            __syncthreads();  // the list of flows that delivered
            const uint32_t nch = red[24 + par];
            for (int q = j; q >= 0 && q < (int)nch; q += (int)blockDim.x - 64) {
                const int fl = (int)dlist[q];
                const int f = dflow[fl];
                const uint32_t mk = dmark[fl];
                const int slot = (mk >> 31) ? 0 : 1;
                st_dev(&d.gd_dslot[2 * f + slot], ((unsigned long long)(t + 1) << 32) | deliv[fl]);
                dmark[fl] = (mk & 0x7FFFFFFFu) | (slot ? 0x80000000u : 0u);
            }
            // delivered counts are read after the barrier: they are complete
            // before this workgroup arrives
            __builtin_amdgcn_s_waitcnt(0x0F70);
        }
        // -------------------------------------------------------------- time
        const int p4 = par * 4;
        {
            const bool wdep = __ballot(dep > 0) != 0, wact = __ballot(act) != 0;
            uint32_t v = next;
#pragma unroll
            for (int sh = 32; sh >= 1; sh >>= 1) {
                const uint32_t u = (uint32_t)__shfl_xor((int)v, sh);
                v = u < v ? u : v;
            }
            if ((tid & 63) == 0) {
                if (wdep) red[p4] = 1u;
                if (wact) red[p4 + 1] = 1u;
                if (v != kNever) atomicMin(&red[p4 + 2], v);
            }
        }
        __syncthreads();
        bool stuck = false;
        if (tid == 0) {
            const bool any_dep = red[p4] != kNever;
            const bool any_act = red[p4 + 1] != kNever;
            const int r3 = (int)(k % 3u);
            unsigned long long *wordg = reinterpret_cast<unsigned long long *>(d.gd_sync) + r3;
            uint32_t *nxtw = d.gd_sync + 6 + r3;
            if (!any_dep && red[p4 + 2] != kNever)
                __hip_atomic_fetch_min(nxtw, red[p4 + 2], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __builtin_amdgcn_s_waitcnt(0x0F70);  // the offer, and the last reset of the words, have landed
            const unsigned long long mine = 1ull | (any_dep ? 1ull << 16 : 0ull) | (any_act ? 1ull << 32 : 0ull);
            unsigned long long v = __hip_atomic_fetch_add(wordg, mine, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + mine;
            uint32_t spins = 0;
            while ((v & 0xFFFFull) < (unsigned long long)NB) {
                if (++spins > kSpinLimit) {
                    stuck = true;
                    break;
                }
                v = ld_dev(wordg);
            }
            const bool movers = ((v >> 16) & 0xFFFFull) != 0, active = ((v >> 32) & 0xFFFFull) != 0;
            red[16] = movers ? t + 1 : (active && !stuck ? ld_dev(nxtw) : kNever);
            red[17] = (active ? 1u : 0u);
            if (w == 0 && !stuck) {
                const int r5 = (int)((k + 2) % 3u);
                st_dev(reinterpret_cast<unsigned long long *>(d.gd_sync) + r5, 0ull);
                st_dev(d.gd_sync + 6 + r5, kNever);
            }
            red[(4 - p4)] = kNever;
            red[(4 - p4) + 1] = kNever;
            red[(4 - p4) + 2] = kNever;
            red[24 + (par ^ 1)] = 0u;
        } else if (j >= 0) {
            // While wave 0 waits: this thread's appended count (once the
            // entries it covers are stored), then this cycle's counts of this
            // thread's sides, the head entry and its next hop.
            const unsigned long long tagk = (unsigned long long)(uint32_t)k;
            if (ht) {
                if (appended) __builtin_amdgcn_s_waitcnt(0x0F70);
                st_dev(&tpub[((size_t)par * 2) * nl + t_lane], (tagk << 32) | tail);
            }
            bool need_e = hs && !cval && head != tkn;  // an entry known before this cycle
            uint32_t ex = 0, er = 0, ep = 0;
            int32_t nh = kUnresolved;
            if (need_e) {
                uint32_t *e = ring + 4 * (size_t)(s_fb + (head & s_fm));
                ex = ld_dev(e);
                er = ld_dev(e + 1);
                ep = ld_dev(e + 2);
            }
            if (hs && cval && ct == kUnresolved) nh = path[cpp + 1];
            uint32_t ntail = tkn, nkhead = khead;
            uint32_t spins = 0;
            if (hs) {
                unsigned long long *pw = &tpub[((size_t)par * 2) * nl + s_lane];
                unsigned long long v;
                while (((v = ld_dev(pw)) >> 32) != tagk) {
                    if (++spins > kSpinLimit) {
                        stuck = true;
                        break;
                    }
                    __builtin_amdgcn_s_sleep(2);
                }
                ntail = (uint32_t)v;
            }
            if (ht) {
                unsigned long long *pw = &tpub[((size_t)par * 2 + 1) * nl + t_lane];
                unsigned long long v;
                while (((v = ld_dev(pw)) >> 32) != tagk) {
                    if (++spins > kSpinLimit) {
                        stuck = true;
                        break;
                    }
                    __builtin_amdgcn_s_sleep(2);
                }
                nkhead = (uint32_t)v;
            }
            if (need_e) {
                cx = ex, cr = er, cpp = ep;
                ct = kUnresolved;
                cval = true;
            }
            if (nh != kUnresolved) ct = nh;
            // an entry appended this cycle is fetched in the next wait (its
            // ready time, t + L, is known without it)
            tkp = tkn;
            tkn = ntail;
            khead = nkhead;
        }
        if (stuck) red[20] = 1u;
        __syncthreads();
        const uint32_t nxt = red[16];
        const uint32_t flags = red[17];
        k++;
        if (red[20]) {
            state = kRunWatchdog;
        } else if (!(flags & 1u)) {
            state = kRunOk;
        } else if (nxt == kNever) {
            state = kRunDeadlock;
        } else {
            t_prev = t;
            t = nxt;
        }
        if (state == kRunRunning && (uint64_t)t > d.max_cycles) state = kRunMaxCycles;
        if (state == kRunRunning && k > d.watchdog) state = kRunWatchdog;
        __syncthreads();
    }
    if (ht) {
        d.tx_lines[t_link] = tx;
        d.busy[t_link] = tx;  // one line per cycle at most: busy cycles = lines
    }
    if (tid == 0) {
        atomicMax(&d.status[0], state);
        if (w == 0) {
            d.makespan[0] = d.T > 0 ? t + 1 : 0;
            d.cycles[0] = k;
        }
    }
}

// ----------------------------------------------------------------------------
// Windowed form (credit delays): when every traffic link has latency L >= 2
// and credit delay D >= 2, a line appended at cycle t may leave at t + L and
// a slot freed at t is usable from t + D, so within a window of
// W = min(L, D) cycles (over all traffic links) no workgroup's work can
// depend on another's.  Each workgroup then runs its own cycles of a window
// with LDS-only phases and its own event skipping; the workgroups exchange
// once per window:
//   - a source side mirrors the FIFO entries appended in earlier windows into
//     an LDS ring (with their next hops) and publishes its popped count; the
//     cycle each entry left is written into the entry's slot;
//   - a target side reads the cycles its popped entries left at (its credit
//     returns) and publishes its appended count;
//   - the next window starts at the earliest event any workgroup offers: its
//     next local event, the ready time of a line it appended, or the return
//     of a credit it freed (all at or after the window's end).
// Lines that cross no window boundary never leave the workgroup's LDS copy;
// the result is the same as the cycle-by-cycle model, because whatever one
// workgroup does inside a window reaches another only from the next window.
// Every bandwidth is 1 and no line has predecessors.
template <int ARB>
__global__ void __launch_bounds__(1024) engine_gridw(DevNet d) {
    extern __shared__ __align__(16) unsigned char smem[];
    if (blockIdx.x % (unsigned)d.gd_stride) return;
    const int w = (int)(blockIdx.x / (unsigned)d.gd_stride);
    if (w >= d.gd_nb) return;
    const int tid = threadIdx.x;
    const int j = tid - 64;
    const int nl = d.nl, m = d.m, NB = d.gd_nb;
    const int sb = d.gd_sptr[w], ns = d.gd_sptr[w + 1] - sb;
    const int tb = d.gd_tptr[w], nt = d.gd_tptr[w + 1] - tb;
    const int NT = d.gd_nt_max, NS = d.gd_ns_max;
    const bool hs = j >= 0 && j < ns, ht = j >= 0 && j < nt;
    const uint32_t W = (uint32_t)d.gd_window;
    const int nwave = (int)(blockDim.x >> 6);

    size_t off = 0;
    auto carve = [&](size_t bytes) {
        unsigned char *p = smem + off;
        off = (off + bytes + 15) & ~(size_t)15;
        return p;
    };
    unsigned long long *word = (unsigned long long *)carve(8 * (size_t)NT * (ARB == 0 ? 2 : 1));
    unsigned long long *post = (unsigned long long *)carve(ARB == 1 ? 8 * (size_t)NS : 0);
    int32_t *inl = (int32_t *)carve(ARB == 1 ? 4 * (size_t)d.gd_inl_max : 0);
    uint4 *sring = (uint4 *)carve(16 * (size_t)d.gd_sring_max);     // {line, ready, path index, next hop}
    uint32_t *cring = (uint32_t *)carve(4 * (size_t)d.gd_cring_max);  // cycles popped entries left at
    uint32_t *wred = (uint32_t *)carve(4 * 4 * 2 * 16);              // per wave: moved, next (two parities)
    uint32_t *red = (uint32_t *)carve(4 * 32);
    constexpr unsigned long long kNone = ARB == 0 ? ~0ull : 0ull;
    constexpr unsigned long long kWon = ~0ull;

    const int32_t *path = d.gd_path;
    uint32_t *ring = reinterpret_cast<uint32_t *>(d.gfifo);  // {line, ready, path index, cycle it left}
    uint32_t *comp = d.completion;
    unsigned long long *tpub = d.gd_tpub;

    for (int q = tid; q < NT * (ARB == 0 ? 2 : 1); q += blockDim.x) word[q] = kNone;
    if (ARB == 1) {
        const int i0 = d.gd_iptr[w], ni = d.gd_iptr[w + 1] - i0;
        for (int q = tid; q < ni; q += blockDim.x) inl[q] = d.gd_inl[i0 + q];
    }
    if (tid < 32) red[tid] = tid == 2 ? kNever : 0u;  // [0] flags, [2] earliest offer
    if (w == 0)
        for (int q = tid; q < m; q += blockDim.x)
            if (d.link_lane[q] < 0) {
                d.tx_lines[q] = 0;
                d.busy[q] = 0;
            }

    // source side
    uint32_t s_lane = 0, s_fb = 0, s_fm = 0, s_D = 1, s_port = 0, s_lo = 0;
    uint32_t head = 0, tkn = 0;
    if (hs) {
        s_lane = (uint32_t)d.gd_slane[sb + j];
        const int link = d.ln_link[s_lane];
        s_fb = (uint32_t)d.ln_fifo[s_lane];
        s_fm = (uint32_t)d.ln_mask[s_lane];
        s_D = (uint32_t)d.credit[link];
        s_port = (uint32_t)d.ln_port[s_lane];
        s_lo = (uint32_t)d.gd_sro[s_lane];
    }
    // target side
    uint32_t t_lane = 0, t_link = 0, t_L = 0, t_cap = 0, t_P = 1, t_fb = 0, t_fm = 0, t_toff = 0, t_D = 1, t_co = 0;
    uint32_t tail = 0, ret = 0, pk = 0, rr = 0;  // appended, credits back, pops known
    unsigned long long tx = 0;
    int R = 0, rend = 0;
    uint32_t o = 0, r_st = 0, r_len = 0;
    int r_path = 0;
    if (ht) {
        t_lane = (uint32_t)d.gd_tlane[tb + j];
        t_link = (uint32_t)d.ln_link[t_lane];
        t_L = (uint32_t)d.lat[t_link];
        t_cap = (uint32_t)d.cap[t_link];
        t_P = (uint32_t)d.ln_P[t_lane];
        t_fb = (uint32_t)d.ln_fifo[t_lane];
        t_fm = (uint32_t)d.ln_mask[t_lane];
        t_D = (uint32_t)d.credit[t_link];
        t_toff = ARB == 1 ? (uint32_t)d.gd_toff[t_lane] : 0u;
        t_co = (uint32_t)d.gd_tro[t_lane];
        R = d.ln_srbeg[t_lane];
        rend = d.ln_srend[t_lane];
        if (R < rend) {
            r_st = d.r_start[R];
            r_len = d.r_len[R];
            r_path = d.r_path[R];
        }
    }
    __syncthreads();

    uint32_t T0 = 0, maxcomp = 0;
    uint64_t widx = 0, local_cycles = 0;
    int32_t state = d.T > 0 ? kRunRunning : kRunOk;
    uint32_t lpar = 0;  // parity of the per-wave reduction slots

    while (state == kRunRunning) {
        const uint32_t wend = T0 + W;  // this window: cycles T0 .. wend - 1
        uint32_t t = T0;
        uint32_t offer = kNever;       // this thread's events at or after wend
        bool over = false;
        // ------------------------------------------------ cycles of the window
        // A cycle's departures are committed at the start of the next
        // iteration (or before the exchange): whether anything moved is
        // known after the grants (every departure other than to the sink is
        // an append here, and a sink departure is decided with the request),
        // so the workgroup's decision on its next cycle shares the barrier
        // between grants and departures.
        bool pend = false, req_f = false, sink_f = false, sreq = false, sdep = false;
        uint4 he = make_uint4(0, 0, 0, 0);
        uint32_t tD = t;
        unsigned long long *wD = word;
        auto depart = [&]() {
            if (hs && (sink_f || req_f)) {
                bool gone = sink_f;
                if (sink_f) {
                    comp[he.x] = tD + 1;
                    maxcomp = max(maxcomp, tD + 1);
                } else {
                    gone = ARB == 1 ? post[j] == kWon : (uint32_t)(wD[he.w] >> 32) == he.x;
                }
                if (gone) {
                    ring[4 * (size_t)(s_fb + (head & s_fm)) + 3] = tD;  // the cycle it left
                    head++;
                    offer = min(offer, tD + s_D);  // its credit comes back
                }
            }
            if (ht && sreq && (ARB == 1 ? sdep : (uint32_t)(wD[j] >> 32) == r_st + o)) {
                if (++o == r_len) {
                    o = 0;
                    R++;
                    if (R < rend) {
                        r_st = d.r_start[R];
                        r_len = d.r_len[R];
                        r_path = d.r_path[R];
                    }
                }
            }
        };
        for (;;) {
            if (pend) depart();
            unsigned long long *wcur = ARB == 0 ? word + (size_t)(lpar & 1u) * NT : word;
            uint32_t next = kNever;
            bool moved = false;
            req_f = sink_f = false;
            if (hs && head != tkn) {
                he = sring[s_lo + (head & s_fm)];
                if (he.y > t) {
                    next = he.y;
                } else if ((int32_t)he.w < 0) {
                    sink_f = true;
                    moved = true;
                } else {
                    req_f = true;
                    const unsigned long long key = ((unsigned long long)he.x << 32) | (he.z + 1u);
                    if (ARB == 1) {
                        post[j] = key;
                        atomicOr(&wcur[he.w], 1ull << s_port);
                    } else {
                        atomicMin(&wcur[he.w], key);
                    }
                }
            }
            sreq = false;
            if (ht && R < rend) {
                sreq = true;
                if (ARB == 1)
                    atomicOr(&wcur[j], 1ull << (t_P - 1u));
                else
                    atomicMin(&wcur[j], ((unsigned long long)(r_st + o) << 32) | (uint32_t)r_path);
            }
            __syncthreads();
            // ---- grants and appends
            sdep = false;
            if (ht) {
                if (ARB == 0) word[(size_t)((lpar & 1u) ^ 1u) * NT + j] = kNone;
                while (ret != pk && cring[t_co + (ret & t_fm)] + t_D <= t) ret++;  // credits back by t
                const unsigned long long wv = wcur[j];
                if (wv != kNone) {
                    if (ARB == 1) wcur[j] = 0ull;
                    if (tail - ret >= t_cap) {
                        if (ARB == 0) wcur[j] = kNone;
                    } else {
                        uint32_t x, pp;
                        if (ARB == 1) {
                            const unsigned long long hi = wv >> rr;
                            const uint32_t p = hi ? rr + (uint32_t)__builtin_ctzll(hi) : (uint32_t)__builtin_ctzll(wv);
                            const int src = inl[t_toff + p];
                            if (src < 0) {
                                x = r_st + o;
                                pp = (uint32_t)r_path;
                                sdep = true;
                            } else {
                                const unsigned long long pw = post[src];
                                post[src] = kWon;
                                x = (uint32_t)(pw >> 32);
                                pp = (uint32_t)pw;
                            }
                            rr = p + 1u == t_P ? 0u : p + 1u;
                        } else {
                            x = (uint32_t)(wv >> 32);
                            pp = (uint32_t)wv;
                        }
                        // plain stores: they are made visible, all at once, before the exchange
                        *reinterpret_cast<uint4 *>(ring + 4 * (size_t)(t_fb + (tail & t_fm))) =
                            make_uint4(x, t + t_L, pp, 0u);
                        tail++;
                        tx++;
                        moved = true;
                        offer = min(offer, t + t_L);  // its consumer's event
                    }
                }
                if (ret != pk) next = min(next, cring[t_co + (ret & t_fm)] + t_D);  // a credit coming back
            }
            // ---- the workgroup's next cycle
            {
                const bool wm = __ballot(moved) != 0;
                uint32_t v = next;
#pragma unroll
                for (int sh = 32; sh >= 1; sh >>= 1) {
                    const uint32_t u = (uint32_t)__shfl_xor((int)v, sh);
                    v = u < v ? u : v;
                }
                if ((tid & 63) == 0) {
                    wred[(lpar & 1u) * 32 + (tid >> 6) * 2] = wm ? 1u : 0u;
                    wred[(lpar & 1u) * 32 + (tid >> 6) * 2 + 1] = v;
                }
            }
            __syncthreads();
            bool any_moved = false;
            uint32_t nx = kNever;
            for (int q = 0; q < nwave; q++) {
                any_moved = any_moved || wred[(lpar & 1u) * 32 + q * 2] != 0u;
                nx = min(nx, wred[(lpar & 1u) * 32 + q * 2 + 1]);
            }
            pend = true;
            tD = t;
            wD = wcur;
            lpar++;
            local_cycles++;
            if (any_moved) nx = t + 1;
            if (nx >= wend || nx == kNever) {
                depart();
                offer = min(offer, nx);
                break;
            }
            if ((uint64_t)nx > d.max_cycles) {
                depart();
                over = true;
                break;
            }
            t = nx;
        }
        // ------------------------------------------------ exchange
        // the window's entries and departure cycles (plain stores) reach
        // device scope before the counts that cover them: every thread's
        // stores are done, then one write-back of the die's cache
        const unsigned long long tagw = (unsigned long long)(uint32_t)widx;
        const int par = (int)(widx & 1u);
        __builtin_amdgcn_s_waitcnt(0x0F70);
        __syncthreads();
        if (tid == 0) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        __syncthreads();
        if (hs) st_dev(&tpub[((size_t)par * 2 + 1) * nl + s_lane], (tagw << 32) | head);
        if (ht) st_dev(&tpub[((size_t)par * 2) * nl + t_lane], (tagw << 32) | tail);
        // lines left (offer already covers their events)
        bool act = (hs && head != tkn) || (ht && (R < rend || tail != pk));
        {
            const bool wact = __ballot(act) != 0, wover = __ballot(over) != 0;
            uint32_t v = offer;
#pragma unroll
            for (int sh = 32; sh >= 1; sh >>= 1) {
                const uint32_t u = (uint32_t)__shfl_xor((int)v, sh);
                v = u < v ? u : v;
            }
            if ((tid & 63) == 0) {
                if (wact) atomicOr(&red[0], 1u);
                if (wover) atomicOr(&red[0], 2u);
                if (v != kNever) atomicMin(&red[2], v);
            }
        }
        __syncthreads();
        bool stuck = false;
        if (tid == 0) {
            const uint32_t flags = red[0];
            const int r3 = (int)(widx % 3u);
            unsigned long long *wordg = reinterpret_cast<unsigned long long *>(d.gd_sync) + r3;
            uint32_t *nxtw = d.gd_sync + 6 + r3;
            if (red[2] != kNever) __hip_atomic_fetch_min(nxtw, red[2], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __builtin_amdgcn_s_waitcnt(0x0F70);
            const unsigned long long mine = 1ull | ((flags & 1u) ? 1ull << 32 : 0ull) | ((flags & 2u) ? 1ull << 48 : 0ull);
            unsigned long long v = __hip_atomic_fetch_add(wordg, mine, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + mine;
            uint32_t spins = 0;
            while ((v & 0xFFFFull) < (unsigned long long)NB) {
                if (++spins > kSpinLimit) {
                    stuck = true;
                    break;
                }
                v = ld_dev(wordg);
            }
            red[16] = stuck ? kNever : ld_dev(nxtw);
            red[17] = (((v >> 32) & 0xFFFFull) ? 1u : 0u) | ((v >> 48) ? 2u : 0u);
            if (w == 0 && !stuck) {
                const int r5 = (int)((widx + 2) % 3u);
                st_dev(reinterpret_cast<unsigned long long *>(d.gd_sync) + r5, 0ull);
                st_dev(d.gd_sync + 6 + r5, kNever);
            }
            red[0] = 0u;
            red[2] = kNever;
        } else if (j >= 0) {
            // the counts of this window; then the new entries (with their next
            // hops) and the cycles the newly popped entries left at
            uint32_t ntail = tkn, npk = pk;
            uint32_t spins = 0;
            if (hs) {
                unsigned long long *pw = &tpub[((size_t)par * 2) * nl + s_lane];
                unsigned long long v;
                while (((v = ld_dev(pw)) >> 32) != tagw) {
                    if (++spins > kSpinLimit) {
                        stuck = true;
                        break;
                    }
                    __builtin_amdgcn_s_sleep(2);
                }
                ntail = (uint32_t)v;
            }
            if (ht) {
                unsigned long long *pw = &tpub[((size_t)par * 2 + 1) * nl + t_lane];
                unsigned long long v;
                while (((v = ld_dev(pw)) >> 32) != tagw) {
                    if (++spins > kSpinLimit) {
                        stuck = true;
                        break;
                    }
                    __builtin_amdgcn_s_sleep(2);
                }
                npk = (uint32_t)v;
            }
            // in batches, so that the loads of a batch are in flight together
            constexpr int kB = 8;
            for (uint32_t i0 = tkn; hs && i0 != ntail;) {
                const uint32_t nb = ntail - i0 < (uint32_t)kB ? ntail - i0 : (uint32_t)kB;
                uint32_t ex[kB], er[kB], ep[kB];
                int32_t nh[kB];
#pragma unroll
                for (int q = 0; q < kB; q++)
                    if ((uint32_t)q < nb) {
                        uint32_t *e = ring + 4 * (size_t)(s_fb + ((i0 + q) & s_fm));
                        ex[q] = ld_dev(e);
                        er[q] = ld_dev(e + 1);
                        ep[q] = ld_dev(e + 2);
                    }
#pragma unroll
                for (int q = 0; q < kB; q++)
                    if ((uint32_t)q < nb) nh[q] = path[ep[q] + 1];
#pragma unroll
                for (int q = 0; q < kB; q++)
                    if ((uint32_t)q < nb) sring[s_lo + ((i0 + q) & s_fm)] = make_uint4(ex[q], er[q], ep[q], (uint32_t)nh[q]);
                i0 += nb;
            }
            for (uint32_t i0 = pk; ht && i0 != npk;) {
                const uint32_t nb = npk - i0 < (uint32_t)kB ? npk - i0 : (uint32_t)kB;
                uint32_t dc[kB];
#pragma unroll
                for (int q = 0; q < kB; q++)
                    if ((uint32_t)q < nb) dc[q] = ld_dev(ring + 4 * (size_t)(t_fb + ((i0 + q) & t_fm)) + 3);
#pragma unroll
                for (int q = 0; q < kB; q++)
                    if ((uint32_t)q < nb) cring[t_co + ((i0 + q) & t_fm)] = dc[q];
                i0 += nb;
            }
            tkn = ntail;
            pk = npk;
        }
        if (stuck) red[20] = 1u;
        __syncthreads();
        const uint32_t nxt = red[16];
        const uint32_t flags = red[17];
        widx++;
        if (red[20]) {
            state = kRunWatchdog;
        } else if (flags & 2u) {
            state = kRunMaxCycles;
        } else if (!(flags & 1u)) {
            state = kRunOk;
        } else if (nxt == kNever) {
            state = kRunDeadlock;
        } else {
            T0 = nxt;
        }
        if (state == kRunRunning && (uint64_t)T0 > d.max_cycles) state = kRunMaxCycles;
        if (state == kRunRunning && local_cycles > d.watchdog) state = kRunWatchdog;
        __syncthreads();
    }
    if (ht) {
        d.tx_lines[t_link] = tx;
        d.busy[t_link] = tx;
    }
    // makespan: the largest completion of any workgroup
    {
        uint32_t v = maxcomp;
#pragma unroll
        for (int sh = 32; sh >= 1; sh >>= 1) {
            const uint32_t u = (uint32_t)__shfl_xor((int)v, sh);
            v = u > v ? u : v;
        }
        if ((tid & 63) == 0 && v) atomicMax(&d.makespan[0], v);
    }
    if (tid == 0) {
        atomicMax(&d.status[0], state);
        atomicMax(reinterpret_cast<unsigned long long *>(&d.cycles[0]), (unsigned long long)local_cycles);
    }
}

}  // namespace

hipError_t launch_grid_any(const DevNet &d, hipStream_t st) {
    hipLaunchKernelGGL(grid_init, dim3(64), dim3(256), 0, st, d);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const void *k;
    if (d.gd_window > 0)
        k = d.arb == 0 ? (const void *)engine_gridw<0> : (const void *)engine_gridw<1>;
    else if (d.gd_one)
        k = d.arb == 0 ? (d.has_preds ? (const void *)engine_grid1<0, true> : (const void *)engine_grid1<0, false>)
                       : (d.has_preds ? (const void *)engine_grid1<1, true> : (const void *)engine_grid1<1, false>);
    else
        k = d.arb == 0 ? (d.has_preds ? (const void *)engine_grid<0, true> : (const void *)engine_grid<0, false>)
                       : (d.has_preds ? (const void *)engine_grid<1, true> : (const void *)engine_grid<1, false>);
    if (d.lds_bytes > 65536) (void)hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, d.lds_bytes);
    DevNet arg = d;
    void *args[] = {&arg};
    return hipLaunchCooperativeKernel(k, dim3((unsigned)(d.gd_nb * d.gd_stride)), dim3((unsigned)d.gd_threads), args,
                                      (unsigned)d.lds_bytes, st);
}

}  // namespace simgpu
