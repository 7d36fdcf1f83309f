#include <hip/hip_runtime.h>

#include "engine_common.h"

namespace simgpu {

namespace {

using namespace dev;

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
    // delivered counters: in LDS whenever lines have predecessors (the host
    // declines this engine otherwise)
    uint32_t *deliv = reinterpret_cast<uint32_t *>(smem + d.o_b1deliv);
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
        // First every lane completes last cycle's appended entry and issues
        // the head reloads it needs, then the heads are used.  The memory
        // counter also counts stores, so one explicit wait here (for last
        // cycle's next-hop loads, long complete) keeps the compiler from
        // waiting on each lane's store before the next lane's; the reloads
        // are then waited for once.
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
#pragma unroll
        for (int q = 0; q < LPT; q++) {
            const int lane = tid + q * NT;
            // the lane's constants are re-derived each cycle rather than kept
            // (hoisted) in spilled registers
            asm volatile("" : "+v"(pa[q]), "+v"(pb[q]));
            st8[q] &= 0x9FFu;
            if (st8[q] & 2048u) {
                // complete the entry appended last cycle with its next hop
                const uint32_t last = (tail[q] - 1u) & rmask;
                reinterpret_cast<int32_t *>(fifo + ((size_t)lane << lg) + last)[3] = ntg[q];
                if ((st8[q] & 256u) && head[q] == tail[q] - 1u) ctg[q] = ntg[q];
                st8[q] &= ~2048u;
            }
            if (lane < nl && tail[q] != head[q] && !(st8[q] & 256u)) {
                const uint4 e = fifo[((size_t)lane << lg) + (head[q] & rmask)];
                cx[q] = e.x;
                cpp[q] = e.y;
                crdy[q] = e.z;
                ctg[q] = (int32_t)e.w;
                st8[q] |= 256u;
            }
        }
#pragma unroll
        for (int q = 0; q < LPT; q++) {
            const int lane = tid + q * NT;
            if (lane < nl && tail[q] != head[q]) {
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
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): R's stores and reloads
        bool sdep = false;
        // lane-derived addresses are recomputed here rather than kept
        // (hoisted) in spilled registers
        int tq = tid;
        asm volatile("" : "+v"(tq));
#pragma unroll
        for (int q = 0; q < LPT; q++) {
            const int lane = tq + q * NT;
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
        // Departures first (completion stores included), then the next heads'
        // loads, so that no lane's store waits behind another lane's load.
        int dep = 0;
        uint32_t gmask = 0;
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
                gmask |= 1u << q;
            }
        }
#pragma unroll
        for (int q = 0; q < LPT; q++) {
            const int lane = tid + q * NT;
            // fetch the next head now (used next cycle) unless it is the
            // entry appended this cycle, which is completed next cycle
            if (((gmask >> q) & 1u) && tail[q] != head[q] && !((st8[q] & 2048u) && head[q] == tail[q] - 1u)) {
                const uint4 e = fifo[((size_t)lane << lg) + (head[q] & rmask)];
                cx[q] = e.x;
                cpp[q] = e.y;
                crdy[q] = e.z;
                ctg[q] = (int32_t)e.w;
                st8[q] |= 256u;
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

hipError_t launch_b1_any(const DevNet &d, hipStream_t st) {
    return d.arb == 0 ? launch_b1<0>(d, st) : launch_b1<1>(d, st);
}

}  // namespace simgpu
