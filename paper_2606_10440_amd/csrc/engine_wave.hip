// ----------------------------------------------------------------------------
// Wave engine: many small scenarios, several per wavefront.
//
// Lane w of a wavefront simulates traffic link i = w mod nl of scenario slot
// g = w / nl, so a wave advances G = 64 / nl scenarios in lockstep, each with
// its own clock.  A workgroup holds up to 8 such waves, independent of each
// other, each with an LDS region sized for its own scenarios' rings; the
// host packs the waves so that a device-full of workgroups holds them all.
// A lane keeps its link's FIFO ring in
// LDS (8-byte entries {line << 7 | local flow << 5, ready cycle}) and its
// head entries, injection stream, round-robin pointer and counters in
// registers.  At most four flows cross a link; a lane's local-flow table is
// one register of four bytes (next lane, and the flow's local index there;
// a flow's last link names its own lane), so no path table is read inside
// the cycle loop.  A flow's delivered
// counter is kept by the lane of its last link, at (lane, local index).
//
// The LDS operations of one wavefront are performed in issue order, so a
// value one lane writes is seen by every later read of any lane of the same
// wave: the phases of a cycle are separated by compiler barriers only, and
// the only waits are for the data a phase consumes.  A single wave issues at
// most one instruction every four clocks, so the loops avoid divergent
// branches in the common path: a lane with nothing to store writes to a
// trash slot of its own instead of branching around the store.
//
// Two cycle loops:
//   b = 1, lowest id   every requester takes the atomic minimum of its key
//                      (line << 7 | local flow at the target << 5 | 1) on the
//                      target's word; the word was reset at the end of the
//                      previous cycle to "empty" or, when the link is full,
//                      to 0, which no key beats.  A requester departs iff the
//                      word holds its key, the target appends the line the
//                      word names.  One LDS round trip decides a cycle.
//   general            requests go to fixed slots (feeder, k) of the target,
//                      stamped with the cycle's tag so that no slot is ever
//                      cleared.  The target sorts each feeder's requests with
//                      a sorting network, merges them with its stream's
//                      (already ordered) offers keeping the b first, writes
//                      the grant ranks and appends the granted lines at once.
//                      Sources depart their longest granted prefix; a grant
//                      behind a refused line (void) is reported back and its
//                      target compacts the appended lines, in a pass the wave
//                      runs only when some lane has a void.
// Completion stores to HBM are never waited for; the rare global loads of a
// new stream range are drained where they are made, so the loop itself holds
// no wait on the memory counter.

#include <hip/hip_runtime.h>

#include <type_traits>

#include "engine_common.h"

namespace simgpu {

namespace {

using namespace dev;

constexpr uint32_t kWordEmpty = 0xFFFFFFFFu;
constexpr uint32_t kWordFull = 0u;
constexpr uint32_t kXs = kWaveXShift;  // line id position in an entry word

// Compiler-only barrier between the phases of a cycle: a wavefront-scope
// fence emits no instruction and no wait, but keeps LDS accesses in order.
__device__ __forceinline__ void cbar() { __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront"); }
// wait for every outstanding global load/store of this wave (vmcnt(0))
__device__ __forceinline__ void vm_drain() { __builtin_amdgcn_s_waitcnt(0x0F70); }

__device__ __forceinline__ uint32_t byte_of(uint32_t v, uint32_t q) { return __builtin_amdgcn_ubfe(v, q * 8u, 8u); }

// Whole-wave DPP shifts by one lane, register to register: lane w receives
// lane w - 1's value (from_below) or lane w + 1's (from_above); the end lane
// keeps `old`.  A lane that is inactive during the shift hands on `old`
// instead of its value, so a shift must run with every lane active: the
// empty volatile asm on the result pins the shift where it is written (on a
// path every lane takes), so that the compiler cannot move it into a branch.
__device__ __forceinline__ uint32_t from_below(uint32_t v, uint32_t old) {
    uint32_t r = (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, 0x138, 0xF, 0xF, false);  // wave_shr:1
    asm volatile("" : "+v"(r));
    return r;
}
__device__ __forceinline__ uint32_t from_above(uint32_t v, uint32_t old) {
    uint32_t r = (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, 0x130, 0xF, 0xF, false);  // wave_shl:1
    asm volatile("" : "+v"(r));
    return r;
}

__device__ __forceinline__ uint32_t wrap_add(uint32_t a, uint32_t n, uint32_t cap) {
    const uint32_t v = a + n;
    return v >= cap ? v - cap : v;
}

// A stream's current id range: its lines, local flow, and its first two
// predecessor descriptors (delivered-counter index, base); np counts all.
struct WRange {
    uint32_t start, len, lf, np;
    int32_t pd0;
    uint32_t ix0, ix1, pb0, pb1;
};

__device__ __forceinline__ void load_wrange(const DevNet &d, int R, WRange &r) {
    r.start = d.r_start[R];
    r.len = d.r_len[R];
    r.lf = (uint32_t)d.r_lf[R];
    r.pd0 = d.r_pd[R];
    const int pd1 = d.r_pd[R + 1];
    r.np = (uint32_t)(pd1 - r.pd0);
    r.ix0 = r.np > 0 ? (uint32_t)d.pd_dix[r.pd0] : 0u;
    r.pb0 = r.np > 0 ? d.pd_base[r.pd0] : 0u;
    r.ix1 = r.np > 1 ? (uint32_t)d.pd_dix[r.pd0 + 1] : 0u;
    r.pb1 = r.np > 1 ? d.pd_base[r.pd0 + 1] : 0u;
    vm_drain();
}

// Lines released by one predecessor whose flow has delivered v lines, from
// a line that waits for more than bb: v - bb per line (each further line
// waits for one more), all of them per chunk (CH).
template <bool CH>
__device__ __forceinline__ uint32_t pred_allows(uint32_t v, uint32_t bb) {
    return v > bb ? (CH ? 0xFFFFFFFFu : v - bb) : 0u;
}

// Lines of range r from offset o on whose predecessors have all been
// delivered (a prefix: the counts only grow with o), capped at n.  dv0/dv1
// hold the first two predecessors' delivered counts as of the cycle start.
// CH: per-chunk dependencies (every base is the whole chunk's; no offset).
template <bool CH>
__device__ __forceinline__ uint32_t released_count(const DevNet &d, const WRange &r, uint32_t o, uint32_t n,
                                                   uint32_t dv0, uint32_t dv1, const uint32_t *deliv) {
    const uint32_t oo = CH ? 0u : o;
    n = r.np > 0 ? min(n, pred_allows<CH>(dv0, r.pb0 + oo)) : n;
    n = r.np > 1 ? min(n, pred_allows<CH>(dv1, r.pb1 + oo)) : n;
    if ((n != 0u) & (r.np > 2)) {
        for (int idx = r.pd0 + 2; idx < r.pd0 + (int)r.np; idx++)
            n = min(n, pred_allows<CH>(deliv[d.pd_dix[idx]], d.pd_base[idx] + oo));
        vm_drain();
    }
    return n;
}

// Whether line o of range r is released (released_count for one line).
template <bool CH>
__device__ __forceinline__ bool released_one(const DevNet &d, const WRange &r, uint32_t o, uint32_t dv0, uint32_t dv1,
                                             const uint32_t *deliv) {
    const uint32_t oo = CH ? 0u : o;
    bool ok = ((r.np < 1u) | (dv0 > r.pb0 + oo)) & ((r.np < 2u) | (dv1 > r.pb1 + oo));
    if (ok & (r.np > 2u)) {
        for (int idx = r.pd0 + 2; idx < r.pd0 + (int)r.np; idx++)
            ok = ok & (deliv[d.pd_dix[idx]] > d.pd_base[idx] + oo);
        vm_drain();
    }
    return ok;
}

// Same from offset 0, with the delivered counts read from LDS (a range
// entered in the middle of a cycle).
template <bool CH>
__device__ __forceinline__ uint32_t released_direct(const DevNet &d, const WRange &r, uint32_t n,
                                                    const uint32_t *deliv) {
    for (int idx = r.pd0; idx < r.pd0 + (int)r.np; idx++)
        n = min(n, pred_allows<CH>(deliv[d.pd_dix[idx]], d.pd_base[idx]));
    vm_drain();
    return n;
}

// Compare-exchange and sorting networks on register arrays (indices are
// compile-time after unrolling).
template <typename K>
__device__ __forceinline__ void cex(K &a, K &b) {
    const K lo = a < b ? a : b;
    const K hi = a < b ? b : a;
    a = lo;
    b = hi;
}

// Batcher's odd-even merge sort, ascending.
template <typename K, int N>
__device__ __forceinline__ void sort_net(K (&a)[N]) {
#pragma unroll
    for (int p = 1; p < N; p <<= 1)
#pragma unroll
        for (int k = p; k >= 1; k >>= 1)
#pragma unroll
            for (int j = k % p; j + k < N; j += 2 * k)
#pragma unroll
                for (int i = 0; i < k; i++)
                    if (i + j + k < N && (i + j) / (2 * p) == (i + j + k) / (2 * p)) cex(a[i + j], a[i + j + k]);
}

// a, b ascending -> a = the N smallest of both, ascending.
template <typename K, int N>
__device__ __forceinline__ void merge_low(K (&a)[N], const K (&b)[N]) {
#pragma unroll
    for (int i = 0; i < N; i++) a[i] = a[i] < b[N - 1 - i] ? a[i] : b[N - 1 - i];
#pragma unroll
    for (int k = N / 2; k >= 1; k >>= 1)
#pragma unroll
        for (int i = 0; i < N; i++)
            if ((i & k) == 0) cex(a[i], a[i + k]);
}

// NF: request-slot groups per target lane (feeders, then the lane's own
// stream in group NF - 1).  CH: per-chunk step dependencies.  CR: credit
// delays -- a line that leaves keeps its ring slot, with the cycle it left
// in place of its ready time, until its credit is back.
template <int BM, int ARB, int NF, bool CH, bool CR>
__global__ void __launch_bounds__(64 * kWaveMaxWpb) engine_wave(DevNet d) {
    extern __shared__ __align__(16) unsigned char smem[];
    // the workgroup's waves are independent: each has its own LDS region and
    // never waits for the others
    const int slot = blockIdx.x * d.wv_wpb + (threadIdx.x >> 6);
    const int wave = d.blk_wave[slot];
    if (wave < 0) return;
    unsigned char *base = smem + d.blk_off[slot];
    uint2 *ring = reinterpret_cast<uint2 *>(base);  // the wave's rings, then one trash entry per lane

    const int w = threadIdx.x & 63;
    const int nl = d.nl;
    const int G = d.wv_G;
    const int m = d.m;
    const int g = w / nl;
    const int i = w - g * nl;
    const int gl0 = g * nl;
    const int s = g < G ? d.wv_sc[(size_t)wave * G + g] : -1;
    const bool on = s >= 0;

    // lane registers
    int link = 0, b = 1;
    uint32_t L = 1, cap = 1, P = 1;
    uint32_t D = 1;  // credit delay (CR)
    uint32_t lfb = 0, lfx = 0;  // local-flow tables (one byte per local flow)
    uint32_t fl = 0, fp = 0;    // feeder wave lanes and their ports, one byte each
    int R = 0, rend = 0;
    uint32_t o = 0;
    WRange cur{};
    bool feed1 = false;  // the lane's link has exactly one feeder
    if (on) {
        link = d.ln_link[i];
        const size_t pi = (size_t)s * m + link;
        b = d.bw[pi];
        L = (uint32_t)d.lat[pi];
        cap = (uint32_t)d.cap[pi];
        if constexpr (CR) D = (uint32_t)d.credit[pi];
        P = (uint32_t)d.ln_P[i];
        lfb = d.wv_lfb[i];
        lfx = d.wv_lfx[i];
        const int nfeed = d.wv_nfeed[i];
        for (int f = 0; f < nfeed; f++) {
            const uint32_t v = (uint32_t)d.wv_feed[4 * i + f];
            fl |= (((v & 0xFFu) + (uint32_t)gl0) & 0xFFu) << (8 * f);
            fp |= ((v >> 8) & 0xFFu) << (8 * f);
        }
        R = d.ln_srbeg[i];
        rend = d.ln_srend[i];
        feed1 = nfeed == 1;
        if (R < rend) load_wrange(d, R, cur);
    }
    // this lane's ring: exclusive prefix sum over the wave of the capacities,
    // each padded so that lane w's ring starts at an entry = w (mod 16): ring
    // heads that advance in step then fall in different LDS banks
    const uint32_t ralloc = (on ? cap : 0u) + ((1u - (on ? cap : 0u)) & 15u);
    uint32_t incl = ralloc;
#pragma unroll
    for (int sh = 1; sh < 64; sh <<= 1) {
        const uint32_t u = (uint32_t)__shfl_up((int)incl, sh);
        if (w >= sh) incl += u;
    }
    const uint32_t rbase = incl - ralloc;
    const uint32_t rtotal = (uint32_t)__shfl((int)incl, 63);
    unsigned char *tailp = base + (((rtotal + 64u) * 8u + 15u) & ~15u);
    uint32_t *word = reinterpret_cast<uint32_t *>(tailp + d.o_wword);        // [128]
    uint32_t *red = reinterpret_cast<uint32_t *>(tailp + d.o_wred);          // [64 + 64 trash]
    uint32_t *deliv_all = reinterpret_cast<uint32_t *>(tailp + d.o_wdeliv);  // [G*nl*4]
    uint32_t *deliv = deliv_all + (size_t)(g < G ? g : 0) * nl * 4;
    const uint32_t mydx = (uint32_t)i * 4u;  // this lane's delivered counters
    // trash slots: a lane with nothing to store writes here
    const uint32_t ring_trash = rtotal + (uint32_t)w;
    constexpr bool kFast = ARB == 0;             // the b = 1 lowest-id loop exists
    constexpr bool kGeneral = BM > 1 || ARB == 1;  // the general loop exists
    const bool lined = !CR && d.wv_lineup != 0;  // the shift loop runs instead
    const bool fast = kFast && !lined && (!kGeneral || __ballot(on && b != 1) == 0ull);
    // the wave's bandwidth bound: its general loop is unrolled to that width
    int wbm = on ? b : 1;
#pragma unroll
    for (int sh = 32; sh >= 1; sh >>= 1) wbm = max(wbm, __shfl_xor(wbm, sh));

    for (int j = w; j < G * nl * 4; j += 64) deliv_all[j] = 0;
    word[w] = kWordEmpty;
    word[64 + w] = kWordEmpty;
    red[w] = kNever;
    red[64 + w] = kNever;
    // links without traffic report zero counters
    for (int gg = 0; gg < G; gg++) {
        const int ss = d.wv_sc[(size_t)wave * G + gg];
        if (ss < 0) continue;
        for (int j = w; j < m; j += 64)
            if (d.link_lane[j] < 0) {
                d.tx_lines[(size_t)ss * m + j] = 0;
                d.busy[(size_t)ss * m + j] = 0;
            }
    }
    vm_drain();
    cbar();

    uint32_t *comp = d.completion + (size_t)(on ? s : 0) * (size_t)d.T;
    // this lane's scenario as a mask of wave lanes
    const unsigned long long smask = (nl >= 64 ? ~0ull : ((1ull << nl) - 1ull)) << gl0;
    uint32_t t = 0;
    uint32_t processed = 0;  // every processed cycle advances t, so this fits 32 bits
    bool live = on && d.T > 0;
    int32_t state = live ? kRunRunning : kRunOk;
    uint32_t occ = 0, head = 0, tail = 0, rr = 0;
    // CR: owed credits are the ring entries ch .. head-1; crt = cycle the
    // oldest comes back (credits come back in the order the lines left)
    uint32_t owed = 0, ch = 0, crt = kNever;
    uint64_t tx = 0, busy = 0;
    uint32_t dv0 = 0, dv1 = 0;
    // a line id outside [0, T) can only come from an engine fault: the store
    // is skipped and the scenario ends with kRunInternal
    const uint32_t Tu = (uint32_t)d.T;
    bool bad = false;
    const uint32_t maxc = d.max_cycles > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)d.max_cycles;
    const uint32_t wdog = d.watchdog > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)d.watchdog;

    // the stream's current range is done: move to the next non-empty one
    auto next_range = [&]() {
        while (R < rend && o >= cur.len) {
            o -= cur.len;
            R++;
            if (R < rend) load_wrange(d, R, cur);
        }
    };
    // delivered counts of the stream's first two predecessors, as of the
    // start of the next cycle (read only while some lane of the wave needs them)
    auto refresh_dv = [&]() {
        if (__ballot(cur.np > 0u) != 0ull) dv0 = deliv[cur.ix0];
        if (__ballot(cur.np > 1u) != 0ull) dv1 = deliv[cur.ix1];
    };
    // CR: slots whose credit is back by the (new) cycle t are free again
    auto credits_back = [&]() {
        bool pop = live & (owed != 0u) & (crt <= t);
        while (__ballot(pop) != 0ull) {
            if (pop) {
                ch = wrap_add(ch, 1u, cap);
                owed -= 1u;
                crt = owed != 0u ? ring[rbase + ch].y + D : kNever;
            }
            pop = live & (owed != 0u) & (crt <= t);
        }
    };
    // End of cycle: clock and status of every scenario of the wave.  nxt is
    // the lane's FIFO-head ready time if still in the future at the start of
    // the cycle; a scenario in which nothing departed jumps to the minimum of
    // its lanes' nxt, rv, which the caller took during the cycle (an LDS
    // atomic minimum issued with the requests).
    auto time_phase = [&](bool dep, uint32_t rv) {
        const bool act = live & ((occ != 0u) | (R < rend));
        const bool sdep = (__ballot(dep) & smask) != 0ull;
        const bool sact = (__ballot(act) & smask) != 0ull;
        const uint32_t tn = sdep ? t + 1u : rv;
        processed += live ? 1u : 0u;
        const bool go = sact & (sdep | (rv != kNever)) & (tn <= maxc) & (processed <= wdog);
        if (live & !go) {  // the scenario ends this cycle
            int32_t st = kRunWatchdog;
            st = (tn > maxc) ? kRunMaxCycles : st;
            st = (!sdep & (rv == kNever)) ? kRunDeadlock : st;
            st = !sact ? kRunOk : st;
            state = st;
            live = false;
        }
        t = live ? tn : t;
        if (__ballot(bad) != 0ull) {  // engine fault: end the faulty scenarios
            const bool sbad = (__ballot(bad) & smask) != 0ull;
            if (sbad & on) {
                state = kRunInternal;
                live = false;
            }
        }
    };

    // Shift loop, for graphs whose links form paths laid out on consecutive
    // lanes: a link is fed by the lane below it (if by any link) plus,
    // possibly, its own injection stream, and sends the lines that go on to
    // the lane above it.  A link's arbitration then merges two ordered
    // lists -- its feeder's lines bound for it, in the feeder's offer order
    // (id order: one flow under lowest id), and its stream's released lines
    // -- and takes the first min(b, free, both); the feeder's taken lines are
    // the first of its lines bound there, so no grant is void.  Requests move
    // one lane up and the number taken one lane down by DPP shifts, register
    // to register: a cycle needs no LDS round trip.  The target appends the
    // merged lines to its ring in LDS; with one line per cycle the first two
    // FIFO entries stay in registers and the ring is read a cycle ahead.
    //
    // Cycles run through a lean body while every lane's next cycle is a
    // common one: the stream offer stays inside the current range and needs
    // at most two predecessor counts, and every scenario moves a line and
    // goes on.  Otherwise one cycle runs through the complete body (range
    // changes, more predecessors, jumps over idle cycles, a scenario's end).
    auto lineup = [&](auto bmw_tag) {
        constexpr int BMW = decltype(bmw_tag)::value;
        const uint32_t tmask = on ? d.wv_duo[i] : 0u;  // local flows bound for the lane above
        const uint32_t fport = fp & 0xFFu;              // the feeder's port here
        uint2 e[BMW];  // first FIFO entries (meaningful for k < min(occ, b))
#pragma unroll
        for (int k = 0; k < BMW; k++) e[k] = make_uint2(0u, 0u);
        uint2 e1 = make_uint2(0u, 0u);   // BMW == 1: the second entry (occ >= 2) ...
        uint2 e1l = make_uint2(0u, 0u);  // ... or, when pend, the ring read that holds it
        bool pend = false;
        uint32_t tx32 = 0, busy32 = 0;   // link counters of this launch (below 2^32: at most T lines)
        // The time advance of a cycle that is not the common one: a scenario
        // in which nothing moved jumps to its earliest future FIFO-head ready
        // time (nxt: this lane's, as of the cycle's start); scenarios end.
        auto slow_time = [&](bool sdep, bool sact, uint32_t nxt) {
            uint32_t rv = kNever;
            if (__ballot(live & !sdep) != 0ull) {
                cbar();
                atomicMin(&red[nxt != kNever ? (uint32_t)g : 64u + (uint32_t)w], nxt);
                cbar();
                rv = red[g];
                cbar();
                red[i == 0 ? (uint32_t)g : 64u + (uint32_t)w] = kNever;
            }
            const uint32_t tn = sdep ? t + 1u : rv;
            const bool go = sact & (tn != kNever) & (tn <= maxc) & (processed <= wdog);
            if (live & !go) {
                int32_t st = kRunWatchdog;
                st = (tn > maxc) ? kRunMaxCycles : st;
                st = (!sdep & (rv == kNever)) ? kRunDeadlock : st;
                st = !sact ? kRunOk : st;
                state = st;
                live = false;
            }
            t = live ? tn : t;
        };
        // One cycle.  FULL: the complete body; else the lean one, valid when
        // no lane needs the complete one.  Returns whether the next cycle can
        // run through the lean body.
        auto cycle = [&](auto full_tag) -> bool {
            constexpr bool FULL = decltype(full_tag)::value;
            const uint32_t e_y0 = e[0].y;  // the head's ready time at the cycle's start
            const uint32_t occ0 = occ, head0 = head;
            // ---------------------------------------------------------- FIFO offer
            uint32_t noff = 0, kmask = 0;
            uint32_t up[BMW];  // offered lines as entry words at the lane above
            {
                bool open = live;
#pragma unroll
                for (int k = 0; k < BMW; k++) {
                    open = open & (k < b) & ((uint32_t)k < occ) & (e[k].y <= t);
                    noff += open ? 1u : 0u;
                    const uint32_t q = (e[k].x >> 5) & 3u;
                    kmask |= (open & (((tmask >> q) & 1u) != 0u)) ? 1u << k : 0u;
                    up[k] = (e[k].x & ~0x7Fu) | ((byte_of(lfb, q) >> 6) << 5);
                }
            }
            // ---------------------------------------------------------- the feeder's lines, up one lane
            uint32_t fe[BMW];
#pragma unroll
            for (int k = 0; k < BMW; k++) fe[k] = from_below(up[k], 0u);
            const uint32_t fkm = from_below(kmask, 0u) & (feed1 ? ~0u : 0u);
            // ---------------------------------------------------------- stream offer
            uint32_t sword[BMW];
#pragma unroll
            for (int k = 0; k < BMW; k++) sword[k] = ((cur.start + o + k) << kXs) | (cur.lf << 5);
            uint32_t nS;
            if constexpr (FULL) {
                nS = (live & (R < rend)) ? released_count<CH>(d, cur, o, min((uint32_t)b, cur.len - o), dv0, dv1, deliv)
                                         : 0u;
                if ((nS == cur.len - o) & (nS < (uint32_t)b) & (R + 1 < rend) & live) {
                    // the offer runs into the ranges after the current one
                    int sR = R + 1;
                    WRange sr;
                    while (sR < rend && nS < (uint32_t)b) {
                        load_wrange(d, sR, sr);
                        const uint32_t n = released_direct<CH>(d, sr, min((uint32_t)b - nS, sr.len), deliv);
#pragma unroll
                        for (int k = 0; k < BMW; k++)
                            if (((uint32_t)k >= nS) & ((uint32_t)k < nS + n))
                                sword[k] = ((sr.start + (uint32_t)k - nS) << kXs) | (sr.lf << 5);
                        nS += n;
                        if (n < sr.len) break;
                        sR++;
                    }
                }
            } else {
                // at most two predecessors, inside the range (the caller checked)
                const uint32_t oo = CH ? 0u : o;
                uint32_t n = (live & (R < rend)) ? (uint32_t)b : 0u;
                n = cur.np > 0u ? min(n, pred_allows<CH>(dv0, cur.pb0 + oo)) : n;
                n = cur.np > 1u ? min(n, pred_allows<CH>(dv1, cur.pb1 + oo)) : n;
                nS = n;
            }
            // ---------------------------------------------------------- arbitration
            const uint32_t nF = (uint32_t)__builtin_popcount(fkm);
            const uint32_t G = live ? min(min((uint32_t)b, cap - occ), nF + nS) : 0u;
            const uint32_t rotf = fport >= rr ? fport - rr : fport + P - rr;
            const uint32_t rots = (P - 1u) >= rr ? P - 1u - rr : P - 1u + P - rr;
            uint32_t gF = 0, gS = 0, lastS = 0;
            uint32_t Ex = 0;  // BMW == 1: the entry word appended
            const uint32_t ready = t + L;
            // Lowest id, several lines: each list is in id order, and when the
            // two do not interleave (the usual case: each is a run of one flow's
            // lines) one lies wholly before the other, so the ranks need no
            // pairwise comparisons.  first: 1 feeder's list first, 2 the
            // stream's, 0 interleaved (compare pairwise).
            uint32_t first = 0;
            if constexpr (ARB == 0 && BMW > 2) {
                uint32_t fmin = 0xFFFFFFFFu, fmax = 0u;
#pragma unroll
                for (int k = 0; k < BMW; k++) {
                    const bool tb = ((fkm >> k) & 1u) != 0u;
                    fmin = tb ? min(fmin, fe[k]) : fmin;
                    fmax = tb ? max(fmax, fe[k]) : fmax;
                }
                const uint32_t smin = sword[0], smax = sword[nS > 0u ? nS - 1u : 0u];
                first = ((nS == 0u) | (fmax < smin)) ? 1u : (((nF == 0u) | (smax < fmin)) ? 2u : 0u);
            }
            const bool pairwise = ARB == 0 && (BMW <= 2 || __ballot(first == 0u) != 0ull);
#pragma unroll
            for (int k = 0; k < BMW; k++) {  // the feeder's lines bound here (positions in fkm)
                const bool tb = ((fkm >> k) & 1u) != 0u;
                const uint32_t j = (uint32_t)__builtin_popcount(fkm & ((1u << k) - 1u));
                uint32_t ahead;
                if constexpr (ARB == 0) {
                    ahead = first == 2u ? nS : 0u;
                    if (pairwise) {
                        ahead = 0;
#pragma unroll
                        for (int y = 0; y < BMW; y++) ahead += (((uint32_t)y < nS) & (sword[y] < fe[k])) ? 1u : 0u;
                    }
                } else {
                    ahead = min(nS, (uint32_t)k + (rots < rotf ? 1u : 0u));
                }
                const uint32_t rank = j + ahead;
                const bool gk = tb & (rank < G);
                ring[gk ? rbase + wrap_add(tail, rank, cap) : ring_trash] = make_uint2(fe[k], ready);
                gF += gk ? 1u : 0u;
                if (BMW == 1) Ex = gk ? fe[k] : Ex;
            }
#pragma unroll
            for (int k = 0; k < BMW; k++) {  // the stream's lines
                uint32_t ahead;
                if constexpr (ARB == 0) {
                    ahead = first == 1u ? nF : 0u;
                    if (pairwise) {
                        ahead = 0;
#pragma unroll
                        for (int y = 0; y < BMW; y++)
                            ahead += ((((fkm >> y) & 1u) != 0u) & (fe[y] < sword[k])) ? 1u : 0u;
                    }
                } else {
                    const uint32_t lim = (uint32_t)k + (rotf < rots ? 1u : 0u);
                    ahead = (uint32_t)__builtin_popcount(fkm & (lim >= 32u ? ~0u : (1u << lim) - 1u));
                }
                const uint32_t rank = (uint32_t)k + ahead;
                const bool gk = ((uint32_t)k < nS) & (rank < G);
                ring[gk ? rbase + wrap_add(tail, rank, cap) : ring_trash] = make_uint2(sword[k], ready);
                gS += gk ? 1u : 0u;
                lastS = gk ? rank + 1u : lastS;
                if (BMW == 1) Ex = gk ? sword[k] : Ex;
            }
            // ---------------------------------------------------------- the lines taken, down one lane
            const uint32_t got = from_above(gF, 0u);
            uint32_t gout = 0, ejd = 0;
            {
                bool open = true;
#pragma unroll
                for (int k = 0; k < BMW; k++) {
                    const bool tb = ((kmask >> k) & 1u) != 0u;
                    const uint32_t j = (uint32_t)__builtin_popcount(kmask & ((1u << k) - 1u));
                    const bool dk = open & ((uint32_t)k < noff) & (!tb | (j < got));
                    open = dk;
                    gout += dk ? 1u : 0u;
                    ejd |= (dk & !tb) ? 1u << k : 0u;
                }
            }
            if (ejd) {
#pragma unroll
                for (int k = 0; k < BMW; k++) {
                    if ((ejd >> k) & 1u) {
                        const uint32_t x = e[k].x >> kXs;
                        bad |= x >= Tu;
                        comp[x < Tu ? x : 0u] = t + 1u;
                        atomicAdd(&deliv[mydx + ((e[k].x >> 5) & 3u)], 1u);
                    }
                }
            }
            if (ARB == 1 && G != 0u) {  // past the port of the last line appended
                const uint32_t lp = lastS == G ? P - 1u : fport;
                rr = lp + 1u == P ? 0u : lp + 1u;
            }
            // ---------------------------------------------------------- FIFO and stream state
            head = wrap_add(head, gout, cap);
            tail = wrap_add(tail, G, cap);
            occ = occ + G - gout;
            tx32 += G;
            busy32 += G ? 1u : 0u;
            o += gS;
            if constexpr (FULL) {
                if (o >= cur.len) next_range();
            }
            if constexpr (BMW == 1) {
                // the first two entries: kept, moved down by a pop, the line just
                // appended, or (entry 1 after a pop with three or more lines)
                // read from the ring now and used no earlier than the next
                // cycle's end
                const uint2 E = make_uint2(Ex, ready);
                const uint2 e1v = pend ? e1l : e1;
                const bool pop = gout != 0u;
                const uint2 n0 = pop ? (occ0 >= 2u ? e1v : E) : (occ0 >= 1u ? e[0] : E);
                const uint2 n1 = pop ? (occ0 == 2u ? E : e1v) : (occ0 == 1u ? E : e1v);
                e1l = ring[rbase + wrap_add(head0, min(2u, cap - 1u), cap)];
                e[0] = n0;
                e1 = n1;
                pend = pop & (occ0 >= 3u);
            } else {
                cbar();
#pragma unroll
                for (int k = 0; k < BMW; k++) e[k] = ring[rbase + wrap_add(head, min((uint32_t)k, cap - 1u), cap)];
            }
            dv0 = deliv[cur.ix0];  // delivered counts for the next cycle (ix0/ix1 = 0 when unused)
            dv1 = deliv[cur.ix1];
            // ---------------------------------------------------------- time
            const bool dep = (gout | gS) != 0u;
            const bool act = live & ((occ != 0u) | (R < rend));
            const bool sdep = (__ballot(dep) & smask) != 0ull;
            const bool sact = (__ballot(act) & smask) != 0ull;
            processed += live ? 1u : 0u;
            const bool common = sdep & sact & (t + 1u <= maxc) & (processed <= wdog);
            const uint32_t nxt = (live & (occ0 != 0u) & (e_y0 > t)) ? e_y0 : kNever;
            if (__ballot(live & !common) != 0ull) slow_time(sdep, sact, nxt);
            else t = live ? t + 1u : t;
            // the next cycle: the stream's offer inside its range, two predecessors at most
            const bool lean = !live | (R >= rend) | ((o + (uint32_t)b < cur.len) & (cur.np <= 2u));
            return __ballot(!lean) == 0ull;
        };
        // The lean cycle for one line per cycle: one entry word up (none
        // when no line is bound there), one bit down.
        auto cycle1 = [&]() -> bool {
            constexpr uint32_t kNone = 0xFFFFFFFFu;  // above every entry word (line ids < 2^25 - 1)
            const uint32_t hx = e[0].x, hy = e[0].y;
            const uint32_t occ0 = occ, head0 = head;
            const bool hrdy = live & (occ != 0u) & (hy <= t);
            const uint32_t q = (hx >> 5) & 3u;
            const bool upb = ((tmask >> q) & 1u) != 0u;
            const bool tb = hrdy & upb;
            const bool ej = hrdy & !upb;
            const uint32_t fe = from_below(tb ? (hx & ~0x7Fu) | ((byte_of(lfb, q) >> 6) << 5) : kNone, kNone) |
                                (feed1 ? 0u : kNone);
            const uint32_t oo = CH ? 0u : o;
            bool sw = live & (R < rend);
            sw = sw & ((cur.np < 1u) | (pred_allows<CH>(dv0, cur.pb0 + oo) != 0u));
            sw = sw & ((cur.np < 2u) | (pred_allows<CH>(dv1, cur.pb1 + oo) != 0u));
            const uint32_t sx = sw ? ((cur.start + o) << kXs) | (cur.lf << 5) : kNone;
            // the winner: lowest entry word (id), or the first port at or after the pointer
            bool fwin;
            if constexpr (ARB == 0) {
                fwin = fe < sx;
            } else {
                const uint32_t rotf = fport >= rr ? fport - rr : fport + P - rr;
                const uint32_t rots = (P - 1u) >= rr ? P - 1u - rr : P - 1u + P - rr;
                fwin = (fe != kNone) & ((sx == kNone) | (rotf < rots));
            }
            const uint32_t wx = fwin ? fe : sx;
            const bool app = live & (wx != kNone) & (occ < cap);
            const uint32_t ready = t + L;
            ring[app ? rbase + tail : ring_trash] = make_uint2(wx, ready);
            const bool gF = app & fwin;
            const bool gS = app & !fwin;
            const bool got = from_above(gF ? 1u : 0u, 0u) != 0u;
            const bool pop = ej | (tb & got);
            if (ej) {
                const uint32_t x = hx >> kXs;
                bad |= x >= Tu;
                comp[x < Tu ? x : 0u] = t + 1u;
                atomicAdd(&deliv[mydx + q], 1u);
            }
            dv0 = deliv[cur.ix0];  // delivered counts for the next cycle (ix0/ix1 = 0 when unused)
            dv1 = deliv[cur.ix1];
            if (ARB == 1 && app) {
                const uint32_t lp = gS ? P - 1u : fport;
                rr = lp + 1u == P ? 0u : lp + 1u;
            }
            head = pop ? wrap_add(head, 1u, cap) : head;
            tail = app ? wrap_add(tail, 1u, cap) : tail;
            occ = occ + (app ? 1u : 0u) - (pop ? 1u : 0u);
            tx32 += app ? 1u : 0u;
            busy32 += app ? 1u : 0u;
            o += gS ? 1u : 0u;
            // first two entries (as in the complete cycle)
            const uint2 E = make_uint2(wx, ready);
            const uint2 e1v = pend ? e1l : e1;
            const uint2 n0 = pop ? (occ0 >= 2u ? e1v : E) : (occ0 >= 1u ? e[0] : E);
            const uint2 n1 = pop ? (occ0 == 2u ? E : e1v) : (occ0 == 1u ? E : e1v);
            e1l = ring[rbase + wrap_add(head0, min(2u, cap - 1u), cap)];
            e[0] = n0;
            e1 = n1;
            pend = pop & (occ0 >= 3u);
            // time: the common case moves every scenario on by one cycle; any
            // other is left to the caller (slow_time)
            const bool act = live & ((occ != 0u) | (R < rend));
            const bool sdep = (__ballot(pop | gS) & smask) != 0ull;
            const bool sact = (__ballot(act) & smask) != 0ull;
            processed += live ? 1u : 0u;
            const bool common = sdep & sact & (t + 1u <= maxc) & (processed <= wdog);
            if (__ballot(live & !common) != 0ull) slow_time(sdep, sact, (live & (occ0 != 0u) & (hy > t)) ? hy : kNever);
            else t = live ? t + 1u : t;
            const bool lean = !live | (R >= rend) | ((o + 1u < cur.len) & (cur.np <= 2u));
            return __ballot(!lean) == 0ull;
        };
        while (__ballot(live) != 0ull) {
            bool ok = cycle(std::true_type{});
            if constexpr (BMW == 1) {
                while (ok && __ballot(live) != 0ull) ok = cycle1();
            } else {
                while (ok && __ballot(live) != 0ull) ok = cycle(std::false_type{});
            }
        }
        tx += tx32;
        busy += busy32;
        if (__ballot(bad) != 0ull) {  // engine fault: end the faulty scenarios
            const bool sbad = (__ballot(bad) & smask) != 0ull;
            if (sbad & on) state = kRunInternal;
        }
    };
    if (lined) {
        if (wbm <= 1) lineup(std::integral_constant<int, 1>{});
        else if constexpr (BM >= 2) {
            if (wbm <= 2 || BM == 2) lineup(std::integral_constant<int, 2>{});
            else if constexpr (BM >= 4) {
                if (wbm <= 4 || BM == 4) lineup(std::integral_constant<int, 4>{});
                else if constexpr (BM >= 8) lineup(std::integral_constant<int, 8>{});
            }
        }
    }

    // The head entries are re-read from the ring at the end of every cycle,
    // unconditionally: after the cycle's pops and appends the ring holds the
    // next cycle's head, and the read is consumed only by the next cycle.
    if constexpr (kFast) {
      if (fast) {
        uint2 he = make_uint2(0u, 0u);  // head entry
        while (__ballot(live) != 0ull) {
            // ---------------------------------------------------------- requests
            const uint32_t hx = he.x, hr = he.y;
            const bool hrdy = live & (occ != 0u) & (hr <= t);
            const uint32_t q = (hx >> 5) & 3u;
            const uint32_t lb = byte_of(lfb, q);
            const bool sink = (lb & 63u) == (uint32_t)i;  // a last link names itself
            const bool ej = hrdy & sink;
            const bool fw = hrdy & !sink;
            const uint32_t tgw = fw ? (uint32_t)gl0 + (lb & 63u) : 64u + (uint32_t)w;
            const uint32_t fkey = (hx & ~0x7Fu) | ((lb >> 6) << 5) | 1u;
            atomicMin(&word[tgw], fkey);
            const bool sw = live & (R < rend) & released_one<CH>(d, cur, o, dv0, dv1, deliv);
            const uint32_t skey = ((cur.start + o) << kXs) | (cur.lf << 5) | 1u;
            atomicMin(&word[sw ? (uint32_t)w : 64u + (uint32_t)w], skey);
            uint32_t nxt = (live & (occ != 0u) & (hr > t)) ? hr : kNever;
            if constexpr (CR) nxt = min(nxt, (live & (owed != 0u)) ? crt : kNever);
            atomicMin(&red[nxt != kNever ? (uint32_t)g : 64u + (uint32_t)w], nxt);
            cbar();
            const uint32_t wt = word[tgw];
            const uint32_t wm = word[w];
            const uint32_t rv = red[g];
            cbar();
            // ---------------------------------------------------------- commit
            const bool fwon = ej | (fw & (wt == fkey));
            const bool swon = sw & (wm == skey);
            const bool app = live & (wm != kWordEmpty) & (wm != kWordFull);
            if (ej) {
                const uint32_t x = hx >> kXs;
                bad |= x >= Tu;
                comp[x < Tu ? x : 0u] = t + 1u;
                atomicAdd(&deliv[mydx + q], 1u);
            }
            ring[app ? rbase + tail : ring_trash] = make_uint2(wm & ~0x1Fu, t + L);
            if constexpr (CR) {  // the slot stays owed until the credit is back
                ring[fwon ? rbase + head : ring_trash] = make_uint2(hx, t);
                crt = (fwon & (owed == 0u)) ? t + D : crt;
                owed += fwon ? 1u : 0u;
            }
            head = fwon ? wrap_add(head, 1u, cap) : head;
            tail = app ? wrap_add(tail, 1u, cap) : tail;
            occ = occ - (fwon ? 1u : 0u) + (app ? 1u : 0u);
            tx += app ? 1u : 0u;
            o += swon ? 1u : 0u;
            if (o >= cur.len) next_range();
            cbar();
            if constexpr (!CR) word[w] = occ < cap ? kWordEmpty : kWordFull;
            red[i == 0 ? (uint32_t)g : 64u + (uint32_t)w] = kNever;
            he = ring[rbase + head];
            refresh_dv();
            time_phase(fwon | swon, rv);
            if constexpr (CR) {  // fullness at the next processed cycle
                credits_back();
                word[w] = occ + owed < cap ? kWordEmpty : kWordFull;
                cbar();
            }
        }
        busy = tx;  // one line per cycle at most
      }
    }
    // General loop, unrolled to BMW request slots per source and grants per
    // target (BMW >= the wave's largest bandwidth).
    auto general = [&](auto bmw_tag) {
        constexpr int BMW = decltype(bmw_tag)::value;
        uint2 *wreq = reinterpret_cast<uint2 *>(tailp + d.o_wreq);  // [(NF*BMW + 1) * 64] slot-major {entry word, tag}
        constexpr uint32_t kReqSlots = 64u * NF * BMW;
        uint2 *wgnt = reinterpret_cast<uint2 *>(tailp + d.o_wreq + ((kReqSlots + 64u) * 8u + 15u) / 16u * 16u);
        uint32_t *wvoid = reinterpret_cast<uint32_t *>(reinterpret_cast<unsigned char *>(wgnt) +
                                                       ((64u * BMW + 64u) * 8u + 15u) / 16u * 16u);  // [(BMW + 1) * 64] rank-major tag
        const uint32_t req_trash = kReqSlots + (uint32_t)w;
        const uint32_t gnt_trash = 64u * BMW + (uint32_t)w;
        for (int j = w; j < (int)kReqSlots + 64; j += 64) wreq[j] = make_uint2(0u, 0u);
        for (int j = w; j < 64 * BMW + 64; j += 64) {
            wgnt[j] = make_uint2(0u, 0u);
            wvoid[j] = 0u;
        }
        cbar();
        // ARB 0: 32-bit sort keys (entry word | slot); ARB 1: 64-bit with the
        // round-robin rank (k * P + rotated port) above them
        using K = typename std::conditional<ARB == 0, uint32_t, unsigned long long>::type;
        constexpr K kMax = ~(K)0;
        uint2 e[BMW];  // first FIFO entries (meaningful for k < min(occ, b))
#pragma unroll
        for (int k = 0; k < BMW; k++) e[k] = make_uint2(0u, 0u);
        while (__ballot(live) != 0ull) {
            const uint32_t tag = processed + 1u;
            // ---------------------------------------------------------- R
            bool open = live;
            uint32_t nf = 0, ejm = 0;
            uint32_t tgk[BMW];
#pragma unroll
            for (int k = 0; k < BMW; k++) {
                const uint2 ek = e[k];
                const bool offk = open & (k < b) & ((uint32_t)k < occ) & (ek.y <= t);
                const uint32_t q = (ek.x >> 5) & 3u;
                const uint32_t lb = byte_of(lfb, q);
                const bool sk = (lb & 63u) == (uint32_t)i;
                const uint32_t tg = (uint32_t)gl0 + (lb & 63u);
                tgk[k] = tg;
                const bool rq = offk & !sk;
                const uint32_t slot = rq ? (byte_of(lfx, q) * BMW + k) * 64u + tg : req_trash;
                wreq[slot] = make_uint2((ek.x & ~0x7Fu) | ((lb >> 6) << 5), tag);
                ejm |= (offk & sk) ? 1u << k : 0u;
                nf += offk ? 1u : 0u;
                open = offk;
            }
            uint32_t nxt = (live & (occ != 0u) & (e[0].y > t)) ? e[0].y : kNever;
            if constexpr (CR) nxt = min(nxt, (live & (owed != 0u)) ? crt : kNever);
            // the scenario's earliest future event, taken with the requests so
            // that an idle cycle needs no extra LDS round trip to jump
            atomicMin(&red[nxt != kNever ? (uint32_t)g : 64u + (uint32_t)w], nxt);
            // stream offers: the released lines of the current range, then (rarely)
            // of the ranges after it
            // (the lane is their source and their target: they stay in registers)
            uint32_t nsr = (live & (R < rend)) ? released_count<CH>(d, cur, o, min((uint32_t)b, cur.len - o), dv0, dv1, deliv)
                                                : 0u;
            uint32_t sword[BMW];
#pragma unroll
            for (int k = 0; k < BMW; k++) sword[k] = ((cur.start + o + k) << kXs) | (cur.lf << 5);
            if ((nsr == cur.len - o) & (nsr < (uint32_t)b) & (R + 1 < rend) & live) {
                int sR = R + 1;
                WRange sr;
                while (sR < rend && nsr < (uint32_t)b) {
                    load_wrange(d, sR, sr);
                    const uint32_t n = released_direct<CH>(d, sr, min((uint32_t)b - nsr, sr.len), deliv);
#pragma unroll
                    for (int k = 0; k < BMW; k++)
                        if (((uint32_t)k >= nsr) & ((uint32_t)k < nsr + n))
                            sword[k] = ((sr.start + (uint32_t)k - nsr) << kXs) | (sr.lf << 5);
                    nsr += n;
                    if (n < sr.len) break;
                    sR++;
                }
            }
            cbar();
            // ---------------------------------------------------------- G
            uint32_t rv;
            K lst[BMW];
            {
                uint2 qv[(NF - 1) * BMW];
#pragma unroll
                for (int c = 0; c < (NF - 1) * BMW; c++) qv[c] = wreq[c * 64 + w];
                rv = red[g];
                K lists[NF][BMW];
#pragma unroll
                for (int f = 0; f < NF; f++) {
                    const bool fs = f == NF - 1;  // the lane's own stream
                    const uint32_t port = fs ? P - 1u : (fp >> (8 * f)) & 0xFFu;
                    const uint32_t rot = port >= rr ? port - rr : port + P - rr;
#pragma unroll
                    for (int k = 0; k < BMW; k++) {
                        const uint32_t wx = fs ? sword[k] : qv[f * BMW + k].x;
                        const bool valid = fs ? (uint32_t)k < nsr : qv[f * BMW + k].y == tag;
                        const uint32_t lo = wx | (uint32_t)(f * BMW + k);
                        K key;
                        if constexpr (ARB == 0) key = lo;
                        else key = ((unsigned long long)((uint32_t)k * P + rot) << 32) | lo;
                        lists[f][k] = valid ? key : kMax;
                    }
                }
#pragma unroll
                for (int k = 0; k < BMW; k++) lst[k] = lists[NF - 1][k];  // stream offers: already in order
#pragma unroll
                for (int f = 0; f < NF - 1; f++) {
                    sort_net(lists[f]);
                    merge_low(lst, lists[f]);
                }
            }
            uint32_t nval = 0;
#pragma unroll
            for (int r = 0; r < BMW; r++) nval += lst[r] != kMax ? 1u : 0u;
            const uint32_t gcnt = live ? min(min((uint32_t)b, cap - occ - (CR ? owed : 0u)), nval) : 0u;
            uint32_t sgr = 0, lastport = 0;
            const uint32_t ready = t + L;
#pragma unroll
            for (int r = 0; r < BMW; r++) {
                const bool gr = (uint32_t)r < gcnt;
                const uint32_t lo = (uint32_t)lst[r];
                const uint32_t c = lo & 31u;
                const uint32_t f = c / BMW, k = c % BMW;
                const bool fs = f == NF - 1;
                const uint32_t src = byte_of(fl, f);
                wgnt[(gr & !fs) ? k * 64u + src : gnt_trash] = make_uint2(tag, (uint32_t)r);
                sgr += (gr & fs) ? 1u : 0u;
                ring[gr ? rbase + wrap_add(tail, (uint32_t)r, cap) : ring_trash] = make_uint2(lo & ~0x1Fu, ready);
                if (ARB == 1) lastport = gr ? (fs ? P - 1u : byte_of(fp, f)) : lastport;
            }
            cbar();
            // ---------------------------------------------------------- D
            uint2 gv[BMW];
#pragma unroll
            for (int k = 0; k < BMW; k++) gv[k] = wgnt[k * 64 + w];
            uint32_t depf = 0, ejd = 0, vdm = 0;
            {
                bool op = true;
#pragma unroll
                for (int k = 0; k < BMW; k++) {
                    const bool offk = (uint32_t)k < nf;
                    const bool ejk = ((ejm >> k) & 1u) != 0u;
                    const bool gk = ejk | (gv[k].x == tag);
                    const bool dep = op & offk & gk;
                    vdm |= (offk & !ejk & gk & !dep) ? 1u << k : 0u;
                    ejd |= (dep & ejk) ? 1u << k : 0u;
                    depf += dep ? 1u : 0u;
                    op = dep;
                }
            }
            if (ejd) {
#pragma unroll
                for (int k = 0; k < BMW; k++) {
                    if ((ejd >> k) & 1u) {
                        const uint32_t x = e[k].x >> kXs;
                        bad |= x >= Tu;
                        comp[x < Tu ? x : 0u] = t + 1u;
                        atomicAdd(&deliv[mydx + ((e[k].x >> 5) & 3u)], 1u);
                    }
                }
            }
            if constexpr (CR) {  // left slots stay owed until their credits are back
#pragma unroll
                for (int k = 0; k < BMW; k++)
                    ring[(uint32_t)k < depf ? rbase + wrap_add(head, (uint32_t)k, cap) : ring_trash] =
                        make_uint2(e[k].x, t);
                crt = ((depf != 0u) & (owed == 0u)) ? t + D : crt;
                owed += depf;
            }
            head = wrap_add(head, depf, cap);
            occ -= depf;
            o += sgr;
            if (o >= cur.len) next_range();
            uint32_t cnt = gcnt;
            if (__ballot(vdm != 0u) != 0ull) {
                // rare: void grants; their targets keep only the lines that departed
                cbar();
#pragma unroll
                for (int k = 0; k < BMW; k++)
                    wvoid[((vdm >> k) & 1u) ? gv[k].y * 64u + tgk[k] : gnt_trash] = tag;
                cbar();
                uint32_t vt[BMW];  // read every void flag before the first ring write
#pragma unroll
                for (int r = 0; r < BMW; r++) vt[r] = wvoid[r * 64 + w];
                cbar();
                uint32_t j = 0;
#pragma unroll
                for (int r = 0; r < BMW; r++) {
                    const uint32_t lo = (uint32_t)lst[r];
                    const bool keep = ((uint32_t)r < gcnt) & (vt[r] != tag);
                    ring[keep ? rbase + wrap_add(tail, j, cap) : ring_trash] = make_uint2(lo & ~0x1Fu, ready);
                    if (ARB == 1) {
                        const uint32_t f = (lo & 31u) / BMW;
                        lastport = keep ? (f == NF - 1 ? P - 1u : byte_of(fp, f)) : lastport;
                    }
                    j += keep ? 1u : 0u;
                }
                cnt = j;
            }
            tail = wrap_add(tail, cnt, cap);
            occ += cnt;
            tx += cnt;
            busy += cnt ? 1u : 0u;
            if (ARB == 1) rr = cnt ? (lastport + 1u == P ? 0u : lastport + 1u) : rr;
            cbar();
            red[i == 0 ? (uint32_t)g : 64u + (uint32_t)w] = kNever;
#pragma unroll
            for (int k = 0; k < BMW; k++) e[k] = ring[rbase + wrap_add(head, min((uint32_t)k, cap - 1u), cap)];
            refresh_dv();
            time_phase((depf | sgr) != 0u, rv);
            if constexpr (CR) credits_back();
        }
    };
    if constexpr (kGeneral) {
        if (!fast && !lined) {
            if constexpr (BM == 1) {
                general(std::integral_constant<int, 1>{});
            } else {
                if (ARB == 1 && wbm <= 1) general(std::integral_constant<int, 1>{});
                else if (wbm <= 2) general(std::integral_constant<int, 2>{});
                else if constexpr (BM >= 4) {
                    if (wbm <= 4 || BM == 4) general(std::integral_constant<int, 4>{});
                    else if constexpr (BM >= 8) general(std::integral_constant<int, 8>{});
                }
            }
        }
    }

    if (on) {
        d.tx_lines[(size_t)s * m + link] = tx;
        d.busy[(size_t)s * m + link] = busy;
        if (i == 0) {
            d.makespan[s] = d.T > 0 ? t + 1u : 0u;
            d.status[s] = state;
            d.cycles[s] = processed;
        }
    }
}

template <int BM, int ARB, int NF>
hipError_t launch_wave3(const DevNet &d, hipStream_t st) {
    // per-chunk dependencies and credit delays get their own instantiations,
    // so that the base loops carry neither; the host does not pick this
    // engine for the two together
    if (d.credit && d.pd_omask == 0u) return hipErrorInvalidValue;
    auto k = d.credit ? engine_wave<BM, ARB, NF, false, true>
                      : d.pd_omask == 0u ? engine_wave<BM, ARB, NF, true, false> : engine_wave<BM, ARB, NF, false, false>;
    if (d.lds_bytes > 65536)
        (void)hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize, d.lds_bytes);
    hipLaunchKernelGGL(k, dim3((unsigned)d.wv_nblk), dim3(64 * d.wv_wpb), (unsigned)d.lds_bytes, st, d);
    return hipGetLastError();
}

// request-slot groups: 2 (one feeder and the stream) or kWaveMaxNF
template <int BM, int ARB>
hipError_t launch_wave2(const DevNet &d, hipStream_t st) {
    if constexpr (BM == 1 && ARB == 0) {
        return launch_wave3<1, 0, 2>(d, st);  // b = 1 loop only
    } else {
        if (d.wv_nfs <= 2) return launch_wave3<BM, ARB, 2>(d, st);
        if constexpr (BM * kWaveMaxNF <= 32) return launch_wave3<BM, ARB, kWaveMaxNF>(d, st);
        return hipErrorInvalidValue;
    }
}

template <int BM>
hipError_t launch_wave(const DevNet &d, hipStream_t st) {
    return d.arb == 0 ? launch_wave2<BM, 0>(d, st) : launch_wave2<BM, 1>(d, st);
}

}  // namespace

hipError_t launch_wave_any(const DevNet &d, hipStream_t st) {
    switch (d.bm) {
    case 1: return launch_wave<1>(d, st);
    case 2: return launch_wave<2>(d, st);
    case 4: return launch_wave<4>(d, st);
    default: return launch_wave<8>(d, st);
    }
}

}  // namespace simgpu
