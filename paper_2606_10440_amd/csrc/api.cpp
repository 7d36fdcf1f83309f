// Host side of libsimgpu: topology validation, routing tables, workload
// expansion into injection streams, device uploads and the C ABI.
//
// Paper: the infrastructure is a directed attributed graph (Sec. 4.6); the
// Simple backend routes over it with a modular routing function (Sec. 4.5);
// the unit of transfer is the 128 B wavefront request (Sec. 4.4.3); the
// collectives are the textbook ring / direct algorithms (Sec. 1).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstdlib>
#include <cstdio>
#include <cstring>
#include <functional>
#include <map>
#include <new>
#include <string>
#include <unordered_map>
#include <vector>

#include "../../include/simgpu.h"
#include "sim_internal.h"

using simgpu::DevNet;

namespace {

// Per-run device scratch of the engines (statuses, processed-cycle counts,
// and the FIFO rings, per-link scalars and request records of the engines
// that keep them in device memory) as one block: each array at an offset,
// bound to a base address per run.
struct StateLayout {
    size_t bytes = 0;
    std::vector<std::function<void(DevNet &, unsigned char *)>> bind;
    template <class T>
    void add(T *DevNet::*field, size_t count) {
        const size_t off = bytes;
        bytes += (std::max<size_t>(count * sizeof(T), 16) + 255) & ~(size_t)255;
        bind.push_back([field, off](DevNet &d, unsigned char *base) { d.*field = reinterpret_cast<T *>(base + off); });
    }
    void apply(DevNet &d, unsigned char *base) const {
        for (const auto &f : bind) f(d, base);
    }
};

// MurmurHash3's 32-bit finalizer (Appleby): spreads (src, dst) over the
// candidate next hops.
inline uint32_t finalize32(uint32_t v) {
    v ^= v >> 16;
    v *= 0x85ebca6bu;
    v ^= v >> 13;
    v *= 0xc2b2ae35u;
    v ^= v >> 16;
    return v;
}

}  // namespace

struct sim_ctx {
    int32_t n = 0, E = 0, m = 0, S = 0, arb = 0;
    int device = 0;
    std::vector<int32_t> row_ptr, col_idx, tail;
    std::vector<int32_t> bw, lat, cap;
    std::vector<int32_t> credit;  // [S*m] credit return delays; empty = all 1
    // minimal-hop routing: the reversed links, and the hop counts from every
    // node to one destination endpoint at a time (computed when needed)
    std::vector<int32_t> in_ptr, in_src;
    mutable std::vector<int32_t> hop_to;
    mutable std::vector<int32_t> hop_frontier;
    mutable int32_t hop_dst = -1;

    // loaded workload
    bool loaded = false;
    bool expanded = false;  // the host expansion of the last load succeeded (sim_txn_info)
    int64_t T = 0;
    uint64_t line_hops = 0;
    std::unordered_map<uint64_t, int32_t> flow_slot;  // (src << 32 | dst) -> slot
    std::vector<int32_t> flow_path;                   // [nflows] start in path_link
    std::vector<int32_t> path_link;
    // the workload's id ranges in id order, for sim_txn_info
    std::vector<uint32_t> h_start, h_moff;
    std::vector<int32_t> h_src, h_dst, h_step;

    DevNet dn{};
    std::vector<void *> dev_static;  // freed on reload / destroy
    std::vector<void *> dev_state;
    StateLayout state;               // the engines' scratch, bound to dev_state's block in dn
    // where the last run's statuses and cycle counts are (its scratch block)
    int32_t *run_status = nullptr;
    uint64_t *run_cycles = nullptr;
    std::string err = "";
    bool ran = false;
};

namespace {

sim_status fail(sim_ctx *c, sim_status s, const std::string &msg) {
    if (c) c->err = msg;
    return s;
}

void free_list(std::vector<void *> &v) {
    for (void *p : v) (void)hipFree(p);
    v.clear();
}

template <class T>
sim_status upload(sim_ctx *c, std::vector<void *> &owner, const std::vector<T> &h, T **out) {
    size_t bytes = std::max<size_t>(h.size() * sizeof(T), 16);
    void *p = nullptr;
    if (hipMalloc(&p, bytes) != hipSuccess) return fail(c, SIM_ERR_OOM, "hipMalloc failed");
    owner.push_back(p);
    if (!h.empty() && hipMemcpy(p, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice) != hipSuccess)
        return fail(c, SIM_ERR_DEVICE, "hipMemcpy failed");
    *out = static_cast<T *>(p);
    return SIM_OK;
}

template <class T>
sim_status alloc(sim_ctx *c, std::vector<void *> &owner, size_t count, T **out) {
    void *p = nullptr;
    if (hipMalloc(&p, std::max<size_t>(count * sizeof(T), 16)) != hipSuccess)
        return fail(c, SIM_ERR_OOM, "hipMalloc failed (" + std::to_string(count * sizeof(T)) + " B)");
    owner.push_back(p);
    *out = static_cast<T *>(p);
    return SIM_OK;
}

// The reversed links (for each node, the tails of its in-links).
void build_in_links(sim_ctx *c) {
    const int32_t n = c->n, m = c->m;
    c->in_ptr.assign(n + 1, 0);
    c->in_src.assign(m, 0);
    for (int32_t l = 0; l < m; l++) c->in_ptr[c->col_idx[l] + 1]++;
    for (int32_t v = 0; v < n; v++) c->in_ptr[v + 1] += c->in_ptr[v];
    std::vector<int32_t> fill(c->in_ptr.begin(), c->in_ptr.end() - 1);
    for (int32_t l = 0; l < m; l++) c->in_src[fill[c->col_idx[l]]++] = c->tail[l];
    c->hop_dst = -1;
}

// Hop distances from every node to endpoint d (-1: unreachable): a
// breadth-first search from d over the reversed links, kept until the next
// destination is asked for.
const int32_t *hops_to(const sim_ctx *c, int32_t d) {
    if (c->hop_dst == d) return c->hop_to.data();
    c->hop_to.assign(c->n, -1);
    int32_t *h = c->hop_to.data();
    auto &frontier = c->hop_frontier;
    frontier.clear();
    frontier.push_back(d);
    h[d] = 0;
    for (size_t q = 0; q < frontier.size(); q++) {
        const int32_t w = frontier[q];
        for (int32_t e = c->in_ptr[w]; e < c->in_ptr[w + 1]; e++) {
            const int32_t u = c->in_src[e];
            if (h[u] < 0) {
                h[u] = h[w] + 1;
                frontier.push_back(u);
            }
        }
    }
    c->hop_dst = d;
    return h;
}

// Minimal-hop route of flow s -> d.  Among out-links whose head is one hop
// nearer to d (ascending link id), the i-th tie-break uses byte (i mod 4) of
// the finalized (s << 16 | d), re-finalized before every fourth tie-break
// after the first.
bool trace_route(const sim_ctx *c, int32_t s, int32_t d, std::vector<int32_t> &out) {
    out.clear();
    const int32_t *h = hops_to(c, d);
    if (h[s] < 0) return false;
    uint32_t key = finalize32(((uint32_t)s << 16) | (uint32_t)d);
    int32_t ties = 0;
    int32_t v = s;
    while (v != d) {
        const int32_t want = h[v] - 1;
        int32_t count = 0;
        for (int32_t l = c->row_ptr[v]; l < c->row_ptr[v + 1]; l++)
            if (h[c->col_idx[l]] == want) count++;
        int32_t pick = 0;
        if (count > 1) {
            if (ties > 0 && (ties & 3) == 0) key = finalize32(key);
            pick = (int32_t)(((key >> (8 * (ties & 3))) & 0xFFu) % (uint32_t)count);
            ties++;
        }
        int32_t chosen = -1;
        for (int32_t l = c->row_ptr[v]; l < c->row_ptr[v + 1]; l++)
            if (h[c->col_idx[l]] == want && pick-- == 0) {
                chosen = l;
                break;
            }
        out.push_back(chosen);
        v = c->col_idx[chosen];
    }
    return true;
}

// The workload as id ranges: consecutive line ids of one flow whose
// predecessors are, line for line, consecutive lines of earlier ranges.
struct Ranges {
    std::vector<uint32_t> start, len;
    std::vector<int32_t> src, dst;
    std::vector<int32_t> step;   // algorithm step of the range's lines (-1: none)
    std::vector<uint32_t> moff;  // offset of the range's first line in its message
    std::vector<int64_t> pref_beg;   // [nr+1] into pref_rng/pref_delta
    std::vector<int64_t> pref_rng;   // predecessor range
    std::vector<uint32_t> pref_delta;  // line start+o waits for line pref_start+delta+o
    bool whole = false;  // per-chunk: every line waits for the whole predecessor range
    std::vector<uint8_t> cls;  // [T] message class per line (empty: all data)
    void add(uint64_t s, uint64_t l, int32_t a, int32_t b, int64_t st = -1, int64_t mo = 0) {
        start.push_back((uint32_t)s);
        len.push_back((uint32_t)l);
        src.push_back(a);
        dst.push_back(b);
        step.push_back((int32_t)st);
        moff.push_back((uint32_t)mo);
        pref_beg.push_back((int64_t)pref_rng.size());
    }
    void pred(int64_t r, uint64_t delta) {
        pref_rng.push_back(r);
        pref_delta.push_back((uint32_t)delta);
    }
    void close() { pref_beg.push_back((int64_t)pref_rng.size()); }
};

inline int64_t wrap(int64_t a, int64_t m) { return ((a % m) + m) % m; }

// Recursive halving-doubling all-reduce over p = 2^K participants.  Range
// layout: halving step j, participant i -> range j p + i (one message);
// doubling step j, participant i -> one range per chunk of its block, so that
// each range's data arrived in one piece (every range has single-range
// predecessors).  In per-message mode every range of a message waits for the
// last range of each message that feeds the message.
sim_status expand_rhd(sim_ctx *c, int64_t N, const std::vector<int32_t> &rho, Ranges &R) {
    const int64_t p = (int64_t)rho.size();
    if (p & (p - 1)) return fail(c, SIM_ERR_INVALID_ARG, "recursive halving-doubling needs a power-of-two endpoint count");
    if (N % p) return fail(c, SIM_ERR_SIZE, "recursive halving-doubling: lines not divisible by participants");
    int K = 0;
    while ((int64_t(1) << K) < p) K++;
    const int64_t C = N / p;
    auto half = [&](int j) { return N >> (j + 1); };
    // first position of the half participant i sends at halving step j
    auto send_start = [&](int64_t i, int j) {
        const int64_t S = half(j);
        return (i >> (K - j)) * 2 * S + (((i >> (K - 1 - j)) & 1) ? 0 : S);
    };
    auto rs_range = [&](int j, int64_t i) { return (int64_t)j * p + i; };
    // range of doubling step j, participant i, chunk ch (within i's block)
    auto ag_range = [&](int j, int64_t i, int64_t ch) {
        return (int64_t)K * p + p * ((int64_t(1) << j) - 1) + (i << j) + (ch - ((i >> j) << j));
    };
    auto ag_last = [&](int j, int64_t i) { return ag_range(j, i, ((i >> j) << j) + (int64_t(1) << j) - 1); };
    for (int j = 0; j < K; j++) {
        const int64_t S = half(j);
        for (int64_t i = 0; i < p; i++) {
            R.add(p * (N - 2 * S) + i * S, S, rho[i], rho[i ^ (p >> (j + 1))], j);
            for (int j2 = 0; j2 < j; j2++) {
                const int64_t from = i ^ (p >> (j2 + 1));
                R.pred(rs_range(j2, from), R.whole ? 0 : send_start(i, j) - send_start(from, j2));
            }
        }
    }
    const int64_t TRS = N * (p - 1);
    for (int j = 0; j < K; j++) {
        for (int64_t i = 0; i < p; i++) {
            const int64_t b0 = (i >> j) << j;
            for (int64_t ch = b0; ch < b0 + (int64_t(1) << j); ch++) {
                R.add(TRS + N * ((int64_t(1) << j) - 1) + (i << j) * C + (ch - b0) * C, C, rho[i], rho[i ^ (int64_t(1) << j)],
                      K + j, (ch - b0) * C);
                if (R.whole) {
                    for (int j2 = 0; j2 < K; j2++) R.pred(rs_range(j2, i ^ (p >> (j2 + 1))), 0);
                    for (int h = 0; h < j; h++) R.pred(ag_last(h, i ^ (int64_t(1) << h)), 0);
                } else if (ch == i) {
                    // the reduced chunk: every halving-step arrival of it
                    for (int j2 = 0; j2 < K; j2++) {
                        const int64_t from = i ^ (p >> (j2 + 1));
                        R.pred(rs_range(j2, from), ch * C - send_start(from, j2));
                    }
                } else {
                    // arrived at the doubling step of the highest bit where ch and i differ
                    int h = 0;
                    while ((ch ^ i) >> (h + 1)) h++;
                    R.pred(ag_range(h, i ^ (int64_t(1) << h), ch), 0);
                }
            }
        }
    }
    return SIM_OK;
}

// Double binary tree all-reduce: one range per message, range index =
// (phase 2 + tree)(p - 1) + edge.
void expand_dbt(int64_t p, int64_t H, const std::vector<int32_t> &rho, Ranges &R) {
    auto parent = [&](int64_t u) -> int64_t {
        const int64_t b = u & -u;
        const int64_t up = (u - b) | (2 * b);
        return up < p ? up : u - b;
    };
    std::vector<std::vector<int64_t>> kids(p);
    for (int64_t u = 1; u < p; u++) kids[parent(u)].push_back(u);
    auto part = [&](int64_t pos, int t) { return t == 0 ? pos : p - 1 - pos; };  // position <-> participant
    auto edge = [&](int64_t part_c, int t) { return t == 0 ? part_c - 1 : part_c; };
    auto msg = [&](int ph, int t, int64_t e) { return ((int64_t)ph * 2 + t) * (p - 1) + e; };
    for (int ph = 0; ph < 2; ph++)
        for (int t = 0; t < 2; t++)
            for (int64_t e = 0; e < p - 1; e++) {
                const int64_t cpart = t == 0 ? e + 1 : e;
                const int64_t cpos = part(cpart, t);
                const int64_t vpos = parent(cpos), vpart = part(vpos, t);
                R.add(msg(ph, t, e) * H, H, rho[ph == 0 ? cpart : vpart], rho[ph == 0 ? vpart : cpart], ph * 2 + t);
                if (ph == 0 || vpos == 0) {
                    // reduce: the children of c; broadcast from the root: the root's children
                    for (int64_t u : kids[ph == 0 ? cpos : 0]) R.pred(msg(0, t, edge(part(u, t), t)), 0);
                } else {
                    R.pred(msg(1, t, edge(vpart, t)), 0);
                }
            }
}

sim_status expand_collective(sim_ctx *c, int32_t coll, uint64_t bytes, int32_t group,
                             const int32_t *order, int32_t dep, Ranges &R) {
    const int64_t E = c->E;
    if (dep != SIM_DEP_LINE && dep != SIM_DEP_CHUNK) return fail(c, SIM_ERR_INVALID_ARG, "unknown dep");
    if (dep == SIM_DEP_CHUNK && coll == SIM_COLL_HIER_ALLREDUCE)
        return fail(c, SIM_ERR_INVALID_ARG, "per-chunk dependencies are not defined for the hierarchical all-reduce");
    R.whole = dep == SIM_DEP_CHUNK;
    if (bytes == 0 || bytes % SIM_LINE_BYTES) return fail(c, SIM_ERR_SIZE, "bytes must be a positive multiple of 128");
    const int64_t N = (int64_t)(bytes / SIM_LINE_BYTES);
    if (E < 2) return fail(c, SIM_ERR_INVALID_ARG, "a collective needs at least 2 endpoints");
    std::vector<int32_t> rho(E);
    for (int64_t i = 0; i < E; i++) rho[i] = (int32_t)i;
    if (order) {
        if (coll == SIM_COLL_HIER_ALLREDUCE || coll == SIM_COLL_ALLTOALL)
            return fail(c, SIM_ERR_INVALID_ARG, "order does not apply to the hierarchical all-reduce or all-to-all");
        std::vector<char> seen(E, 0);
        for (int64_t i = 0; i < E; i++) {
            if (order[i] < 0 || order[i] >= E || seen[order[i]])
                return fail(c, SIM_ERR_INVALID_ARG, "order is not a permutation of the endpoints");
            seen[order[i]] = 1;
            rho[i] = order[i];
        }
    }
    if (coll == SIM_COLL_RING_ALLREDUCE) {
        const int64_t p = E;
        if (N % p) return fail(c, SIM_ERR_SIZE, "ring: lines not divisible by participants");
        const int64_t C = N / p;
        for (int64_t s = 0; s < 2 * p - 2; s++)
            for (int64_t i = 0; i < p; i++) {
                R.add((s * p + i) * C, C, rho[i], rho[(i + 1) % p], s);
                if (s > 0) R.pred((s - 1) * p + wrap(i - 1, p), 0);
            }
    } else if (coll == SIM_COLL_DIRECT_ALLREDUCE) {
        const int64_t p = E;
        if (N % p) return fail(c, SIM_ERR_SIZE, "direct: lines not divisible by participants");
        const int64_t C = N / p;
        for (int64_t ph = 0; ph < 2; ph++)
            for (int64_t k = 1; k < p; k++)
                for (int64_t i = 0; i < p; i++) {
                    int64_t idx = (ph * (p - 1) + (k - 1)) * p + i;
                    R.add(idx * C, C, rho[i], rho[(i + k) % p], ph * (p - 1) + k - 1);
                    if (ph == 1)
                        for (int64_t i2 = 0; i2 < p; i2++)
                            if (i2 != i) R.pred(((wrap(i - i2, p) - 1) * p + i2), 0);
                }
    } else if (coll == SIM_COLL_HIER_ALLREDUCE) {
        const int64_t M = group;
        if (M < 2 || E % M || E / M < 2)
            return fail(c, SIM_ERR_INVALID_ARG, "hierarchical: group_size must split endpoints into >= 2 domains of >= 2");
        const int64_t G = E / M;
        if (N % M) return fail(c, SIM_ERR_SIZE, "hierarchical: lines not divisible by group size");
        const int64_t C1 = N / M;
        if (C1 % G) return fail(c, SIM_ERR_SIZE, "hierarchical: chunk not divisible by domain count");
        const int64_t C2 = C1 / G;
        const int64_t R1 = (M - 1) * G * M, R2 = (2 * G - 2) * M * G;
        const int64_t B2 = R1 * C1, B3 = B2 + R2 * C2;
        // phase 1: direct reduce-scatter inside each domain
        for (int64_t k = 1; k < M; k++)
            for (int64_t d = 0; d < G; d++)
                for (int64_t r = 0; r < M; r++)
                    R.add((((k - 1) * G + d) * M + r) * C1, C1, (int32_t)(d * M + r),
                          (int32_t)(d * M + (r + k) % M), k - 1);
        // phase 2: ring over the domains on each rail r
        for (int64_t s = 0; s < 2 * G - 2; s++)
            for (int64_t r = 0; r < M; r++)
                for (int64_t d = 0; d < G; d++) {
                    R.add(B2 + ((s * M + r) * G + d) * C2, C2, (int32_t)(d * M + r),
                          (int32_t)(((d + 1) % G) * M + r), (M - 1) + s);
                    // Up to the first all-gather step the sent sub-chunk (d - s) mod G
                    // includes this node's own copy, reduced inside the domain first.
                    if (s <= G - 1)
                        for (int64_t r2 = 0; r2 < M; r2++)
                            if (r2 != r) R.pred(((wrap(r - r2, M) - 1) * G + d) * M + r2, wrap(d - s, G) * C2);
                    if (s >= 1) R.pred(R1 + ((s - 1) * M + r) * G + wrap(d - 1, G), 0);
                }
        // phase 3: direct all-gather inside each domain, split per sub-chunk
        for (int64_t k = 1; k < M; k++)
            for (int64_t d = 0; d < G; d++)
                for (int64_t r = 0; r < M; r++)
                    for (int64_t sub = 0; sub < G; sub++) {
                        R.add(B3 + (((k - 1) * G + d) * M + r) * C1 + sub * C2, C2, (int32_t)(d * M + r),
                              (int32_t)(d * M + (r + k) % M), (M - 1) + (2 * G - 2) + (k - 1), sub * C2);
                        const bool owned = sub == (d + 1) % G;  // fully reduced here by the ring
                        int64_t s = owned ? G - 2 : G - 1 + wrap(d - sub, G);
                        if (owned)
                            for (int64_t r2 = 0; r2 < M; r2++)
                                if (r2 != r) R.pred(((wrap(r - r2, M) - 1) * G + d) * M + r2, sub * C2);
                        R.pred(R1 + (s * M + r) * G + wrap(d - 1, G), 0);
                    }
    } else if (coll == SIM_COLL_ALLTOALL) {
        const int64_t C = N;
        for (int64_t k = 1; k < E; k++)
            for (int64_t i = 0; i < E; i++) R.add(((k - 1) * E + i) * C, C, (int32_t)i, (int32_t)((i + k) % E), k - 1);
    } else if (coll == SIM_COLL_RING_ALLGATHER || coll == SIM_COLL_RING_REDUCESCATTER) {
        const int64_t p = E;
        if (N % p) return fail(c, SIM_ERR_SIZE, "ring: lines not divisible by participants");
        const int64_t C = N / p;
        for (int64_t s = 0; s < p - 1; s++)
            for (int64_t i = 0; i < p; i++) {
                R.add((s * p + i) * C, C, rho[i], rho[(i + 1) % p], s);
                if (s > 0) R.pred((s - 1) * p + wrap(i - 1, p), 0);
            }
    } else if (coll == SIM_COLL_DIRECT_ALLGATHER || coll == SIM_COLL_DIRECT_REDUCESCATTER) {
        const int64_t p = E;
        if (N % p) return fail(c, SIM_ERR_SIZE, "direct: lines not divisible by participants");
        const int64_t C = N / p;
        for (int64_t k = 1; k < p; k++)
            for (int64_t i = 0; i < p; i++) R.add(((k - 1) * p + i) * C, C, rho[i], rho[(i + k) % p], k - 1);
    } else if (coll == SIM_COLL_RHD_ALLREDUCE) {
        const sim_status st = expand_rhd(c, N, rho, R);
        if (st != SIM_OK) return st;
    } else if (coll == SIM_COLL_DBT_ALLREDUCE) {
        if (N % 2) return fail(c, SIM_ERR_SIZE, "double binary tree: lines not divisible by 2");
        expand_dbt(E, N / 2, rho, R);
    } else {
        return fail(c, SIM_ERR_INVALID_ARG, "unknown collective");
    }
    R.close();
    return SIM_OK;
}

// Grid engine layout: node -> workgroup, the lanes of every workgroup as
// source sides (head node owned) and target sides (tail node owned), request
// slots, the flows whose delivered counts each workgroup keeps, and the LDS
// size (the kernel carves the same arrays in the same order).
struct GridLayout {
    int32_t nb = 0, threads = 64, ns_max = 0, nt_max = 0, req_max = 0, fl_max = 0;
    int64_t bytes = INT64_MAX;
    std::vector<int32_t> sptr, slane, tptr, tlane, tloc, rqoff, floc, fptr, fown;
    // one-line-per-cycle form
    bool one = false;
    int32_t one_threads = 64, inl_max = 0;
    int64_t one_bytes = INT64_MAX;
    std::vector<int32_t> toff, iptr, inl;
    // windowed form
    int32_t window = 0, sring_max = 0, cring_max = 0;
    std::vector<int32_t> sro, tro;
};

GridLayout grid_layout(const sim_ctx *c, const std::vector<int32_t> &fsrc, const std::vector<char> &has_stream,
                       const std::vector<std::vector<int32_t>> &feeders, const std::vector<int32_t> &fsrc_pos,
                       int32_t bmax, int32_t bm, int32_t nflows, const std::vector<int32_t> &pd_flow, int want_nb,
                       const std::vector<int32_t> &port_at_head, const std::vector<int32_t> &nports) {
    GridLayout g;
    const int32_t nl = (int32_t)fsrc.size();
    std::vector<int64_t> wgt(c->n, 0);
    for (int32_t i = 0; i < nl; i++) {
        const int32_t l = fsrc[i];
        wgt[c->tail[l]] += 1 + (has_stream[l] ? 1 : 0);
        wgt[c->col_idx[l]] += 1;
    }
    std::vector<int32_t> nodes;
    for (int32_t v = 0; v < c->n; v++)
        if (wgt[v] > 0) nodes.push_back(v);
    const int32_t nb = std::max<int32_t>(1, std::min<int32_t>(want_nb, (int32_t)nodes.size()));
    std::stable_sort(nodes.begin(), nodes.end(), [&](int32_t a, int32_t b) { return wgt[a] > wgt[b]; });
    std::vector<int32_t> part(c->n, 0);
    std::vector<int64_t> load(nb, 0);
    for (int32_t v : nodes) {
        const int32_t w = (int32_t)(std::min_element(load.begin(), load.end()) - load.begin());
        part[v] = w;
        load[w] += wgt[v];
    }
    g.nb = nb;
    std::vector<std::vector<int32_t>> src(nb), tgt(nb);
    for (int32_t i = 0; i < nl; i++) {  // lanes in fsrc order
        src[part[c->col_idx[fsrc[i]]]].push_back(i);
        tgt[part[c->tail[fsrc[i]]]].push_back(i);
    }
    g.tloc.assign(nl, 0);
    g.rqoff.assign(nl, 0);
    g.sptr.push_back(0);
    g.tptr.push_back(0);
    for (int32_t w = 0; w < nb; w++) {
        int64_t r = 0;
        for (size_t j = 0; j < tgt[w].size(); j++) {
            const int32_t i = tgt[w][j];
            g.tloc[i] = (int32_t)j;
            g.rqoff[i] = (int32_t)r;
            r += (int64_t)((int32_t)feeders[fsrc_pos[fsrc[i]]].size() + (has_stream[fsrc[i]] ? 1 : 0)) * bmax;
        }
        g.slane.insert(g.slane.end(), src[w].begin(), src[w].end());
        g.tlane.insert(g.tlane.end(), tgt[w].begin(), tgt[w].end());
        g.sptr.push_back((int32_t)g.slane.size());
        g.tptr.push_back((int32_t)g.tlane.size());
        g.ns_max = std::max(g.ns_max, (int32_t)src[w].size());
        g.nt_max = std::max(g.nt_max, (int32_t)tgt[w].size());
        g.req_max = (int32_t)std::max<int64_t>(g.req_max, r);
    }
    // delivered counters: kept for the flows some line waits on, by the
    // workgroup of the flow's destination endpoint
    g.floc.assign(nflows, -1);
    std::vector<char> waited(nflows, 0);
    for (int32_t f : pd_flow) waited[f] = 1;
    std::vector<std::vector<int32_t>> own(nb);
    for (int32_t f = 0; f < nflows; f++) {
        if (!waited[f]) continue;
        int32_t q = c->flow_path[f];
        while (c->path_link[q] >= 0) q++;
        const int32_t w = part[c->col_idx[c->path_link[q - 1]]];
        g.floc[f] = (int32_t)own[w].size();
        own[w].push_back(f);
    }
    g.fptr.push_back(0);
    for (int32_t w = 0; w < nb; w++) {
        g.fown.insert(g.fown.end(), own[w].begin(), own[w].end());
        g.fptr.push_back((int32_t)g.fown.size());
        g.fl_max = std::max(g.fl_max, (int32_t)own[w].size());
    }
    if (g.fown.empty()) g.fown.push_back(0);
    // wave 0 runs the barrier; one thread per lane after it
    const int32_t most = std::max(g.ns_max, g.nt_max);
    g.threads = std::min<int32_t>(1024, 64 + std::max<int32_t>(64, ((most + 63) / 64) * 64));
    auto a16 = [](int64_t v) { return (v + 15) & ~(int64_t)15; };
    const int64_t NS = g.ns_max, NT = g.nt_max, BM = bm, KC = 4;
    const bool preds = !pd_flow.empty();
    int64_t b = 0;
    for (int q = 0; q < 11; q++) b += a16(4 * NS);     // constants, head, counts, cache fill, offers
    for (int q = 0; q < 4; q++) b += a16(4 * NS * KC); // cached entries
    for (int q = 0; q < 3; q++) b += a16(4 * NS * BM); // offered lines, targets, grants
    for (int q = 0; q < 24; q++) b += a16(4 * NT);     // constants, counts, stream cursor and range
    for (int q = 0; q < 3; q++) b += a16(preds ? 4 * NT * 2 : 0);  // stream predecessor descriptors, counts
    for (int q = 0; q < 2; q++) b += a16(8 * NT);      // counters
    for (int q = 0; q < 3; q++) b += a16(4 * NT * BM); // grant list, departs, stream grants
    b += a16(16 * (int64_t)g.req_max);
    b += a16(preds ? 4 * ((int64_t)g.fl_max + 1) : 0);  // delivered counters (+ one for the rest)
    for (int q = 0; q < 3; q++) b += a16(preds ? 4 * (int64_t)g.fl_max : 0);  // flow ids, marks, list
    b += a16(4 * 32);
    g.bytes = b;
    // one-line-per-cycle form: one source and one target side per thread
    // after the barrier wave, and every input-port set in one 64-bit mask
    if (bmax == 1 && most <= 960) {
        g.one = true;
        g.one_threads = 64 + std::max<int32_t>(64, ((most + 63) / 64) * 64);
        std::vector<int32_t> sloc(nl, -1);
        for (int32_t w = 0; w < nb; w++)
            for (int32_t q = g.sptr[w]; q < g.sptr[w + 1]; q++) sloc[g.slane[q]] = q - g.sptr[w];
        std::vector<int32_t> lane_of(c->m, -1);
        for (int32_t i = 0; i < nl; i++) lane_of[fsrc[i]] = i;
        std::vector<std::vector<int32_t>> in_links(c->n);
        for (int32_t l = 0; l < c->m; l++) in_links[c->col_idx[l]].push_back(l);
        g.toff.assign(nl, 0);
        g.iptr.push_back(0);
        std::vector<int32_t> node_off(c->n, -1);
        for (int32_t w = 0; w < nb; w++) {
            const size_t base = g.inl.size();
            for (int32_t q = g.tptr[w]; q < g.tptr[w + 1]; q++) {
                const int32_t i = g.tlane[q];
                const int32_t u = c->tail[fsrc[i]];
                if (node_off[u] < 0) {
                    node_off[u] = (int32_t)(g.inl.size() - base);
                    if (nports[u] > 64) g.one = false;
                    std::vector<int32_t> tab(nports[u], -1);
                    for (int32_t l : in_links[u])
                        if (lane_of[l] >= 0) tab[port_at_head[l]] = sloc[lane_of[l]];
                    g.inl.insert(g.inl.end(), tab.begin(), tab.end());
                }
                g.toff[i] = node_off[u];
            }
            g.iptr.push_back((int32_t)g.inl.size());
            g.inl_max = std::max(g.inl_max, (int32_t)(g.inl.size() - base));
        }
        if (g.inl.empty()) g.inl.push_back(-1);
        int64_t b1 = a16(8 * NT * (c->arb == SIM_ARB_LOWEST_ID ? 2 : 1));
        if (c->arb == SIM_ARB_ROUND_ROBIN) b1 += a16(8 * NS) + a16(4 * (int64_t)g.inl_max);
        b1 += a16(preds ? 4 * ((int64_t)g.fl_max + 1) : 0);
        for (int q = 0; q < 3; q++) b1 += a16(preds ? 4 * (int64_t)g.fl_max : 0);
        b1 += a16(4 * 32);
        g.one_bytes = b1;
    }
    return g;
}

// Turn ranges into device tables: flow slots, paths, streams, predecessor
// descriptors, FIFO/request layouts; allocate per-scenario state.
sim_status finish_load(sim_ctx *c, Ranges &R) {
    free_list(c->dev_static);
    free_list(c->dev_state);
    c->loaded = false;
    c->expanded = false;
    const int64_t nr = (int64_t)R.start.size();
    int64_t T = 0;
    for (int64_t i = 0; i < nr; i++) {
        if ((int64_t)R.start[i] != T) return fail(c, SIM_ERR_INVALID_ARG, "internal: ranges not contiguous");
        T += R.len[i];
    }
    if (T >= (int64_t)0xFFFFFFFFll) return fail(c, SIM_ERR_SIZE, "more than 2^32-2 transactions");
    c->T = T;
    c->h_start = R.start;
    c->h_src = R.src;
    c->h_dst = R.dst;
    c->h_step = R.step;
    c->h_moff = R.moff;

    // flow slots and paths
    c->flow_slot.clear();
    c->flow_path.clear();
    c->path_link.clear();
    std::vector<int32_t> rflow(nr);
    std::vector<int32_t> flow_hops;
    // flow slots in order of first appearance; their routes are traced
    // destination by destination (one hop table alive at a time)
    std::vector<std::pair<int32_t, int32_t>> fpair;
    for (int64_t i = 0; i < nr; i++) {
        uint64_t key = ((uint64_t)(uint32_t)R.src[i] << 32) | (uint32_t)R.dst[i];
        auto it = c->flow_slot.find(key);
        if (it == c->flow_slot.end()) {
            it = c->flow_slot.emplace(key, (int32_t)fpair.size()).first;
            fpair.emplace_back(R.src[i], R.dst[i]);
        }
        rflow[i] = it->second;
    }
    const int32_t nflows = (int32_t)fpair.size();
    {
        std::vector<int32_t> by_dst(nflows);
        for (int32_t f = 0; f < nflows; f++) by_dst[f] = f;
        std::stable_sort(by_dst.begin(), by_dst.end(),
                         [&](int32_t a, int32_t b) { return fpair[a].second < fpair[b].second; });
        std::vector<std::vector<int32_t>> routes(nflows);
        for (int32_t f : by_dst) {
            if (!trace_route(c, fpair[f].first, fpair[f].second, routes[f]))
                return fail(c, SIM_ERR_UNREACHABLE, "no path from endpoint " + std::to_string(fpair[f].first) +
                                                        " to endpoint " + std::to_string(fpair[f].second));
        }
        size_t total = 0;
        for (const auto &r : routes) total += r.size() + 1;
        if (total >= (size_t)INT32_MAX) return fail(c, SIM_ERR_SIZE, "path table too large");
        c->path_link.reserve(total);
        for (int32_t f = 0; f < nflows; f++) {
            c->flow_path.push_back((int32_t)c->path_link.size());
            c->path_link.insert(c->path_link.end(), routes[f].begin(), routes[f].end());
            c->path_link.push_back(-(1 + f));
            flow_hops.push_back((int32_t)routes[f].size());
        }
    }
    if (c->path_link.size() >= (size_t)INT32_MAX) return fail(c, SIM_ERR_SIZE, "path table too large");

    // per-flow sequence numbers (flows deliver in id order) and predecessor descriptors
    std::vector<uint32_t> seq0(nr);
    {
        std::vector<uint64_t> cnt(nflows, 0);
        for (int64_t i = 0; i < nr; i++) {
            seq0[i] = (uint32_t)cnt[rflow[i]];
            cnt[rflow[i]] += R.len[i];
        }
    }
    c->line_hops = 0;
    for (int64_t i = 0; i < nr; i++) c->line_hops += (uint64_t)R.len[i] * (uint64_t)flow_hops[rflow[i]];

    // streams: ranges grouped by first link, ascending id inside a stream
    const int32_t m = c->m;
    std::vector<int64_t> first_cnt(m + 1, 0);
    for (int64_t i = 0; i < nr; i++) first_cnt[c->path_link[c->flow_path[rflow[i]]] + 1]++;
    std::vector<int32_t> s_link, s_rbeg, s_rend;
    std::vector<int64_t> pos(m, -1);
    int64_t acc = 0;
    for (int32_t l = 0; l < m; l++) {
        if (first_cnt[l + 1] == 0) continue;
        s_link.push_back(l);
        s_rbeg.push_back((int32_t)acc);
        pos[l] = acc;
        acc += first_cnt[l + 1];
        s_rend.push_back((int32_t)acc);
    }
    if (acc >= INT32_MAX) return fail(c, SIM_ERR_SIZE, "too many ranges");
    std::vector<uint32_t> r_start(nr), r_len(nr);
    std::vector<int32_t> r_path(nr), r_pd(nr + 1);
    std::vector<int32_t> pd_flow;
    std::vector<uint32_t> pd_base;
    std::vector<int64_t> order(nr);
    for (int64_t i = 0; i < nr; i++) {
        int32_t f = c->path_link[c->flow_path[rflow[i]]];
        order[pos[f]++] = i;
    }
    for (int64_t j = 0; j < nr; j++) {
        int64_t i = order[j];
        r_start[j] = R.start[i];
        r_len[j] = R.len[i];
        r_path[j] = c->flow_path[rflow[i]];
        r_pd[j] = (int32_t)pd_flow.size();
        for (int64_t q = R.pref_beg[i]; q < R.pref_beg[i + 1]; q++) {
            int64_t pr = R.pref_rng[q];
            if (!R.whole && (uint64_t)R.pref_delta[q] + R.len[i] > R.len[pr])
                return fail(c, SIM_ERR_INVALID_ARG, "internal: predecessor range too short");
            pd_flow.push_back(rflow[pr]);
            pd_base.push_back(R.whole ? seq0[pr] + R.len[pr] - 1 : seq0[pr] + R.pref_delta[q]);
        }
    }
    r_pd[nr] = (int32_t)pd_flow.size();

    // links carrying traffic; ports; FIFO and request layouts
    std::vector<char> used(m, 0);
    for (int32_t v : c->path_link)
        if (v >= 0) used[v] = 1;
    std::vector<int32_t> fsrc;
    for (int32_t l = 0; l < m; l++)
        if (used[l]) fsrc.push_back(l);
    // Lined-up graphs: every traffic link is fed by at most one other link
    // and sends lines on to at most one other link, and these links form
    // paths (no cycle).  The traffic links are then ordered path by path, so
    // that in lane order a link's feeder is the link just before it and its
    // next link the one just after it (the wave engine's shift loop).
    // (The wave engine's shift loop also needs, under lowest-id arbitration
    // with several lines per cycle, one flow at most per pair of consecutive
    // links, and no credit delays; otherwise the links keep their order.)
    int32_t bmax_all = 1;
    for (int32_t v : c->bw) bmax_all = std::max(bmax_all, v);
    bool lineup = c->credit.empty();
    {
        std::vector<int32_t> pre(m, -1), nxt(m, -1), npair(m, 0);
        for (size_t q = 0; q + 1 < c->path_link.size() && lineup; q++) {
            const int32_t a = c->path_link[q], b2 = c->path_link[q + 1];
            if (a < 0 || b2 < 0) continue;
            if ((pre[b2] >= 0 && pre[b2] != a) || (nxt[a] >= 0 && nxt[a] != b2)) lineup = false;
            pre[b2] = a;
            nxt[a] = b2;
            if (++npair[a] > 1 && c->arb == SIM_ARB_LOWEST_ID && bmax_all > 1) lineup = false;
        }
        std::vector<int32_t> order;
        std::vector<char> seen(m, 0);
        for (int32_t l : fsrc) {
            if (!lineup || pre[l] >= 0) continue;
            for (int32_t v = l; v >= 0; v = nxt[v]) {
                if (seen[v]) { lineup = false; break; }
                seen[v] = 1;
                order.push_back(v);
            }
        }
        if (lineup && order.size() == fsrc.size()) fsrc = order;
        else lineup = false;  // a cycle of feeders (never reached from a path start)
    }
    std::vector<int32_t> nports(c->n, 0), port_at_head(m), nports_tail(m);
    for (int32_t l = 0; l < m; l++) port_at_head[l] = nports[c->col_idx[l]]++;
    for (int32_t v = 0; v < c->E; v++) nports[v]++;  // injection port last
    for (int32_t l = 0; l < m; l++) nports_tail[l] = nports[c->tail[l]];
    int32_t bmax = 1;
    for (int32_t v : c->bw) bmax = std::max(bmax, v);
    std::vector<int32_t> fifo_off(m, 0), fifo_mask(m, 0), req_off(m, 0);
    int64_t ftot = 0, rtot = 0;
    for (int32_t l = 0; l < m; l++) {
        int32_t capmax = 1;
        for (int32_t s = 0; s < c->S; s++) capmax = std::max(capmax, c->cap[(size_t)s * m + l]);
        int32_t ring = 1;
        while (ring < capmax) ring <<= 1;
        if (!used[l]) ring = 1;
        fifo_off[l] = (int32_t)ftot;
        fifo_mask[l] = ring - 1;
        ftot += ring;
        req_off[l] = (int32_t)rtot;
        if (used[l]) rtot += (int64_t)nports_tail[l] * bmax;
    }
    if (ftot >= INT32_MAX || rtot >= INT32_MAX) return fail(c, SIM_ERR_SIZE, "state too large");

    // Which links carry traffic, and which of them start an injection stream.
    const int32_t nl = (int32_t)fsrc.size();
    std::vector<char> has_stream(m, 0);
    for (int32_t f : s_link) has_stream[f] = 1;
    int32_t bm = 1;
    while (bm < bmax) bm <<= 1;
    bool rr_ports_fit = true;  // every input-port set fits a 64-bit mask
    for (int32_t l : fsrc)
        if (nports_tail[l] > 64) rr_ports_fit = false;
    const bool any_preds = !pd_flow.empty();

    // Engine choice.  Wave engine for small graphs batched many to a
    // wavefront; lane engine with FIFO rings in LDS when a scenario fits a
    // workgroup's LDS; the compact b = 1 engine for large single-line-rate
    // graphs; the lane engine with FIFO rings in HBM when only its mailboxes
    // fit; else the workgroup engine, resident in LDS when its per-scenario
    // state fits.  One large topology goes to the grid engine when its
    // one-line or windowed form applies.
    auto align16 = [](int64_t v) { return (v + 15) & ~(int64_t)15; };
    const int64_t kLds = 160 * 1024;
    int64_t lf = 0;
    for (int32_t l : fsrc) lf += fifo_mask[l] + 1;
    // mailbox slots of the lane engine: feeders of each target lane x bmax
    std::vector<int32_t> link_lane(m, -1);
    for (int32_t i = 0; i < nl; i++) link_lane[fsrc[i]] = i;
    const std::vector<int32_t> fsrc_pos(link_lane);  // position of a traffic link in fsrc
    std::vector<std::vector<int32_t>> feeders(nl);
    for (size_t q = 0; q + 1 < c->path_link.size(); q++) {
        const int32_t a = c->path_link[q], b2 = c->path_link[q + 1];
        if (a >= 0 && b2 >= 0) feeders[link_lane[b2]].push_back(link_lane[a]);
    }
    int64_t lr = 0;
    for (int32_t i = 0; i < nl; i++) {
        auto &fv = feeders[i];
        std::sort(fv.begin(), fv.end());
        fv.erase(std::unique(fv.begin(), fv.end()), fv.end());
        lr += (int64_t)((int32_t)fv.size() + (has_stream[fsrc[i]] ? 1 : 0)) * bmax;
    }
    // Wave engine tables: every lane's local flows (at most four cross a
    // link), the feeders of every lane as a target, each range's local flow
    // at its first lane, and the scenario slots of every wave (scenarios
    // with the most lines per cycle of bandwidth on their busiest link first,
    // so that the longest runs start first).
    struct WaveLayout {
        bool ok = false;
        bool lineup = false;  // the shift loop: paths of links on consecutive lanes
        int32_t G = 0, W = 0, nfs = 0;
        int32_t nblk = 0, wpb = 0;
        int64_t o_word = 0, o_red = 0, o_deliv = 0, o_req = 0, o_gnt = 0, o_gdep = 0, bytes = 0;
    };
    WaveLayout wv;
    std::vector<uint32_t> wv_lfb, wv_lfx;
    std::vector<int32_t> wv_feed, wv_nfeed, wv_sc, r_lf, pd_dix, blk_wave, blk_off;
    std::vector<uint32_t> wv_duo;
    constexpr int64_t kWaveBlockLds = 160 * 1024;  // LDS of a compute unit
    // compute units of the current device (256 on MI355X)
    int32_t wave_blocks = 256;
    {
        int cur = 0, ncu = 0;
        if (hipGetDevice(&cur) == hipSuccess &&
            hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, cur) == hipSuccess && ncu > 0)
            wave_blocks = ncu;
    }
    {
        std::vector<std::vector<int32_t>> lflows(nl);
        bool ok = nl >= 1 && nl <= 64 && T < (1ll << 25) - 1 && bm <= 8;
        for (int32_t f = 0; ok && f < nflows; f++)
            for (int64_t q = c->flow_path[f]; ok && c->path_link[q] >= 0; q++) {
                auto &v = lflows[link_lane[c->path_link[q]]];
                v.push_back(f);
                if (v.size() > 4) ok = false;
                if (c->path_link[q + 1] == c->path_link[q]) ok = false;  // the sink encoding needs this
            }
        int32_t maxfeed = 0;
        for (int32_t i = 0; i < nl; i++) maxfeed = std::max(maxfeed, (int32_t)feeders[i].size());
        const int32_t nfs = maxfeed + 1 <= 2 ? 2 : simgpu::kWaveMaxNF;
        if (maxfeed + 1 > simgpu::kWaveMaxNF || nfs * bm > 32) ok = false;
        for (int32_t l : fsrc)
            if (nports_tail[l] > 255) ok = false;
        if (ok) {
            auto lf_index = [&](int32_t lane, int32_t f) {
                const auto &v = lflows[lane];
                return (int32_t)(std::find(v.begin(), v.end(), f) - v.begin());
            };
            // byte q of wv_lfb: local index at the next lane << 6 | next lane (the
            // lane itself: the line leaves the network, as a minimal path never
            // takes a link twice); byte q of wv_lfx: this lane's feeder
            // index at the next lane.  A flow's delivered counter sits at
            // (its last lane) * 4 + (its local index there).
            wv_lfb.assign(nl, 0u);
            wv_lfx.assign(nl, 0u);
            std::vector<int32_t> flow_dix(nflows, 0);
            for (int32_t f = 0; f < nflows; f++)
                for (int64_t q = c->flow_path[f]; c->path_link[q] >= 0; q++) {
                    const int32_t ln = link_lane[c->path_link[q]];
                    const int32_t nx = c->path_link[q + 1];
                    const uint32_t sh = 8u * (uint32_t)lf_index(ln, f);
                    if (nx < 0) {
                        wv_lfb[ln] |= (uint32_t)ln << sh;
                        flow_dix[f] = ln * 4 + lf_index(ln, f);
                    } else {
                        const int32_t ln2 = link_lane[nx];
                        const auto &fv = feeders[ln2];
                        const int32_t fi = (int32_t)(std::find(fv.begin(), fv.end(), ln) - fv.begin());
                        wv_lfb[ln] |= ((uint32_t)ln2 | ((uint32_t)lf_index(ln2, f) << 6)) << sh;
                        wv_lfx[ln] |= (uint32_t)fi << sh;
                    }
                }
            pd_dix.resize(pd_flow.size());
            for (size_t q = 0; q < pd_flow.size(); q++) pd_dix[q] = flow_dix[pd_flow[q]];
            wv_feed.assign((size_t)nl * 4, 0);
            wv_nfeed.assign(nl, 0);
            for (int32_t i = 0; i < nl; i++) {
                wv_nfeed[i] = (int32_t)feeders[i].size();
                for (size_t f = 0; f < feeders[i].size(); f++)
                    wv_feed[(size_t)i * 4 + f] = feeders[i][f] | (port_at_head[fsrc[feeders[i][f]]] << 8);
            }
            // The shift loop (no credit delays): a lane's feeder is the lane
            // before it and the lines it sends on go to the lane after it;
            // wv_duo[i] = the local flows bound for that lane.  Under lowest-id
            // arbitration with several lines per cycle, one flow at most is
            // bound for it, so that the lines it offers there are in id order.
            wv.lineup = lineup && c->credit.empty();
            wv_duo.assign(nl, 0);
            for (int32_t i = 0; i < nl && wv.lineup; i++) {
                uint32_t tm = 0;
                for (size_t q = 0; q < lflows[i].size(); q++) {
                    const int32_t lb = (int32_t)((wv_lfb[i] >> (8 * q)) & 63u);
                    if (lb == i) continue;
                    if (lb != i + 1) wv.lineup = false;
                    tm |= 1u << q;
                }
                if (feeders[i].size() > 1 || (feeders[i].size() == 1 && feeders[i][0] != i - 1)) wv.lineup = false;
                if (c->arb == SIM_ARB_LOWEST_ID && bmax > 1 && __builtin_popcount(tm) > 1) wv.lineup = false;
                wv_duo[i] = tm;
            }
            if (const char *ev = std::getenv("SIMGPU_WAVE_LOOP"))
                if (!std::strcmp(ev, "general")) wv.lineup = false;  // tests: the arbitration loops on such graphs
            r_lf.assign(nr, 0);
            for (int64_t j = 0; j < nr; j++)
                r_lf[j] = lf_index(link_lane[c->path_link[r_path[j]]], rflow[order[j]]);
            const int32_t S = c->S;
            const int32_t G = std::min(64 / nl, S);
            std::vector<double> lcnt(nl, 0.0);
            for (int64_t j = 0; j < nr; j++)
                for (int64_t q = r_path[j]; c->path_link[q] >= 0; q++) lcnt[link_lane[c->path_link[q]]] += r_len[j];
            // A wave runs the b = 1 loop only if all its scenarios can, and runs
            // as long as its longest scenario: waves hold scenarios of one
            // bandwidth bound only, in order of expected length (lines per unit
            // of bandwidth on the busiest link, then smaller buffers first).
            std::vector<double> est(S, 0.0);
            std::vector<int32_t> mincap(S, SIM_MAX_CAP), sbmax(S, 1), ord(S);
            for (int32_t s = 0; s < S; s++) {
                for (int32_t i = 0; i < nl; i++) {
                    const size_t pi = (size_t)s * m + fsrc[i];
                    est[s] = std::max(est[s], lcnt[i] / c->bw[pi]);
                    mincap[s] = std::min(mincap[s], c->cap[pi]);
                    sbmax[s] = std::max(sbmax[s], c->bw[pi]);
                }
                ord[s] = s;
            }
            std::stable_sort(ord.begin(), ord.end(), [&](int32_t a, int32_t b2) {
                if (sbmax[a] != sbmax[b2]) return sbmax[a] < sbmax[b2];
                return est[a] != est[b2] ? est[a] > est[b2] : mincap[a] < mincap[b2];
            });
            wv_sc.clear();
            for (int32_t k = 0; k < S; k++) {
                const bool new_wave = wv_sc.size() % G == 0 || sbmax[ord[k]] != sbmax[ord[k - 1]];
                if (new_wave)
                    while (wv_sc.size() % G) wv_sc.push_back(-1);
                wv_sc.push_back(ord[k]);
            }
            while (wv_sc.size() % G) wv_sc.push_back(-1);
            const int32_t W = (int32_t)(wv_sc.size() / G);
            // A wave's LDS region: its rings (+ one trash entry per lane), then
            // words (64 + 64 trash) | reduction slots (64 + 64 trash) | delivered counters |
            // for the general loop: request slots, grants, void flags (each +
            // 64 trash).  Offsets below are relative to the end of the rings.
            const bool general = bm > 1 || c->arb == SIM_ARB_ROUND_ROBIN;
            int64_t off = 0;
            wv.o_word = off;
            off += 128 * 4;
            wv.o_red = off;
            off += 128 * 4;
            wv.o_deliv = off;
            off = align16(off + (int64_t)G * nl * 4 * 4);
            const int64_t tail_fast = off;
            wv.o_req = off;
            // the general loop's slots, grants and void flags for a wave whose
            // bandwidth bound rounds up to wb
            auto tail_gen = [&](int64_t wb) {
                return tail_fast + align16(((int64_t)64 * nfs * wb + 64) * 8) + align16(((int64_t)64 * wb + 64) * 8) +
                       align16(((int64_t)64 * wb + 64) * 4);
            };
            std::vector<int64_t> wbytes(W);
            bool fits = true;
            for (int32_t q = 0; q < W; q++) {
                int64_t ringn = 0;
                int32_t wbmax = 1;
                for (int32_t g = 0; g < G; g++) {
                    const int32_t s = wv_sc[(size_t)q * G + g];
                    if (s < 0) continue;
                    for (int32_t i = 0; i < nl; i++) {
                        const int64_t cp = c->cap[(size_t)s * m + fsrc[i]];
                        ringn += cp + ((1 - cp) & 15);  // padded as the kernel does
                        wbmax = std::max(wbmax, c->bw[(size_t)s * m + fsrc[i]]);
                    }
                }
                // lanes without a link still take one padding entry each
                int32_t on_lanes = 0;
                for (int32_t g = 0; g < G; g++)
                    if (wv_sc[(size_t)q * G + g] >= 0) on_lanes += nl;
                ringn += 64 - on_lanes;
                int64_t wb = 1;
                while (wb < wbmax) wb <<= 1;
                const bool fast = c->arb == SIM_ARB_LOWEST_ID && wbmax == 1;
                wbytes[q] = align16((ringn + 64) * 8) + ((general && !fast && !wv.lineup) ? tail_gen(wb) : tail_fast);
                if (wbytes[q] > kWaveBlockLds) fits = false;
            }
            // Estimated run time of each wave, for placement only: its longest
            // scenario's processed cycles (lines on the busiest link per cycle
            // of bandwidth, plus a few fill/drain cycles per buffer's worth of
            // lines) times the relative cost of a cycle of the loop it runs
            // (the b = 1 loop, or the general loop unrolled to 1, 2, 4, 8).
            std::vector<double> wtime(W, 0.0);
            for (int32_t q = 0; q < W; q++) {
                double cyc = 0.0;
                int32_t wbmax = 1;
                for (int32_t g = 0; g < G; g++) {
                    const int32_t s = wv_sc[(size_t)q * G + g];
                    if (s < 0) continue;
                    for (int32_t i = 0; i < nl; i++) {
                        const size_t pi = (size_t)s * m + fsrc[i];
                        cyc = std::max(cyc, lcnt[i] / c->bw[pi] + 4.0 * lcnt[i] / c->cap[pi]);
                        wbmax = std::max(wbmax, c->bw[pi]);
                    }
                }
                const bool fast = c->arb == SIM_ARB_LOWEST_ID && wbmax == 1;
                const double per = wv.lineup ? (wbmax <= 1 ? 0.5 : wbmax <= 2 ? 0.8 : wbmax <= 4 ? 1.2 : 2.0)
                                   : fast ? 1.0 : wbmax <= 1 ? 1.5 : wbmax <= 2 ? 1.8 : wbmax <= 4 ? 2.9 : 5.5;
                wtime[q] = cyc * per;
            }
            std::vector<std::vector<int32_t>> blk;
            int64_t lds_floor = 0;
            // A compute unit has four SIMDs and runs the waves of one workgroup
            // on them in turn (wave j on SIMD j mod 4).  When there are more
            // waves than SIMDs, the shortest waves share a SIMD two by two
            // (a pair sits at positions j and j + 4 of a workgroup) and the
            // longest run alone; each workgroup takes four SIMD slots and has a
            // compute unit to itself (below).
            const int32_t nsimd = 4 * wave_blocks;
            if (fits && W > nsimd && W <= 2 * nsimd) {
                const int32_t E = W - nsimd;  // SIMDs holding two waves
                std::vector<int32_t> qs(W);
                for (int32_t q = 0; q < W; q++) qs[q] = q;
                std::stable_sort(qs.begin(), qs.end(), [&](int32_t a, int32_t b2) { return wtime[a] > wtime[b2]; });
                // slots: the W - 2E longest alone; the 2E shortest paired,
                // longest of them with shortest
                struct Slot { int32_t a, b; int64_t bytes; };
                std::vector<Slot> slots;
                for (int32_t k = 0; k < W - 2 * E; k++) slots.push_back({qs[k], -1, wbytes[qs[k]]});
                for (int32_t k = 0; k < E; k++) {
                    const int32_t a = qs[W - 2 * E + k], b2 = qs[W - 1 - k];
                    slots.push_back({a, b2, wbytes[a] + wbytes[b2]});
                }
                std::stable_sort(slots.begin(), slots.end(), [](const Slot &x, const Slot &y) { return x.bytes > y.bytes; });
                std::vector<std::vector<Slot>> bs(wave_blocks);
                std::vector<int64_t> bb(wave_blocks, 0);
                bool ok2 = true;
                for (const Slot &sl : slots) {
                    int32_t best = -1;
                    for (int32_t k = 0; k < wave_blocks; k++) {
                        if (bs[k].size() >= 4 || bb[k] + sl.bytes > kWaveBlockLds) continue;
                        if (best < 0 || bb[k] < bb[best]) best = k;
                    }
                    if (best < 0) {
                        ok2 = false;
                        break;
                    }
                    bs[best].push_back(sl);
                    bb[best] += sl.bytes;
                }
                if (ok2) {
                    // positions: pairs' first waves, lone waves, then the pairs'
                    // second waves at position + 4 (-1 = no wave)
                    blk.resize(wave_blocks);
                    for (int32_t k = 0; k < wave_blocks; k++) {
                        std::stable_sort(bs[k].begin(), bs[k].end(), [](const Slot &x, const Slot &y) {
                            return (x.b >= 0) > (y.b >= 0);
                        });
                        auto &v = blk[k];
                        for (const Slot &sl : bs[k]) v.push_back(sl.a);
                        while (v.size() < 4) v.push_back(-1);
                        for (const Slot &sl : bs[k])
                            if (sl.b >= 0) v.push_back(sl.b);
                    }
                }
            }
            if (blk.empty()) {
                // Otherwise pack the waves into workgroups of up to kWaveMaxWpb
                // independent waves and at most kWaveBlockLds bytes, aiming at one
                // workgroup per compute unit so that every wave is resident at
                // once: largest first, each into the workgroup with the fewest
                // waves that has room.
                std::vector<int32_t> qord(W);
                for (int32_t q = 0; q < W; q++) qord[q] = q;
                std::stable_sort(qord.begin(), qord.end(), [&](int32_t a, int32_t b2) { return wbytes[a] > wbytes[b2]; });
                blk.resize(std::min<int32_t>(wave_blocks, W));
                std::vector<int64_t> bbytes(blk.size(), 0);
                for (int32_t q : qord) {
                    if (!fits) break;
                    int32_t best = -1;
                    for (int32_t k = 0; k < (int32_t)blk.size(); k++) {
                        if ((int32_t)blk[k].size() >= simgpu::kWaveMaxWpb || bbytes[k] + wbytes[q] > kWaveBlockLds) continue;
                        if (best < 0 || blk[k].size() < blk[best].size() ||
                            (blk[k].size() == blk[best].size() && bbytes[k] < bbytes[best]))
                            best = k;
                    }
                    if (best < 0) {
                        blk.emplace_back();
                        bbytes.push_back(0);
                        best = (int32_t)blk.size() - 1;
                    }
                    blk[best].push_back(q);
                    bbytes[best] += wbytes[q];
                }
                // waves of a workgroup in scenario order (longest expected first);
                // workgroups ordered by their first wave
                for (auto &v : blk) std::sort(v.begin(), v.end());
                std::stable_sort(blk.begin(), blk.end(), [](const std::vector<int32_t> &a, const std::vector<int32_t> &b2) {
                    return (a.empty() ? INT32_MAX : a[0]) < (b2.empty() ? INT32_MAX : b2[0]);
                });
            }
            int32_t wpb = 1;
            int64_t lmax = 16;
            for (auto &v : blk) wpb = std::max(wpb, (int32_t)v.size());
            blk_wave.assign(blk.size() * wpb, -1);
            blk_off.assign(blk.size() * wpb, 0);
            for (size_t k = 0; k < blk.size(); k++) {
                int64_t o2 = 0;
                for (size_t j = 0; j < blk[k].size(); j++) {
                    const int32_t q = blk[k][j];
                    blk_wave[k * wpb + j] = q;
                    blk_off[k * wpb + j] = (int32_t)o2;
                    if (q >= 0) o2 += wbytes[q];
                }
                lmax = std::max(lmax, o2);
            }
            // no more workgroups than compute units: each reserves more than half
            // of the LDS, so that no two share a compute unit while another idles
            if ((int32_t)blk.size() <= wave_blocks) lds_floor = kWaveBlockLds / 2 + 16;
            lmax = std::max(lmax, lds_floor);
            wv.bytes = lmax;
            wv.G = G;
            wv.W = W;
            wv.nblk = (int32_t)blk.size();
            wv.wpb = wpb;
            wv.nfs = nfs;
            wv.ok = fits && wv.bytes <= kWaveBlockLds;
        }
    }
    const int64_t path_bytes = (int64_t)c->path_link.size() * 4;
    struct LaneLayout { int64_t o_path, o_deliv, o_reqcnt, o_reqb, o_req, o_glist, o_grant, o_gdep, o_red, bytes; bool path_lds; };
    auto lane_layout = [&](bool fifo_lds) {
        LaneLayout L{};
        int64_t off = fifo_lds ? lf * 16 : 0;
        L.o_path = off;
        L.path_lds = path_bytes <= 16384;
        if (L.path_lds) off = align16(off + path_bytes);
        L.o_deliv = off;
        off = align16(off + (int64_t)nflows * 4);
        L.o_reqcnt = off;
        off = align16(off + (int64_t)nl * 4);
        L.o_reqb = off;
        off = align16(off + (int64_t)nl * 8);
        L.o_req = off;
        off = align16(off + lr * 16);
        L.o_glist = off;
        off = align16(off + (int64_t)nl * bm * 4);
        L.o_grant = off;
        off = align16(off + (int64_t)2 * nl * bm * 4);
        L.o_gdep = off;
        off = align16(off + (int64_t)nl * bm * 4);
        L.o_red = off;
        L.bytes = align16(off + 64);
        return L;
    };
    const LaneLayout lay_lds = lane_layout(true), lay_hbm = lane_layout(false);
    // compact engine LDS: one request word per target lane (+ grant words and
    // the in-link lane table for round-robin), delivered counters if they fit
    // words (lowest-id: two buffers) | grant words + in-lane table (round-robin)
    // | per-lane counters | delivered counters if they fit | reduction slots
    // round-robin: request masks + posts (8 B per lane) + in-lane table (u16);
    // lowest-id: two buffers of request words; then one counter per lane
    // (+ in-lane offsets, u16) then one counter per lane
    const int64_t b1_words = (c->arb == SIM_ARB_ROUND_ROBIN ? (int64_t)nl * 16 + align16((int64_t)m * 2) +
                                                                  align16((int64_t)nl * 2)
                                                            : (int64_t)nl * 16) +
                             (int64_t)nl * 4;
    int32_t b1_ring = 1;
    for (int32_t l : fsrc) b1_ring = std::max(b1_ring, fifo_mask[l] + 1);
    const bool b1_deliv_lds = any_preds && align16(b1_words) + (int64_t)nflows * 4 + 64 <= kLds;
    const int64_t b1_bytes = align16(align16(b1_words) + (b1_deliv_lds ? (int64_t)nflows * 4 : 0)) + 64;
    // the compact engine keeps delivered counters in LDS only (its phases wait
    // on LDS, never on global memory), and round-robin keeps the in-link lane
    // table and each lane's offset in it as 16-bit values
    const bool b1_ok = bmax == 1 && (int64_t)s_link.size() <= 1024 && nl <= 8 * 1024 && b1_bytes <= kLds &&
                       (!any_preds || b1_deliv_lds) &&
                       (c->arb == SIM_ARB_LOWEST_ID || (rr_ports_fit && m < 65536));
    // credit delays above 1 are simulated by the wave engine (not together
    // with per-chunk dependencies), the workgroup engine (both forms) and the
    // grid engine's windowed form; class-fair arbitration by the workgroup
    // engine (both forms)
    const bool credits = !c->credit.empty();
    const bool fair = (c->arb & SIM_ARB_FAIR_CLASSES) != 0;
    // Grid engine (one scenario over many workgroups): nodes are split over
    // the workgroups by longest-processing-time assignment of their lanes
    // (target sides of out-links, source sides of in-links, a stream), so
    // that every workgroup's per-cycle work is about the same.
    GridLayout gl;
    const bool grid_try = c->S == 1 && !fair && nl >= 1 && bm <= 64;
    if (grid_try) {
        int want_nb = 32;
        if (const char *ev = std::getenv("SIMGPU_GRID_WGS")) want_nb = std::max(1, std::min(32, std::atoi(ev)));
        gl = grid_layout(c, fsrc, has_stream, feeders, fsrc_pos, bmax, bm, nflows, pd_flow, want_nb, port_at_head,
                         nports);
        if (std::getenv("SIMGPU_GRID_GENERAL")) gl.one = false;  // tests: the general form on b = 1 graphs
        if (gl.one && gl.one_bytes <= kLds) {
            gl.bytes = gl.one_bytes;
            gl.threads = gl.one_threads;
        } else {
            gl.one = false;
        }
        // Credit delays: the windowed form, when every traffic link has
        // latency and credit delay of at least 2 and no line waits on another.
        if (credits) {
            int32_t win = INT32_MAX;
            for (int32_t l : fsrc) win = std::min(win, std::min(c->lat[l], c->credit[l]));
            if (gl.one && !any_preds && win >= 2) {
                std::vector<int32_t> ring_of(nl);
                for (int32_t i = 0; i < nl; i++) ring_of[i] = fifo_mask[fsrc[i]] + 1;
                gl.sro.assign(nl, 0);
                gl.tro.assign(nl, 0);
                int64_t smax = 0, tmax = 0;
                for (int32_t w = 0; w < gl.nb; w++) {
                    int64_t so = 0, to = 0;
                    for (int32_t q = gl.sptr[w]; q < gl.sptr[w + 1]; q++) {
                        gl.sro[gl.slane[q]] = (int32_t)so;
                        so += ring_of[gl.slane[q]];
                    }
                    for (int32_t q = gl.tptr[w]; q < gl.tptr[w + 1]; q++) {
                        gl.tro[gl.tlane[q]] = (int32_t)to;
                        to += ring_of[gl.tlane[q]];
                    }
                    smax = std::max(smax, so);
                    tmax = std::max(tmax, to);
                }
                auto a16 = [](int64_t v) { return (v + 15) & ~(int64_t)15; };
                int64_t b = a16(8 * (int64_t)gl.nt_max * (c->arb == SIM_ARB_LOWEST_ID ? 2 : 1));
                if (c->arb == SIM_ARB_ROUND_ROBIN) b += a16(8 * (int64_t)gl.ns_max) + a16(4 * (int64_t)gl.inl_max);
                b += a16(16 * smax) + a16(4 * tmax) + a16(4 * 4 * 2 * 16) + a16(4 * 32);
                gl.window = win;
                gl.sring_max = (int32_t)smax;
                gl.cring_max = (int32_t)tmax;
                gl.bytes = b;
            } else {
                gl.bytes = INT64_MAX;  // credit delays need the windowed form
            }
        }
    }
    const bool grid_ok = grid_try && gl.bytes <= kLds;
    // Resident workgroup engine: a scenario's per-link state and parameters
    // and the cycle's request records in LDS.  16-bit positions and counts
    // (rings of at most 2^15 entries, fewer than 2^16 requests per target
    // and cycle, links and sources below 2^16, latencies and credit delays
    // below 2^16), records past the LDS capacity in HBM.  Workgroups per CU:
    // the most (up to 4, as many as the batch needs) whose LDS leaves room
    // for at least 256 records.
    struct ResLayout {
        bool ok = false;
        int64_t off[24] = {};
        int64_t bytes = 0, rcap = 0, scap = 0, ovf = 0, tcap = 0, tovf = 0;
        int32_t threads = 256, nw = 1;
    } res;
    {
        const int64_t nsrc_all = (int64_t)m + (int64_t)s_link.size();
        bool ok = m <= 65535 && nsrc_all <= 65535 && bmax <= 64;
        int64_t qmax = 0;  // request records one cycle can need
        for (int32_t l : fsrc) {
            ok = ok && fifo_mask[l] + 1 <= 32768 && (int64_t)nports_tail[l] * bmax <= 65533 && nports_tail[l] <= 255;
            int32_t bl = 1;
            for (int32_t sc = 0; sc < c->S; sc++) bl = std::max(bl, c->bw[(size_t)sc * m + l]);
            qmax += std::min<int64_t>(bl, fifo_mask[l] + 1) + (has_stream[l] ? bl : 0);
        }
        for (size_t i = 0; i < c->lat.size() && ok; i++) ok = c->lat[i] <= 65535;
        for (size_t i = 0; i < c->credit.size() && ok; i++) ok = c->credit[i] <= 65535;
        ok = ok && qmax < (1 << 24);
        auto a4 = [](int64_t v) { return (v + 3) & ~(int64_t)3; };
        int64_t scap = bmax > 4 ? std::min<int64_t>(512, (int64_t)m * ((bmax - 1) / 4)) : 0;
        if (const char *ev = std::getenv("SIMGPU_SPILL_CAP"))  // tests: a short spill list (later chunks inline)
            scap = std::max<int64_t>(0, std::min<int64_t>(scap, std::atoll(ev)));
        const int64_t sizes[17] = {2 * (int64_t)m, 2 * (int64_t)m, credits ? 2 * (int64_t)m : 0, 2 * (int64_t)m,
                                   4 * (int64_t)m, m, (c->arb & SIM_ARB_ROUND_ROBIN) ? m : 0, 2 * (int64_t)m,
                                   2 * (int64_t)m, credits ? 2 * (int64_t)m : 0, 4 * nsrc_all,
                                   4 * (int64_t)s_link.size(), 4 * (int64_t)s_link.size(),
                                   4 * ((nsrc_all + 31) / 32), 2 * nsrc_all, 2 * (int64_t)m, 4 * scap};
        int64_t o = 0;
        for (int i = 0; i < 17; i++) {
            res.off[i] = o;
            o += a4(sizes[i]);
        }
        res.off[18] = o;  // input ports per link (round-robin)
        o += a4((c->arb & SIM_ARB_ROUND_ROBIN) ? m : 0);
        int32_t sbw = 1;  // widest stream link: windows of ranges per stream
        for (int32_t f : s_link)
            for (int32_t sc = 0; sc < c->S; sc++) sbw = std::max(sbw, c->bw[(size_t)sc * m + f]);
        res.nw = (sbw + simgpu::kResWindow - 1) / simgpu::kResWindow;
        res.off[19] = o;  // a check result per stream window
        o += a4(2 * (int64_t)s_link.size() * res.nw);
        res.tcap = std::min<int64_t>(m, 256);  // per-target words of a cycle's targets
        if (const char *ev = std::getenv("SIMGPU_RES_TCAP"))  // tests: later targets' words in HBM
            res.tcap = std::max<int64_t>(1, std::min<int64_t>(res.tcap, std::atoll(ev)));
        res.tovf = (int64_t)m - res.tcap;
        res.off[21] = o;  // per stream: its link, one past its last range
        o += 4 * (int64_t)s_link.size();
        res.off[22] = o;
        o += 4 * (int64_t)s_link.size();
        res.off[23] = o;  // class-fair arbitration: the class whose turn it is per link
        o += a4(fair ? m : 0);
        o = (o + 7) & ~(int64_t)7;  // 64-bit words first
        res.off[20] = o;
        o += 14 * res.tcap;
        o = (o + 7) & ~(int64_t)7;
        res.off[17] = o;  // request records last
        const int64_t room = kLds - 1024;  // room for the static LDS
        const int want = c->S > 512 ? 4 : c->S > 256 ? 2 : 1;
        for (int k = want; k >= 1 && ok && !res.ok; k--) {
            const int64_t avail = room / k - o;
            const int64_t rb = fair ? 32 : 30;  // record bytes (class-fair: a count of requests ahead)
            const int64_t rcap = std::min<int64_t>({qmax, avail / rb, 4096});
            if (rcap < std::min<int64_t>(qmax, 256)) continue;
            res.ok = true;
            res.rcap = std::max<int64_t>(rcap, 1);
            if (const char *ev = std::getenv("SIMGPU_RES_RCAP"))  // tests: later request records in HBM
                res.rcap = std::max<int64_t>(1, std::min<int64_t>(res.rcap, std::atoll(ev)));
            res.scap = scap;
            res.ovf = std::max<int64_t>(0, qmax - res.rcap);
            res.bytes = o + rb * res.rcap;
            res.threads = k == 1 ? 1024 : k == 2 ? 512 : 256;
        }
    }
    if ((credits && R.whole) || fair) wv.ok = false;
    const bool lane_ok = !credits && !fair && nl >= 1 && nl <= 1024 && bm <= 64 && lay_lds.bytes <= kLds;
    const bool lanehbm_ok = !credits && !fair && nl >= 1 && nl <= 1024 && bm <= 64 && lay_hbm.bytes <= kLds;
    const bool b1_usable = !credits && !fair && nl >= 1 && b1_ok;
    int engine = simgpu::kEngineWorkgroup;
    if (wv.ok) engine = simgpu::kEngineWave;
    else if (lane_ok) engine = simgpu::kEngineLane;
    else if (b1_usable) engine = simgpu::kEngineB1;
    else if (lanehbm_ok) engine = simgpu::kEngineLaneHbm;
    // One large topology whose lines move one per cycle per link: the grid
    // engine's one-line form spreads it over many CUs at a lower time per
    // processed cycle than the single-workgroup compact and HBM engines.
    if (grid_ok && gl.one && (engine == simgpu::kEngineB1 || engine == simgpu::kEngineLaneHbm ||
                              engine == simgpu::kEngineWorkgroup))
        engine = simgpu::kEngineGrid;
    if (engine == simgpu::kEngineWorkgroup && res.ok) engine = simgpu::kEngineResident;
    bool wg_scan = false;  // workgroup engine without active sets (tests)
    if (const char *ev = std::getenv("SIMGPU_ENGINE")) {
        int want = -1;
        if (!std::strcmp(ev, "workgroup")) want = simgpu::kEngineWorkgroup;
        if (!std::strcmp(ev, "workgroup_scan")) {
            want = simgpu::kEngineWorkgroup;
            wg_scan = true;
        }
        if (!std::strcmp(ev, "lane")) want = simgpu::kEngineLane;
        if (!std::strcmp(ev, "lanehbm")) want = simgpu::kEngineLaneHbm;
        if (!std::strcmp(ev, "b1")) want = simgpu::kEngineB1;
        if (!std::strcmp(ev, "wave")) want = simgpu::kEngineWave;
        if (!std::strcmp(ev, "grid")) want = simgpu::kEngineGrid;
        if (!std::strcmp(ev, "resident")) want = simgpu::kEngineResident;
        const bool ok = want == simgpu::kEngineWorkgroup || (want == simgpu::kEngineWave && wv.ok) ||
                        (want == simgpu::kEngineResident && res.ok) ||
                        (want == simgpu::kEngineGrid && grid_ok) ||
                        (want == simgpu::kEngineLane && lane_ok) || (want == simgpu::kEngineLaneHbm && lanehbm_ok) ||
                        (want == simgpu::kEngineB1 && b1_usable);
        if (want < 0 || !ok) return fail(c, SIM_ERR_INVALID_ARG, std::string("SIMGPU_ENGINE=") + ev + " is not usable here");
        engine = want;
    }

    // Lane order: traffic links ascending; the compact engine puts the links
    // that start a stream first so that stream j is owned by thread j.
    std::vector<int32_t> lane_link(fsrc);
    if (engine == simgpu::kEngineB1)
        std::stable_partition(lane_link.begin(), lane_link.end(), [&](int32_t l) { return has_stream[l] != 0; });
    for (int32_t i = 0; i < nl; i++) link_lane[lane_link[i]] = i;
    std::vector<int32_t> path_lane(c->path_link.size());
    for (size_t q = 0; q < c->path_link.size(); q++) {
        int32_t v = c->path_link[q];
        path_lane[q] = v >= 0 ? link_lane[v] : v;
    }
    std::vector<int32_t> ln_P(nl), ln_port(nl), ln_fifo(nl), ln_mask(nl), ln_req(nl), ln_reqcap(nl),
        ln_srbeg(nl, 0), ln_srend(nl, 0);
    for (size_t j = 0; j < s_link.size(); j++) {
        ln_srbeg[link_lane[s_link[j]]] = s_rbeg[j];
        ln_srend[link_lane[s_link[j]]] = s_rend[j];
    }
    {
        int64_t f = 0, r = 0;
        for (int32_t i = 0; i < nl; i++) {
            const int32_t l = lane_link[i];
            ln_P[i] = nports_tail[l];
            ln_port[i] = port_at_head[l];
            ln_fifo[i] = (int32_t)f;
            ln_mask[i] = fifo_mask[l];
            f += fifo_mask[l] + 1;
            // feeders were collected in fsrc order
            const int32_t nfeed = (int32_t)feeders[fsrc_pos[l]].size() +
                                  (has_stream[l] ? 1 : 0);
            ln_req[i] = (int32_t)r;
            ln_reqcap[i] = nfeed * bmax;
            r += (int64_t)nfeed * bmax;
        }
    }
    // round-robin port -> lane table of the compact engine: for every node,
    // the lanes of its in-links in port order (-1 for links without traffic)
    std::vector<int32_t> node_inoff(c->n + 1, 0), in_lane(m, -1), ln_inoff(nl, 0);
    for (int32_t l = 0; l < m; l++) node_inoff[c->col_idx[l] + 1]++;
    for (int32_t v = 0; v < c->n; v++) node_inoff[v + 1] += node_inoff[v];
    for (int32_t l = 0; l < m; l++) in_lane[node_inoff[c->col_idx[l]] + port_at_head[l]] = link_lane[l];
    for (int32_t i = 0; i < nl; i++) ln_inoff[i] = node_inoff[c->tail[lane_link[i]]];
    const LaneLayout &lay = engine == simgpu::kEngineLane ? lay_lds : lay_hbm;
    const bool path_in_lds = lay.path_lds;
    const int64_t lds_bytes = engine == simgpu::kEngineB1     ? b1_bytes
                              : engine == simgpu::kEngineWave ? wv.bytes
                              : engine == simgpu::kEngineGrid ? gl.bytes
                              : engine == simgpu::kEngineResident ? res.bytes
                                                              : lay.bytes;

    // everything below touches the device
    c->expanded = true;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return fail(c, SIM_ERR_DEVICE, "no HIP device");
    if (c->device >= 0 && dev != c->device)
        return fail(c, SIM_ERR_DEVICE, "current HIP device differs from the context's device");
    c->device = dev;
    DevNet d{};
    d.m = m;
    d.n_fsrc = (int32_t)fsrc.size();
    d.ns = (int32_t)s_link.size();
    d.nflows = nflows;
    d.S = c->S;
    d.arb = c->arb;
    d.bmax = bmax;
    d.fifo_total = (int32_t)ftot;
    d.req_total = (int32_t)rtot;
    d.T = T;
    d.engine = engine;
    d.nl = nl;
    d.has_preds = any_preds ? 1 : 0;
    d.pd_omask = R.whole ? 0u : 0xFFFFFFFFu;
    {   // workgroup engine: the active sets (a bit and a list entry per source, a list
        // entry per link) in LDS unless the graph is too large for them or the full
        // scan is asked for; then 7 words per link, one per source, two per stream
        // in LDS too when they fit and every scenario's workgroup is resident at once
        // (else fewer resident workgroups hide less HBM latency than the LDS saves)
        const int64_t nsrc_all = (int64_t)m + (int64_t)s_link.size();
        const int64_t rcap = std::min<int64_t>(1024, nsrc_all * bmax);  // request list (8 B each)
        // spill list (4 B each): the chunks after the first of FIFO offers longer than one chunk
        int64_t scap = bmax > 4 ? std::min<int64_t>(512, (int64_t)m * ((bmax - 1) / 4)) : 0;
        if (const char *ev = std::getenv("SIMGPU_SPILL_CAP"))  // tests: a short spill list (later chunks inline)
            scap = std::max<int64_t>(0, std::min<int64_t>(scap, std::atoll(ev)));
        // (+ one word: the request list is 8-byte aligned)
        const int64_t act = 4 * ((nsrc_all + 31) / 32 + nsrc_all + (int64_t)m + 1) + 8 * rcap + 4 * scap;
        const int64_t room = kLds - 1024;  // room for the static LDS
        d.wg_act = (act <= room / 2 && !wg_scan) ? (int32_t)act : 0;
        d.wg_rcap = (int32_t)rcap;
        d.wg_scap = (int32_t)scap;
        const int64_t words = 7 * (int64_t)m + nsrc_all + 2 * (int64_t)s_link.size();
        const int64_t bytes = words * 4 + d.wg_act;
        const int64_t per_cu = bytes <= room ? room / bytes : 0;
        d.wg_lds = per_cu > 0 && (int64_t)c->S <= 256 * per_cu ? (int32_t)(words * 4) : 0;
    }
    d.b1_ns = (int32_t)s_link.size();
    d.b1_lpt = (nl + 1023) / 1024;
    d.b1_deliv_lds = b1_deliv_lds ? 1 : 0;
    d.o_word = 0;
    d.o_gnt = (int32_t)((int64_t)nl * 8);   // round-robin posts
    d.o_inl = (int32_t)((int64_t)nl * 16);
    d.o_b1ino = (int32_t)((int64_t)nl * 16 + align16((int64_t)m * 2));
    d.o_b1cnt = (int32_t)(c->arb == SIM_ARB_ROUND_ROBIN ? d.o_b1ino + align16((int64_t)nl * 2) : (int64_t)nl * 16);
    d.b1_ring_lg = 0;
    while ((1 << d.b1_ring_lg) < b1_ring) d.b1_ring_lg++;
    d.o_b1deliv = (int32_t)align16(b1_words);
    d.o_b1red = (int32_t)(b1_bytes - 64);
    d.lane_threads = ((nl + 63) / 64) * 64;
    if (const char *ev = std::getenv("SIMGPU_LANE_THREADS")) {
        const int v = std::atoi(ev);
        if (v >= d.lane_threads && v <= 1024 && v % 64 == 0) d.lane_threads = v;
    }
    d.bm = bm;
    d.lds_bytes = (int32_t)lds_bytes;
    d.o_path = (int32_t)lay.o_path;
    d.o_deliv = (int32_t)lay.o_deliv;
    d.o_reqcnt = (int32_t)lay.o_reqcnt;
    d.o_reqb = (int32_t)lay.o_reqb;
    d.o_req = (int32_t)lay.o_req;
    d.o_glist = (int32_t)lay.o_glist;
    d.o_grant = (int32_t)lay.o_grant;
    d.o_gdep = (int32_t)lay.o_gdep;
    d.o_red = (int32_t)lay.o_red;
    d.wv_G = wv.G;
    d.wv_W = wv.W;
    d.wv_nblk = wv.nblk;
    d.wv_wpb = wv.wpb;
    d.wv_nfs = wv.nfs;
    d.wv_lineup = wv.lineup ? 1 : 0;
    d.o_wword = (int32_t)wv.o_word;
    d.o_wred = (int32_t)wv.o_red;
    d.o_wdeliv = (int32_t)wv.o_deliv;
    d.o_wreq = (int32_t)wv.o_req;
    d.o_wgnt = (int32_t)wv.o_gnt;
    d.o_wgdep = (int32_t)wv.o_gdep;
    d.path_len = (int32_t)path_lane.size();
    d.path_in_lds = path_in_lds ? 1 : 0;
    d.req_slots = (int32_t)lr;
    // lane engines: rings of the traffic links only, in lane order
    if (engine != simgpu::kEngineWorkgroup && engine != simgpu::kEngineResident) d.fifo_total = (int32_t)lf;
    for (int i = 0; i < 24; i++) d.wr_off[i] = (int32_t)res.off[i];
    d.wr_rcap = (int32_t)res.rcap;
    d.wr_scap = (int32_t)res.scap;
    d.wr_ovf = res.ovf;
    d.wr_threads = res.threads;
    d.wr_nw = res.nw;
    d.wr_tcap = (int32_t)res.tcap;
    d.wr_tovf = res.tovf;
    sim_status st;
    auto &own = c->dev_static;
#define UP(vec, field)                                         \
    if ((st = upload(c, own, vec, &tmp_##field)) != SIM_OK) return st; \
    d.field = tmp_##field;
    int32_t *tmp_fsrc_link, *tmp_port_at_head, *tmp_nports_tail, *tmp_fifo_off, *tmp_fifo_mask, *tmp_req_off;
    int32_t *tmp_s_link, *tmp_s_rbeg, *tmp_s_rend, *tmp_r_path, *tmp_r_pd, *tmp_pd_flow, *tmp_path_link;
    uint32_t *tmp_r_start, *tmp_r_len, *tmp_pd_base;
    int32_t *tmp_bw, *tmp_lat, *tmp_cap;
    UP(fsrc, fsrc_link);
    UP(port_at_head, port_at_head);
    UP(nports_tail, nports_tail);
    UP(fifo_off, fifo_off);
    UP(fifo_mask, fifo_mask);
    UP(req_off, req_off);
    UP(s_link, s_link);
    UP(s_rbeg, s_rbeg);
    UP(s_rend, s_rend);
    UP(r_start, r_start);
    UP(r_len, r_len);
    UP(r_path, r_path);
    UP(r_pd, r_pd);
    UP(pd_flow, pd_flow);
    UP(pd_base, pd_base);
    UP(c->path_link, path_link);
    UP(c->bw, bw);
    UP(c->lat, lat);
    UP(c->cap, cap);
    if (credits) {
        int32_t *tmp_credit;
        UP(c->credit, credit);
    }
    if (engine == simgpu::kEngineWorkgroup || engine == simgpu::kEngineResident) {
        // streams to wake when a flow delivers: every flow that a range of the
        // stream waits on (flow-major CSR, each stream once per flow)
        std::vector<std::pair<int32_t, int32_t>> fs;
        for (size_t j = 0; j < s_link.size(); j++)
            for (int32_t r = s_rbeg[j]; r < s_rend[j]; r++)
                for (int32_t q = r_pd[r]; q < r_pd[r + 1]; q++) fs.emplace_back(pd_flow[q], (int32_t)j);
        std::sort(fs.begin(), fs.end());
        fs.erase(std::unique(fs.begin(), fs.end()), fs.end());
        std::vector<int32_t> fw_ptr(nflows + 1, 0), fw_str(fs.size());
        for (size_t q = 0; q < fs.size(); q++) {
            fw_ptr[fs[q].first + 1]++;
            fw_str[q] = fs[q].second;
        }
        for (int32_t f = 0; f < nflows; f++) fw_ptr[f + 1] += fw_ptr[f];
        if (fw_str.empty()) fw_str.push_back(0);
        int32_t *tmp_fw_ptr, *tmp_fw_str;
        UP(fw_ptr, fw_ptr);
        UP(fw_str, fw_str);
    }
    if (engine == simgpu::kEngineResident) {
        // descriptor spans shared by consecutive ranges of a stream whose
        // descriptors are equal
        std::vector<char> first(r_start.size() + 1, 0);
        for (int32_t b0 : s_rbeg) first[b0] = 1;
        std::vector<int32_t> rpb(r_start.size() + 1, 0), rpe(r_start.size() + 1, 0), pdf;
        std::vector<uint32_t> pdb;
        for (size_t j = 0; j < r_start.size(); j++) {
            const int32_t a1 = r_pd[j], b1 = r_pd[j + 1];
            bool same = j > 0 && !first[j] && a1 - r_pd[j - 1] == b1 - a1;
            for (int32_t q = 0; same && q < b1 - a1; q++)
                same = pd_flow[r_pd[j - 1] + q] == pd_flow[a1 + q] && pd_base[r_pd[j - 1] + q] == pd_base[a1 + q];
            if (same) {
                rpb[j] = rpb[j - 1];
                rpe[j] = rpe[j - 1];
                continue;
            }
            rpb[j] = (int32_t)pdf.size();
            for (int32_t q = a1; q < b1; q++) {
                pdf.push_back(pd_flow[q]);
                pdb.push_back(pd_base[q]);
            }
            rpe[j] = (int32_t)pdf.size();
        }
        if (pdf.empty()) {
            pdf.push_back(0);
            pdb.push_back(0);
        }
        int32_t *tmp_wr_rpb, *tmp_wr_rpe, *tmp_wr_pdf;
        uint32_t *tmp_wr_pdb;
        UP(rpb, wr_rpb);
        UP(rpe, wr_rpe);
        UP(pdf, wr_pdf);
        UP(pdb, wr_pdb);
    }
    if (fair && !R.cls.empty()) {
        uint8_t *tmp_line_cls;
        UP(R.cls, line_cls);
    }
    int32_t *tmp_ln_P, *tmp_ln_port, *tmp_ln_fifo, *tmp_ln_mask, *tmp_ln_req, *tmp_ln_reqcap, *tmp_ln_srbeg,
        *tmp_ln_srend, *tmp_link_lane, *tmp_path_lane;
    UP(ln_P, ln_P);
    UP(ln_port, ln_port);
    UP(ln_fifo, ln_fifo);
    UP(ln_mask, ln_mask);
    UP(ln_req, ln_req);
    UP(ln_reqcap, ln_reqcap);
    UP(ln_srbeg, ln_srbeg);
    UP(ln_srend, ln_srend);
    UP(link_lane, link_lane);
    UP(path_lane, path_lane);
    int32_t *tmp_ln_link, *tmp_in_lane, *tmp_ln_inoff;
    UP(lane_link, ln_link);
    UP(in_lane, in_lane);
    UP(ln_inoff, ln_inoff);
    if (engine == simgpu::kEngineGrid) {
        // the layout was made in fsrc order; lanes are in lane_link order
        // (the same order for this engine), and paths are re-expressed in the
        // tail workgroups' local target indices
        std::vector<int32_t> gpath(path_lane.size());
        // a sink entry names the delivered counter of its flow in the
        // destination's workgroup (the last one if nothing waits on the flow)
        for (size_t q = 0; q < path_lane.size(); q++) {
            const int32_t v = path_lane[q];
            gpath[q] = v >= 0 ? gl.tloc[v] : -1 - (gl.floc[-v - 1] >= 0 ? gl.floc[-v - 1] : gl.fl_max);
        }
        d.gd_nb = gl.nb;
        d.gd_stride = 8;  // blocks w * 8: one die's CUs when blocks go round-robin over the 8 dies
        if (const char *ev = std::getenv("SIMGPU_GRID_STRIDE")) {  // tests: workgroups spread over the dies
            const int v = std::atoi(ev);
            if (v >= 1 && v <= 8) d.gd_stride = v;
        }
        d.gd_threads = gl.threads;
        d.gd_ns_max = gl.ns_max;
        d.gd_nt_max = gl.nt_max;
        d.gd_req_max = gl.req_max;
        d.gd_fl_max = gl.fl_max;
        d.gd_one = gl.one ? 1 : 0;
        d.gd_inl_max = gl.inl_max;
        d.gd_window = gl.window;
        d.gd_sring_max = gl.sring_max;
        d.gd_cring_max = gl.cring_max;
        int32_t *tmp_gd_sptr, *tmp_gd_slane, *tmp_gd_tptr, *tmp_gd_tlane, *tmp_gd_rqoff, *tmp_gd_path, *tmp_gd_floc,
            *tmp_gd_fptr, *tmp_gd_fown;
        UP(gl.sptr, gd_sptr);
        UP(gl.slane, gd_slane);
        UP(gl.tptr, gd_tptr);
        UP(gl.tlane, gd_tlane);
        UP(gl.rqoff, gd_rqoff);
        UP(gpath, gd_path);
        UP(gl.floc, gd_floc);
        UP(gl.fptr, gd_fptr);
        UP(gl.fown, gd_fown);
        if (gl.one) {
            int32_t *tmp_gd_toff, *tmp_gd_iptr, *tmp_gd_inl;
            UP(gl.toff, gd_toff);
            UP(gl.iptr, gd_iptr);
            UP(gl.inl, gd_inl);
        }
        if (gl.window > 0) {
            int32_t *tmp_gd_sro, *tmp_gd_tro;
            UP(gl.sro, gd_sro);
            UP(gl.tro, gd_tro);
        }
    }
    if (engine == simgpu::kEngineWave) {
        uint32_t *tmp_wv_lfb, *tmp_wv_lfx, *tmp_wv_duo;
        if (wv_duo.empty()) wv_duo.push_back(0);
        UP(wv_duo, wv_duo);
        int32_t *tmp_wv_feed, *tmp_wv_nfeed, *tmp_wv_sc, *tmp_r_lf, *tmp_pd_dix;
        UP(wv_lfb, wv_lfb);
        UP(wv_lfx, wv_lfx);
        UP(pd_dix, pd_dix);
        UP(wv_feed, wv_feed);
        UP(wv_nfeed, wv_nfeed);
        UP(wv_sc, wv_sc);
        int32_t *tmp_blk_wave, *tmp_blk_off;
        UP(blk_wave, blk_wave);
        UP(blk_off, blk_off);
        UP(r_lf, r_lf);
    }
#undef UP
    const size_t S = (size_t)c->S;
    const size_t nsrc = (size_t)m + (size_t)d.ns;
    StateLayout &sl = c->state;
    sl = StateLayout{};
    sl.add(&DevNet::status, S);
    sl.add(&DevNet::cycles, S);
    if (engine == simgpu::kEngineLaneHbm || engine == simgpu::kEngineGrid) sl.add(&DevNet::gfifo, S * (size_t)lf);
    if (engine == simgpu::kEngineGrid) {
        sl.add(&DevNet::gd_pub, 4 * (size_t)nl);
        if (gl.one) sl.add(&DevNet::gd_tpub, 4 * (size_t)nl);
        sl.add(&DevNet::gd_dslot, 2 * (size_t)nflows);
        sl.add(&DevNet::gd_sync, 16);
    }
    if (engine == simgpu::kEngineB1) {  // uniform rings: lane i owns entries [i << lg, (i + 1) << lg)
        d.fifo_total = nl << d.b1_ring_lg;
        sl.add(&DevNet::gfifo, S * (size_t)d.fifo_total);
    }
    if (engine == simgpu::kEngineResident) {
        sl.add(&DevNet::wr_frec, S * ftot);
        sl.add(&DevNet::delivered, S * nflows);
        if (res.ovf > 0) {
            const size_t ov = S * (size_t)res.ovf;
            sl.add(&DevNet::wr_ox, ov);
            sl.add(&DevNet::wr_opp, ov);
            sl.add(&DevNet::wr_okey, ov);
            sl.add(&DevNet::wr_ots, ov);
            sl.add(&DevNet::wr_osidx, ov);
            sl.add(&DevNet::wr_ogl, ov);
            sl.add(&DevNet::wr_osrc, ov);
            sl.add(&DevNet::wr_og, ov);
            sl.add(&DevNet::wr_osrcid, ov);
            if (fair) sl.add(&DevNet::wr_oaux, ov);
        }
        if (res.tovf > 0) {
            const size_t tv = S * (size_t)res.tovf;
            sl.add(&DevNet::wr_otmask, tv);
            sl.add(&DevNet::wr_otseg, tv);
            sl.add(&DevNet::wr_otq, tv);
        }
    }
    if (engine == simgpu::kEngineWorkgroup) {
        sl.add(&DevNet::fifo_x, S * ftot);
        sl.add(&DevNet::fifo_rdy, S * ftot);
        sl.add(&DevNet::fifo_pp, S * ftot);
        sl.add(&DevNet::qhead, S * m);
        sl.add(&DevNet::qcred, S * m);
        sl.add(&DevNet::cptr, S * m);
        if (fair) sl.add(&DevNet::req_aux, S * rtot);
        sl.add(&DevNet::qtail, S * m);
        sl.add(&DevNet::rr, S * m);
        sl.add(&DevNet::cur_rng, S * d.ns);
        sl.add(&DevNet::cur_off, S * d.ns);
        sl.add(&DevNet::delivered, S * nflows);
        sl.add(&DevNet::req_cnt, S * m);
        sl.add(&DevNet::req_rec, S * rtot);
        sl.add(&DevNet::sreq_x, S * nsrc * bmax);
        sl.add(&DevNet::sreq_pp, S * nsrc * bmax);
        sl.add(&DevNet::sreq_n, S * nsrc);
        sl.add(&DevNet::grant, S * nsrc * bmax);
        sl.add(&DevNet::gcount, S * m);
        sl.add(&DevNet::glist, S * m * bmax);
        sl.add(&DevNet::gdep, S * m * bmax);
    }
    unsigned char *block = nullptr;
    if ((st = alloc(c, c->dev_state, sl.bytes, &block))) return st;
    sl.apply(d, block);
    c->dn = d;
    c->loaded = true;
    c->ran = false;
    return SIM_OK;
}

}  // namespace

namespace {

// Entry points; their extern "C" wrappers follow.

sim_status create_impl(int32_t n_nodes, int32_t n_endpoints, const int32_t *row_ptr, const int32_t *col_idx,
                      int32_t n_scenarios, const int32_t *bw, const int32_t *lat, const int32_t *cap,
                      int32_t arb, sim_ctx **out) {
    if (!out || !row_ptr || !col_idx || !bw || !lat || !cap) return SIM_ERR_INVALID_ARG;
    *out = nullptr;
    if (n_nodes < 1 || n_endpoints < 1 || n_endpoints > n_nodes || n_scenarios < 1) return SIM_ERR_INVALID_ARG;
    if (arb < 0 || arb > (SIM_ARB_ROUND_ROBIN | SIM_ARB_FAIR_CLASSES)) return SIM_ERR_INVALID_ARG;
    if (n_endpoints > 65536) return SIM_ERR_INVALID_ARG;  // (src << 16 | dst) hash key
    if (row_ptr[0] != 0) return SIM_ERR_TOPOLOGY;
    for (int32_t v = 0; v < n_nodes; v++)
        if (row_ptr[v + 1] < row_ptr[v]) return SIM_ERR_TOPOLOGY;
    const int32_t m = row_ptr[n_nodes];
    for (int32_t v = 0; v < n_nodes; v++)
        for (int32_t l = row_ptr[v]; l < row_ptr[v + 1]; l++)
            if (col_idx[l] < 0 || col_idx[l] >= n_nodes || col_idx[l] == v) return SIM_ERR_TOPOLOGY;
    const size_t pm = (size_t)n_scenarios * (size_t)m;
    for (size_t i = 0; i < pm; i++)
        if (bw[i] < 1 || bw[i] > SIM_MAX_BW || lat[i] < 1 || lat[i] > SIM_MAX_LAT || cap[i] < 1 ||
            cap[i] > SIM_MAX_CAP)
            return SIM_ERR_TOPOLOGY;
    sim_ctx *c = new (std::nothrow) sim_ctx();
    if (!c) return SIM_ERR_OOM;
    c->device = -1;  // bound to the current HIP device by the first load
    c->n = n_nodes;
    c->E = n_endpoints;
    c->m = m;
    c->S = n_scenarios;
    c->arb = arb;
    c->row_ptr.assign(row_ptr, row_ptr + n_nodes + 1);
    c->col_idx.assign(col_idx, col_idx + m);
    c->tail.resize(m);
    for (int32_t v = 0; v < n_nodes; v++)
        for (int32_t l = row_ptr[v]; l < row_ptr[v + 1]; l++) c->tail[l] = v;
    c->bw.assign(bw, bw + pm);
    c->lat.assign(lat, lat + pm);
    c->cap.assign(cap, cap + pm);
    build_in_links(c);
    *out = c;
    return SIM_OK;
}

sim_status load_collective_impl(sim_ctx *c, int32_t coll, uint64_t bytes, int32_t group_size, const int32_t *order,
                               int32_t dep) {
    if (!c) return SIM_ERR_INVALID_ARG;
    if (coll != SIM_COLL_HIER_ALLREDUCE && group_size != 0)
        return fail(c, SIM_ERR_INVALID_ARG, "group_size applies to the hierarchical all-reduce only");
    Ranges R;
    sim_status st = expand_collective(c, coll, bytes, group_size, order, dep, R);
    if (st != SIM_OK) return st;
    return finish_load(c, R);
}

sim_status load_transactions_impl(sim_ctx *c, int64_t n, const int32_t *src, const int32_t *dst,
                                 const int64_t *pred_ptr, const int64_t *pred_idx) {
    if (!c || n < 0 || (n > 0 && (!src || !dst || !pred_ptr))) return SIM_ERR_INVALID_ARG;
    if (n >= (int64_t)0xFFFFFFFFll) return fail(c, SIM_ERR_SIZE, "more than 2^32-2 transactions");
    if (n > 0 && pred_ptr[0] != 0) return fail(c, SIM_ERR_INVALID_ARG, "pred_ptr[0] must be 0");
    Ranges R;
    for (int64_t x = 0; x < n; x++) {
        if (src[x] < 0 || src[x] >= c->E || dst[x] < 0 || dst[x] >= c->E || src[x] == dst[x])
            return fail(c, SIM_ERR_INVALID_ARG, "transaction " + std::to_string(x) + ": bad endpoints");
        if (pred_ptr[x + 1] < pred_ptr[x]) return fail(c, SIM_ERR_INVALID_ARG, "pred_ptr not monotone");
        R.add((uint64_t)x, 1, src[x], dst[x]);
        for (int64_t q = pred_ptr[x]; q < pred_ptr[x + 1]; q++) {
            if (!pred_idx || pred_idx[q] < 0 || pred_idx[q] >= n)
                return fail(c, SIM_ERR_INVALID_ARG, "predecessor out of range");
            R.pred(pred_idx[q], 0);
        }
    }
    R.close();
    return finish_load(c, R);
}

// GPU programs (copies with one or more sources, releases, acquires) turned
// into lines; the rules are those of sim_load_gpu_ops.
sim_status load_gpu_ops_impl(sim_ctx *c, int64_t n_ops, const int32_t *kind, const int32_t *cu,
                             const int64_t *src_ptr, const int32_t *src_space, const int64_t *src_line,
                             const int32_t *dst_space, const int64_t *dst_line, const int64_t *n_lines,
                             int32_t n_spaces, int32_t n_ch, const int32_t *space_ch, int32_t unroll,
                             int32_t window) {
    if (!c || n_ops < 0 || n_spaces < 1 || n_ch < 1 || !space_ch || unroll < 1 || window < 1 || !src_ptr ||
        (n_ops > 0 && (!kind || !cu || !dst_space || !dst_line || !n_lines)))
        return c ? fail(c, SIM_ERR_INVALID_ARG, "gpu ops: null array or bad n_spaces/n_ch/unroll/window")
                 : SIM_ERR_INVALID_ARG;
    if (src_ptr[0] != 0) return fail(c, SIM_ERR_INVALID_ARG, "gpu ops: src_ptr[0] must be 0");
    if (n_ops > 0 && src_ptr[n_ops] > 0 && (!src_space || !src_line))
        return fail(c, SIM_ERR_INVALID_ARG, "gpu ops: null source arrays");
    for (int64_t q = 0; q < (int64_t)n_spaces * n_ch; q++)
        if (space_ch[q] < 0 || space_ch[q] >= c->E) return fail(c, SIM_ERR_INVALID_ARG, "gpu ops: channel is not an endpoint");
    enum : uint8_t { kLoad, kStore, kRelease, kAcquire };
    // One wavefront request of a CU's program.  A store waits for the data of
    // loads [g0, g0 + gn) of the same program; a release or acquire names its
    // semaphore by its index in `sems`.
    struct Req {
        uint8_t what;
        int32_t chan;
        int64_t g0;
        int64_t gn;
    };
    auto two = [](const Req &r) { return r.what == kLoad || r.what == kAcquire; };
    std::map<std::pair<int32_t, int64_t>, std::pair<int32_t, int64_t>> rel_at;  // semaphore -> (CU, index)
    std::map<int32_t, std::vector<Req>> prog;                                     // by CU, ascending
    std::vector<std::pair<int32_t, int64_t>> sems;                                // acquires' semaphores
    uint64_t lines = 0;
    auto chan_of = [&](int32_t s, int64_t a) { return space_ch[(int64_t)s * n_ch + a % n_ch]; };
    for (int64_t o = 0; o < n_ops; o++) {
        const std::string where = "gpu ops: operation " + std::to_string(o);
        const int64_t K = src_ptr[o + 1] - src_ptr[o];
        if (cu[o] < 0 || cu[o] >= c->E) return fail(c, SIM_ERR_INVALID_ARG, where + ": CU is not an endpoint");
        if (K < 0 || dst_space[o] < 0 || dst_space[o] >= n_spaces || dst_line[o] < 0 || n_lines[o] < 0)
            return fail(c, SIM_ERR_INVALID_ARG, where + " out of range");
        auto &pr = prog[cu[o]];
        const int64_t first = (int64_t)pr.size();
        if (kind[o] == SIM_OP_RELEASE || kind[o] == SIM_OP_ACQUIRE) {
            if (K != 0 || n_lines[o] != 1)
                return fail(c, SIM_ERR_INVALID_ARG, where + ": a release or acquire has no source and one line");
            const auto sem = std::make_pair(dst_space[o], dst_line[o]);
            if (kind[o] == SIM_OP_RELEASE) {
                if (!rel_at.emplace(sem, std::make_pair(cu[o], first)).second)
                    return fail(c, SIM_ERR_INVALID_ARG, where + ": semaphore released twice");
                pr.push_back({kRelease, chan_of(sem.first, sem.second), -1, 0});
                lines += 1;
            } else {
                pr.push_back({kAcquire, chan_of(sem.first, sem.second), (int64_t)sems.size(), 0});
                sems.push_back(sem);
                lines += 2;
            }
        } else if (kind[o] == SIM_OP_COPY) {
            if (K < 1) return fail(c, SIM_ERR_INVALID_ARG, where + ": a copy needs a source");
            for (int64_t s = src_ptr[o]; s < src_ptr[o + 1]; s++)
                if (src_space[s] < 0 || src_space[s] >= n_spaces || src_line[s] < 0)
                    return fail(c, SIM_ERR_INVALID_ARG, where + ": source out of range");
            lines += (uint64_t)(2 * K + 1) * (uint64_t)n_lines[o];
            if (lines >= 0xFFFFFFFFull) return fail(c, SIM_ERR_SIZE, "more than 2^32-2 transactions");
            for (int64_t j0 = 0; j0 < n_lines[o]; j0 += unroll) {
                const int64_t gn = std::min<int64_t>(unroll, n_lines[o] - j0);
                const int64_t g0 = (int64_t)pr.size();
                for (int64_t s = src_ptr[o]; s < src_ptr[o + 1]; s++)
                    for (int64_t u = 0; u < gn; u++) pr.push_back({kLoad, chan_of(src_space[s], src_line[s] + j0 + u), 0, 0});
                const int64_t nl = (int64_t)pr.size() - g0;
                for (int64_t u = 0; u < gn; u++) pr.push_back({kStore, chan_of(dst_space[o], dst_line[o] + j0 + u), g0, nl});
            }
        } else {
            return fail(c, SIM_ERR_INVALID_ARG, where + ": unknown kind " + std::to_string(kind[o]));
        }
        if (lines >= 0xFFFFFFFFull) return fail(c, SIM_ERR_SIZE, "more than 2^32-2 transactions");
        for (int64_t q = first; q < (int64_t)pr.size(); q++)
            if (pr[q].chan == cu[o]) return fail(c, SIM_ERR_INVALID_ARG, where + ": a CU is the channel of its own line");
    }
    for (const auto &s : sems)
        if (!rel_at.count(s))
            return fail(c, SIM_ERR_INVALID_ARG, "gpu ops: acquire of semaphore (" + std::to_string(s.first) + ", " +
                                                    std::to_string(s.second) + ") that nothing releases");
    // ids, step-major over the CUs
    std::vector<std::pair<int32_t, std::vector<Req> *>> cus;
    std::map<int32_t, size_t> cu_row;
    for (auto &kv : prog) {
        cu_row[kv.first] = cus.size();
        cus.push_back({kv.first, &kv.second});
    }
    std::vector<std::vector<int64_t>> id(cus.size());
    size_t kmax = 0;
    for (size_t q = 0; q < cus.size(); q++) {
        id[q].resize(cus[q].second->size());
        kmax = std::max(kmax, cus[q].second->size());
    }
    int64_t T = 0;
    for (size_t k = 0; k < kmax; k++)
        for (size_t q = 0; q < cus.size(); q++)
            if (k < cus[q].second->size()) {
                id[q][k] = T;
                T += two((*cus[q].second)[k]) ? 2 : 1;
            }
    auto done = [&](size_t q, size_t k) { return id[q][k] + (two((*cus[q].second)[k]) ? 1 : 0); };
    // Per CU: the latest store or release per channel since the CU's last
    // release.  Lines of one (CU, channel) pair share a path, so they complete
    // in id order and the latest one stands for all of them.
    std::vector<std::map<int32_t, int64_t>> pending(cus.size());
    Ranges R;
    int64_t next = 0;
    for (size_t k = 0; k < kmax; k++)
        for (size_t q = 0; q < cus.size(); q++) {
            const auto &pr = *cus[q].second;
            if (k >= pr.size()) continue;
            const Req &r = pr[k];
            const int64_t x = id[q][k];
            if (x != next) return fail(c, SIM_ERR_INVALID_ARG, "internal: gpu op ids not dense");
            R.add((uint64_t)x, 1, cus[q].first, r.chan, (int64_t)k, 0);
            if (k >= (size_t)window) R.pred(done(q, k - (size_t)window), 0);  // retired before this one issues
            if (k >= 1 && pr[k - 1].what == kAcquire && window != 1) R.pred(done(q, k - 1), 0);
            if (r.what == kStore)
                for (int64_t g = r.g0; g < r.g0 + r.gn; g++) R.pred(id[q][g] + 1, 0);
            if (r.what == kRelease) {
                for (const auto &kv : pending[q]) R.pred(kv.second, 0);
                pending[q].clear();
            }
            if (r.what == kStore || r.what == kRelease) pending[q][r.chan] = x;
            if (r.what == kAcquire) {
                const auto &at = rel_at[sems[(size_t)r.g0]];
                R.pred(id[cu_row[at.first]][(size_t)at.second], 0);
            }
            R.cls.push_back(r.what == kStore ? 0 : 1);
            next = x + 1;
            if (two(r)) {  // the data line or reply
                R.add((uint64_t)x + 1, 1, r.chan, cus[q].first, (int64_t)k, 1);
                R.pred(x, 0);
                R.cls.push_back(r.what == kLoad ? 0 : 1);
                next = x + 2;
            }
        }
    R.close();
    return finish_load(c, R);
}

sim_status load_memcpy_impl(sim_ctx *c, int64_t n_ops, const int32_t *cu, const int32_t *src_space,
                           const int32_t *dst_space, const int64_t *src_line, const int64_t *dst_line,
                           const int64_t *n_lines, int32_t n_spaces, int32_t n_ch, const int32_t *space_ch,
                           int32_t unroll, int32_t window) {
    if (!c || n_ops < 0 || (n_ops > 0 && (!src_space || !src_line)))
        return c ? fail(c, SIM_ERR_INVALID_ARG, "memcpy: null array or negative n_ops") : SIM_ERR_INVALID_ARG;
    std::vector<int32_t> kinds((size_t)n_ops, SIM_OP_COPY);
    std::vector<int64_t> sp((size_t)n_ops + 1);
    for (int64_t o = 0; o <= n_ops; o++) sp[(size_t)o] = o;
    return load_gpu_ops_impl(c, n_ops, kinds.data(), cu, sp.data(), src_space, src_line, dst_space, dst_line,
                             n_lines, n_spaces, n_ch, space_ch, unroll, window);
}


// scratch == nullptr: the engines' scratch is the context's block; else the
// caller's scratch_bytes at scratch (nothing is allocated either way)
sim_status run_impl(sim_ctx *c, void *stream, uint32_t *d_completion, uint64_t *d_tx_lines,
                   uint64_t *d_busy_cycles, uint32_t *d_makespan, uint64_t max_cycles,
                   unsigned char *scratch = nullptr, size_t scratch_bytes = 0) {
    if (!c) return SIM_ERR_INVALID_ARG;
    if (!c->loaded) return fail(c, SIM_ERR_STATE, "sim_run before a workload was loaded");
    if ((!d_completion && c->T > 0) || !d_tx_lines || !d_busy_cycles || !d_makespan)
        return fail(c, SIM_ERR_INVALID_ARG, "null output buffer");
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev != c->device)
        return fail(c, SIM_ERR_DEVICE, "current HIP device differs from the context's device");
    DevNet d = c->dn;
    if (scratch) {
        if (c->state.bytes > scratch_bytes)
            return fail(c, SIM_ERR_SIZE, "the loaded workload needs " + std::to_string(c->state.bytes) +
                                             " B of engine scratch, more than the " + std::to_string(scratch_bytes) +
                                             " B of the allocation-free run");
        c->state.apply(d, scratch);
    }
    d.completion = d_completion;
    d.tx_lines = d_tx_lines;
    d.busy = d_busy_cycles;
    d.makespan = d_makespan;
    d.max_cycles = (max_cycles == 0 || max_cycles > simgpu::kCycleLimit) ? simgpu::kCycleLimit : max_cycles;
    // Between two departing cycles at most fifo_total event jumps can happen
    // (each lands on a distinct FIFO-head ready time); departing cycles are at
    // most line_hops + T.
    d.watchdog = (c->line_hops + (uint64_t)c->T + 1) * ((uint64_t)d.fifo_total + 2) + 1000000ull;
    int e = simgpu::launch_engine(d, stream);
    if (e != 0) return fail(c, SIM_ERR_DEVICE, std::string("kernel launch failed: ") + hipGetErrorString((hipError_t)e));
    c->run_status = d.status;
    c->run_cycles = d.cycles;
    c->ran = true;
    return SIM_OK;
}

sim_status status_after_sync_impl(sim_ctx *c, int32_t *status, uint64_t *cycles) {
    if (!c) return SIM_ERR_INVALID_ARG;
    if (!c->loaded || !c->ran) return fail(c, SIM_ERR_STATE, "no run to report on");
    std::vector<int32_t> st(c->S);
    if (hipMemcpy(st.data(), c->run_status, sizeof(int32_t) * c->S, hipMemcpyDeviceToHost) != hipSuccess)
        return fail(c, SIM_ERR_DEVICE, "hipMemcpy of status failed");
    if (status) std::memcpy(status, st.data(), sizeof(int32_t) * c->S);
    if (cycles &&
        hipMemcpy(cycles, c->run_cycles, sizeof(uint64_t) * c->S, hipMemcpyDeviceToHost) != hipSuccess)
        return fail(c, SIM_ERR_DEVICE, "hipMemcpy of cycles failed");
    for (int32_t s = 0; s < c->S; s++) {
        if (st[s] == simgpu::kRunDeadlock) return fail(c, SIM_ERR_DEADLOCK, "scenario " + std::to_string(s) + " deadlocked");
        if (st[s] == simgpu::kRunMaxCycles)
            return fail(c, SIM_ERR_MAX_CYCLES, "scenario " + std::to_string(s) + " exceeded max_cycles");
        if (st[s] == simgpu::kRunInternal)
            return fail(c, SIM_ERR_DEVICE, "scenario " + std::to_string(s) + ": internal engine error (request slot overflow or line id out of range)");
        if (st[s] == simgpu::kRunWatchdog)
            return fail(c, SIM_ERR_DEVICE, "scenario " + std::to_string(s) + ": engine watchdog fired");
        if (st[s] != simgpu::kRunOk) return fail(c, SIM_ERR_DEVICE, "scenario " + std::to_string(s) + " did not finish");
    }
    return SIM_OK;
}

sim_status txn_info_impl(const sim_ctx *c, int64_t id, int32_t *src, int32_t *dst, int32_t *step, int32_t *line) {
    if (!c) return SIM_ERR_INVALID_ARG;
    if (!c->expanded) return SIM_ERR_STATE;
    if (id < 0 || id >= c->T) return SIM_ERR_INVALID_ARG;
    // the range holding id: the last one whose first id is <= id
    const size_t r = (size_t)(std::upper_bound(c->h_start.begin(), c->h_start.end(), (uint32_t)id) - c->h_start.begin()) - 1;
    if (src) *src = c->h_src[r];
    if (dst) *dst = c->h_dst[r];
    if (step) *step = c->h_step[r];
    if (line) *line = c->h_step[r] < 0 ? 0 : (int32_t)(c->h_moff[r] + ((uint32_t)id - c->h_start[r]));
    return SIM_OK;
}

sim_status route_impl(const sim_ctx *c, int32_t src, int32_t dst, int32_t *links, int32_t cap, int32_t *len) {
    if (!c || !len || src < 0 || dst < 0 || src >= c->E || dst >= c->E) return SIM_ERR_INVALID_ARG;
    std::vector<int32_t> hops;
    if (src == dst) {
        *len = 0;
        return SIM_OK;
    }
    if (!trace_route(c, src, dst, hops)) return SIM_ERR_UNREACHABLE;
    *len = (int32_t)hops.size();
    if ((int32_t)hops.size() > cap || (!links && !hops.empty())) return SIM_ERR_SIZE;
    std::copy(hops.begin(), hops.end(), links);
    return SIM_OK;
}



sim_status set_credit_impl(sim_ctx *c, const int32_t *credit) {
    if (!c) return SIM_ERR_INVALID_ARG;
    const size_t pm = (size_t)c->S * (size_t)c->m;
    bool any = false;
    for (size_t i = 0; credit && i < pm; i++) {
        if (credit[i] < 1 || credit[i] > SIM_MAX_LAT) return fail(c, SIM_ERR_INVALID_ARG, "credit delay out of range");
        any |= credit[i] > 1;
    }
    if (any) c->credit.assign(credit, credit + pm);
    else c->credit.clear();
    // the engine and its tables depend on the delays: the workload is loaded again
    free_list(c->dev_static);
    free_list(c->dev_state);
    c->loaded = false;
    c->expanded = false;
    c->ran = false;
    return SIM_OK;
}

}  // namespace

// No C++ exception crosses the C ABI: allocation failures become
// SIM_ERR_OOM, anything else SIM_ERR_DEVICE.
template <typename F>
sim_status guarded(sim_ctx *c, F &&f) {
    try {
        return f();
    } catch (const std::bad_alloc &) {
        if (c) c->err = "host allocation failed";
        return SIM_ERR_OOM;
    } catch (...) {
        if (c) c->err = "unexpected host error";
        return SIM_ERR_DEVICE;
    }
}

namespace simgpu {
// The allocation-free run (noalloc.hip): sim_run with the engines' scratch at
// the caller's device address.
sim_status run_on_scratch(sim_ctx *c, void *stream, uint32_t *d_completion, uint64_t *d_tx_lines,
                          uint64_t *d_busy_cycles, uint32_t *d_makespan, uint64_t max_cycles, void *scratch,
                          size_t scratch_bytes) {
    if (!scratch) return SIM_ERR_INVALID_ARG;
    return guarded(c, [&] {
        return run_impl(c, stream, d_completion, d_tx_lines, d_busy_cycles, d_makespan, max_cycles,
                        static_cast<unsigned char *>(scratch), scratch_bytes);
    });
}
}  // namespace simgpu

extern "C" {

sim_status sim_create(int32_t n_nodes, int32_t n_endpoints, const int32_t *row_ptr, const int32_t *col_idx,
                      int32_t n_scenarios, const int32_t *bw, const int32_t *lat, const int32_t *cap,
                      int32_t arb, sim_ctx **out) {
    return guarded(nullptr, [&] { return create_impl(n_nodes, n_endpoints, row_ptr, col_idx, n_scenarios, bw, lat, cap, arb, out); });
}

sim_status sim_set_credit(sim_ctx *c, const int32_t *credit) {
    return guarded(c, [&] { return set_credit_impl(c, credit); });
}

sim_status sim_load_collective(sim_ctx *c, int32_t coll, uint64_t bytes, int32_t group_size, const int32_t *order,
                               int32_t dep) {
    return guarded(c, [&] { return load_collective_impl(c, coll, bytes, group_size, order, dep); });
}

sim_status sim_load_transactions(sim_ctx *c, int64_t n, const int32_t *src, const int32_t *dst,
                                 const int64_t *pred_ptr, const int64_t *pred_idx) {
    return guarded(c, [&] { return load_transactions_impl(c, n, src, dst, pred_ptr, pred_idx); });
}

sim_status sim_load_memcpy(sim_ctx *c, int64_t n_ops, const int32_t *cu, const int32_t *src_space,
                           const int32_t *dst_space, const int64_t *src_line, const int64_t *dst_line,
                           const int64_t *n_lines, int32_t n_spaces, int32_t n_ch, const int32_t *space_ch,
                           int32_t unroll, int32_t window) {
    return guarded(c, [&] { return load_memcpy_impl(c, n_ops, cu, src_space, dst_space, src_line, dst_line, n_lines, n_spaces, n_ch, space_ch, unroll, window); });
}

sim_status sim_load_gpu_ops(sim_ctx *c, int64_t n_ops, const int32_t *kind, const int32_t *cu,
                            const int64_t *src_ptr, const int32_t *src_space, const int64_t *src_line,
                            const int32_t *dst_space, const int64_t *dst_line, const int64_t *n_lines,
                            int32_t n_spaces, int32_t n_ch, const int32_t *space_ch, int32_t unroll, int32_t window) {
    return guarded(c, [&] { return load_gpu_ops_impl(c, n_ops, kind, cu, src_ptr, src_space, src_line, dst_space, dst_line, n_lines, n_spaces, n_ch, space_ch, unroll, window); });
}

sim_status sim_run(sim_ctx *c, void *stream, uint32_t *d_completion, uint64_t *d_tx_lines,
                   uint64_t *d_busy_cycles, uint32_t *d_makespan, uint64_t max_cycles) {
    return guarded(c, [&] { return run_impl(c, stream, d_completion, d_tx_lines, d_busy_cycles, d_makespan, max_cycles); });
}

sim_status sim_status_after_sync(sim_ctx *c, int32_t *status, uint64_t *cycles) {
    return guarded(c, [&] { return status_after_sync_impl(c, status, cycles); });
}

sim_status sim_route(const sim_ctx *c, int32_t src, int32_t dst, int32_t *links, int32_t cap, int32_t *len) {
    return guarded(const_cast<sim_ctx *>(c), [&] { return route_impl(c, src, dst, links, cap, len); });
}

sim_status sim_txn_info(const sim_ctx *c, int64_t id, int32_t *src, int32_t *dst, int32_t *phase_step, int32_t *line) {
    return guarded(const_cast<sim_ctx *>(c), [&] { return txn_info_impl(c, id, src, dst, phase_step, line); });
}

sim_status sim_sizes(const sim_ctx *c, int64_t *n_txn, int32_t *n_links, int32_t *n_scenarios, uint64_t *line_hops) {
    if (!c) return SIM_ERR_INVALID_ARG;
    if (n_links) *n_links = c->m;
    if (n_scenarios) *n_scenarios = c->S;
    if (!c->loaded) return SIM_ERR_STATE;
    if (n_txn) *n_txn = c->T;
    if (line_hops) *line_hops = c->line_hops;
    return SIM_OK;
}

const char *sim_last_error(const sim_ctx *c) { return c ? c->err.c_str() : "null context"; }

void sim_destroy(sim_ctx *c) {
    if (!c) return;
    free_list(c->dev_static);
    free_list(c->dev_state);
    delete c;
}

}  // extern "C"
