/*
 * simgpu -- line-granularity network simulation on one MI355X (gfx950).
 *
 * C ABI of libsimgpu.so.  Every call returns a sim_status; no C++ exception
 * crosses this boundary.  Plain pointers and sizes only.
 *
 * What is simulated.  The paper ("ASTRA-sim 3.0") makes the cache-line-sized
 * wavefront request the unit that the network backend simulates (Sec. 4.4.3,
 * "Wavefront Request") and extends the Simple network backend to a graph of
 * endpoints, switches and links with a modular routing function (Sec. 4.5);
 * the Simple backend itself is an alpha-beta model (Sec. 2.1).  This library
 * advances every 128 B line of a collective hop by hop through such a graph.
 * The paper does not state the queueing discipline; the model implemented
 * here is:
 *   - link l = bounded FIFO with integer bandwidth b_l (lines/cycle), latency
 *     L_l (cycles) and capacity cap_l (lines in flight plus waiting);
 *   - per cycle t, from the state at the start of t: every FIFO offers its
 *     first <= b ready entries, every injection stream (source endpoint,
 *     first link) its first <= b released lines in id order; each link grants
 *     min(b, cap - occupancy, #requests) requests, ordered by lowest line id
 *     or round-robin over its tail node's input ports (key (k, port offset));
 *     the longest granted prefix of each source departs; lines enter the
 *     target FIFO in grant order and may leave at t + L; a line leaving its
 *     last link completes at t + 1;
 *   - cycles in which nothing can change are skipped;
 *   - optionally (sim_set_credit) a freed slot returns to its link's
 *     arbiter only some cycles after the line left;
 *   - routes are minimal-hop paths; ties between next hops are broken by the
 *     MurmurHash3 32-bit finalizer of (src << 16 | dst) (hash ECMP);
 *   - a line is injected once all its predecessor lines have completed
 *     (per line, or per whole chunk: sim_dep).
 *
 * Threading: a context is used by one host thread at a time; there is no
 * global mutable state, so distinct contexts may be used concurrently.
 */
#ifndef SIMGPU_H
#define SIMGPU_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sim_ctx sim_ctx; /* opaque, owned by the library */

typedef enum {
    SIM_OK = 0,
    SIM_ERR_INVALID_ARG = 1, /* null pointer, bad enum, out-of-range argument    */
    SIM_ERR_TOPOLOGY = 2,    /* malformed CSR, self-loop, parameter out of range */
    SIM_ERR_UNREACHABLE = 3, /* a needed endpoint pair has no path               */
    SIM_ERR_SIZE = 4,        /* message not divisible into whole lines/chunks    */
    SIM_ERR_OOM = 5,         /* host or device allocation failed                 */
    SIM_ERR_DEVICE = 6,      /* HIP runtime error                                */
    SIM_ERR_DEADLOCK = 7,    /* device: no departure and no future event         */
    SIM_ERR_MAX_CYCLES = 8,  /* device: cycle guard exceeded                     */
    SIM_ERR_STATE = 9        /* call out of order (e.g. run before load)         */
} sim_status;

/* Arbitration: lowest line id, or round-robin over input ports; either may
 * add SIM_ARB_FAIR_CLASSES (Sec. 5.2: fair arbitration of control and data
 * messages).  Then a link ranks its requests by class turns: starting with
 * the class its pointer names (data at first), each pick takes the lowest
 * base key of the class whose turn it is among the sources' heads (requests
 * with no earlier request of the same source left at this link, so that no
 * source's lines are reordered), or of either class if that class has none,
 * and hands the turn to the other class.  After a cycle in which it appended
 * lines, the pointer names the class other than that of the last line
 * appended.  Load requests of sim_load_memcpy are control messages; every
 * other line is data.  The workgroup engine (generic and LDS-resident)
 * simulates SIM_ARB_FAIR_CLASSES. */
typedef enum { SIM_ARB_LOWEST_ID = 0, SIM_ARB_ROUND_ROBIN = 1, SIM_ARB_FAIR_CLASSES = 2 } sim_arb;

/* Collectives (the paper's textbook algorithms, Sec. 1 and 2.2: ring,
 * all-pairs (direct), double binary tree and recursive halving-doubling; the
 * hierarchical form composes direct and ring steps over scale-up domains).
 * p = participants = all endpoints; participant i is endpoint order[i].
 * Transaction ids are step-major (a mixed-radix number whose leading digit
 * is the step), so that lowest-id arbitration favours earlier steps; a
 * message is one step's transfer between two participants.
 *
 *   RING_*          step s, participant i sends C = N/p lines to i+1; id
 *                   (s p + i) C + j.  Line j of step s >= 1 waits for line j
 *                   that i received at step s-1.  All-reduce: 2(p-1) steps;
 *                   reduce-scatter and all-gather: p-1 steps (the same DAG:
 *                   a reduction costs no time).
 *   DIRECT_ALLREDUCE  reduce-scatter: i sends chunk i+k to i+k (k = 1..p-1),
 *                   then all-gather: i sends its reduced chunk i to i+k, line
 *                   j waiting for line j of every reduce-scatter chunk into i;
 *                   id ((phase (p-1) + k-1) p + i) C + j.
 *   DIRECT_ALLGATHER / _REDUCESCATTER  one all-pairs exchange, id
 *                   ((k-1) p + i) C + j, no waits.
 *   RHD_ALLREDUCE   p = 2^K.  Halving step j = 0..K-1: partner i ^ (p >>
 *                   (j+1)); i keeps the half of its block chosen by that bit
 *                   of i and sends the other N >> (j+1) lines, id p(N - 2S) +
 *                   i S + o.  Doubling step j: partner i ^ (1 << j); i sends
 *                   its block of 2^j chunks (starting at chunk (i >> j) << j),
 *                   id N(p-1) + N(2^j - 1) + i 2^j C + o.  A sent position
 *                   waits for every earlier arrival of it at the sender.
 *   DBT_ALLREDUCE   half t of the buffer (H = N/2 lines) is reduced up and
 *                   broadcast down tree t.  Tree shape over positions: 0 is
 *                   the root; position u with lowest set bit b hangs below u
 *                   with bit b cleared and bit 2b set if that is < p, else
 *                   below u with bit b cleared.  Tree 0 puts participant i at
 *                   position i, tree 1 at p-1-i.  Edge e joins non-root
 *                   participant c (e = c-1 in tree 0, c in tree 1) to its
 *                   parent; id ((phase 2 + t)(p-1) + e) H + j, phase 0 = reduce
 *                   (c -> parent, waits for line j from each child), 1 =
 *                   broadcast (parent -> c, waits for line j from each child
 *                   of the root if the parent is the root, else for line j
 *                   broadcast to the parent).
 *   HIER_ALLREDUCE  see sim_load_collective.
 *   ALLTOALL        i sends N lines to i+k (k = 1..p-1), id ((k-1) p + i) N + j.
 */
typedef enum {
    SIM_COLL_RING_ALLREDUCE = 0,       /* reduce-scatter + all-gather ring, 2(p-1) steps */
    SIM_COLL_DIRECT_ALLREDUCE = 1,     /* all-pairs reduce-scatter then all-gather       */
    SIM_COLL_HIER_ALLREDUCE = 2,       /* direct RS in domain, ring per rail, direct AG  */
    SIM_COLL_ALLTOALL = 3,             /* linear-shift all-to-all                        */
    SIM_COLL_RING_ALLGATHER = 4,       /* p-1 ring steps                                 */
    SIM_COLL_RING_REDUCESCATTER = 5,   /* p-1 ring steps                                 */
    SIM_COLL_DIRECT_ALLGATHER = 6,     /* one all-pairs exchange                         */
    SIM_COLL_DIRECT_REDUCESCATTER = 7, /* one all-pairs exchange                         */
    SIM_COLL_RHD_ALLREDUCE = 8,        /* recursive halving-doubling, p a power of two   */
    SIM_COLL_DBT_ALLREDUCE = 9         /* double binary tree                             */
} sim_coll;

/* Granularity of the step-to-step dependencies of a collective (Sec. 4.2
 * and 5.2 contrast get-style transfers, which overlap steps line by line,
 * with put + signal, where a step waits for the signal that the whole
 * message of the step before has arrived). */
typedef enum {
    SIM_DEP_LINE = 0,  /* a line waits for the lines that brought its data to the sender */
    SIM_DEP_CHUNK = 1  /* a message waits for every message that delivers any of its data */
} sim_dep;

/* Limits checked by sim_create. */
#define SIM_MAX_BW 64           /* lines per cycle */
#define SIM_MAX_LAT (1 << 20)   /* cycles          */
#define SIM_MAX_CAP (1 << 16)   /* lines           */
#define SIM_LINE_BYTES 128

/*
 * Create a context from a directed graph (paper Sec. 4.6: the infrastructure
 * as a directed attributed graph whose vertices are hardware units and whose
 * edges carry bandwidth/latency annotations).
 *   n_nodes, n_endpoints : nodes 0..n_endpoints-1 are endpoints (they inject
 *                          and eject lines); the rest are switches.
 *   row_ptr[n_nodes+1], col_idx[m] : CSR out-adjacency; m = row_ptr[n_nodes];
 *                          link id = CSR index; col_idx[l] = head node of l.
 *                          No self-loops.  Parallel links are allowed.
 *   n_scenarios          : S >= 1 independent scenarios sharing topology,
 *                          routing and workload (batched design sweeps).
 *   bw, lat, cap         : [S*m] int32, scenario-major; 1 <= bw <= SIM_MAX_BW,
 *                          1 <= lat <= SIM_MAX_LAT, 1 <= cap <= SIM_MAX_CAP.
 *   arb                  : sim_arb: SIM_ARB_LOWEST_ID or SIM_ARB_ROUND_ROBIN,
 *                          optionally | SIM_ARB_FAIR_CLASSES.
 * Host arrays are copied; the caller keeps ownership.  Routing distances are
 * built here.  Uses the current HIP device.  *out is set only on SIM_OK.
 */
sim_status sim_create(int32_t n_nodes, int32_t n_endpoints, const int32_t *row_ptr,
                      const int32_t *col_idx, int32_t n_scenarios, const int32_t *bw,
                      const int32_t *lat, const int32_t *cap, int32_t arb, sim_ctx **out);

/*
 * Credit-delay flow control (a flow-control variant of the model).
 *   credit : [S*m] int32, scenario-major like bw/lat/cap; 1 <= credit <=
 *            SIM_MAX_LAT; NULL = every delay 1.
 * A slot that a line frees by leaving link l at cycle t is seen free by l's
 * arbiter from cycle t + credit[l] on (1 = the start-of-cycle snapshot of
 * the base model): credits that travel back to the sender take time, which
 * also bounds how soon a link's state can affect its upstream neighbours.
 * Returns of owed credits are events of the time advance.  Delays above 1
 * are simulated by the wave engine (not together with SIM_DEP_CHUNK), the
 * workgroup engine (generic and LDS-resident) and, for one large topology,
 * the grid engine's windowed form.  Any loaded workload is dropped:
 * call sim_load_* again before sim_run.  The array is copied.
 */
sim_status sim_set_credit(sim_ctx *ctx, const int32_t *credit);

/*
 * Load a collective (replaces any previous workload).
 *   coll       : sim_coll.
 *   bytes      : N * 128: the buffer per endpoint (all-reduce; the input of
 *                reduce-scatter; the output of all-gather) or per ordered
 *                pair (all-to-all).  N must divide by the collective's chunk
 *                divisor (p for ring/direct/RHD, 2 for DBT, M*G for
 *                hierarchical), else SIM_ERR_SIZE.
 *   group_size : hierarchical only: endpoints per domain M (endpoint d*M + r);
 *                0 otherwise.
 *   order      : participant order, a permutation of the endpoints (NULL =
 *                rank order); must be NULL for hierarchical and all-to-all.
 *                RHD needs a power-of-two endpoint count (SIM_ERR_INVALID_ARG).
 *   dep        : sim_dep.  Hierarchical all-reduce takes SIM_DEP_LINE only
 *                (SIM_ERR_INVALID_ARG otherwise); for collectives without
 *                waits the two are the same.
 * Builds the routes of every flow used (SIM_ERR_UNREACHABLE if one has no
 * path), the injection streams and the predecessor tables, and uploads them.
 */
sim_status sim_load_collective(sim_ctx *ctx, int32_t coll, uint64_t bytes, int32_t group_size,
                               const int32_t *order, int32_t dep);

/*
 * Load a custom transaction list: line x (0 <= x < n) goes src[x] -> dst[x]
 * (endpoints, src != dst) and may be injected once every line in
 * pred_idx[pred_ptr[x] .. pred_ptr[x+1]) has completed (paper Sec. 4.2: the
 * custom collective algorithms are dependency-ordered transfer lists).  A
 * cyclic predecessor relation is reported as SIM_ERR_DEADLOCK by the run.
 */
sim_status sim_load_transactions(sim_ctx *ctx, int64_t n, const int32_t *src, const int32_t *dst,
                                 const int64_t *pred_ptr, const int64_t *pred_idx);

/*
 * Load memcpy programs run by compute units: the injection side of the GPU
 * model (Sec. 4.4.3 wavefront requests, Sec. 4.4.4 loop unrolling, the
 * outstanding-request limit of Sec. 5.3).  Replaces any previous workload.
 *   n_ops, cu[], src_space[], dst_space[], src_line[], dst_line[], n_lines[]:
 *       operation o copies n_lines[o] lines from line address src_line[o] of
 *       address space src_space[o] to dst_line[o] of dst_space[o]; it runs on
 *       endpoint cu[o].  A CU runs its operations in array order.
 *   n_spaces, n_ch, space_ch[n_spaces * n_ch]: line a of space s lives on the
 *       memory-channel endpoint space_ch[s * n_ch + a mod n_ch].
 *   unroll U >= 1: the copy loop issues U loads, waits for their data, then
 *       issues the U stores (an operation's last group may be shorter).
 *   window W >= 1: a CU's wavefront requests (load requests and stores) are
 *       issued in program order with at most W outstanding, retired in order:
 *       request k waits until request k - W is done.
 * Lines: a load is a request (CU -> source channel) and a data line
 * (channel -> CU) that may leave once the request has arrived; a store
 * (CU -> destination channel) may leave once the data of every load of its
 * group has arrived; a load is done when its data has arrived, a store when
 * it has.  Program order is kept by the network: all of a CU's requests
 * leave through the CU's first link in id order.  Ids are step-major: for
 * issue index k = 0, 1, ... and the CUs in ascending endpoint order, a load
 * takes two ids (request, data), a store one.  Arrays are copied.
 * SIM_ERR_INVALID_ARG for an endpoint out of range, a CU that is also the
 * channel of one of its lines, a space out of range, negative sizes or
 * addresses, U or W < 1; SIM_ERR_SIZE beyond 2^32 - 2 lines.
 */
sim_status sim_load_memcpy(sim_ctx *ctx, int64_t n_ops, const int32_t *cu, const int32_t *src_space,
                           const int32_t *dst_space, const int64_t *src_line, const int64_t *dst_line,
                           const int64_t *n_lines, int32_t n_spaces, int32_t n_ch, const int32_t *space_ch,
                           int32_t unroll, int32_t window);

/* Operation kinds of sim_load_gpu_ops. */
#define SIM_OP_COPY 0
#define SIM_OP_RELEASE 1
#define SIM_OP_ACQUIRE 2

/*
 * Load GPU programs with data and control operations (paper Sec. 4.1.1 GPU
 * instructions, Sec. 4.1.2 GPU operations: memcpy, reduce, acquire and
 * release; Sec. 4.4.2 compute unit; Sec. 4.4.3 a semaphore access is one
 * wavefront request; Sec. 5.2 get- and put-based collectives).  Replaces any
 * previous workload.  sim_load_memcpy is this call with one-source copies.
 *   kind[o]: SIM_OP_COPY, SIM_OP_RELEASE or SIM_OP_ACQUIRE; cu[o] runs it (a
 *       CU runs its operations in array order).
 *   src_ptr[n_ops + 1] (src_ptr[0] = 0), src_space[], src_line[]: the sources
 *       of operation o are entries src_ptr[o] .. src_ptr[o+1] - 1.
 *   SIM_OP_COPY: n_lines[o] lines from each source (line address src_line,
 *       address space src_space) into dst_line[o] of dst_space[o]; one source
 *       is a memcpy, several are a reduce of the sources into the
 *       destination.  Per group of at most U lines the CU issues the loads of
 *       source 0, then of source 1, ..., waits for all of their data, then
 *       issues the group's stores.  The reduce arithmetic itself is taken to
 *       cost no cycles: only its wait for every input is modelled.
 *   SIM_OP_RELEASE: no source, n_lines 1; one store to the semaphore line
 *       (dst_space[o], dst_line[o]) that leaves once every earlier store of
 *       the CU has arrived.  Each semaphore is released exactly once.
 *   SIM_OP_ACQUIRE: no source, n_lines 1; one load of the semaphore line
 *       (request and reply).  Of the polls of a waiting wavefront only the
 *       successful one is simulated: its request leaves once the release of
 *       that semaphore has arrived, and the CU's next request waits for the
 *       reply.
 *   n_spaces, n_ch, space_ch[n_spaces * n_ch], unroll U >= 1, window W >= 1:
 *       as for sim_load_memcpy (W bounds every issued request: load and
 *       acquire requests, stores and releases).
 * Ids are step-major: for issue index k = 0, 1, ... and the CUs in ascending
 * endpoint order, a load or acquire takes two ids (request, then data or
 * reply), a store or release one.  Stores and data lines are data messages
 * (class 0); load requests and every line of a release or acquire are control
 * messages (class 1).  A memory channel returns its lines in id order: an
 * acquire whose reply waits for a late release holds back that channel's
 * later replies, and a program in which that closes a cycle of waits is
 * reported as SIM_ERR_DEADLOCK by the run.  Arrays are copied.
 * SIM_ERR_INVALID_ARG for an unknown kind, a copy without a source, a release
 * or acquire with a source or n_lines != 1, a semaphore released twice or
 * acquired but never released, and the errors of sim_load_memcpy;
 * SIM_ERR_SIZE beyond 2^32 - 2 lines.
 */
sim_status sim_load_gpu_ops(sim_ctx *ctx, int64_t n_ops, const int32_t *kind, const int32_t *cu,
                            const int64_t *src_ptr, const int32_t *src_space, const int64_t *src_line,
                            const int32_t *dst_space, const int64_t *dst_line, const int64_t *n_lines,
                            int32_t n_spaces, int32_t n_ch, const int32_t *space_ch, int32_t unroll,
                            int32_t window);

/* Sizes of the loaded problem: transactions T, links m, scenarios S and
 * line-hops per scenario (sum of path lengths; a line-hop is one admission of
 * a 128 B wavefront request onto a link, the per-line, per-hop unit of work
 * of Sec. 4.4.3).  Any pointer may be NULL.  SIM_ERR_STATE before a load
 * (n_links and n_scenarios are still written). */
sim_status sim_sizes(const sim_ctx *ctx, int64_t *n_txn, int32_t *n_links, int32_t *n_scenarios,
                     uint64_t *line_hops);

/*
 * Enqueue one full simulation of every scenario on hip_stream (a
 * hipStream_t; NULL = the null stream) and return.  This is the network
 * side of the fine-grained simulation: every wavefront request (one 128 B
 * cache line, Sec. 4.4.3) is advanced link by link through the graph of
 * endpoints and switches with the routing of Sec. 4.5, under the queueing
 * rules stated at the top of this header.  Outputs are caller-owned
 * device buffers that must stay valid until the stream reaches this work:
 *   d_completion  [S*T] u32 : completion cycle of every line (scenario-major)
 *   d_tx_lines    [S*m] u64 : lines admitted onto each link
 *   d_busy_cycles [S*m] u64 : cycles in which each link admitted >= 1 line
 *   d_makespan    [S]   u32 : max completion per scenario
 * max_cycles bounds the simulated cycle (0 = the largest supported guard).
 * Argument errors return synchronously.  Deadlock / guard overrun are found
 * on the device: read them with sim_status_after_sync once the stream has
 * been synchronised; the outputs of a failed scenario are unspecified.
 */
sim_status sim_run(sim_ctx *ctx, void *hip_stream, uint32_t *d_completion, uint64_t *d_tx_lines,
                   uint64_t *d_busy_cycles, uint32_t *d_makespan, uint64_t max_cycles);

/*
 * sim_run without any device allocation, for callers that cannot allocate:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments, outputs and errors as sim_run; the engines'
 * per-run scratch (per-scenario statuses and cycle counts, and the FIFO
 * rings, per-link scalars and request records of the engines that keep
 * them in device memory) comes from a fixed array of
 * SIM_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on
 * until the process ends, instead of from the context.  SIM_ERR_SIZE (and
 * nothing enqueued) if the loaded workload needs more scratch than that.
 * The call allocates nothing; the first call on a device looks the array's
 * address up.  Every call on a GPU uses the same array and leaves its
 * contents behind (each run initialises what it reads): runs that overlap
 * on one GPU -- on different streams, or from different contexts before the
 * earlier run has finished -- race on it, and a later run overwrites the
 * statuses sim_status_after_sync reports for an earlier one, so synchronise
 * and read the status before the next call.
 */
#define SIM_NOALLOC_SCRATCH_BYTES (8u << 20)
sim_status sim_run_noalloc(sim_ctx *ctx, void *hip_stream, uint32_t *d_completion, uint64_t *d_tx_lines,
                           uint64_t *d_busy_cycles, uint32_t *d_makespan, uint64_t max_cycles);

/* After the caller has synchronised the run's stream: SIM_OK, or the first
 * device-detected error (DEADLOCK / MAX_CYCLES) over the scenarios.  (Error
 * reporting of this library; the paper has no counterpart.)  If
 * status/cycles are non-NULL they receive per-scenario statuses ([S] int32)
 * and processed-cycle counts ([S] u64) on the host. */
sim_status sim_status_after_sync(sim_ctx *ctx, int32_t *status, uint64_t *cycles);

/* Route of flow src -> dst as link ids (host copy; *len = hop count): the
 * routing function of Sec. 4.5 over the graph of Sec. 4.6, here minimal-hop
 * paths with MurmurHash3-finalizer ECMP tie-breaks (see the top of this
 * header).  src == dst gives *len = 0.  SIM_ERR_INVALID_ARG for endpoints out
 * of range or a NULL len; SIM_ERR_UNREACHABLE if dst cannot be reached;
 * SIM_ERR_SIZE if cap < hop count or links is NULL for a non-empty route
 * (then *len still holds the count).  links (cap entries) is caller-owned. */
sim_status sim_route(const sim_ctx *ctx, int32_t src, int32_t dst, int32_t *links, int32_t cap,
                     int32_t *len);

/*
 * Decode line id of the loaded workload: the unit transfer of the network
 * model is one 128 B wavefront request (Sec. 4.4.3); this names which
 * transfer of the workload it is.
 *   *src, *dst  : its source and destination endpoints;
 *   *phase_step : the algorithm step of the line, the leading digit of the
 *                 step-major id (see sim_coll): ring s; direct all-reduce
 *                 phase (p-1) + k-1; direct all-gather / reduce-scatter and
 *                 all-to-all k-1; hierarchical: phase 1 k-1, phase 2 (M-1) +
 *                 s, phase 3 (M-1) + (2G-2) + k-1; RHD: halving step j,
 *                 doubling step K + j; DBT: 2 phase + tree.  memcpy
 *                 programs: the issue index of the request in its CU's
 *                 program.  Custom transaction lists: -1;
 *   *line       : the line's offset within its message (one step's transfer
 *                 between two participants); memcpy: 0 for a load request or
 *                 a store, 1 for a load's data line; custom lists: 0.
 * Any output pointer may be NULL.  SIM_ERR_STATE before a load;
 * SIM_ERR_INVALID_ARG if id is outside [0, T).  Host-only, no device work:
 * it answers for the last load whose workload expansion succeeded, also when
 * that load then failed to bind device memory (SIM_ERR_DEVICE / SIM_ERR_OOM).
 */
sim_status sim_txn_info(const sim_ctx *ctx, int64_t id, int32_t *src, int32_t *dst, int32_t *phase_step,
                        int32_t *line);

/* Last error message of this context (owned by the context; never NULL).
 * Error reporting of this library; the paper has no counterpart. */
const char *sim_last_error(const sim_ctx *ctx);

/* Free the context and all its device memory.  NULL is allowed.  (Resource
 * management of this library; the paper has no counterpart.) */
void sim_destroy(sim_ctx *ctx);

#ifdef __cplusplus
}
#endif
#endif /* SIMGPU_H */
