/*
 * CPU oracle for the line-granularity network model -- TEST INFRASTRUCTURE.
 *
 * This file is the plain, slow, single-threaded reference that the GPU
 * library is checked against.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load it; the product never does.  It
 * shares no code, header or table with the GPU library.
 *
 * What it computes (paper: Sec. 4.4.3 "Wavefront Request" -- a 128 B
 * cache-line transfer is the unit the network simulates; Sec. 4.5 "Detailed
 * Simple Network Modeling" -- the network is a graph of endpoints and
 * switches with a routing function; Sec. 2.1 -- the Simple backend is an
 * alpha-beta model; Sec. 1/2 list ring and direct collectives).  The paper
 * leaves the queueing discipline unstated, so the model below is the reading
 * this project adopts (all readings are listed with the design notes):
 *
 *   link l : FIFO of (line, ready) entries; integer bandwidth b (lines per
 *            cycle), latency L (cycles), capacity cap (lines in flight plus
 *            waiting).  Entered at cycle t -> may leave at t + L.
 *   cycle t (every decision uses the state at the start of t):
 *     requests  each FIFO offers its first <= b entries with ready <= t
 *               (stopping at the first not-ready one); each injection stream
 *               (src endpoint, first link) offers its first <= b released
 *               lines in ascending id (stopping at the first unreleased one).
 *               The k-th offered line requests the next link of its path, or
 *               the sink when the current link is its last hop.
 *     grants    per link f: order the requests (lowest line id first, or
 *               round-robin: ascending (k, (port - rr_f) mod P)) and grant
 *               the first min(b_f, cap_f - occ_f, #requests); the sink
 *               grants everything.
 *     departures from every source exactly the longest granted prefix
 *               (k = 0, 1, ...) departs; a grant beyond it is void.
 *     enter     departing lines join their target FIFO in grant order with
 *               ready = t + L; counters; round-robin pointer moves past the
 *               port of the last appended line.
 *     eject     a line leaving to the sink completes at t + 1.
 *     time      next cycle is t + 1 if anything departed, else the earliest
 *               future FIFO-head ready time; no such time while lines remain
 *               is a deadlock.
 *   routing   minimal hop paths; among equal-length next hops, a choice by
 *             the MurmurHash3 32-bit finalizer of (src << 16 | dst).
 *   release   a line may be injected once all its predecessor lines have
 *             completed (rel = max predecessor completion, 0 if none).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <time.h>

#define OR_OK 0
#define OR_ERR_INVALID_ARG 1
#define OR_ERR_TOPOLOGY 2
#define OR_ERR_UNREACHABLE 3
#define OR_ERR_SIZE 4
#define OR_ERR_OOM 5
#define OR_ERR_DEADLOCK 7
#define OR_ERR_MAX_CYCLES 8
#define OR_ERR_INVARIANT 100

#define NEVER 0xFFFFFFFFu
#define SINK (-1)

/* ---------------------------------------------------------------- hashing */

/* MurmurHash3 (Appleby) 32-bit finalizer: xor-shift 16, multiply by
 * 0x85ebca6b, xor-shift 13, multiply by 0xc2b2ae35, xor-shift 16. */
uint32_t oracle_fmix32(uint32_t h)
{
    h ^= h >> 16;
    h *= 0x85ebca6bu;
    h ^= h >> 13;
    h *= 0xc2b2ae35u;
    h ^= h >> 16;
    return h;
}

/* ---------------------------------------------------------------- routing */

/* Hop distance from every node to endpoint d: breadth-first search from d
 * over the reversed links (in_ptr/in_tail list, for each node w, the tails
 * of the links entering w).  dist = -1 when d is unreachable. */
static void bfs_to(int32_t n, const int32_t *in_ptr, const int32_t *in_tail,
                   int32_t d, int32_t *dist, int32_t *queue)
{
    for (int32_t v = 0; v < n; v++) dist[v] = -1;
    dist[d] = 0;
    int32_t qh = 0, qt = 0;
    queue[qt++] = d;
    while (qh < qt) {
        int32_t w = queue[qh++];
        for (int32_t q = in_ptr[w]; q < in_ptr[w + 1]; q++) {
            int32_t u = in_tail[q];
            if (dist[u] >= 0) continue;
            dist[u] = dist[w] + 1;
            queue[qt++] = u;
        }
    }
}

/* Path of flow (s, d) given dist-to-d.  At each node the candidates are the
 * out-links (ascending id) whose head is one hop closer to d; at the j-th
 * node with two or more candidates, the choice is byte (j mod 4) of the hash
 * modulo the candidate count, and the hash is re-mixed before every fourth
 * choice point after the first.  cand has room for the largest out-degree.
 * Returns the hop count. */
static int32_t trace_path(const int32_t *row_ptr, const int32_t *col_idx,
                          const int32_t *dist, int32_t s, int32_t d,
                          int32_t *out, int32_t *cand)
{
    uint32_t h = oracle_fmix32(((uint32_t)s << 16) | (uint32_t)d);
    int32_t v = s, len = 0, j = 0;
    while (v != d) {
        int32_t nc = 0;
        for (int32_t l = row_ptr[v]; l < row_ptr[v + 1]; l++)
            if (dist[col_idx[l]] == dist[v] - 1) cand[nc++] = l;
        int32_t pick;
        if (nc == 1) {
            pick = cand[0];
        } else {
            if (j > 0 && j % 4 == 0) h = oracle_fmix32(h);
            pick = cand[((h >> (8 * (j % 4))) & 255u) % (uint32_t)nc];
            j++;
        }
        out[len++] = pick;
        v = col_idx[pick];
    }
    return len;
}

/* All E*E flow paths.  path_ptr has E*E+1 entries (flow = s*E + d).  A pair
 * with s == d or with no path gets an empty path.  Returns OR_ERR_SIZE if
 * path_cap is too small (path_ptr[E*E] then holds the need). */
int oracle_paths(int32_t n, int32_t E, const int32_t *row_ptr,
                 const int32_t *col_idx, int64_t *path_ptr, int32_t *path_link,
                 int64_t path_cap)
{
    int32_t *dist = malloc(sizeof(int32_t) * (size_t)n * (size_t)E);
    int32_t *queue = malloc(sizeof(int32_t) * (size_t)n);
    int32_t *tmp = malloc(sizeof(int32_t) * (size_t)(n + 1));
    int32_t m = row_ptr[n];
    int32_t maxdeg = 1;
    for (int32_t u = 0; u < n; u++)
        if (row_ptr[u + 1] - row_ptr[u] > maxdeg) maxdeg = row_ptr[u + 1] - row_ptr[u];
    int32_t *cand = malloc(sizeof(int32_t) * (size_t)maxdeg);
    if (!dist || !queue || !tmp || !cand) { free(dist); free(queue); free(tmp); free(cand); return OR_ERR_OOM; }
    int rc = OR_OK;
    int32_t *in_ptr = calloc((size_t)n + 1, sizeof(int32_t));
    int32_t *in_tail = malloc(sizeof(int32_t) * (size_t)(m + 1));
    int32_t *fill = calloc((size_t)n, sizeof(int32_t));
    for (int32_t l = 0; l < m; l++) in_ptr[col_idx[l] + 1]++;
    for (int32_t v = 0; v < n; v++) in_ptr[v + 1] += in_ptr[v];
    for (int32_t u = 0; u < n; u++)
        for (int32_t l = row_ptr[u]; l < row_ptr[u + 1]; l++)
            in_tail[in_ptr[col_idx[l]] + fill[col_idx[l]]++] = u;
    for (int32_t d = 0; d < E; d++) bfs_to(n, in_ptr, in_tail, d, dist + (size_t)d * n, queue);
    free(in_ptr); free(in_tail); free(fill);
    int64_t pos = 0;
    for (int32_t s = 0; s < E && rc == OR_OK; s++) {
        for (int32_t d = 0; d < E; d++) {
            path_ptr[(int64_t)s * E + d] = pos;
            if (s == d) continue;
            const int32_t *dd = dist + (size_t)d * n;
            if (dd[s] < 0) continue;  /* unreachable: empty path */
            int32_t len = trace_path(row_ptr, col_idx, dd, s, d, tmp, cand);
            if (pos + len <= path_cap) memcpy(path_link + pos, tmp, sizeof(int32_t) * (size_t)len);
            pos += len;
        }
    }
    path_ptr[(int64_t)E * E] = pos;
    if (rc == OR_OK && pos > path_cap) rc = OR_ERR_SIZE;
    free(dist); free(queue); free(tmp); free(cand);
    return rc;
}

/* Routes of the (source, destination) pairs one workload uses, for graphs
 * whose all-pairs table would not fit: an open-addressing hash from the key
 * s * E + d to the pair's path, each traced as above, destination by
 * destination so that one distance array is alive at a time. */
typedef struct {
    int64_t cap;        /* hash slots (power of two) */
    int64_t *key;       /* -1: empty */
    int64_t *idx;       /* pair index of the slot */
    int64_t np;         /* pairs */
    int64_t *pkey;      /* [np] keys in insertion order */
    int64_t *ptr;       /* [np + 1] path start in link */
    int32_t *link;
} routes_t;

static int64_t route_slot(const routes_t *r, int64_t key)
{
    uint64_t h = (uint64_t)key * 0x9E3779B97F4A7C15ull;   /* Fibonacci hashing */
    int64_t i = (int64_t)(h >> 20) & (r->cap - 1);
    while (r->key[i] != -1 && r->key[i] != key) i = (i + 1) & (r->cap - 1);
    return i;
}

static int routes_add(routes_t *r, int64_t key)
{
    if (2 * (r->np + 1) > r->cap) {                    /* grow to keep the load under one half */
        routes_t g = *r;
        g.cap = r->cap ? 2 * r->cap : 1024;
        g.key = malloc(sizeof(int64_t) * (size_t)g.cap);
        g.idx = malloc(sizeof(int64_t) * (size_t)g.cap);
        g.pkey = realloc(r->pkey, sizeof(int64_t) * (size_t)g.cap);
        if (!g.key || !g.idx || !g.pkey) return OR_ERR_OOM;
        for (int64_t i = 0; i < g.cap; i++) g.key[i] = -1;
        for (int64_t q = 0; q < r->np; q++) {
            int64_t i = route_slot(&g, g.pkey[q]);
            g.key[i] = g.pkey[q];
            g.idx[i] = q;
        }
        free(r->key); free(r->idx);
        *r = g;
    }
    int64_t i = route_slot(r, key);
    if (r->key[i] == -1) {
        r->key[i] = key;
        r->idx[i] = r->np;
        r->pkey[r->np++] = key;
    }
    return OR_OK;
}

static int64_t routes_find(const routes_t *r, int64_t key)
{
    if (!r->cap) return -1;
    int64_t i = route_slot(r, key);
    return r->key[i] == key ? r->idx[i] : -1;
}

/* Trace every pair (unreachable: empty path). */
static int routes_trace(routes_t *r, int32_t n, int32_t E, const int32_t *row_ptr, const int32_t *col_idx)
{
    int32_t m = row_ptr[n];
    int32_t maxdeg = 1;
    for (int32_t u = 0; u < n; u++)
        if (row_ptr[u + 1] - row_ptr[u] > maxdeg) maxdeg = row_ptr[u + 1] - row_ptr[u];
    int32_t *dist = malloc(sizeof(int32_t) * (size_t)n), *queue = malloc(sizeof(int32_t) * (size_t)n);
    int32_t *cand = malloc(sizeof(int32_t) * (size_t)maxdeg);
    int32_t *in_ptr = calloc((size_t)n + 1, sizeof(int32_t)), *in_tail = malloc(sizeof(int32_t) * (size_t)(m + 1));
    int32_t *fill = calloc((size_t)n, sizeof(int32_t));
    int64_t *order = malloc(sizeof(int64_t) * (size_t)(r->np > 0 ? r->np : 1));
    int32_t *len = malloc(sizeof(int32_t) * (size_t)(r->np > 0 ? r->np : 1));
    r->ptr = malloc(sizeof(int64_t) * (size_t)(r->np + 1));
    if (!dist || !queue || !cand || !in_ptr || !in_tail || !fill || !order || !len || !r->ptr) return OR_ERR_OOM;
    for (int32_t l = 0; l < m; l++) in_ptr[col_idx[l] + 1]++;
    for (int32_t v = 0; v < n; v++) in_ptr[v + 1] += in_ptr[v];
    for (int32_t u = 0; u < n; u++)
        for (int32_t l = row_ptr[u]; l < row_ptr[u + 1]; l++)
            in_tail[in_ptr[col_idx[l]] + fill[col_idx[l]]++] = u;
    /* pairs grouped by destination (counting sort) */
    int64_t *dcnt = calloc((size_t)E + 1, sizeof(int64_t));
    if (!dcnt) return OR_ERR_OOM;
    for (int64_t q = 0; q < r->np; q++) dcnt[r->pkey[q] % E + 1]++;
    for (int32_t d = 0; d < E; d++) dcnt[d + 1] += dcnt[d];
    for (int64_t q = 0; q < r->np; q++) order[dcnt[r->pkey[q] % E]++] = q;
    free(dcnt);
    /* path lengths are the distances: a first pass sizes the table */
    int64_t total = 0;
    for (int64_t a = 0; a < r->np; a++) {
        int32_t d = (int32_t)(r->pkey[order[a]] % E), s = (int32_t)(r->pkey[order[a]] / E);
        if (a == 0 || r->pkey[order[a - 1]] % E != d) bfs_to(n, in_ptr, in_tail, d, dist, queue);
        len[order[a]] = s == d || dist[s] < 0 ? 0 : dist[s];
        total += len[order[a]];
    }
    r->ptr[0] = 0;
    for (int64_t q = 0; q < r->np; q++) r->ptr[q + 1] = r->ptr[q] + len[q];
    r->link = malloc(sizeof(int32_t) * (size_t)(total > 0 ? total : 1));
    if (!r->link) return OR_ERR_OOM;
    for (int64_t a = 0; a < r->np; a++) {
        int32_t d = (int32_t)(r->pkey[order[a]] % E), s = (int32_t)(r->pkey[order[a]] / E);
        if (a == 0 || r->pkey[order[a - 1]] % E != d) bfs_to(n, in_ptr, in_tail, d, dist, queue);
        if (len[order[a]]) trace_path(row_ptr, col_idx, dist, s, d, r->link + r->ptr[order[a]], cand);
    }
    free(dist); free(queue); free(cand); free(in_ptr); free(in_tail); free(fill); free(order); free(len);
    return OR_OK;
}

static void routes_free(routes_t *r)
{
    free(r->key); free(r->idx); free(r->pkey); free(r->ptr); free(r->link);
    memset(r, 0, sizeof(*r));
}

/* ------------------------------------------------------ workload expansion */

enum {
    COLL_RING = 0, COLL_DIRECT = 1, COLL_HIER = 2, COLL_A2A = 3,
    COLL_RING_AG = 4, COLL_RING_RS = 5, COLL_DIRECT_AG = 6, COLL_DIRECT_RS = 7,
    COLL_RHD = 8, COLL_DBT = 9, COLL_CUSTOM = -1
};

/* Dependency granularity of a collective step (Sec. 4.2, 5.2): per line (a
 * line may leave once the same line of the previous step has arrived, the
 * get-style overlap), or per chunk (put + signal: a message -- one step's
 * transfer from one participant to another -- starts once every message
 * that delivers any of its inputs has arrived whole). */
enum { DEP_LINE = 0, DEP_CHUNK = 1 };

typedef struct {
    int coll;
    int dep;                /* DEP_LINE or DEP_CHUNK */
    int32_t E;              /* endpoints */
    int32_t p;              /* participants (ring/direct: all endpoints) */
    const int32_t *rho;     /* ring order (NULL = rank order) */
    int64_t C;              /* ring/direct/a2a/rhd chunk lines */
    int64_t N;              /* rhd: buffer lines */
    int32_t K;              /* rhd: log2 p */
    int64_t H;              /* dbt: lines per tree (half the buffer) */
    int64_t G, M, C1, C2, B2, B3;  /* hierarchical */
    int64_t T;
    /* custom */
    const int32_t *csrc, *cdst;
    const int64_t *pptr, *pidx;
} work_t;

static int32_t rho_of(const work_t *w, int64_t i) { return w->rho ? w->rho[i] : (int32_t)i; }

/* Transaction-id spaces are step-major: for each collective the id is a
 * mixed-radix number whose most significant digit is the algorithm step, so
 * that lowest-id arbitration favours earlier steps. */
static int setup_work(work_t *w, int coll, uint64_t bytes, int32_t group, int32_t E,
                      const int32_t *order, int dep)
{
    memset(w, 0, sizeof(*w));
    w->coll = coll; w->E = E; w->p = E; w->rho = order; w->dep = dep;
    if (dep != DEP_LINE && dep != DEP_CHUNK) return OR_ERR_INVALID_ARG;
    if (dep == DEP_CHUNK && coll == COLL_HIER) return OR_ERR_INVALID_ARG;  /* not defined here */
    if (order && (coll == COLL_HIER || coll == COLL_A2A)) return OR_ERR_INVALID_ARG;
    if (bytes == 0 || bytes % 128 != 0) return OR_ERR_SIZE;
    int64_t N = (int64_t)(bytes / 128);  /* lines */
    if (E < 2) return OR_ERR_INVALID_ARG;
    switch (coll) {
    case COLL_RING:
        if (N % E) return OR_ERR_SIZE;
        w->C = N / E;
        w->T = (2 * (int64_t)E - 2) * E * w->C;
        break;
    case COLL_DIRECT:
        if (N % E) return OR_ERR_SIZE;
        w->C = N / E;
        w->T = 2 * (int64_t)(E - 1) * E * w->C;
        break;
    case COLL_HIER:
        if (group < 2 || E % group || E / group < 2) return OR_ERR_INVALID_ARG;
        w->M = group; w->G = E / group;
        if (N % w->M) return OR_ERR_SIZE;
        w->C1 = N / w->M;
        if (w->C1 % w->G) return OR_ERR_SIZE;
        w->C2 = w->C1 / w->G;
        w->B2 = (w->M - 1) * w->G * w->M * w->C1;
        w->B3 = w->B2 + (2 * w->G - 2) * w->M * w->G * w->C2;
        w->T = w->B3 + (w->M - 1) * w->G * w->M * w->C1;
        break;
    case COLL_A2A:
        w->C = N;
        w->T = (int64_t)(E - 1) * E * w->C;
        break;
    case COLL_RING_AG: case COLL_RING_RS: case COLL_DIRECT_AG: case COLL_DIRECT_RS:
        if (N % E) return OR_ERR_SIZE;
        w->C = N / E;
        w->T = (int64_t)(E - 1) * E * w->C;
        break;
    case COLL_RHD:
        if (E & (E - 1)) return OR_ERR_INVALID_ARG;   /* power of two participants */
        if (N % E) return OR_ERR_SIZE;
        while ((1 << w->K) < E) w->K++;
        w->N = N;
        w->C = N / E;
        w->T = 2 * N * (int64_t)(E - 1);
        break;
    case COLL_DBT:
        if (N % 2) return OR_ERR_SIZE;
        w->H = N / 2;
        w->T = 4 * (int64_t)(E - 1) * w->H;
        break;
    default:
        return OR_ERR_INVALID_ARG;
    }
    if (w->T >= (int64_t)0xFFFFFFFF) return OR_ERR_SIZE;
    return OR_OK;
}

static int64_t pmod(int64_t a, int64_t m) { int64_t r = a % m; return r < 0 ? r + m : r; }

/* ---- recursive halving-doubling all-reduce (Thakur et al., cited in Sec. 1)
 * p = 2^K participants, N lines per buffer, chunk C = N/p.
 * Reduce-scatter step j (0 <= j < K): partner at distance p >> (j+1).
 *   Before the step participant i holds the block of 2 S_j lines (S_j =
 *   N >> (j+1)) starting at (i >> (K-j)) * 2 S_j; it keeps the half chosen by
 *   bit (K-1-j) of i and sends the other half to the partner.  After K steps
 *   i holds chunk i reduced.
 *   ids: p (N - 2 S_j) + i S_j + o.
 * All-gather step j: partner at distance 1 << j; i sends its block of 2^j
 *   chunks, which starts at chunk (i >> j) << j.
 *   ids: N (p-1) + N (2^j - 1) + i 2^j C + o.
 * A sent line at buffer position q waits, per line, for every earlier
 * arrival of position q at its sender: in reduce-scatter the partial sums of
 * all earlier steps; in all-gather, for the sender's own chunk, all K
 * reduce-scatter arrivals, else the all-gather step that brought q. */
static int64_t rhd_rs_len(const work_t *w, int32_t j) { return w->N >> (j + 1); }
static int64_t rhd_rs_base(const work_t *w, int32_t j) { return (int64_t)w->p * (w->N - 2 * rhd_rs_len(w, j)); }
static int64_t rhd_ag_len(const work_t *w, int32_t j) { return w->C << j; }
static int64_t rhd_ag_base(const work_t *w, int32_t j)
{
    return w->N * (int64_t)(w->p - 1) + w->N * (((int64_t)1 << j) - 1);
}
/* first buffer position of the half participant i sends at reduce-scatter step j */
static int64_t rhd_rs_send_start(const work_t *w, int64_t i, int32_t j)
{
    int64_t S = rhd_rs_len(w, j);
    int64_t block = (i >> (w->K - j)) * 2 * S;
    int64_t keep_upper = (i >> (w->K - 1 - j)) & 1;
    return block + (keep_upper ? 0 : S);
}
/* id of the line that brought position q to participant i at reduce-scatter step j */
static int64_t rhd_rs_arrival(const work_t *w, int64_t i, int32_t j, int64_t q)
{
    int64_t from = i ^ ((int64_t)w->p >> (j + 1));
    return rhd_rs_base(w, j) + from * rhd_rs_len(w, j) + (q - rhd_rs_send_start(w, from, j));
}
/* id of the line that brought position q to participant i at all-gather step h */
static int64_t rhd_ag_arrival(const work_t *w, int64_t i, int32_t h, int64_t q)
{
    int64_t from = i ^ ((int64_t)1 << h);
    return rhd_ag_base(w, h) + from * rhd_ag_len(w, h) + (q - ((from >> h) << h) * w->C);
}

/* ---- double binary tree all-reduce (Jeaugey, cited in Sec. 1)
 * Half t of the buffer (H lines) is reduced up tree t to its root and then
 * broadcast down it.  Both trees have one shape over positions 0..p-1:
 * position 0 is the root; any other position u with lowest set bit b hangs
 * below u with bit b cleared and bit 2b set, when that is a position, else
 * below u with bit b cleared (the in-order binary tree).  Tree 0
 * puts participant i at position i, tree 1 at position p-1-i, so the leaves
 * of one are inner nodes of the other.
 * Edge e of tree t joins its non-root participant c (e = c-1 in tree 0, c in
 * tree 1) to the parent.  ids: ((phase*2 + t)(p-1) + e) H + j, phase 0 =
 * reduce (c -> parent), 1 = broadcast (parent -> c).
 * A reduce line waits for the same line from each child; a broadcast line
 * from the root waits for the same line from each child of the root, from
 * any other node for the same line broadcast to it. */
static int64_t dbt_parent_pos(int64_t u, int64_t p)
{
    if (u == 0) return -1;
    int64_t b = u & -u;
    int64_t up = (u - b) | (2 * b);
    return up < p ? up : u - b;
}
static int64_t dbt_pos(int64_t i, int t, int64_t p) { return t == 0 ? i : p - 1 - i; }  /* its own inverse */
static int64_t dbt_edge(int64_t c, int t) { return t == 0 ? c - 1 : c; }
static int64_t dbt_edge_part(int64_t e, int t) { return t == 0 ? e + 1 : e; }

/* Message of a line (chunk mode): one step's transfer between two
 * participants, a contiguous id range. */
static int64_t msg_of(const work_t *w, int64_t x)
{
    if (w->coll == COLL_DBT) return x / w->H;
    if (w->coll == COLL_RHD) {
        if (x < rhd_ag_base(w, 0)) {
            int32_t j = 0;
            while (j + 1 < w->K && x >= rhd_rs_base(w, j + 1)) j++;
            return (int64_t)j * w->p + (x - rhd_rs_base(w, j)) / rhd_rs_len(w, j);
        }
        int32_t j = 0;
        while (j + 1 < w->K && x >= rhd_ag_base(w, j + 1)) j++;
        return (int64_t)(w->K + j) * w->p + (x - rhd_ag_base(w, j)) / rhd_ag_len(w, j);
    }
    return x / w->C;
}
static int64_t msg_count(const work_t *w)
{
    if (w->coll == COLL_DBT) return w->T / w->H;
    if (w->coll == COLL_RHD) return 2 * (int64_t)w->K * w->p;
    return w->T / w->C;
}
static int64_t msg_first(const work_t *w, int64_t m)
{
    if (w->coll == COLL_DBT) return m * w->H;
    if (w->coll == COLL_RHD) {
        int32_t j = (int32_t)(m / w->p);
        int64_t i = m % w->p;
        if (j < w->K) return rhd_rs_base(w, j) + i * rhd_rs_len(w, j);
        return rhd_ag_base(w, j - w->K) + i * rhd_ag_len(w, j - w->K);
    }
    return m * w->C;
}
static int64_t msg_len(const work_t *w, int64_t m)
{
    if (w->coll == COLL_DBT) return w->H;
    if (w->coll == COLL_RHD) {
        int32_t j = (int32_t)(m / w->p);
        return j < w->K ? rhd_rs_len(w, j) : rhd_ag_len(w, j - w->K);
    }
    return w->C;
}

/* Most predecessors decode() can write for one line of this workload: the
 * longest list of a custom workload; for the collectives, the sender's
 * arrivals of one position, which the endpoint count bounds (direct: p - 1;
 * hierarchical: M; RHD: K + j < 2K; DBT: at most two children). */
static int64_t pred_bound(const work_t *w)
{
    if (w->coll == COLL_CUSTOM) {
        int64_t most = 1;
        for (int64_t x = 0; x < w->T; x++)
            if (w->pptr[x + 1] - w->pptr[x] > most) most = w->pptr[x + 1] - w->pptr[x];
        return most;
    }
    return (int64_t)w->E + 2 * (int64_t)w->K + 8;
}

/* Decode transaction x into (src, dst) and its predecessor list.
 * Returns the number of predecessors written to preds, which must have room
 * for pred_bound(w) entries.  A
 * predecessor p >= 0 is a line; in chunk mode a predecessor is a whole chunk,
 * written -1 - c for chunk c = the C lines [c*C, (c+1)*C). */
static int32_t decode(const work_t *w, int64_t x, int32_t *src, int32_t *dst, int64_t *preds)
{
    int32_t np = 0;
    if (w->coll == COLL_CUSTOM) {
        *src = w->csrc[x]; *dst = w->cdst[x];
        for (int64_t q = w->pptr[x]; q < w->pptr[x + 1]; q++) preds[np++] = w->pidx[q];
        return np;
    }
    if (w->coll == COLL_RING || w->coll == COLL_RING_AG || w->coll == COLL_RING_RS) {
        /* id = (s*p + i)*C + j; sends rho(i) -> rho(i+1); waits for the same
         * line of the previous step received from rho(i-1).  All-reduce runs
         * 2(p-1) steps; reduce-scatter and all-gather p-1, whose dependency
         * structure is the same (the reduction itself costs no time). */
        int64_t p = w->p, C = w->C;
        int64_t j = x % C, q = x / C, i = q % p, s = q / p;
        *src = rho_of(w, i); *dst = rho_of(w, (i + 1) % p);
        if (s >= 1) {
            int64_t prev = (s - 1) * p + pmod(i - 1, p);
            preds[np++] = w->dep == DEP_CHUNK ? -1 - prev : prev * C + j;
        }
        return np;
    }
    if (w->coll == COLL_DIRECT) {
        /* id = ((ph*(p-1) + (k-1))*p + i)*C + j; i -> i+k.  Reduce-scatter
         * (ph 0) has no predecessors; all-gather line j of chunk i waits for
         * every reduce-scatter line j of chunk i delivered to i. */
        int64_t p = w->p, C = w->C;
        int64_t j = x % C, q = x / C, i = q % p;
        q /= p;
        int64_t k = q % (p - 1) + 1, ph = q / (p - 1);
        *src = rho_of(w, i); *dst = rho_of(w, (i + k) % p);
        if (ph == 1)
            for (int64_t i2 = 0; i2 < p; i2++) {
                if (i2 == i) continue;
                int64_t k2 = pmod(i - i2, p);
                int64_t rs = (0 * (p - 1) + (k2 - 1)) * p + i2;  /* reduce-scatter chunk into i */
                preds[np++] = w->dep == DEP_CHUNK ? -1 - rs : rs * C + j;
            }
        return np;
    }
    if (w->coll == COLL_HIER) {
        int64_t G = w->G, M = w->M, C1 = w->C1, C2 = w->C2;
        if (x < w->B2) {
            /* phase 1: intra-domain reduce-scatter, (d, r) -> (d, r+k) */
            int64_t q = x / C1, r = q % M;
            q /= M;
            int64_t d = q % G, k = q / G + 1;
            *src = (int32_t)(d * M + r); *dst = (int32_t)(d * M + (r + k) % M);
            return 0;
        }
        if (x < w->B3) {
            /* phase 2: ring over domains on rail r, (d, r) -> (d+1, r) */
            int64_t y = x - w->B2;
            int64_t j = y % C2, q = y / C2, d = q % G;
            q /= G;
            int64_t r = q % M, s = q / M;
            *src = (int32_t)(d * M + r); *dst = (int32_t)(((d + 1) % G) * M + r);
            if (s <= G - 1) {
                /* reduce-scatter steps and the first all-gather step send
                 * sub-chunk (d - s) mod G combined with this node's own copy,
                 * which must first be reduced inside the domain: all phase-1
                 * lines sub*C2 + j of chunk r delivered to (d, r) */
                int64_t sub = pmod(d - s, G);
                for (int64_t r2 = 0; r2 < M; r2++) {
                    if (r2 == r) continue;
                    int64_t k = pmod(r - r2, M);
                    preds[np++] = (((k - 1) * G + d) * M + r2) * C1 + sub * C2 + j;
                }
            }
            if (s >= 1)  /* the same line received from (d - 1, r) one step earlier */
                preds[np++] = w->B2 + (((s - 1) * M + r) * G + pmod(d - 1, G)) * C2 + j;
            return np;
        }
        /* phase 3: intra-domain all-gather of chunk r, (d, r) -> (d, r+k) */
        int64_t y = x - w->B3;
        int64_t j = y % C1, q = y / C1, r = q % M;
        q /= M;
        int64_t d = q % G, k = q / G + 1;
        *src = (int32_t)(d * M + r); *dst = (int32_t)(d * M + (r + k) % M);
        int64_t sub = j / C2, jj = j % C2, dm = pmod(d - 1, G), s;
        if (sub == (d + 1) % G) {
            /* owned after reduce-scatter: the last reduce-scatter line from
             * (d - 1, r) combined with this node's domain-reduced copy */
            s = G - 2;
            for (int64_t r2 = 0; r2 < M; r2++) {
                if (r2 == r) continue;
                int64_t k2 = pmod(r - r2, M);
                preds[np++] = (((k2 - 1) * G + d) * M + r2) * C1 + j;
            }
        } else {
            s = G - 1 + pmod(d - sub, G);               /* arrives during all-gather */
        }
        preds[np++] = w->B2 + ((s * M + r) * G + dm) * C2 + jj;
        return np;
    }
    if (w->coll == COLL_DIRECT_AG || w->coll == COLL_DIRECT_RS) {
        /* id = ((k-1)*p + i)*C + j; rho(i) -> rho(i+k), no predecessors: in
         * reduce-scatter i sends its part of chunk i+k to that chunk's owner,
         * in all-gather its own chunk to every peer. */
        int64_t p = w->p, C = w->C;
        int64_t q = x / C, i = q % p, k = q / p + 1;
        *src = rho_of(w, i); *dst = rho_of(w, (i + k) % p);
        return 0;
    }
    if (w->coll == COLL_RHD) {
        int64_t p = w->p, C = w->C;
        int32_t K = w->K;
        if (x < rhd_ag_base(w, 0)) {
            int32_t j = 0;
            while (j + 1 < K && x >= rhd_rs_base(w, j + 1)) j++;
            int64_t y = x - rhd_rs_base(w, j), S = rhd_rs_len(w, j);
            int64_t i = y / S, q = rhd_rs_send_start(w, i, j) + y % S;
            *src = rho_of(w, i); *dst = rho_of(w, i ^ (p >> (j + 1)));
            for (int32_t j2 = 0; j2 < j; j2++)
                preds[np++] = w->dep == DEP_CHUNK ? -1 - ((int64_t)j2 * p + (i ^ (p >> (j2 + 1))))
                                                  : rhd_rs_arrival(w, i, j2, q);
            return np;
        }
        int32_t j = 0;
        while (j + 1 < K && x >= rhd_ag_base(w, j + 1)) j++;
        int64_t y = x - rhd_ag_base(w, j), A = rhd_ag_len(w, j);
        int64_t i = y / A, q = ((i >> j) << j) * C + y % A;
        *src = rho_of(w, i); *dst = rho_of(w, i ^ ((int64_t)1 << j));
        if (w->dep == DEP_CHUNK) {
            for (int32_t j2 = 0; j2 < K; j2++) preds[np++] = -1 - ((int64_t)j2 * p + (i ^ (p >> (j2 + 1))));
            for (int32_t h = 0; h < j; h++) preds[np++] = -1 - ((int64_t)(K + h) * p + (i ^ ((int64_t)1 << h)));
            return np;
        }
        int64_t c = q / C;
        if (c == i) {
            for (int32_t j2 = 0; j2 < K; j2++) preds[np++] = rhd_rs_arrival(w, i, j2, q);
        } else {
            int32_t h = 0;
            while ((c ^ i) >> (h + 1)) h++;   /* highest differing bit */
            preds[np++] = rhd_ag_arrival(w, i, h, q);
        }
        return np;
    }
    if (w->coll == COLL_DBT) {
        int64_t p = w->p, H = w->H;
        int64_t j = x % H, q = x / H, e = q % (p - 1);
        q /= p - 1;
        int t = (int)(q % 2), ph = (int)(q / 2);
        int64_t c = dbt_edge_part(e, t);
        int64_t vpos = dbt_parent_pos(dbt_pos(c, t, p), p);
        int64_t v = dbt_pos(vpos, t, p);
        *src = rho_of(w, ph == 0 ? c : v);
        *dst = rho_of(w, ph == 0 ? v : c);
        /* reduce: children of c; broadcast from the root: children of the root */
        int64_t gather = ph == 0 ? dbt_pos(c, t, p) : (vpos == 0 ? 0 : -1);
        if (gather >= 0) {
            for (int64_t u = 1; u < p; u++)
                if (dbt_parent_pos(u, p) == gather) {
                    int64_t mm = (int64_t)t * (p - 1) + dbt_edge(dbt_pos(u, t, p), t);
                    preds[np++] = w->dep == DEP_CHUNK ? -1 - mm : mm * H + j;
                }
        } else {
            int64_t mm = ((int64_t)2 + t) * (p - 1) + dbt_edge(v, t);
            preds[np++] = w->dep == DEP_CHUNK ? -1 - mm : mm * H + j;
        }
        return np;
    }
    /* all-to-all, linear shift: id = ((k-1)*E + i)*C + j; i -> i+k */
    {
        int64_t E = w->E, C = w->C;
        int64_t j = x % C, q = x / C, i = q % E, k = q / E + 1;
        (void)j;
        *src = (int32_t)i; *dst = (int32_t)((i + k) % E);
        return 0;
    }
}

/* Public decoder (tests use it to pin the expansion).  preds has room for
 * pred_cap entries; a line with more predecessors returns OR_ERR_SIZE with
 * *npred set to the count needed. */
int oracle_txn(int coll, uint64_t bytes, int32_t group, int32_t E, const int32_t *order, int32_t dep,
               int64_t x, int32_t *src, int32_t *dst, int32_t *npred, int64_t *preds, int32_t pred_cap,
               int64_t *T_out)
{
    work_t w;
    int rc = setup_work(&w, coll, bytes, group, E, order, dep);
    if (rc) return rc;
    if (T_out) *T_out = w.T;
    if (x < 0 || x >= w.T) return OR_ERR_INVALID_ARG;
    int64_t *all = malloc(sizeof(int64_t) * (size_t)pred_bound(&w));
    if (!all) return OR_ERR_OOM;
    int32_t np = decode(&w, x, src, dst, all);
    *npred = np;
    if (np <= pred_cap) memcpy(preds, all, sizeof(int64_t) * (size_t)np);
    else rc = OR_ERR_SIZE;
    free(all);
    return rc;
}

/* ------------------------------------------------------------ GPU programs
 * The injection side of the GPU model (Sec. 4.1.1 GPU instructions, 4.1.2
 * GPU operations, 4.4.2 compute unit, 4.4.3 wavefront requests, 4.4.4 loop
 * unrolling; the outstanding-request limit of Sec. 5.3).  A CU runs its
 * operations in list order:
 *   COPY    n lines from K >= 1 sources (space s_k, first line a_k) into one
 *           destination.  Unrolled by U, each group of gn <= U lines issues
 *           the loads of source 0 (lines j0 .. j0 + gn - 1), then of source
 *           1, ..., waits for all of their data, then issues the gn stores.
 *           K = 1 is memcpy; K > 1 is a reduce of the K inputs into the
 *           destination.  The arithmetic of the reduce is taken to cost no
 *           cycles (the paper gives no count); its effect is that the stores
 *           wait for every input.
 *   RELEASE one store to a semaphore line; a release completes the CU's
 *           earlier stores first (it waits for every earlier store of the
 *           CU), and it is a control message.
 *   ACQUIRE one load of a semaphore line (request and reply, both control
 *           messages).  The wavefront polls the semaphore until the release
 *           is visible; of those polls only the one that finds it released
 *           is simulated: its request leaves once the release of the same
 *           semaphore has arrived.  The CU's next request waits for the
 *           reply.
 *   load  = a request line (CU -> the channel of the source line) and a data
 *           line (that channel -> CU) that may leave once the request has
 *           arrived;
 *   store = one line (CU -> the channel of the destination line).
 * The CU's requests (load requests, stores, releases, acquire requests) are
 * its issued wavefront requests, in program order; request k may be issued
 * only once request k - W is done (its data or reply arrived / the store
 * arrived): at most W outstanding, retired in order.  Program order itself
 * comes from the network: all of a CU's requests leave through its one
 * link, in id order.  Line a of space s lives on channel
 * space_ch[s * n_ch + a mod n_ch].  Each semaphore (space, line) is released
 * by exactly one RELEASE; every ACQUIRE names a released semaphore.
 * Ids are step-major: for issue index k = 0, 1, ... and the CUs in ascending
 * endpoint order, a load or acquire takes two ids (request, then data or
 * reply), a store or release one.  Data lines and stores are data (class
 * 0); load requests and everything of a release or acquire are control
 * (class 1). */
enum { IN_LOAD = 0, IN_STORE = 1, IN_RELEASE = 2, IN_ACQUIRE = 3 };
typedef struct {
    int kind;
    int32_t chan;
    int64_t g0, gn;      /* store: the loads [g0, g0 + gn) of its group */
    int32_t sem_sp;      /* release / acquire: the semaphore */
    int64_t sem_ln;
} minstr_t;
typedef struct { int32_t sp; int64_t ln; int32_t q; int64_t k; } sem_t;

static int sem_cmp(const void *a, const void *b)
{
    const sem_t *x = a, *y = b;
    if (x->sp != y->sp) return x->sp < y->sp ? -1 : 1;
    return x->ln < y->ln ? -1 : x->ln > y->ln;
}

int oracle_gpu_ops(int64_t n_ops, const int32_t *kind, const int32_t *cu, const int64_t *src_ptr,
                   const int32_t *ssp, const int64_t *sline, const int32_t *dsp, const int64_t *dline,
                   const int64_t *nlines, int32_t n_spaces, int32_t n_ch, const int32_t *space_ch, int32_t U,
                   int32_t W, int64_t cap_txn, int64_t cap_pred, int32_t *src, int32_t *dst,
                   int64_t *pred_ptr, int64_t *pred_idx, uint8_t *cls, int64_t *T_out, int64_t *P_out)
{
    if (n_ops < 0 || n_ch < 1 || n_spaces < 1 || U < 1 || W < 1 || src_ptr[0] != 0) return OR_ERR_INVALID_ARG;
    #define CHAN(s, a) space_ch[(int64_t)(s) * n_ch + (a) % n_ch]
    for (int64_t o = 0; o < n_ops; o++) {
        int64_t K = src_ptr[o + 1] - src_ptr[o];
        if (K < 0 || dsp[o] < 0 || dsp[o] >= n_spaces || dline[o] < 0 || nlines[o] < 0) return OR_ERR_INVALID_ARG;
        if (kind[o] == 0) {
            if (K < 1) return OR_ERR_INVALID_ARG;
            for (int64_t s = src_ptr[o]; s < src_ptr[o + 1]; s++)
                if (ssp[s] < 0 || ssp[s] >= n_spaces || sline[s] < 0) return OR_ERR_INVALID_ARG;
        } else if (kind[o] == 1 || kind[o] == 2) {
            if (K != 0 || nlines[o] != 1) return OR_ERR_INVALID_ARG;
        } else {
            return OR_ERR_INVALID_ARG;
        }
    }
    /* the CUs, ascending */
    int32_t *cus = malloc(sizeof(int32_t) * (size_t)(n_ops > 0 ? n_ops : 1));
    int32_t ncu = 0;
    for (int64_t o = 0; o < n_ops; o++) {
        int found = 0;
        for (int32_t q = 0; q < ncu; q++) found |= cus[q] == cu[o];
        if (!found) cus[ncu++] = cu[o];
    }
    for (int32_t a = 1; a < ncu; a++)          /* insertion sort */
        for (int32_t b = a; b > 0 && cus[b - 1] > cus[b]; b--) { int32_t t = cus[b]; cus[b] = cus[b - 1]; cus[b - 1] = t; }
    /* each CU's program */
    minstr_t **prog = calloc((size_t)(ncu > 0 ? ncu : 1), sizeof(minstr_t *));
    int64_t *plen = calloc((size_t)(ncu > 0 ? ncu : 1), sizeof(int64_t));
    int64_t kmax = 0, nrel = 0;
    int rc = OR_OK;
    for (int32_t q = 0; q < ncu; q++) {
        int64_t len = 0;
        for (int64_t o = 0; o < n_ops; o++)
            if (cu[o] == cus[q]) len += kind[o] == 0 ? (src_ptr[o + 1] - src_ptr[o] + 1) * nlines[o] : 1;
        prog[q] = malloc(sizeof(minstr_t) * (size_t)(len > 0 ? len : 1));
        int64_t k = 0;
        for (int64_t o = 0; o < n_ops; o++) {
            if (cu[o] != cus[q]) continue;
            if (kind[o] != 0) {
                prog[q][k++] = (minstr_t){kind[o] == 1 ? IN_RELEASE : IN_ACQUIRE, CHAN(dsp[o], dline[o]), 0, 0,
                                          dsp[o], dline[o]};
                nrel += kind[o] == 1;
                continue;
            }
            for (int64_t j0 = 0; j0 < nlines[o]; j0 += U) {
                int64_t gn = nlines[o] - j0 < U ? nlines[o] - j0 : U;
                int64_t g0 = k;                       /* first load of the group */
                for (int64_t s = src_ptr[o]; s < src_ptr[o + 1]; s++)
                    for (int64_t j = j0; j < j0 + gn; j++)
                        prog[q][k++] = (minstr_t){IN_LOAD, CHAN(ssp[s], sline[s] + j), 0, 0, -1, -1};
                int64_t nload = k - g0;               /* K gn loads */
                for (int64_t j = j0; j < j0 + gn; j++)
                    prog[q][k++] = (minstr_t){IN_STORE, CHAN(dsp[o], dline[o] + j), g0, nload, -1, -1};
            }
        }
        plen[q] = k;
        if (k > kmax) kmax = k;
        for (int64_t j = 0; j < k; j++)
            if (prog[q][j].chan == cus[q]) rc = OR_ERR_INVALID_ARG;   /* a line to itself */
    }
    /* the releases, sorted by semaphore: one each */
    sem_t *rel = malloc(sizeof(sem_t) * (size_t)(nrel > 0 ? nrel : 1));
    int64_t nr = 0;
    for (int32_t q = 0; q < ncu; q++)
        for (int64_t k = 0; k < plen[q]; k++)
            if (prog[q][k].kind == IN_RELEASE) rel[nr++] = (sem_t){prog[q][k].sem_sp, prog[q][k].sem_ln, q, k};
    qsort(rel, (size_t)nr, sizeof(sem_t), sem_cmp);
    for (int64_t r = 1; r < nr; r++)
        if (sem_cmp(&rel[r - 1], &rel[r]) == 0) rc = OR_ERR_INVALID_ARG;
    /* ids: first id of every instruction */
    int64_t **id = calloc((size_t)(ncu > 0 ? ncu : 1), sizeof(int64_t *));
    for (int32_t q = 0; q < ncu; q++) id[q] = malloc(sizeof(int64_t) * (size_t)(plen[q] > 0 ? plen[q] : 1));
    #define TWO(in) ((in)->kind == IN_LOAD || (in)->kind == IN_ACQUIRE)
    int64_t T = 0;
    for (int64_t k = 0; k < kmax; k++)
        for (int32_t q = 0; q < ncu; q++)
            if (k < plen[q]) { id[q][k] = T; T += TWO(&prog[q][k]) ? 2 : 1; }
    /* the line that marks instruction k of CU q done */
    #define DONE(q, k) (TWO(&prog[q][k]) ? id[q][k] + 1 : id[q][k])
    int64_t P = 0;
    if (T >= (int64_t)0xFFFFFFFF) rc = OR_ERR_SIZE;
    int64_t *pl = malloc(sizeof(int64_t) * (size_t)(kmax + 2));   /* one line's predecessors */
    for (int64_t k = 0; k < kmax && rc == OR_OK; k++)
        for (int32_t q = 0; q < ncu && rc == OR_OK; q++) {
            if (k >= plen[q]) continue;
            const minstr_t *in = &prog[q][k];
            int64_t x = id[q][k];
            /* the issued line's predecessors, each once */
            int64_t np = 0;
            if (k >= W) pl[np++] = DONE(q, k - W);
            if (k >= 1 && prog[q][k - 1].kind == IN_ACQUIRE && !(k >= W && W == 1))
                pl[np++] = DONE(q, k - 1);               /* after an acquire: its reply */
            if (in->kind == IN_STORE)
                for (int64_t g = in->g0; g < in->g0 + in->gn; g++) pl[np++] = id[q][g] + 1;
            if (in->kind == IN_RELEASE)                  /* stores back to the previous release, inclusive */
                for (int64_t j = k - 1; j >= 0; j--) {
                    if (prog[q][j].kind == IN_STORE || prog[q][j].kind == IN_RELEASE) pl[np++] = id[q][j];
                    if (prog[q][j].kind == IN_RELEASE) break;
                }
            if (in->kind == IN_ACQUIRE) {
                sem_t key = {in->sem_sp, in->sem_ln, 0, 0};
                const sem_t *r = nr ? bsearch(&key, rel, (size_t)nr, sizeof(sem_t), sem_cmp) : NULL;
                if (!r) { rc = OR_ERR_INVALID_ARG; break; }
                pl[np++] = id[r->q][r->k];
            }
            int64_t need = np + (TWO(in) ? 1 : 0);
            if (cap_txn >= T && cap_pred >= P + need) {
                src[x] = cus[q];
                dst[x] = in->chan;
                if (cls) cls[x] = in->kind == IN_STORE ? 0 : 1;
                pred_ptr[x] = P;
                for (int64_t i = 0; i < np; i++) pred_idx[P + i] = pl[i];
                pred_ptr[x + 1] = P + np;
                if (TWO(in)) {       /* the data line or reply: waits for its request */
                    src[x + 1] = in->chan;
                    dst[x + 1] = cus[q];
                    if (cls) cls[x + 1] = in->kind == IN_LOAD ? 0 : 1;
                    pred_idx[P + np] = x;
                    pred_ptr[x + 2] = P + np + 1;
                }
            }
            P += need;
        }
    #undef DONE
    #undef TWO
    #undef CHAN
    if (T_out) *T_out = T;
    if (P_out) *P_out = P;
    for (int32_t q = 0; q < ncu; q++) { free(prog[q]); free(id[q]); }
    free(prog); free(id); free(plen); free(cus); free(rel); free(pl);
    return rc;
}

/* memcpy programs: every operation a COPY from one source. */
int oracle_memcpy(int64_t n_ops, const int32_t *cu, const int32_t *ssp, const int32_t *dsp,
                  const int64_t *sline, const int64_t *dline, const int64_t *nlines,
                  int32_t n_spaces, int32_t n_ch, const int32_t *space_ch, int32_t U, int32_t W,
                  int64_t cap_txn, int64_t cap_pred, int32_t *src, int32_t *dst,
                  int64_t *pred_ptr, int64_t *pred_idx, uint8_t *cls, int64_t *T_out, int64_t *P_out)
{
    if (n_ops < 0) return OR_ERR_INVALID_ARG;
    int32_t *kind = calloc((size_t)(n_ops > 0 ? n_ops : 1), sizeof(int32_t));
    int64_t *sp = malloc(sizeof(int64_t) * (size_t)(n_ops + 1));
    for (int64_t o = 0; o <= n_ops; o++) sp[o] = o;
    int rc = oracle_gpu_ops(n_ops, kind, cu, sp, ssp, sline, dsp, dline, nlines, n_spaces, n_ch, space_ch, U, W,
                            cap_txn, cap_pred, src, dst, pred_ptr, pred_idx, cls, T_out, P_out);
    free(kind);
    free(sp);
    return rc;
}

/* ------------------------------------------------------------- simulation */

/* FIFO entry: line id, first cycle it may leave, hop index of this link on
 * its path, and the path itself (start in the path table, hop count). */
typedef struct { uint32_t x; uint32_t ready; int32_t hop; int32_t plen; int64_t pp; } entry_t;

typedef struct {
    int32_t src;        /* source id: FIFO l -> l, stream of link f -> m + f */
    int32_t k;          /* position in the source's offer */
    uint32_t x;         /* line id */
    int32_t target;     /* link id, or SINK */
    int32_t port;       /* input port at the target's tail node */
    int32_t hop;        /* hop index of the target on the line's path */
    int32_t plen;       /* path of the line: hop count and start */
    int64_t pp;
    int granted;
    int departs;
} req_t;

typedef struct {
    uint64_t processed_cycles;
    uint64_t line_hops;
    double seconds;     /* event loop only */
} oracle_stats;

/* A decoded stream head: its predecessors and its path. */
typedef struct {
    uint32_t x;
    int32_t np;
    int64_t *preds;
    int64_t pp;
    int32_t plen;
} hcache_t;

static const hcache_t *head_info(hcache_t *c, int64_t *slot, const work_t *w, uint32_t x,
                                 const routes_t *rt, int32_t E)
{
    if (c->x == x) return c;
    int32_t s, d;
    if (w->coll == COLL_CUSTOM) {
        /* custom lists may have any number of predecessors */
        int64_t n = w->pptr[x + 1] - w->pptr[x];
        free(c->preds);
        c->preds = malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
        slot = c->preds;
    } else {
        c->preds = slot;
    }
    c->np = decode(w, x, &s, &d, slot);
    const int64_t q = routes_find(rt, (int64_t)s * E + d);
    c->pp = rt->ptr[q];
    c->plen = (int32_t)(rt->ptr[q + 1] - c->pp);
    c->x = x;
    return c;
}

/* rel(x) = max completion over predecessors; "never" while any is pending.
 * A whole-message predecessor is complete once all its lines are; its
 * completion is the latest of theirs (counted in chunk_done / chunk_max as
 * lines complete). */
static uint64_t release_of(const hcache_t *c, const uint32_t *completion, const int64_t *chunk_done,
                           const uint32_t *chunk_max, const work_t *w)
{
    uint64_t rel = 0;
    for (int32_t q = 0; q < c->np; q++) {
        int64_t p = c->preds[q];
        uint32_t v;
        if (p >= 0) {
            v = completion[p];
            if (v == NEVER) return UINT64_MAX;
        } else {
            if (chunk_done[-1 - p] < msg_len(w, -1 - p)) return UINT64_MAX;
            v = chunk_max[-1 - p];
        }
        if (v > rel) rel = v;
    }
    return rel;
}

static int key_less(const req_t *a, const req_t *b, int arb, int32_t rr, int32_t P)
{
    if ((arb & 1) == 0) return a->x < b->x;
    if (a->k != b->k) return a->k < b->k;
    return pmod(a->port - rr, P) < pmod(b->port - rr, P);
}

/*
 * Run one scenario.  Inputs: CSR topology (endpoints are nodes 0..E-1), the
 * per-link bw/lat/cap, the arbitration policy (0 lowest id, 1 round-robin,
 * plus 2 for class-fair arbitration, see below),
 * and either a collective (coll >= 0) or a custom transaction list
 * (coll == -1: n_txn lines with src/dst and predecessor CSR).  Outputs:
 * completion[T] (cycle, NEVER if not delivered), tx_lines[m], busy[m],
 * makespan.  max_cycles bounds the processed cycle (0 = 2^32 - 2).
 * check != 0 verifies the per-cycle and end-of-run invariants.
 * credit (NULL = all 1): per-link credit return delay D >= 1.  A slot that a
 * line frees by leaving link l at cycle t is seen free by l's arbiter from
 * cycle t + D on; D = 1 is the start-of-cycle snapshot of the base model.
 * (A flow-control variant: credits that travel back over the link take
 * time, which also gives a parallel simulation D cycles of lookahead.)
 * cls (NULL = all 0): class of every line of a custom list, 0 data, 1
 * control.  With arb & 2 (the fair arbitration of control and data messages
 * of Sec. 5.2) a link ranks its requests by class turns: starting with the
 * class its pointer names, each pick takes the lowest-key request of the
 * class whose turn it is among the sources' heads (requests with no earlier
 * request of the same source left; a source's lines are never reordered),
 * or of either class if that class has none, and the turn passes to the
 * other class.  After a cycle in which it appended lines, the pointer names
 * the class other than that of the last line appended.  Pointers start at
 * data.
 */
int oracle_simulate(int32_t n, int32_t E, const int32_t *row_ptr, const int32_t *col_idx,
                    const int32_t *bw, const int32_t *lat, const int32_t *cap, const int32_t *credit, int32_t arb,
                    int32_t coll, uint64_t bytes, int32_t group, const int32_t *order, int32_t dep,
                    int64_t n_txn, const int32_t *csrc, const int32_t *cdst, const uint8_t *cls,
                    const int64_t *pred_ptr, const int64_t *pred_idx,
                    uint64_t max_cycles, int32_t check,
                    uint32_t *completion, uint64_t *tx_lines, uint64_t *busy,
                    uint32_t *makespan, oracle_stats *stats)
{
    if (n < 1 || E < 1 || E > n || !row_ptr || !col_idx) return OR_ERR_INVALID_ARG;
    int32_t m = row_ptr[n];
    for (int32_t l = 0; l < m; l++) {
        if (bw[l] < 1 || lat[l] < 1 || cap[l] < 1 || (credit && credit[l] < 1)) return OR_ERR_TOPOLOGY;
        if (col_idx[l] < 0 || col_idx[l] >= n) return OR_ERR_TOPOLOGY;
    }
    for (int32_t u = 0; u < n; u++)
        for (int32_t l = row_ptr[u]; l < row_ptr[u + 1]; l++)
            if (col_idx[l] == u) return OR_ERR_TOPOLOGY;
    if (max_cycles == 0 || max_cycles > 0xFFFFFFFEull) max_cycles = 0xFFFFFFFEull;

    work_t w;
    int rc;
    if (coll == COLL_CUSTOM) {
        memset(&w, 0, sizeof(w));
        w.coll = COLL_CUSTOM; w.E = E; w.T = n_txn;
        w.csrc = csrc; w.cdst = cdst; w.pptr = pred_ptr; w.pidx = pred_idx;
        for (int64_t x = 0; x < n_txn; x++) {
            if (csrc[x] < 0 || csrc[x] >= E || cdst[x] < 0 || cdst[x] >= E || csrc[x] == cdst[x])
                return OR_ERR_INVALID_ARG;
            for (int64_t q = pred_ptr[x]; q < pred_ptr[x + 1]; q++)
                if (pred_idx[q] < 0 || pred_idx[q] >= n_txn) return OR_ERR_INVALID_ARG;
        }
    } else {
        rc = setup_work(&w, coll, bytes, group, E, order, dep);
        if (rc) return rc;
    }
    int64_t T = w.T;
    /* chunk mode: lines completed per message and the latest completion */
    int64_t nchunks = (w.dep == DEP_CHUNK && T > 0) ? msg_count(&w) : 0;
    int64_t *chunk_done = nchunks ? calloc((size_t)nchunks, sizeof(int64_t)) : NULL;
    uint32_t *chunk_max = nchunks ? calloc((size_t)nchunks, sizeof(uint32_t)) : NULL;

    /* routes of the pairs the workload uses */
    routes_t rt;
    memset(&rt, 0, sizeof(rt));
    int64_t *preds = malloc(sizeof(int64_t) * (size_t)pred_bound(&w));
    for (int64_t x = 0; x < T && rc == OR_OK; x++) {
        int32_t s, d;
        decode(&w, x, &s, &d, preds);
        rc = routes_add(&rt, (int64_t)s * E + d);
    }
    if (rc == OR_OK) rc = routes_trace(&rt, n, E, row_ptr, col_idx);
    if (rc) { routes_free(&rt); free(preds); free(chunk_done); free(chunk_max); return rc; }
    const int64_t *path_ptr = rt.ptr;
    const int32_t *path_link = rt.link;
    /* the path of flow (s, d): start and one past its end in path_link */
    #define PATH_LO(s, d) path_ptr[routes_find(&rt, (int64_t)(s) * E + (d))]
    #define PATH_HI(s, d) path_ptr[routes_find(&rt, (int64_t)(s) * E + (d)) + 1]

    /* input ports: in-links of v sorted by id, then the injection port */
    int32_t *port_of = malloc(sizeof(int32_t) * (size_t)(m + 1));
    int32_t *nports = calloc((size_t)n, sizeof(int32_t));
    int32_t *tail_of = malloc(sizeof(int32_t) * (size_t)(m + 1));
    for (int32_t u = 0; u < n; u++)
        for (int32_t l = row_ptr[u]; l < row_ptr[u + 1]; l++) tail_of[l] = u;
    for (int32_t l = 0; l < m; l++) port_of[l] = nports[col_idx[l]]++;
    for (int32_t v = 0; v < E; v++) nports[v]++;

    /* injection streams: per first link, the lines in ascending id */
    int64_t *s_ptr = calloc((size_t)m + 1, sizeof(int64_t));
    uint32_t *s_list = malloc(sizeof(uint32_t) * (size_t)(T > 0 ? T : 1));
    int64_t *s_cur = calloc((size_t)m, sizeof(int64_t));
    int64_t line_hops = 0;
    int32_t maxp = 1;   /* most predecessors of any line (sizes the head cache) */
    for (int64_t x = 0; x < T; x++) {
        int32_t s, d;
        int32_t np = decode(&w, x, &s, &d, preds);
        if (np > maxp) maxp = np;
        int64_t f0 = PATH_LO(s, d);
        if (PATH_HI(s, d) == f0) {   /* needed pair without a path */
            rc = OR_ERR_UNREACHABLE;
            break;
        }
        s_ptr[path_link[f0] + 1]++;
        line_hops += PATH_HI(s, d) - f0;
    }
    if (rc) {
        routes_free(&rt); free(port_of); free(nports); free(tail_of);
        free(s_ptr); free(s_list); free(s_cur); free(preds); free(chunk_done); free(chunk_max);
        return rc;
    }
    for (int32_t l = 0; l < m; l++) s_ptr[l + 1] += s_ptr[l];
    for (int64_t x = 0; x < T; x++) {
        int32_t s, d;
        decode(&w, x, &s, &d, preds);
        int32_t f = path_link[PATH_LO(s, d)];
        s_list[s_ptr[f] + s_cur[f]++] = (uint32_t)x;
    }
    memset(s_cur, 0, sizeof(int64_t) * (size_t)m);

    /* FIFOs */
    int64_t *q_off = malloc(sizeof(int64_t) * ((size_t)m + 1));
    q_off[0] = 0;
    for (int32_t l = 0; l < m; l++) q_off[l + 1] = q_off[l] + cap[l];
    entry_t *qbuf = malloc(sizeof(entry_t) * (size_t)(q_off[m] > 0 ? q_off[m] : 1));
    int32_t *qhead = calloc((size_t)m, sizeof(int32_t));
    int32_t *qocc = calloc((size_t)m, sizeof(int32_t));
    /* credits not yet returned: per link a queue (at most cap entries) of
     * (return cycle, count), and the total owed */
    uint64_t *owe_t = malloc(sizeof(uint64_t) * (size_t)(q_off[m] > 0 ? q_off[m] : 1));
    int32_t *owe_n = malloc(sizeof(int32_t) * (size_t)(q_off[m] > 0 ? q_off[m] : 1));
    int32_t *owe_h = calloc((size_t)m, sizeof(int32_t));    /* queue head */
    int32_t *owe_c = calloc((size_t)m, sizeof(int32_t));    /* queue length */
    int32_t *owed = calloc((size_t)m, sizeof(int32_t));     /* credits owed */
    int32_t *cptr = calloc((size_t)m, sizeof(int32_t));     /* class-fair pointer */
    int32_t *rr = calloc((size_t)m, sizeof(int32_t));

    int32_t bmax = 1;
    for (int32_t l = 0; l < m; l++) if (bw[l] > bmax) bmax = bw[l];
    size_t rcap = (size_t)2 * m * bmax + 1;
    req_t *reqs = malloc(sizeof(req_t) * rcap);
    int32_t *fair_a = malloc(sizeof(int32_t) * rcap);
    /* per-target request slots: at most (input ports of its tail) * bmax */
    int32_t *bucket_n = calloc((size_t)m, sizeof(int32_t));
    int64_t *bucket_off = malloc(sizeof(int64_t) * ((size_t)m + 1));
    bucket_off[0] = 0;
    for (int32_t f = 0; f < m; f++) bucket_off[f + 1] = bucket_off[f] + (int64_t)nports[tail_of[f]] * bmax;
    int32_t *bucket = malloc(sizeof(int32_t) * (size_t)(bucket_off[m] + 1));
    int32_t *touched = malloc(sizeof(int32_t) * ((size_t)m + 1));
    int32_t *active = malloc(sizeof(int32_t) * ((size_t)2 * m + 1));
    int32_t *src_first = malloc(sizeof(int32_t) * (size_t)2 * m);
    int32_t *src_cnt = calloc((size_t)2 * m, sizeof(int32_t));
    /* decoded stream heads (re-used while a head waits) */
    if (w.coll == COLL_CUSTOM) maxp = 1;  /* custom heads allocate their own */
    hcache_t *hcache = malloc(sizeof(hcache_t) * (size_t)m * bmax);
    int64_t *hpred = malloc(sizeof(int64_t) * (size_t)m * bmax * maxp);
    for (size_t i = 0; i < (size_t)m * bmax; i++) { hcache[i].x = NEVER; hcache[i].preds = NULL; }
    uint32_t *admit0 = check ? malloc(sizeof(uint32_t) * (size_t)(T > 0 ? T : 1)) : NULL;
    int32_t *adm_cnt = check ? calloc((size_t)m, sizeof(int32_t)) : NULL;

    for (int64_t x = 0; x < T; x++) completion[x] = NEVER;
    for (int32_t l = 0; l < m; l++) { tx_lines[l] = 0; busy[l] = 0; }
    if (admit0) for (int64_t x = 0; x < T; x++) admit0[x] = NEVER;

    int64_t remaining = T;
    uint64_t t = 0, processed = 0;
    rc = OR_OK;
    struct timespec t0, t1;
    clock_gettime(CLOCK_MONOTONIC, &t0);

    while (remaining > 0) {
        if (t > max_cycles) { rc = OR_ERR_MAX_CYCLES; break; }
        processed++;
        size_t nr = 0;
        int32_t ntouched = 0, nactive = 0;
        /* --- credits that are back by this cycle */
        for (int32_t l = 0; l < m; l++)
            while (owe_c[l] && owe_t[q_off[l] + owe_h[l]] <= t) {
                owed[l] -= owe_n[q_off[l] + owe_h[l]];
                owe_h[l] = (owe_h[l] + 1) % cap[l];
                owe_c[l]--;
            }
        /* --- requests from FIFOs */
        for (int32_t l = 0; l < m; l++) {
            if (qocc[l] == 0) continue;
            src_first[l] = (int32_t)nr;
            src_cnt[l] = 0;
            for (int32_t k = 0; k < bw[l] && k < qocc[l]; k++) {
                entry_t *e = &qbuf[q_off[l] + (qhead[l] + k) % cap[l]];
                if (e->ready > t) break;
                req_t *r = &reqs[nr++];
                r->src = l; r->k = k; r->x = e->x;
                r->hop = e->hop + 1;
                r->pp = e->pp; r->plen = e->plen;
                r->target = (r->hop < e->plen) ? path_link[e->pp + r->hop] : SINK;
                r->port = port_of[l];
                r->granted = 0; r->departs = 0;
                src_cnt[l]++;
            }
            if (src_cnt[l]) active[nactive++] = l;
        }
        /* --- requests from injection streams */
        for (int32_t f = 0; f < m; f++) {
            int32_t sid = m + f;
            int64_t len = s_ptr[f + 1] - s_ptr[f];
            if (s_cur[f] >= len) continue;
            src_first[sid] = (int32_t)nr;
            src_cnt[sid] = 0;
            for (int32_t k = 0; k < bw[f] && s_cur[f] + k < len; k++) {
                uint32_t x = s_list[s_ptr[f] + s_cur[f] + k];
                const hcache_t *hc = head_info(&hcache[(size_t)f * bmax + k], hpred + ((size_t)f * bmax + k) * maxp,
                                               &w, x, &rt, E);
                uint64_t rel = release_of(hc, completion, chunk_done, chunk_max, &w);
                if (rel > t) break;
                req_t *r = &reqs[nr++];
                r->src = sid; r->k = k; r->x = x;
                r->hop = 0; r->target = f;
                r->pp = hc->pp; r->plen = hc->plen;
                r->port = nports[tail_of[f]] - 1;
                r->granted = 0; r->departs = 0;
                src_cnt[sid]++;
            }
            if (src_cnt[sid]) active[nactive++] = sid;
        }
        /* --- grants: bucket requests by target link, order, grant a prefix */
        for (size_t i = 0; i < nr; i++) {
            if (reqs[i].target == SINK) { reqs[i].granted = 1; continue; }
            int32_t f = reqs[i].target;
            if (bucket_n[f] == 0) touched[ntouched++] = f;
            bucket[bucket_off[f] + bucket_n[f]++] = (int32_t)i;
        }
        for (int32_t ti = 0; ti < ntouched; ti++) {
            int32_t f = touched[ti];
            int32_t cnt = bucket_n[f];
            int32_t *bk = bucket + bucket_off[f];
            int32_t P = nports[tail_of[f]];
            for (int32_t a = 1; a < cnt; a++) {      /* insertion sort by key */
                int32_t v = bk[a], b = a - 1;
                while (b >= 0 && key_less(&reqs[v], &reqs[bk[b]], arb, rr[f], P)) {
                    bk[b + 1] = bk[b];
                    b--;
                }
                bk[b + 1] = v;
            }
            if (arb & 2) {
                /* class turns over the sources' heads: each pick takes, among
                 * the requests whose source has no earlier request left, the
                 * lowest key of the class whose turn it is (of either class if
                 * none), and hands the turn to the other class */
                int32_t turn = cptr[f];
                for (int32_t a = 0; a < cnt; a++) fair_a[a] = bk[a];   /* key order */
                for (int32_t pos = 0; pos < cnt; pos++) {
                    int32_t pick = -1, any = -1;
                    for (int32_t a = 0; a < cnt; a++) {
                        if (fair_a[a] < 0) continue;
                        const req_t *ra = &reqs[fair_a[a]];
                        int head = 1;
                        for (int32_t b2 = 0; b2 < cnt && head; b2++)
                            if (fair_a[b2] >= 0 && reqs[fair_a[b2]].src == ra->src && reqs[fair_a[b2]].k < ra->k) head = 0;
                        if (!head) continue;
                        if (any < 0) any = a;
                        if (pick < 0 && (cls ? cls[ra->x] : 0) == turn) pick = a;
                    }
                    if (pick < 0) pick = any;
                    bk[pos] = fair_a[pick];
                    turn = 1 - (cls ? cls[reqs[fair_a[pick]].x] : 0);
                    fair_a[pick] = -1;
                }
            }
            int32_t g = bw[f];
            if (cap[f] - qocc[f] - owed[f] < g) g = cap[f] - qocc[f] - owed[f];
            if (cnt < g) g = cnt;
            for (int32_t a = 0; a < g; a++) reqs[bk[a]].granted = 1;
        }
        /* --- departures: longest granted prefix of each source */
        int64_t departed = 0;
        for (int32_t ai = 0; ai < nactive; ai++) {
            int32_t sid = active[ai];
            for (int32_t k = 0; k < src_cnt[sid]; k++) {
                req_t *r = &reqs[src_first[sid] + k];
                if (!r->granted) break;
                r->departs = 1;
            }
        }
        /* --- enter target FIFOs in grant order */
        for (int32_t ti = 0; ti < ntouched; ti++) {
            int32_t f = touched[ti];
            int32_t cnt = bucket_n[f];
            bucket_n[f] = 0;
            int32_t *bk = bucket + bucket_off[f];
            int32_t entered = 0, last_port = -1, last_cls = 0;
            for (int32_t a = 0; a < cnt; a++) {
                req_t *r = &reqs[bk[a]];
                if (!r->departs) continue;
                entry_t *e = &qbuf[q_off[f] + (qhead[f] + qocc[f]) % cap[f]];
                e->x = r->x; e->ready = (uint32_t)(t + (uint64_t)lat[f]); e->hop = r->hop;
                e->pp = r->pp; e->plen = r->plen;
                qocc[f]++;
                entered++;
                last_port = r->port;
                last_cls = cls ? cls[r->x] : 0;
                if (admit0 && r->hop == 0) admit0[r->x] = (uint32_t)t;
            }
            if (entered) {
                tx_lines[f] += (uint64_t)entered;
                busy[f] += 1;
                if (arb & 1) rr[f] = (last_port + 1) % nports[tail_of[f]];
                if (arb & 2) cptr[f] = 1 - last_cls;
                if (check) {
                    if (entered > bw[f]) rc = OR_ERR_INVARIANT;         /* admissions <= b */
                    if (qocc[f] > cap[f]) rc = OR_ERR_INVARIANT;         /* occupancy <= cap */
                }
            }
        }
        /* --- pop sources, eject to sink */
        for (int32_t ai = 0; ai < nactive; ai++) {
            int32_t sid = active[ai];
            int32_t dep = 0;
            for (int32_t k = 0; k < src_cnt[sid]; k++) {
                req_t *r = &reqs[src_first[sid] + k];
                if (!r->departs) break;
                dep++;
                if (r->target == SINK) {
                    if (check && completion[r->x] != NEVER) rc = OR_ERR_INVARIANT;  /* once */
                    completion[r->x] = (uint32_t)(t + 1);
                    remaining--;
                    if (chunk_done) {
                        int64_t ch = msg_of(&w, (int64_t)r->x);
                        chunk_done[ch]++;
                        if ((uint32_t)(t + 1) > chunk_max[ch]) chunk_max[ch] = (uint32_t)(t + 1);
                    }
                }
            }
            if (!dep) continue;
            departed += dep;
            if (sid < m) {
                if (check && dep > bw[sid]) rc = OR_ERR_INVARIANT;       /* departures <= b */
                qhead[sid] = (qhead[sid] + dep) % cap[sid];
                qocc[sid] -= dep;
                if (credit && credit[sid] > 1) {   /* the freed slots come back later */
                    int32_t at = (owe_h[sid] + owe_c[sid]) % cap[sid];
                    owe_t[q_off[sid] + at] = t + (uint64_t)credit[sid];
                    owe_n[q_off[sid] + at] = (int32_t)dep;
                    owe_c[sid]++;
                    owed[sid] += (int32_t)dep;
                    if (check && qocc[sid] + owed[sid] > cap[sid]) rc = OR_ERR_INVARIANT;
                }
            } else {
                s_cur[sid - m] += dep;
            }
        }
        if (check) {
            /* FIFO order: ready times never decrease from head to tail */
            for (int32_t l = 0; l < m && rc == OR_OK; l++)
                for (int32_t k = 1; k < qocc[l]; k++) {
                    entry_t *a = &qbuf[q_off[l] + (qhead[l] + k - 1) % cap[l]];
                    entry_t *b = &qbuf[q_off[l] + (qhead[l] + k) % cap[l]];
                    if (a->ready > b->ready) { rc = OR_ERR_INVARIANT; break; }
                }
        }
        if (rc) break;
        if (remaining == 0) break;
        /* --- time advance */
        if (departed > 0) {
            t++;
            continue;
        }
        uint64_t next = UINT64_MAX;
        for (int32_t l = 0; l < m; l++)
            for (int32_t k = 0; k < bw[l] && k < qocc[l]; k++) {
                entry_t *e = &qbuf[q_off[l] + (qhead[l] + k) % cap[l]];
                if (e->ready > t) { if (e->ready < next) next = e->ready; break; }
            }
        for (int32_t f = 0; f < m; f++) {
            int64_t len = s_ptr[f + 1] - s_ptr[f];
            for (int32_t k = 0; k < bw[f] && s_cur[f] + k < len; k++) {
                uint32_t x = s_list[s_ptr[f] + s_cur[f] + k];
                const hcache_t *hc = head_info(&hcache[(size_t)f * bmax + k], hpred + ((size_t)f * bmax + k) * maxp,
                                               &w, x, &rt, E);
                uint64_t rel = release_of(hc, completion, chunk_done, chunk_max, &w);
                if (rel > t) { if (rel < next) next = rel; break; }
            }
        }
        for (int32_t l = 0; l < m; l++)   /* the next credit to come back */
            if (owe_c[l] && owe_t[q_off[l] + owe_h[l]] < next) next = owe_t[q_off[l] + owe_h[l]];
        if (next == UINT64_MAX) { rc = OR_ERR_DEADLOCK; break; }
        t = next;
    }
    clock_gettime(CLOCK_MONOTONIC, &t1);

    uint32_t mk = 0;
    for (int64_t x = 0; x < T; x++)
        if (completion[x] != NEVER && completion[x] > mk) mk = completion[x];
    *makespan = mk;

    if (check && rc == OR_OK) {
        /* sum of admissions equals the sum of path lengths */
        uint64_t sum = 0;
        for (int32_t l = 0; l < m; l++) {
            sum += tx_lines[l];
            if (busy[l] > tx_lines[l] || tx_lines[l] > (uint64_t)bw[l] * busy[l]) rc = OR_ERR_INVARIANT;
        }
        if (sum != (uint64_t)line_hops) rc = OR_ERR_INVARIANT;
        /* completion >= release + path latency + 1, release = max pred completion */
        for (int64_t x = 0; x < T && rc == OR_OK; x++) {
            int32_t s, d;
            int32_t np = decode(&w, x, &s, &d, preds);
            uint64_t rel = 0;
            for (int32_t q = 0; q < np; q++) {
                /* a whole-message predecessor: the latest of its lines */
                int64_t lo = preds[q] >= 0 ? preds[q] : msg_first(&w, -1 - preds[q]);
                int64_t hi = preds[q] >= 0 ? preds[q] + 1 : lo + msg_len(&w, -1 - preds[q]);
                for (int64_t y = lo; y < hi; y++)
                    if (completion[y] > rel) rel = completion[y];
            }
            uint64_t lsum = 0;
            for (int64_t q = PATH_LO(s, d); q < PATH_HI(s, d); q++)
                lsum += (uint64_t)lat[path_link[q]];
            if (admit0[x] < rel) rc = OR_ERR_INVARIANT;
            if ((uint64_t)completion[x] < rel + lsum + 1) rc = OR_ERR_INVARIANT;
        }
        /* a flow (same source and destination, so the same path) delivers its
         * lines in id order: no arbitration reorders a source's lines */
        uint32_t *flow_last = calloc((size_t)E * E, sizeof(uint32_t));
        for (int64_t x = 0; x < T && rc == OR_OK && flow_last; x++) {
            int32_t s, d;
            decode(&w, x, &s, &d, preds);
            uint32_t *fl = &flow_last[(int64_t)s * E + d];
            if (completion[x] < *fl) rc = OR_ERR_INVARIANT;
            *fl = completion[x];
        }
        free(flow_last);
    }

    if (stats) {
        stats->processed_cycles = processed;
        stats->line_hops = (uint64_t)line_hops;
        stats->seconds = (double)(t1.tv_sec - t0.tv_sec) + 1e-9 * (double)(t1.tv_nsec - t0.tv_nsec);
    }
    routes_free(&rt); free(port_of); free(nports); free(tail_of);
    free(s_ptr); free(s_list); free(s_cur); free(preds); free(q_off); free(qbuf);
    #undef PATH_LO
    #undef PATH_HI
    free(qhead); free(qocc); free(owe_t); free(owe_n); free(owe_h); free(owe_c); free(owed); free(cptr); free(rr);
    free(fair_a); free(reqs); free(bucket_n); free(bucket_off);
    free(bucket); free(touched); free(active);
    for (size_t i = 0; w.coll == COLL_CUSTOM && i < (size_t)m * bmax; i++) free(hcache[i].preds);
    free(hcache); free(hpred); free(src_first); free(src_cnt); free(admit0); free(adm_cnt);
    free(chunk_done); free(chunk_max);
    return rc;
}
