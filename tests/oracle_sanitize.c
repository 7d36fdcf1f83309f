/*
 * Host-side sanitizer driver for the CPU oracle (test infrastructure).
 * Built with AddressSanitizer and UndefinedBehaviorSanitizer together with
 * oracle/oracle.c by tests/test_oracle_sanitize.py; it runs every
 * collective in both dependency modes and every arbitration policy, memcpy
 * programs, credit delays and the error paths with the invariant checks
 * on, and exits non-zero if a status is not the expected one.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

typedef struct { uint64_t processed_cycles, line_hops; double seconds; } oracle_stats;

int oracle_txn(int coll, uint64_t bytes, int32_t group, int32_t E, const int32_t *order, int32_t dep,
               int64_t x, int32_t *src, int32_t *dst, int32_t *npred, int64_t *preds, int32_t pred_cap,
               int64_t *T_out);
int oracle_simulate(int32_t n, int32_t E, const int32_t *row_ptr, const int32_t *col_idx,
                    const int32_t *bw, const int32_t *lat, const int32_t *cap, const int32_t *credit, int32_t arb,
                    int32_t coll, uint64_t bytes, int32_t group, const int32_t *order, int32_t dep,
                    int64_t n_txn, const int32_t *csrc, const int32_t *cdst, const uint8_t *cls,
                    const int64_t *pred_ptr, const int64_t *pred_idx, uint64_t max_cycles, int32_t check,
                    uint32_t *completion, uint64_t *tx_lines, uint64_t *busy, uint32_t *makespan,
                    oracle_stats *stats);
int oracle_memcpy(int64_t n_ops, const int32_t *cu, const int32_t *ssp, const int32_t *dsp,
                  const int64_t *sline, const int64_t *dline, const int64_t *nlines,
                  int32_t n_spaces, int32_t n_ch, const int32_t *space_ch, int32_t U, int32_t W,
                  int64_t cap_txn, int64_t cap_pred, int32_t *src, int32_t *dst,
                  int64_t *pred_ptr, int64_t *pred_idx, uint8_t *cls, int64_t *T_out, int64_t *P_out);

enum { P = 4, M_LINKS = P * (P - 1) };
static int32_t row_ptr[P + 1], col_idx[M_LINKS], bw[M_LINKS], lat[M_LINKS], cap[M_LINKS], credit[M_LINKS];
static int failures;

static void expect(int got, int want, const char *what, int a, int b)
{
    if (got != want) {
        fprintf(stderr, "%s (%d, %d): status %d, expected %d\n", what, a, b, got, want);
        failures++;
    }
}

static int run(int coll, int group, int dep, int arb, const int32_t *cr, uint64_t max_cycles)
{
    const uint64_t bytes = 128 * 4 * 6;
    int64_t T = 0;
    int32_t s, d, np;
    int64_t preds[64];
    int rc = oracle_txn(coll, bytes, group, P, NULL, dep, 0, &s, &d, &np, preds, 64, &T);
    if (rc) return rc;
    uint32_t *comp = malloc(sizeof(uint32_t) * (size_t)T), mk;
    uint64_t tx[M_LINKS], busy[M_LINKS];
    oracle_stats st;
    rc = oracle_simulate(P, P, row_ptr, col_idx, bw, lat, cap, cr, arb, coll, bytes, group, NULL, dep, 0, NULL,
                         NULL, NULL, NULL, NULL, max_cycles, 1, comp, tx, busy, &mk, &st);
    free(comp);
    return rc;
}

int main(void)
{
    int l = 0;
    for (int u = 0; u < P; u++) {   /* full mesh */
        row_ptr[u] = l;
        for (int v = 0; v < P; v++)
            if (v != u) { col_idx[l] = v; bw[l] = 1 + l % 2; lat[l] = 1 + l % 3; cap[l] = 2 + l % 3; credit[l] = 1 + l % 4; l++; }
    }
    row_ptr[P] = l;
    for (int coll = 0; coll <= 9; coll++)
        for (int dep = 0; dep <= 1; dep++)
            for (int arb = 0; arb <= 3; arb++) {
                int group = coll == 2 ? 2 : 0;
                int want = (coll == 2 && dep == 1) ? 1 : 0;   /* hierarchical: per line only */
                expect(run(coll, group, dep, arb, NULL, 0), want, "collective", coll, dep * 4 + arb);
                expect(run(coll, group, dep, arb, credit, 0), want, "collective+credit", coll, dep * 4 + arb);
            }
    expect(run(0, 0, 0, 0, NULL, 3), 8, "max_cycles", 0, 0);
    expect(run(8, 0, 0, 0, NULL, 0), 0, "rhd", 8, 0);

    /* memcpy: CU 0 copies 7 lines from space 0 to space 1 (channels 1..3) */
    int32_t cu[2] = {0, 0}, ssp[2] = {0, 1}, dsp[2] = {1, 0}, chans[6] = {1, 2, 3, 3, 2, 1};
    int64_t sl[2] = {0, 5}, dl[2] = {9, 0}, nl[2] = {7, 3}, T = 0, NP = 0;
    expect(oracle_memcpy(2, cu, ssp, dsp, sl, dl, nl, 2, 3, chans, 2, 3, 0, 0, NULL, NULL, NULL, NULL, NULL, &T,
                         &NP), 0, "memcpy sizes", 0, 0);
    int32_t *src = malloc(sizeof(int32_t) * (size_t)T), *dst = malloc(sizeof(int32_t) * (size_t)T);
    int64_t *pptr = malloc(sizeof(int64_t) * (size_t)(T + 1)), *pidx = malloc(sizeof(int64_t) * (size_t)(NP + 1));
    uint8_t *cls = malloc((size_t)T);
    expect(oracle_memcpy(2, cu, ssp, dsp, sl, dl, nl, 2, 3, chans, 2, 3, T, NP, src, dst, pptr, pidx, cls, &T, &NP),
           0, "memcpy", 0, 0);
    uint32_t *comp = malloc(sizeof(uint32_t) * (size_t)T), mk;
    uint64_t tx[M_LINKS], busy[M_LINKS];
    oracle_stats st;
    for (int arb = 0; arb <= 3; arb++)
        expect(oracle_simulate(P, P, row_ptr, col_idx, bw, lat, cap, credit, arb, -1, 0, 0, NULL, 0, T, src, dst, cls,
                               pptr, pidx, 0, 1, comp, tx, busy, &mk, &st), 0, "memcpy run", arb, 0);
    /* a cyclic dependency deadlocks */
    int32_t cs[2] = {0, 1}, cd[2] = {1, 0};
    int64_t cp[3] = {0, 1, 2}, ci[2] = {1, 0};
    expect(oracle_simulate(P, P, row_ptr, col_idx, bw, lat, cap, NULL, 0, -1, 0, 0, NULL, 0, 2, cs, cd, NULL, cp, ci,
                           0, 1, comp, tx, busy, &mk, &st), 7, "cyclic", 0, 0);
    free(src); free(dst); free(pptr); free(pidx); free(cls); free(comp);

    /* a custom DAG whose last line waits for all 5000 lines before it */
    {
        enum { N = 5001 };
        int32_t *s5 = malloc(sizeof(int32_t) * N), *d5 = malloc(sizeof(int32_t) * N);
        int64_t *p5 = malloc(sizeof(int64_t) * (N + 1)), *i5 = malloc(sizeof(int64_t) * (N - 1));
        uint32_t *c5 = malloc(sizeof(uint32_t) * N);
        for (int x = 0; x < N; x++) { s5[x] = x % P; d5[x] = (x + 1 + x / P % (P - 1)) % P; p5[x] = 0; }
        for (int x = 0; x < N - 1; x++) i5[x] = x;
        p5[N] = N - 1;
        for (int arb = 0; arb <= 1; arb++)
            expect(oracle_simulate(P, P, row_ptr, col_idx, bw, lat, cap, NULL, arb, -1, 0, 0, NULL, 0, N, s5, d5, NULL,
                                   p5, i5, 0, 1, c5, tx, busy, &mk, &st), 0, "fan-in 5000", arb, 0);
        free(s5); free(d5); free(p5); free(i5); free(c5);
    }
    /* a node with 5000 parallel out-links to one neighbour (route choice
     * among 5000 candidates) */
    {
        enum { K = 5000 };
        int32_t rp[3] = {0, K, K + 1}, *ci5 = malloc(sizeof(int32_t) * (K + 1));
        int32_t *b5 = malloc(sizeof(int32_t) * (K + 1)), *l5 = malloc(sizeof(int32_t) * (K + 1)),
                *k5 = malloc(sizeof(int32_t) * (K + 1));
        for (int l2 = 0; l2 <= K; l2++) { ci5[l2] = l2 < K ? 1 : 0; b5[l2] = 1; l5[l2] = 3; k5[l2] = 8; }
        uint64_t *tx5 = malloc(sizeof(uint64_t) * (K + 1)), *bu5 = malloc(sizeof(uint64_t) * (K + 1));
        uint32_t c5[2 * 64];
        expect(oracle_simulate(2, 2, rp, ci5, b5, l5, k5, NULL, 1, 3, 128 * 64, 0, NULL, 0, 0, NULL, NULL, NULL,
                               NULL, NULL, 0, 1, c5, tx5, bu5, &mk, &st), 0, "out-degree 5000", 0, 0);
        int32_t s, d, np;
        int64_t one[1], T5;
        /* direct all-reduce over 4100 endpoints: an all-gather line has 4099 predecessors */
        expect(oracle_txn(1, 128 * 4100, 0, 4100, NULL, 0, (int64_t)4099 * 4100, &s, &d, &np, one, 1, &T5), 4,
               "txn needs more room", np, 0);
        if (np != 4099) { fprintf(stderr, "txn predecessor count %d\n", np); failures++; }
        free(ci5); free(b5); free(l5); free(k5); free(tx5); free(bu5);
    }
    if (failures) return 1;
    printf("oracle sanitizer driver: ok\n");
    return 0;
}
