/*
 * oracle_sanitize.c -- drives every function of the CPU oracle
 * (oracle/mpt_oracle.c, compiled into this program) under AddressSanitizer
 * and UndefinedBehaviorSanitizer, on instances whose results the paper fixes:
 *
 *   - the complete 3-uniform family on four chunks (Theorem 4): OPT_free 8,
 *     every global order 9, the read-off layout abc, abd, cda, cdb;
 *   - the leave-one-out family L_n (Theorem 5, Eq. 5) for n = 1..12:
 *     OPT_free = n ceil(log2 n) - 2^ceil(log2 n) + n, every global order
 *     (n-1)(n+2)/2, and the greedy reaching the optimum on L_8;
 *   - seeded random instances: the read-off layout's trie cost, the
 *     hierarchy's Eq. (2) cost and OPT_free agree (Theorem 1); the spanning
 *     tree bound and the greedy's savings bracket the optimum (Section 6.3);
 *     capacity 0 bills sum_i w(R_i) and the DFS order at capacity
 *     max_i w(R_i) bills the trie cost (Theorem 7).
 *
 * Exit status 0 when every check holds; a sanitizer report aborts the run.
 * Test infrastructure only (the oracle is).
 */
#include "../../oracle/mpt_oracle.c"

#include <stdio.h>

static int failures = 0;
#define CHECK(cond)                                                       \
    do {                                                                  \
        if (!(cond)) {                                                    \
            fprintf(stderr, "FAIL %s:%d: %s\n", __FILE__, __LINE__, #cond); \
            ++failures;                                                   \
        }                                                                 \
    } while (0)

typedef struct {
    int m;
    int64_t u, nnz;
    int64_t *w, *off;
    int32_t *ch;
} inst_t;

static inst_t make(int m, int64_t u, int64_t nnz) {
    inst_t t;
    t.m = m;
    t.u = u;
    t.nnz = nnz;
    t.w = (int64_t *)calloc((size_t)(u > 0 ? u : 1), sizeof(int64_t));
    t.off = (int64_t *)calloc((size_t)m + 1, sizeof(int64_t));
    t.ch = (int32_t *)calloc((size_t)(nnz > 0 ? nnz : 1), sizeof(int32_t));
    return t;
}

static void release(inst_t *t) {
    free(t->w);
    free(t->off);
    free(t->ch);
}

static uint64_t lcg = 12345u;
static uint32_t rnd(uint32_t n) {
    lcg = lcg * 6364136223846793005ull + 1442695040888963407ull;
    return (uint32_t)((lcg >> 33) % n);
}

/* the whole exact path; returns OPT_free and fills the orders */
static int64_t solve(const inst_t *t, int32_t *orders, uint32_t **split_out) {
    const size_t n = (size_t)1 << t->m;
    int64_t *W = (int64_t *)malloc(n * sizeof(int64_t));
    int64_t *M = (int64_t *)malloc(n * sizeof(int64_t));
    int64_t *C = (int64_t *)malloc(n * sizeof(int64_t));
    uint32_t *split = (uint32_t *)malloc(n * sizeof(uint32_t));
    CHECK(oracle_intersection_weights(t->m, t->u, t->w, t->off, t->ch, W) == OR_OK);
    CHECK(oracle_exact_dp(t->m, W, M, split, 2) == OR_OK);
    CHECK(oracle_cost_table(t->m, W, M, C) == OR_OK);
    CHECK(oracle_orders(t->m, t->u, t->off, t->ch, split, orders) == OR_OK);
    const int64_t opt = C[n - 1];
    free(W);
    free(M);
    free(C);
    if (split_out) *split_out = split; else free(split);
    return opt;
}

static int64_t request_total(const inst_t *t) {
    int64_t s = 0;
    for (int64_t j = 0; j < t->nnz; ++j) s += t->w[t->ch[j]];
    return s;
}

static void k4(void) {
    static const int sets[4][3] = {{0, 1, 2}, {0, 1, 3}, {0, 2, 3}, {1, 2, 3}};
    inst_t t = make(4, 4, 12);
    for (int x = 0; x < 4; ++x) t.w[x] = 1;
    for (int i = 0; i < 4; ++i) {
        t.off[i + 1] = 3 * (i + 1);
        for (int j = 0; j < 3; ++j) t.ch[3 * i + j] = sets[i][j];
    }
    int32_t orders[12];
    uint32_t *split = NULL;
    CHECK(solve(&t, orders, &split) == 8);
    static const int expect[12] = {0, 1, 2, 0, 1, 3, 2, 3, 0, 2, 3, 1};   /* abc abd cda cdb */
    for (int j = 0; j < 12; ++j) CHECK(orders[j] == expect[j]);
    CHECK(oracle_trie_cost(4, 4, t.w, t.off, orders) == 8);
    CHECK(oracle_hierarchy_cost(4, 4, t.w, t.off, t.ch, split) == 8);
    int32_t rank[4], seqs[12];
    CHECK(oracle_popularity_rank(4, 4, t.off, t.ch, rank) == OR_OK);
    CHECK(oracle_global_order_layout(4, 4, t.off, t.ch, rank, seqs) == OR_OK);
    CHECK(oracle_trie_cost(4, 4, t.w, t.off, seqs) == 9);
    free(split);
    release(&t);
}

static void leave_one_out(void) {
    for (int n = 1; n <= 12; ++n) {
        inst_t t = make(n, n, (int64_t)n * (n - 1));
        for (int x = 0; x < n; ++x) t.w[x] = 1;
        int64_t at = 0;
        for (int i = 0; i < n; ++i) {
            for (int x = 0; x < n; ++x)
                if (x != i) t.ch[at++] = x;
            t.off[i + 1] = at;
        }
        int c = 0;
        while ((1 << c) < n) ++c;
        int32_t *orders = (int32_t *)malloc(sizeof(int32_t) * (size_t)(at > 0 ? at : 1));
        CHECK(solve(&t, orders, NULL) == (int64_t)n * c - (1 << c) + n);
        int32_t *rank = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
        int32_t *seqs = (int32_t *)malloc(sizeof(int32_t) * (size_t)(at > 0 ? at : 1));
        CHECK(oracle_popularity_rank(n, n, t.off, t.ch, rank) == OR_OK);
        CHECK(oracle_global_order_layout(n, n, t.off, t.ch, rank, seqs) == OR_OK);
        CHECK(oracle_trie_cost(n, n, t.w, t.off, seqs) == (int64_t)(n - 1) * (n + 2) / 2);
        if (n == 8) {
            int32_t ma[7], mb[7], parent[15];
            int64_t gain[7];
            const int64_t sav = oracle_greedy(n, n, t.w, t.off, t.ch, ma, mb, gain, parent, 2);
            CHECK(request_total(&t) - sav == (int64_t)n * c - (1 << c) + n);
            CHECK(oracle_tree_savings(n, n, t.w, t.off, t.ch, 2 * n - 1, parent) == sav);
        }
        free(orders);
        free(rank);
        free(seqs);
        release(&t);
    }
}

static void random_instances(void) {
    for (int trial = 0; trial < 6; ++trial) {
        const int m = 3 + trial;
        const int64_t u = 12 + 3 * trial;
        inst_t t = make(m, u, (int64_t)m * u);
        for (int64_t x = 0; x < u; ++x) t.w[x] = 1 + rnd(40);
        int64_t at = 0;
        for (int i = 0; i < m; ++i) {
            for (int64_t x = 0; x < u; ++x)
                if (rnd(3) == 0) t.ch[at++] = (int32_t)x;
            t.off[i + 1] = at;
        }
        t.nnz = at;
        int32_t *orders = (int32_t *)malloc(sizeof(int32_t) * (size_t)(at > 0 ? at : 1));
        uint32_t *split = NULL;
        const int64_t opt = solve(&t, orders, &split);
        CHECK(oracle_trie_cost(m, u, t.w, t.off, orders) == opt);
        CHECK(oracle_hierarchy_cost(m, u, t.w, t.off, t.ch, split) == opt);
        /* Section 6.3: spanning-tree lower bound and the greedy's half savings */
        int64_t *P = (int64_t *)malloc(sizeof(int64_t) * (size_t)m * m);
        CHECK(oracle_pair_weights(m, u, t.w, t.off, t.ch, P, 2) == OR_OK);
        const int64_t total = request_total(&t);
        CHECK(total - oracle_max_spanning_tree(m, P) <= opt);
        int32_t ma[16], mb[16], parent[32];
        int64_t gain[16];
        const int64_t sav = oracle_greedy(m, u, t.w, t.off, t.ch, ma, mb, gain, parent, 2);
        CHECK(sav <= total - opt && 2 * sav >= total - opt);
        int32_t *gorders = (int32_t *)malloc(sizeof(int32_t) * (size_t)(at > 0 ? at : 1));
        CHECK(oracle_tree_orders(m, u, t.off, t.ch, 2 * m - 1, parent, gorders) == OR_OK);
        CHECK(oracle_trie_cost(m, u, t.w, t.off, gorders) <= total - sav);
        /* Theorem 7: DFS order at one request's capacity bills the trie cost */
        int32_t order[16];
        int64_t wmax = 0;
        for (int i = 0; i < m; ++i) {
            int64_t s = 0;
            for (int64_t j = t.off[i]; j < t.off[i + 1]; ++j) s += t.w[t.ch[j]];
            if (s > wmax) wmax = s;
        }
        CHECK(oracle_dfs_schedule(m, t.off, orders, order) == OR_OK);
        CHECK(oracle_lru_cache_cost(m, u, t.w, t.off, orders, order, wmax) == opt);
        CHECK(oracle_window_schedule(m, t.off, orders, 2, order) == OR_OK);
        CHECK(oracle_lru_cache_cost(m, u, t.w, t.off, orders, order, 0) == total);
        free(P);
        free(gorders);
        free(orders);
        free(split);
        release(&t);
    }
}

int main(void) {
    k4();
    leave_one_out();
    random_instances();
    if (failures) fprintf(stderr, "%d checks failed\n", failures);
    else printf("oracle under sanitizers: all checks hold\n");
    return failures ? 1 : 0;
}
