/*
 * CPU oracle for the exact MPT solver -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke entry point and the benchmark's CPU-baseline
 * leg may load or call this file's library. The product path never does, and
 * this file shares no code, header or table with it.
 *
 * It is a plain, slow and deliberately unoptimised restatement of
 * "Prefix Sharing Is a Sorting Problem":
 *
 *   demand sets      S_x = { i : x in R_i }                     (Section 3)
 *   intersections    I(B) = intersection of R_i over i in B,
 *                    W(B) = w(I(B)), I(empty) = U                (proof of Thm 1)
 *   exact DP         M(B) = w(I(B)) + max over B = B1 (+) B2 of
 *                    M(B1) + M(B2), M({i}) = 0                    (Section 3.1)
 *   optimum          OPT_free = sum_i w(R_i) - M([m])             (Thm 1, Eq. 3)
 *   layout           top-down: node B emits I(B) \ I(parent(B))  (proof of Thm 1)
 *   trie cost        sum over non-root trie nodes of w(chunk)     (Section 2, Eq. 1)
 *   hierarchy cost   sum_x w(x) t_x(H), t_x = number of maximal
 *                    clusters of H inside S_x                     (Thm 1, Eq. 2)
 *
 * Readings where the paper is silent (each one is listed with its reason in
 * the design notes of the repository):
 *   - both parts of a bipartition are non-empty; a singleton has M = 0;
 *   - the part that contains the lowest request of B is called B1, and among
 *     optimal bipartitions the one with the numerically smallest B1 is kept;
 *   - inside a node the newly common chunks are emitted in ascending id;
 *   - I(empty) = U, so W(empty) counts every chunk, even unrequested ones.
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC mpt_oracle.c -o libmpt_oracle.so
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

#define OR_OK 0
#define OR_E_INVALID (-1)
#define OR_E_RANGE (-2)
#define OR_E_DUP (-3)
#define OR_E_NOMEM (-4)

static int popcount32(uint32_t v) { return __builtin_popcount(v); }

/* S_x for every chunk x: bit i is set iff x is in R_i (Section 3). */
int oracle_demand_sets(int m, int64_t n_chunks, const int64_t *req_off,
                       const int32_t *req_chunks, uint32_t *sx)
{
    if (m < 1 || m > 30 || n_chunks < 0) return OR_E_INVALID;
    for (int64_t x = 0; x < n_chunks; ++x) sx[x] = 0;
    for (int i = 0; i < m; ++i) {
        if (req_off[i + 1] < req_off[i]) return OR_E_INVALID;
        for (int64_t j = req_off[i]; j < req_off[i + 1]; ++j) {
            int32_t x = req_chunks[j];
            if (x < 0 || x >= n_chunks) return OR_E_RANGE;
            if (sx[x] & (1u << i)) return OR_E_DUP;
            sx[x] |= 1u << i;
        }
    }
    return OR_OK;
}

/*
 * W(B) = w(I(B)) for every request subset B (2^m entries).
 * A chunk x lies in I(B) exactly when every request of B needs it, that is
 * when B is a subset of S_x. So each chunk adds w(x) to W(B) for every
 * subset B of S_x, which the loop below enumerates one by one.
 */
int oracle_intersection_weights(int m, int64_t n_chunks, const int64_t *w,
                                const int64_t *req_off, const int32_t *req_chunks,
                                int64_t *W)
{
    uint32_t *sx = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)(n_chunks > 0 ? n_chunks : 1));
    if (!sx) return OR_E_NOMEM;
    int rc = oracle_demand_sets(m, n_chunks, req_off, req_chunks, sx);
    if (rc != OR_OK) { free(sx); return rc; }
    uint64_t n = 1ull << m;
    for (uint64_t b = 0; b < n; ++b) W[b] = 0;
    for (int64_t x = 0; x < n_chunks; ++x) {
        uint32_t s = sx[x];
        uint32_t b = s;
        for (;;) {                       /* every subset b of S_x, S_x first */
            W[b] += w[x];
            if (b == 0) break;
            b = (b - 1) & s;
        }
    }
    free(sx);
    return OR_OK;
}

/*
 * The exact DP of Section 3.1 in its savings form:
 *   M({i}) = 0,  M(B) = W(B) + max over B = B1 (+) B2, both non-empty,
 *                               of M(B1) + M(B2).
 * Each unordered bipartition is visited once, as the B1 that holds the
 * lowest request of B. Ties keep the smallest B1; split[B] = that B1,
 * split = 0 for |B| <= 1. Subsets are handled in order of size, so every
 * part has its value before it is read; subsets of one size are independent
 * and are shared out over `threads` OpenMP threads.
 */
int oracle_exact_dp(int m, const int64_t *W, int64_t *M, uint32_t *split, int threads)
{
    if (m < 1 || m > 30) return OR_E_INVALID;
    if (threads < 1) threads = 1;
    int64_t n = (int64_t)1 << m;
    for (int64_t b = 0; b < n; ++b) { M[b] = 0; split[b] = 0; }
    for (int p = 2; p <= m; ++p) {
        #pragma omp parallel for schedule(dynamic, 16) num_threads(threads)
        for (int64_t bi = 0; bi < n; ++bi) {
            uint32_t B = (uint32_t)bi;
            if (popcount32(B) != p) continue;
            uint32_t low = B & (0u - B);
            uint32_t rest = B ^ low;
            int64_t best = INT64_MIN;
            uint32_t best_b1 = 0;
            /* proper subsets r of rest (rest itself would leave B2 empty) */
            uint32_t r = (rest - 1) & rest;
            for (;;) {
                uint32_t B1 = r | low;
                uint32_t B2 = B ^ B1;
                int64_t v = M[B1] + M[B2];
                if (v > best || (v == best && B1 < best_b1)) { best = v; best_b1 = B1; }
                if (r == 0) break;
                r = (r - 1) & rest;
            }
            M[B] = W[B] + best;
            split[B] = best_b1;
        }
    }
    return OR_OK;
}

/* Cost form of the same table: C(B) = sum_{i in B} w(R_i) - M(B), the
 * optimum of the sub-instance {R_i : i in B} by Eq. (3); w(R_i) = W({i}).
 * C(empty) = 0. */
int oracle_cost_table(int m, const int64_t *W, const int64_t *M, int64_t *C)
{
    if (m < 1 || m > 30) return OR_E_INVALID;
    int64_t n = (int64_t)1 << m;
    for (int64_t b = 0; b < n; ++b) {
        int64_t s = 0;
        for (int i = 0; i < m; ++i)
            if ((b >> i) & 1) s += W[(int64_t)1 << i];
        C[b] = s - M[b];
    }
    return OR_OK;
}

/* ----- hierarchy helpers ------------------------------------------------- */

/* Nodes of the binary hierarchy H encoded by split[] (children of B are
 * split[B] and B \ split[B]), listed root first with their parents.
 * Returns the node count (2m-1) or a negative status. */
static int hierarchy_nodes(int m, const uint32_t *split, uint32_t *node, uint32_t *parent)
{
    uint32_t full = (m == 32) ? 0xffffffffu : ((1u << m) - 1u);
    int cnt = 0, head = 0;
    node[cnt] = full; parent[cnt] = 0; ++cnt;
    while (head < cnt) {
        uint32_t B = node[head++];
        if (popcount32(B) < 2) continue;
        uint32_t A = split[B];
        uint32_t low = B & (0u - B);
        if ((A & ~B) || A == 0 || A == B || !(A & low)) return OR_E_INVALID;
        if (cnt + 2 > 2 * m) return OR_E_INVALID;
        node[cnt] = A; parent[cnt] = B; ++cnt;
        node[cnt] = B ^ A; parent[cnt] = B; ++cnt;
    }
    return cnt;
}

/*
 * Layout read off the hierarchy (proof of Theorem 1, "<=" half): at node B,
 * with I(parent(B)) already emitted, every request below B emits the chunks
 * of I(B) \ I(parent(B)), in ascending chunk id; I(parent(root)) = empty.
 * pi_i is written to order_chunks[req_off[i] .. req_off[i+1]).
 */
int oracle_orders(int m, int64_t n_chunks, const int64_t *req_off, const int32_t *req_chunks,
                  const uint32_t *split, int32_t *order_chunks)
{
    if (m < 1 || m > 30 || n_chunks < 0) return OR_E_INVALID;
    int rc = OR_OK;
    size_t u = (size_t)(n_chunks > 0 ? n_chunks : 1);
    unsigned char *member = (unsigned char *)calloc((size_t)m * u, 1);  /* member[i*u+x] = x in R_i */
    unsigned char *in_node = (unsigned char *)malloc(u);
    unsigned char *in_par = (unsigned char *)malloc(u);
    uint32_t *node = (uint32_t *)malloc(sizeof(uint32_t) * 2 * (size_t)m);
    uint32_t *parent = (uint32_t *)malloc(sizeof(uint32_t) * 2 * (size_t)m);
    int64_t *cursor = (int64_t *)malloc(sizeof(int64_t) * (size_t)m);
    if (!member || !in_node || !in_par || !node || !parent || !cursor) { rc = OR_E_NOMEM; goto done; }
    for (int i = 0; i < m; ++i) {
        cursor[i] = req_off[i];
        for (int64_t j = req_off[i]; j < req_off[i + 1]; ++j) {
            int32_t x = req_chunks[j];
            if (x < 0 || x >= n_chunks) { rc = OR_E_RANGE; goto done; }
            if (member[(size_t)i * u + (size_t)x]) { rc = OR_E_DUP; goto done; }
            member[(size_t)i * u + (size_t)x] = 1;
        }
    }
    int cnt = hierarchy_nodes(m, split, node, parent);
    if (cnt < 0) { rc = cnt; goto done; }
    /* nodes are listed parents-before-children, so the emission order along
     * every root-to-leaf path is preserved */
    for (int v = 0; v < cnt; ++v) {
        uint32_t B = node[v], P = parent[v];
        for (size_t x = 0; x < (size_t)n_chunks; ++x) {
            unsigned char a = 1, b = (P != 0);
            for (int i = 0; i < m; ++i) {
                if ((B >> i) & 1) a &= member[(size_t)i * u + x];
                if ((P >> i) & 1) b &= member[(size_t)i * u + x];
            }
            in_node[x] = a;   /* x in I(B) */
            in_par[x] = b;    /* x in I(parent(B)); empty above the root */
        }
        for (size_t x = 0; x < (size_t)n_chunks; ++x) {
            if (!in_node[x] || in_par[x]) continue;
            for (int i = 0; i < m; ++i) {
                if (!((B >> i) & 1)) continue;
                if (cursor[i] >= req_off[i + 1]) { rc = OR_E_INVALID; goto done; }
                order_chunks[cursor[i]++] = (int32_t)x;
            }
        }
    }
    for (int i = 0; i < m; ++i)
        if (cursor[i] != req_off[i + 1]) { rc = OR_E_INVALID; goto done; }
done:
    free(member); free(in_node); free(in_par); free(node); free(parent); free(cursor);
    return rc;
}

/*
 * Eq. (1): the cost of a layout is the total weight of the non-root nodes of
 * the trie of the m chunk sequences. The trie is built explicitly: each node
 * keeps its children in a singly linked list. Returns the cost, or a
 * negative status.
 */
int64_t oracle_trie_cost(int m, int64_t n_chunks, const int64_t *w,
                         const int64_t *seq_off, const int32_t *seqs)
{
    if (m < 0 || n_chunks < 0) return OR_E_INVALID;
    int64_t total = seq_off[m];
    int64_t cap = total + 1;
    int32_t *chunk = (int32_t *)malloc(sizeof(int32_t) * (size_t)cap);
    int64_t *first_child = (int64_t *)malloc(sizeof(int64_t) * (size_t)cap);
    int64_t *next_sib = (int64_t *)malloc(sizeof(int64_t) * (size_t)cap);
    if (!chunk || !first_child || !next_sib) { free(chunk); free(first_child); free(next_sib); return OR_E_NOMEM; }
    int64_t nodes = 1, cost = 0;
    chunk[0] = -1; first_child[0] = -1; next_sib[0] = -1;
    for (int i = 0; i < m; ++i) {
        int64_t cur = 0;
        for (int64_t j = seq_off[i]; j < seq_off[i + 1]; ++j) {
            int32_t x = seqs[j];
            if (x < 0 || x >= n_chunks) { cost = OR_E_RANGE; goto done; }
            int64_t c = first_child[cur];
            while (c >= 0 && chunk[c] != x) c = next_sib[c];
            if (c < 0) {
                c = nodes++;
                chunk[c] = x; first_child[c] = -1;
                next_sib[c] = first_child[cur]; first_child[cur] = c;
                cost += w[x];
            }
            cur = c;
        }
    }
done:
    free(chunk); free(first_child); free(next_sib);
    return cost;
}

/*
 * Eq. (2) evaluated for the hierarchy in split[]: sum_x w(x) t_x(H), where
 * t_x(H) counts the maximal clusters of H contained in S_x -- the nodes v
 * with v a subset of S_x whose parent is not (or that are the root).
 */
int64_t oracle_hierarchy_cost(int m, int64_t n_chunks, const int64_t *w,
                              const int64_t *req_off, const int32_t *req_chunks,
                              const uint32_t *split)
{
    if (m < 1 || m > 30 || n_chunks < 0) return OR_E_INVALID;
    uint32_t *sx = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)(n_chunks > 0 ? n_chunks : 1));
    uint32_t *node = (uint32_t *)malloc(sizeof(uint32_t) * 2 * (size_t)m);
    uint32_t *parent = (uint32_t *)malloc(sizeof(uint32_t) * 2 * (size_t)m);
    int64_t cost = 0;
    if (!sx || !node || !parent) { cost = OR_E_NOMEM; goto done; }
    int rc = oracle_demand_sets(m, n_chunks, req_off, req_chunks, sx);
    if (rc != OR_OK) { cost = rc; goto done; }
    int cnt = hierarchy_nodes(m, split, node, parent);
    if (cnt < 0) { cost = cnt; goto done; }
    for (int64_t x = 0; x < n_chunks; ++x) {
        int64_t t = 0;
        for (int v = 0; v < cnt; ++v) {
            int inside = (node[v] & ~sx[x]) == 0;
            int parent_inside = (v > 0) && ((parent[v] & ~sx[x]) == 0);
            if (inside && !parent_inside) ++t;
        }
        cost += w[x] * t;
    }
done:
    free(sx); free(node); free(parent);
    return cost;
}

int oracle_max_threads(void) { return omp_get_max_threads(); }
