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
 *   greedy H_g       merge the two clusters sharing the most
 *                    weight, signature = intersection         (Section 6.2)
 *   spanning tree    OPT_free >= sum_i w(R_i) - max spanning tree
 *                    of w(R_i ∩ R_j)                  (Section 6.3, Thm 6)
 *   global orders    every request sorted by one chunk order (Section 7)
 *   DFS schedule     requests in lexicographic order of their sequences,
 *                    whole stream or per arrival window   (Thm 7, Sec. 8.1)
 *   radix cache      LRU-leaf eviction under a weight capacity (Section 8)
 *
 * Readings where the paper is silent (each one is listed with its reason in
 * the design notes of the repository):
 *   - both parts of a bipartition are non-empty; a singleton has M = 0;
 *   - the part that contains the lowest request of B is called B1, and among
 *     optimal bipartitions the one with the numerically smallest B1 is kept;
 *   - inside a node the newly common chunks are emitted in ascending id;
 *   - I(empty) = U, so W(empty) counts every chunk, even unrequested ones;
 *   - greedy ties: a cluster is named by its smallest request, the
 *     lexicographically smallest pair of names merges, the merge keeps the
 *     smaller name.
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

/* ===== Sections 6.2-6.3: agglomerative hierarchy, spanning-tree bound =====
 *
 * These functions take any m (requests are identified by index, not by a
 * bit of a mask) and work on sorted chunk lists.
 */

static int cmp_i32(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

/* Every request as an ascending chunk list at out[req_off[i] ..). Rejects
 * ids out of range and chunks repeated inside a request. */
static int sorted_requests(int m, int64_t n_chunks, const int64_t *req_off,
                           const int32_t *req_chunks, int32_t *out)
{
    for (int i = 0; i < m; ++i) {
        int64_t lo = req_off[i], hi = req_off[i + 1];
        if (hi < lo) return OR_E_INVALID;
        for (int64_t j = lo; j < hi; ++j) {
            if (req_chunks[j] < 0 || req_chunks[j] >= n_chunks) return OR_E_RANGE;
            out[j] = req_chunks[j];
        }
        qsort(out + lo, (size_t)(hi - lo), sizeof(int32_t), cmp_i32);
        for (int64_t j = lo + 1; j < hi; ++j)
            if (out[j] == out[j - 1]) return OR_E_DUP;
    }
    return OR_OK;
}

/* w(a ∩ b) of two ascending lists */
static int64_t inter_weight(const int32_t *a, int64_t na, const int32_t *b, int64_t nb,
                            const int64_t *w)
{
    int64_t i = 0, j = 0, s = 0;
    while (i < na && j < nb) {
        if (a[i] < b[j]) ++i;
        else if (a[i] > b[j]) ++j;
        else { s += w[a[i]]; ++i; ++j; }
    }
    return s;
}

/* a ∩ b of two ascending lists, written ascending to out; returns its size */
static int64_t inter_list(const int32_t *a, int64_t na, const int32_t *b, int64_t nb, int32_t *out)
{
    int64_t i = 0, j = 0, n = 0;
    while (i < na && j < nb) {
        if (a[i] < b[j]) ++i;
        else if (a[i] > b[j]) ++j;
        else { out[n++] = a[i]; ++i; ++j; }
    }
    return n;
}

/*
 * Pair weights P[i*m + j] = w(R_i ∩ R_j) for all requests i, j, so the
 * diagonal holds w(R_i). These are the edge weights of the spanning-tree
 * bound and the values of the greedy's first merge (Sections 6.2-6.3).
 */
int oracle_pair_weights(int m, int64_t n_chunks, const int64_t *w, const int64_t *req_off,
                        const int32_t *req_chunks, int64_t *P, int threads)
{
    if (m < 1 || n_chunks < 0) return OR_E_INVALID;
    int32_t *srt = (int32_t *)malloc(sizeof(int32_t) * (size_t)(req_off[m] > 0 ? req_off[m] : 1));
    if (!srt) return OR_E_NOMEM;
    int rc = sorted_requests(m, n_chunks, req_off, req_chunks, srt);
    if (rc == OR_OK) {
        if (threads > 0) omp_set_num_threads(threads);
#pragma omp parallel for schedule(dynamic, 4)
        for (int i = 0; i < m; ++i)
            for (int j = 0; j < m; ++j)
                P[(size_t)i * m + j] = inter_weight(srt + req_off[i], req_off[i + 1] - req_off[i],
                                                    srt + req_off[j], req_off[j + 1] - req_off[j], w);
    }
    free(srt);
    return rc;
}

/*
 * Agglomerative common-prefix hierarchy (Section 6.2; H_g of Theorem 6).
 * Every request starts as a cluster whose signature is R_i. While two or
 * more clusters remain, the pair whose signatures share the most weight is
 * merged, and the merged signature is the intersection of the two.
 *
 * Reading where the paper is silent (ties): a cluster is named by its
 * smallest request; among pairs of equal value the lexicographically
 * smallest pair of names (a, b), a < b, merges, and the merged cluster keeps
 * the name a.
 *
 * Plain: each step scans all active pairs for the maximum and recomputes
 * the values of the new cluster against every other one from the lists.
 *
 * Outputs for step t = 0 .. m-2: merge_a[t] < merge_b[t], gain[t] =
 * w(I(A) ∩ I(B)). node_parent[v] for the 2m-1 nodes: leaf i is node i, the
 * merge of step t creates node m + t, the root's parent is -1.
 * Returns SAV(H_g) = sum of the gains (Theorem 6), or a negative status.
 */
int64_t oracle_greedy(int m, int64_t n_chunks, const int64_t *w, const int64_t *req_off,
                      const int32_t *req_chunks, int32_t *merge_a, int32_t *merge_b,
                      int64_t *gain, int32_t *node_parent, int threads)
{
    if (m < 1 || n_chunks < 0) return OR_E_INVALID;
    int64_t nnz = req_off[m];
    int64_t sav = 0;
    int32_t *srt = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nnz > 0 ? nnz : 1));
    int32_t *tmp = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nnz > 0 ? nnz : 1));
    int64_t *len = (int64_t *)malloc(sizeof(int64_t) * (size_t)m);
    int64_t *V = (int64_t *)malloc(sizeof(int64_t) * (size_t)m * (size_t)m);
    unsigned char *active = (unsigned char *)malloc((size_t)m);
    int32_t *node_of = (int32_t *)malloc(sizeof(int32_t) * (size_t)m);
    int64_t *row_best = (int64_t *)malloc(sizeof(int64_t) * (size_t)m);
    int32_t *row_arg = (int32_t *)malloc(sizeof(int32_t) * (size_t)m);
    if (!srt || !tmp || !len || !V || !active || !node_of || !row_best || !row_arg) { sav = OR_E_NOMEM; goto done; }
    int rc = sorted_requests(m, n_chunks, req_off, req_chunks, srt);
    if (rc != OR_OK) { sav = rc; goto done; }
    if (threads > 0) omp_set_num_threads(threads);
    /* signature of cluster a lives at srt[req_off[a] ..), len[a] entries;
     * it only ever shrinks, so it stays in place */
    for (int a = 0; a < m; ++a) {
        len[a] = req_off[a + 1] - req_off[a];
        active[a] = 1;
        node_of[a] = a;
        node_parent[a] = -1;
    }
#pragma omp parallel for schedule(dynamic, 4)
    for (int a = 0; a < m; ++a)
        for (int b = 0; b < m; ++b)
            V[(size_t)a * m + b] = inter_weight(srt + req_off[a], len[a], srt + req_off[b], len[b], w);
    for (int t = 0; t + 1 < m; ++t) {
        /* the first maximum in (a, b) order is the lexicographically smallest */
#pragma omp parallel for schedule(dynamic, 16)
        for (int a = 0; a < m; ++a) {
            row_best[a] = -1; row_arg[a] = -1;
            if (!active[a]) continue;
            for (int b = a + 1; b < m; ++b)
                if (active[b] && V[(size_t)a * m + b] > row_best[a]) { row_best[a] = V[(size_t)a * m + b]; row_arg[a] = b; }
        }
        int ba = -1, bb = -1;
        int64_t bv = -1;
        for (int a = 0; a < m; ++a)
            if (row_arg[a] >= 0 && row_best[a] > bv) { bv = row_best[a]; ba = a; bb = row_arg[a]; }
        if (ba < 0) { sav = OR_E_INVALID; goto done; }
        merge_a[t] = ba; merge_b[t] = bb; gain[t] = bv;
        sav += bv;
        int64_t n = inter_list(srt + req_off[ba], len[ba], srt + req_off[bb], len[bb], tmp);
        memcpy(srt + req_off[ba], tmp, sizeof(int32_t) * (size_t)n);
        len[ba] = n;
        active[bb] = 0;
        node_parent[node_of[ba]] = m + t;
        node_parent[node_of[bb]] = m + t;
        node_parent[m + t] = -1;
        node_of[ba] = m + t;
#pragma omp parallel for schedule(dynamic, 16)
        for (int c = 0; c < m; ++c) {
            if (!active[c] || c == ba) continue;
            int64_t v = inter_weight(srt + req_off[ba], len[ba], srt + req_off[c], len[c], w);
            V[(size_t)ba * m + c] = v;
            V[(size_t)c * m + ba] = v;
        }
    }
done:
    free(srt); free(tmp); free(len); free(V); free(active); free(node_of); free(row_best); free(row_arg);
    return sav;
}

/* Nodes of an explicit hierarchy in an order where every child comes before
 * its parent; fills child lists. Returns the root or a negative status. */
static int tree_children(int m, int n_nodes, const int32_t *node_parent, int32_t *kid0, int32_t *kid1,
                         int32_t *order)
{
    int root = -1;
    for (int v = 0; v < n_nodes; ++v) { kid0[v] = -1; kid1[v] = -1; }
    for (int v = 0; v < n_nodes; ++v) {
        int p = node_parent[v];
        if (p < 0) { if (root >= 0) return OR_E_INVALID; root = v; continue; }
        if (p < m || p >= n_nodes) return OR_E_INVALID;
        if (kid0[p] < 0) kid0[p] = v;
        else if (kid1[p] < 0) kid1[p] = v;
        else return OR_E_INVALID;
    }
    if (root < 0) return OR_E_INVALID;
    /* post-order by an explicit stack */
    int32_t *stack = (int32_t *)malloc(sizeof(int32_t) * 2 * (size_t)n_nodes);
    unsigned char *seen = (unsigned char *)calloc((size_t)n_nodes, 1);
    if (!stack || !seen) { free(stack); free(seen); return OR_E_NOMEM; }
    int sp = 0, cnt = 0;
    stack[sp++] = root;
    while (sp > 0) {
        int v = stack[sp - 1];
        if (v >= m && !seen[v]) {
            seen[v] = 1;
            if (kid0[v] < 0 || kid1[v] < 0) { free(stack); free(seen); return OR_E_INVALID; }
            stack[sp++] = kid0[v];
            stack[sp++] = kid1[v];
        } else {
            --sp;
            order[cnt++] = v;
        }
    }
    free(stack); free(seen);
    if (cnt != n_nodes) return OR_E_INVALID;
    return root;
}

/* I(v) of every node of an explicit hierarchy, as ascending lists:
 * I(leaf i) = R_i, I(v) = I(kid0) ∩ I(kid1). list[v] is malloc'd. */
static int node_intersections(int m, int64_t n_chunks, const int64_t *req_off, const int32_t *req_chunks,
                              int n_nodes, const int32_t *node_parent, int32_t **list, int64_t *len,
                              int32_t *parent_out, int *root_out)
{
    int32_t *kid0 = (int32_t *)malloc(sizeof(int32_t) * (size_t)n_nodes);
    int32_t *kid1 = (int32_t *)malloc(sizeof(int32_t) * (size_t)n_nodes);
    int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)n_nodes);
    int64_t nnz = req_off[m];
    int32_t *srt = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nnz > 0 ? nnz : 1));
    int rc = OR_OK;
    if (!kid0 || !kid1 || !order || !srt) { rc = OR_E_NOMEM; goto done; }
    for (int v = 0; v < n_nodes; ++v) { list[v] = NULL; len[v] = 0; parent_out[v] = node_parent[v]; }
    rc = sorted_requests(m, n_chunks, req_off, req_chunks, srt);
    if (rc != OR_OK) goto done;
    rc = tree_children(m, n_nodes, node_parent, kid0, kid1, order);
    if (rc < 0) goto done;
    *root_out = rc;
    rc = OR_OK;
    for (int k = 0; k < n_nodes; ++k) {
        int v = order[k];
        if (v < m) {
            len[v] = req_off[v + 1] - req_off[v];
            list[v] = (int32_t *)malloc(sizeof(int32_t) * (size_t)(len[v] > 0 ? len[v] : 1));
            if (!list[v]) { rc = OR_E_NOMEM; goto done; }
            memcpy(list[v], srt + req_off[v], sizeof(int32_t) * (size_t)len[v]);
        } else {
            int a = kid0[v], b = kid1[v];
            int64_t cap = len[a] < len[b] ? len[a] : len[b];
            list[v] = (int32_t *)malloc(sizeof(int32_t) * (size_t)(cap > 0 ? cap : 1));
            if (!list[v]) { rc = OR_E_NOMEM; goto done; }
            len[v] = inter_list(list[a], len[a], list[b], len[b], list[v]);
        }
    }
done:
    free(kid0); free(kid1); free(order); free(srt);
    return rc;
}

/*
 * Layout read off an explicit hierarchy (proof of Theorem 1, "<=" half), for
 * any m: leaves 0 .. m-1 are the requests, node_parent[v] is the parent of
 * node v (-1 at the root) and internal nodes m .. n_nodes-1 have two
 * children each. Node v emits I(v) \ I(parent(v)) in ascending chunk id,
 * top-down; pi_i goes to order_chunks[req_off[i] ..).
 */
int oracle_tree_orders(int m, int64_t n_chunks, const int64_t *req_off, const int32_t *req_chunks,
                       int n_nodes, const int32_t *node_parent, int32_t *order_chunks)
{
    if (m < 1 || n_nodes != 2 * m - 1) return OR_E_INVALID;
    int32_t **list = (int32_t **)calloc((size_t)n_nodes, sizeof(int32_t *));
    int64_t *len = (int64_t *)malloc(sizeof(int64_t) * (size_t)n_nodes);
    int32_t *par = (int32_t *)malloc(sizeof(int32_t) * (size_t)n_nodes);
    int32_t *path = (int32_t *)malloc(sizeof(int32_t) * (size_t)n_nodes);
    int root = -1, rc = OR_OK;
    if (!list || !len || !par || !path) { rc = OR_E_NOMEM; goto done; }
    rc = node_intersections(m, n_chunks, req_off, req_chunks, n_nodes, node_parent, list, len, par, &root);
    if (rc != OR_OK) goto done;
    for (int i = 0; i < m; ++i) {
        int d = 0;
        for (int v = i; v >= 0; v = par[v]) path[d++] = v;     /* leaf .. root */
        int64_t pos = req_off[i];
        for (int k = d - 1; k >= 0; --k) {                      /* root .. leaf */
            int v = path[k], p = par[v];
            for (int64_t e = 0; e < len[v]; ++e) {
                int32_t x = list[v][e];
                int in_parent = 0;
                if (p >= 0)
                    for (int64_t f = 0; f < len[p]; ++f)
                        if (list[p][f] == x) { in_parent = 1; break; }
                if (in_parent) continue;
                if (pos >= req_off[i + 1]) { rc = OR_E_INVALID; goto done; }
                order_chunks[pos++] = x;
            }
        }
        if (pos != req_off[i + 1]) { rc = OR_E_INVALID; goto done; }
    }
done:
    if (list) for (int v = 0; v < n_nodes; ++v) free(list[v]);
    free(list); free(len); free(par); free(path);
    return rc;
}

/* SAV(H) = sum over internal nodes v of w(I(v)) for an explicit hierarchy
 * (Theorem 1, Eq. 3), computed from the node lists. */
int64_t oracle_tree_savings(int m, int64_t n_chunks, const int64_t *w, const int64_t *req_off,
                            const int32_t *req_chunks, int n_nodes, const int32_t *node_parent)
{
    if (m < 1 || n_nodes != 2 * m - 1) return OR_E_INVALID;
    int32_t **list = (int32_t **)calloc((size_t)n_nodes, sizeof(int32_t *));
    int64_t *len = (int64_t *)malloc(sizeof(int64_t) * (size_t)n_nodes);
    int32_t *par = (int32_t *)malloc(sizeof(int32_t) * (size_t)n_nodes);
    int root = -1;
    int64_t sav = 0;
    if (!list || !len || !par) { sav = OR_E_NOMEM; goto done; }
    int rc = node_intersections(m, n_chunks, req_off, req_chunks, n_nodes, node_parent, list, len, par, &root);
    if (rc != OR_OK) { sav = rc; goto done; }
    for (int v = m; v < n_nodes; ++v)
        for (int64_t e = 0; e < len[v]; ++e) sav += w[list[v][e]];
done:
    if (list) for (int v = 0; v < n_nodes; ++v) free(list[v]);
    free(list); free(len); free(par);
    return sav;
}

/*
 * Spanning-tree bound (Section 6.3, after Theorem 6): the savings of any
 * hierarchy are at most the weight of a maximum spanning tree of the
 * complete graph on the requests with edge weights P[i][j] = w(R_i ∩ R_j),
 * so OPT_free >= sum_i w(R_i) - MST. Prim's algorithm, O(m^2). Returns the
 * weight of a maximum spanning tree.
 */
int64_t oracle_max_spanning_tree(int m, const int64_t *P)
{
    if (m < 1) return OR_E_INVALID;
    int64_t *key = (int64_t *)malloc(sizeof(int64_t) * (size_t)m);
    unsigned char *in = (unsigned char *)calloc((size_t)m, 1);
    if (!key || !in) { free(key); free(in); return OR_E_NOMEM; }
    int64_t total = 0;
    for (int v = 0; v < m; ++v) key[v] = -1;
    key[0] = 0;
    for (int it = 0; it < m; ++it) {
        int u = -1;
        for (int v = 0; v < m; ++v)
            if (!in[v] && (u < 0 || key[v] > key[u])) u = v;
        in[u] = 1;
        total += key[u];
        for (int v = 0; v < m; ++v)
            if (!in[v] && v != u && P[(size_t)u * m + v] > key[v]) key[v] = P[(size_t)u * m + v];
    }
    free(key); free(in);
    return total;
}

/* ===== Sections 7-8: layouts, schedules and the radix cache ================
 *
 * A layout is a CSR of chunk sequences (seq_off[m+1], seqs[nnz]); request i's
 * sequence is seqs[seq_off[i] .. seq_off[i+1]).
 */

/* Global-order layout (Section 3.1, global orders; the popularity and id
 * orders of the Section 7 comparisons): every request is sorted by
 * rank[chunk] ascending. */
static const int32_t *g_rank_for_sort;
static int cmp_by_rank(const void *a, const void *b)
{
    int32_t x = g_rank_for_sort[*(const int32_t *)a], y = g_rank_for_sort[*(const int32_t *)b];
    return (x > y) - (x < y);
}

int oracle_global_order_layout(int m, int64_t n_chunks, const int64_t *req_off, const int32_t *req_chunks,
                               const int32_t *rank, int32_t *seqs)
{
    if (m < 1 || n_chunks < 0) return OR_E_INVALID;
    for (int i = 0; i < m; ++i) {
        for (int64_t j = req_off[i]; j < req_off[i + 1]; ++j) {
            if (req_chunks[j] < 0 || req_chunks[j] >= n_chunks) return OR_E_RANGE;
            seqs[j] = req_chunks[j];
        }
        g_rank_for_sort = rank;
        qsort(seqs + req_off[i], (size_t)(req_off[i + 1] - req_off[i]), sizeof(int32_t), cmp_by_rank);
    }
    return OR_OK;
}

/* Popularity order: chunks by the number of requests that hold them,
 * descending, ties by id ascending; rank[x] = position of x. */
int oracle_popularity_rank(int m, int64_t n_chunks, const int64_t *req_off, const int32_t *req_chunks, int32_t *rank)
{
    if (m < 1 || n_chunks < 0) return OR_E_INVALID;
    int64_t *cnt = (int64_t *)calloc((size_t)(n_chunks > 0 ? n_chunks : 1), sizeof(int64_t));
    if (!cnt) return OR_E_NOMEM;
    for (int64_t j = 0; j < req_off[m]; ++j) {
        if (req_chunks[j] < 0 || req_chunks[j] >= n_chunks) { free(cnt); return OR_E_RANGE; }
        cnt[req_chunks[j]]++;
    }
    /* counts from high to low, ids ascending inside each count */
    int64_t maxc = 0;
    for (int64_t x = 0; x < n_chunks; ++x) if (cnt[x] > maxc) maxc = cnt[x];
    int64_t pos = 0;
    for (int64_t c = maxc; c >= 0; --c)
        for (int64_t x = 0; x < n_chunks; ++x)
            if (cnt[x] == c) rank[x] = (int32_t)pos++;
    free(cnt);
    return OR_OK;
}

/* The DFS serving order of the layout's trie (Theorem 7): requests sorted
 * lexicographically by their sequences (a proper prefix first), equal
 * sequences by request index. */
static const int64_t *g_seq_off;
static const int32_t *g_seqs;
static int cmp_seq(const void *pa, const void *pb)
{
    int a = *(const int *)pa, b = *(const int *)pb;
    int64_t la = g_seq_off[a + 1] - g_seq_off[a], lb = g_seq_off[b + 1] - g_seq_off[b];
    const int32_t *sa = g_seqs + g_seq_off[a], *sb = g_seqs + g_seq_off[b];
    for (int64_t j = 0; j < la && j < lb; ++j)
        if (sa[j] != sb[j]) return sa[j] < sb[j] ? -1 : 1;
    if (la != lb) return la < lb ? -1 : 1;
    return (a > b) - (a < b);
}

int oracle_dfs_schedule(int m, const int64_t *seq_off, const int32_t *seqs, int32_t *order)
{
    if (m < 1) return OR_E_INVALID;
    for (int i = 0; i < m; ++i) order[i] = i;
    g_seq_off = seq_off; g_seqs = seqs;
    qsort(order, (size_t)m, sizeof(int32_t), cmp_seq);
    return OR_OK;
}

/* Windowed reordering (Section 8.1): the arrival stream 0, 1, ..., m-1 is cut
 * into consecutive windows of `window` requests and each window is served
 * in DFS order; window <= 0 means the whole stream. */
int oracle_window_schedule(int m, const int64_t *seq_off, const int32_t *seqs, int64_t window, int32_t *order)
{
    if (m < 1) return OR_E_INVALID;
    if (window <= 0 || window > m) window = m;
    g_seq_off = seq_off; g_seqs = seqs;
    for (int i = 0; i < m; ++i) order[i] = i;
    for (int64_t s = 0; s < m; s += window) {
        int64_t n = (s + window <= m) ? window : m - s;
        qsort(order + s, (size_t)n, sizeof(int32_t), cmp_seq);
    }
    return OR_OK;
}

/*
 * Radix cache with least-recently-used leaf eviction (Section 8): the
 * cached nodes of the layout's trie always include their ancestors. Serving
 * a request touches every node of its root-to-leaf path (all at the serving
 * time); the nodes not cached are computed, which costs their weight, and
 * inserted; then, while the cached weight exceeds `capacity`, the cached
 * leaf used least recently is evicted. The cache starts empty. Returns the
 * total computed weight (the prefill bill), or a negative status.
 * The trie is explicit; each eviction scans every node for the LRU leaf.
 */
int64_t oracle_lru_cache_cost(int m, int64_t n_chunks, const int64_t *w, const int64_t *seq_off,
                              const int32_t *seqs, const int32_t *order, int64_t capacity)
{
    if (m < 1 || n_chunks < 0 || capacity < 0) return OR_E_INVALID;
    int64_t total = seq_off[m];
    int64_t cap = total + 1;
    int32_t *chunk = (int32_t *)malloc(sizeof(int32_t) * (size_t)cap);
    int64_t *parent = (int64_t *)malloc(sizeof(int64_t) * (size_t)cap);
    int64_t *first_child = (int64_t *)malloc(sizeof(int64_t) * (size_t)cap);
    int64_t *next_sib = (int64_t *)malloc(sizeof(int64_t) * (size_t)cap);
    unsigned char *cached = (unsigned char *)calloc((size_t)cap, 1);
    int64_t *last = (int64_t *)malloc(sizeof(int64_t) * (size_t)cap);
    int64_t *kids_cached = (int64_t *)calloc((size_t)cap, sizeof(int64_t));
    int64_t *path = (int64_t *)malloc(sizeof(int64_t) * (size_t)cap);
    int64_t cost = 0;
    if (!chunk || !parent || !first_child || !next_sib || !cached || !last || !kids_cached || !path) { cost = OR_E_NOMEM; goto done; }
    /* the trie of all sequences (node 0 = root, never cached, weight 0) */
    int64_t nodes = 1;
    chunk[0] = -1; parent[0] = -1; first_child[0] = -1; next_sib[0] = -1;
    for (int i = 0; i < m; ++i) {
        int64_t cur = 0;
        for (int64_t j = seq_off[i]; j < seq_off[i + 1]; ++j) {
            int32_t x = seqs[j];
            if (x < 0 || x >= n_chunks) { cost = OR_E_RANGE; goto done; }
            int64_t c = first_child[cur];
            while (c >= 0 && chunk[c] != x) c = next_sib[c];
            if (c < 0) {
                c = nodes++;
                chunk[c] = x; parent[c] = cur; first_child[c] = -1;
                next_sib[c] = first_child[cur]; first_child[cur] = c;
            }
            cur = c;
        }
    }
    int64_t used = 0;
    for (int t = 0; t < m; ++t) {
        int i = order[t];
        if (i < 0 || i >= m) { cost = OR_E_INVALID; goto done; }
        /* the path of request i */
        int64_t len = 0, cur = 0;
        for (int64_t j = seq_off[i]; j < seq_off[i + 1]; ++j) {
            int64_t c = first_child[cur];
            while (chunk[c] != seqs[j]) c = next_sib[c];
            path[len++] = c;
            cur = c;
        }
        for (int64_t d = 0; d < len; ++d) {
            int64_t v = path[d];
            last[v] = t;
            if (!cached[v]) {
                cached[v] = 1;
                cost += w[chunk[v]];
                used += w[chunk[v]];
                if (parent[v] > 0) kids_cached[parent[v]]++;
            }
        }
        while (used > capacity) {
            int64_t best = -1;
            for (int64_t v = 1; v < nodes; ++v)
                if (cached[v] && kids_cached[v] == 0 && (best < 0 || last[v] < last[best])) best = v;
            if (best < 0) break;
            cached[best] = 0;
            used -= w[chunk[best]];
            if (parent[best] > 0) kids_cached[parent[best]]--;
        }
    }
done:
    free(chunk); free(parent); free(first_child); free(next_sib); free(cached); free(last); free(kids_cached); free(path);
    return cost;
}
