/*
 * mpt.h -- C ABI of libmpt.so, an exact solver for the Minimum Prefix Trie
 * with Free Permutations (MPT) problem on AMD Instinct MI355X (gfx950).
 *
 * Problem (Section 2 of "Prefix Sharing Is a Sorting Problem"): a universe
 * of n_chunks chunks with weights w(x) > 0 and m requests R_i (sets of chunk
 * ids). Choose one permutation pi_i of every R_i so that the trie of the m
 * resulting sequences has the smallest total weight of non-root nodes
 * (Eq. 1). By the structure theorem (Theorem 1, Eqs. 2-3) the optimum is
 *     OPT_free = sum_i w(R_i) - max_H sum_{v internal in H} w(I(v)),
 * a maximum over binary hierarchies H on the requests, with
 * I(B) = intersection of R_i over i in B. The solver computes it with the
 * O(3^m) subset DP of Section 3.1, in cost form:
 *     C({i}) = w(R_i),
 *     C(S)   = min over A (+) B = S, A holding the lowest request of S,
 *              both non-empty, of C(A) + C(B)  -  W(S),     W(S) = w(I(S)),
 * and reads the orders off the optimal hierarchy top-down (proof of
 * Theorem 1, "<=" half).
 *
 * Conventions shared by every entry point
 *  - Subsets of requests are m-bit masks: bit i set = request i is in the set.
 *  - Every array argument is DEVICE memory (HBM) owned by the caller; the
 *    library allocates nothing and keeps no pointer after a call returns.
 *  - `stream` is a hipStream_t (NULL = the null stream). All device work of a
 *    call is enqueued on it. Calls that return a host value synchronise it.
 *  - `workspace` is caller-owned device scratch of at least
 *    mpt_workspace_bytes(m, nnz) bytes, 256-byte aligned. Calls that share
 *    one workspace must not run concurrently.
 *  - Return value: MPT_OK (0) or a negative mpt_status. On error no output is
 *    guaranteed to be written; mpt_last_error() describes the failure for
 *    the calling thread. No C++ exception crosses this interface.
 *  - Integer ranges: 1 <= m <= MPT_MAX_M; 0 <= n_chunks <= MPT_MAX_CHUNKS;
 *    0 <= nnz <= 2^31 - 1 (request slots, the same for every call below);
 *    1 <= w(x) <= MPT_MAX_CHUNK_WEIGHT; sum_i w(R_i) < 2^61. These keep
 *    every W, C and pair sum inside int64.
 */
#ifndef MPT_H
#define MPT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MPT_MAX_M 30
#define MPT_MAX_CHUNKS (1LL << 30)
#define MPT_MAX_CHUNK_WEIGHT (1LL << 32)
/* C[0] after mpt_solve_exact: the empty set never takes part in a split. */
#define MPT_COST_SENTINEL (1LL << 62)

enum mpt_status {
    MPT_OK = 0,
    MPT_E_INVALID = -1,   /* bad size, null pointer, or req_off not a CSR offset array */
    MPT_E_RANGE = -2,     /* a chunk id outside [0, n_chunks) */
    MPT_E_DUP = -3,       /* a chunk repeated inside one request */
    MPT_E_WEIGHT = -4,    /* a weight <= 0 or > MPT_MAX_CHUNK_WEIGHT */
    MPT_E_OVERFLOW = -5,  /* sum_i w(R_i) >= 2^61 */
    MPT_E_WORKSPACE = -6, /* workspace missing, misaligned or too small */
    MPT_E_STATE = -7,     /* context call out of order (e.g. a solve before a build) */
    MPT_E_DEVICE = -8,    /* HIP runtime error (detail in mpt_last_error) */
    MPT_E_INTERNAL = -9   /* internal error (e.g. a host allocation failed) */
};

/* Bytes of device workspace that every entry point below needs for an
 * instance with m requests and nnz = req_off[m] request slots. */
size_t mpt_workspace_bytes(int m, int64_t nnz);

/*
 * Phase 1 -- intersection weights W(B) = w(I(B)) for all 2^m subsets B
 * (W(B) is the weight of the chunks shared by every request of B; Section 3,
 * proof of Theorem 1; I(empty) = U, so W(0) is the total weight of all
 * chunks). Also returns the demand sets S_x = { i : x in R_i } (Section 3).
 *
 *   chunk_w    [n_chunks]  int64 weights w(x)
 *   req_off    [m+1]       int64 CSR offsets, req_off[0] = 0, non-decreasing,
 *                          req_off[m] = nnz; request i is
 *                          req_chunks[req_off[i] .. req_off[i+1])
 *   req_chunks [nnz]       int32 chunk ids, distinct inside each request;
 *                          requests may be empty or equal to each other
 *   sig        [n_chunks]  out: uint32 S_x masks
 *   W          [2^m]       out: int64 table, 16-byte aligned
 * Validates the device inputs (MPT_E_INVALID / RANGE / DUP / WEIGHT /
 * OVERFLOW) and synchronises `stream` to report the result.
 */
int mpt_build_weights(int m, int64_t n_chunks, int64_t nnz,
                      const int64_t *chunk_w, const int64_t *req_off,
                      const int32_t *req_chunks, uint32_t *sig, int64_t *W,
                      void *workspace, size_t workspace_bytes, void *stream);

/*
 * Phase 2 -- the exact DP of Section 3.1 over all 2^m subsets, layer by
 * layer in |S|.
 *   W      [2^m]  int64 table from mpt_build_weights
 *   C      [2^m]  out: C(S) = OPT_free of the sub-instance {R_i : i in S};
 *                 C[0] = MPT_COST_SENTINEL
 *   split  [2^m]  out: for |S| >= 2 the optimal part A that holds the lowest
 *                 request of S; among optimal parts the numerically smallest;
 *                 0 for |S| <= 1. split encodes the optimal hierarchy: the
 *                 children of S are split[S] and S ^ split[S].
 *   opt_cost      HOST out, nullable: C(full set) = OPT_free (Theorem 1).
 *                 When non-null the call synchronises `stream`.
 * W, C and split need only the alignment of their element types.
 * For m >= 13 the call also synchronises `stream` once before its kernels,
 * to read sum_i W({i}) back: that total picks the key representation of the
 * packed kernels (32-bit keys for the cross and self pairs while it is below
 * 2^20 - 1, else exact doubles, uint64, or the plain kernels). Every
 * representation gives the same C and split.
 */
int mpt_solve_exact(int m, const int64_t *W, int64_t *C, uint32_t *split,
                    int64_t *opt_cost, void *workspace, size_t workspace_bytes,
                    void *stream);

/*
 * Phase 3 -- the layout read off the hierarchy (proof of Theorem 1): at node
 * B of the hierarchy each request below B emits I(B) \ I(parent(B)) in
 * ascending chunk id, with I(parent(root)) = empty. Chunk x of R_i is thus
 * emitted at the first node on request i's root-to-leaf path that is a
 * subset of S_x.
 *   req_off, req_chunks  the instance (as for mpt_build_weights)
 *   sig, split           outputs of the two calls above
 *   order_chunks [nnz]   out: pi_i at order_chunks[req_off[i] .. req_off[i+1])
 * Fails with MPT_E_INVALID (offsets, or a split table that does not encode
 * a hierarchy below the full set) or MPT_E_RANGE (a chunk id) before
 * anything is written; synchronises `stream` once to report those checks.
 */
int mpt_extract_orders(int m, int64_t n_chunks, int64_t nnz,
                       const int64_t *req_off, const int32_t *req_chunks,
                       const uint32_t *sig, const uint32_t *split,
                       int32_t *order_chunks, void *workspace,
                       size_t workspace_bytes, void *stream);

/*
 * mpt_solve_exact without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops, harnesses that
 * forbid hipMalloc). Same arguments, outputs and errors as mpt_solve_exact;
 * the scratch is a device array of MPT_NOALLOC_SCRATCH_BYTES inside the
 * library (one per device, kept until the process ends), enough for
 * m <= MPT_NOALLOC_MAX_M; larger m fails with MPT_E_INVALID. The call itself
 * allocates nothing. All calls on one device share that array: calls that
 * overlap on one device (other threads or streams) race and must be
 * serialised by the caller; consecutive calls on one stream are safe.
 */
#define MPT_NOALLOC_MAX_M 20
#define MPT_NOALLOC_SCRATCH_BYTES (37u << 20)
int mpt_solve_exact_noalloc(int m, const int64_t *W, int64_t *C, uint32_t *split, int64_t *opt_cost,
                            void *stream);

/*
 * ---- The context layer: the three phases of one instance on one device ----
 *
 * A context holds a device, a stream, a caller-owned workspace and the state
 * of one instance: created -> built (mpt_ctx_build_weights) -> solved
 * (mpt_ctx_solve_exact) -> extracted (mpt_ctx_extract_orders). Each phase
 * needs the one before it (else MPT_E_STATE); a new build starts over. A
 * failed build leaves the context created (no instance); a failed solve or
 * extraction leaves it where it was before that phase. Inputs are borrowed
 * for the duration of the build and copied into the workspace, which also
 * holds W, C, split, the demand sets and the orders; mpt_copy_table reads
 * them out. Compared with the stateless calls above, the solve needs no
 * read-back of sum_i w(R_i) (the build keeps it) and the extraction no
 * validation of a split table the library made, so the solve and the
 * extraction synchronise the stream only when they return host data.
 * A context serves one thread at a time; contexts are independent.
 */
typedef struct mpt_ctx mpt_ctx;

#define MPT_TABLE_W 0       /* int64 [2^m]      after a build */
#define MPT_TABLE_SIG 1     /* uint32 [n_chunks] after a build */
#define MPT_TABLE_C 2       /* int64 [2^m]      after a solve (C[0] = MPT_COST_SENTINEL) */
#define MPT_TABLE_SPLIT 3   /* uint32 [2^m]     after a solve */
#define MPT_TABLE_ORDERS 4  /* int32 [nnz]      after an extraction (CSR with req_off) */

/* Options (mpt_set_option). MPT_OPT_CHUNK_PAIRS: 0 (default) lets the
 * library plan how the cross pairs of each DP level are split over
 * workgroups; k >= 1 runs every level in chunks of at most k pairs (a level
 * whose pairs fit one chunk finishes its rows in the same kernel). Results
 * do not depend on it (it exists to test exactly that); it changes the
 * workspace size. */
#define MPT_OPT_CHUNK_PAIRS 1

/* MPT_OPT_WEIGHT_ROUTE: how a build computes W (Section 3.1's superset
 * sums). 0 (default) picks by size; MPT_ROUTE_LIST makes each 2^12-subset
 * tile scan the list of (S_x, w(x)) and write its part of W once (cost grows
 * with tiles x list length); MPT_ROUTE_DENSE scatters the list into W and
 * runs the superset zeta in place over the whole table (cost grows with
 * 2^m). The tables are the same on either route. */
#define MPT_OPT_WEIGHT_ROUTE 2
#define MPT_ROUTE_AUTO 0
#define MPT_ROUTE_LIST 1
#define MPT_ROUTE_DENSE 2

/* New context on HIP device hip_device, enqueueing on hip_stream (a
 * hipStream_t created on that device; NULL = its null stream). *out = NULL
 * on failure. Every context call makes hip_device current for its duration
 * and restores the caller's device. */
int mpt_create(mpt_ctx **out, int hip_device, void *hip_stream);

/* Frees the context (host memory only: the workspace is the caller's).
 * NULL-safe. Waits for nothing: the caller must not destroy a context whose
 * work is still in flight on its stream and then reuse the workspace. */
void mpt_destroy(mpt_ctx *ctx);

/* Sets an option (see MPT_OPT_*); MPT_E_INVALID for an unknown option or
 * value. Resets the context to created. */
int mpt_set_option(mpt_ctx *ctx, int option, int64_t value);

/* Device bytes the context needs for an instance of m requests, n_chunks
 * chunks and nnz request slots, with the context's options (ctx NULL:
 * default options). 0 for sizes out of range. */
size_t mpt_ctx_workspace_bytes(const mpt_ctx *ctx, int m, int64_t n_chunks, int64_t nnz);

/* Hands the context a caller-owned device workspace (256-byte aligned, on
 * the context's device, alive until the next mpt_set_workspace or
 * mpt_destroy). Its size is checked at each build. Resets the context to
 * created. dev_ptr NULL detaches it. */
int mpt_set_workspace(mpt_ctx *ctx, void *dev_ptr, size_t bytes);

/*
 * Phase 1 (as mpt_build_weights): copies the instance into the workspace,
 * validates it and builds W and the demand sets. chunk_w [n_chunks],
 * req_off [m+1] and req_chunks [nnz] may be host or device memory (copied
 * with hipMemcpyDefault). Synchronises the stream to report validation
 * errors. MPT_E_WORKSPACE if the workspace is missing or smaller than
 * mpt_ctx_workspace_bytes(ctx, m, n_chunks, nnz).
 */
int mpt_ctx_build_weights(mpt_ctx *ctx, int m, int64_t n_chunks, int64_t nnz, const int64_t *chunk_w,
                          const int64_t *req_off, const int32_t *req_chunks);

/*
 * Phase 2 (as mpt_solve_exact), after a build (else MPT_E_STATE).
 *   opt_cost    HOST out, nullable: OPT_free = C(full set) (Theorem 1)
 *   savings     HOST out, nullable: sum_i w(R_i) - OPT_free, the weight the
 *               optimal trie saves over no sharing (Eq. 3)
 *   split_host  HOST out, nullable: uint32 [2^m] split table
 * Synchronises the stream only if one of them is non-NULL.
 */
int mpt_ctx_solve_exact(mpt_ctx *ctx, int64_t *opt_cost, int64_t *savings, uint32_t *split_host);

/*
 * OPT_free and the savings of the last solve (HOST outs, nullable), after a
 * solve (else MPT_E_STATE): reads C(full set) back, synchronising the stream.
 * With this call a solve that returns no host data, the extraction and the
 * read-back run as one stream of work with a single synchronisation.
 */
int mpt_ctx_optimum(const mpt_ctx *ctx, int64_t *opt_cost, int64_t *savings);

/*
 * Phase 3 (as mpt_extract_orders), after a solve (else MPT_E_STATE).
 *   order_chunks_host  HOST out, nullable: int32 [nnz], pi_i at
 *                      [req_off[i], req_off[i+1])
 * Synchronises the stream only if order_chunks_host is non-NULL.
 */
int mpt_ctx_extract_orders(mpt_ctx *ctx, int32_t *order_chunks_host);

/*
 * Copies table `which` (MPT_TABLE_*) to host_dst, which holds `bytes` bytes
 * (at least the table's size, else MPT_E_INVALID); MPT_E_STATE if the phase
 * that writes the table has not run since the last build. Synchronises.
 */
int mpt_copy_table(const mpt_ctx *ctx, int which, void *host_dst, size_t bytes);

/* Device address and size of table `which` inside the workspace (valid
 * until the next build or workspace change), under the same state rules. */
int mpt_table_device(const mpt_ctx *ctx, int which, const void **dev_ptr, size_t *bytes);

/*
 * ---- Sections 6.2-6.3: heuristic and bound for large request counts ----
 *
 * These calls take any m in [1, MPT_GREEDY_MAX_M]; requests are identified
 * by index. Same conventions as above; they share one workspace of
 * mpt_greedy_workspace_bytes(m, n_chunks, nnz) bytes (about 8 m^2 + 44 nnz
 * + 8 n_chunks + 110 m bytes). Instances are validated as for
 * mpt_build_weights.
 */
#define MPT_GREEDY_MAX_M 16384

/* Bytes of device workspace for the calls below (0 for sizes out of range). */
size_t mpt_greedy_workspace_bytes(int m, int64_t n_chunks, int64_t nnz);

/*
 * Pair weights P[i*m + j] = w(R_i ∩ R_j) for all requests i, j (so
 * P[i*m + i] = w(R_i)): the edge weights of the spanning-tree bound and the
 * values of the greedy's first merge (Sections 6.2-6.3).
 *   P [m*m]         out: int64, row-major, device
 *   request_total   HOST out, nullable: sum_i w(R_i)
 * Cost: one write of P plus sum_x |S_x|^2 additions, in on-chip memory,
 * one per pair of requests sharing a chunk -- meant for sparse demand
 * (small |S_x|).
 * Synchronises `stream` (twice) to report validation errors.
 */
int mpt_pair_weights(int m, int64_t n_chunks, int64_t nnz, const int64_t *chunk_w,
                     const int64_t *req_off, const int32_t *req_chunks, int64_t *P,
                     int64_t *request_total, void *workspace, size_t workspace_bytes,
                     void *stream);

/*
 * Agglomerative common-prefix hierarchy H_g (Section 6.2; Theorem 6 shows
 * SAV(H_g) >= SAV* / 2). Every request starts as a cluster with signature
 * R_i; m-1 times, the two clusters whose signatures share the most weight
 * merge, and the merged signature is their intersection. A cluster is named
 * by its smallest request; among pairs of equal value the lexicographically
 * smallest pair of names (a, b), a < b, merges and keeps the name a.
 *   merge_a, merge_b [m-1]  out: int32 names of step t's pair, a < b
 *   gain [m-1]              out: int64 w(I(A) ∩ I(B)) of step t
 *                           (non-increasing, Theorem 6 part i)
 *   node_parent [2m-1]      out: int32 parent of each node (-1 at the root);
 *                           leaf i is node i, step t creates node m + t
 *   order_chunks [nnz]      out, nullable: the layout read off H_g (proof of
 *                           Theorem 1): top-down, node v emits
 *                           I(v) \ I(parent(v)) in ascending chunk id;
 *                           pi_i at order_chunks[req_off[i] ..)
 *   savings                 HOST out, nullable: SAV(H_g) = sum of the gains;
 *                           the layout costs at most sum_i w(R_i) - SAV(H_g)
 * The merges are found in parallel rounds (every mutually best pair of
 * clusters at once) and put in the sequence above afterwards; the outputs
 * are those of the one-merge-at-a-time procedure. Synchronises `stream`
 * once per eight rounds and before returning.
 */
int mpt_greedy_hierarchy(int m, int64_t n_chunks, int64_t nnz, const int64_t *chunk_w,
                         const int64_t *req_off, const int32_t *req_chunks,
                         int32_t *merge_a, int32_t *merge_b, int64_t *gain,
                         int32_t *node_parent, int32_t *order_chunks, int64_t *savings,
                         void *workspace, size_t workspace_bytes, void *stream);

/*
 * Spanning-tree lower bound (Section 6.3): every hierarchy's savings are at
 * most the weight of a maximum spanning tree of the complete graph on the
 * requests with edge weights P[i][j] (from mpt_pair_weights), so
 *     OPT_free >= sum_i P[i][i] - MST.
 *   P            [m*m] int64 pair weights, device
 *   mst_weight   HOST out: weight of a maximum spanning tree
 * Boruvka rounds over the whole device (ceil(log2 m) of them); uses
 * 256 + 32 m bytes of the workspace (rounded up per array); synchronises
 * `stream`.
 */
int mpt_spanning_tree_bound(int m, const int64_t *P, int64_t *mst_weight,
                            void *workspace, size_t workspace_bytes, void *stream);

/*
 * ---- Sections 7-8: layouts, serving schedules and the radix cache ----
 *
 * A layout is a CSR of chunk sequences: seq_off[m+1] (int64, device) and
 * seqs[nnz] (int32 chunk ids, device), e.g. the order_chunks output of
 * mpt_extract_orders or mpt_greedy_hierarchy with the request offsets.
 * Chunk ids must lie in [0, n_chunks); weights as above. The calls share one
 * workspace of mpt_layout_workspace_bytes(m, n_chunks, nnz, n_configs) bytes
 * (n_configs = 0 for the first two calls).
 */
#define MPT_LAYOUT_MAX_M (1 << 24)
#define MPT_CACHE_MAX_CONFIGS 256
#define MPT_ORDER_ID 0          /* chunk id ascending */
#define MPT_ORDER_POPULARITY 1  /* number of requests holding the chunk descending, id ascending */

size_t mpt_layout_workspace_bytes(int m, int64_t n_chunks, int64_t nnz, int n_configs);

/*
 * Global-order layout (Section 3.1's global orders; the id and popularity
 * baselines of Section 7): every request's chunks sorted by one order of the
 * chunks.
 *   req_off, req_chunks  the instance (as for mpt_build_weights)
 *   order_kind           MPT_ORDER_ID or MPT_ORDER_POPULARITY
 *   seqs [nnz]           out: the layout, CSR with req_off
 * Synchronises `stream` once to report validation errors.
 */
int mpt_global_order_layout(int m, int64_t n_chunks, int64_t nnz, const int64_t *req_off,
                            const int32_t *req_chunks, int order_kind, int32_t *seqs,
                            void *workspace, size_t workspace_bytes, void *stream);

/*
 * Trie cost of a layout (Eq. 1: the total weight of the non-root nodes of
 * the trie of the m sequences), and the DFS serving order of that trie
 * (Theorem 7): requests sorted lexicographically by their sequences, a
 * proper prefix first, equal sequences by request index.
 *   dfs_order [m]   out, nullable: request ids in DFS order
 *   trie_cost       HOST out
 * Synchronises `stream`.
 */
int mpt_layout_cost(int m, int64_t n_chunks, int64_t nnz, const int64_t *chunk_w,
                    const int64_t *seq_off, const int32_t *seqs, int32_t *dfs_order,
                    int64_t *trie_cost, void *workspace, size_t workspace_bytes, void *stream);

/*
 * Radix cache (Section 8): serving a request touches every node of its
 * root-to-leaf path in the layout's trie; the nodes not cached are computed
 * (their weight is billed) and inserted; then, while the cached weight
 * exceeds the capacity, the least-recently-used cached leaf is evicted
 * (cached nodes always include their ancestors). The cache starts empty.
 * Configuration c serves the requests in arrival order 0 .. m-1 cut into
 * windows of windows[c] requests, each window in DFS order (Section 8.1;
 * windows[c] <= 0 or >= m: the whole stream in DFS order, 1: arrival
 * order), with capacity capacities[c] (weight units; Theorem 7: in DFS
 * order max_i w(R_i) already bills exactly the trie cost).
 *   n_configs              1 .. MPT_CACHE_MAX_CONFIGS
 *   windows, capacities    HOST arrays [n_configs]
 *   costs                  HOST out [n_configs]: the billed weight
 *   trie_cost              HOST out, nullable: the unbounded-cache bill
 * Such a cache always holds the longest prefix of its recency stack that
 * fits (the stack property of LRU), so an access hits iff the distinct
 * weight accessed since its node's previous access, plus its own, fits.
 * Configurations with equal windows share one schedule and one pass that
 * prices all their capacities. Synchronises `stream`.
 */
int mpt_cache_simulate(int m, int64_t n_chunks, int64_t nnz, const int64_t *chunk_w,
                       const int64_t *seq_off, const int32_t *seqs, int n_configs,
                       const int64_t *windows, const int64_t *capacities, int64_t *costs,
                       int64_t *trie_cost, void *workspace, size_t workspace_bytes, void *stream);

/*
 * ---- Section 7.1: the quality-preserving pinned variant ----
 *
 * The first t chunks of every request in its input (relevance) order are
 * pinned at the end of its sequence, most relevant last; the rest (the free
 * part) is permuted. The construction: the distinct free sets are laid out
 * by the exact DP (mpt_build_weights, mpt_solve_exact, mpt_extract_orders)
 * or the greedy (mpt_greedy_hierarchy), every request takes its set's free
 * sequence, then its pinned suffix. Requests with equal free sets thereby
 * share one free sequence, and their suffixes can share trie nodes.
 */
size_t mpt_pinned_workspace_bytes(int m, int64_t nnz);

/*
 * Split into free sets and pinned suffixes.
 *   t                 pinned chunks per request (0: nothing pinned)
 *   dmap [m]          out: index of each request's free set among the
 *                     distinct sets, numbered in order of their first request
 *   free_off [m+1]    out: CSR offsets of the distinct free sets (the first
 *                     n_distinct + 1 entries are written)
 *   free_chunks [nnz] out: the distinct free sets, each in ascending chunk id
 *   n_distinct        HOST out: number of distinct free sets (>= 1)
 * Synchronises `stream`.
 */
int mpt_pinned_split(int m, int64_t n_chunks, int64_t nnz, const int64_t *req_off,
                     const int32_t *req_chunks, int t, int32_t *dmap, int64_t *free_off,
                     int32_t *free_chunks, int *n_distinct, void *workspace,
                     size_t workspace_bytes, void *stream);

/*
 * The layout: seqs[req_off[i] ..) = free sequence of set dmap[i] (from
 * free_layout, CSR with free_off, e.g. the orders of the exact or greedy
 * call on the distinct sets) followed by request i's pinned suffix.
 * Uses the first 256 bytes of the workspace; synchronises `stream`.
 */
int mpt_pinned_assemble(int m, int64_t nnz, const int64_t *req_off, const int32_t *req_chunks,
                        int t, const int32_t *dmap, int n_distinct, const int64_t *free_off,
                        const int32_t *free_layout, int32_t *seqs, void *workspace,
                        size_t workspace_bytes, void *stream);

/* Static text for a status code. */
const char *mpt_status_string(int status);

/* Detail of the calling thread's last failed call ("" if none). */
const char *mpt_last_error(void);

/*
 * Diagnostics: per-kernel device time with HIP events recorded on the
 * caller's stream around every launch. mpt_profile_begin() clears and
 * enables recording (process-wide); mpt_profile_begin_prefix(p) does the
 * same for the launches whose label starts with p only (the events add a few
 * microseconds between launches, so a timing run records only the kernels it
 * needs); mpt_profile_end() waits for the events,
 * fills up to max_entries rows, disables recording and returns the number of
 * distinct kernels seen (or a negative status).
 *   work: the algorithmic units the launches processed -- evaluated
 *         bipartitions for the DP kernels, bytes written for the W kernel.
 */
typedef struct mpt_profile_row {
    char kernel[48];
    int64_t launches;
    double total_ms;
    double work;
} mpt_profile_row;

int mpt_profile_begin(void);
int mpt_profile_begin_prefix(const char *prefix);
int mpt_profile_end(mpt_profile_row *rows, int max_entries);

#ifdef __cplusplus
}
#endif

#endif /* MPT_H */
