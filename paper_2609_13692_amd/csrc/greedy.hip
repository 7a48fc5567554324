// libmpt.so, Sections 6.2-6.3 of "Prefix Sharing Is a Sorting Problem",
// for any number of requests up to MPT_GREEDY_MAX_M:
//   mpt_pair_weights         P[i][j] = w(R_i ∩ R_j)
//   mpt_greedy_hierarchy     the agglomerative common-prefix hierarchy H_g
//                            (Section 6.2, Theorem 6) and its layout
//   mpt_spanning_tree_bound  the maximum spanning tree of P, whence
//                            OPT_free >= sum_i w(R_i) - MST (Section 6.3)
//
// Requests are sorted once (a bitonic sort of (request, chunk) keys); the
// transposed (chunk, request) keys give the demand list S_x of every chunk.
// Pair weights are a scatter over the pairs of every demand list: request
// families of retrieval shape have small |S_x|, so this touches
// sum_x |S_x|^2 entries instead of a dense m x m x u contraction.
//
// The greedy's m-1 merges depend on each other, so one workgroup runs them
// all. Per merge it reduces the per-row best pairs to the global one,
// intersects the two signatures, scatters the new cluster's values through
// the demand lists of its signature (an LDS accumulator), and rescans only
// the rows whose best partner was one of the merged clusters (merge values
// never grow, Theorem 6 part i, so no other row's best can change).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>

#include "bitonic.h"
#include "common.h"
#include "mpt.h"

namespace {

using mptlib::align256;
using mptlib::fail;
using mptlib::grid_for;
using mptlib::LaunchScope;
using mptlib::kSortTile;
using mptlib::sort_keys;

constexpr int kWave = 64;
constexpr int kLoopThreads = 1024;           // the one workgroup of the merge loop
constexpr int kLoopWaves = kLoopThreads / kWave;

enum : uint32_t { GERR_INVALID = 1u, GERR_RANGE = 2u, GERR_DUP = 4u, GERR_WEIGHT = 8u, GERR_OVERFLOW = 16u };

// first 256 bytes of the workspace
struct GHeader {
    uint32_t err;
    uint32_t pad0;
    unsigned long long total;    // sum_i w(R_i), unsigned so it cannot wrap before the check
    int64_t pad[30];
};
static_assert(sizeof(GHeader) == 256, "header is one 256-byte block");

inline int64_t pow2_at_least(int64_t n) {
    int64_t p = 1;
    while (p < n) p <<= 1;
    return p;
}

struct GLayout {
    size_t keys1, keys2, sig, sig_len, dem, dem_off, V, best_v, best_p, active, node_of, dbuf, d_off, d_len,
        key, total;
    int64_t npad;
};

GLayout g_layout(int m, int64_t n_chunks, int64_t nnz) {
    GLayout L{};
    const size_t mm = (size_t)m;
    L.npad = std::max<int64_t>(pow2_at_least(std::max<int64_t>(nnz, 1)), kSortTile);
    size_t o = align256(sizeof(GHeader));
    auto take = [&](size_t bytes) { size_t at = o; o = align256(o + std::max<size_t>(bytes, 1)); return at; };
    L.keys1 = take(8 * (size_t)L.npad);
    L.keys2 = take(8 * (size_t)L.npad);
    L.sig = take(4 * (size_t)std::max<int64_t>(nnz, 1));
    L.sig_len = take(4 * mm);
    L.dem = take(4 * (size_t)std::max<int64_t>(nnz, 1));
    L.dem_off = take(8 * ((size_t)n_chunks + 1));
    L.V = take(8 * mm * mm);
    L.best_v = take(8 * mm);
    L.best_p = take(4 * mm);
    L.active = take(4 * mm);
    L.node_of = take(4 * mm);
    L.dbuf = take(4 * (size_t)std::max<int64_t>(nnz, 1));
    L.d_off = take(8 * (2 * mm));
    L.d_len = take(4 * (2 * mm));
    L.key = take(4 * mm);       // signature starts (int32) when they do not fit on chip
    L.total = o;
    return L;
}

// ---------------------------------------------------------------------------
// block helpers

// (value, index) pair order of a maximum with ties to the smallest index
__device__ inline bool better(int64_t v, int32_t i, int64_t ov, int32_t oi) {
    return v > ov || (v == ov && (unsigned)i < (unsigned)oi);
}

__device__ inline void wave_best(int64_t &v, int32_t &i) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const int64_t ov = __shfl_xor(v, off, kWave);
        const int32_t oi = __shfl_xor(i, off, kWave);
        if (better(ov, oi, v, i)) { v = ov; i = oi; }
    }
}

// best (value, index) over the workgroup, every thread gets the result. No
// closing barrier: the scratch (sv, si) must not be written again before
// some other barrier of the workgroup.
__device__ inline void block_best_once(int64_t &v, int32_t &i, int64_t *sv, int32_t *si) {
    wave_best(v, i);
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    if (lane == 0) { sv[wid] = v; si[wid] = i; }
    __syncthreads();
    v = sv[0]; i = si[0];
    for (int k = 1; k < (int)(blockDim.x / kWave); ++k)
        if (better(sv[k], si[k], v, i)) { v = sv[k]; i = si[k]; }
}


// exclusive prefix sum of one int per thread over the workgroup; returns
// the thread's offset, *total gets the sum
__device__ inline int block_scan(int x, int *total, int *sw) {
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    int incl = x;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int y = __shfl_up(incl, off, kWave);
        if (lane >= off) incl += y;
    }
    if (lane == kWave - 1) sw[wid] = incl;
    __syncthreads();
    int before = 0, all = 0;
    for (int k = 0; k < (int)(blockDim.x / kWave); ++k) {
        if (k < wid) before += sw[k];
        all += sw[k];
    }
    __syncthreads();
    *total = all;
    return before + incl - x;
}

// position of x in the ascending list a[0 .. n), or -1
__device__ inline int64_t find_sorted(const int32_t *a, int64_t n, int32_t x) {
    int64_t lo = 0, hi = n;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (a[mid] < x) lo = mid + 1; else hi = mid;
    }
    return (lo < n && a[lo] == x) ? lo : -1;
}

// ---------------------------------------------------------------------------
// validation and keys

__global__ void k_g_header(GHeader *h) {
    if (threadIdx.x == 0) { h->err = 0; h->total = 0; }
}

__global__ void k_g_check_offsets(int m, int64_t nnz, const int64_t *req_off, GHeader *h) {
    bool ok = true;
    for (int i = threadIdx.x; i < m; i += blockDim.x) ok = ok && req_off[i] <= req_off[i + 1];
    if (threadIdx.x == 0) ok = ok && req_off[0] == 0 && req_off[m] == nnz;
    if (!ok) atomicOr(&h->err, GERR_INVALID);
}

__global__ void k_g_check_weights(int64_t n_chunks, const int64_t *w, GHeader *h) {
    for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < n_chunks; x += (int64_t)gridDim.x * blockDim.x)
        if (w[x] <= 0 || w[x] > MPT_MAX_CHUNK_WEIGHT) atomicOr(&h->err, GERR_WEIGHT);
}

// (request, chunk) and (chunk, request) keys of every slot; keys past nnz
// are padding that sorts last
__global__ void k_g_keys(int m, int64_t n_chunks, int64_t nnz, int64_t npad, const int64_t *req_off,
                         const int32_t *req_chunks, const int64_t *w, uint64_t *keys1, uint64_t *keys2, GHeader *h) {
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < npad; j += (int64_t)gridDim.x * blockDim.x) {
        if (j >= nnz) { keys1[j] = ~0ull; keys2[j] = ~0ull; continue; }
        int lo = 0, hi = m - 1;                     // request of slot j: last i with req_off[i] <= j
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (req_off[mid] <= j) lo = mid; else hi = mid - 1;
        }
        const int32_t x = req_chunks[j];
        if (x < 0 || (int64_t)x >= n_chunks) {
            atomicOr(&h->err, GERR_RANGE);
            keys1[j] = ~0ull; keys2[j] = ~0ull;
            continue;
        }
        keys1[j] = ((uint64_t)lo << 32) | (uint32_t)x;
        keys2[j] = ((uint64_t)x << 32) | (uint32_t)lo;
        const int64_t wx = w[x];
        if (wx > 0 && wx <= MPT_MAX_CHUNK_WEIGHT) atomicAdd(&h->total, (unsigned long long)wx);
    }
}

// ---------------------------------------------------------------------------
// lists and pair weights

// sorted keys -> request lists (chunk ids ascending inside each request),
// demand lists (request ids ascending inside each chunk); a repeated chunk
// inside a request is two equal adjacent (request, chunk) keys
__global__ void k_g_lists(int m, int64_t nnz, const uint64_t *keys1, const uint64_t *keys2, int32_t *sig,
                          int32_t *sig_len, int32_t *dem, const int64_t *req_off, GHeader *h) {
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < nnz; j += (int64_t)gridDim.x * blockDim.x) {
        sig[j] = (int32_t)(keys1[j] & 0xffffffffu);
        dem[j] = (int32_t)(keys2[j] & 0xffffffffu);
        if (j > 0 && keys1[j] == keys1[j - 1]) atomicOr(&h->err, GERR_DUP);
    }
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < m; i += (int64_t)gridDim.x * blockDim.x)
        sig_len[i] = (int32_t)(req_off[i + 1] - req_off[i]);
}

// dem_off[x] = first slot of chunk x in the (chunk, request) order
__global__ void k_g_dem_off(int64_t n_chunks, int64_t nnz, const uint64_t *keys2, int64_t *dem_off) {
    for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x <= n_chunks; x += (int64_t)gridDim.x * blockDim.x) {
        const uint64_t key = (uint64_t)x << 32;
        int64_t lo = 0, hi = nnz;
        while (lo < hi) {
            const int64_t mid = (lo + hi) >> 1;
            if (keys2[mid] < key) lo = mid + 1; else hi = mid;
        }
        dem_off[x] = lo;
    }
}

__global__ void k_g_fill64(int64_t *p, int64_t n, int64_t v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = v;
}

// slot e = (chunk x, request a) adds w(x) to P[a][a] and to P[a][b], P[b][a]
// for every later request b of S_x; one wave per slot, so a long demand
// list is spread over 64 lanes
__global__ void k_g_pairs(int m, int64_t nnz, const uint64_t *keys2, const int32_t *dem, const int64_t *dem_off,
                          const int64_t *w, unsigned long long *P) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t waves = (int64_t)gridDim.x * blockDim.x / kWave;
    for (int64_t e = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave; e < nnz; e += waves) {
        const int64_t x = (int64_t)(keys2[e] >> 32);
        const unsigned long long wx = (unsigned long long)w[x];
        const size_t a = (size_t)dem[e];
        if (lane == 0) atomicAdd(&P[a * m + a], wx);
        const int64_t end = dem_off[x + 1];
        for (int64_t f = e + 1 + lane; f < end; f += kWave) {
            const size_t b = (size_t)dem[f];
            atomicAdd(&P[a * m + b], wx);
            atomicAdd(&P[b * m + a], wx);
        }
    }
}

// ---------------------------------------------------------------------------
// agglomerative hierarchy

// best partner of every row: max over d != c of V[c][d], ties to the
// smallest d; one wave per row
__global__ void k_g_row_best(int m, const int64_t *V, int64_t *best_v, int32_t *best_p) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
    if (row >= m) return;
    int64_t v = -1;
    int32_t p = -1;
    for (int d = lane; d < m; d += kWave)
        if (d != row && better(V[row * m + d], d, v, p)) { v = V[row * m + d]; p = d; }
    wave_best(v, p);
    if (lane == 0) { best_v[row] = v; best_p[row] = p; }
}

struct LoopArgs {
    int m;
    const int64_t *w;
    const int64_t *req_off;     // start of cluster a's signature
    int32_t *sig;               // signatures, ascending, shrinking in place
    int32_t *sig_len;
    int32_t *sig_at;            // req_off as int32 (workspace copy, used when m > kMetaCap)
    int64_t *V;                 // V[a][c] = w(I(a) ∩ I(c)) for live a, c
    int64_t *best_v;
    int32_t *best_p;
    int32_t *node_of;           // tree node of live cluster a
    int32_t *dbuf;              // D(v) = I(v) \ I(parent(v)), packed
    int64_t dcap;               // entries of dbuf (nnz: the D lists never need more)
    int64_t *d_off;
    int32_t *d_len;
    int32_t *merge_a, *merge_b;
    int64_t *gain;
    int32_t *node_parent;
    GHeader *h;
};

// The columns of the candidate pass and of the new row are owned by the
// waves other than wave 0, which intersects the signatures meanwhile.
constexpr int kColThreads = kLoopThreads - kWave;
constexpr int kColsPerThread = (MPT_GREEDY_MAX_M + kColThreads - 1) / kColThreads;
static_assert(kColsPerThread <= 32, "the column flags of a thread fit 32 bits");
constexpr int kScCap = 2048;                                        // I(C) kept in LDS up to this size
constexpr int kSigCap = 1024;                                       // I(A), I(B) copied to LDS up to this size
constexpr int kMetaCap = 4096;                                      // per-cluster state in LDS up to this m
constexpr int kCandCap = 2048;                                      // candidate columns listed in LDS per merge
constexpr int kRescParts = 4;                                       // waves per rescanned row
constexpr int kRescRows = kLoopWaves / kRescParts;                  // rows rescanned together

__device__ inline uint64_t lanes_below(int lane) { return (1ull << lane) - 1ull; }

// w(I(C) ∩ list) for an ascending list: I(C) and the weights of its
// chunks in LDS; the list is read 8 entries at a time so that its loads
// overlap
__device__ inline int64_t inter_weight_lds(const int32_t *ic, const int64_t *icw, int64_t n_ic, const int32_t *list,
                                           int64_t n) {
    int64_t s = 0;
    constexpr int U = 8;
    for (int64_t j0 = 0; j0 < n; j0 += U) {
        int32_t y[U];
#pragma unroll
        for (int u = 0; u < U; ++u) y[u] = j0 + u < n ? list[j0 + u] : -1;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (y[u] < 0) continue;
            const int64_t pos = find_sorted(ic, n_ic, y[u]);
            if (pos >= 0) s += icw[pos];
        }
    }
    return s;
}

// the same with I(C) in global memory (too long for the LDS copy)
__device__ inline int64_t inter_weight_global(const int32_t *ic, int64_t n_ic, const int32_t *list, int64_t n,
                                              const int64_t *w) {
    int64_t s = 0;
    for (int64_t j = 0; j < n; ++j) {
        const int32_t y = list[j];
        if (find_sorted(ic, n_ic, y) >= 0) s += w[y];
    }
    return s;
}

// Each step: (1) the pair to merge from the threads' cached row bests;
// (2) candidate columns c, where both V[a][c] and V[b][c] are positive (the
// new value is at most their minimum), on waves 1 and up; (3) at the same
// time wave 0 intersects the signatures: I(C) = I(A) ∩ I(B) in place and
// in LDS, D(A), D(B) to the packed lists; (4) the new row and column of a,
// from intersections at the candidates; (5) rows whose best partner was a
// or b are rescanned.
__global__ __launch_bounds__(kLoopThreads) void k_g_merge_loop(LoopArgs A) {
    __shared__ uint8_t act[MPT_GREEDY_MAX_M];    // 1 while r names a live cluster
    __shared__ int32_t sc[kScCap];               // I(C) of the current merge
    __shared__ int64_t scw[kScCap];              // w(x) of the chunks of I(C)
    __shared__ int32_t s_in[2 * kSigCap];        // I(A), I(B) while they are intersected
    __shared__ uint8_t dirty[kLoopThreads];      // a row owned by this thread changed its best
    // reduction scratch of steps (1) and (4): each is written again only
    // after barriers of the other steps, so neither reduction needs a
    // closing barrier
    __shared__ int64_t red1_v[kLoopWaves], red4_v[kLoopWaves];
    __shared__ int32_t red1_i[kLoopWaves], red4_i[kLoopWaves];
    __shared__ int scan_w[kLoopWaves];
    __shared__ int64_t cursor;                   // next free slot of dbuf
    __shared__ int64_t s_kept;                   // |I(C)|
    __shared__ int n_resc;
    __shared__ int32_t resc[kLoopThreads];       // rows to rescan (overflow: rescan all)
    __shared__ int resc_all;
    __shared__ int64_t part_v[kRescRows][kRescParts];
    __shared__ int32_t part_p[kRescRows][kRescParts];
    __shared__ int32_t m_at[kMetaCap];           // signature start of each cluster (m <= kMetaCap)
    __shared__ int32_t m_len[kMetaCap];          // signature length of each cluster (m <= kMetaCap)
    __shared__ int64_t m_bv[kMetaCap];           // best value of each row (m <= kMetaCap)
    __shared__ int32_t m_bp[kMetaCap];           // best partner of each row (m <= kMetaCap)
    __shared__ int32_t cand_list[kCandCap];
    __shared__ int n_cand;
    const int m = A.m;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1), wid = tid / kWave;
    // signature starts and lengths: on chip when they fit (generic pointers
    // read either)
    const bool meta_lds = m <= kMetaCap;
    int32_t *sat = meta_lds ? m_at : A.sig_at;
    int32_t *slen = meta_lds ? m_len : A.sig_len;
    int64_t *best_v = meta_lds ? m_bv : A.best_v;
    int32_t *best_p = meta_lds ? m_bp : A.best_p;
    if (tid == 0) cursor = 0;
    for (int v = tid; v < 2 * m - 1; v += blockDim.x) { A.node_parent[v] = -1; A.d_off[v] = 0; A.d_len[v] = 0; }
    for (int r = tid; r < m; r += blockDim.x) {
        A.node_of[r] = r;
        act[r] = 1;
        const int32_t at = (int32_t)A.req_off[r], len = (int32_t)(A.req_off[r + 1] - A.req_off[r]);
        if (meta_lds) { m_at[r] = at; m_len[r] = len; m_bv[r] = A.best_v[r]; m_bp[r] = A.best_p[r]; }
        else { A.sig_at[r] = at; }
    }
    dirty[tid] = 1;
    if (tid == 0) n_cand = 0;
    __syncthreads();
    int64_t cv = -1;                             // best (value, row) over the rows this thread owns
    int32_t ci = -1;
    int t = 0;
    for (; t + 1 < m; ++t) {
        // (1) the best row value, ties to the smallest row; that row's best
        // partner is larger than the row (a smaller partner would be a
        // smaller row with the same value)
        if (dirty[tid]) {
            cv = -1; ci = -1;
            for (int r = tid; r < m; r += blockDim.x)
                if (act[r] && best_p[r] >= 0 && better(best_v[r], r, cv, ci)) { cv = best_v[r]; ci = r; }
            dirty[tid] = 0;
        }
        int64_t g = cv;
        int32_t a = ci;
        block_best_once(g, a, red1_v, red1_i);
        if (a < 0 || g <= 0) break;              // every remaining value is 0
        const int32_t b = best_p[a];
        // (2) candidate columns of this thread, and which old values of a
        // are not zero (only changed entries are written back)
        uint32_t cand = 0, nonzero = 0, flag = 0, listed = 0;
        const int ct = tid - kWave;              // column owner index (wave 0 owns none)
#pragma unroll 1
        for (int k = 0; k < kColsPerThread && ct >= 0; ++k) {
            const int c = ct + k * kColThreads;
            if (c >= m) break;
            if (!act[c] || c == a) continue;
            const int64_t va = A.V[(size_t)a * m + c];
            const int64_t vb = A.V[(size_t)b * m + c];
            const int32_t p = best_p[c];
            if (va != 0) nonzero |= 1u << k;
            if (c != b && va > 0 && vb > 0) {
                cand |= 1u << k;
                const int i = atomicAdd(&n_cand, 1);       // cleared at the end of the previous step
                if (i < kCandCap) { cand_list[i] = c; listed |= 1u << k; }
            }
            if (p == a || p == b) flag |= 1u << k;
        }
        // (3) signatures, by wave 0 alone
        const int64_t na = slen[a], nb = slen[b];
        const int64_t dstart = cursor;
        if (dstart + na + nb > A.dcap) {         // cannot happen for a valid run: stop with an error
            if (tid == 0) atomicOr(&A.h->err, GERR_INVALID);
            return;
        }
        if (wid == 0) {
            int32_t *sa = A.sig + sat[a];
            const int32_t *sb_g = A.sig + sat[b];
            // the two signatures in LDS when they fit (searches stay on chip)
            const bool in_lds = na <= kSigCap && nb <= kSigCap;
            const int32_t *sa_r = sa, *sb = sb_g;
            if (in_lds) {
                for (int64_t e = lane; e < na; e += kWave) s_in[e] = sa[e];
                for (int64_t e = lane; e < nb; e += kWave) s_in[kSigCap + e] = sb_g[e];
                sa_r = s_in;
                sb = s_in + kSigCap;
            }
            int64_t dcur = dstart;
            // D(B) = I(B) \ I(A)
            for (int64_t base = 0; base < nb; base += kWave) {
                const int64_t e = base + lane;
                int32_t x = 0;
                bool keep = false;
                if (e < nb) { x = sb[e]; keep = find_sorted(sa_r, na, x) < 0; }
                const uint64_t mk = __ballot(keep);
                if (keep) A.dbuf[dcur + __popcll(mk & lanes_below(lane))] = x;
                dcur += __popcll(mk);
            }
            const int64_t d_a_at = dcur;
            // I(C) = I(A) ∩ I(B) over I(A) in place (and to LDS), D(A) = the rest
            int64_t kept = 0;
            for (int64_t base = 0; base < na; base += kWave) {
                const int64_t e = base + lane;
                int32_t x = 0;
                bool in_b = false;
                if (e < na) { x = sa_r[e]; in_b = find_sorted(sb, nb, x) >= 0; }
                const uint64_t mi = __ballot(in_b);
                const uint64_t mo = __ballot(e < na && !in_b);
                if (in_b) {
                    const int64_t pos = kept + __popcll(mi & lanes_below(lane));
                    sa[pos] = x;
                    if (pos < kScCap) { sc[pos] = x; scw[pos] = A.w[x]; }
                } else if (e < na) {
                    A.dbuf[dcur + __popcll(mo & lanes_below(lane))] = x;
                }
                kept += __popcll(mi);
                dcur += __popcll(mo);
            }
            if (lane == 0) {
                const int node_a = A.node_of[a], node_b = A.node_of[b], node_c = m + t;
                A.merge_a[t] = a; A.merge_b[t] = b; A.gain[t] = g;
                if (b <= a) atomicOr(&A.h->err, GERR_INVALID);
                A.d_off[node_b] = dstart; A.d_len[node_b] = (int32_t)(d_a_at - dstart);
                A.d_off[node_a] = d_a_at; A.d_len[node_a] = (int32_t)(dcur - d_a_at);
                A.node_parent[node_a] = node_c;
                A.node_parent[node_b] = node_c;
                A.node_of[a] = node_c;
                slen[a] = (int32_t)kept;
                act[b] = 0;
                dirty[b % kLoopThreads] = 1;
                dirty[a % kLoopThreads] = 1;
                cursor = dcur;
                s_kept = kept;
                n_resc = 0;
                resc_all = 0;
            }
        }
        __syncthreads();
        // (4) the new values of a against every live c: the listed
        // candidates are shared out evenly, every other column is 0 (or its
        // owner computes it when the list overflowed)
        const int64_t kept = s_kept;
        const bool ic_lds = kept <= kScCap;
        int64_t bv = -1;
        int32_t bp = -1;
        const int ncl = min(n_cand, kCandCap);
        for (int i = tid; i < ncl; i += blockDim.x) {
            const int c = cand_list[i];
            int64_t v = 0;
            if (kept > 0) {
                const int32_t *list = A.sig + sat[c];
                const int64_t n = slen[c];       // c != a: unchanged by this merge
                v = ic_lds ? inter_weight_lds(sc, scw, kept, list, n)
                           : inter_weight_global(A.sig + sat[a], kept, list, n, A.w);
            }
            A.V[(size_t)a * m + c] = v;
            A.V[(size_t)c * m + a] = v;
            if (better(v, c, bv, bp)) { bv = v; bp = c; }
        }
#pragma unroll 1
        for (int k = 0; k < kColsPerThread && ct >= 0; ++k) {
            const int c = ct + k * kColThreads;
            if (c >= m) break;
            if (!act[c] || c == a) continue;
            if (!((listed >> k) & 1u)) {
                const bool is_cand = kept > 0 && ((cand >> k) & 1u);
                int64_t v = 0;
                if (is_cand) {
                    const int32_t *list = A.sig + sat[c];
                    const int64_t n = slen[c];
                    v = ic_lds ? inter_weight_lds(sc, scw, kept, list, n)
                               : inter_weight_global(A.sig + sat[a], kept, list, n, A.w);
                }
                if (is_cand || ((nonzero >> k) & 1u)) {  // the old value may differ
                    A.V[(size_t)a * m + c] = v;
                    A.V[(size_t)c * m + a] = v;
                }
                if (better(v, c, bv, bp)) { bv = v; bp = c; }
            }
            if ((flag >> k) & 1u) {
                const int r = atomicAdd(&n_resc, 1);
                if (r < kLoopThreads) resc[r] = c; else resc_all = 1;
                dirty[c % kLoopThreads] = 1;
            }
        }
        block_best_once(bv, bp, red4_v, red4_i);   // its barrier comes after the V writes
        if (tid == 0) { best_v[a] = bv; best_p[a] = bp; n_cand = 0; }
        // (5) rows whose best partner was a or b: rescan. Values never grow,
        // so the row's old best bounds every entry now: scanning in index
        // order, the first entry at that bound is the answer (largest value,
        // smallest index) and the scan can stop there. Rows go four at a
        // time, each split into four quarters of columns, one wave each.
        const int nr = resc_all ? m : n_resc;
        for (int r0 = 0; r0 < nr; r0 += kRescRows) {
            const int slot = wid / kRescParts, part = wid % kRescParts;
            const int k = r0 + slot;
            int c = -1;
            if (k < nr) {
                c = resc_all ? k : resc[k];
                if (!act[c] || c == a || (resc_all && best_p[c] != a && best_p[c] != b)) c = -1;
            }
            if (c >= 0) {
                const int64_t ub = best_v[c];
                const int64_t *row = A.V + (size_t)c * m;
                const int q = (m + kRescParts - 1) / kRescParts;
                const int lo = part * q, hi = min(m, lo + q);
                int64_t v = -1;
                int32_t p = -1;
                bool hit = false;
                constexpr int G = 8;             // chunks of 64 columns loaded together
                for (int base = lo; base < hi && !hit; base += G * kWave) {
                    int64_t x[G];
#pragma unroll
                    for (int j = 0; j < G; ++j) {
                        const int d = base + j * kWave + lane;
                        x[j] = (d < hi && d != c && act[d]) ? row[d] : -1;
                    }
#pragma unroll
                    for (int j = 0; j < G; ++j) {
                        const int d = base + j * kWave + lane;
                        const uint64_t at_ub = __ballot(x[j] == ub && x[j] >= 0);
                        if (!hit && at_ub) {
                            v = ub;
                            p = base + j * kWave + __ffsll((long long)at_ub) - 1;
                            hit = true;
                        }
                        if (!hit && better(x[j], d, v, p)) { v = x[j]; p = d; }
                    }
                }
                if (!hit) wave_best(v, p);
                if (lane == 0) { part_v[slot][part] = v; part_p[slot][part] = p; }
            }
            __syncthreads();
            // quarters in index order: the first that holds a best equal to
            // the bound decides, otherwise the best of the four
            if (part == 0 && lane == 0 && c >= 0) {
                const int64_t ub = best_v[c];
                int64_t v = -1;
                int32_t p = -1;
                for (int j = 0; j < kRescParts; ++j) {
                    if (part_p[slot][j] < 0) continue;
                    if (part_v[slot][j] == ub) { v = ub; p = part_p[slot][j]; break; }
                    if (better(part_v[slot][j], part_p[slot][j], v, p)) { v = part_v[slot][j]; p = part_p[slot][j]; }
                }
                best_v[c] = v;
                best_p[c] = p;
            }
            __syncthreads();
        }
    }
    // Every remaining pair shares nothing: the merges take the two smallest
    // live names in turn (n0, n1), (n0, n2), ... with gain 0, and every
    // merged signature is empty, so D(child) is the child's whole signature
    // (the root's whole signature if only one cluster is left) and the
    // chain's own nodes emit nothing. Live names in ascending order, one
    // round of the workgroup at a time.
    __shared__ int32_t first_name;
    if (tid == 0) first_name = -1;
    __syncthreads();
    const int t0 = t;
    int64_t dcur = cursor;
    int done = 0;                                // live names ranked so far
    for (int base = 0; base < m; base += blockDim.x) {
        const int r = base + tid;
        const int live = r < m && act[r];
        const int len = live ? slen[r] : 0;
        int tot, ltot;
        const int rank = done + block_scan(live, &tot, scan_w);
        const int loff = block_scan(len, &ltot, scan_w);
        if (dcur + ltot > A.dcap) {              // cannot happen for a valid run
            if (tid == 0) atomicOr(&A.h->err, GERR_INVALID);
            return;
        }
        if (live) {
            const int node = A.node_of[r];
            const int32_t *src = A.sig + sat[r];
            for (int e = 0; e < len; ++e) A.dbuf[dcur + loff + e] = src[e];
            A.d_off[node] = dcur + loff;
            A.d_len[node] = len;
            if (rank == 0) {
                first_name = r;
            } else {
                const int tt = t0 + rank - 1;    // the merge that takes r
                A.merge_b[tt] = r;
                A.gain[tt] = 0;
                A.node_parent[node] = m + tt;
            }
        }
        done += tot;
        dcur += ltot;
        __syncthreads();
    }
    const int n_live = done;
    // the chain: node m+t0 holds the first two names, node m+t0+k holds
    // node m+t0+k-1 and the name of rank k+1
    for (int k = tid; k + 1 < n_live; k += blockDim.x) {
        A.merge_a[t0 + k] = first_name;
        A.d_off[m + t0 + k] = dcur;
        A.d_len[m + t0 + k] = 0;
        if (k > 0) A.node_parent[m + t0 + k - 1] = m + t0 + k;
    }
    if (tid == 0 && n_live >= 2) A.node_parent[A.node_of[first_name]] = m + t0;
    if (tid == 0 && t0 + n_live - 1 != m - 1) atomicOr(&A.h->err, GERR_INVALID);
}

// pi_i: walk from leaf i to the root, placing D(v) of every node on the
// path right to left (the root's list comes first); one wave per request
__global__ void k_g_orders(int m, int64_t nnz, const int64_t *req_off, const int32_t *node_parent,
                           const int32_t *dbuf, const int64_t *d_off, const int32_t *d_len, int32_t *order_chunks,
                           GHeader *h) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
    if (i >= m) return;
    int64_t end = req_off[i + 1];
    const int64_t begin = req_off[i];
    int steps = 0;
    for (int v = (int)i; v >= 0 && steps < 2 * m; v = node_parent[v], ++steps) {
        if (v >= 2 * m - 1) { if (lane == 0) atomicOr(&h->err, GERR_INVALID); return; }
        const int64_t len = d_len[v];
        if (len < 0 || end - len < begin || d_off[v] < 0 || d_off[v] + len > nnz) {
            if (lane == 0) atomicOr(&h->err, GERR_INVALID);
            return;
        }
        const int32_t *src = dbuf + d_off[v];
        for (int64_t e = lane; e < len; e += kWave) order_chunks[end - len + e] = src[e];
        end -= len;
    }
    if (end != begin && lane == 0) atomicOr(&h->err, GERR_INVALID);
}

// ---------------------------------------------------------------------------
// maximum spanning tree (Boruvka). Edges are ordered by (weight desc, then
// the pair (lo, hi) of their endpoints ascending), a strict total order, so
// every round's chosen edges form a forest plus mutual pairs and no cycle
// can close. Every round at least halves the number of components; the
// complete graph keeps an edge between any two, so ceil(log2 m) rounds
// leave one. The tree's weight does not depend on which order breaks ties.

__device__ inline uint32_t edge_id(int u, int v) {
    const uint32_t lo = (uint32_t)min(u, v), hi = (uint32_t)max(u, v);
    return (lo << 14) | hi;                      // m <= 2^14
}

__global__ void k_bv_init(int m, int32_t *comp, unsigned long long *total) {
    for (int v = blockIdx.x * blockDim.x + threadIdx.x; v < m; v += gridDim.x * blockDim.x) comp[v] = v;
    if (blockIdx.x == 0 && threadIdx.x == 0) *total = 0;
}

__global__ void k_bv_reset(int m, int64_t *cw, uint32_t *ce) {
    for (int v = blockIdx.x * blockDim.x + threadIdx.x; v < m; v += gridDim.x * blockDim.x) { cw[v] = -1; ce[v] = ~0u; }
}

// best edge of every vertex to another component (one wave per vertex),
// folded into its component's best weight
__global__ void k_bv_vertex(int m, const int64_t *P, const int32_t *comp, int64_t *vw, uint32_t *ve, int64_t *cw) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t u = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
    if (u >= m) return;
    const int32_t cu = comp[u];
    int64_t bw = -1;
    uint32_t be = ~0u;
    for (int v = lane; v < m; v += kWave) {
        if (comp[v] == cu) continue;
        const int64_t x = P[u * m + v];
        const uint32_t e = edge_id((int)u, v);
        if (x > bw || (x == bw && e < be)) { bw = x; be = e; }
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const int64_t ow = __shfl_xor(bw, off, kWave);
        const uint32_t oe = (uint32_t)__shfl_xor((int)be, off, kWave);
        if (ow > bw || (ow == bw && oe < be)) { bw = ow; be = oe; }
    }
    if (lane == 0) {
        vw[u] = bw; ve[u] = be;
        if (bw >= 0) atomicMax((long long *)&cw[cu], (long long)bw);
    }
}

// among the vertices that reach their component's best weight, the smallest edge
__global__ void k_bv_edge(int m, const int32_t *comp, const int64_t *vw, const uint32_t *ve, const int64_t *cw,
                          uint32_t *ce) {
    for (int u = blockIdx.x * blockDim.x + threadIdx.x; u < m; u += gridDim.x * blockDim.x) {
        const int32_t cu = comp[u];
        if (vw[u] >= 0 && vw[u] == cw[cu]) atomicMin(&ce[cu], ve[u]);
    }
}

// every component hooks onto the component across its best edge, except
// the smaller one of a mutual pair; the hooking side adds the edge weight
__global__ void k_bv_hook(int m, const int32_t *comp, const int64_t *cw, const uint32_t *ce, int32_t *par,
                          unsigned long long *total) {
    for (int c = blockIdx.x * blockDim.x + threadIdx.x; c < m; c += gridDim.x * blockDim.x) {
        par[c] = c;
        if (comp[c] != c || ce[c] == ~0u) continue;
        const int lo = (int)(ce[c] >> 14), hi = (int)(ce[c] & 0x3fffu);
        const int32_t d = comp[lo] == c ? comp[hi] : comp[lo];
        if (ce[d] == ce[c] && c < d) continue;           // d hooks onto c
        par[c] = d;
        atomicAdd(total, (unsigned long long)cw[c]);
    }
}

// new component of every vertex: follow the hooks to a root
__global__ void k_bv_jump(int m, int32_t *comp, const int32_t *par) {
    for (int v = blockIdx.x * blockDim.x + threadIdx.x; v < m; v += gridDim.x * blockDim.x) {
        int32_t r = comp[v];
        for (int guard = 0; par[r] != r && guard < m; ++guard) r = par[r];
        comp[v] = r;
    }
}

// ---------------------------------------------------------------------------
// host side

int g_check_common(int m, int64_t n_chunks, int64_t nnz) {
    if (m < 1 || m > MPT_GREEDY_MAX_M) return fail(MPT_E_INVALID, "m = %d outside [1, %d]", m, MPT_GREEDY_MAX_M);
    if (n_chunks < 0 || n_chunks > MPT_MAX_CHUNKS) return fail(MPT_E_INVALID, "n_chunks = %lld out of range", (long long)n_chunks);
    if (nnz < 0 || nnz > (int64_t)INT32_MAX) return fail(MPT_E_INVALID, "nnz = %lld out of range", (long long)nnz);
    return MPT_OK;
}

int g_check_ws(const GLayout &L, void *ws, size_t bytes) {
    if (!ws) return fail(MPT_E_WORKSPACE, "workspace is NULL");
    if (((uintptr_t)ws & 255u) != 0) return fail(MPT_E_WORKSPACE, "workspace is not 256-byte aligned");
    if (bytes < L.total) return fail(MPT_E_WORKSPACE, "workspace has %zu bytes, needs %zu", bytes, L.total);
    return MPT_OK;
}

int g_read_errors(GHeader *h, hipStream_t s, int64_t *request_total = nullptr) {
    GHeader hh;
    MPT_HIP_TRY(hipMemcpyAsync(&hh, h, sizeof hh, hipMemcpyDeviceToHost, s));
    MPT_HIP_TRY(hipStreamSynchronize(s));
    if (hh.err & GERR_INVALID) return fail(MPT_E_INVALID, "req_off is not a CSR offset array of length m+1 ending at nnz");
    if (hh.err & GERR_RANGE) return fail(MPT_E_RANGE, "a chunk id is outside [0, n_chunks)");
    if (hh.err & GERR_WEIGHT) return fail(MPT_E_WEIGHT, "a chunk weight is <= 0 or > 2^32");
    if (hh.err & GERR_DUP) return fail(MPT_E_DUP, "a chunk is repeated inside one request");
    if (hh.total >= (1ull << 61)) return fail(MPT_E_OVERFLOW, "sum of request weights reaches 2^61");
    if (request_total) *request_total = (int64_t)hh.total;
    return MPT_OK;
}

// Validate the instance and build the sorted lists, the demand lists and
// (when P is given) the pair weights. Synchronises once to report errors.
int g_prepare(int m, int64_t n_chunks, int64_t nnz, const int64_t *chunk_w, const int64_t *req_off,
              const int32_t *req_chunks, int64_t *P, const GLayout &L, char *ws, hipStream_t s,
              int64_t *request_total = nullptr) {
    GHeader *h = (GHeader *)ws;
    uint64_t *keys1 = (uint64_t *)(ws + L.keys1), *keys2 = (uint64_t *)(ws + L.keys2);
    k_g_header<<<1, 64, 0, s>>>(h);
    k_g_check_offsets<<<1, 256, 0, s>>>(m, nnz, req_off, h);
    if (n_chunks > 0) k_g_check_weights<<<grid_for(n_chunks, 256), 256, 0, s>>>(n_chunks, chunk_w, h);
    {
        LaunchScope ls("g_keys", (double)nnz, s);
        k_g_keys<<<grid_for(L.npad, 256), 256, 0, s>>>(m, n_chunks, nnz, L.npad, req_off, req_chunks, chunk_w, keys1,
                                                      keys2, h);
    }
    MPT_HIP_TRY(hipGetLastError());
    int rc = g_read_errors(h, s);
    if (rc) return rc;
    {
        LaunchScope ls("g_sort", 2.0 * (double)L.npad, s);
        if ((rc = sort_keys(keys1, L.npad, s))) return rc;
        if ((rc = sort_keys(keys2, L.npad, s))) return rc;
    }
    int32_t *sig = (int32_t *)(ws + L.sig), *sig_len = (int32_t *)(ws + L.sig_len), *dem = (int32_t *)(ws + L.dem);
    int64_t *dem_off = (int64_t *)(ws + L.dem_off);
    k_g_lists<<<grid_for(std::max<int64_t>(nnz, m), 256), 256, 0, s>>>(m, nnz, keys1, keys2, sig, sig_len, dem, req_off, h);
    k_g_dem_off<<<grid_for(n_chunks + 1, 256), 256, 0, s>>>(n_chunks, nnz, keys2, dem_off);
    MPT_HIP_TRY(hipGetLastError());
    if ((rc = g_read_errors(h, s, request_total))) return rc;
    if (P) {
        const int64_t mm = (int64_t)m * m;
        LaunchScope ls("g_pairs", 8.0 * (double)mm, s);
        k_g_fill64<<<grid_for(mm, 256, 16384), 256, 0, s>>>(P, mm, 0);
        if (nnz > 0)
            k_g_pairs<<<grid_for(nnz * kWave, 256, 16384), 256, 0, s>>>(m, nnz, keys2, dem, dem_off, chunk_w,
                                                                         (unsigned long long *)P);
        MPT_HIP_TRY(hipGetLastError());
    }
    return MPT_OK;
}

}  // namespace

extern "C" size_t mpt_greedy_workspace_bytes(int m, int64_t n_chunks, int64_t nnz) {
    if (m < 1 || m > MPT_GREEDY_MAX_M || n_chunks < 0 || nnz < 0) return 0;
    return g_layout(m, n_chunks, nnz).total;
}

extern "C" int mpt_pair_weights(int m, int64_t n_chunks, int64_t nnz, const int64_t *chunk_w, const int64_t *req_off,
                                const int32_t *req_chunks, int64_t *P, int64_t *request_total, void *workspace,
                                size_t workspace_bytes, void *stream) {
    mptlib::clear_error();
    int rc = g_check_common(m, n_chunks, nnz);
    if (rc) return rc;
    if (!req_off || !P) return fail(MPT_E_INVALID, "req_off and P must not be NULL");
    if (n_chunks > 0 && !chunk_w) return fail(MPT_E_INVALID, "chunk_w must not be NULL");
    if (nnz > 0 && !req_chunks) return fail(MPT_E_INVALID, "req_chunks must not be NULL");
    const GLayout L = g_layout(m, n_chunks, nnz);
    if ((rc = g_check_ws(L, workspace, workspace_bytes))) return rc;
    return g_prepare(m, n_chunks, nnz, chunk_w, req_off, req_chunks, P, L, (char *)workspace, (hipStream_t)stream,
                     request_total);
}

extern "C" int mpt_greedy_hierarchy(int m, int64_t n_chunks, int64_t nnz, const int64_t *chunk_w,
                                    const int64_t *req_off, const int32_t *req_chunks, int32_t *merge_a,
                                    int32_t *merge_b, int64_t *gain, int32_t *node_parent, int32_t *order_chunks,
                                    int64_t *savings, void *workspace, size_t workspace_bytes, void *stream) {
    mptlib::clear_error();
    int rc = g_check_common(m, n_chunks, nnz);
    if (rc) return rc;
    if (!req_off || !node_parent) return fail(MPT_E_INVALID, "req_off and node_parent must not be NULL");
    if (m > 1 && (!merge_a || !merge_b || !gain)) return fail(MPT_E_INVALID, "merge_a, merge_b and gain must not be NULL");
    if (n_chunks > 0 && !chunk_w) return fail(MPT_E_INVALID, "chunk_w must not be NULL");
    if (nnz > 0 && !req_chunks) return fail(MPT_E_INVALID, "req_chunks must not be NULL");
    const GLayout L = g_layout(m, n_chunks, nnz);
    if ((rc = g_check_ws(L, workspace, workspace_bytes))) return rc;
    hipStream_t s = (hipStream_t)stream;
    char *ws = (char *)workspace;
    int64_t *V = (int64_t *)(ws + L.V);
    if ((rc = g_prepare(m, n_chunks, nnz, chunk_w, req_off, req_chunks, V, L, ws, s))) return rc;
    LoopArgs A{};
    A.m = m;
    A.w = chunk_w;
    A.req_off = req_off;
    A.sig = (int32_t *)(ws + L.sig);
    A.sig_len = (int32_t *)(ws + L.sig_len);
    A.sig_at = (int32_t *)(ws + L.key);
    A.V = V;
    A.best_v = (int64_t *)(ws + L.best_v);
    A.best_p = (int32_t *)(ws + L.best_p);
    A.node_of = (int32_t *)(ws + L.node_of);
    A.dbuf = (int32_t *)(ws + L.dbuf);
    A.dcap = std::max<int64_t>(nnz, 1);
    A.d_off = (int64_t *)(ws + L.d_off);
    A.d_len = (int32_t *)(ws + L.d_len);
    A.merge_a = merge_a;
    A.merge_b = merge_b;
    A.gain = gain;
    A.node_parent = node_parent;
    A.h = (GHeader *)ws;
    {
        LaunchScope ls("g_row_best", 8.0 * (double)m * m, s);
        k_g_row_best<<<(m + 3) / 4, 4 * kWave, 0, s>>>(m, V, A.best_v, A.best_p);
    }
    {
        LaunchScope ls("g_merge_loop", (double)(m - 1), s);
        k_g_merge_loop<<<1, kLoopThreads, 0, s>>>(A);
    }
    MPT_HIP_TRY(hipGetLastError());
    if (order_chunks) {
        LaunchScope ls("g_orders", 4.0 * (double)nnz, s);
        k_g_orders<<<(m + 3) / 4, 4 * kWave, 0, s>>>(m, nnz, req_off, node_parent, A.dbuf, A.d_off, A.d_len,
                                                     order_chunks, A.h);
        MPT_HIP_TRY(hipGetLastError());
    }
    if ((rc = g_read_errors(A.h, s))) return rc;
    if (savings) {
        *savings = 0;
        if (m > 1) {
            // the gains are copied back and summed on the host (m - 1 values)
            int64_t *hg = new int64_t[m - 1];
            const hipError_t e1 = hipMemcpyAsync(hg, gain, sizeof(int64_t) * (size_t)(m - 1), hipMemcpyDeviceToHost, s);
            const hipError_t e2 = e1 == hipSuccess ? hipStreamSynchronize(s) : e1;
            if (e2 != hipSuccess) { delete[] hg; return fail(MPT_E_DEVICE, "copy of the gains: %s", hipGetErrorString(e2)); }
            for (int t = 0; t < m - 1; ++t) *savings += hg[t];
            delete[] hg;
        }
    }
    return MPT_OK;
}

extern "C" int mpt_spanning_tree_bound(int m, const int64_t *P, int64_t *mst_weight, void *workspace,
                                       size_t workspace_bytes, void *stream) {
    mptlib::clear_error();
    if (m < 1 || m > MPT_GREEDY_MAX_M) return fail(MPT_E_INVALID, "m = %d outside [1, %d]", m, MPT_GREEDY_MAX_M);
    if (!P || !mst_weight) return fail(MPT_E_INVALID, "P and mst_weight must not be NULL");
    if (!workspace) return fail(MPT_E_WORKSPACE, "workspace is NULL");
    if (((uintptr_t)workspace & 255u) != 0) return fail(MPT_E_WORKSPACE, "workspace is not 256-byte aligned");
    // header, then comp, par, vertex-best and component-best arrays
    const size_t mm = (size_t)m;
    const size_t off_comp = align256(sizeof(GHeader)), off_par = off_comp + align256(4 * mm),
                 off_vw = off_par + align256(4 * mm), off_ve = off_vw + align256(8 * mm),
                 off_cw = off_ve + align256(4 * mm), off_ce = off_cw + align256(8 * mm), need = off_ce + align256(4 * mm);
    if (workspace_bytes < need) return fail(MPT_E_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
    hipStream_t s = (hipStream_t)stream;
    GHeader *h = (GHeader *)workspace;
    char *ws = (char *)workspace;
    int32_t *comp = (int32_t *)(ws + off_comp), *par = (int32_t *)(ws + off_par);
    int64_t *vw = (int64_t *)(ws + off_vw), *cw = (int64_t *)(ws + off_cw);
    uint32_t *ve = (uint32_t *)(ws + off_ve), *ce = (uint32_t *)(ws + off_ce);
    int rounds = 0;
    while ((1 << rounds) < m) ++rounds;
    const int gv = grid_for(m, 256);
    k_bv_init<<<gv, 256, 0, s>>>(m, comp, &h->total);
    for (int r = 0; r < rounds; ++r) {
        LaunchScope ls("g_boruvka", 8.0 * (double)m * m, s);
        k_bv_reset<<<gv, 256, 0, s>>>(m, cw, ce);
        k_bv_vertex<<<(m + 3) / 4, 4 * kWave, 0, s>>>(m, P, comp, vw, ve, cw);
        k_bv_edge<<<gv, 256, 0, s>>>(m, comp, vw, ve, cw, ce);
        k_bv_hook<<<gv, 256, 0, s>>>(m, comp, cw, ce, par, &h->total);
        k_bv_jump<<<gv, 256, 0, s>>>(m, comp, par);
    }
    MPT_HIP_TRY(hipGetLastError());
    unsigned long long total = 0;
    MPT_HIP_TRY(hipMemcpyAsync(&total, &h->total, sizeof total, hipMemcpyDeviceToHost, s));
    MPT_HIP_TRY(hipStreamSynchronize(s));
    *mst_weight = (int64_t)total;
    return MPT_OK;
}
