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

#include "common.h"
#include "mpt.h"

namespace {

using mptlib::align256;
using mptlib::fail;
using mptlib::grid_for;
using mptlib::LaunchScope;

constexpr int kWave = 64;
constexpr int kLoopThreads = 1024;           // the one workgroup of the merge loop and of Prim
constexpr int kLoopWaves = kLoopThreads / kWave;
constexpr int kSortTile = 4096;              // keys sorted in LDS per workgroup
constexpr int kSortThreads = 1024;

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
    L.key = take(8 * mm);
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

// best (value, index) over the workgroup; every thread gets the result
__device__ inline void block_best(int64_t &v, int32_t &i, int64_t *sv, int32_t *si) {
    wave_best(v, i);
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    if (lane == 0) { sv[wid] = v; si[wid] = i; }
    __syncthreads();
    v = sv[0]; i = si[0];
    for (int k = 1; k < (int)(blockDim.x / kWave); ++k)
        if (better(sv[k], si[k], v, i)) { v = sv[k]; i = si[k]; }
    __syncthreads();
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
// bitonic sort of n = 2^k >= kSortTile uint64 keys, ascending

__device__ inline void cswap(uint64_t &a, uint64_t &b, bool up) {
    if ((a > b) == up) { const uint64_t t = a; a = b; b = t; }
}

// every stage k <= kSortTile inside one tile (direction from the global index)
__global__ __launch_bounds__(kSortThreads) void k_sort_tile(uint64_t *keys) {
    __shared__ uint64_t t[kSortTile];
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
    for (int e = threadIdx.x; e < kSortTile; e += kSortThreads) t[e] = keys[base + e];
    __syncthreads();
    for (int k = 2; k <= kSortTile; k <<= 1)
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int p = threadIdx.x; p < kSortTile / 2; p += kSortThreads) {
                const int i = ((p / j) * 2 * j) + (p % j), l = i + j;
                cswap(t[i], t[l], ((base + i) & k) == 0);
            }
            __syncthreads();
        }
    for (int e = threadIdx.x; e < kSortTile; e += kSortThreads) keys[base + e] = t[e];
}

// one compare-exchange step of stage k with stride j >= kSortTile
__global__ void k_sort_global(uint64_t *keys, int64_t n, int64_t k, int64_t j) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n / 2; p += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = ((p / j) * 2 * j) + (p % j), l = i + j;
        uint64_t a = keys[i], b = keys[l];
        cswap(a, b, (i & k) == 0);
        keys[i] = a; keys[l] = b;
    }
}

// the strides j < kSortTile of stage k > kSortTile inside one tile
__global__ __launch_bounds__(kSortThreads) void k_sort_tile_merge(uint64_t *keys, int64_t k) {
    __shared__ uint64_t t[kSortTile];
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
    for (int e = threadIdx.x; e < kSortTile; e += kSortThreads) t[e] = keys[base + e];
    __syncthreads();
    const bool up = (base & k) == 0;            // the tile lies inside one run of stage k
    for (int j = kSortTile >> 1; j > 0; j >>= 1) {
        for (int p = threadIdx.x; p < kSortTile / 2; p += kSortThreads) {
            const int i = ((p / j) * 2 * j) + (p % j), l = i + j;
            cswap(t[i], t[l], up);
        }
        __syncthreads();
    }
    for (int e = threadIdx.x; e < kSortTile; e += kSortThreads) keys[base + e] = t[e];
}

int sort_keys(uint64_t *keys, int64_t n, hipStream_t s) {
    const int tiles = (int)(n / kSortTile);
    k_sort_tile<<<tiles, kSortThreads, 0, s>>>(keys);
    for (int64_t k = 2 * kSortTile; k <= n; k <<= 1) {
        for (int64_t j = k >> 1; j >= kSortTile; j >>= 1)
            k_sort_global<<<grid_for(n / 2, 256, 16384), 256, 0, s>>>(keys, n, k, j);
        k_sort_tile_merge<<<tiles, kSortThreads, 0, s>>>(keys, k);
    }
    MPT_HIP_TRY(hipGetLastError());
    return MPT_OK;
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
// for every later request b of S_x
__global__ void k_g_pairs(int m, int64_t nnz, const uint64_t *keys2, const int32_t *dem, const int64_t *dem_off,
                          const int64_t *w, unsigned long long *P) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < nnz; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t x = (int64_t)(keys2[e] >> 32);
        const unsigned long long wx = (unsigned long long)w[x];
        const size_t a = (size_t)dem[e];
        atomicAdd(&P[a * m + a], wx);
        const int64_t end = dem_off[x + 1];
        for (int64_t f = e + 1; f < end; ++f) {
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
__global__ void k_g_row_best(int m, const int64_t *V, int64_t *best_v, int32_t *best_p, int32_t *active) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
    if (row >= m) return;
    int64_t v = -1;
    int32_t p = -1;
    for (int d = lane; d < m; d += kWave)
        if (d != row && better(V[row * m + d], d, v, p)) { v = V[row * m + d]; p = d; }
    wave_best(v, p);
    if (lane == 0) { best_v[row] = v; best_p[row] = p; active[row] = 1; }
}

struct LoopArgs {
    int m;
    const int64_t *w;
    const int64_t *req_off;     // start of cluster a's signature
    int32_t *sig;               // signatures, ascending, shrinking in place
    int32_t *sig_len;
    const int32_t *dem;
    const int64_t *dem_off;
    int64_t *V;                 // V[a][c] = w(I(a) ∩ I(c)) for live a, c
    int64_t *best_v;
    int32_t *best_p;
    int32_t *active;            // 1 while a is the name of a live cluster
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

__global__ __launch_bounds__(kLoopThreads) void k_g_merge_loop(LoopArgs A) {
    extern __shared__ int64_t newv[];            // m entries: values of the new cluster
    __shared__ int64_t red_v[kLoopWaves];
    __shared__ int32_t red_i[kLoopWaves];
    __shared__ int scan_w[kLoopWaves];
    __shared__ int64_t cursor;                   // next free slot of dbuf
    __shared__ int n_resc;
    __shared__ int32_t resc[kLoopThreads];       // rows to rescan (overflow: rescan all)
    __shared__ int resc_all;
    const int m = A.m;
    const int tid = threadIdx.x;
    if (tid == 0) cursor = 0;
    for (int v = tid; v < 2 * m - 1; v += blockDim.x) { A.node_parent[v] = -1; A.d_off[v] = 0; A.d_len[v] = 0; }
    for (int a = tid; a < m; a += blockDim.x) A.node_of[a] = a;
    __syncthreads();
    int t = 0;
    for (; t + 1 < m; ++t) {
        // the pair to merge: the best row value, ties to the smallest row;
        // that row's best partner is larger than the row (a smaller partner
        // would be a smaller row with the same value)
        int64_t g = -1;
        int32_t a = -1;
        for (int r = tid; r < m; r += blockDim.x)
            if (A.active[r] && A.best_p[r] >= 0 && better(A.best_v[r], r, g, a)) { g = A.best_v[r]; a = r; }
        block_best(g, a, red_v, red_i);
        if (a < 0 || g <= 0) break;              // every remaining value is 0
        const int32_t b = A.best_p[a];
        if (tid == 0) {
            A.merge_a[t] = a; A.merge_b[t] = b; A.gain[t] = g;
            if (b <= a) atomicOr(&A.h->err, GERR_INVALID);
        }
        // D(B) = I(B) \ I(A), then I(A) <- I(A) ∩ I(B) in place with
        // D(A) = I(A) \ I(B) on the side
        int32_t *sa = A.sig + A.req_off[a];
        const int32_t *sb = A.sig + A.req_off[b];
        const int64_t na = A.sig_len[a], nb = A.sig_len[b];
        const int node_a = A.node_of[a], node_b = A.node_of[b];
        int64_t dcur = cursor;
        if (dcur + na + nb > A.dcap) {                 // cannot happen for a valid run: stop with an error
            if (tid == 0) atomicOr(&A.h->err, GERR_INVALID);
            return;
        }
        const int64_t d_b_at = dcur;
        for (int64_t base = 0; base < nb; base += blockDim.x) {
            const int64_t e = base + tid;
            int32_t x = 0;
            int keep = 0;
            if (e < nb) { x = sb[e]; keep = find_sorted(sa, na, x) < 0; }
            int tot;
            const int off = block_scan(keep, &tot, scan_w);
            if (keep) A.dbuf[dcur + off] = x;
            dcur += tot;
        }
        const int64_t d_a_at = dcur;
        int64_t kept = 0;
        for (int64_t base = 0; base < na; base += blockDim.x) {
            const int64_t e = base + tid;
            int32_t x = 0;
            int in_b = 0;
            if (e < na) { x = sa[e]; in_b = find_sorted(sb, nb, x) >= 0; }
            int tot_in;
            const int off_in = block_scan(in_b, &tot_in, scan_w);
            const int off_out = (int)(e - base) - off_in;   // position among this round's dropped entries
            __syncthreads();                                // every read of this round of sa is done
            if (e < na) {
                if (in_b) sa[kept + off_in] = x;
                else A.dbuf[dcur + off_out] = x;
            }
            const int64_t round = std::min<int64_t>((int64_t)blockDim.x, na - base);
            kept += tot_in;
            dcur += round - tot_in;
        }
        const int node_c = m + t;
        if (tid == 0) {
            A.d_off[node_b] = d_b_at; A.d_len[node_b] = (int32_t)(d_a_at - d_b_at);
            A.d_off[node_a] = d_a_at; A.d_len[node_a] = (int32_t)(dcur - d_a_at);
            A.node_parent[node_a] = node_c;
            A.node_parent[node_b] = node_c;
            A.node_of[a] = node_c;
            A.sig_len[a] = (int32_t)kept;
            A.active[b] = 0;
            cursor = dcur;
            n_resc = 0;
            resc_all = 0;
        }
        for (int c = tid; c < m; c += blockDim.x) newv[c] = 0;
        __syncthreads();
        // values of the new cluster: x in I(C) counts for cluster c iff the
        // name c (its smallest request) holds x and x is in I(c)
        for (int64_t e = 0; e < kept; ++e) {
            const int32_t x = sa[e];
            const int64_t wx = A.w[x];
            for (int64_t f = A.dem_off[x] + tid; f < A.dem_off[x + 1]; f += blockDim.x) {
                const int32_t c = A.dem[f];
                if (c != a && A.active[c] && find_sorted(A.sig + A.req_off[c], A.sig_len[c], x) >= 0)
                    atomicAdd((unsigned long long *)&newv[c], (unsigned long long)wx);
            }
        }
        __syncthreads();
        int64_t bv = -1;
        int32_t bp = -1;
        for (int c = tid; c < m; c += blockDim.x) {
            if (!A.active[c] || c == a) continue;
            const int64_t v = newv[c];
            A.V[(size_t)a * m + c] = v;
            A.V[(size_t)c * m + a] = v;
            if (better(v, c, bv, bp)) { bv = v; bp = c; }
            const int32_t p = A.best_p[c];
            if (p == a || p == b) {
                const int k = atomicAdd(&n_resc, 1);
                if (k < kLoopThreads) resc[k] = c; else resc_all = 1;
            }
        }
        block_best(bv, bp, red_v, red_i);        // includes a barrier after the V writes
        if (tid == 0) { A.best_v[a] = bv; A.best_p[a] = bp; }
        // rows whose best partner was a or b: rescan, one wave per row
        const int lane = tid & (kWave - 1), wid = tid / kWave;
        const int nr = resc_all ? m : n_resc;
        for (int k = wid; k < nr; k += kLoopWaves) {
            const int c = resc_all ? k : resc[k];
            if (!A.active[c] || c == a || (resc_all && A.best_p[c] != a && A.best_p[c] != b)) continue;
            int64_t v = -1;
            int32_t p = -1;
            for (int d = lane; d < m; d += kWave)
                if (d != c && A.active[d] && better(A.V[(size_t)c * m + d], d, v, p)) { v = A.V[(size_t)c * m + d]; p = d; }
            wave_best(v, p);
            if (lane == 0) { A.best_v[c] = v; A.best_p[c] = p; }
        }
        __syncthreads();
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
        const int live = r < m && A.active[r];
        const int len = live ? A.sig_len[r] : 0;
        int tot, ltot;
        const int rank = done + block_scan(live, &tot, scan_w);
        const int loff = block_scan(len, &ltot, scan_w);
        if (dcur + ltot > A.dcap) {              // cannot happen for a valid run
            if (tid == 0) atomicOr(&A.h->err, GERR_INVALID);
            return;
        }
        if (live) {
            const int node = A.node_of[r];
            const int32_t *src = A.sig + A.req_off[r];
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
// maximum spanning tree (Prim), one workgroup; key[] in LDS

__global__ __launch_bounds__(kLoopThreads) void k_g_prim(int m, const int64_t *P, unsigned long long *out) {
    extern __shared__ int64_t key[];             // -1: in the tree
    __shared__ int64_t red_v[kLoopWaves];
    __shared__ int32_t red_i[kLoopWaves];
    const int tid = threadIdx.x;
    for (int v = tid; v < m; v += blockDim.x) key[v] = v == 0 ? 0 : INT64_MIN;
    __syncthreads();
    unsigned long long total = 0;
    for (int it = 0; it < m; ++it) {
        int64_t bv = INT64_MIN;
        int32_t bu = -1;
        for (int v = tid; v < m; v += blockDim.x)
            if (key[v] != -1 && (bu < 0 || better(key[v], v, bv, bu))) { bv = key[v]; bu = v; }
        block_best(bv, bu, red_v, red_i);
        if (bu < 0) break;
        total += (unsigned long long)bv;
        if (tid == 0) key[bu] = -1;
        __syncthreads();
        const int64_t *row = P + (size_t)bu * m;
        for (int v = tid; v < m; v += blockDim.x) {
            const int64_t k = key[v];
            if (k != -1 && row[v] > k) key[v] = row[v];
        }
        __syncthreads();
    }
    if (tid == 0) *out = total;
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
            k_g_pairs<<<grid_for(nnz, 256), 256, 0, s>>>(m, nnz, keys2, dem, dem_off, chunk_w, (unsigned long long *)P);
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
    A.dem = (int32_t *)(ws + L.dem);
    A.dem_off = (int64_t *)(ws + L.dem_off);
    A.V = V;
    A.best_v = (int64_t *)(ws + L.best_v);
    A.best_p = (int32_t *)(ws + L.best_p);
    A.active = (int32_t *)(ws + L.active);
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
        k_g_row_best<<<(m + 3) / 4, 4 * kWave, 0, s>>>(m, V, A.best_v, A.best_p, A.active);
    }
    {
        const size_t lds = sizeof(int64_t) * (size_t)m;
        MPT_HIP_TRY(hipFuncSetAttribute((const void *)k_g_merge_loop, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
        LaunchScope ls("g_merge_loop", (double)(m - 1), s);
        k_g_merge_loop<<<1, kLoopThreads, lds, s>>>(A);
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
    if (workspace_bytes < sizeof(GHeader)) return fail(MPT_E_WORKSPACE, "workspace has %zu bytes, needs %zu",
                                                       workspace_bytes, sizeof(GHeader));
    hipStream_t s = (hipStream_t)stream;
    GHeader *h = (GHeader *)workspace;
    {
        const size_t lds = sizeof(int64_t) * (size_t)m;
        MPT_HIP_TRY(hipFuncSetAttribute((const void *)k_g_prim, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
        LaunchScope ls("g_prim", 8.0 * (double)m * m, s);
        k_g_prim<<<1, kLoopThreads, lds, s>>>(m, P, &h->total);
    }
    MPT_HIP_TRY(hipGetLastError());
    unsigned long long total = 0;
    MPT_HIP_TRY(hipMemcpyAsync(&total, &h->total, sizeof total, hipMemcpyDeviceToHost, s));
    MPT_HIP_TRY(hipStreamSynchronize(s));
    *mst_weight = (int64_t)total;
    return MPT_OK;
}
