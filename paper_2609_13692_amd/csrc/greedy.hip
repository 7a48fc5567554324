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
// The greedy's merges run in rounds over the whole chip: every round merges
// all pairs of clusters that are each other's best partner (merge values
// never grow, Theorem 6 part i, so each such pair is one of the greedy's
// merges), intersects their signatures, recomputes the new rows and only
// the best partners that can have changed. A sort of the merges by the
// lowest priority in their subtrees then gives the greedy's sequence.
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
using mptlib::kSegMax;
using mptlib::kSortTile;
using mptlib::seg_rank;
using mptlib::sort_keys;

constexpr int kWave = 64;

enum : uint32_t { GERR_INVALID = 1u, GERR_RANGE = 2u, GERR_DUP = 4u, GERR_WEIGHT = 8u, GERR_OVERFLOW = 16u };

// first 256 bytes of the workspace
struct GHeader {
    uint32_t err;
    uint32_t pad0;
    unsigned long long total;    // sum_i w(R_i), unsigned so it cannot wrap before the check
    int32_t n_rec;               // merge records so far
    int32_t lo;                  // first record of the current round
    int32_t n_resc[2];           // rows marked for a rescan, by round parity
    int32_t last_pairs;          // merges of the last finished round
    int32_t bv_done;             // spanning tree: 1 once one component is left
    unsigned long long dcursor;  // next free slot of the packed D lists
    int64_t max_len;             // longest request list
    int64_t pad[25];
};
static_assert(sizeof(GHeader) == 256, "header is one 256-byte block");

inline int64_t pow2_at_least(int64_t n) {
    int64_t p = 1;
    while (p < n) p <<= 1;
    return p;
}

struct GLayout {
    size_t keys1, keys2, sig, sig_len, dem, dem_off, V, best_v, best_p, active, last, touched, resc, dbuf, d_off,
        d_len, rec32, rec64, total;
    int64_t npad;
};
constexpr int kRec32 = 7;    // int32 arrays of the merge records
constexpr int kRec64 = 3;    // int64 arrays of the merge records

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
    L.last = take(4 * mm);
    L.touched = take(4 * mm);
    L.resc = take(4 * mm);
    L.dbuf = take(4 * (size_t)std::max<int64_t>(nnz, 1));
    L.d_off = take(8 * (2 * mm));
    L.d_len = take(4 * (2 * mm));
    L.rec32 = take(4 * mm * kRec32);
    L.rec64 = take(8 * mm * kRec64);
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
    if (threadIdx.x == 0) { h->err = 0; h->total = 0; h->max_len = 0; }
}

__global__ void k_g_check_offsets(int m, int64_t nnz, const int64_t *req_off, GHeader *h) {
    bool ok = true;
    int64_t mx = 0;
    for (int i = threadIdx.x; i < m; i += blockDim.x) {
        const int64_t len = req_off[i + 1] - req_off[i];
        ok = ok && len >= 0;
        mx = len > mx ? len : mx;
    }
    if (threadIdx.x == 0) ok = ok && req_off[0] == 0 && req_off[m] == nnz;
    if (!ok) atomicOr(&h->err, GERR_INVALID);
    if (mx > 0) atomicMax((long long *)&h->max_len, (long long)mx);
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
// inside a request is two equal adjacent (request, chunk) keys. keys1 null:
// the request lists are already in sig (k_g_sig_short).
__global__ void k_g_lists(int m, int64_t nnz, const uint64_t *keys1, const uint64_t *keys2, int32_t *sig,
                          int32_t *sig_len, int32_t *dem, const int64_t *req_off, GHeader *h) {
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < nnz; j += (int64_t)gridDim.x * blockDim.x) {
        dem[j] = (int32_t)(keys2[j] & 0xffffffffu);
        if (!keys1) continue;
        sig[j] = (int32_t)(keys1[j] & 0xffffffffu);
        if (j > 0 && keys1[j] == keys1[j - 1]) atomicOr(&h->err, GERR_DUP);
    }
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < m; i += (int64_t)gridDim.x * blockDim.x)
        sig_len[i] = (int32_t)(req_off[i + 1] - req_off[i]);
}

// request lists when every request has at most kSegMax chunks: one wave
// per request ranks its chunks (chunk ids validated already)
__global__ void k_g_sig_short(int m, const int64_t *req_off, const int32_t *req_chunks, int32_t *sig, GHeader *h) {
    const int lane = (int)(threadIdx.x & (kWave - 1));
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) / kWave;
    for (int64_t i = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) / kWave; i < m; i += nwaves) {
        const int64_t o = req_off[i];
        const int n = (int)(req_off[i + 1] - o);
        const uint32_t c = lane < n ? (uint32_t)req_chunks[o + lane] : 0u;
        bool dup;
        const int pos = seg_rank(c, n, dup);
        if (lane < n) {
            sig[o + pos] = (int32_t)c;
            if (dup) atomicOr(&h->err, GERR_DUP);
        }
    }
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

// row a of P, a tile of kPairTile columns per workgroup: every chunk x of
// R_a adds w(x) to the columns of the requests in its demand list S_x (one
// wave per chunk, lanes along S_x), summed in LDS and written once. The
// row's tiles cover every column, so P needs no zeroing.
constexpr int kPairTile = 4096;
constexpr int kPairThreads = 256;
__global__ __launch_bounds__(kPairThreads) void k_g_pair_rows(int m, const int32_t *sig, const int64_t *req_off,
                                                              const int32_t *dem, const int64_t *dem_off,
                                                              const int64_t *w, int64_t *P) {
    __shared__ unsigned long long row[kPairTile];
    const int tiles = (m + kPairTile - 1) / kPairTile;
    const int64_t a = blockIdx.x / tiles;
    const int c0 = (int)(blockIdx.x % tiles) * kPairTile;
    const int width = min(kPairTile, m - c0);
    for (int j = threadIdx.x; j < width; j += kPairThreads) row[j] = 0ull;
    __syncthreads();
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    const int64_t s0 = req_off[a], s1 = req_off[a + 1];
    for (int64_t q = s0 + wid; q < s1; q += kPairThreads / kWave) {
        const int32_t x = sig[q];
        const unsigned long long wx = (unsigned long long)w[x];
        for (int64_t f = dem_off[x] + lane; f < dem_off[x + 1]; f += kWave) {
            const int b = dem[f] - c0;
            if (b >= 0 && b < width) atomicAdd(&row[b], wx);
        }
    }
    __syncthreads();
    int64_t *out = P + a * (int64_t)m + c0;
    for (int j = threadIdx.x; j < width; j += kPairThreads) out[j] = (int64_t)row[j];
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

// The greedy's merges in rounds. Merge values never grow (Theorem 6 part
// i): a cluster formed from A and B shares with any C at most what A and B
// each share with C. Order pairs by (value desc, smaller name asc, larger
// name asc), where a cluster's name is its smallest request; the sequential
// greedy merges the first pair in this order every time. A pair (a, b) in
// which each is the other's best partner stays so under every other merge,
// so the sequential greedy merges it at some point: every round merges all
// such mutual-best pairs of positive value at once (the first pair overall
// is always one), until no positive value is left. The rounds produce the
// greedy's merges, not its sequence; the sequence is the pair order itself.
// A merge X that forms a cluster taking part in a later merge Y of names
// p < q comes first: X's value is at least Y's, and if equal, the parts
// named p and q already shared that value when X was chosen (their
// signatures contain those of Y's clusters), so X's pair preceded (p, q).
struct Rac {
    int m;
    const int64_t *w;
    const int64_t *req_off;     // start of each cluster's signature in sig
    int32_t *sig;               // signatures, ascending, shrinking in place
    int32_t *sig_len;
    int64_t *V;                 // V[a][c] = w(I(a) ∩ I(c)) for live a, c
    int64_t *best_v;
    int32_t *best_p;
    int32_t *act;               // 1 while the name is a live cluster
    int32_t *last;              // last merge record into each name (-1: a leaf)
    int32_t *touched;           // round in which the name last merged
    int32_t *resc;              // rows whose best partner is recomputed this round
    // merge records, in the order the rounds produce them
    int32_t *ra, *rb, *rca, *rcb, *rpos, *rdal, *rdbl;
    int64_t *rgain, *rdao, *rdbo;
    int32_t *dbuf;              // D(v) = I(v) \ I(parent(v)), packed
    int64_t dcap;               // entries of dbuf (nnz: the D lists never need more)
    int64_t *d_off;
    int32_t *d_len;
    int32_t *merge_a, *merge_b;
    int64_t *gain;
    int32_t *node_parent;
    GHeader *h;
};

__device__ inline uint64_t lanes_below(int lane) { return (1ull << lane) - 1ull; }

// w(p ∩ q) for ascending lists: the shorter searched in the longer
__device__ inline int64_t inter_weight(const int32_t *p, int64_t np, const int32_t *q, int64_t nq, const int64_t *w) {
    if (np > nq) { const int32_t *t = p; p = q; q = t; const int64_t n = np; np = nq; nq = n; }
    int64_t s = 0;
    for (int64_t j = 0; j < np; ++j) {
        const int32_t y = p[j];
        if (find_sorted(q, nq, y) >= 0) s += w[y];
    }
    return s;
}

// pair order (gain, a, b): true when x comes after y in the greedy's order
// (smaller gain; equal gains, larger names)
__device__ inline bool after(int64_t xg, int32_t xa, int32_t xb, int64_t yg, int32_t ya, int32_t yb) {
    return xg < yg || (xg == yg && (xa > ya || (xa == ya && xb > yb)));
}

__global__ void k_rac_init(Rac R) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    for (int64_t r = t0; r < R.m; r += stride) { R.act[r] = 1; R.last[r] = -1; R.touched[r] = -1; R.rpos[r] = 0; }
    for (int64_t v = t0; v < 2 * (int64_t)R.m - 1; v += stride) { R.node_parent[v] = -1; R.d_off[v] = 0; R.d_len[v] = 0; }
    if (t0 == 0) {
        R.h->n_rec = 0;
        R.h->lo = 0;
        R.h->n_resc[0] = 0;
        R.h->n_resc[1] = 0;
        R.h->last_pairs = -1;
        R.h->dcursor = 0;
    }
}

// One wave per row a: if a and its best partner b > a are mutual best with
// positive value, a new merge record i (a, b, value) is taken, and the wave
// merges: I(C) = I(A) ∩ I(B) in place of I(A), D(B) = I(B) \ I(A) and
// D(A) = I(A) \ I(B) to the packed lists, and the merges that formed A and
// B. The pair test reads only values that no merge of the round writes
// (best values and partners; a partner b that a merge deactivates fails the
// test b > best partner as well), so merging while other waves still test
// finds the same pairs. Record numbers within a round follow the atomic
// order; the sequence is recovered by sorting on the pair order.
__global__ void k_rac_pairs_merge(Rac R, int round) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) / kWave;
    for (int64_t a = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) / kWave; a < R.m; a += nwaves) {
        int rec = -1;
        int32_t b = -1;
        if (lane == 0 && R.act[a] && R.best_v[a] > 0) {
            b = R.best_p[a];
            if (b > a && R.best_p[b] == (int32_t)a) {
                const int i = atomicAdd(&R.h->n_rec, 1);
                if (i >= R.m - 1) {
                    atomicOr(&R.h->err, GERR_INVALID);   // cannot happen
                } else {
                    R.ra[i] = (int32_t)a;
                    R.rb[i] = b;
                    R.rgain[i] = R.best_v[a];
                    rec = i;
                }
            }
        }
        rec = __shfl(rec, 0, kWave);
        if (rec < 0) continue;
        b = __shfl(b, 0, kWave);
        const int64_t i = rec;
        int32_t *sa = R.sig + R.req_off[a];
        const int32_t *sb = R.sig + R.req_off[b];
        const int64_t na = R.sig_len[a], nb = R.sig_len[b];
        int64_t kept = 0;
        for (int64_t base = 0; base < na; base += kWave) {
            const int64_t e = base + lane;
            kept += __popcll(__ballot(e < na && find_sorted(sb, nb, sa[e]) >= 0));
        }
        const int64_t dlen = na + nb - 2 * kept;
        unsigned long long dstart = 0;
        if (lane == 0) dstart = atomicAdd(&R.h->dcursor, (unsigned long long)dlen);
        dstart = __shfl(dstart, 0, kWave);
        if ((int64_t)dstart + dlen > R.dcap) {   // cannot happen for a valid run
            if (lane == 0) atomicOr(&R.h->err, GERR_INVALID);
            continue;
        }
        int64_t dcur = (int64_t)dstart;
        for (int64_t base = 0; base < nb; base += kWave) {
            const int64_t e = base + lane;
            int32_t x = 0;
            bool keep = false;
            if (e < nb) { x = sb[e]; keep = find_sorted(sa, na, x) < 0; }
            const uint64_t mk = __ballot(keep);
            if (keep) R.dbuf[dcur + __popcll(mk & lanes_below(lane))] = x;
            dcur += __popcll(mk);
        }
        const int64_t d_a_at = dcur;
        // in place: a lane writes at or below the entry it read, and the
        // entries above the current 64 are not written yet
        int64_t k = 0;
        for (int64_t base = 0; base < na; base += kWave) {
            const int64_t e = base + lane;
            int32_t x = 0;
            bool in_b = false;
            if (e < na) { x = sa[e]; in_b = find_sorted(sb, nb, x) >= 0; }
            const uint64_t mi = __ballot(in_b);
            const uint64_t mo = __ballot(e < na && !in_b);
            if (in_b) sa[k + __popcll(mi & lanes_below(lane))] = x;
            else if (e < na) R.dbuf[dcur + __popcll(mo & lanes_below(lane))] = x;
            k += __popcll(mi);
            dcur += __popcll(mo);
        }
        if (lane == 0) {
            R.sig_len[a] = (int32_t)kept;
            R.act[b] = 0;
            R.touched[a] = round;
            R.touched[b] = round;
            const int32_t ca = R.last[a], cb = R.last[b];
            R.rca[i] = ca;
            R.rcb[i] = cb;
            R.last[a] = (int32_t)i;
            R.rdbo[i] = (int64_t)dstart;
            R.rdbl[i] = (int32_t)(d_a_at - (int64_t)dstart);
            R.rdao[i] = d_a_at;
            R.rdal[i] = (int32_t)(dcur - d_a_at);
        }
    }
}

// the new clusters' rows against every live column. A value is positive
// only where both old values are; the row of a is written by its own merge
// (columns of clusters merged in the same round included: both sides
// compute the same value), the column entry of every other row here.
// The same launch marks the rows whose best partner may have changed: the
// new clusters and the rows whose best partner merged (no other row's best
// can change: values fall).
__global__ void k_rac_rows(Rac R, int round) {
    const int lo = R.h->lo, hi = min(R.h->n_rec, R.m - 1);
    const int64_t m = R.m;
    const int64_t total = (int64_t)(hi - lo) * m;
    const int64_t t0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x, stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t f = t0; f < total; f += stride) {
        const int64_t i = lo + f / m;
        const int32_t x = (int32_t)(f % m);
        const int32_t a = R.ra[i], b = R.rb[i];
        if (x == a || !R.act[x]) continue;
        const int64_t va = R.V[a * m + x], vb = R.V[b * m + x];
        const int64_t kept = R.sig_len[a];
        int64_t v = 0;
        if (va > 0 && vb > 0 && kept > 0)
            v = inter_weight(R.sig + R.req_off[a], kept, R.sig + R.req_off[x], R.sig_len[x], R.w);
        if (v != va) {
            R.V[a * m + x] = v;
            if (R.touched[x] != round) R.V[(int64_t)x * m + a] = v;
        }
    }
    if (hi <= lo) return;                        // nothing merged, nothing to rescan
    for (int64_t x = t0; x < m; x += stride) {
        if (!R.act[x]) continue;
        const int32_t p = R.best_p[x];
        if (R.touched[x] == round || (p >= 0 && R.touched[p] == round))
            R.resc[atomicAdd(&R.h->n_resc[round & 1], 1)] = (int32_t)x;
    }
}

// one workgroup per marked row: best partner, ties to the smallest index;
// each thread loads 8 columns before comparing them. Block 0 also closes
// the round: the next round's records start at the current count, and its
// rescan counter starts at 0.
constexpr int kRescThreads = 256;
__global__ __launch_bounds__(kRescThreads) void k_rac_rescan(Rac R, int round) {
    __shared__ int64_t sv[kRescThreads / kWave];
    __shared__ int32_t si[kRescThreads / kWave];
    const int n = R.h->n_resc[round & 1];
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        R.h->last_pairs = R.h->n_rec - R.h->lo;
        R.h->lo = R.h->n_rec;
        R.h->n_resc[(round + 1) & 1] = 0;
    }
    const int64_t m = R.m;
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    constexpr int U = 8;
    for (int j = blockIdx.x; j < n; j += gridDim.x) {
        const int32_t x = R.resc[j];
        const int64_t *row = R.V + x * m;
        int64_t v = -1;
        int32_t p = -1;
        for (int64_t d0 = threadIdx.x; d0 < m; d0 += (int64_t)kRescThreads * U) {
            int64_t val[U];
            int32_t live[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t d = d0 + (int64_t)u * kRescThreads;
                val[u] = d < m ? row[d] : -1;
                live[u] = d < m ? R.act[d] : 0;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t d = (int32_t)(d0 + (int64_t)u * kRescThreads);
                if (live[u] && d != x && better(val[u], d, v, p)) { v = val[u]; p = d; }
            }
        }
        wave_best(v, p);
        if (lane == 0) { sv[wid] = v; si[wid] = p; }
        __syncthreads();
        if (threadIdx.x == 0) {
            for (int k = 1; k < kRescThreads / kWave; ++k)
                if (better(sv[k], si[k], v, p)) { v = sv[k]; p = si[k]; }
            R.best_v[x] = v;
            R.best_p[x] = p;
        }
        __syncthreads();
    }
}

// position of every record in the greedy's sequence: the records before it
// in the pair order. Blocks take a tile of records (x) against a tile of
// others (y), held in LDS, and add their counts (positions start at 0).
constexpr int kRankThreads = 256;
__global__ __launch_bounds__(kRankThreads) void k_rac_rank(Rac R, int n) {
    __shared__ int64_t tg[kRankThreads];
    __shared__ int32_t ta[kRankThreads], tb[kRankThreads];
    const int i = blockIdx.x * kRankThreads + threadIdx.x;
    const int j0 = blockIdx.y * kRankThreads;
    const int j = j0 + threadIdx.x;
    if (j < n) { tg[threadIdx.x] = R.rgain[j]; ta[threadIdx.x] = R.ra[j]; tb[threadIdx.x] = R.rb[j]; }
    __syncthreads();
    if (i >= n) return;
    const int64_t g = R.rgain[i];
    const int32_t a = R.ra[i], b = R.rb[i];
    const int cnt = min(kRankThreads, n - j0);
    int pos = 0;
    for (int k = 0; k < cnt; ++k) pos += after(g, a, b, tg[k], ta[k], tb[k]) ? 1 : 0;
    if (pos) atomicAdd(&R.rpos[i], pos);
}

// tree node of merge record i is m + its position; leaves are 0 .. m - 1
__device__ inline int32_t rec_node(const Rac &R, int32_t rec, int32_t leaf) {
    return rec >= 0 ? R.m + R.rpos[rec] : leaf;
}

__global__ void k_rac_emit(Rac R, int n) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
        const int t = R.rpos[i];
        const int32_t a = R.ra[i], b = R.rb[i];
        R.merge_a[t] = a;
        R.merge_b[t] = b;
        R.gain[t] = R.rgain[i];
        const int32_t node = R.m + t;
        const int32_t na = rec_node(R, R.rca[i], a), nb = rec_node(R, R.rcb[i], b);
        R.node_parent[na] = node;
        R.node_parent[nb] = node;
        R.d_off[na] = R.rdao[i];
        R.d_len[na] = R.rdal[i];
        R.d_off[nb] = R.rdbo[i];
        R.d_len[nb] = R.rdbl[i];
    }
}

// Every remaining pair shares nothing: the merges take the two smallest
// live names in turn (n0, n1), (n0, n2), ... with gain 0, and every
// merged signature is empty, so D(child) is the child's whole signature
// (the root's whole signature if only one cluster is left) and the
// chain's own nodes emit nothing. Live names in ascending order, one
// round of the workgroup at a time.
constexpr int kChainThreads = 1024;
__global__ __launch_bounds__(kChainThreads) void k_rac_chain(Rac R, int t0) {
    __shared__ int scan_w[kChainThreads / kWave];
    __shared__ int32_t first_name;
    const int m = R.m, tid = threadIdx.x;
    if (tid == 0) first_name = -1;
    __syncthreads();
    int64_t dcur = (int64_t)R.h->dcursor;
    int done = 0;                                // live names ranked so far
    for (int base = 0; base < m; base += kChainThreads) {
        const int r = base + tid;
        const int live = r < m && R.act[r];
        const int len = live ? R.sig_len[r] : 0;
        int tot, ltot;
        const int rank = done + block_scan(live, &tot, scan_w);
        const int loff = block_scan(len, &ltot, scan_w);
        if (dcur + ltot > R.dcap) {              // cannot happen for a valid run
            if (tid == 0) atomicOr(&R.h->err, GERR_INVALID);
            return;
        }
        if (live) {
            const int32_t node = rec_node(R, R.last[r], r);
            const int32_t *src = R.sig + R.req_off[r];
            for (int e = 0; e < len; ++e) R.dbuf[dcur + loff + e] = src[e];
            R.d_off[node] = dcur + loff;
            R.d_len[node] = len;
            if (rank == 0) {
                first_name = r;
            } else {
                const int tt = t0 + rank - 1;    // the merge that takes r
                if (tt < m - 1) {
                    R.merge_b[tt] = r;
                    R.gain[tt] = 0;
                    R.node_parent[node] = m + tt;
                }
            }
        }
        done += tot;
        dcur += ltot;
        __syncthreads();
    }
    const int n_live = done;
    // the chain: node m+t0 holds the first two names, node m+t0+k holds
    // node m+t0+k-1 and the name of rank k+1
    for (int k = tid; k + 1 < n_live && t0 + k < m - 1; k += kChainThreads) {
        R.merge_a[t0 + k] = first_name;
        R.d_off[m + t0 + k] = dcur;
        R.d_len[m + t0 + k] = 0;
        if (k > 0) R.node_parent[m + t0 + k - 1] = m + t0 + k;
    }
    if (tid == 0 && n_live >= 2) R.node_parent[rec_node(R, R.last[first_name], first_name)] = m + t0;
    if (tid == 0 && t0 + n_live - 1 != m - 1) atomicOr(&R.h->err, GERR_INVALID);
}

// pi_i: walk from leaf i to the root, placing D(v) of every node on the
// path right to left (the root's list comes first); one wave per request.
// The zero-gain merges (nodes m + chain_from and up) emit nothing and
// every node above one of them is one of them, so a walk ends there.
__global__ void k_g_orders(int m, int64_t nnz, const int64_t *req_off, const int32_t *node_parent,
                           const int32_t *dbuf, const int64_t *d_off, const int32_t *d_len, int32_t *order_chunks,
                           int chain_from, GHeader *h) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
    if (i >= m) return;
    int64_t end = req_off[i + 1];
    const int64_t begin = req_off[i];
    int steps = 0;
    for (int v = (int)i; v >= 0 && steps < 2 * m; v = node_parent[v], ++steps) {
        if (v >= 2 * m - 1) { if (lane == 0) atomicOr(&h->err, GERR_INVALID); return; }
        if (v >= m + chain_from) break;
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

// Borůvka's rounds after the last component has formed change nothing:
// the hook kernel raises h->bv_done when a root finds no edge out of its
// component (P is complete, so that root's component holds every vertex),
// and the later rounds' kernels return at once.
__global__ void k_bv_init(int m, int32_t *comp, GHeader *h) {
    for (int v = blockIdx.x * blockDim.x + threadIdx.x; v < m; v += gridDim.x * blockDim.x) comp[v] = v;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        h->total = 0;
        h->bv_done = 0;
    }
}

__global__ void k_bv_reset(int m, int64_t *cw, uint32_t *ce, const GHeader *h) {
    if (h->bv_done) return;
    for (int v = blockIdx.x * blockDim.x + threadIdx.x; v < m; v += gridDim.x * blockDim.x) { cw[v] = -1; ce[v] = ~0u; }
}

// best edge of every vertex to another component (one wave per vertex),
// folded into its component's best weight
__global__ void k_bv_vertex(int m, const int64_t *P, const int32_t *comp, int64_t *vw, uint32_t *ve, int64_t *cw,
                            const GHeader *h) {
    if (h->bv_done) return;
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
                          uint32_t *ce, const GHeader *h) {
    if (h->bv_done) return;
    for (int u = blockIdx.x * blockDim.x + threadIdx.x; u < m; u += gridDim.x * blockDim.x) {
        const int32_t cu = comp[u];
        if (vw[u] >= 0 && vw[u] == cw[cu]) atomicMin(&ce[cu], ve[u]);
    }
}

// every component hooks onto the component across its best edge, except
// the smaller one of a mutual pair; the hooking side adds the edge weight
// (no early return here: a workgroup that saw bv_done raised by another
// one of this launch would skip hooks; with one component there are none)
__global__ void k_bv_hook(int m, const int32_t *comp, const int64_t *cw, const uint32_t *ce, int32_t *par,
                          GHeader *h) {
    for (int c = blockIdx.x * blockDim.x + threadIdx.x; c < m; c += gridDim.x * blockDim.x) {
        par[c] = c;
        if (comp[c] != c) continue;
        if (ce[c] == ~0u) {
            h->bv_done = 1;
            continue;
        }
        const int lo = (int)(ce[c] >> 14), hi = (int)(ce[c] & 0x3fffu);
        const int32_t d = comp[lo] == c ? comp[hi] : comp[lo];
        if (ce[d] == ce[c] && c < d) continue;           // d hooks onto c
        par[c] = d;
        atomicAdd(&h->total, (unsigned long long)cw[c]);
    }
}

// new component of every vertex: follow the hooks to a root
__global__ void k_bv_jump(int m, int32_t *comp, const int32_t *par, const GHeader *h) {
    if (h->bv_done) return;
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

int g_read_errors(GHeader *h, hipStream_t s, int64_t *request_total = nullptr, int64_t *max_len = nullptr) {
    GHeader hh;
    MPT_HIP_TRY(hipMemcpyAsync(&hh, h, sizeof hh, hipMemcpyDeviceToHost, s));
    MPT_HIP_TRY(hipStreamSynchronize(s));
    if (hh.err & GERR_INVALID) return fail(MPT_E_INVALID, "req_off is not a CSR offset array of length m+1 ending at nnz");
    if (hh.err & GERR_RANGE) return fail(MPT_E_RANGE, "a chunk id is outside [0, n_chunks)");
    if (hh.err & GERR_WEIGHT) return fail(MPT_E_WEIGHT, "a chunk weight is <= 0 or > 2^32");
    if (hh.err & GERR_DUP) return fail(MPT_E_DUP, "a chunk is repeated inside one request");
    if (hh.total >= (1ull << 61)) return fail(MPT_E_OVERFLOW, "sum of request weights reaches 2^61");
    if (request_total) *request_total = (int64_t)hh.total;
    if (max_len) *max_len = hh.max_len;
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
    int64_t max_len = 0;
    int rc = g_read_errors(h, s, nullptr, &max_len);
    if (rc) return rc;
    int32_t *sig = (int32_t *)(ws + L.sig), *sig_len = (int32_t *)(ws + L.sig_len), *dem = (int32_t *)(ws + L.dem);
    int64_t *dem_off = (int64_t *)(ws + L.dem_off);
    // short requests: the request lists by ranks inside each request, the
    // (request, chunk) keys unsorted and unused
    const bool short_lists = max_len <= kSegMax;
    {
        LaunchScope ls("g_sort", 2.0 * (double)L.npad, s);
        if (short_lists) k_g_sig_short<<<std::max(1, (m + 3) / 4), 4 * kWave, 0, s>>>(m, req_off, req_chunks, sig, h);
        else if ((rc = sort_keys(keys1, L.npad, s))) return rc;
        if ((rc = sort_keys(keys2, L.npad, s))) return rc;
    }
    k_g_lists<<<grid_for(std::max<int64_t>(nnz, m), 256), 256, 0, s>>>(m, nnz, short_lists ? nullptr : keys1, keys2, sig,
                                                                        sig_len, dem, req_off, h);
    k_g_dem_off<<<grid_for(n_chunks + 1, 256), 256, 0, s>>>(n_chunks, nnz, keys2, dem_off);
    MPT_HIP_TRY(hipGetLastError());
    if ((rc = g_read_errors(h, s, request_total))) return rc;
    if (P) {
        const int64_t mm = (int64_t)m * m;
        LaunchScope ls("g_pairs", 8.0 * (double)mm, s);
        const int64_t blocks = (int64_t)m * ((m + kPairTile - 1) / kPairTile);
        k_g_pair_rows<<<(unsigned)blocks, kPairThreads, 0, s>>>(m, sig, req_off, dem, dem_off, chunk_w, P);
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
    Rac R{};
    R.m = m;
    R.w = chunk_w;
    R.req_off = req_off;
    R.sig = (int32_t *)(ws + L.sig);
    R.sig_len = (int32_t *)(ws + L.sig_len);
    R.V = V;
    R.best_v = (int64_t *)(ws + L.best_v);
    R.best_p = (int32_t *)(ws + L.best_p);
    R.act = (int32_t *)(ws + L.active);
    R.last = (int32_t *)(ws + L.last);
    R.touched = (int32_t *)(ws + L.touched);
    R.resc = (int32_t *)(ws + L.resc);
    int32_t *r32 = (int32_t *)(ws + L.rec32);
    int32_t **f32[kRec32] = {&R.ra, &R.rb, &R.rca, &R.rcb, &R.rpos, &R.rdal, &R.rdbl};
    for (int k = 0; k < kRec32; ++k) *f32[k] = r32 + (size_t)k * m;
    int64_t *r64 = (int64_t *)(ws + L.rec64);
    int64_t **f64[kRec64] = {&R.rgain, &R.rdao, &R.rdbo};
    for (int k = 0; k < kRec64; ++k) *f64[k] = r64 + (size_t)k * m;
    R.dbuf = (int32_t *)(ws + L.dbuf);
    R.dcap = std::max<int64_t>(nnz, 1);
    R.d_off = (int64_t *)(ws + L.d_off);
    R.d_len = (int32_t *)(ws + L.d_len);
    R.merge_a = merge_a;
    R.merge_b = merge_b;
    R.gain = gain;
    R.node_parent = node_parent;
    R.h = (GHeader *)ws;
    {
        LaunchScope ls("g_row_best", 8.0 * (double)m * m, s);
        k_g_row_best<<<(m + 3) / 4, 4 * kWave, 0, s>>>(m, V, R.best_v, R.best_p);
        k_rac_init<<<grid_for(2 * (int64_t)m, 256), 256, 0, s>>>(R);
    }
    // rounds in batches without host synchronisation; a round that finds
    // no pair changes nothing, so the batch's last round tells whether the
    // rounds are over. Batches of 8, 8, 16 and then 32 rounds: few
    // synchronisations, at most 31 empty rounds (a few µs each) at the end.
    int n_rec = 0;
    {
        LaunchScope ls("g_rounds", (double)(m - 1), s);
        const int g_rec = std::max(1, std::min(4096, (m + 3) / 4));        // waves: one per row
        const int g_cols = grid_for((int64_t)m * std::max(1, m / 2), 256, 4096);   // (2048: 1% slower, 512: 17%)
        const int g_resc = std::max(1, std::min(m, 2048));                  // workgroups: one per marked row
        for (int round = 0;;) {
            const int batch = round < 16 ? 8 : round < 32 ? 16 : 32;
            for (int k = 0; k < batch; ++k, ++round) {
                k_rac_pairs_merge<<<g_rec, 4 * kWave, 0, s>>>(R, round);
                k_rac_rows<<<g_cols, 256, 0, s>>>(R, round);
                k_rac_rescan<<<g_resc, kRescThreads, 0, s>>>(R, round);
            }
            MPT_HIP_TRY(hipGetLastError());
            GHeader hh;
            MPT_HIP_TRY(hipMemcpyAsync(&hh, R.h, sizeof hh, hipMemcpyDeviceToHost, s));
            MPT_HIP_TRY(hipStreamSynchronize(s));
            if (hh.err) return fail(MPT_E_INTERNAL, "greedy rounds left an inconsistent state");   // cannot happen
            n_rec = std::min(hh.n_rec, m - 1);
            if (hh.last_pairs == 0) break;
            if (round > m + 32) return fail(MPT_E_INTERNAL, "greedy rounds do not end");   // cannot happen
        }
    }
    {
        LaunchScope ls("g_sequence", (double)m, s);
        if (n_rec > 0) {
            const unsigned tiles = (unsigned)((n_rec + kRankThreads - 1) / kRankThreads);
            k_rac_rank<<<dim3(tiles, tiles), kRankThreads, 0, s>>>(R, n_rec);
            k_rac_emit<<<grid_for(n_rec, 256), 256, 0, s>>>(R, n_rec);
        }
        k_rac_chain<<<1, kChainThreads, 0, s>>>(R, n_rec);
    }
    MPT_HIP_TRY(hipGetLastError());
    if (order_chunks) {
        LaunchScope ls("g_orders", 4.0 * (double)nnz, s);
        k_g_orders<<<(m + 3) / 4, 4 * kWave, 0, s>>>(m, nnz, req_off, node_parent, R.dbuf, R.d_off, R.d_len,
                                                     order_chunks, n_rec, R.h);
        MPT_HIP_TRY(hipGetLastError());
    }
    if ((rc = g_read_errors(R.h, s))) return rc;
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
    k_bv_init<<<gv, 256, 0, s>>>(m, comp, h);
    for (int r = 0; r < rounds; ++r) {
        LaunchScope ls("g_boruvka", 8.0 * (double)m * m, s);
        k_bv_reset<<<gv, 256, 0, s>>>(m, cw, ce, h);
        k_bv_vertex<<<(m + 3) / 4, 4 * kWave, 0, s>>>(m, P, comp, vw, ve, cw, h);
        k_bv_edge<<<gv, 256, 0, s>>>(m, comp, vw, ve, cw, ce, h);
        k_bv_hook<<<gv, 256, 0, s>>>(m, comp, cw, ce, par, h);
        k_bv_jump<<<gv, 256, 0, s>>>(m, comp, par, h);
    }
    MPT_HIP_TRY(hipGetLastError());
    unsigned long long total = 0;
    MPT_HIP_TRY(hipMemcpyAsync(&total, &h->total, sizeof total, hipMemcpyDeviceToHost, s));
    MPT_HIP_TRY(hipStreamSynchronize(s));
    *mst_weight = (int64_t)total;
    return MPT_OK;
}
