// libmpt.so, Sections 7-8 of "Prefix Sharing Is a Sorting Problem":
// layouts, serving schedules and the radix cache.
//   mpt_global_order_layout  every request sorted by one chunk order: chunk
//                            id, or popularity (the global-order baselines)
//   mpt_layout_cost          trie cost (Eq. 1) of any layout, and the DFS
//                            serving order of its trie (Theorem 7)
//   mpt_cache_simulate       the prefill bill of serving a layout through a
//                            radix cache with least-recently-used leaf
//                            eviction, for many (reorder window, capacity)
//                            pairs at once (Section 8, 8.1)
//
// Trie cost. Sorted lexicographically, request s shares with all earlier
// requests exactly the longest common prefix (LCP) with its predecessor, so
// it adds the trie nodes past that LCP: the cost is a sum over requests of
// the weights past their LCP, and the sorted order is a DFS order of the
// trie. Nodes get ids in that order.
//
// Radix cache. Serving a request touches its whole path, so an ancestor is
// never older than a descendant, and the least-recently-used leaf is the
// deepest of the least-recently-used nodes: the policy is plain LRU over
// nodes, with each request's path touched from the leaf up. Such a cache
// always holds the longest prefix of its recency stack that fits, so an
// access hits iff the distinct weight accessed since its node's previous
// access, plus its own, fits the capacity. That stack distance does not
// depend on the capacity: configurations with the same window share one
// schedule, one access log and one pass that prices all their capacities,
// every log entry on its own thread.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <vector>

#include "bitonic.h"
#include "common.h"
#include "mpt.h"
#include "seqsort.h"

namespace {

using mptlib::align256;
using mptlib::fail;
using mptlib::grid_for;
using mptlib::kSegMax;
using mptlib::kSortTile;
using mptlib::LaunchScope;
using mptlib::seg_rank;
using mptlib::sort_keys;
using mptlib::kSeqSortTile;
using mptlib::sort_requests;

constexpr int kWave = 64;

enum : uint32_t { LERR_INVALID = 1u, LERR_RANGE = 2u, LERR_WEIGHT = 8u, LERR_OVERFLOW = 16u };

struct LHeader {
    uint32_t err;
    uint32_t pad0;
    unsigned long long total;   // sum of the sequence weights
    unsigned long long cost;    // trie cost
    int64_t max_len;            // longest sequence
    int64_t pad[28];
};
static_assert(sizeof(LHeader) == 256, "header is one 256-byte block");

inline int64_t pow2_at_least(int64_t n) {
    int64_t p = 1;
    while (p < n) p <<= 1;
    return p;
}

struct LLayout {
    size_t ord, rank, lcp, base, pn, nw, mtree, crank, cinv, keys, sched, log_off, logs, acc_start, prev, next, accw,
        bnext, bsum, cfg_win, cfg_cap, cfg_off, cfg_list, costs, total;
    int64_t mpad, kpad;
};

// nnz bounds the trie's node count
LLayout l_layout(int m, int64_t n_chunks, int64_t nnz, int n_cfg) {
    LLayout L{};
    const size_t mm = (size_t)m, nz = (size_t)std::max<int64_t>(nnz, 1), nc = (size_t)std::max(n_cfg, 0);
    L.mpad = std::max<int64_t>(pow2_at_least(m), kSeqSortTile);
    L.kpad = std::max<int64_t>(
        pow2_at_least(std::max(std::max<int64_t>(nnz, n_chunks), (int64_t)nc * std::max<int64_t>(m, nnz))), kSortTile);
    const size_t nblk = (nz + 255) / 256;       // sorted blocks of the access logs (kStackBlock entries)
    size_t o = align256(sizeof(LHeader));
    auto take = [&](size_t bytes) { size_t at = o; o = align256(o + std::max<size_t>(bytes, 1)); return at; };
    L.ord = take(4 * (size_t)L.mpad);
    L.rank = take(4 * mm);
    L.lcp = take(4 * mm);
    L.base = take(8 * (mm + 1));
    L.pn = take(4 * nz);
    L.nw = take(8 * nz);
    L.mtree = take(8 * (size_t)L.mpad);          // min segment tree over the LCPs
    L.crank = take(4 * (size_t)n_chunks);
    L.cinv = take(4 * (size_t)n_chunks);
    L.keys = take(8 * (size_t)L.kpad);
    L.sched = take(4 * nc * mm);
    L.log_off = take(8 * nc * mm);
    L.logs = take(4 * nc * nz);
    L.acc_start = take(4 * nc * nz);
    L.prev = take(4 * nc * nz);
    L.next = take(4 * nc * nz);
    L.accw = take(8 * nc * nz);
    L.bnext = take(4 * nc * nblk * 256);
    L.bsum = take(8 * nc * nblk * 256);
    L.cfg_win = take(8 * nc);
    L.cfg_cap = take(8 * nc);
    L.cfg_off = take(4 * (nc + 1));
    L.cfg_list = take(4 * nc);
    L.costs = take(8 * nc);
    L.total = o;
    return L;
}

// ---------------------------------------------------------------------------
// validation

__global__ void k_l_header(LHeader *h) {
    if (threadIdx.x == 0) { h->err = 0; h->total = 0; h->cost = 0; h->max_len = 0; }
}

__global__ void k_l_check_offsets(int m, int64_t nnz, const int64_t *off, LHeader *h) {
    bool ok = true;
    int64_t mx = 0;
    for (int i = threadIdx.x; i < m; i += blockDim.x) {
        const int64_t len = off[i + 1] - off[i];
        ok = ok && len >= 0;
        mx = len > mx ? len : mx;
    }
    if (threadIdx.x == 0) ok = ok && off[0] == 0 && off[m] == nnz;
    if (!ok) atomicOr(&h->err, LERR_INVALID);
    if (mx > 0) atomicMax((long long *)&h->max_len, (long long)mx);
}

__global__ void k_l_check_chunks(int64_t nnz, int64_t n_chunks, const int32_t *seqs, const int64_t *w, LHeader *h) {
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < nnz; j += (int64_t)gridDim.x * blockDim.x) {
        const int32_t x = seqs[j];
        if (x < 0 || (int64_t)x >= n_chunks) { atomicOr(&h->err, LERR_RANGE); continue; }
        if (w) {
            const int64_t wx = w[x];
            if (wx <= 0 || wx > MPT_MAX_CHUNK_WEIGHT) atomicOr(&h->err, LERR_WEIGHT);
            else atomicAdd(&h->total, (unsigned long long)wx);
        }
    }
}

int l_read_errors(LHeader *h, hipStream_t s, int64_t *max_len = nullptr) {
    LHeader hh;
    MPT_HIP_TRY(hipMemcpyAsync(&hh, h, sizeof hh, hipMemcpyDeviceToHost, s));
    MPT_HIP_TRY(hipStreamSynchronize(s));
    if (hh.err & LERR_INVALID) return fail(MPT_E_INVALID, "offsets are not a CSR offset array of length m+1 ending at nnz");
    if (hh.err & LERR_RANGE) return fail(MPT_E_RANGE, "a chunk id is outside [0, n_chunks)");
    if (hh.err & LERR_WEIGHT) return fail(MPT_E_WEIGHT, "a chunk weight is <= 0 or > 2^32");
    if (hh.total >= (1ull << 61)) return fail(MPT_E_OVERFLOW, "sum of sequence weights reaches 2^61");
    if (max_len) *max_len = hh.max_len;
    return MPT_OK;
}

// ---------------------------------------------------------------------------
// global-order layouts

__global__ void k_l_fill_i32(int32_t *p, int64_t n, int32_t v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = v;
}

__global__ void k_l_fill_u64(uint64_t *p, int64_t n, uint64_t v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = v;
}

// demand of every chunk (into the rank array, reused below)
__global__ void k_l_count(int64_t nnz, const int32_t *chunks, int32_t *cnt) {
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < nnz; j += (int64_t)gridDim.x * blockDim.x)
        atomicAdd(&cnt[chunks[j]], 1);
}

// popularity key of chunk x: demand descending, then id ascending
__global__ void k_l_pop_keys(int64_t n_chunks, const int32_t *cnt, uint64_t *keys) {
    for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < n_chunks; x += (int64_t)gridDim.x * blockDim.x)
        keys[x] = ((uint64_t)(0x7fffffffu - (uint32_t)cnt[x]) << 32) | (uint32_t)x;
}

// sorted popularity keys -> rank[x]
__global__ void k_l_pop_rank(int64_t n_chunks, const uint64_t *keys, int32_t *rank) {
    for (int64_t r = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; r < n_chunks; r += (int64_t)gridDim.x * blockDim.x)
        rank[(uint32_t)(keys[r] & 0xffffffffu)] = (int32_t)r;
}

// key of slot j: its request in the high 32 bits, the chunk's position in
// the order in the low 32 bits (for the id order the position is the id)
__global__ void k_l_layout_keys(int m, int64_t nnz, int64_t npad, const int64_t *req_off, const int32_t *chunks,
                                const int32_t *rank, int kind, uint64_t *keys) {
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < npad; j += (int64_t)gridDim.x * blockDim.x) {
        if (j >= nnz) { keys[j] = ~0ull; continue; }
        int lo = 0, hi = m - 1;                 // request of slot j
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (req_off[mid] <= j) lo = mid; else hi = mid - 1;
        }
        const uint32_t x = (uint32_t)chunks[j];
        const uint32_t r = kind == MPT_ORDER_ID ? x : (uint32_t)rank[x];
        keys[j] = ((uint64_t)lo << 32) | r;
    }
}

// sorted keys -> sequences (position -> chunk through the inverse of rank)
__global__ void k_l_layout_out(int64_t nnz, const uint64_t *keys, const int32_t *inv, int kind, int32_t *seqs) {
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < nnz; j += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t r = (uint32_t)(keys[j] & 0xffffffffu);
        seqs[j] = kind == MPT_ORDER_ID ? (int32_t)r : inv[r];
    }
}

// the layout when every request has at most kSegMax chunks: one wave per
// request ranks its chunks by their position in the order (the id, or the
// popularity rank), ties by slot
__global__ void k_l_layout_short(int m, const int64_t *req_off, const int32_t *chunks, const int32_t *rank, int kind,
                                 int32_t *seqs) {
    const int lane = (int)(threadIdx.x & (kWave - 1));
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) / kWave;
    for (int64_t i = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) / kWave; i < m; i += nwaves) {
        const int64_t o = req_off[i];
        const int n = (int)(req_off[i + 1] - o);
        const int32_t x = lane < n ? chunks[o + lane] : 0;
        const uint32_t r = lane < n ? (kind == MPT_ORDER_ID ? (uint32_t)x : (uint32_t)rank[x]) : 0u;
        bool dup;
        const int pos = seg_rank(r, n, dup);
        if (lane < n) seqs[o + pos] = x;
    }
}

__global__ void k_l_inverse(int64_t n, const int32_t *rank, int32_t *inv) {
    for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < n; x += (int64_t)gridDim.x * blockDim.x)
        inv[rank[x]] = (int32_t)x;
}

// ---------------------------------------------------------------------------
// trie cost, ranks, node ids

// position s of the sorted order: LCP with s-1, the weight it adds, the
// count of its new nodes (into base[s + 1] for the scan), rank of its request
__global__ void k_l_lcp(int m, const int32_t *ord, const int64_t *off, const int32_t *seqs, const int64_t *w,
                        int32_t *lcp, int64_t *base, int32_t *rank, LHeader *h) {
    for (int s = blockIdx.x * blockDim.x + threadIdx.x; s < m; s += gridDim.x * blockDim.x) {
        const int i = ord[s];
        const int64_t li = off[i + 1] - off[i];
        const int32_t *si = seqs + off[i];
        int64_t l = 0;
        if (s > 0) {
            const int p = ord[s - 1];
            const int64_t lp = off[p + 1] - off[p];
            const int32_t *sp = seqs + off[p];
            while (l < li && l < lp && si[l] == sp[l]) ++l;
        }
        unsigned long long add = 0;
        for (int64_t j = l; j < li; ++j) add += (unsigned long long)w[si[j]];
        if (add) atomicAdd(&h->cost, add);
        lcp[s] = (int32_t)l;
        base[s + 1] = li - l;
        rank[i] = s;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) base[0] = 0;
}

// in-place inclusive scan of base[1 .. m] (one workgroup): base[s] becomes
// the first node id of sorted position s, base[m] the node count
__global__ __launch_bounds__(1024) void k_l_scan(int m, int64_t *base) {
    __shared__ int64_t sw[16];
    __shared__ int64_t carry;
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (int b0 = 1; b0 <= m; b0 += blockDim.x) {
        const int i = b0 + threadIdx.x;
        int64_t x = i <= m ? base[i] : 0;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const int64_t y = __shfl_up(x, o, kWave);
            if (lane >= o) x += y;
        }
        if (lane == kWave - 1) sw[wid] = x;
        __syncthreads();
        int64_t before = carry;
        for (int k = 0; k < wid; ++k) before += sw[k];
        if (i <= m) base[i] = before + x;
        __syncthreads();
        if (threadIdx.x == blockDim.x - 1) carry = before + x;
        __syncthreads();
    }
}

// weight of every trie node: sorted position s creates the nodes of depths
// LCP .. len-1 of its request, with ids base[s] + (j - LCP)
__global__ void k_l_node_weights(int m, const int32_t *ord, const int64_t *off, const int32_t *seqs, const int64_t *w,
                                 const int32_t *lcp, const int64_t *base, int64_t *nw) {
    for (int s = blockIdx.x * blockDim.x + threadIdx.x; s < m; s += gridDim.x * blockDim.x) {
        const int i = ord[s];
        const int64_t li = off[i + 1] - off[i], l = lcp[s], b = base[s];
        for (int64_t j = l; j < li; ++j) nw[b + (j - l)] = w[seqs[off[i] + j]];
    }
}

// node ids of every request's path. Request s (in sorted order) creates the
// nodes of depths LCP(s) .. len-1, with ids base[s] + (j - LCP(s)); a
// shallower depth j < LCP(s) holds the node of the previous request, and so
// on back to the last request t <= s with LCP(t) <= j, which created it. A
// min segment tree over the LCPs finds t in O(log m), so every slot of the
// layout is one independent thread.
constexpr int kTreeBlock = 2048;               // leaves of the subtree one workgroup builds in LDS

// leaves mtree[mpad + t] = LCP(t) (padding: INT32_MAX) and the levels of each
// workgroup's subtree of kTreeBlock leaves (heap order: node n has children
// 2n, 2n + 1; the root is 1)
__global__ __launch_bounds__(1024) void k_l_mtree_low(int m, int64_t mpad, const int32_t *lcp, int32_t *mtree) {
    __shared__ int32_t t[kTreeBlock];
    const int64_t S = min<int64_t>(kTreeBlock, mpad);
    const int64_t first = (int64_t)blockIdx.x * S;
    for (int64_t e = threadIdx.x; e < S; e += blockDim.x) {
        const int64_t leaf = first + e;
        const int32_t v = leaf < m ? lcp[leaf] : INT32_MAX;
        t[e] = v;
        mtree[mpad + leaf] = v;
    }
    __syncthreads();
    for (int64_t len = S >> 1, k = 1; len >= 1; len >>= 1, ++k) {
        int32_t v = 0;
        const int64_t e = threadIdx.x;
        if (e < len) v = min(t[2 * e], t[2 * e + 1]);
        __syncthreads();
        if (e < len) {
            t[e] = v;
            mtree[(mpad >> k) + (first >> k) + e] = v;
        }
        __syncthreads();
    }
}

// the levels above the subtrees, one workgroup
__global__ __launch_bounds__(1024) void k_l_mtree_top(int64_t top, int32_t *mtree) {
    for (int64_t len = top >> 1; len >= 1; len >>= 1) {
        for (int64_t n = len + threadIdx.x; n < 2 * len; n += blockDim.x) mtree[n] = min(mtree[2 * n], mtree[2 * n + 1]);
        __syncthreads();
    }
}

// last position t <= r whose LCP is at most j (exists: LCP(0) = 0)
__device__ inline int64_t last_at_most(const int32_t *mtree, int64_t mpad, int64_t r, int32_t j) {
    int64_t n = mpad + r;
    if (mtree[n] <= j) return r;
    while (n > 1) {
        if ((n & 1) && mtree[n - 1] <= j) { n -= 1; break; }   // the left neighbour's subtree holds one
        n >>= 1;
    }
    while (n < mpad) n = mtree[2 * n + 1] <= j ? 2 * n + 1 : 2 * n;
    return n - mpad;
}

__global__ void k_l_paths(int m, int64_t nnz, int64_t mpad, const int64_t *off, const int32_t *rank, const int32_t *lcp,
                          const int64_t *base, const int32_t *mtree, int32_t *pn) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < nnz; k += (int64_t)gridDim.x * blockDim.x) {
        // the request holding slot k: the last i with off[i] <= k
        int lo = 0, hi = m - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (off[mid] <= k) lo = mid; else hi = mid - 1;
        }
        const int64_t j = k - off[lo];
        const int64_t s = rank[lo];
        const int64_t t = j < lcp[s] ? last_at_most(mtree, mpad, s - 1, (int32_t)j) : s;
        pn[k] = (int32_t)(base[t] + (j - lcp[t]));
    }
}

// ---------------------------------------------------------------------------
// schedules and access logs

// key of request i under configuration c: window index, then the request's
// position in the DFS order (windowed DFS = sort inside every window)
__global__ void k_l_sched_keys(int m, int n_cfg, int64_t npad, const int64_t *windows, const int32_t *rank,
                               uint64_t *keys) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < npad; e += (int64_t)gridDim.x * blockDim.x) {
        if (e >= (int64_t)n_cfg * m) { keys[e] = ~0ull; continue; }
        const int c = (int)(e / m), i = (int)(e % m);
        const int64_t W = windows[c];
        const uint64_t win = (uint64_t)(i / W);
        keys[e] = ((uint64_t)c << 56) | (win << 28) | (uint64_t)rank[i];
    }
}

// sorted keys -> schedule of every configuration (request ids) and the
// access-log length of each served request
__global__ void k_l_sched_out(int m, int n_cfg, const uint64_t *keys, const int32_t *ord, const int64_t *off,
                              int32_t *sched, int64_t *log_off) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < (int64_t)n_cfg * m;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int r = (int)(keys[e] & ((1u << 28) - 1u));
        const int i = ord[r];
        sched[e] = i;
        log_off[e] = off[i + 1] - off[i];
    }
}

// exclusive scan of the log lengths of every configuration (one workgroup
// per configuration)
__global__ __launch_bounds__(1024) void k_l_log_scan(int m, int64_t *log_off) {
    __shared__ int64_t sw[16];
    __shared__ int64_t carry;
    int64_t *a = log_off + (int64_t)blockIdx.x * m;
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (int b0 = 0; b0 < m; b0 += blockDim.x) {
        const int i = b0 + threadIdx.x;
        const int64_t v = i < m ? a[i] : 0;
        int64_t x = v;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const int64_t y = __shfl_up(x, o, kWave);
            if (lane >= o) x += y;
        }
        if (lane == kWave - 1) sw[wid] = x;
        __syncthreads();
        int64_t before = carry;
        for (int k = 0; k < wid; ++k) before += sw[k];
        if (i < m) a[i] = before + x - v;
        __syncthreads();
        if (threadIdx.x == blockDim.x - 1) carry = before + x;
        __syncthreads();
    }
}

// the access log of every configuration: served requests in order, each
// path from its leaf up to the root
__global__ void k_l_logs(int m, int n_cfg, int64_t nnz, const int32_t *sched, const int64_t *log_off,
                         const int64_t *off, const int32_t *pn, int32_t *logs, int32_t *acc_start) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < (int64_t)n_cfg * m;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int c = (int)(e / m);
        const int i = sched[e];
        const int64_t li = off[i + 1] - off[i], at = log_off[e];
        int32_t *dst = logs + (int64_t)c * nnz + at;
        int32_t *st = acc_start + (int64_t)c * nnz + at;
        const int32_t *path = pn + off[i];
        for (int64_t j = 0; j < li; ++j) {
            dst[j] = path[li - 1 - j];
            st[j] = (int32_t)at;                 // where the request's accesses start
        }
    }
}

// ---------------------------------------------------------------------------
// the radix cache by stack distances
//
// Serving a request touches its whole path, each node of it more recently
// than its descendants, and every miss is inserted before the cache evicts
// (least-recently-used leaf first, which is the least-recently-used node,
// since an ancestor is never older than its descendants). By induction over
// the requests, the cache after each request holds exactly the longest
// prefix of the recency stack (nodes by latest access, most recent first)
// whose weight fits the capacity: the stack property of LRU (Mattson et al.,
// 1970), here with weights. So node v of the request whose accesses start at
// log position s is a hit iff it was accessed before and the nodes above it
// in the stack together with v fit: D + w(v) <= capacity, where D is the
// weight of the distinct nodes accessed between v's previous access p and s,
// i.e. the sum of w_j over log entries p < j < s whose node is not accessed
// again before s (next_j >= s). D does not depend on the capacity: one pass
// over a schedule's log bills all its capacities.

constexpr int kStackBlock = 256;               // log entries per sorted block
static_assert(kStackBlock == 256, "the lockstep searches of k_l_bill take 9 halvings");

// sort keys of the access logs of schedules d0 .. d0 + nd - 1: (schedule,
// node, log position); the padding sorts last
__global__ void k_l_acc_keys(int64_t nnz, int d0, int nd, int be, int bn, int64_t npad, const int32_t *logs,
                             uint64_t *keys) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < npad; k += (int64_t)gridDim.x * blockDim.x) {
        if (k >= (int64_t)nd * nnz) { keys[k] = ~0ull; continue; }
        const int64_t dl = k / nnz, e = k % nnz;
        const uint64_t v = (uint64_t)logs[(d0 + dl) * nnz + e];
        keys[k] = ((uint64_t)dl << (bn + be)) | (v << be) | (uint64_t)e;
    }
}

// previous and next access of the same node (-1 / nnz when there is none);
// schedule d0 + dl holds sorted positions [dl nnz, (dl + 1) nnz)
__global__ void k_l_prev_next(int64_t nnz, int d0, int nd, int be, const uint64_t *keys, int32_t *prev,
                              int32_t *next) {
    const uint64_t emask = (1ull << be) - 1ull;
    const int64_t n = (int64_t)nd * nnz;
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < n; k += (int64_t)gridDim.x * blockDim.x) {
        const uint64_t key = keys[k], grp = key >> be;
        const int64_t at = (d0 + k / nnz) * nnz + (int64_t)(key & emask);
        const bool has_prev = (k % nnz) > 0 && (keys[k - 1] >> be) == grp;
        const bool has_next = (k + 1) % nnz != 0 && (keys[k + 1] >> be) == grp;
        prev[at] = has_prev ? (int32_t)(keys[k - 1] & emask) : -1;
        next[at] = has_next ? (int32_t)(keys[k + 1] & emask) : (int32_t)nnz;
    }
}

// one workgroup per block of 256 log entries of one schedule: the entries'
// weights, and the block sorted by next access descending with the running
// weight sum, so that the weight of the entries with next >= s is a prefix
__global__ __launch_bounds__(kStackBlock) void k_l_stack_blocks(int64_t nnz, int64_t nblk, const int32_t *logs,
                                                                const int64_t *nw, const int32_t *next,
                                                                int64_t *accw, int32_t *bnext, int64_t *bsum) {
    __shared__ uint64_t t[kStackBlock];
    __shared__ int64_t ws[kStackBlock];
    const int64_t d = blockIdx.x / nblk, b = blockIdx.x % nblk;
    const int64_t j = b * kStackBlock + threadIdx.x;
    const int64_t at = d * nnz + j;
    int64_t w = 0;
    int32_t nx = -1;                                     // padding: never counted
    if (j < nnz) {
        w = nw[logs[at]];
        nx = next[at];
        accw[at] = w;
    }
    ws[threadIdx.x] = w;
    // key: next access in the high half (biased so that -1 sorts lowest),
    // entry index in the low half; sorted descending
    t[threadIdx.x] = ((uint64_t)(uint32_t)(nx + 1) << 32) | (uint64_t)threadIdx.x;
    __syncthreads();
    for (int k = 2; k <= kStackBlock; k <<= 1)
        for (int s = k >> 1; s > 0; s >>= 1) {
            const int i = threadIdx.x, pj = i ^ s;
            if (pj > i) {
                const bool desc = (i & k) == 0;
                const uint64_t a = t[i], c = t[pj];
                if (desc ? (a < c) : (a > c)) { t[i] = c; t[pj] = a; }
            }
            __syncthreads();
        }
    const uint64_t key = t[threadIdx.x];
    int64_t x = ws[key & 0xffffffffull];
    // inclusive scan of the weights in sorted order
    __shared__ int64_t sw[kStackBlock / kWave];
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int64_t y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    if (lane == kWave - 1) sw[wid] = x;
    __syncthreads();
    for (int k = 0; k < wid; ++k) x += sw[k];
    const int64_t out = d * nblk * kStackBlock + j;
    bnext[out] = (int32_t)(key >> 32) - 1;
    bsum[out] = x;
}

// one thread per log entry of one schedule: its stack distance, then its
// bill under every capacity of the schedule, summed per workgroup in LDS
// and added to the configurations' costs
constexpr int kBillThreads = 256;
__global__ __launch_bounds__(kBillThreads) void k_l_bill(int64_t nnz, int64_t nblk, const int32_t *prev,
                                                         const int32_t *next, const int32_t *acc_start,
                                                         const int64_t *accw, const int32_t *bnext,
                                                         const int64_t *bsum, const int32_t *cfg_off,
                                                         const int32_t *cfg_list, const int64_t *caps,
                                                         unsigned long long *costs) {
    __shared__ unsigned long long acc[MPT_CACHE_MAX_CONFIGS];
    const int d = blockIdx.y;
    const int c0 = cfg_off[d], nc = cfg_off[d + 1] - c0;
    for (int k = threadIdx.x; k < nc; k += kBillThreads) acc[k] = 0ull;
    __syncthreads();
    const int64_t e = blockIdx.x * (int64_t)kBillThreads + threadIdx.x;
    if (e < nnz) {
        const int64_t base = (int64_t)d * nnz;
        const int64_t w = accw[base + e];
        const int64_t p = prev[base + e];
        int64_t dist = -1;                               // -1: first access, a miss everywhere
        if (p >= 0) {
            const int64_t s = acc_start[base + e];
            dist = 0;
            // a range of single entries, 8 loads in flight at a time
            auto singles = [&](int64_t from, int64_t to) {
                for (int64_t q = from; q < to; q += 8) {
                    int32_t nx[8];
                    int64_t wq[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        nx[u] = q + u < to ? next[base + q + u] : -1;
                        wq[u] = q + u < to ? accw[base + q + u] : 0;
                    }
#pragma unroll
                    for (int u = 0; u < 8; ++u) dist += nx[u] >= s ? wq[u] : 0;
                }
            };
            const int64_t j0 = p + 1;
            const int64_t first_full = (j0 + kStackBlock - 1) / kStackBlock * kStackBlock;
            const int64_t end_full = s / kStackBlock * kStackBlock;
            if (first_full >= end_full) {
                singles(j0, s);                          // no whole block in between
            } else {
                singles(j0, first_full);
                singles(end_full, s);
                // whole blocks: the prefix of each block with next >= s, four
                // binary searches in lockstep
                const int64_t bbase = (int64_t)d * nblk * kStackBlock;
                int64_t j = first_full;
                for (; j + 4 * kStackBlock <= end_full; j += 4 * kStackBlock) {
                    int lo[4] = {0, 0, 0, 0}, hi[4] = {kStackBlock, kStackBlock, kStackBlock, kStackBlock};
                    for (int it = 0; it <= 8; ++it) {           // log2(kStackBlock) + 1 halvings
                        int32_t v[4];
#pragma unroll
                        for (int u = 0; u < 4; ++u) {
                            const int mid = (lo[u] + hi[u]) >> 1;
                            v[u] = lo[u] < hi[u] ? bnext[bbase + j + u * kStackBlock + mid] : 0;
                        }
#pragma unroll
                        for (int u = 0; u < 4; ++u) {
                            if (lo[u] >= hi[u]) continue;
                            const int mid = (lo[u] + hi[u]) >> 1;
                            if (v[u] >= s) lo[u] = mid + 1; else hi[u] = mid;
                        }
                    }
#pragma unroll
                    for (int u = 0; u < 4; ++u)
                        if (lo[u] > 0) dist += bsum[bbase + j + u * kStackBlock + lo[u] - 1];
                }
                for (; j < end_full; j += kStackBlock) {
                    int lo = 0, hi = kStackBlock;              // first sorted entry with next < s
                    while (lo < hi) {
                        const int mid = (lo + hi) >> 1;
                        if (bnext[bbase + j + mid] >= s) lo = mid + 1; else hi = mid;
                    }
                    if (lo > 0) dist += bsum[bbase + j + lo - 1];
                }
            }
        }
        for (int k = 0; k < nc; ++k) {
            const bool miss = dist < 0 || dist + w > caps[cfg_list[c0 + k]];
            if (miss) atomicAdd(&acc[k], (unsigned long long)w);
        }
    }
    __syncthreads();
    for (int k = threadIdx.x; k < nc; k += kBillThreads)
        if (acc[k]) atomicAdd(&costs[cfg_list[c0 + k]], acc[k]);
}

// ---------------------------------------------------------------------------
// host side

int l_check(int m, int64_t n_chunks, int64_t nnz) {
    if (m < 1 || m > MPT_LAYOUT_MAX_M) return fail(MPT_E_INVALID, "m = %d outside [1, %d]", m, MPT_LAYOUT_MAX_M);
    if (n_chunks < 0 || n_chunks > MPT_MAX_CHUNKS) return fail(MPT_E_INVALID, "n_chunks = %lld out of range", (long long)n_chunks);
    if (nnz < 0 || nnz > (int64_t)INT32_MAX) return fail(MPT_E_INVALID, "nnz = %lld out of range", (long long)nnz);
    return MPT_OK;
}

int l_check_ws(const LLayout &L, void *ws, size_t bytes) {
    if (!ws) return fail(MPT_E_WORKSPACE, "workspace is NULL");
    if (((uintptr_t)ws & 255u) != 0) return fail(MPT_E_WORKSPACE, "workspace is not 256-byte aligned");
    if (bytes < L.total) return fail(MPT_E_WORKSPACE, "workspace has %zu bytes, needs %zu", bytes, L.total);
    return MPT_OK;
}

// validation + lexicographic order + LCPs + trie cost (+ node ids)
int l_prepare(int m, int64_t n_chunks, int64_t nnz, const int64_t *w, const int64_t *off, const int32_t *seqs,
              const LLayout &L, char *ws, hipStream_t s, bool paths, int64_t *trie_cost, int64_t *n_nodes) {
    LHeader *h = (LHeader *)ws;
    k_l_header<<<1, 64, 0, s>>>(h);
    k_l_check_offsets<<<1, 256, 0, s>>>(m, nnz, off, h);
    if (nnz > 0) k_l_check_chunks<<<grid_for(nnz, 256), 256, 0, s>>>(nnz, n_chunks, seqs, w, h);
    MPT_HIP_TRY(hipGetLastError());
    int rc = l_read_errors(h, s);
    if (rc) return rc;
    int32_t *ord = (int32_t *)(ws + L.ord), *rank = (int32_t *)(ws + L.rank), *lcp = (int32_t *)(ws + L.lcp);
    int64_t *base = (int64_t *)(ws + L.base);
    {
        LaunchScope ls("l_sort_requests", (double)m, s);
        if ((rc = sort_requests(ord, rank, m, L.mpad, off, seqs, s))) return rc;
    }
    {
        LaunchScope ls("l_lcp", (double)nnz, s);
        k_l_lcp<<<grid_for(m, 256), 256, 0, s>>>(m, ord, off, seqs, w, lcp, base, rank, h);
        k_l_scan<<<1, 1024, 0, s>>>(m, base);
    }
    MPT_HIP_TRY(hipGetLastError());
    if (paths) {
        int32_t *pn = (int32_t *)(ws + L.pn), *mtree = (int32_t *)(ws + L.mtree);
        int64_t *nw = (int64_t *)(ws + L.nw);
        LaunchScope ls("l_paths", (double)nnz, s);
        k_l_node_weights<<<grid_for(m, 256), 256, 0, s>>>(m, ord, off, seqs, w, lcp, base, nw);
        const int64_t sub = std::min<int64_t>(kTreeBlock, L.mpad);
        k_l_mtree_low<<<(unsigned)(L.mpad / sub), 1024, 0, s>>>(m, L.mpad, lcp, mtree);
        if (L.mpad > sub) k_l_mtree_top<<<1, 1024, 0, s>>>(L.mpad / sub, mtree);
        if (nnz > 0)
            k_l_paths<<<grid_for(nnz, 256), 256, 0, s>>>(m, nnz, L.mpad, off, rank, lcp, base, mtree, pn);
        MPT_HIP_TRY(hipGetLastError());
    }
    int64_t hv[2] = {0, 0};
    MPT_HIP_TRY(hipMemcpyAsync(&hv[0], &h->cost, sizeof(int64_t), hipMemcpyDeviceToHost, s));
    MPT_HIP_TRY(hipMemcpyAsync(&hv[1], &base[m], sizeof(int64_t), hipMemcpyDeviceToHost, s));
    MPT_HIP_TRY(hipStreamSynchronize(s));
    if (trie_cost) *trie_cost = hv[0];
    if (n_nodes) *n_nodes = hv[1];
    return MPT_OK;
}

}  // namespace

extern "C" size_t mpt_layout_workspace_bytes(int m, int64_t n_chunks, int64_t nnz, int n_configs) {
    if (m < 1 || m > MPT_LAYOUT_MAX_M || n_chunks < 0 || nnz < 0 || n_configs < 0 ||
        n_configs > MPT_CACHE_MAX_CONFIGS)
        return 0;
    return l_layout(m, n_chunks, nnz, n_configs).total;
}

extern "C" int mpt_global_order_layout(int m, int64_t n_chunks, int64_t nnz, const int64_t *req_off,
                                       const int32_t *req_chunks, int order_kind, int32_t *seqs, void *workspace,
                                       size_t workspace_bytes, void *stream) {
    mptlib::clear_error();
    int rc = l_check(m, n_chunks, nnz);
    if (rc) return rc;
    if (order_kind != MPT_ORDER_ID && order_kind != MPT_ORDER_POPULARITY)
        return fail(MPT_E_INVALID, "order_kind = %d is not MPT_ORDER_ID or MPT_ORDER_POPULARITY", order_kind);
    if (!req_off || (nnz > 0 && (!req_chunks || !seqs))) return fail(MPT_E_INVALID, "req_off, req_chunks and seqs must not be NULL");
    const LLayout L = l_layout(m, n_chunks, nnz, 0);
    if ((rc = l_check_ws(L, workspace, workspace_bytes))) return rc;
    hipStream_t s = (hipStream_t)stream;
    char *ws = (char *)workspace;
    LHeader *h = (LHeader *)ws;
    k_l_header<<<1, 64, 0, s>>>(h);
    k_l_check_offsets<<<1, 256, 0, s>>>(m, nnz, req_off, h);
    if (nnz > 0) k_l_check_chunks<<<grid_for(nnz, 256), 256, 0, s>>>(nnz, n_chunks, req_chunks, nullptr, h);
    MPT_HIP_TRY(hipGetLastError());
    int64_t max_len = 0;
    if ((rc = l_read_errors(h, s, &max_len))) return rc;
    if (nnz == 0) return MPT_OK;
    uint64_t *keys = (uint64_t *)(ws + L.keys);
    int32_t *rank = (int32_t *)(ws + L.crank), *inv = (int32_t *)(ws + L.cinv);
    const int64_t kpad = L.kpad;
    LaunchScope ls("l_global_order", (double)nnz, s);
    if (order_kind == MPT_ORDER_POPULARITY) {
        // (count, id) keys of the chunks, padded to a power of two
        const int64_t cpad = std::max<int64_t>(pow2_at_least(n_chunks), kSortTile);
        k_l_fill_i32<<<grid_for(n_chunks, 256), 256, 0, s>>>(rank, n_chunks, 0);
        k_l_count<<<grid_for(nnz, 256), 256, 0, s>>>(nnz, req_chunks, rank);
        k_l_fill_u64<<<grid_for(cpad, 256), 256, 0, s>>>(keys, cpad, ~0ull);
        k_l_pop_keys<<<grid_for(n_chunks, 256), 256, 0, s>>>(n_chunks, rank, keys);
        if ((rc = sort_keys(keys, cpad, s))) return rc;
        k_l_pop_rank<<<grid_for(n_chunks, 256), 256, 0, s>>>(n_chunks, keys, rank);
        if (max_len > kSegMax) k_l_inverse<<<grid_for(n_chunks, 256), 256, 0, s>>>(n_chunks, rank, inv);
    }
    if (max_len <= kSegMax) {
        k_l_layout_short<<<std::max(1, (m + 3) / 4), 4 * kWave, 0, s>>>(m, req_off, req_chunks, rank, order_kind, seqs);
        MPT_HIP_TRY(hipGetLastError());
        return MPT_OK;
    }
    k_l_layout_keys<<<grid_for(kpad, 256), 256, 0, s>>>(m, nnz, kpad, req_off, req_chunks, rank, order_kind, keys);
    if ((rc = sort_keys(keys, kpad, s))) return rc;
    k_l_layout_out<<<grid_for(nnz, 256), 256, 0, s>>>(nnz, keys, inv, order_kind, seqs);
    MPT_HIP_TRY(hipGetLastError());
    return MPT_OK;
}

extern "C" int mpt_layout_cost(int m, int64_t n_chunks, int64_t nnz, const int64_t *chunk_w, const int64_t *seq_off,
                               const int32_t *seqs, int32_t *dfs_order, int64_t *trie_cost, void *workspace,
                               size_t workspace_bytes, void *stream) {
    mptlib::clear_error();
    int rc = l_check(m, n_chunks, nnz);
    if (rc) return rc;
    if (!seq_off || !trie_cost || (nnz > 0 && !seqs) || (n_chunks > 0 && !chunk_w))
        return fail(MPT_E_INVALID, "seq_off, seqs, chunk_w and trie_cost must not be NULL");
    const LLayout L = l_layout(m, n_chunks, nnz, 0);
    if ((rc = l_check_ws(L, workspace, workspace_bytes))) return rc;
    hipStream_t s = (hipStream_t)stream;
    char *ws = (char *)workspace;
    if ((rc = l_prepare(m, n_chunks, nnz, chunk_w, seq_off, seqs, L, ws, s, false, trie_cost, nullptr))) return rc;
    if (dfs_order) {
        MPT_HIP_TRY(hipMemcpyAsync(dfs_order, ws + L.ord, sizeof(int32_t) * (size_t)m, hipMemcpyDeviceToDevice, s));
        MPT_HIP_TRY(hipStreamSynchronize(s));
    }
    return MPT_OK;
}

extern "C" int mpt_cache_simulate(int m, int64_t n_chunks, int64_t nnz, const int64_t *chunk_w,
                                  const int64_t *seq_off, const int32_t *seqs, int n_configs,
                                  const int64_t *windows, const int64_t *capacities, int64_t *costs,
                                  int64_t *trie_cost, void *workspace, size_t workspace_bytes, void *stream) {
    mptlib::clear_error();
    int rc = l_check(m, n_chunks, nnz);
    if (rc) return rc;
    if (n_configs < 1 || n_configs > MPT_CACHE_MAX_CONFIGS)
        return fail(MPT_E_INVALID, "n_configs = %d outside [1, %d]", n_configs, MPT_CACHE_MAX_CONFIGS);
    if (!seq_off || !windows || !capacities || !costs || (nnz > 0 && !seqs) || (n_chunks > 0 && !chunk_w))
        return fail(MPT_E_INVALID, "seq_off, seqs, chunk_w, windows, capacities and costs must not be NULL");
    for (int c = 0; c < n_configs; ++c)
        if (capacities[c] < 0) return fail(MPT_E_INVALID, "capacity %d is negative", c);
    const LLayout L = l_layout(m, n_chunks, nnz, n_configs);
    if ((rc = l_check_ws(L, workspace, workspace_bytes))) return rc;
    hipStream_t s = (hipStream_t)stream;
    char *ws = (char *)workspace;
    int64_t tc = 0, n_nodes = 0;
    if ((rc = l_prepare(m, n_chunks, nnz, chunk_w, seq_off, seqs, L, ws, s, true, &tc, &n_nodes))) return rc;
    if (trie_cost) *trie_cost = tc;
    // configurations: window <= 0 or > m means the whole stream. Equal
    // windows share one schedule (and log); cfg_off / cfg_list list the
    // configurations of every schedule.
    std::vector<int64_t> win;
    std::vector<int> sched_of(n_configs);
    for (int c = 0; c < n_configs; ++c) {
        const int64_t wc = (windows[c] <= 0 || windows[c] > m) ? m : windows[c];
        int d = 0;
        while (d < (int)win.size() && win[d] != wc) ++d;
        if (d == (int)win.size()) win.push_back(wc);
        sched_of[c] = d;
    }
    const int n_sched = (int)win.size();
    std::vector<int32_t> cfg_off(n_sched + 1, 0), cfg_list;
    for (int d = 0; d < n_sched; ++d) {
        for (int c = 0; c < n_configs; ++c)
            if (sched_of[c] == d) cfg_list.push_back(c);
        cfg_off[d + 1] = (int32_t)cfg_list.size();
    }
    std::vector<int64_t> capv(capacities, capacities + n_configs);
    int64_t *dev_win = (int64_t *)(ws + L.cfg_win), *dev_capacity = (int64_t *)(ws + L.cfg_cap);
    int32_t *dev_cfg_off = (int32_t *)(ws + L.cfg_off), *dev_cfg_list = (int32_t *)(ws + L.cfg_list);
    MPT_HIP_TRY(hipMemcpyAsync(dev_win, win.data(), sizeof(int64_t) * n_sched, hipMemcpyHostToDevice, s));
    MPT_HIP_TRY(hipMemcpyAsync(dev_capacity, capv.data(), sizeof(int64_t) * n_configs, hipMemcpyHostToDevice, s));
    MPT_HIP_TRY(hipMemcpyAsync(dev_cfg_off, cfg_off.data(), sizeof(int32_t) * (n_sched + 1), hipMemcpyHostToDevice, s));
    MPT_HIP_TRY(hipMemcpyAsync(dev_cfg_list, cfg_list.data(), sizeof(int32_t) * n_configs, hipMemcpyHostToDevice, s));
    uint64_t *keys = (uint64_t *)(ws + L.keys);
    int32_t *sched = (int32_t *)(ws + L.sched), *logs = (int32_t *)(ws + L.logs);
    int32_t *acc_start = (int32_t *)(ws + L.acc_start), *prev = (int32_t *)(ws + L.prev), *next = (int32_t *)(ws + L.next);
    int64_t *log_off = (int64_t *)(ws + L.log_off), *accw = (int64_t *)(ws + L.accw);
    const int32_t *ord = (const int32_t *)(ws + L.ord), *rank = (const int32_t *)(ws + L.rank);
    {
        LaunchScope ls("l_schedules", (double)n_sched * m, s);
        const int64_t spad = std::max<int64_t>(pow2_at_least((int64_t)n_sched * m), kSortTile);
        k_l_sched_keys<<<grid_for(spad, 256), 256, 0, s>>>(m, n_sched, spad, dev_win, rank, keys);
        if ((rc = sort_keys(keys, spad, s))) return rc;
        k_l_sched_out<<<grid_for((int64_t)n_sched * m, 256), 256, 0, s>>>(m, n_sched, keys, ord, seq_off, sched,
                                                                          log_off);
        k_l_log_scan<<<n_sched, 1024, 0, s>>>(m, log_off);
        if (nnz > 0)
            k_l_logs<<<grid_for((int64_t)n_sched * m, 256), 256, 0, s>>>(m, n_sched, nnz, sched, log_off, seq_off,
                                                                         (const int32_t *)(ws + L.pn), logs, acc_start);
    }
    MPT_HIP_TRY(hipGetLastError());
    int64_t *dev_costs = (int64_t *)(ws + L.costs);
    k_l_fill_u64<<<1, 256, 0, s>>>((uint64_t *)dev_costs, n_configs, 0ull);
    if (nnz > 0) {
        {
            // previous and next access of every log entry: a sort of
            // (schedule, node, position) keys, as many schedules per sort as
            // the 63 key bits hold
            LaunchScope ls("l_reuse", (double)n_sched * nnz, s);
            auto bits = [](int64_t n) { int b = 1; while (b < 62 && ((int64_t)1 << b) < n) ++b; return b; };
            const int be = bits(nnz), bn = bits(std::max<int64_t>(n_nodes, 1));
            const int gb = 63 - be - bn;                  // >= 1: nnz and the node count stay below 2^31
            const int group = gb >= 8 ? n_sched : std::min(n_sched, 1 << gb);
            for (int d0 = 0; d0 < n_sched; d0 += group) {
                const int nd = std::min(group, n_sched - d0);
                const int64_t npad = std::max<int64_t>(pow2_at_least((int64_t)nd * nnz), kSortTile);
                k_l_acc_keys<<<grid_for(npad, 256), 256, 0, s>>>(nnz, d0, nd, be, bn, npad, logs, keys);
                if ((rc = sort_keys(keys, npad, s))) return rc;
                k_l_prev_next<<<grid_for((int64_t)nd * nnz, 256), 256, 0, s>>>(nnz, d0, nd, be, keys, prev, next);
            }
        }
        LaunchScope ls("l_simulate", (double)n_configs * nnz, s);
        const int64_t nblk = (nnz + kStackBlock - 1) / kStackBlock;
        int32_t *bnext = (int32_t *)(ws + L.bnext);
        int64_t *bsum = (int64_t *)(ws + L.bsum);
        k_l_stack_blocks<<<(unsigned)(n_sched * nblk), kStackBlock, 0, s>>>(nnz, nblk, logs, (const int64_t *)(ws + L.nw),
                                                                            next, accw, bnext, bsum);
        k_l_bill<<<dim3((unsigned)((nnz + kBillThreads - 1) / kBillThreads), (unsigned)n_sched), kBillThreads, 0, s>>>(
            nnz, nblk, prev, next, acc_start, accw, bnext, bsum, dev_cfg_off, dev_cfg_list, dev_capacity,
            (unsigned long long *)dev_costs);
    }
    MPT_HIP_TRY(hipGetLastError());
    MPT_HIP_TRY(hipMemcpyAsync(costs, dev_costs, sizeof(int64_t) * n_configs, hipMemcpyDeviceToHost, s));
    MPT_HIP_TRY(hipStreamSynchronize(s));
    return MPT_OK;
}
