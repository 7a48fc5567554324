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
// nodes, with each request's path touched from the leaf up. An LRU cache of
// weighted items always holds the longest suffix of its access log whose
// distinct items fit the capacity, so eviction walks the log from its tail,
// dropping entries that are still the latest access of their node. One
// wave runs one (window, capacity) pair, 64 log entries per step, with the
// latest access of every node in LDS.
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
using mptlib::kSortTile;
using mptlib::LaunchScope;
using mptlib::sort_keys;
using mptlib::kSeqSortTile;
using mptlib::sort_requests;

constexpr int kWave = 64;
constexpr int kSimNodesLds = 36 * 1024;       // nodes whose latest access fits the LDS of one workgroup

enum : uint32_t { LERR_INVALID = 1u, LERR_RANGE = 2u, LERR_WEIGHT = 8u, LERR_OVERFLOW = 16u };

struct LHeader {
    uint32_t err;
    uint32_t pad0;
    unsigned long long total;   // sum of the sequence weights
    unsigned long long cost;    // trie cost
    int64_t pad[29];
};
static_assert(sizeof(LHeader) == 256, "header is one 256-byte block");

inline int64_t pow2_at_least(int64_t n) {
    int64_t p = 1;
    while (p < n) p <<= 1;
    return p;
}

struct LLayout {
    size_t ord, rank, lcp, base, pn, nw, cur, crank, cinv, keys, sched, log_off, logs, state, cfg_win, cfg_cap,
        costs, total;
    int64_t mpad, kpad;
};

// nnz bounds the trie's node count
LLayout l_layout(int m, int64_t n_chunks, int64_t nnz, int n_cfg) {
    LLayout L{};
    const size_t mm = (size_t)m, nz = (size_t)std::max<int64_t>(nnz, 1), nc = (size_t)std::max(n_cfg, 0);
    L.mpad = std::max<int64_t>(pow2_at_least(m), kSeqSortTile);
    L.kpad = std::max<int64_t>(pow2_at_least(std::max<int64_t>(std::max<int64_t>(nnz, n_chunks), (int64_t)nc * m)),
                               kSortTile);
    size_t o = align256(sizeof(LHeader));
    auto take = [&](size_t bytes) { size_t at = o; o = align256(o + std::max<size_t>(bytes, 1)); return at; };
    L.ord = take(4 * (size_t)L.mpad);
    L.rank = take(4 * mm);
    L.lcp = take(4 * mm);
    L.base = take(8 * (mm + 1));
    L.pn = take(4 * nz);
    L.nw = take(8 * nz);
    L.cur = take(4 * nz);
    L.crank = take(4 * (size_t)n_chunks);
    L.cinv = take(4 * (size_t)n_chunks);
    L.keys = take(8 * (size_t)L.kpad);
    L.sched = take(4 * nc * mm);
    L.log_off = take(8 * nc * mm);
    L.logs = take(4 * nc * nz);
    L.state = take(nz > (size_t)kSimNodesLds ? 4 * nc * nz : 0);
    L.cfg_win = take(8 * nc);
    L.cfg_cap = take(8 * nc);
    L.costs = take(8 * nc);
    L.total = o;
    return L;
}

// ---------------------------------------------------------------------------
// validation

__global__ void k_l_header(LHeader *h) {
    if (threadIdx.x == 0) { h->err = 0; h->total = 0; h->cost = 0; }
}

__global__ void k_l_check_offsets(int m, int64_t nnz, const int64_t *off, LHeader *h) {
    bool ok = true;
    for (int i = threadIdx.x; i < m; i += blockDim.x) ok = ok && off[i] <= off[i + 1];
    if (threadIdx.x == 0) ok = ok && off[0] == 0 && off[m] == nnz;
    if (!ok) atomicOr(&h->err, LERR_INVALID);
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

int l_read_errors(LHeader *h, hipStream_t s) {
    LHeader hh;
    MPT_HIP_TRY(hipMemcpyAsync(&hh, h, sizeof hh, hipMemcpyDeviceToHost, s));
    MPT_HIP_TRY(hipStreamSynchronize(s));
    if (hh.err & LERR_INVALID) return fail(MPT_E_INVALID, "offsets are not a CSR offset array of length m+1 ending at nnz");
    if (hh.err & LERR_RANGE) return fail(MPT_E_RANGE, "a chunk id is outside [0, n_chunks)");
    if (hh.err & LERR_WEIGHT) return fail(MPT_E_WEIGHT, "a chunk weight is <= 0 or > 2^32");
    if (hh.total >= (1ull << 61)) return fail(MPT_E_OVERFLOW, "sum of sequence weights reaches 2^61");
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

// node ids of every request's path: depth j < LCP takes the node of the
// same depth of the previous request in sorted order, deeper ones are the
// request's own new nodes. One wave walks the sorted requests, 64 at a time
// (their offsets, lengths, LCPs and bases loaded together); lane l owns the
// depths l, l + 64, ..., the first kRegDepth of them in registers and the
// rest in `cur` (only ever read back by the same lane).
constexpr int kRegDepth = 4;
__global__ __launch_bounds__(kWave) void k_l_paths(int m, const int32_t *ord, const int64_t *off, const int32_t *lcp,
                                                   const int64_t *base, int32_t *pn, int32_t *cur) {
    const int lane = threadIdx.x;
    int32_t reg[kRegDepth];
#pragma unroll
    for (int r = 0; r < kRegDepth; ++r) reg[r] = -1;
    for (int s0 = 0; s0 < m; s0 += kWave) {
        const int s = s0 + lane;
        int64_t my_off = 0, my_len = 0, my_b = 0;
        int my_l = 0;
        if (s < m) {
            const int i = ord[s];
            my_off = off[i];
            my_len = off[i + 1] - my_off;
            my_l = lcp[s];
            my_b = base[s];
        }
        const int cnt = min(kWave, m - s0);
        for (int q = 0; q < cnt; ++q) {
            const int64_t io = __shfl(my_off, q, kWave), len = __shfl(my_len, q, kWave), b = __shfl(my_b, q, kWave);
            const int l = __shfl(my_l, q, kWave);
#pragma unroll
            for (int r = 0; r < kRegDepth; ++r) {
                const int64_t j = lane + (int64_t)r * kWave;
                if (j < len) {
                    if (j >= l) reg[r] = (int32_t)(b + (j - l));
                    pn[io + j] = reg[r];
                }
            }
            for (int64_t j = lane + (int64_t)kRegDepth * kWave; j < len; j += kWave) {
                int32_t v;
                if (j >= l) { v = (int32_t)(b + (j - l)); cur[j] = v; }
                else v = cur[j];
                pn[io + j] = v;
            }
        }
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
                         const int64_t *off, const int32_t *pn, int32_t *logs) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < (int64_t)n_cfg * m;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int c = (int)(e / m);
        const int i = sched[e];
        const int64_t li = off[i + 1] - off[i], at = log_off[e];
        int32_t *dst = logs + (int64_t)c * nnz + at;
        const int32_t *path = pn + off[i];
        for (int64_t j = 0; j < li; ++j) dst[j] = path[li - 1 - j];
    }
}

// ---------------------------------------------------------------------------
// the radix cache, one wave per configuration

template <bool kLds>
__global__ __launch_bounds__(kWave) void k_l_simulate(int m, int64_t nnz, int64_t n_nodes, const int64_t *capacities,
                                                      const int32_t *sched, const int64_t *off, const int32_t *pn,
                                                      const int64_t *nw, const int32_t *logs, int32_t *state_g,
                                                      int64_t *costs) {
    extern __shared__ int32_t state_s[];
    const int c = blockIdx.x;
    const int lane = threadIdx.x;
    int32_t *last = kLds ? state_s : state_g + (int64_t)c * nnz;   // latest log position of a cached node, -1 if not cached
    const int32_t *log = logs + (int64_t)c * nnz;
    const int32_t *sc = sched + (int64_t)c * m;
    const int64_t cap = capacities[c];
    for (int64_t v = lane; v < n_nodes; v += kWave) last[v] = -1;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    int64_t used = 0, cost = 0, head = 0, tail = 0;
    for (int t = 0; t < m; ++t) {
        const int i = sc[t];
        const int64_t li = off[i + 1] - off[i];
        const int32_t *path = pn + off[i];
        // misses: the nodes not cached (the cached ones are the top of the
        // path); then every node of the path becomes the latest access
        int64_t miss = 0;
        for (int64_t j0 = 0; j0 < li; j0 += kWave) {
            const int64_t j = j0 + lane;
            if (j < li) {
                const int32_t v = path[j];
                if (last[v] < 0) miss += nw[v];
                last[v] = (int32_t)(head + (li - 1 - j));
            }
        }
#pragma unroll
        for (int o = kWave / 2; o > 0; o >>= 1) miss += __shfl_xor(miss, o, kWave);
        cost += miss;
        used += miss;
        head += li;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        // evict from the log tail: an entry that is still its node's latest
        // access is a cached node, the oldest one left
        while (used > cap && tail < head) {
            const int64_t e = tail + lane;
            int64_t wl = 0;
            int32_t v = -1;
            if (e < head) {
                v = log[e];
                if (last[v] == (int32_t)e) wl = nw[v];
            }
            int64_t incl = wl;
#pragma unroll
            for (int o = 1; o < kWave; o <<= 1) {
                const int64_t y = __shfl_up(incl, o, kWave);
                if (lane >= o) incl += y;
            }
            // first lane after which the cache fits; all 64 if none
            const uint64_t fits = __ballot(e < head && used - incl <= cap);
            const int cut = fits ? __ffsll((long long)fits) - 1 : kWave - 1;
            if (lane <= cut && wl > 0) last[v] = -1;
            const int64_t dropped = __shfl(incl, cut, kWave);
            used -= dropped;
            tail += cut + 1;
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        }
        if (tail > head) tail = head;
    }
    if (lane == 0) costs[c] = cost;
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
        if ((rc = sort_requests(ord, m, L.mpad, off, seqs, s))) return rc;
    }
    {
        LaunchScope ls("l_lcp", (double)nnz, s);
        k_l_lcp<<<grid_for(m, 256), 256, 0, s>>>(m, ord, off, seqs, w, lcp, base, rank, h);
        k_l_scan<<<1, 1024, 0, s>>>(m, base);
    }
    MPT_HIP_TRY(hipGetLastError());
    if (paths) {
        int32_t *pn = (int32_t *)(ws + L.pn), *cur = (int32_t *)(ws + L.cur);
        int64_t *nw = (int64_t *)(ws + L.nw);
        LaunchScope ls("l_paths", (double)nnz, s);
        k_l_node_weights<<<grid_for(m, 256), 256, 0, s>>>(m, ord, off, seqs, w, lcp, base, nw);
        k_l_paths<<<1, kWave, 0, s>>>(m, ord, off, lcp, base, pn, cur);
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
    if ((rc = l_read_errors(h, s))) return rc;
    if (nnz == 0) return MPT_OK;
    uint64_t *keys = (uint64_t *)(ws + L.keys);
    int32_t *rank = (int32_t *)(ws + L.crank), *inv = (int32_t *)(ws + L.cinv);
    const int64_t kpad = L.kpad;
    LaunchScope ls("l_global_order", (double)nnz, s);
    if (order_kind == MPT_ORDER_POPULARITY) {
        k_l_fill_i32<<<grid_for(n_chunks, 256), 256, 0, s>>>(rank, n_chunks, 0);
        k_l_count<<<grid_for(nnz, 256), 256, 0, s>>>(nnz, req_chunks, rank);
        k_l_fill_u64<<<grid_for(kpad, 256), 256, 0, s>>>(keys, kpad, ~0ull);
        k_l_pop_keys<<<grid_for(n_chunks, 256), 256, 0, s>>>(n_chunks, rank, keys);
        if ((rc = sort_keys(keys, kpad, s))) return rc;
        k_l_pop_rank<<<grid_for(n_chunks, 256), 256, 0, s>>>(n_chunks, keys, rank);
        k_l_inverse<<<grid_for(n_chunks, 256), 256, 0, s>>>(n_chunks, rank, inv);
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
    // configurations: window <= 0 or > m means the whole stream
    std::vector<int64_t> win(n_configs), capv(capacities, capacities + n_configs);
    for (int c = 0; c < n_configs; ++c) win[c] = (windows[c] <= 0 || windows[c] > m) ? m : windows[c];
    int64_t *dev_cfg = (int64_t *)(ws + L.cfg_win), *dev_capacity = (int64_t *)(ws + L.cfg_cap);
    MPT_HIP_TRY(hipMemcpyAsync(dev_cfg, win.data(), sizeof(int64_t) * n_configs, hipMemcpyHostToDevice, s));
    MPT_HIP_TRY(hipMemcpyAsync(dev_capacity, capv.data(), sizeof(int64_t) * n_configs, hipMemcpyHostToDevice, s));
    uint64_t *keys = (uint64_t *)(ws + L.keys);
    int32_t *sched = (int32_t *)(ws + L.sched), *logs = (int32_t *)(ws + L.logs);
    int64_t *log_off = (int64_t *)(ws + L.log_off);
    const int32_t *ord = (const int32_t *)(ws + L.ord), *rank = (const int32_t *)(ws + L.rank);
    {
        LaunchScope ls("l_schedules", (double)n_configs * m, s);
        k_l_sched_keys<<<grid_for(L.kpad, 256), 256, 0, s>>>(m, n_configs, L.kpad, dev_cfg, rank, keys);
        if ((rc = sort_keys(keys, L.kpad, s))) return rc;
        k_l_sched_out<<<grid_for((int64_t)n_configs * m, 256), 256, 0, s>>>(m, n_configs, keys, ord, seq_off, sched,
                                                                           log_off);
        k_l_log_scan<<<n_configs, 1024, 0, s>>>(m, log_off);
        if (nnz > 0)
            k_l_logs<<<grid_for((int64_t)n_configs * m, 256), 256, 0, s>>>(m, n_configs, nnz, sched, log_off, seq_off,
                                                                          (const int32_t *)(ws + L.pn), logs);
    }
    MPT_HIP_TRY(hipGetLastError());
    int64_t *dev_costs = (int64_t *)(ws + L.costs);
    {
        LaunchScope ls("l_simulate", (double)n_configs * nnz, s);
        if (n_nodes <= kSimNodesLds) {
            const size_t lds = sizeof(int32_t) * (size_t)std::max<int64_t>(n_nodes, 1);
            MPT_HIP_TRY(hipFuncSetAttribute((const void *)k_l_simulate<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                            (int)lds));
            k_l_simulate<true><<<n_configs, kWave, lds, s>>>(m, nnz, n_nodes, dev_capacity, sched, seq_off,
                                                             (const int32_t *)(ws + L.pn), (const int64_t *)(ws + L.nw),
                                                             logs, nullptr, dev_costs);
        } else {
            k_l_simulate<false><<<n_configs, kWave, 0, s>>>(m, nnz, n_nodes, dev_capacity, sched, seq_off,
                                                            (const int32_t *)(ws + L.pn), (const int64_t *)(ws + L.nw),
                                                            logs, (int32_t *)(ws + L.state), dev_costs);
        }
    }
    MPT_HIP_TRY(hipGetLastError());
    MPT_HIP_TRY(hipMemcpyAsync(costs, dev_costs, sizeof(int64_t) * n_configs, hipMemcpyDeviceToHost, s));
    MPT_HIP_TRY(hipStreamSynchronize(s));
    return MPT_OK;
}
