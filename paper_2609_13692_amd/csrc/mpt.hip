// libmpt.so -- exact MPT solver for MI355X (gfx950): kernels and the C ABI.
//
// Phases (declared in include/mpt.h):
//   1. mpt_build_weights: demand sets S_x, then W(B) = w(I(B)) for all 2^m
//      request subsets in ONE pass over HBM (each output element is written
//      once and the dense table is never read back).
//   2. mpt_solve_exact: the Section 3.1 subset DP in cost form, one launch
//      per popcount layer, with argmin splits.
//   3. mpt_extract_orders: per-request chunk orders from the hierarchy.
//
// Everything here is integer arithmetic (int64 weights and costs, uint32
// masks); there is no floating point and no dense contraction, so no MFMA.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstddef>
#include <cstring>
#include <mutex>
#include <string>
#include <type_traits>
#include <vector>

#include "bitonic.h"
#include "common.h"
#include "core.h"
#include "mpt.h"

namespace {

using mptlib::fail;
using mptlib::grid_for;
using mptlib::LaunchScope;
using mptlib::align256;

constexpr int kWave = 64;
constexpr int64_t kInf = MPT_COST_SENTINEL;   // C[empty]: never part of a minimum
constexpr int64_t kCostLimit = 1LL << 61;     // every C(S) stays below this

// ---------------------------------------------------------------------------
// binomial coefficients for colex (un)ranking of the subsets of one layer
struct BinomTable { uint32_t v[32][32]; };
constexpr BinomTable make_binom() {
    BinomTable t{};
    for (int n = 0; n < 32; ++n) {
        t.v[n][0] = 1;
        for (int k = 1; k <= n; ++k) t.v[n][k] = t.v[n - 1][k - 1] + (k <= n - 1 ? t.v[n - 1][k] : 0u);
    }
    return t;
}
constexpr BinomTable kBinom = make_binom();
__constant__ BinomTable c_binom = make_binom();

// error bits set by device-side validation
enum : uint32_t {
    ERR_INVALID = 1u, ERR_RANGE = 2u, ERR_DUP = 4u, ERR_WEIGHT = 8u, ERR_OVERFLOW = 16u
};

// workspace header (first 256 bytes of the caller's workspace)
struct WsHeader {
    uint32_t err;          // OR of ERR_* bits
    uint32_t n_list;       // entries of the compact (S_x, w) list
    int64_t zero_weight;   // total weight of chunks that no request holds
    int64_t total;         // sum_i w(R_i) = sum_i W({i}) (saturated)
    int64_t pad[29];
};
static_assert(sizeof(WsHeader) == 256, "header is one 256-byte block");

// ---------------------------------------------------------------------------
// small device helpers

// S with popcount k and colex rank r among the m-bit masks
__device__ inline uint32_t unrank_colex(uint32_t r, int k, int m) {
    uint32_t s = 0;
    for (int pos = m - 1; pos >= 0 && k > 0; --pos) {
        uint32_t c = c_binom.v[pos][k];
        if (r >= c) { s |= 1u << pos; r -= c; --k; }
    }
    return s;
}

// XCD-aware block order: the hardware hands consecutive workgroups to the 8
// XCDs in turn; renumber so that each XCD gets one contiguous range of
// logical blocks (neighbouring subsets share most of their submasks, so they
// should share one L2).
__device__ inline uint32_t xcd_block(uint32_t bid, uint32_t nblocks) {
    const uint32_t nx = 8;
    uint32_t q = nblocks / nx, r = nblocks % nx;
    uint32_t x = bid % nx, i = bid / nx;
    uint32_t first = x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q;
    return first + i;
}

// Workgroup barrier that orders LDS only. Global stores issued before it
// may still be in flight afterwards: for kernels whose waves exchange data
// through LDS alone (global results are read by later launches only).
__device__ inline void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ inline void lex_min(int64_t &v, uint32_t &a, int64_t ov, uint32_t oa) {
    if (ov < v || (ov == v && oa < a)) { v = ov; a = oa; }
}

__device__ inline void wave_lex_min(int64_t &v, uint32_t &a) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        int64_t ov = __shfl_xor(v, off, kWave);
        uint32_t oa = __shfl_xor(a, off, kWave);
        lex_min(v, a, ov, oa);
    }
}

// ---------------------------------------------------------------------------
// phase 1 kernels

__global__ void k_fill_u32(uint32_t *p, int64_t n, uint32_t v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void k_header_init(WsHeader *h) {
    if (threadIdx.x == 0) { h->err = 0; h->n_list = 0; h->zero_weight = 0; h->total = 0; }
}

// req_off must be a CSR offset array: req_off[0] = 0, non-decreasing, = nnz at m
__global__ void k_check_offsets(int m, int64_t nnz, const int64_t *req_off, WsHeader *h) {
    if (threadIdx.x != 0) return;
    bool ok = req_off[0] == 0 && req_off[m] == nnz;
    for (int i = 0; i < m; ++i) ok = ok && req_off[i] <= req_off[i + 1];
    if (!ok) atomicOr(&h->err, ERR_INVALID);
}

// S_x: every request slot sets bit i of its chunk's mask; a bit that was
// already set means the chunk is repeated inside request i.
__global__ void k_demand_sets(int m, int64_t n_chunks, int64_t nnz, const int64_t *req_off,
                              const int32_t *req_chunks, uint32_t *sig, WsHeader *h) {
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < nnz; j += (int64_t)gridDim.x * blockDim.x) {
        // request of slot j: the last i with req_off[i] <= j
        int lo = 0, hi = m - 1;
        while (lo < hi) {
            int mid = (lo + hi + 1) >> 1;
            if (req_off[mid] <= j) lo = mid; else hi = mid - 1;
        }
        int32_t x = req_chunks[j];
        if (x < 0 || (int64_t)x >= n_chunks) { atomicOr(&h->err, ERR_RANGE); continue; }
        uint32_t bit = 1u << lo;
        uint32_t old = atomicOr(&sig[x], bit);
        if (old & bit) atomicOr(&h->err, ERR_DUP);
    }
}

// weight check and compaction of the chunks that some request holds into a
// (S_x, w(x)) list, in chunk order; the others only reach W(empty) and are
// summed apart. Three passes without contended atomics: each block counts
// its contiguous range, one workgroup scans the counts (and sums the
// unrequested weight), each block writes its range at its offset.
constexpr int kCompactThreads = 256;
constexpr int kCompactMaxBlocks = 4096;

struct CompactPlan {
    int64_t per;     // chunks per block (a multiple of the block size)
    uint32_t blocks;
};

inline CompactPlan compact_plan(int64_t n_chunks) {
    const int64_t want = (n_chunks + 4095) / 4096;
    const uint32_t blocks = (uint32_t)std::max<int64_t>(1, std::min<int64_t>(want, kCompactMaxBlocks));
    int64_t per = (n_chunks + blocks - 1) / blocks;
    per = (per + kCompactThreads - 1) / kCompactThreads * kCompactThreads;
    return {std::max<int64_t>(per, kCompactThreads), blocks};
}

__device__ inline int64_t block_sum_i64(int64_t v, int64_t *red) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
    if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = v;
    __syncthreads();
    int64_t s = 0;
    for (int i = 0; i < kCompactThreads / kWave; ++i) s += red[i];
    return s;
}

__global__ __launch_bounds__(kCompactThreads) void k_compact_count(int64_t n_chunks, int64_t per, const int64_t *w,
                                                                    const uint32_t *sig, uint32_t *bcount,
                                                                    int64_t *bzero, WsHeader *h) {
    __shared__ int64_t red[2][kCompactThreads / kWave];
    const int64_t lo = blockIdx.x * per, hi = min(n_chunks, lo + per);
    int64_t taken = 0, zw = 0;
    bool bad = false;
    for (int64_t x = lo + threadIdx.x; x < hi; x += kCompactThreads) {
        const int64_t wx = w[x];
        const uint32_t sx = sig[x];
        if (wx <= 0 || wx > MPT_MAX_CHUNK_WEIGHT) { bad = true; continue; }
        if (sx) ++taken; else zw += wx;
    }
    if (bad) atomicOr(&h->err, ERR_WEIGHT);
    taken = block_sum_i64(taken, red[0]);
    zw = block_sum_i64(zw, red[1]);
    if (threadIdx.x == 0) { bcount[blockIdx.x] = (uint32_t)taken; bzero[blockIdx.x] = zw; }
}

// exclusive scan of the block counts, the list length and the unrequested
// weight into the header; one workgroup
constexpr int kScanThreads = 1024;
__global__ __launch_bounds__(kScanThreads) void k_compact_scan(uint32_t blocks, const uint32_t *bcount,
                                                               const int64_t *bzero, uint32_t *boff, WsHeader *h) {
    __shared__ uint64_t part[kScanThreads];
    __shared__ int64_t zpart[kScanThreads];
    const uint32_t t = threadIdx.x;
    const uint32_t per = (blocks + kScanThreads - 1) / kScanThreads;
    const uint32_t lo = min(blocks, t * per), hi = min(blocks, lo + per);
    uint64_t sum = 0;
    int64_t zs = 0;
    for (uint32_t i = lo; i < hi; ++i) { sum += bcount[i]; zs += bzero[i]; }
    part[t] = sum;
    zpart[t] = zs;
    __syncthreads();
    for (uint32_t off = 1; off < kScanThreads; off <<= 1) {
        const uint64_t v = t >= off ? part[t - off] : 0u;
        const int64_t z = t >= off ? zpart[t - off] : 0;
        __syncthreads();
        part[t] += v;
        zpart[t] += z;
        __syncthreads();
    }
    uint64_t run = t ? part[t - 1] : 0u;
    for (uint32_t i = lo; i < hi; ++i) {
        boff[i] = (uint32_t)run;
        run += bcount[i];
    }
    if (t == kScanThreads - 1) {
        h->n_list = (uint32_t)part[t];
        h->zero_weight = zpart[t];
    }
}

__global__ __launch_bounds__(kCompactThreads) void k_compact_write(int64_t n_chunks, int64_t per, int64_t cap,
                                                                    const int64_t *w, const uint32_t *sig,
                                                                    const uint32_t *boff, uint32_t *list_sig,
                                                                    int64_t *list_w, WsHeader *h) {
    constexpr int kWaves = kCompactThreads / kWave;
    __shared__ uint32_t wcount[kWaves];
    const int lane = (int)(threadIdx.x & (kWave - 1)), wv = (int)(threadIdx.x / kWave);
    const uint64_t below = lane ? (~0ull >> (kWave - lane)) : 0ull;     // lanes under this one
    const int64_t lo = blockIdx.x * per, hi = min(n_chunks, lo + per);
    uint32_t base = boff[blockIdx.x];
    bool over = false;
    // every thread of the block runs the same iterations (out-of-range lanes idle)
    for (int64_t x0 = lo; x0 < hi; x0 += kCompactThreads) {
        const int64_t x = x0 + threadIdx.x;
        const int64_t wx = x < hi ? w[x] : 0;
        const uint32_t sx = x < hi ? sig[x] : 0u;
        const bool take = sx != 0 && wx > 0 && wx <= MPT_MAX_CHUNK_WEIGHT;
        const uint64_t mask = __ballot(take);
        if (lane == 0) wcount[wv] = (uint32_t)__popcll(mask);
        __syncthreads();
        uint32_t before = 0, all = 0;
#pragma unroll
        for (int i = 0; i < kWaves; ++i) {
            before += i < wv ? wcount[i] : 0u;
            all += wcount[i];
        }
        if (take) {
            const uint32_t idx = base + before + (uint32_t)__popcll(mask & below);
            if ((int64_t)idx < cap) { list_sig[idx] = sx; list_w[idx] = wx; }
            else over = true;
        }
        base += all;
        __syncthreads();
    }
    if (over) atomicOr(&h->err, ERR_INVALID);
}

// W table, one workgroup per tile of 2^13 consecutive subsets that share the
// high bits H = tile id (for m < 13 one tile whose missing request bits no
// chunk holds). A chunk reaches W(H|L) iff H|L is inside S_x, i.e. iff S_x's
// high part contains H and its low part contains L. So the tile keeps
// f(L) = sum of w(x) over chunks whose high part contains H and whose low
// part equals L, and a superset-sum (zeta) over the 13 low bits turns f into
// W. The zeta over the high bits is thereby done on the sparse list, and the
// dense table is written exactly once and never read.
// The zeta over the low bits: bits 0..4 are also summed on the sparse list
// (a chunk with low part L adds w to every L' with L' = L outside bits 0..4
// and L' a subset of L inside them); bits 5..8 and 9..11 are two register
// passes, with 16 elements per thread and with two groups of 8. LDS holds
// 16 elements per 144 bytes, which keeps both passes free of bank
// conflicts; the last pass holds elements g + 512 k for g = t and t + 256,
// so each store instruction covers 2 KiB of contiguous bytes. A tile takes
// 36 KiB of LDS, so four workgroups share a CU: the stores of one tile
// drain while others are built, and each workgroup's first tile, built
// before any of its stores start, is short.
constexpr int kZetaBits = 12;
constexpr int kZetaThreads = 256;
constexpr int kZetaN = 1 << kZetaBits;
constexpr uint32_t kZetaSparseMask = 31u;     // bits summed on the sparse list
__device__ inline int zpos(int e) { return e + 2 * (e >> 4); }

// superset zeta over the index bits of N = 2^J register elements
template <int N>
__device__ inline void zeta_regs(int64_t v[N]) {
#pragma unroll
    for (int j = 0; (1 << j) < N; ++j)
#pragma unroll
        for (int k = 0; k < N; ++k)
            if (!((k >> j) & 1)) v[k] += v[k | (1 << j)];
}

// w(x) onto every position below low part L inside the sparse bits
__device__ inline void zeta_scatter(int64_t *tile, uint32_t low, int64_t w) {
    const uint32_t fixed = low & ~kZetaSparseMask;
    const uint32_t sm = low & kZetaSparseMask;
    uint32_t sub = sm;
    for (;;) {
        atomicAdd((unsigned long long *)&tile[zpos((int)(fixed | sub))], (unsigned long long)w);
        if (sub == 0) break;
        sub = (sub - 1u) & sm;
    }
}

// Persistent: each workgroup keeps up to kZetaHeld list entries per thread
// in registers and walks tiles blockIdx.x, + gridDim.x, ...; a tile's stores
// drain while the next tile is built.
constexpr int kZetaHeld = 4;
// the dense route pays once the tiles' list checks (tiles x slots, about
// 1 ps each) cost more than its passes over the table (about 10 ps per
// subset at m = 25) plus its launches (about 30 us)
inline bool dense_route_pays(int m, int64_t nnz) {
    const double tiles = m > 12 ? std::ldexp(1.0, m - 12) : 1.0;
    return tiles * (double)nnz > 10.0 * std::ldexp(1.0, m) + 3.0e7;
}

__global__ __launch_bounds__(kZetaThreads) void k_weights_tile(
        int m, uint32_t cap, uint32_t n_tiles, const uint32_t *list_sig, const int64_t *list_w, const WsHeader *h,
        int64_t *W) {
    __shared__ __align__(16) int64_t tile[kZetaN + kZetaN / 8];
    const int b = kZetaBits;
    const uint32_t lowmask = (uint32_t)kZetaN - 1u;
    const int t = threadIdx.x;
    const uint32_t cnt = min(h->n_list, cap);
    const int64_t zero_weight = h->zero_weight;
    uint32_t my_sig[kZetaHeld];
    int64_t my_w[kZetaHeld];
#pragma unroll
    for (int i = 0; i < kZetaHeld; ++i) {
        const uint32_t j = (uint32_t)t + (uint32_t)i * kZetaThreads;
        my_sig[i] = j < cnt ? list_sig[j] : 0u;
        my_w[i] = j < cnt ? list_w[j] : 0;
    }
    for (uint32_t hi = blockIdx.x; hi < n_tiles; hi += gridDim.x) {   // hi: high part H of the tile
        lds_barrier();
        for (int e = t; e < (kZetaN + kZetaN / 8) / 2; e += kZetaThreads)
            reinterpret_cast<longlong2 *>(tile)[e] = make_longlong2(0, 0);
        lds_barrier();
#pragma unroll
        for (int i = 0; i < kZetaHeld; ++i) {
            const uint32_t sg = my_sig[i];
            if (my_w[i] != 0 && ((sg >> b) & hi) == hi) zeta_scatter(tile, sg & lowmask, my_w[i]);
        }
        for (uint32_t j = t + kZetaHeld * kZetaThreads; j < cnt; j += kZetaThreads) {
            const uint32_t sg = list_sig[j];
            if (((sg >> b) & hi) == hi) zeta_scatter(tile, sg & lowmask, list_w[j]);
        }
        if (hi == 0 && t == 0)
            atomicAdd((unsigned long long *)&tile[0], (unsigned long long)zero_weight);
        lds_barrier();
        static_assert(kZetaBits == 12 && kZetaThreads == 256, "pass shapes below");
        int64_t v[16];
        // bits 5..8: element (t >> 5) << 9 | k << 5 | (t & 31)
        const int eb = ((t >> 5) << 9) | (t & 31);
#pragma unroll
        for (int k = 0; k < 16; ++k) v[k] = tile[zpos(eb | (k << 5))];
        zeta_regs<16>(v);
#pragma unroll
        for (int k = 0; k < 16; ++k) tile[zpos(eb | (k << 5))] = v[k];
        lds_barrier();
        // bits 9..11: elements g + 512 k for the groups g = t and t + 256,
        // stored straight to HBM (each store instruction covers 2 KiB)
        int64_t *out = W + ((int64_t)hi << b);
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int g = t + half * kZetaThreads;
            int64_t u[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) u[k] = tile[zpos(g + (k << 9))];
            zeta_regs<8>(u);
            if (m >= b) {
#pragma unroll
                for (int k = 0; k < 8; ++k) out[g + (k << 9)] = u[k];
            } else {                    // one partial tile: only the first 2^m subsets exist
#pragma unroll
                for (int k = 0; k < 8; ++k)
                    if (g + (k << 9) < (1 << m)) out[g + (k << 9)] = u[k];
            }
        }
    }
}

// Dense route for long chunk lists (the tile kernel scans the whole list
// once per tile, tiles x entries in all): f(S) = the weight of the chunks
// with S_x = S, scattered into a zeroed W, then the superset zeta
// W(S) = sum_{T superset of S} f(T) in place, in read-write passes of up to
// 11 bits (low bits) and 5 bits (the others) that keep every subset a
// thread touches in registers: at m = 25, the zeroing plus four passes.
__global__ void k_dense_zero(int64_t n, int64_t *W) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        W[i] = 0;
}

// The scatter adds each workgroup's slice of the list into an LDS hash table
// first: demand sets repeat (chunks held by the same few requests share
// S_x), and device-wide atomics on one address serialize, so each distinct
// set of a slice costs one global atomic. Entries that find no slot within
// the probe limit go to W directly. Integer sums: the result does not depend
// on the order.
constexpr int kScatterThreads = 1024;
constexpr int kScatterSlice = 8192;          // list entries per workgroup pass
constexpr int kHashBits = 13;
constexpr int kHashSlots = 1 << kHashBits;
constexpr int kHashProbes = 16;

__global__ __launch_bounds__(kScatterThreads) void k_dense_scatter(uint32_t cap, const uint32_t *list_sig,
                                                                    const int64_t *list_w, const WsHeader *h,
                                                                    int64_t *W) {
    __shared__ uint32_t key[kHashSlots];              // 0 = empty (no listed chunk has S_x = 0)
    __shared__ unsigned long long sum[kHashSlots];
    const uint64_t cnt = min(h->n_list, cap);
    for (uint64_t lo = (uint64_t)blockIdx.x * kScatterSlice; lo < cnt; lo += (uint64_t)gridDim.x * kScatterSlice) {
        for (int i = threadIdx.x; i < kHashSlots; i += kScatterThreads) { key[i] = 0u; sum[i] = 0ull; }
        __syncthreads();
        const uint64_t hi = min(cnt, lo + kScatterSlice);
        for (uint64_t j = lo + threadIdx.x; j < hi; j += kScatterThreads) {
            const uint32_t sx = list_sig[j];
            const unsigned long long wx = (unsigned long long)list_w[j];
            uint32_t slot = (sx * 2654435761u) >> (32 - kHashBits);
            bool done = false;
            for (int p = 0; p < kHashProbes && !done; ++p) {
                const uint32_t k = atomicCAS(&key[slot], 0u, sx);
                if (k == 0u || k == sx) {
                    atomicAdd(&sum[slot], wx);
                    done = true;
                }
                slot = (slot + 1u) & (kHashSlots - 1u);
            }
            if (!done) atomicAdd((unsigned long long *)&W[sx], wx);
        }
        __syncthreads();
        for (int i = threadIdx.x; i < kHashSlots; i += kScatterThreads)
            if (key[i]) atomicAdd((unsigned long long *)&W[key[i]], sum[i]);
        __syncthreads();
    }
    if (blockIdx.x == 0 && threadIdx.x == 0)
        atomicAdd((unsigned long long *)&W[0], (unsigned long long)h->zero_weight);
}

// superset zeta over 2^K values in registers: v[r] += v[r | 2^b], bit by bit
template <int K>
__device__ inline void zeta_reg_bits(int64_t (&v)[1 << K]) {
#pragma unroll
    for (int b = 0; b < K; ++b)
#pragma unroll
        for (int r = 0; r < (1 << K); ++r)
            if (!(r & (1 << b))) v[r] += v[r | (1 << b)];
}

// the low min(m, 11) bits: a wave owns 2^11 consecutive subsets, lane l
// holds subsets l + 64 r (r < 32), so every load and store is 64
// consecutive values; bits 6..10 are register bits, bits 0..5 lane bits
// (lane l adds lane l + 2^b when its bit b is clear). Subsets past 2^m read
// as 0 and are not stored: adding them changes nothing.
constexpr int kLaneRegBits = 5;
constexpr int kLowPassBits = 6 + kLaneRegBits;
constexpr int kDenseThreads = 256;
__global__ __launch_bounds__(kDenseThreads) void k_dense_zeta_low(int64_t n, int64_t *W) {
    constexpr int R = 1 << kLaneRegBits;
    const int lane = (int)(threadIdx.x & (kWave - 1));
    const int64_t base = ((blockIdx.x * (int64_t)kDenseThreads + threadIdx.x) >> 6) << kLowPassBits;
    if (base >= n) return;                            // whole waves
    int64_t v[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t i = base + lane + ((int64_t)r << 6);
        v[r] = i < n ? W[i] : 0;
    }
    zeta_reg_bits<kLaneRegBits>(v);
#pragma unroll
    for (int b = 0; b < 6; ++b) {
        const bool add = !(lane & (1 << b));
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int64_t up = __shfl_down(v[r], 1u << b, kWave);
            if (add) v[r] += up;
        }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t i = base + lane + ((int64_t)r << 6);
        if (i < n) W[i] = v[r];
    }
}

// bits j .. j + K - 1 (j >= 11, j + K <= m): a thread owns the 2^K subsets
// that differ only in those bits; consecutive threads take consecutive low
// subsets, so each of its loads and stores is coalesced across the wave
template <int K>
__global__ __launch_bounds__(kDenseThreads) void k_dense_zeta_high(int m, int j, int64_t *W) {
    const int64_t g = blockIdx.x * (int64_t)kDenseThreads + threadIdx.x;
    if (g >= ((int64_t)1 << (m - K))) return;
    const int64_t s = ((g >> j) << (j + K)) | (g & (((int64_t)1 << j) - 1));
    int64_t v[1 << K];
#pragma unroll
    for (int r = 0; r < (1 << K); ++r) v[r] = W[s + ((int64_t)r << j)];
    zeta_reg_bits<K>(v);
#pragma unroll
    for (int r = 0; r + 1 < (1 << K); ++r) W[s + ((int64_t)r << j)] = v[r];   // the full-set value is unchanged
}

// bits j .. j + K - 1 for K of 6 or 7 (too many values for one thread's
// registers), over the 2^K x 16 tile of the 16 consecutive low subsets
// s0 .. s0 + 15 (16 x 8 bytes = one 128-byte line per row): thread (c, g)
// loads rows 2^(K-4) g .. 2^(K-4) (g + 1) - 1 of column c and adds along
// their K - 4 low row bits in registers; the tile goes through LDS once;
// then a thread per column and low row part adds along the 4 high row bits
// in registers and writes back: one HBM read and write of every value for K
// bits, one barrier
constexpr int kTileCols = 16;
template <int K>
__global__ __launch_bounds__(kDenseThreads) void k_dense_zeta_tile(int j, int64_t *W) {
    constexpr int R = 1 << K, KR = K - 4, RB = 1 << KR;
    static_assert(R * kTileCols == kDenseThreads * RB, "one thread per column and run of RB rows");
    __shared__ int64_t t[R][kTileCols];
    const int64_t g0 = (int64_t)blockIdx.x * kTileCols;          // first of the tile's low subsets
    const int64_t s0 = ((g0 >> j) << (j + K)) | (g0 & (((int64_t)1 << j) - 1));
    const int c = (int)threadIdx.x % kTileCols, g = (int)threadIdx.x / kTileCols;
    int64_t v[RB];
#pragma unroll
    for (int i = 0; i < RB; ++i) v[i] = W[s0 + c + ((int64_t)(g * RB + i) << j)];
    zeta_reg_bits<KR>(v);
#pragma unroll
    for (int i = 0; i < RB; ++i) t[g * RB + i][c] = v[i];
    __syncthreads();
    if ((int)threadIdx.x < RB * kTileCols) {
        const int lo = g;                                          // rows lo + 2^KR h, h < 16
        int64_t u[16];
#pragma unroll
        for (int h = 0; h < 16; ++h) u[h] = t[lo + (h << KR)][c];
        zeta_reg_bits<4>(u);
#pragma unroll
        for (int h = 0; h < 16; ++h) {
            const int r = lo + (h << KR);
            if (r != R - 1) W[s0 + c + ((int64_t)r << j)] = u[h];     // the full-set row is unchanged
        }
    }
}

// the high bits 11 .. m - 1 in as few passes of at most 7 bits as they
// need, their widths as even as possible (m = 25: 7 + 7)
constexpr int kHighPassMax = 7;
void dense_zeta_high(int m, int j, int K, int64_t *W, hipStream_t s) {
    if (K > kLaneRegBits) {
        const uint32_t blocks = (uint32_t)(((int64_t)1 << (m - K)) / kTileCols);
        if (K == 6) k_dense_zeta_tile<6><<<blocks, kDenseThreads, 0, s>>>(j, W);
        else k_dense_zeta_tile<7><<<blocks, kDenseThreads, 0, s>>>(j, W);
        return;
    }
    const uint32_t blocks = (uint32_t)((((int64_t)1 << (m - K)) + kDenseThreads - 1) / kDenseThreads);
    switch (K) {
    case 1: k_dense_zeta_high<1><<<blocks, kDenseThreads, 0, s>>>(m, j, W); break;
    case 2: k_dense_zeta_high<2><<<blocks, kDenseThreads, 0, s>>>(m, j, W); break;
    case 3: k_dense_zeta_high<3><<<blocks, kDenseThreads, 0, s>>>(m, j, W); break;
    case 4: k_dense_zeta_high<4><<<blocks, kDenseThreads, 0, s>>>(m, j, W); break;
    default: k_dense_zeta_high<5><<<blocks, kDenseThreads, 0, s>>>(m, j, W); break;
    }
}

// every C(S) is at most sum_{i in S} w(R_i) = sum_{i in S} W({i}); the DP
// needs that total below 2^61
__global__ void k_check_total(int m, const int64_t *W, WsHeader *h) {
    if (threadIdx.x != 0) return;
    int64_t tot = 0;
    bool over = false;
    for (int i = 0; i < m; ++i) {
        int64_t v = W[(int64_t)1 << i];
        if (v >= kCostLimit - tot) over = true; else tot += v;
    }
    h->total = over ? kCostLimit : tot;
    if (over) atomicOr(&h->err, ERR_OVERFLOW);
}

// ---------------------------------------------------------------------------
// phase 2 kernels: C(S) = min_{A (+) B = S, lowbit(S) in A} C(A) + C(B) - W(S)

// C[0] = sentinel, C[{i}] = w(R_i), all other entries 0 so that the one
// pair (S, empty) that an enumeration may touch sums to >= the sentinel;
// split = 0 for |S| <= 1 (every other entry is written by its layer).
__global__ void k_dp_init(int m, const int64_t *W, int64_t *C, uint32_t *split) {
    const int64_t n = (int64_t)1 << m;
    for (int64_t s = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; s < n; s += (int64_t)gridDim.x * blockDim.x) {
        int pc = __popc((uint32_t)s);
        C[s] = s == 0 ? kInf : (pc == 1 ? W[s] : 0);
        if (pc <= 1) split[s] = 0;
    }
}

// small layers (|S| <= 6, at most 31 pairs per subset): one subset per lane
__global__ __launch_bounds__(256) void k_dp_lane(int m, int p, uint32_t n_sets, const int64_t *__restrict__ W,
                                                 int64_t *__restrict__ C, uint32_t *__restrict__ split) {
    uint32_t g = blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= n_sets) return;
    const uint32_t S = unrank_colex(g, p, m);
    const uint32_t l = S & (0u - S);
    const uint32_t R = S ^ l;
    int64_t best = INT64_MAX;
    uint32_t best_a = 0;
    // proper submasks r of R in increasing order (r = R would leave B empty)
    for (uint32_t r = 0; r != R; r = ((r | ~R) + 1u) & R) {
        const uint32_t A = r | l;
        const int64_t v = C[A] + C[S ^ A];
        if (v < best) { best = v; best_a = A; }
    }
    C[S] = best - W[S];
    split[S] = best_a;
}

// larger layers: one wave per (subset, segment of 2^seg_bits enumeration
// indices). Enumeration index t of A' = deposit(t, R) (order preserving);
// the 6 low bits of t are the lane, the rest a wave-uniform counter that is
// stepped in deposited form. Each lane therefore visits its A in increasing
// order, so a strict '<' keeps the smallest optimal A per lane and the
// lexicographic wave reduction keeps it overall.
__global__ __launch_bounds__(256) void k_dp_wave(int m, int p, int seg_bits, uint32_t n_tasks, int seg_log,
                                                 const int64_t *__restrict__ W, int64_t *__restrict__ C,
                                                 uint32_t *__restrict__ split, int64_t *__restrict__ part_v,
                                                 uint32_t *__restrict__ part_a) {
    const uint32_t lb = xcd_block(blockIdx.x, gridDim.x);
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const uint32_t lane = threadIdx.x % kWave;
    const uint32_t waves = gridDim.x * (blockDim.x / kWave);
    // a grid of at most kMaxGrid blocks walks the tasks (wave-uniform)
    for (uint32_t task = lb * (blockDim.x / kWave) + wave; task < n_tasks; task += waves) {
        const uint32_t set_rank = task >> seg_log;
        const uint32_t seg = task & ((1u << seg_log) - 1u);
        const uint32_t S = unrank_colex(set_rank, p, m);
        const uint32_t l = S & (0u - S);
        const uint32_t R = S ^ l;
        // lane part: deposit of the lane id into the 6 lowest bits of R
        uint32_t rr = R, lane_part = 0;
#pragma unroll
        for (int k = 0; k < 6; ++k) {
            uint32_t bit = rr & (0u - rr);
            rr ^= bit;
            if ((lane >> k) & 1u) lane_part |= bit;
        }
        const uint32_t R_hi = rr;
        const uint32_t nh = 1u << (seg_bits - 6);
        // deposit of the segment's first counter value into R_hi
        uint32_t hp = 0;
        {
            uint32_t hh = seg * nh, rem = R_hi;
            while (hh) {
                uint32_t bit = rem & (0u - rem);
                rem ^= bit;
                if (hh & 1u) hp |= bit;
                hh >>= 1;
            }
        }
        const uint32_t base_a = lane_part | l;
        int64_t best = INT64_MAX;
        uint32_t best_a = 0;
#pragma unroll 4
        for (uint32_t it = 0; it < nh; ++it) {
            const uint32_t A = base_a | hp;
            const int64_t v = C[A] + C[S ^ A];
            if (v < best) { best = v; best_a = A; }
            hp = ((hp | ~R_hi) + 1u) & R_hi;
        }
        wave_lex_min(best, best_a);
        if (lane == 0) {
            if (seg_log == 0) {
                C[S] = best - W[S];
                split[S] = best_a;
            } else {
                part_v[task] = best;
                part_a[task] = best_a;
            }
        }
    }
}

// second stage for split layers: one wave per subset
__global__ __launch_bounds__(256) void k_dp_reduce(int m, int p, uint32_t n_sets, int seg_log,
                                                   const int64_t *__restrict__ W, int64_t *__restrict__ C,
                                                   uint32_t *__restrict__ split, const int64_t *__restrict__ part_v,
                                                   const uint32_t *__restrict__ part_a) {
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const uint32_t lane = threadIdx.x % kWave;
    const uint32_t waves = gridDim.x * (blockDim.x / kWave);
    const uint32_t nseg = 1u << seg_log;
    for (uint32_t set_rank = blockIdx.x * (blockDim.x / kWave) + wave; set_rank < n_sets; set_rank += waves) {
        int64_t best = INT64_MAX;
        uint32_t best_a = 0xffffffffu;
        for (uint32_t j = lane; j < nseg; j += kWave) {
            const uint32_t t = (set_rank << seg_log) + j;
            lex_min(best, best_a, part_v[t], part_a[t]);
        }
        wave_lex_min(best, best_a);
        if (lane == 0) {
            const uint32_t S = unrank_colex(set_rank, p, m);
            C[S] = best - W[S];
            split[S] = best_a;
        }
    }
}

// ---------------------------------------------------------------------------
// phase 2, row-blocked DP (packed keys).
//
// A mask X splits into a row part X_H, its low H = m - L bits, and an
// in-row part X_L, its high L bits: X = X_H | X_L << H, with X_L made of a
// middle part X2 (its high L - CB bits) and a low part X1 (its low CB bits).
// Row X_H is the 2^L table entries that share X_H, stored together. Every
// unordered bipartition of S = S_H | S_L << H with S_H non-empty is visited
// once, from the part A holding lowbit(S_H) -- which is lowbit(S), since
// S_H holds the low bits:
//   cross pairs  (A_H, B_H), A_H holding lowbit(S_H), B_H non-empty: rows
//                A_H and B_H are complete (lower level), and C(S) gets
//                min over A_L of rowA[A_L] + rowB[S_L ^ A_L];
//   self pair    (S_H, 0): rowA is row S_H itself, filled in order of |S_L|,
//                rowB is row 0.
// Row 0 (S_H = 0) is the DP over the L in-row requests alone, done first by
// one workgroup. Levels h = |S_H| run one after the other; within a level
// every S_H is independent. Inside a pair, a thread takes the block of 2^CB
// entries for a middle mask and does the CB-bit min-plus subset convolution
// in registers.
//
// Packed keys: C'(X) = C(X) << m. A candidate's key is C'(A) + C'(B) + A,
// with A the mask of the part holding lowbit(S), below 2^m. The smallest key
// is the smallest cost and, among equal costs, the numerically smallest such
// part -- the documented tie rule. That part is always the one from the A
// row, so the table is kept twice: tagged (C'(X) + X, an OR, since C' leaves
// the low m bits zero) for rows on the A side and plain (C') for rows on the
// B side, and a key is one add. Keys are exact integers held as doubles (one
// v_add_f64 and one v_min_f64 per candidate) while sum_i w(R_i) < 2^(51-m),
// otherwise as uint64 (below 2^62); larger instances take the plain kernels.
namespace rb {
#ifndef MPT_RB_L
#define MPT_RB_L 12
#endif
constexpr int L = MPT_RB_L;           // row bits
constexpr int CB = 3;                 // register-block bits
constexpr int R2 = L - CB;            // middle bits
#ifndef MPT_RB_THREADS
#define MPT_RB_THREADS 1024
#endif
constexpr int NB = 1 << CB;           // entries per block
constexpr int ROW = 1 << L;           // entries per row
constexpr int NS2 = 1 << R2;          // blocks per row
constexpr int THREADS = MPT_RB_THREADS;
constexpr int CUS = 256;              // MI355X compute units

constexpr int cpop(int x) { int c = 0; while (x) { c += x & 1; x >>= 1; } return c; }

constexpr uint32_t cdeposit(uint32_t t, uint32_t mask) {
    uint32_t r = 0;
    while (t && mask) {
        const uint32_t bit = mask & (0u - mask);
        mask ^= bit;
        if (t & 1u) r |= bit;
        t >>= 1;
    }
    return r;
}

// the middle masks of each popcount, for the one-thread-per-block steps
struct Blocks { uint16_t v[NS2]; int begin[R2 + 1]; int end[R2 + 1]; };
constexpr Blocks make_blocks() {
    Blocks b{};
    int n = 0;
    for (int k = 0; k <= R2; ++k) {
        b.begin[k] = n;
        for (int s = 0; s < NS2; ++s)
            if (cpop(s) == k) b.v[n++] = (uint16_t)s;
        b.end[k] = n;
    }
    return b;
}
constexpr Blocks kBlocks = make_blocks();
__constant__ Blocks c_blocks = kBlocks;

// Self-pair work items of level k = |S2|: chunks of 2^t_k submasks A2 of
// S2 in increasing order, t_k the least that keeps the level's items within
// one pass of the workgroup, so a level's critical path is one item.
// Grouped by level from R2 down to 0; entry = S2 | first A2 << 16 |
// t_k << 28 | 1 << 31. Inside a level, up to 8 chunks of one S2 sit in
// adjacent lanes (their flushes combine in registers) and neighbouring
// groups of 8 lanes hold different S2 (so the accumulator flushes of one
// wave spread over several blocks).
struct Items {
    uint32_t v[8192];
    int begin[R2 + 1];
    int end[R2 + 1];
    int n;
};
constexpr int self_item_log(const Blocks &b, int k) {
    for (int t = 0; t < k; ++t)
        if ((b.end[k] - b.begin[k]) * (1 << (k - t)) <= THREADS) return t;
    return k;
}
constexpr Items make_items() {
    Items it{};
    const Blocks b = make_blocks();
    int n = 0;
    for (int k = R2; k >= 0; --k) {
        it.begin[k] = n;
        const int tb = self_item_log(b, k);
        const int chunks = 1 << (k - tb);
        const int lo = chunks < 8 ? chunks : 8;          // chunks of one S2 that sit in adjacent lanes
        for (int jh = 0; jh < chunks / lo; ++jh)
            for (int bi = b.begin[k]; bi < b.end[k]; ++bi) {
                const int s = b.v[bi];
                for (int jl = 0; jl < lo; ++jl)
                    it.v[n++] = (uint32_t)s | (cdeposit((uint32_t)(jh * lo + jl) << tb, (uint32_t)s) << 16) |
                                ((uint32_t)tb << 28) | (1u << 31);
            }
        it.end[k] = n;
    }
    it.n = n;
    return it;
}
constexpr Items kItems = make_items();
static_assert(kItems.n <= 8192, "item table too small");
constexpr bool levels_fit(const Items &it, const Blocks &b) {
    for (int k = 0; k <= R2; ++k)
        if (it.end[k] - it.begin[k] > THREADS || b.end[k] - b.begin[k] > THREADS) return false;
    return true;
}
static_assert(levels_fit(kItems, kBlocks), "every level of the self pair runs in one pass of the workgroup");
__constant__ Items c_items = kItems;

// Cross-pair work of the threads of a workgroup, lifted on the top middle
// bit E = 1 << (R2-1): a base iteration (S2', A2') over the other R2-1 middle
// bits also covers (S2'|E, A2') and (S2'|E, A2'|E), which reuse its blocks,
// so four block loads serve three block convolutions. Each thread owns
// exactly one item -- the same for every row pair of its chunk -- and keeps
// the best keys of its two output blocks in registers across all pairs,
// flushing them once. An item is a run of consecutive submasks A2' of one
// S2' (in increasing order), starting at an even index with an even count
// (the S2' = 0 item is its single submask).
//
// The waves of a workgroup go to the four SIMDs in turn, and every pair ends
// at a workgroup barrier, so the SIMD with the most steps sets the pace. The
// runs are cut to step capacities by wave: the first half of the waves take
// runs of 8, the next quarter runs of up to 6, the last quarter runs of up to
// 4, so that each SIMD gets two waves of 8, one of 6 and one of 4 steps
// (26, against 3^(R2-1) / 64 / 4 = 25.6 at least). The S2' are taken by
// decreasing popcount; a run never leaves a remainder of 2 that would need
// a lane of its own. Entry: S2' | first A2' << 8 | count << 16 | 1 << 31
// (0 = no item).
constexpr int RL = R2 - 1;
struct ThreadItems { uint32_t v[THREADS]; bool ok; };
constexpr uint32_t titem(int s2, int a2, int cnt) {
    return (uint32_t)s2 | ((uint32_t)a2 << 8) | ((uint32_t)cnt << 16) | (1u << 31);
}
constexpr ThreadItems make_thread_items() {
    ThreadItems t{};
    constexpr int WAVES = THREADS / kWave;
    // lane classes: [0, nA) capacity 8, [nA, nA + nB) 6, the rest 4
    const int nA = WAVES / 2 * kWave, nB = WAVES / 4 * kWave;
    int at[3] = {0, nA, nA + nB};
    const int end[3] = {nA, nA + nB, THREADS};
    t.ok = true;
    for (int k = RL; k >= 0; --k)
        for (int s = 0; s < (1 << RL); ++s) {
            if (cpop(s) != k) continue;
            int n = 1 << k, first = 0;
            while (n > 0) {
                int cls = -1, take = 0;
                if (n >= 8 && at[0] < end[0]) { cls = 0; take = 8; }
                else if (n >= 6 && at[1] < end[1] && (n == 6 || n >= 10)) { cls = 1; take = 6; }
                else if (n >= 4 && at[2] < end[2]) { cls = 2; take = 4; }
                else if (at[1] < end[1]) { cls = 1; take = n < 4 ? n : 4; }
                else if (at[2] < end[2] && n < 4) { cls = 2; take = n; }
                if (cls < 0) { t.ok = false; return t; }
                t.v[at[cls]++] = titem(s, (int)cdeposit((uint32_t)first, (uint32_t)s), take);
                first += take;
                n -= take;
            }
        }
    return t;
}
constexpr ThreadItems kTItems = make_thread_items();
static_assert(kTItems.ok, "every cross-pair run needs a thread of its own");
// the cross-pair loop steps two submasks at a time: an item of S2' != 0
// starts at a submask without lowbit(S2') and has an even count; the item
// of S2' = 0 is its single submask; every submask of every S2' is covered once
constexpr bool items_pair_up(const ThreadItems &t) {
    int steps[1 << RL] = {};
    for (int i = 0; i < THREADS; ++i) {
        const uint32_t v = t.v[i];
        if (!(v >> 31)) continue;
        const uint32_t s2 = v & 0xffu, a2 = (v >> 8) & 0xffu, cnt = (v >> 16) & 15u;
        if (s2 == 0 ? (cnt != 1 || a2 != 0) : (cnt == 0 || (cnt & 1u) || (a2 & (s2 & (0u - s2))) != 0)) return false;
        steps[s2] += (int)cnt;
    }
    for (int s = 0; s < (1 << RL); ++s)
        if (steps[s] != (1 << cpop(s))) return false;
    return true;
}
static_assert(items_pair_up(kTItems), "cross-pair items must pair up their submasks and cover each once");
__constant__ ThreadItems c_titems = kTItems;

// The lanes whose items have one S2', for combining their best keys after
// the pairs: the items of an S2' are handed out in one go, class by class,
// so they sit in runs of adjacent lanes, at most two with this table.
// Entry: first lane | count << 16 (count 0: no run).
constexpr int kRuns = 2;
struct ItemRuns { uint32_t r[1 << RL][kRuns]; bool ok; };
constexpr ItemRuns make_item_runs(const ThreadItems &t) {
    ItemRuns g{};
    g.ok = true;
    int n[1 << RL] = {};
    for (int i = 0; i < THREADS; ++i) {
        if (!(t.v[i] >> 31)) continue;
        const int sp = (int)(t.v[i] & 0xffu);
        if (n[sp] > 0) {
            uint32_t &last = g.r[sp][n[sp] - 1];
            if ((int)(last & 0xffffu) + (int)(last >> 16) == i) {
                last += 1u << 16;
                continue;
            }
        }
        if (n[sp] == kRuns) {
            g.ok = false;
            return g;
        }
        g.r[sp][n[sp]++] = (uint32_t)i | (1u << 16);
    }
    return g;
}
constexpr ItemRuns kItemRuns = make_item_runs(kTItems);
static_assert(kItemRuns.ok, "the lanes of one S2' form at most two runs");
// the runs cover exactly the lanes with items, each S2' with at least one
constexpr bool runs_cover(const ThreadItems &t, const ItemRuns &g) {
    int owner[THREADS] = {};
    for (int i = 0; i < THREADS; ++i) owner[i] = -1;
    for (int sp = 0; sp < (1 << RL); ++sp) {
        int lanes = 0;
        for (int q = 0; q < kRuns; ++q)
            for (int i = 0; i < (int)(g.r[sp][q] >> 16); ++i) {
                const int l = (int)(g.r[sp][q] & 0xffffu) + i;
                if (l >= THREADS || owner[l] != -1 || !(t.v[l] >> 31) || (int)(t.v[l] & 0xffu) != sp) return false;
                owner[l] = sp;
                ++lanes;
            }
        if (lanes == 0) return false;
    }
    for (int i = 0; i < THREADS; ++i)
        if ((t.v[i] >> 31) && owner[i] == -1) return false;
    return true;
}
static_assert(runs_cover(kTItems, kItemRuns), "every lane with an item is in one run of its S2'");

// The combining plan. Each 16-lane quarter of a wave takes four S2' in
// turn, lane q the entry q of each (q < 8: entry q of block S2', else entry
// q - 8 of block S2'|E), and reads the staged keys of the S2''s lanes. The
// quarters of a wave step together, so a step costs its costliest S2' (one
// read per lane of it): the S2' are grouped four to a step by decreasing
// cost, and the groups go to the waves, four each, costliest first onto the
// least loaded wave. Entry [wave][quarter]: the four S2' (8 bits each, step
// j in bits 8j..8j+7) and, per step, their runs as first lane | count << 10
// in 16 bits each.
constexpr int kWaves = THREADS / kWave;
static_assert((1 << RL) == kWaves * 4 * 4, "four steps of four quarters per wave cover every S2'");
struct alignas(16) GatherSlot { uint32_t runs[4]; uint32_t s2; uint32_t pad[3]; };
struct GatherPlan { GatherSlot s[kWaves][4]; bool ok; };
constexpr GatherPlan make_gather_plan(const ItemRuns &g) {
    GatherPlan plan{};
    plan.ok = true;
    int cost[1 << RL] = {};
    int maxc = 0;
    for (int sp = 0; sp < (1 << RL); ++sp) {
        for (int q = 0; q < kRuns; ++q) cost[sp] += (int)(g.r[sp][q] >> 16);
        maxc = cost[sp] > maxc ? cost[sp] : maxc;
    }
    int order[1 << RL] = {};
    int n = 0;
    for (int c = maxc; c >= 0; --c)
        for (int sp = 0; sp < (1 << RL); ++sp)
            if (cost[sp] == c) order[n++] = sp;
    int load[kWaves] = {}, used[kWaves] = {};
    for (int gi = 0; gi < (1 << RL) / 4; ++gi) {
        int w = -1;
        for (int x = 0; x < kWaves; ++x)
            if (used[x] < 4 && (w < 0 || load[x] < load[w])) w = x;
        for (int u = 0; u < 4; ++u) {
            const int sp = order[4 * gi + u];
            uint32_t word = 0;
            for (int q = 0; q < kRuns; ++q) {
                const uint32_t first = g.r[sp][q] & 0xffffu, cnt = g.r[sp][q] >> 16;
                if (first >= 1024u || cnt >= 64u) plan.ok = false;
                word |= (first | cnt << 10) << (16 * q);
            }
            plan.s[w][u].runs[used[w]] = word;
            plan.s[w][u].s2 |= (uint32_t)sp << (8 * used[w]);
        }
        load[w] += cost[order[4 * gi]];
        ++used[w];
    }
    return plan;
}
constexpr GatherPlan kGatherPlan = make_gather_plan(kItemRuns);
static_assert(kRuns == 2 && THREADS <= 1024 && kGatherPlan.ok, "runs fit 16 bits each");
constexpr bool gather_covers(const GatherPlan &plan) {
    bool seen[1 << RL] = {};
    for (int w = 0; w < kWaves; ++w)
        for (int u = 0; u < 4; ++u)
            for (int j = 0; j < 4; ++j) {
                const int sp = (int)((plan.s[w][u].s2 >> (8 * j)) & 0xffu);
                if (seen[sp]) return false;
                seen[sp] = true;
            }
    return true;
}
static_assert(gather_covers(kGatherPlan), "every S2' is combined by one quarter of one wave");
__constant__ GatherPlan c_gather = kGatherPlan;


// Key arithmetic. A table entry carries the packed value v = C' or, tagged,
// C' | X.
//   uint64: an entry is v itself; a key is the sum of two entries.
//   double: an entry is the double 2^52 + 2v. Its exponent is fixed, so its
//   low mantissa bits are the integer 2v. The sum of two entries is
//   2^53 + 2(v_A + v_B): even, so exact below 2^54, and its mantissa is the
//   packed key v_A + v_B. That needs 2v < 2^52 for every entry, i.e.
//   sum_i w(R_i) < 2^(51-m).
template <class K> struct Key;
template <> struct Key<uint64_t> {
    static __device__ inline uint64_t entry(uint64_t v) { return v; }
    static __device__ inline uint64_t entry_value(uint64_t e) { return e; }
    static __device__ inline uint64_t add(uint64_t a, uint64_t b) { return a + b; }
    static __device__ inline uint64_t min(uint64_t a, uint64_t b) { return b < a ? b : a; }
    static __device__ inline uint64_t none() { return ~0ull; }
    static __device__ inline uint64_t bits(uint64_t k) { return k; }
    static __device__ inline uint64_t from_bits(uint64_t b) { return b; }
    // key bits (as kept in the accumulators) -> packed key; ~0 for none
    static __device__ inline uint64_t key_value(uint64_t b) { return b; }
    // the packed table in HBM holds each entry's bits
    static __device__ inline uint64_t store(uint64_t v) { return v; }
    static __device__ inline uint64_t stored_value(uint64_t b) { return b; }
    static __device__ inline uint64_t load(uint64_t b) { return b; }
    // packed key -> the bits the accumulators hold
    static __device__ inline uint64_t key_bits(uint64_t k) { return k; }
};
template <> struct Key<double> {
    static constexpr uint64_t E52 = 0x4330000000000000ull;  // bits of 2^52
    static constexpr uint64_t MANT = (1ull << 52) - 1u;
    static __device__ inline uint64_t bits(double k) { return (uint64_t)__double_as_longlong(k); }
    static __device__ inline double from_bits(uint64_t b) { return __longlong_as_double((long long)b); }
    static __device__ inline double entry(uint64_t v) { return from_bits(E52 | (v << 1)); }
    static __device__ inline uint64_t entry_value(double e) { return (bits(e) & MANT) >> 1; }
    static __device__ inline double add(double a, double b) { return a + b; }
    static __device__ inline double min(double a, double b) { return fmin(a, b); }
    static __device__ inline double none() { return __builtin_inf(); }
    // keys are positive doubles: they order like their bit patterns
    static __device__ inline uint64_t key_value(uint64_t b) { return b >= 0x7ff0000000000000ull ? ~0ull : b & MANT; }
    static __device__ inline uint64_t store(uint64_t v) { return E52 | (v << 1); }
    static __device__ inline uint64_t stored_value(uint64_t b) { return (b & MANT) >> 1; }
    static __device__ inline double load(uint64_t b) { return from_bits(b); }
    // packed key -> the bits of the sum that carries it: 2^53 + 2k
    static __device__ inline uint64_t key_bits(uint64_t k) { return 0x4340000000000000ull | k; }
};

// Narrow keys, for the cross pairs while sum_i w(R_i) < 2^20 - 1. Every
// C(A) + C(B) is then below 2^20 - 1 (a sub-instance costs at most the sum
// of its request weights), and a candidate's key fits 32 bits:
// (C(A) + C(B)) << L | A_L, A_L the in-row part of the part holding
// lowbit(S). Inside one row pair A_H is fixed, so the order of these keys is
// the order of (cost, A). The entries are C(X) << L | X_L (tagged) and
// C(X) << L (plain), so a key is again one add, and the minimum over a
// candidate chain becomes v_min3_u32 (two candidates per instruction).
// Across the pairs of a chunk, taken in increasing A_H, each output entry
// keeps beside its best key the A_H of the first pair that reached it.
template <> struct Key<uint32_t> {
    static __device__ inline uint32_t add(uint32_t a, uint32_t b) { return a + b; }
    static __device__ inline uint32_t min(uint32_t a, uint32_t b) { return b < a ? b : a; }
    static __device__ inline uint32_t none() { return 0xffffffffu; }
};
constexpr int64_t kNarrowTotal = (int64_t)1 << (32 - L);   // sum_i w(R_i) must stay below this - 1
static_assert(32 - L >= 20, "narrow keys leave 20 bits for the cost");

// Rows, in HBM and in LDS alike. Block x2 (the NB entries sharing the
// middle mask x2) sits at slot(x2) = x2 ^ (x2 >> 3 & 7) ^ (x2 >> 6 & 3)
// (for R2 = 9; the last term takes the bits between 6 and E), a GF(2)-linear
// involution, so slot(S2 ^ A2) = slot(S2) ^ slot(A2); it maps the low R2-1
// middle bits onto themselves and the top one, E, onto NS2/2, so
// slot(X | E) = slot(X) + NS2/2 for X below E. A row is stored as NB/2
// planes of 16-byte pieces: plane q holds entries 2q and 2q+1 of every
// block, block at slot s in piece s. A lane's four reads of one block are
// then 8 KiB apart (immediate offsets), and a 16-lane pass of reads is free
// of bank conflicts when its lanes' slots differ mod 16 (gfx950 serves a
// 16-byte read 16 lanes at a time from 16 groups of 16 bytes; a plane is a
// multiple of 256 bytes). Because HBM holds the rows in this same layout, a
// row reaches LDS as a plain copy, straight from global memory.
constexpr int PLANE = 2 * NS2;        // K elements per plane
// element index inside a row of entry x of the block at slot
__host__ __device__ constexpr uint32_t lpos(uint32_t slot, int x) {
    return (uint32_t)(x >> 1) * PLANE + slot * 2u + (uint32_t)(x & 1);
}
__host__ __device__ constexpr uint32_t slot_of(uint32_t x2) {
    return x2 ^ ((x2 >> 3) & 7u) ^ ((x2 >> 6) & ((1u << (R2 - 7)) - 1u));
}
constexpr bool slots_ok() {
    bool seen[NS2] = {};
    for (uint32_t x = 0; x < (uint32_t)NS2; ++x) {
        const uint32_t sl = slot_of(x);
        if (sl >= (uint32_t)NS2 || seen[sl] || slot_of(sl) != x) return false;
        seen[sl] = true;
        if (x < (uint32_t)NS2 / 2 && (sl >= (uint32_t)NS2 / 2 || slot_of(x | NS2 / 2) != sl + NS2 / 2)) return false;
    }
    return true;
}
static_assert(R2 >= 7 && slots_ok(), "slot_of is an involution that puts the E half NS2/2 above the rest");
static_assert(NB == 8 && (PLANE * 8) % 256 == 0, "four planes of 16-byte pieces, each a multiple of 256 bytes");
// Narrow tables use the same slots with 4-byte elements: NB/4 planes of
// 16-byte pieces, plane q holding entries 4q..4q+3 of every block, block at
// slot s in piece s (a plane is 8 KiB, a row 16 KiB).
constexpr int NPLANE = 4 * NS2;       // uint32 elements per narrow plane
__host__ __device__ constexpr uint32_t npos(uint32_t slot, int x) {
    return (uint32_t)(x >> 2) * NPLANE + slot * 4u + (uint32_t)(x & 3);
}

// two buffers of the (A, B) row pair: the next pair's rows are copied in
// while the current pair runs
template <class K> struct alignas(16) Lds {
    K r[2][2][ROW];        // [buffer][A side (tagged), B side (plain)]
    uint64_t acc[ROW];     // best key bits per entry of the output row
};
static_assert(sizeof(Lds<double>) <= 160 * 1024, "rows and accumulators fit one CU's LDS");
// workgroups that run on one CU at a time (their LDS takes the CU)
constexpr int WGS_PER_CU = (int)((160 * 1024) / sizeof(Lds<double>));

// block at slot -> v[x] = entry x
template <class K>
__device__ inline void load_blk(const K *row, uint32_t slot, K v[NB]) {
    // each 16-byte piece is read as one 128-bit integer: a vector of two
    // keys whose lanes are used apart gets split into 8-byte reads
    const __uint128_t *p = reinterpret_cast<const __uint128_t *>(row + slot * 2u);
#pragma unroll
    for (int q = 0; q < NB / 2; ++q) {
        const __uint128_t t = p[q * (PLANE / 2)];
        v[2 * q] = Key<K>::from_bits((uint64_t)t);
        v[2 * q + 1] = Key<K>::from_bits((uint64_t)(t >> 64));
    }
}

// narrow block at slot -> v[x] = entry x (two 16-byte reads)
__device__ inline void load_blk(const uint32_t *row, uint32_t slot, uint32_t v[NB]) {
    const uint4 *p = reinterpret_cast<const uint4 *>(row + slot * 4u);
#pragma unroll
    for (int q = 0; q < NB / 4; ++q) {
        const uint4 t = p[q * (NPLANE / 4)];
        v[4 * q] = t.x;
        v[4 * q + 1] = t.y;
        v[4 * q + 2] = t.z;
        v[4 * q + 3] = t.w;
    }
}

// row xh of a table of E-byte elements -> LDS dst, as direct global-to-LDS
// copies of 16 bytes per lane (no registers held), by a workgroup of NT
// threads. Completion: this thread's vmcnt, then a workgroup barrier.
typedef __attribute__((address_space(3))) void lds_void;
template <class E, int NT = THREADS>
__device__ inline void copy_row(void *dst, const E *__restrict__ tab, uint32_t xh) {
    constexpr int PIECES = ROW * (int)sizeof(E) / 16;    // 16-byte pieces per row
    constexpr int PER_WAVE = PIECES / (NT / kWave);
    static_assert(PER_WAVE % kWave == 0, "whole wave copies");
    const int w = (int)(threadIdx.x / kWave), lane = (int)(threadIdx.x & (kWave - 1));
    const uint4 *src = reinterpret_cast<const uint4 *>(tab + ((size_t)xh << L));
#pragma unroll
    for (int i = 0; i < PER_WAVE / kWave; ++i) {
        const int p0 = w * PER_WAVE + i * kWave;         // first piece of this wave copy (uniform)
        __builtin_amdgcn_global_load_lds(src + p0 + lane, (lds_void *)((char *)dst + p0 * 16), 16, 0, 0);
    }
}
// copy_row, with each direct copy issued through inline
// assembly so that the compiler's wait insertion does not see it: while it
// knows of a pending direct copy into LDS, it makes every LDS read wait for
// all earlier LDS reads. These copies are retired explicitly (copies_done,
// then a workgroup barrier) before their rows are read, and they add only
// to the in-order count of vector loads, so the compiler's own waits stay
// correct (at worst longer). M0, which carries the LDS address of a copy,
// is saved and restored around it.
template <class E>
__device__ inline void copy_row_quiet(void *dst, const E *__restrict__ tab, uint32_t xh) {
    constexpr int PIECES = ROW * (int)sizeof(E) / 16;
    constexpr int PER_WAVE = PIECES / (THREADS / kWave);
    static_assert(PER_WAVE % kWave == 0, "whole wave copies");
    const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
    const int lane = (int)(threadIdx.x & (kWave - 1));
    const uint4 *src = reinterpret_cast<const uint4 *>(tab + ((size_t)xh << L));
    typedef __attribute__((address_space(3))) char lds_c;
    const uint32_t base = (uint32_t)(uintptr_t)(lds_c *)dst;
#pragma unroll
    for (int i = 0; i < PER_WAVE / kWave; ++i) {
        const int p0 = w * PER_WAVE + i * kWave;
        const uint32_t at = base + (uint32_t)p0 * 16u;     // the wave's 1 KiB of LDS
        uint32_t saved;
        asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %2, off\n\ts_nop 0\n\ts_mov_b32 m0, %0"
                     : "=&s"(saved)
                     : "s"(at), "v"(src + p0 + lane)
                     : "memory");
    }
}
// vmcnt(0), expcnt and lgkmcnt untouched (gfx9 encoding). The builtin, not
// inline asm, so that the compiler's wait insertion sees the copies retire:
// a pending direct-to-LDS copy (a flat-encoded instruction) makes it treat
// the LDS counter as out of order and wait for every outstanding LDS read.
__device__ inline void copies_done() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// deposit the low bits of t into the set bits of mask (in order)
__device__ inline uint32_t deposit(uint32_t t, uint32_t mask) {
    uint32_t r = 0;
    while (t && mask) {
        const uint32_t bit = mask & (0u - mask);
        mask ^= bit;
        if (t & 1u) r |= bit;
        t >>= 1;
    }
    return r;
}

// CB-bit min-plus subset convolution of one block pair, a[] from the A row
// (tagged) and b[] from the B row (plain):
//   best[S1] = min(best[S1], min over A1 in S1 of a[A1] + b[S1 ^ A1]).
template <class K>
__device__ inline void conv_full(const K a[NB], const K b[NB], K best[NB]) {
#pragma unroll
    for (int s1 = 0; s1 < NB; ++s1)
#pragma unroll
        for (int a1 = 0; a1 < NB; ++a1)
            if (!(a1 & ~s1)) best[s1] = Key<K>::min(best[s1], Key<K>::add(a[a1], b[s1 ^ a1]));
}

// the same, folding into out[] the keys of in[] (in and out may be one array)
template <class K>
__device__ inline void conv_into(const K a[NB], const K b[NB], const K in[NB], K out[NB]) {
#pragma unroll
    for (int s1 = 0; s1 < NB; ++s1) {
        K v = in[s1];
#pragma unroll
        for (int a1 = 0; a1 < NB; ++a1)
            if (!(a1 & ~s1)) v = Key<K>::min(v, Key<K>::add(a[a1], b[s1 ^ a1]));
        out[s1] = v;
    }
}

// minimum of v over an aligned group of seg = 1, 2, 4, 8 or 16 lanes (every
// lane of the group gets it): quad permutations, then the half-row mirror
// that pairs the two quads of 8 lanes, then the row mirror that pairs the
// two halves of 16
__device__ inline uint32_t group_min32(uint32_t v, uint32_t seg) {
    auto take = [&](uint32_t o) { v = o < v ? o : v; };
    if (seg >= 2) take((uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));    // quad_perm [1,0,3,2]
    if (seg >= 4) take((uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));    // quad_perm [2,3,0,1]
    if (seg >= 8) take((uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));   // row_half_mirror
    if (seg >= 16) take((uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false));  // row_mirror
    return v;
}

// Flush of best keys (one block of the output row) from lanes that share S2
// in aligned groups of seg lanes: the group minimum of each entry's key bits
// (the high words, then the low words among the lanes holding the least
// high word) and one LDS atomic per group and entry -- 64-bit LDS atomics
// are slow, and lanes that hit one address in the same instruction are
// served one at a time.
template <class K>
__device__ inline void flush_group(const K best[NB], uint32_t s2, uint32_t seg, uint64_t *acc) {
    const uint32_t lane = threadIdx.x & (kWave - 1);
#pragma unroll
    for (int x = 0; x < NB; ++x) {
        const uint64_t b = Key<K>::bits(best[x]);     // unsigned order = key order
        const uint32_t hi = group_min32((uint32_t)(b >> 32), seg);
        const uint32_t lo = group_min32((uint32_t)(b >> 32) == hi ? (uint32_t)b : 0xffffffffu, seg);
        const uint64_t g = ((uint64_t)hi << 32) | lo;
        if ((lane & (seg - 1)) == 0 && g != Key<K>::bits(Key<K>::none()))
            atomicMin((unsigned long long *)&acc[(s2 << CB) | x], (unsigned long long)g);
    }
}

// one self-pair work item (S2, first A2, t) of row S_H against row 0: 2^t
// submasks A2 of S2 in increasing order, skipping A2 == S2 (B2 would be
// empty); rA is row S_H (tagged), rB row 0 (plain)
template <class K>
__device__ inline void run_item(uint32_t item, const K *rA, const K *rB, uint64_t *acc) {
    const uint32_t s2 = item & 0xffffu;
    const int k = __popc(s2);
    const int tb = (int)((item >> 28) & 7u);
    const uint32_t cnt = 1u << tb;
    const uint32_t slot_s2 = slot_of(s2);
    uint32_t a2 = (item >> 16) & 0xfffu;
    K best[NB];
#pragma unroll
    for (int x = 0; x < NB; ++x) best[x] = Key<K>::none();
    for (uint32_t i = 0; i < cnt; ++i) {
        if (a2 != s2) {
            const uint32_t sa = slot_of(a2), sb = slot_s2 ^ sa;
            K a[NB], b[NB];
            load_blk(rA, sa, a);
            load_blk(rB, sb, b);
            conv_full<K>(a, b, best);
        }
        a2 = ((a2 | ~s2) + 1u) & s2;
    }
    const uint32_t chunks = 1u << (k - tb);
    flush_group<K>(best, s2, chunks < 8u ? chunks : 8u, acc);
}

// The block that thread t completes when it finishes a row, and its W: the
// t-th middle mask in order of popcount, so that the blocks of one level sit
// in consecutive threads (threads past NS2 take none). Loaded before the
// row's setup, whose waits then cover these loads too. WT: int64_t, or
// uint32_t for narrow keys, which hold sum_i w(R_i) < 2^20 (every W fits 32
// bits).
template <class WT>
struct OwnBlock {
    uint32_t s2;
    WT w[NB];
};
template <class WT>
__device__ inline void own_block_load(uint32_t sh, const int64_t *__restrict__ Wr, OwnBlock<WT> &o) {
    const uint32_t t = threadIdx.x < (uint32_t)NS2 ? threadIdx.x : NS2 - 1u;
    o.s2 = c_blocks.v[t];
    const uint4 *wp = reinterpret_cast<const uint4 *>(Wr + ((sh << L) | (o.s2 << CB)));
#pragma unroll
    for (int q = 0; q < NB / 2; ++q) {
        const uint4 v = wp[q];
        if constexpr (sizeof(WT) == 4) {
            o.w[2 * q] = v.x;
            o.w[2 * q + 1] = v.z;
        } else {
            o.w[2 * q] = (int64_t)(((uint64_t)v.y << 32) | v.x);
            o.w[2 * q + 1] = (int64_t)(((uint64_t)v.w << 32) | v.z);
        }
    }
}

// A thread's self-pair item of level k (k at most R2): entry i of the
// level's items, any valid entry past the level's end (validity is tested
// where the entry is used, so that no wait for the load comes earlier).
template <int NT>
__device__ inline uint32_t item_load(int k, int i) {
    constexpr int last = kItems.n - 1;
    const int it = c_items.begin[k] + (int)threadIdx.x + i * NT;
    return c_items.v[it < last ? it : last];
}

// Complete row S_H (non-empty) on 64-bit keys (narrow rows have
// finalize_row_narrow). s.acc holds the best cross-pair key bits (or ~0);
// rS receives row S_H (tagged), r0 holds row 0 (plain), both in LDS; own:
// this thread's block (own_block_load). Writes the row to the plain and the
// tagged table and its splits to Sr (row-major, mask order inside a row).
// As in finalize_row_narrow, the levels issue no global stores (a finished
// block's plain entries go to its acc entries, its splits to s.r[1][0]) and
// load only the next level's item entries, into the other of two registers.
template <class K>
__device__ __attribute__((always_inline)) inline void finalize_row(int m, uint32_t sh, const OwnBlock<int64_t> &own,
                                                                   Lds<K> &s, K *rS, const K *r0,
                                                                   uint64_t *__restrict__ Tt,
                                                                   uint64_t *__restrict__ Pt,
                                                                   uint32_t *__restrict__ Sr) {
    const int H = m - L;
    const uint32_t row = sh << L;
    const uint64_t mask = ((uint64_t)1 << m) - 1u;
    const int tid = (int)threadIdx.x;
    uint32_t *split = reinterpret_cast<uint32_t *>(s.r[1][0]);
    // block 0 of row 0, plain: C'(X1 << H) for every low part X1
    uint64_t b0[NB];
#pragma unroll
    for (int x = 0; x < NB; ++x) b0[x] = Key<K>::entry_value(r0[lpos(0u, x)]);
    // S = (S_H, 0, 0) with one request in S_H is a leaf: C = W
    const bool single = (sh & (sh - 1u)) == 0;
    auto level = [&](int k, const uint32_t &cur, uint32_t &nxt) __attribute__((always_inline)) {
        nxt = item_load<THREADS>(k < R2 ? k + 1 : R2, 0);
        // A2 a proper submask of S2
        if (tid < c_items.end[k] - c_items.begin[k]) run_item<K>(cur, rS, r0, s.acc);
        lds_barrier();
        // A2 = S2: in-block pairs, one thread per block of this level; A =
        // (S_H, S2, A1) holds lowbit(S), B = (0, 0, S1 ^ A1) is in block 0
        // of row 0
        if (tid >= c_blocks.begin[k] && tid < c_blocks.end[k]) {
            const uint32_t s2 = own.s2;
            const uint32_t tag = s2 << CB;
            const uint32_t base = sh | (tag << H);               // mask of (S_H, S2, X1 = 0)
            uint64_t out[NB];
            uint32_t sp[NB];
            // the block's accumulated keys (cross pairs and this level's
            // items), read together before the dependent chain below
            uint64_t kacc[NB];
#pragma unroll
            for (int x = 0; x < NB; ++x) kacc[x] = Key<K>::key_value(s.acc[tag | x]);
            const bool leaf0 = s2 == 0 && single;
            // S1 in order of popcount so that every A1 < S1 is ready; no
            // branches, so the reads above stay ahead of the chain
#pragma unroll
            for (int pc = 0; pc <= CB; ++pc) {
#pragma unroll
                for (int s1 = 0; s1 < NB; ++s1) {
                    if (cpop(s1) != pc) continue;
                    const int64_t w = own.w[s1];
                    uint64_t kb = kacc[s1];
#pragma unroll
                    for (int a1 = 0; a1 < NB; ++a1) {
                        if ((a1 & ~s1) || a1 == s1) continue;
                        const uint64_t c = out[a1] + b0[s1 ^ a1] + (base | ((uint32_t)a1 << H));
                        kb = c < kb ? c : kb;
                    }
                    const bool leaf = s1 == 0 && leaf0;
                    out[s1] = leaf ? (uint64_t)w << m : ((kb >> m) - (uint64_t)w) << m;
                    sp[s1] = leaf ? 0u : (uint32_t)(kb & mask);
                }
            }
            const uint32_t sl = slot_of(s2);
            // the tagged entries to the row, the plain ones and the splits
            // over the entries just read
#pragma unroll
            for (int x = 0; x < NB; ++x) {
                rS[lpos(sl, x)] = Key<K>::entry(out[x] | base | ((uint32_t)x << H));
                s.acc[tag | x] = Key<K>::store(out[x]);
            }
            uint4 *sp4 = reinterpret_cast<uint4 *>(split + tag);
            sp4[0] = make_uint4(sp[0], sp[1], sp[2], sp[3]);
            sp4[1] = make_uint4(sp[4], sp[5], sp[6], sp[7]);
        }
        lds_barrier();
    };
    uint32_t ia = item_load<THREADS>(0, 0), ib;
    for (int k = 0; k <= R2; k += 2) {
        level(k, ia, ib);
        if (k + 1 <= R2) level(k + 1, ib, ia);
    }
    // the row to HBM: plain entries (the block at slot p, plane by plane),
    // tagged entries (the LDS row's bits: an entry and its stored form are
    // the same bits), splits (mask order)
    for (int p = tid; p < NS2; p += THREADS) {
        const uint4 *src = reinterpret_cast<const uint4 *>(s.acc + (slot_of((uint32_t)p) << CB));
#pragma unroll
        for (int q = 0; q < NB / 2; ++q) *reinterpret_cast<uint4 *>(Pt + row + lpos((uint32_t)p, 2 * q)) = src[q];
    }
    for (int p = tid; p < ROW / 2; p += THREADS)
        reinterpret_cast<uint4 *>(Tt + row)[p] = reinterpret_cast<const uint4 *>(rS)[p];
    for (int p = tid; p < ROW / 4; p += THREADS)
        reinterpret_cast<uint4 *>(Sr + row)[p] = reinterpret_cast<const uint4 *>(split)[p];
}

// One self-pair item (as run_item, on narrow rows) whose group minimum goes to the
// narrow self-pair minima sacc (32-bit LDS atomics): every candidate of the
// self pair has A_H = S_H, so the 32-bit key order is the (cost, A) order.
__device__ inline void run_item_self(uint32_t item, const uint32_t *rA, const uint32_t *rB, uint32_t *sacc) {
    const uint32_t s2 = item & 0xffffu;
    const int k = __popc(s2);
    const int tb = (int)((item >> 28) & 7u);
    const uint32_t cnt = 1u << tb;
    const uint32_t slot_s2 = slot_of(s2);
    uint32_t a2 = (item >> 16) & 0xfffu;
    uint32_t best[NB];
#pragma unroll
    for (int x = 0; x < NB; ++x) best[x] = Key<uint32_t>::none();
    for (uint32_t i = 0; i < cnt; ++i) {
        if (a2 != s2) {
            const uint32_t sa = slot_of(a2), sb = slot_s2 ^ sa;
            uint32_t a[NB], b[NB];
            load_blk(rA, sa, a);
            load_blk(rB, sb, b);
            conv_full<uint32_t>(a, b, best);
        }
        a2 = ((a2 | ~s2) + 1u) & s2;
    }
    const uint32_t chunks = 1u << (k - tb);
    const uint32_t seg = chunks < 8u ? chunks : 8u;
    const uint32_t lane = threadIdx.x & (kWave - 1);
#pragma unroll
    for (int x = 0; x < NB; ++x) {
        uint32_t b = best[x];
        if (seg >= 2) { const uint32_t o = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)b, 0xB1, 0xF, 0xF, false); b = o < b ? o : b; }
        if (seg >= 4) { const uint32_t o = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)b, 0x4E, 0xF, 0xF, false); b = o < b ? o : b; }
        if (seg >= 8) { const uint32_t o = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)b, 0x141, 0xF, 0xF, false); b = o < b ? o : b; }
        best[x] = b;
    }
    if ((lane & (seg - 1)) == 0) {
#pragma unroll
        for (int x = 0; x < NB; ++x)
            if (best[x] != Key<uint32_t>::none()) atomicMin(&sacc[(s2 << CB) | x], best[x]);
    }
}

// Completes row S_H (non-empty) on narrow keys. In LDS: acc, the 64-bit
// cross-pair keys of the row; rSn, row S_H (tagged, filled here); r0n, row 0
// (plain); sacc, the narrow self-pair minima (4096 entries set to all ones
// before the caller's barrier). own: this thread's block (own_block_load).
// Writes the row to the plain 64-bit table, to both narrow tables and its
// splits to Sr (row-major, mask order inside a row). The self pair's
// candidates (A_H = S_H) are kept as 32-bit keys up to the comparison with
// the cross pairs' key of each entry. NT threads: each takes THREADS / NT
// items of a level (the item table is laid out for THREADS; its lane groups
// stay aligned since NT is a multiple of the wave).
//
// The levels issue no global stores: a finished block leaves its plain
// entries in its (no longer needed) acc entries and its splits in its sacc
// entries, and the whole row goes to HBM in coalesced pieces after the last
// level. The only global loads inside the levels are the next level's item
// entries, read unconditionally (clamped index, validity tested where they
// are used) into the other of two register sets, so that no wait for them
// comes before the next level: vector memory operations retire in order,
// and a wait for an older load would wait for every newer one.
template <class K, int NT = THREADS>
__device__ __attribute__((always_inline)) inline void finalize_row_narrow(
        int m, uint32_t sh, const OwnBlock<uint32_t> &own, uint64_t *acc, uint32_t *rSn, const uint32_t *r0n,
        uint32_t *sacc, uint64_t *__restrict__ Pt, uint32_t *__restrict__ Tn, uint32_t *__restrict__ Pn,
        uint32_t *__restrict__ Sr) {
    static_assert(THREADS % NT == 0 && NT % kWave == 0 && NT >= NS2 / 4, "items and blocks per thread");
    constexpr int IPT = THREADS / NT;
    const int H = m - L;
    const uint32_t row = sh << L;
    const uint64_t mask = ((uint64_t)1 << m) - 1u;
    const int tid = (int)threadIdx.x;
    // block 0 of row 0, plain narrow: C(X1 << H) << L for every low part X1
    uint32_t b0n[NB];
#pragma unroll
    for (int x = 0; x < NB; ++x) b0n[x] = r0n[npos(0u, x)];
    // S = (S_H, 0, 0) with one request in S_H is a leaf: C = W
    const bool single = (sh & (sh - 1u)) == 0;
    auto level = [&](int k, const uint32_t (&cur)[IPT], uint32_t (&nxt)[IPT]) __attribute__((always_inline)) {
        const int kn = k < R2 ? k + 1 : R2;     // (the last level reads entries it does not use)
#pragma unroll
        for (int i = 0; i < IPT; ++i) nxt[i] = item_load<NT>(kn, i);
        // A2 a proper submask of S2
        const int n_items = c_items.end[k] - c_items.begin[k];
#pragma unroll
        for (int i = 0; i < IPT; ++i)
            if (tid + i * NT < n_items) run_item_self(cur[i], rSn, r0n, sacc);
        lds_barrier();
        // A2 = S2: in-block pairs, one thread per block of this level; A =
        // (S_H, S2, A1) holds lowbit(S), B = (0, 0, S1 ^ A1) is in block 0
        // of row 0
        if (tid >= c_blocks.begin[k] && tid < c_blocks.end[k]) {
            const uint32_t s2 = own.s2;
            const uint32_t tag = s2 << CB;                       // in-row part of (S2, X1 = 0)
            // the block's self-pair minima and cross-pair keys, read together
            uint32_t sself[NB];
            {
                const uint4 *sp4 = reinterpret_cast<const uint4 *>(sacc + tag);
                const uint4 u0 = sp4[0], u1 = sp4[1];
                sself[0] = u0.x; sself[1] = u0.y; sself[2] = u0.z; sself[3] = u0.w;
                sself[4] = u1.x; sself[5] = u1.y; sself[6] = u1.z; sself[7] = u1.w;
            }
            // The cross pairs' keys (cost << m | A_L << H | A_H) as narrow
            // keys nacc = cost << L | A_L, and the least self-pair key that
            // loses to them: the self pair's key (A_H = S_H) wins where
            // nk < thr, with thr = nacc + 1 where S_H < A_H (equal narrow
            // keys go to the smaller A_H); none stays all ones. The cost is
            // below 2^20, so nacc + 1 does not overflow. The dependent chain
            // below then runs on 32-bit keys alone.
            uint32_t nacc[NB], thr[NB], aacc[NB];
            const uint32_t hmask = (1u << H) - 1u;
#pragma unroll
            for (int x = 0; x < NB; ++x) {
                const uint64_t ka = Key<K>::key_value(acc[tag | x]);
                const bool none = ka == ~0ull;
                const uint32_t n = ((uint32_t)(ka >> m) << L) | ((uint32_t)(ka >> H) & (ROW - 1u));
                nacc[x] = none ? ~0u : n;
                thr[x] = none ? ~0u : n + (sh < ((uint32_t)ka & hmask) ? 1u : 0u);
                aacc[x] = (uint32_t)(ka & mask);
            }
            const bool leaf0 = s2 == 0 && single;
            uint32_t on[NB], sp[NB];
            uint64_t cm[NB];
            // S1 in order of popcount so that every A1 < S1 is ready
#pragma unroll
            for (int pc = 0; pc <= CB; ++pc) {
#pragma unroll
                for (int s1 = 0; s1 < NB; ++s1) {
                    if (cpop(s1) != pc) continue;
                    uint32_t nk = sself[s1];
#pragma unroll
                    for (int a1 = 0; a1 < NB; ++a1) {
                        if ((a1 & ~s1) || a1 == s1) continue;
                        const uint32_t c = on[a1] + b0n[s1 ^ a1];
                        nk = c < nk ? c : nk;
                    }
                    const bool self = nk < thr[s1];
                    const uint32_t best = self ? nk : nacc[s1];
                    const uint32_t w = own.w[s1];
                    const bool leaf = s1 == 0 && leaf0;
                    const uint32_t c = leaf ? w : (best >> L) - w;
                    on[s1] = (c << L) | tag | (uint32_t)s1;
                    // off the chain: the split A (A_L << H | A_H) and the
                    // plain entry
                    sp[s1] = leaf ? 0u : self ? ((nk & (ROW - 1u)) << H) | sh : aacc[s1];
                    cm[s1] = (uint64_t)c << m;
                }
            }
            // the plain entries and the splits, over the entries just read
#pragma unroll
            for (int x = 0; x < NB; ++x) acc[tag | x] = Key<K>::store(cm[x]);
            uint4 *sp4 = reinterpret_cast<uint4 *>(sacc + tag);
            sp4[0] = make_uint4(sp[0], sp[1], sp[2], sp[3]);
            sp4[1] = make_uint4(sp[4], sp[5], sp[6], sp[7]);
            // C(X) << L, tagged with X_L = S2 << CB | X1
            const uint32_t sl = slot_of(s2);
#pragma unroll
            for (int q = 0; q < NB / 4; ++q)
                *reinterpret_cast<uint4 *>(rSn + npos(sl, 4 * q)) =
                    make_uint4(on[4 * q], on[4 * q + 1], on[4 * q + 2], on[4 * q + 3]);
        }
        lds_barrier();
    };
    uint32_t ia[IPT], ib[IPT];
#pragma unroll
    for (int i = 0; i < IPT; ++i) ia[i] = item_load<NT>(0, i);
    for (int k = 0; k <= R2; k += 2) {
        level(k, ia, ib);
        if (k + 1 <= R2) level(k + 1, ib, ia);
    }
    // the row to HBM: plain entries (the block at slot p, plane by plane),
    // splits (mask order), and the tagged and plain narrow rows (the LDS
    // layout is the table's)
    for (int p = tid; p < NS2; p += NT) {
        const uint4 *src = reinterpret_cast<const uint4 *>(acc + (slot_of((uint32_t)p) << CB));
#pragma unroll
        for (int q = 0; q < NB / 2; ++q) *reinterpret_cast<uint4 *>(Pt + row + lpos((uint32_t)p, 2 * q)) = src[q];
    }
    const uint32_t lo = ~(ROW - 1u);
    for (int p = tid; p < ROW / 4; p += NT) {
        reinterpret_cast<uint4 *>(Sr + row)[p] = reinterpret_cast<const uint4 *>(sacc)[p];
        const uint4 tv = reinterpret_cast<const uint4 *>(rSn)[p];
        reinterpret_cast<uint4 *>(Tn + row)[p] = tv;
        reinterpret_cast<uint4 *>(Pn + row)[p] = make_uint4(tv.x & lo, tv.y & lo, tv.z & lo, tv.w & lo);
    }
}

template <class K>
__device__ inline const K *lds_at(uint32_t off) {
    return (const K *)(__attribute__((address_space(3))) const K *)(uintptr_t)off;
}

// one base step (S2', A2') of the lifted cross-pair loop: three block
// convolutions from four block loads. off_a, off_b: LDS byte offsets of
// blocks A2' (tagged row) and B2' = S2' ^ A2' (plain row); the blocks with
// E sit NS2/2 slots above those without, a constant offset. KI is the key
// type in LDS: a wide K, or uint32_t for narrow rows. The keys of in0/in1
// (outputs S2' and S2'|E) are folded into out0/out1 (in and out may be the
// same arrays).
template <class KI>
__device__ __attribute__((always_inline)) inline void cross_step(uint32_t off_a, uint32_t off_b, const KI in0[NB],
                                                                 const KI in1[NB], KI out0[NB], KI out1[NB]) {
    constexpr uint32_t HALF = NS2 / 2;
    const KI *pa = lds_at<KI>(off_a), *pb = lds_at<KI>(off_b);
    KI a0[NB], a1[NB], b0[NB], b1[NB];
    load_blk(pa, 0u, a0);                                 // A2'
    load_blk(pb, HALF, b1);                               // B2'|E
    load_blk(pb, 0u, b0);                                 // B2'
    load_blk(pa, HALF, a1);                               // A2'|E
    conv_into<KI>(a0, b1, in1, out1);                     // (S2'|E, A2')
    conv_into<KI>(a0, b0, in0, out0);                     // (S2', A2')
    conv_into<KI>(a1, b0, out1, out1);                    // (S2'|E, A2'|E)
    // 64-bit keys: steps kept apart (measured faster). Narrow keys leave
    // registers for the compiler to start a step's reads during the
    // previous step's arithmetic (measured faster there).
    if (!std::is_same<KI, uint32_t>::value) __builtin_amdgcn_sched_barrier(0);
}

// Cross pairs of one (S_H, chunk). The level's rows (colex ranks) come in
// two parts: the first head_rows rows in chunks of per_chunk pairs (one
// chunk, with fused set: the row is finished in place), then the other rows
// in tail_chunks chunks of tail_per_chunk pairs, so that the level's last
// round of workgroups is filled with short ones. The head's workgroups come
// first in launch order. Chunk partials: head chunk b of the launch at slot
// b, tail chunk b' at slot tail_base + b'. NARROW: the pairs run on the
// narrow tables (Tn tagged, Pn plain), in the wide rows' space.
template <class K, bool NARROW>
__global__ __launch_bounds__(THREADS) void k_rb_cross(int m, int h, uint32_t n_pairs, uint32_t chunks,
                                                      uint32_t per_chunk, int fused, uint32_t head_rows,
                                                      uint32_t tail_chunks, uint32_t tail_per_chunk, uint32_t tail_base,
                                                      const int64_t *__restrict__ Wr,
                                                      uint64_t *__restrict__ Tt, uint64_t *__restrict__ Pt,
                                                      uint32_t *__restrict__ Tn, uint32_t *__restrict__ Pn,
                                                      uint32_t *__restrict__ Sr, uint64_t *__restrict__ partial) {
    typedef typename std::conditional<NARROW, uint32_t, K>::type KI;
    __shared__ Lds<K> s;
    const uint32_t head_wgs = head_rows * chunks;
    uint32_t r, j, pc, slot;
    bool fz;
    if (blockIdx.x < head_wgs) {
        const uint32_t b = xcd_block(blockIdx.x, head_wgs);
        r = b / chunks;
        j = b % chunks;
        pc = per_chunk;
        fz = fused != 0;
        slot = b;
    } else {
        const uint32_t b = xcd_block(blockIdx.x - head_wgs, gridDim.x - head_wgs);
        r = head_rows + b / tail_chunks;
        j = b % tail_chunks;
        pc = tail_per_chunk;
        fz = false;
        slot = tail_base + b;
    }
    const uint32_t sh = unrank_colex(r, h, m - L);
    const uint32_t lowh = sh & (0u - sh);
    const uint32_t rest = sh ^ lowh;
    const uint32_t t0 = j * pc;
    const uint32_t t1 = min(n_pairs, t0 + pc);
    uint32_t ah = t0 < t1 ? (lowh | deposit(t0, rest)) : 0u;
    // this thread's item, its best keys for outputs S2' and S2'|E
    constexpr uint32_t E = 1u << RL;
    const uint32_t item = c_titems.v[threadIdx.x];
    const bool has_item = (item >> 31) != 0;
    const uint32_t s2 = item & 0xffu;
    const uint32_t a2_first = (item >> 8) & 0xffu;
    const uint32_t cnt = (item >> 16) & 15u;
    const uint32_t slot_s2 = slot_of(s2);
    const uint32_t low2 = s2 & (0u - s2);
    const uint32_t low_off = slot_of(low2) * 16u;                    // block offset of lowbit(S2')
    static_assert(RL == R2 - 1 && (1u << RL) == NS2 / 2, "E is the top middle bit");
    static_assert(NS2 / 2 * 16 <= 16 * 1024, "slot offsets stay below the row size");
    // Best keys of the two output blocks. Narrow keys use two register sets:
    // pair t of the chunk folds set (t - t0) & 1 into the other one, so the
    // keys a pair starts from are still there when it ends, for the A_H
    // tracking to compare with no copies.
    KI bp0[NB], bp1[NB], bq0[NB], bq1[NB];
    uint32_t bh0[NB], bh1[NB];                                       // NARROW: A_H of each best key
#pragma unroll
    for (int x = 0; x < NB; ++x) {
        bp0[x] = Key<KI>::none();
        bp1[x] = Key<KI>::none();
        bq0[x] = Key<KI>::none();
        bq1[x] = Key<KI>::none();
        bh0[x] = 0u;
        bh1[x] = 0u;
    }
    // The item's block offsets (bytes inside a row) of the even submask of
    // each of its up to four two-step rounds, the same for every pair: an
    // item starts at a submask without lowbit(S2') and has an even count, the
    // odd submask is the even one plus lowbit(S2'), and slot_of is
    // GF(2)-linear, so the odd step's offsets are the even step's XOR
    // low_off. The item of S2' = 0 (its one submask) runs the same way: with
    // lowbit 0 both steps are that submask, and a repeated candidate leaves a
    // minimum as it is.
    // (Narrow keys keep them in registers; wide keys, short of registers,
    // compute each round's as it comes.)
    auto round_offsets = [&](uint32_t &a2, uint32_t &fa, uint32_t &fb) {
        const uint32_t sa = slot_of(a2) & (NS2 / 2 - 1u);
        fa = sa * 16u;
        fb = ((slot_s2 ^ sa) & (NS2 / 2 - 1u)) * 16u;
        a2 = ((a2 | low2 | ~s2) + 1u) & s2;                          // two submasks on
    };
    uint32_t oa_item[4], ob_item[4];
    if constexpr (NARROW) {
        uint32_t a2 = a2_first;
#pragma unroll
        for (int i = 0; i < 4; ++i) round_offsets(a2, oa_item[i], ob_item[i]);
    }
    // row buffer [buf][side] of this kernel's key type
    auto buf = [&](int b, int side) -> KI * {
        if constexpr (NARROW) return reinterpret_cast<uint32_t *>(&s.r[0][0][0]) + (b * 2 + side) * ROW;
        else return s.r[b][side];
    };
    auto copy_pair = [&](int b, uint32_t a_h) {
        if constexpr (NARROW) {
            copy_row_quiet(buf(b, 0), Tn, a_h);
            copy_row_quiet(buf(b, 1), Pn, sh ^ a_h);
        } else {
            copy_row_quiet(buf(b, 0), Tt, a_h);
            copy_row_quiet(buf(b, 1), Pt, sh ^ a_h);
        }
    };
    // A_H tracking of a finished pair (narrow keys): a key the pair lowered
    // came from it; an equal key keeps the earlier, smaller A_H. It runs at
    // the start of the next pair, where it overlaps that pair's first LDS
    // reads (that pair writes its keys over the set compared here only
    // after those reads), and after the last pair.
    uint32_t ah_prev = 0;
    auto track = [&](const KI *o0, const KI *o1, const KI *i0, const KI *i1) {
#pragma unroll
        for (int x = 0; x < NB; ++x) {
            bh0[x] = o0[x] < i0[x] ? ah_prev : bh0[x];
            bh1[x] = o1[x] < i1[x] ? ah_prev : bh1[x];
        }
    };
    // (wide keys) pair t of the chunk runs on buffer (t - t0) & 1 while the
    // rows of pair t + 1 are copied into the other one
    auto pair = [&](auto cur_c, uint32_t t) {
        constexpr int CUR = decltype(cur_c)::value;
        // (wide keys track nothing: one set, updated in place)
        KI *in0 = (NARROW && CUR) ? bq0 : bp0, *in1 = (NARROW && CUR) ? bq1 : bp1;
        KI *out0 = !NARROW ? bp0 : CUR ? bp0 : bq0, *out1 = !NARROW ? bp1 : CUR ? bp1 : bq1;
        copies_done();
        lds_barrier();     // rows of pair t in place; pair t - 1 done with the other buffer
        const uint32_t ah_cur = ah;
        const uint32_t an = lowh | (((ah | ~rest) + 1u) & rest);    // next A_H holding lowbit(S_H)
        if (t + 1 < t1) copy_pair(CUR ^ 1, an);
        ah = an;
        // The buffers' LDS offsets (multiples of the row size). Wide buffer 1
        // lies beyond the 16-bit immediates, so wide bases are kept opaque to
        // the compiler and added once per address.
        typedef __attribute__((address_space(3))) const KI lds_k;
        uint32_t oa = (uint32_t)(uintptr_t)(lds_k *)buf(CUR, 0);
        uint32_t ob = (uint32_t)(uintptr_t)(lds_k *)buf(CUR, 1);
        if constexpr (!NARROW) asm("" : "+s"(oa), "+s"(ob));
        if (has_item) {
            // pair t - 1 folded this pair's output set into its input set
            if constexpr (NARROW)
                if (t > t0) track(in0, in1, out0, out1);
            uint32_t a2 = a2_first;
            auto two = [&](int i, const KI *i0, const KI *i1) {
                uint32_t fa, fb;
                if constexpr (NARROW) {
                    fa = oa_item[i];
                    fb = ob_item[i];
                } else {
                    round_offsets(a2, fa, fb);
                }
                cross_step<KI>(oa + fa, ob + fb, i0, i1, out0, out1);
                cross_step<KI>(oa + (fa ^ low_off), ob + (fb ^ low_off), out0, out1, out0, out1);
            };
            // (the next pair's copies, unseen by the compiler's wait
            // insertion, land while this pair runs and are awaited when the
            // next pair starts)
            two(0, in0, in1);
            if constexpr (NARROW) {
                if (cnt > 2) two(1, out0, out1);
                if (cnt > 4) two(2, out0, out1);
                if (cnt > 6) two(3, out0, out1);
            } else {
                for (uint32_t i = 2; i < cnt; i += 2) two(0, out0, out1);
            }
        }
        ah_prev = ah_cur;
    };
    if constexpr (NARROW) {
        // Narrow keys run the pairs in sets of two: the four narrow row pairs
        // fill the 128 KiB of row buffers (set 0 in slots 0, 1, set 1 in
        // slots 2, 3), so one barrier and one batch of copies serve two
        // pairs; the copies of the next set (unseen by the compiler's wait
        // insertion) stay in flight for the whole set and are awaited when
        // the next set starts. Set 1 lies 64 KiB up, past the reads' 16-bit immediate
        // offsets: its pairs add 64 KiB to the items' offset registers and
        // take set 0's immediates.
        auto adv = [&](uint32_t x) __attribute__((always_inline)) { return lowh | (((x | ~rest) + 1u) & rest); };
        uint32_t ah_copy = ah, ah_run = ah;
        auto copy_set = [&](int S, uint32_t t) __attribute__((always_inline)) {
            if (t < t1) { copy_pair(2 * S, ah_copy); ah_copy = adv(ah_copy); }
            if (t + 1 < t1) { copy_pair(2 * S + 1, ah_copy); ah_copy = adv(ah_copy); }
        };
        auto pair_n = [&](auto cur_c, uint32_t t) __attribute__((always_inline)) {
            constexpr int CUR = decltype(cur_c)::value;
            KI *in0 = CUR ? bq0 : bp0, *in1 = CUR ? bq1 : bp1;
            KI *out0 = CUR ? bp0 : bq0, *out1 = CUR ? bp1 : bq1;
            const uint32_t ah_cur = ah_run;
            ah_run = adv(ah_run);
            typedef __attribute__((address_space(3))) const KI lds_k;
            const uint32_t oa = (uint32_t)(uintptr_t)(lds_k *)buf(CUR, 0);
            const uint32_t ob = (uint32_t)(uintptr_t)(lds_k *)buf(CUR, 1);
            if (has_item) {
                if (t > t0) track(in0, in1, out0, out1);
                auto two = [&](int i, const KI *i0, const KI *i1) __attribute__((always_inline)) {
                    const uint32_t fa = oa_item[i], fb = ob_item[i];
                    cross_step<KI>(oa + fa, ob + fb, i0, i1, out0, out1);
                    cross_step<KI>(oa + (fa ^ low_off), ob + (fb ^ low_off), out0, out1, out0, out1);
                };
                two(0, in0, in1);
                if (cnt > 2) two(1, out0, out1);
                if (cnt > 4) two(2, out0, out1);
                if (cnt > 6) two(3, out0, out1);
            }
            ah_prev = ah_cur;
        };
        auto shift = [&](uint32_t d) __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                oa_item[i] += d;
                ob_item[i] += d;
                // opaque: the old values die here instead of being kept for after set 1
                asm volatile("" : "+v"(oa_item[i]), "+v"(ob_item[i]));
            }
        };
        auto set_run = [&](auto s_c, uint32_t t) __attribute__((always_inline)) {
            constexpr int S = decltype(s_c)::value;
            copies_done();
            lds_barrier();     // rows of this set in place; the previous set done with the other one
            copy_set(S ^ 1, t + 2);
            if constexpr (S == 1) shift(0x10000u);
            pair_n(std::integral_constant<int, 0>{}, t);
            if (t + 1 < t1) pair_n(std::integral_constant<int, 1>{}, t + 1);
            if constexpr (S == 1) shift(0u - 0x10000u);
        };
        if (t0 < t1) copy_set(0, t0);
        for (uint32_t t = t0; t < t1; t += 4) {
            set_run(std::integral_constant<int, 0>{}, t);
            if (t + 2 < t1) set_run(std::integral_constant<int, 1>{}, t + 2);
        }
    } else {
        if (t0 < t1) copy_pair(0, ah);
        for (uint32_t t = t0; t < t1; t += 2) {
            pair(std::integral_constant<int, 0>{}, t);
            if (t + 1 < t1) pair(std::integral_constant<int, 1>{}, t + 1);
        }
    }
    // The lanes' best keys are combined through LDS: every lane stages its
    // 16 keys (8 of block S2', 8 of S2'|E) as accumulator key bits (~0 for
    // none) in the row buffers, and each quarter of a wave then takes the
    // minimum over the lanes of its S2' for each of the S2''s 16 entries
    // (the gather plan). The minimum of the packed keys is the (cost, A)
    // order, so this equals one atomic minimum per lane and entry, without
    // the atomics. Key q of lane i sits at 16 i + (q ^ (i & 15)): a lane's
    // 16 stores and a quarter's 16 reads of one lane fall in distinct banks.
    uint64_t *stage = reinterpret_cast<uint64_t *>(&s.r[0][0][0]);
    static_assert(2 * NB * THREADS * sizeof(uint64_t) <= sizeof(s.r), "the staged keys fit the row buffers");
    const uint32_t quarter = (threadIdx.x / 16u) & 3u, q16 = threadIdx.x & 15u;
    const GatherSlot &gslot = c_gather.s[threadIdx.x / kWave][quarter];
    const uint4 gruns = *reinterpret_cast<const uint4 *>(gslot.runs);   // loaded ahead of the barriers
    const uint32_t gs2 = gslot.s2;
    lds_barrier();     // every wave is done with the rows
    if (has_item) {
        // the last pair's tracking; an odd number of pairs leaves the keys in
        // the second set
        // (a branch, not a pointer select, keeps both sets in registers)
        auto stage_set = [&](const KI *f0, const KI *f1) {
            const int H = m - L;
            uint64_t *own = stage + 16u * threadIdx.x;
            const uint32_t sw = threadIdx.x & 15u;
#pragma unroll
            for (int q = 0; q < 2 * NB; ++q) {
                const KI b = q < NB ? f0[q] : f1[q - NB];
                uint64_t v;
                if constexpr (NARROW) {
                    const uint32_t h = q < NB ? bh0[q] : bh1[q - NB];
                    const uint64_t key = ((uint64_t)(b >> L) << m) | ((uint64_t)(b & (ROW - 1u)) << H) | h;
                    v = b == Key<uint32_t>::none() ? ~0ull : Key<K>::key_bits(key);
                } else {
                    v = b == Key<K>::none() ? ~0ull : Key<K>::bits(b);
                }
                own[(uint32_t)q ^ sw] = v;
            }
        };
        if (NARROW && ((t1 - t0) & 1u)) {
            track(bq0, bq1, bp0, bp1);
            stage_set(bq0, bq1);
        } else {
            if (NARROW && t1 > t0) track(bp0, bp1, bq0, bq1);
            stage_set(bp0, bp1);
        }
    }
    lds_barrier();
    {
        const uint32_t gw[4] = {gruns.x, gruns.y, gruns.z, gruns.w};
        auto m2 = [](uint64_t a, uint64_t b) { return a < b ? a : b; };
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            uint64_t v = ~0ull;
#pragma unroll
            for (int r = 0; r < kRuns; ++r) {
                const uint32_t word = gw[jj] >> (16 * r);
                const uint32_t first = word & 1023u, n = (word >> 10) & 63u;
                // four reads in flight; a lane past the run repeats its last
                for (uint32_t i = 0; i < n; i += 4) {
                    auto at = [&](uint32_t k) {
                        const uint32_t ln = first + min(i + k, n - 1u);
                        return stage[16u * ln + (q16 ^ (ln & 15u))];
                    };
                    const uint64_t o0 = at(0), o1 = at(1), o2 = at(2), o3 = at(3);
                    v = m2(v, m2(m2(o0, o1), m2(o2, o3)));
                }
            }
            const uint32_t sp = (gs2 >> (8 * jj)) & 0xffu;
            const uint32_t e = ((q16 < NB ? sp : (sp | E)) << CB) | (q16 & (NB - 1u));
            if (fz) s.acc[e] = v;
            else partial[(size_t)slot * ROW + e] = v;
        }
    }
    lds_barrier();     // the staged keys are read before the buffers are reused
    if (fz) {
        OwnBlock<typename std::conditional<NARROW, uint32_t, int64_t>::type> own;
        own_block_load(sh, Wr, own);
        if constexpr (NARROW) {
            copy_row(buf(0, 1), Pn, 0u);
            uint32_t *sacc = buf(1, 0);
            for (int e = threadIdx.x; e < ROW; e += THREADS) sacc[e] = Key<uint32_t>::none();
        } else {
            copy_row(s.r[0][1], Pt, 0u);
        }
        copies_done();
        lds_barrier();
        if constexpr (NARROW) finalize_row_narrow<K>(m, sh, own, s.acc, buf(0, 0), buf(0, 1), buf(1, 0), Pt, Tn, Pn, Sr);
        else finalize_row<K>(m, sh, own, s, s.r[0][0], s.r[0][1], Tt, Pt, Sr);
    }
}

// min over the chunks of one S_H, into chunk 0's slot. Block (r, e-range,
// g) folds chunks 1 + g, 1 + g + G, ... of entries e into chunk 0 with a
// 64-bit atomic min (unsigned order = key order).
constexpr int RED_CHUNKS_PER_BLOCK = 32;
__global__ __launch_bounds__(256) void k_rb_reduce(uint32_t chunks, uint32_t groups, uint64_t *__restrict__ partial) {
    const uint32_t per_set = (ROW / 256) * groups;
    const uint32_t r = blockIdx.x / per_set;
    const uint32_t rem = blockIdx.x % per_set;
    const uint32_t e = (rem % (ROW / 256)) * 256 + threadIdx.x;
    const uint32_t g = rem / (ROW / 256);
    uint64_t *base = partial + (size_t)r * chunks * ROW + e;
    uint64_t v = ~0ull;
    for (uint32_t j = 1 + g; j < chunks; j += groups) {
        const uint64_t o = base[(size_t)j * ROW];
        v = o < v ? o : v;
    }
    if (v != ~0ull) atomicMin((unsigned long long *)base, (unsigned long long)v);
}

// A row's cross-pair keys into LDS acc from its c chunk slots (the first
// at slot; as k_rb_cross lays them out: head rows in chunks, the others in
// tail_chunks from tail_base), by NT threads: none without chunks (level 1
// has no cross pairs); up to kFoldChunks chunks folded here, with every
// thread's loads in flight together (16 bytes each); more chunks were
// folded into the first slot by k_rb_reduce, which is then copied directly.
// Completion: copies_done, then a workgroup barrier.
constexpr uint32_t kFoldChunks = 16;
template <int NT>
__device__ inline void load_row_keys(uint64_t *acc, const uint64_t *__restrict__ partial, size_t slot, uint32_t c) {
    if (c == 0) {
        for (int e = threadIdx.x; e < ROW; e += NT) acc[e] = ~0ull;
    } else if (c > kFoldChunks) {
        copy_row<uint64_t, NT>(acc, partial, (uint32_t)slot);
    } else {
        const ulonglong2 *src = reinterpret_cast<const ulonglong2 *>(partial + slot * ROW);
        constexpr int PER = ROW / 2 / NT;                       // 16-byte pieces per thread
        ulonglong2 v[PER];
#pragma unroll
        for (int q = 0; q < PER; ++q) v[q] = src[threadIdx.x + q * NT];
        for (uint32_t j = 1; j < c; ++j) {
            ulonglong2 o[PER];
#pragma unroll
            for (int q = 0; q < PER; ++q) o[q] = src[(size_t)j * (ROW / 2) + threadIdx.x + q * NT];
#pragma unroll
            for (int q = 0; q < PER; ++q) {
                v[q].x = o[q].x < v[q].x ? o[q].x : v[q].x;
                v[q].y = o[q].y < v[q].y ? o[q].y : v[q].y;
            }
        }
        ulonglong2 *dst = reinterpret_cast<ulonglong2 *>(acc);
#pragma unroll
        for (int q = 0; q < PER; ++q) dst[threadIdx.x + q * NT] = v[q];
    }
}

// finish rows row_offset + blockIdx.x of one level on 64-bit keys (narrow
// rows: k_rb_final_narrow), acc from the row's chunk slots (load_row_keys)
template <class K>
__global__ __launch_bounds__(THREADS) void k_rb_final(int m, int h, uint32_t row_offset, uint32_t head_rows,
                                                      uint32_t chunks, uint32_t tail_chunks, uint32_t tail_base,
                                                      const int64_t *__restrict__ Wr,
                                                      uint64_t *__restrict__ Tt, uint64_t *__restrict__ Pt,
                                                      uint32_t *__restrict__ Sr, const uint64_t *__restrict__ partial) {
    __shared__ Lds<K> s;
    const uint32_t r = row_offset + blockIdx.x;
    const uint32_t sh = unrank_colex(r, h, m - L);
    const uint32_t c = r < head_rows ? chunks : tail_chunks;
    const size_t slot = r < head_rows ? (size_t)r * chunks : tail_base + (size_t)(r - head_rows) * tail_chunks;
    OwnBlock<int64_t> own;
    own_block_load(sh, Wr, own);
    load_row_keys<THREADS>(s.acc, partial, slot, c);
    copy_row(s.r[0][1], Pt, 0u);
    copies_done();
    lds_barrier();
    finalize_row<K>(m, sh, own, s, s.r[0][0], s.r[0][1], Tt, Pt, Sr);
}

// k_rb_final on narrow rows, in NT threads and half the CU's LDS (the
// accumulator row and three narrow rows). With NT = FINAL_THREADS, half the
// threads of a CU, two rows are finished on a CU at a time: the finishing's
// phases are bound by latency, and the two workgroups' phases overlap. A
// launch of at most one row per CU takes NT = THREADS: every row then has
// all of its CU's threads.
constexpr int FINAL_THREADS = THREADS / 2;
struct alignas(16) LdsFinalNarrow {
    uint64_t acc[ROW];
    uint32_t nr[3 * ROW];      // row S_H (tagged), row 0 (plain), the self-pair minima
};
static_assert(2 * sizeof(LdsFinalNarrow) <= 160 * 1024, "two narrow finishing workgroups per CU");
template <class K, int NT>
__global__ __launch_bounds__(NT) void k_rb_final_narrow(int m, int h, uint32_t row_offset,
                                                                   uint32_t head_rows, uint32_t chunks,
                                                                   uint32_t tail_chunks, uint32_t tail_base,
                                                                   const int64_t *__restrict__ Wr,
                                                                   uint64_t *__restrict__ Pt,
                                                                   uint32_t *__restrict__ Tn,
                                                                   uint32_t *__restrict__ Pn,
                                                                   uint32_t *__restrict__ Sr,
                                                                   const uint64_t *__restrict__ partial) {
    __shared__ LdsFinalNarrow s;
    const uint32_t r = row_offset + blockIdx.x;
    const uint32_t sh = unrank_colex(r, h, m - L);
    const uint32_t c = r < head_rows ? chunks : tail_chunks;
    const size_t slot = r < head_rows ? (size_t)r * chunks : tail_base + (size_t)(r - head_rows) * tail_chunks;
    OwnBlock<uint32_t> own;
    own_block_load(sh, Wr, own);
    load_row_keys<NT>(s.acc, partial, slot, c);
    copy_row<uint32_t, NT>(s.nr + ROW, Pn, 0u);
    for (int e = threadIdx.x; e < ROW; e += NT) s.nr[2 * ROW + e] = Key<uint32_t>::none();
    copies_done();
    lds_barrier();
    finalize_row_narrow<K, NT>(m, sh, own, s.acc, s.nr, s.nr + ROW, s.nr + 2 * ROW, Pt, Tn, Pn, Sr);
}

// the in-row masks grouped by popcount, for the row-0 DP
struct Subsets { uint16_t v[ROW]; int begin[L + 2]; };
constexpr Subsets make_subsets() {
    Subsets t{};
    int count[L + 1] = {};
    for (int e = 0; e < ROW; ++e) ++count[cpop(e)];
    t.begin[0] = 0;
    for (int k = 0; k <= L; ++k) t.begin[k + 1] = t.begin[k] + count[k];
    int at[L + 1] = {};
    for (int k = 0; k <= L; ++k) at[k] = t.begin[k];
    for (int e = 0; e < ROW; ++e) t.v[at[cpop(e)]++] = (uint16_t)e;
    return t;
}
__constant__ Subsets c_subsets = make_subsets();

// Row 0: the DP over the L requests of the in-row part alone (S_H empty),
// level by level in |S_L|, a group of lanes per subset; the key of a candidate is
// C'(A) + C'(S ^ A) + A's mask, with A holding lowbit(S). Writes row 0 to the
// plain table (it is only ever a B row; NARROW: to the narrow plain table as
// well, for the self pairs) and its splits.
template <class K, bool NARROW>
__global__ __launch_bounds__(THREADS) void k_rb_row0(int m, const int64_t *__restrict__ Wr,
                                                     uint64_t *__restrict__ Pt, uint32_t *__restrict__ Pn,
                                                     uint32_t *__restrict__ Sr) {
    __shared__ uint64_t c[ROW];
    __shared__ int64_t wrow[ROW];          // W of row 0, read once
    __shared__ uint32_t spl[ROW];
    const int H = m - L;
    const uint64_t mask = ((uint64_t)1 << m) - 1u;
    for (int e = threadIdx.x; e < ROW; e += THREADS) {
        const int64_t w = Wr[e];
        wrow[e] = w;
        c[e] = __popc((uint32_t)e) == 1 ? (uint64_t)w << m : 0u;         // C(empty) = 0 is never a part
        spl[e] = 0u;
    }
    __syncthreads();
    const int wv = (int)(threadIdx.x / kWave), lane = (int)(threadIdx.x & (kWave - 1));
    for (int p = 2; p <= L; ++p) {
        // one thread per subset while a subset has at most 63 candidates,
        // two at |S| = 8 (each level is then one round of the workgroup), a
        // wave per subset above; lane li of a group takes candidates li,
        // li + G, ..., its A' stepping by a masked add of G
        const int G = p <= 7 ? 1 : p == 8 ? 2 : kWave;
        const uint32_t n_sub = (uint32_t)(c_subsets.begin[p + 1] - c_subsets.begin[p]);
        const uint32_t per_wave = (uint32_t)(kWave / G);
        const uint32_t gl = (uint32_t)(lane / G), li = (uint32_t)(lane % G);
        for (uint32_t r0 = (uint32_t)wv * per_wave; r0 < n_sub; r0 += (uint32_t)(THREADS / kWave) * per_wave) {
            const uint32_t r = r0 + gl;
            uint64_t kb = ~0ull;
            uint32_t S = 0;
            if (r < n_sub) {
                S = c_subsets.v[c_subsets.begin[p] + (int)r];
                const uint32_t lb = S & (0u - S), rest = S ^ lb;
                const uint32_t n_a = (1u << (p - 1)) - 1u;   // A = lb | A', A' a proper subset of rest
                const uint32_t step = deposit((uint32_t)G, rest);
                uint32_t ap = deposit(li, rest);
                for (uint32_t t = li; t < n_a; t += (uint32_t)G) {
                    const uint32_t A = lb | ap;
                    const uint64_t key = c[A] + c[S ^ A] + ((uint64_t)A << H);
                    kb = key < kb ? key : kb;
                    ap = ((ap | ~rest) + step) & rest;
                }
            }
            for (int off = G / 2; off > 0; off >>= 1) {
                const uint64_t o = __shfl_xor(kb, off, kWave);
                kb = o < kb ? o : kb;
            }
            if (r < n_sub && li == 0) {
                c[S] = ((kb >> m) - (uint64_t)wrow[S]) << m;
                spl[S] = (uint32_t)(kb & mask);
            }
        }
        __syncthreads();
    }
    for (int e = threadIdx.x; e < ROW; e += THREADS) {
        Pt[lpos(slot_of((uint32_t)e >> CB), e & (NB - 1))] = Key<K>::store(c[e]);
        if (NARROW) Pn[npos(slot_of((uint32_t)e >> CB), e & (NB - 1))] = (uint32_t)(c[e] >> m) << L;
        Sr[e] = spl[e];
    }
}

// plain table -> C in mask order: C[S_H | S_L << H] = C'(S) >> m (C[0]
// keeps the documented sentinel). Tiles of 64 rows x 64 stored elements go
// through LDS, so reads run along rows and writes along S_H; VEC writes two
// entries per 16-byte store (C 16-byte aligned).
template <class K, bool VEC>
__global__ __launch_bounds__(256) void k_rb_unpack(int m, const uint64_t *__restrict__ Pt, int64_t *__restrict__ C) {
    __shared__ int64_t tile[64][65];
    const int H = m - L;
    const uint32_t R = 1u << H;                                // rows, a power of two >= 2
    const uint32_t r0 = blockIdx.x * 64u, e0 = blockIdx.y * 64u;
    const int tx = (int)(threadIdx.x & 31u), ty = (int)(threadIdx.x >> 5);
    // reads: 16 bytes (two stored elements) per lane along a row
    for (int i = ty; i < 64; i += 8) {
        const uint32_t r = r0 + (uint32_t)i;
        if (r < R) {
            const ulonglong2 v = *reinterpret_cast<const ulonglong2 *>(Pt + ((size_t)r << L) + e0 + 2u * (uint32_t)tx);
            tile[i][2 * tx] = (int64_t)(Key<K>::stored_value(v.x) >> m);
            tile[i][2 * tx + 1] = (int64_t)(Key<K>::stored_value(v.y) >> m);
        }
    }
    __syncthreads();
    // writes: 16 bytes (two consecutive S_H) per lane along mask order
    for (int jj = ty; jj < 64; jj += 8) {
        const uint32_t e = e0 + (uint32_t)jj;                  // stored element of every row in the tile
        const uint32_t q = e / PLANE, o = e % PLANE;
        const uint32_t sl = (slot_of(o >> 1) << CB) | (2u * q + (o & 1u));   // its in-row mask
        const uint32_t r = r0 + 2u * (uint32_t)tx;
        if (r < R) {
            const int64_t x = (r == 0 && sl == 0) ? kInf : tile[2 * tx][jj], y = tile[2 * tx + 1][jj];
            int64_t *dst = C + ((size_t)r | ((size_t)sl << H));
            if (VEC) {
                *reinterpret_cast<longlong2 *>(dst) = make_longlong2(x, y);
            } else {
                dst[0] = x;
                dst[1] = y;
            }
        }
    }
}

// out[c][r] = in[r][c] for a row-major R x Cn matrix, tiles of 64 x 64.
// Each lane moves V consecutive elements per global access (R and Cn are
// multiples of V).
template <class T, int V>
__global__ __launch_bounds__(256) void k_transpose(const T *__restrict__ in, T *__restrict__ out, uint32_t R,
                                                   uint32_t Cn) {
    constexpr int TW = 64 / V;                 // lanes across 64 elements
    constexpr int TH = 256 / TW;               // tile rows per pass
    typedef T Vec __attribute__((ext_vector_type(V)));
    __shared__ T tile[64][65];
    const uint32_t r0 = blockIdx.y * 64u, c0 = blockIdx.x * 64u;
    const int tx = (int)(threadIdx.x % TW), ty = (int)(threadIdx.x / TW);
    for (int i = ty; i < 64; i += TH) {
        const uint32_t r = r0 + (uint32_t)i, c = c0 + (uint32_t)(tx * V);
        if (r < R && c < Cn) {
            const Vec v = *reinterpret_cast<const Vec *>(in + (size_t)r * Cn + c);
#pragma unroll
            for (int k = 0; k < V; ++k) tile[i][tx * V + k] = v[k];
        }
    }
    __syncthreads();
    for (int jj = ty; jj < 64; jj += TH) {
        const uint32_t c = c0 + (uint32_t)jj, r = r0 + (uint32_t)(tx * V);
        if (r < R && c < Cn) {
            Vec v;
#pragma unroll
            for (int k = 0; k < V; ++k) v[k] = tile[tx * V + k][jj];
            *reinterpret_cast<Vec *>(out + (size_t)c * R + r) = v;
        }
    }
}

// sum_i W({i}), saturated, for the packed-key eligibility test
__global__ void k_request_total(int m, const int64_t *W, WsHeader *h) {
    if (threadIdx.x != 0) return;
    int64_t tot = 0;
    for (int i = 0; i < m; ++i) {
        const int64_t v = W[(int64_t)1 << i];
        tot = (v >= INT64_MAX - tot) ? INT64_MAX : tot + v;
    }
    h->total = tot;
}
}  // namespace rb

// ---------------------------------------------------------------------------
// phase 3: one workgroup per request i. Chunk x of R_i is emitted at the
// first node of i's root-to-leaf path that lies inside S_x; inside a node
// chunks go in ascending id. Every slot gets the key (request, depth, id);
// one sort of all keys then leaves each request's chunks in its own slot
// range, in emission order (keys are distinct: ids are distinct within R_i).
__global__ __launch_bounds__(256) void k_extract(int m, int64_t n_chunks, int64_t nnz, const int64_t *req_off,
                                                 const int32_t *req_chunks, const uint32_t *sig,
                                                 const uint32_t *split, uint64_t *keys, WsHeader *h) {
    __shared__ uint32_t path[32];
    __shared__ int depth_n;
    __shared__ int bad;
    const int i = blockIdx.x;
    const int64_t lo = req_off[i], hi = req_off[i + 1];
    if (lo < 0 || hi < lo || hi > nnz) {
        if (threadIdx.x == 0) atomicOr(&h->err, ERR_INVALID);
        return;
    }
    if (threadIdx.x == 0) {
        const uint32_t full = (m == 32) ? 0xffffffffu : ((1u << m) - 1u);
        uint32_t node = full;
        int d = 0;
        int b = 0;
        path[0] = node;
        while (__popc(node) > 1 && d < 31) {
            uint32_t a = split[node];
            uint32_t low = node & (0u - node);
            if ((a & ~node) || a == 0 || a == node || !(a & low)) { b = 1; break; }
            node = ((a >> i) & 1u) ? a : (node ^ a);
            path[++d] = node;
        }
        depth_n = d + 1;
        bad = b;
    }
    __syncthreads();
    if (bad) {
        if (threadIdx.x == 0) atomicOr(&h->err, ERR_INVALID);
        return;
    }
    const int dn = depth_n;
    for (int64_t j = lo + threadIdx.x; j < hi; j += blockDim.x) {
        int32_t x = req_chunks[j];
        uint64_t key = ~0ull;
        if (x < 0 || (int64_t)x >= n_chunks) {
            atomicOr(&h->err, ERR_RANGE);
        } else {
            const uint32_t s = sig[x];
            int d = 0;
            while (d < dn - 1 && (path[d] & ~s)) ++d;
            key = ((uint64_t)i << 37) | ((uint64_t)d << 32) | (uint32_t)x;   // i < 32, d < 32
        }
        keys[j] = key;
    }
}

__global__ void k_fill_u64(uint64_t *p, int64_t from, int64_t to, uint64_t v) {
    for (int64_t i = from + blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < to; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void k_extract_out(int64_t nnz, const uint64_t *keys, int32_t *order_chunks) {
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < nnz; j += (int64_t)gridDim.x * blockDim.x)
        order_chunks[j] = (int32_t)(keys[j] & 0xffffffffu);
}

// ---------------------------------------------------------------------------
// host side


// layer plan of the DP: which kernel and how many segments per subset
struct LayerPlan { int p; uint32_t n_sets; int kind; int seg_bits; int seg_log; uint32_t n_tasks; };
enum { KIND_LANE = 0, KIND_WAVE = 1 };
constexpr uint32_t kTargetWaves = 32768;   // enough waves to fill 256 CUs several times over
// grids of the plain kernels stay within 2^32 work-items; they walk the rest
constexpr uint32_t kMaxGrid = 1u << 20;

LayerPlan plan_layer(int m, int p) {
    LayerPlan L{};
    L.p = p;
    L.n_sets = kBinom.v[m][p];
    if (p <= 6) {
        L.kind = KIND_LANE;
        L.n_tasks = L.n_sets;
        return L;
    }
    L.kind = KIND_WAVE;
    int seg_bits = p - 1;
    while (seg_bits > 6 && ((uint64_t)L.n_sets << (p - 1 - seg_bits)) < kTargetWaves) --seg_bits;
    L.seg_bits = seg_bits;
    L.seg_log = p - 1 - seg_bits;
    L.n_tasks = L.n_sets << L.seg_log;
    return L;
}

size_t dp_partial_entries(int m) {
    size_t mx = 0;
    for (int p = 2; p <= m; ++p) {
        LayerPlan L = plan_layer(m, p);
        if (L.kind == KIND_WAVE && L.seg_log > 0) mx = std::max(mx, (size_t)L.n_tasks);
    }
    return mx;
}

// row-blocked DP: one entry per level h = |S_H| of the high part
// One level of the row-blocked DP: n_sets rows; the first n_sets - tail_rows
// (the head) run their n_pairs cross pairs in `chunks` chunks of per_chunk
// pairs (one chunk: finished in the same kernel), the other tail_rows in
// tail_chunks chunks of tail_per_chunk.
struct RbLevel {
    int h;
    uint32_t n_sets, n_pairs, chunks, per_chunk;
    uint32_t tail_rows, tail_chunks, tail_per_chunk;
};
constexpr int kRbMinM = rb::L + 1;
constexpr int kRbMaxLevels = MPT_MAX_M - rb::L + 1;
constexpr uint32_t kRbMaxChunks = 4096;
struct RbPlan { RbLevel v[kRbMaxLevels]; int n; };

// chunk_pairs = 0: the chunk count of every level from the cost model below.
// chunk_pairs > 0: every level runs its cross pairs in chunks of at most
// chunk_pairs pairs (at most kRbMaxChunks chunks); a level whose pairs fit one
// chunk finishes its rows in the same kernel. Every plan gives the same tables:
// the chunks' keys are folded by exact minima.
RbPlan rb_plan(int m, int64_t chunk_pairs) {
    RbPlan plan{};
    const int m_hi = m - rb::L;
    for (int h = 0; h <= m_hi; ++h) {
        RbLevel L{};
        L.h = h;
        L.n_sets = kBinom.v[m_hi][h];
        L.n_pairs = h >= 2 ? (1u << (h - 1)) - 1u : 0u;
        if (L.n_pairs == 0) {
            L.chunks = 0;
        } else if (chunk_pairs > 0) {
            const int64_t c = ((int64_t)L.n_pairs + chunk_pairs - 1) / chunk_pairs;
            L.chunks = (uint32_t)std::min<int64_t>(c, kRbMaxChunks);
        } else {
            // A fixed number of workgroups runs per CU at a time (their LDS
            // takes the CU), so W equal workgroups take ceil(W / slots)
            // rounds. In units of one row pair's time, a workgroup also pays
            // about one pair of fixed cost (accumulator, flush, partials) and
            // finishing a row about four; a split level finishes its rows in
            // a separate pass. Pick the chunk count c with the least
            // modelled time (ties to fewer chunks).
            const double slots = rb::CUS * rb::WGS_PER_CU;
            constexpr double kWgCost = 1.0, kFinishCost = 4.1;
            auto rounds = [&](double w) { return std::ceil(w / slots); };
            auto cost = [&](uint32_t c) {
                const double per = std::ceil((double)L.n_pairs / c);
                if (c == 1) return rounds(L.n_sets) * (per + kWgCost + kFinishCost);
                return rounds((double)L.n_sets * c) * (per + kWgCost) + rounds(L.n_sets) * (kFinishCost + 0.3);
            };
            uint32_t best = 1;
            double best_cost = cost(1);
            for (uint32_t c = 2; c <= std::min<uint32_t>(L.n_pairs, kRbMaxChunks); ++c) {
                const double e = cost(c);
                if (e < best_cost - 1e-9) { best = c; best_cost = e; }
            }
            L.chunks = best;
            // A tail: the rows whose workgroups would make up the last,
            // partial round run in more, shorter chunks, which the CUs left
            // free in that round (and then all CUs) take after the head's
            // workgroups. Head workgroups take a, tail ones b: the head runs
            // q full rounds and r more workgroups; the free CUs run tail
            // workgroups while those r finish, all CUs the rest. The tail's
            // rows are finished by a separate pass (fused head), and their
            // partials take one more reduce launch.
            constexpr double kLaunch = 1.0;
            const uint32_t rem = (uint32_t)(((uint64_t)L.n_sets * best) % (uint64_t)slots);
            const uint32_t nb = (rem + best - 1) / best;
            if (rem != 0 && nb < L.n_sets && L.n_pairs >= 2) {
                const double a = std::ceil((double)L.n_pairs / best) + kWgCost + (best == 1 ? kFinishCost : 0.0);
                const double head = (double)(L.n_sets - nb) * best;
                const double q = std::floor(head / slots), r = head - q * slots;
                const double finals = best == 1 ? rounds(nb) * (kFinishCost + 0.3) + 2 * kLaunch
                                                : rounds(L.n_sets) * (kFinishCost + 0.3) + kLaunch;
                for (uint32_t c = 2; c <= std::min<uint32_t>(L.n_pairs, 64u); ++c) {
                    const double b = std::ceil((double)L.n_pairs / c) + kWgCost;
                    const double wb = (double)nb * c;
                    double t;
                    if (r == 0) {
                        t = q * a + rounds(wb) * b;
                    } else {
                        const double f = slots - r, k = std::floor(a / b);
                        t = wb <= f * k ? (q + 1) * a : (q + 1) * a + rounds(wb - f * k) * b;
                    }
                    if (t + finals < best_cost - 1e-9) {
                        best_cost = t + finals;
                        L.tail_rows = nb;
                        L.tail_chunks = c;
                    }
                }
            }
        }
        L.per_chunk = L.chunks ? (L.n_pairs + L.chunks - 1) / L.chunks : 0;
        L.tail_per_chunk = L.tail_chunks ? (L.n_pairs + L.tail_chunks - 1) / L.tail_chunks : 0;
        plan.v[plan.n++] = L;
    }
    return plan;
}

size_t rb_partial_entries(int m, int64_t chunk_pairs) {
    if (m < kRbMinM) return 0;
    size_t mx = 0;
    const RbPlan plan = rb_plan(m, chunk_pairs);
    for (int i = 0; i < plan.n; ++i) {
        const RbLevel &L = plan.v[i];
        const size_t head = L.chunks > 1 ? (size_t)(L.n_sets - L.tail_rows) * L.chunks : 0;
        mx = std::max(mx, (head + (size_t)L.tail_rows * L.tail_chunks) * rb::ROW);
    }
    return mx;
}

struct WsLayout {
    size_t list_sig, list_w, part_v, part_a, keys, rb_part, rb_tagged, rb_plain, rb_wrow, rb_srow;
    size_t compact_count, compact_zero, compact_off;
    size_t build_end, extract_end;   // bytes the build and the extraction use
    size_t total;                    // bytes every phase fits in
};

// keys sorted by the extraction: a power of two, at least one sort tile
inline size_t extract_keys(int64_t nnz) {
    size_t n = (size_t)mptlib::kSortTile;
    while (n < (size_t)nnz) n <<= 1;
    return n;
}

WsLayout ws_layout(int m, int64_t nnz, int64_t chunk_pairs) {
    WsLayout L{};
    const size_t nz = (size_t)std::max<int64_t>(nnz, 1);
    const size_t P = std::max<size_t>(dp_partial_entries(m), 1);
    size_t off = sizeof(WsHeader);
    // build-phase list, DP partials and extraction keys are never live at
    // the same time, so they share the region after the header
    L.list_sig = off;
    L.list_w = off + align256(nz * 4);
    size_t build_end = L.list_w + align256(nz * 8);
    // the compaction's per-block counts, unrequested weights and offsets
    L.compact_count = build_end;
    L.compact_zero = L.compact_count + align256((size_t)kCompactMaxBlocks * 4);
    L.compact_off = L.compact_zero + align256((size_t)kCompactMaxBlocks * 8);
    build_end = L.compact_off + align256((size_t)kCompactMaxBlocks * 4);
    L.part_v = off;
    L.part_a = off + align256(P * 8);
    size_t dp_end = L.part_a + align256(P * 4);
    L.keys = off;
    size_t ex_end = L.keys + align256(extract_keys(nnz) * 8);
    L.rb_part = off;
    size_t rb_end = L.rb_part + align256(rb_partial_entries(m, chunk_pairs) * 8);
    if (m >= kRbMinM) {
        // the packed DP's tagged and plain tables, W and split in row order
        L.rb_tagged = rb_end;
        rb_end += align256((size_t)8 << m);
        L.rb_plain = rb_end;
        rb_end += align256((size_t)8 << m);
        L.rb_wrow = rb_end;
        rb_end += align256((size_t)8 << m);
        L.rb_srow = rb_end;
        rb_end += align256((size_t)4 << m);
    }
    L.build_end = build_end;
    L.extract_end = ex_end;
    L.total = std::max(std::max(build_end, rb_end), std::max(dp_end, ex_end));
    return L;
}

// need: the bytes the calling phase uses (at most mpt_workspace_bytes)
int check_ws(void *ws, size_t bytes, size_t need) {
    if (!ws) return fail(MPT_E_WORKSPACE, "workspace is NULL");
    if (((uintptr_t)ws & 255u) != 0) return fail(MPT_E_WORKSPACE, "workspace is not 256-byte aligned");
    if (bytes < need) return fail(MPT_E_WORKSPACE, "workspace has %zu bytes, needs %zu", bytes, need);
    return MPT_OK;
}

// the first fields of the header, as the host reads them back
struct HeaderHead { uint32_t err; uint32_t n_list; int64_t zero_weight; int64_t total; };
static_assert(offsetof(WsHeader, total) == offsetof(HeaderHead, total), "header prefix");

int read_errors(WsHeader *h, hipStream_t s, int64_t *total = nullptr) {
    HeaderHead hh{};
    MPT_HIP_TRY(hipMemcpyAsync(&hh, h, sizeof hh, hipMemcpyDeviceToHost, s));
    MPT_HIP_TRY(hipStreamSynchronize(s));
    const uint32_t err = hh.err;
    if (err & ERR_INVALID) return fail(MPT_E_INVALID, "req_off is not a CSR offset array of length m+1 ending at nnz, or split is not a hierarchy");
    if (err & ERR_RANGE) return fail(MPT_E_RANGE, "a chunk id is outside [0, n_chunks)");
    if (err & ERR_DUP) return fail(MPT_E_DUP, "a chunk is repeated inside one request");
    if (err & ERR_WEIGHT) return fail(MPT_E_WEIGHT, "a chunk weight is <= 0 or > 2^32");
    if (err & ERR_OVERFLOW) return fail(MPT_E_OVERFLOW, "sum of request weights reaches 2^61");
    if (total) *total = hh.total;
    return MPT_OK;
}

int check_common(int m, int64_t n_chunks, int64_t nnz) {
    if (m < 1 || m > MPT_MAX_M) return fail(MPT_E_INVALID, "m = %d outside [1, %d]", m, MPT_MAX_M);
    if (n_chunks < 0 || n_chunks > MPT_MAX_CHUNKS) return fail(MPT_E_INVALID, "n_chunks = %lld out of range", (long long)n_chunks);
    if (nnz < 0 || nnz > (int64_t)INT32_MAX) return fail(MPT_E_INVALID, "nnz = %lld out of range", (long long)nnz);
    return MPT_OK;
}

template <class K, bool NARROW>
int solve_rb(int m, const int64_t *W, int64_t *C, uint32_t *split, char *ws, const WsLayout &Lw,
             int64_t chunk_pairs, hipStream_t s) {
    // NARROW: the two narrow tables take the wide tagged table's space
    uint64_t *Tt = NARROW ? nullptr : (uint64_t *)(ws + Lw.rb_tagged);
    uint32_t *Tn = NARROW ? (uint32_t *)(ws + Lw.rb_tagged) : nullptr;
    uint32_t *Pn = NARROW ? Tn + ((size_t)1 << m) : nullptr;
    uint64_t *Pt = (uint64_t *)(ws + Lw.rb_plain);
    // profiling label of the cross-pair launches: names the key width
    const char *kCrossLabel = NARROW ? "rb_cross_u32" : (std::is_same<K, double>::value ? "rb_cross_f64" : "rb_cross_u64");
    int64_t *Wr = (int64_t *)(ws + Lw.rb_wrow);
    uint32_t *Sr = (uint32_t *)(ws + Lw.rb_srow);
    uint64_t *partial = (uint64_t *)(ws + Lw.rb_part);
    const int H = m - rb::L;
    const uint32_t R = 1u << H;
    const int64_t n = (int64_t)1 << m;
    double pair_work = 1.0;
    for (int i = 0; i < rb::L; ++i) pair_work *= 3.0;        // ordered (A_L, S_L) pairs of one row pair
    // the caller's W, C and split need not be 16-byte aligned: 16-byte
    // accesses only where they are
    auto aligned16 = [](const void *p) { return ((uintptr_t)p & 15u) == 0; };
    {
        // W in mask order is a 2^L x 2^H matrix (S_L, S_H); rows need it transposed
        LaunchScope ls("rb_wrows", 16.0 * n, s);
        const dim3 grid((R + 63) / 64, rb::ROW / 64);
        if (aligned16(W))
            rb::k_transpose<int64_t, 2><<<grid, 256, 0, s>>>(W, Wr, (uint32_t)rb::ROW, R);
        else
            rb::k_transpose<int64_t, 1><<<grid, 256, 0, s>>>(W, Wr, (uint32_t)rb::ROW, R);
    }
    {
        LaunchScope ls("rb_row0", pair_work / 2, s);
        rb::k_rb_row0<K, NARROW><<<1, rb::THREADS, 0, s>>>(m, Wr, Pt, Pn, Sr);
    }
    const RbPlan plan = rb_plan(m, chunk_pairs);
    for (int li = 0; li < plan.n; ++li) {
        const RbLevel &P = plan.v[li];
        if (P.h == 0) continue;                               // row 0: done above
        // narrow finishing of rows first .. first + rows - 1: a whole CU per
        // row when the rows fit one per CU, else two rows per CU
        auto final_narrow = [&](uint32_t rows, uint32_t first, uint32_t head, uint32_t chunks, uint32_t tail_chunks,
                                uint32_t tail_base) {
            if (rows <= (uint32_t)rb::CUS)
                rb::k_rb_final_narrow<K, rb::THREADS><<<rows, rb::THREADS, 0, s>>>(
                    m, P.h, first, head, chunks, tail_chunks, tail_base, Wr, Pt, Tn, Pn, Sr, partial);
            else
                rb::k_rb_final_narrow<K, rb::FINAL_THREADS><<<rows, rb::FINAL_THREADS, 0, s>>>(
                    m, P.h, first, head, chunks, tail_chunks, tail_base, Wr, Pt, Tn, Pn, Sr, partial);
        };
        if (P.n_pairs == 0) {
            LaunchScope ls("rb_final", pair_work * P.n_sets, s);
            if constexpr (NARROW)
                final_narrow(P.n_sets, 0u, P.n_sets, 0u, 0u, 0u);
            else
                rb::k_rb_final<K><<<P.n_sets, rb::THREADS, 0, s>>>(m, P.h, 0u, P.n_sets, 0u, 0u, 0u, Wr, Tt, Pt, Sr,
                                                                   partial);
        } else {
            const uint32_t head = P.n_sets - P.tail_rows;
            const uint32_t head_wgs = head * P.chunks, tail_wgs = P.tail_rows * P.tail_chunks;
            const bool fused = P.chunks == 1;
            const uint32_t tail_base = fused ? 0u : head_wgs;
            {
                // work: the row pairs, and a fused row's self pair
                LaunchScope ls(kCrossLabel, pair_work * ((double)P.n_sets * P.n_pairs + (fused ? head : 0u)), s);
                rb::k_rb_cross<K, NARROW><<<head_wgs + tail_wgs, rb::THREADS, 0, s>>>(
                    m, P.h, P.n_pairs, P.chunks, P.per_chunk, fused ? 1 : 0, head, P.tail_chunks, P.tail_per_chunk,
                    tail_base, Wr, Tt, Pt, Tn, Pn, Sr, partial);
            }
            auto reduce = [&](uint32_t rows, uint32_t chunks, uint64_t *part) {
                LaunchScope ls("rb_reduce", (double)rows * chunks * rb::ROW * 8.0, s);
                const uint32_t groups = (chunks - 1 + rb::RED_CHUNKS_PER_BLOCK - 1) / rb::RED_CHUNKS_PER_BLOCK;
                rb::k_rb_reduce<<<rows * (rb::ROW / 256) * groups, 256, 0, s>>>(chunks, groups, part);
            };
            // (up to kFoldChunks chunks are folded by the finishing kernel)
            if (!fused && P.chunks > rb::kFoldChunks) reduce(head, P.chunks, partial);
            if (P.tail_rows && P.tail_chunks > rb::kFoldChunks)
                reduce(P.tail_rows, P.tail_chunks, partial + (size_t)tail_base * rb::ROW);
            if (!fused || P.tail_rows) {
                const uint32_t first = fused ? head : 0u;
                LaunchScope ls("rb_final", pair_work * (P.n_sets - first), s);
                if constexpr (NARROW)
                    final_narrow(P.n_sets - first, first, head, P.chunks, P.tail_chunks, tail_base);
                else
                    rb::k_rb_final<K><<<P.n_sets - first, rb::THREADS, 0, s>>>(
                        m, P.h, first, head, P.chunks, P.tail_chunks, tail_base, Wr, Tt, Pt, Sr, partial);
            }
        }
        MPT_HIP_TRY(hipGetLastError());
    }
    {
        LaunchScope ls("rb_unpack", 16.0 * n, s);
        const dim3 grid((R + 63) / 64, rb::ROW / 64);
        if (aligned16(C))
            rb::k_rb_unpack<K, true><<<grid, 256, 0, s>>>(m, Pt, C);
        else
            rb::k_rb_unpack<K, false><<<grid, 256, 0, s>>>(m, Pt, C);
    }
    {
        LaunchScope ls("rb_split", 8.0 * n, s);
        // 16-byte accesses need R (2^(m-12) rows) to be a multiple of 4
        if (R >= 4 && aligned16(split))
            rb::k_transpose<uint32_t, 4><<<dim3(rb::ROW / 64, (R + 63) / 64), 256, 0, s>>>(Sr, split, R,
                                                                                       (uint32_t)rb::ROW);
        else
            rb::k_transpose<uint32_t, 1><<<dim3(rb::ROW / 64, (R + 63) / 64), 256, 0, s>>>(Sr, split, R,
                                                                                       (uint32_t)rb::ROW);
    }
    MPT_HIP_TRY(hipGetLastError());
    return MPT_OK;
}

}  // namespace

// ===========================================================================
// Phases behind the C ABI. The exported calls below and the context layer
// (ctx.hip) validate their arguments and call these.

namespace mptcore {

size_t workspace_bytes(int m, int64_t nnz, int64_t chunk_pairs) {
    if (m < 1 || m > MPT_MAX_M || nnz < 0) return 0;
    return ws_layout(m, nnz, chunk_pairs).total;
}

int build(int m, int64_t n_chunks, int64_t nnz, const int64_t *chunk_w, const int64_t *req_off,
          const int32_t *req_chunks, uint32_t *sig, int64_t *W, void *workspace, size_t workspace_bytes,
          hipStream_t s, int64_t *total, int route) {
    mptlib::Range range("mpt build_weights");
    int rc = check_common(m, n_chunks, nnz);
    if (rc) return rc;
    if (!req_off || !W) return fail(MPT_E_INVALID, "req_off and W must not be NULL");
    if ((uintptr_t)W & 15u) return fail(MPT_E_INVALID, "W must be 16-byte aligned");
    if (n_chunks > 0 && (!chunk_w || !sig)) return fail(MPT_E_INVALID, "chunk_w and sig must not be NULL");
    if (nnz > 0 && !req_chunks) return fail(MPT_E_INVALID, "req_chunks must not be NULL");
    const WsLayout L = ws_layout(m, nnz, 0);
    if ((rc = check_ws(workspace, workspace_bytes, L.build_end))) return rc;
    char *ws = (char *)workspace;
    WsHeader *h = (WsHeader *)ws;
    uint32_t *list_sig = (uint32_t *)(ws + L.list_sig);
    int64_t *list_w = (int64_t *)(ws + L.list_w);

    k_header_init<<<1, 64, 0, s>>>(h);
    k_check_offsets<<<1, 64, 0, s>>>(m, nnz, req_off, h);
    if (n_chunks > 0) {
        {
            LaunchScope ls("fill_sig", 4.0 * n_chunks, s);
            k_fill_u32<<<grid_for(n_chunks, 256), 256, 0, s>>>(sig, n_chunks, 0u);
        }
        if (nnz > 0) {
            LaunchScope ls("demand_sets", (double)nnz, s);
            k_demand_sets<<<grid_for(nnz, 256), 256, 0, s>>>(m, n_chunks, nnz, req_off, req_chunks, sig, h);
        }
        {
            LaunchScope ls("compact", (double)n_chunks, s);
            const CompactPlan cp = compact_plan(n_chunks);
            uint32_t *bcount = (uint32_t *)(ws + L.compact_count), *boff = (uint32_t *)(ws + L.compact_off);
            int64_t *bzero = (int64_t *)(ws + L.compact_zero);
            k_compact_count<<<cp.blocks, kCompactThreads, 0, s>>>(n_chunks, cp.per, chunk_w, sig, bcount, bzero, h);
            k_compact_scan<<<1, kScanThreads, 0, s>>>(cp.blocks, bcount, bzero, boff, h);
            k_compact_write<<<cp.blocks, kCompactThreads, 0, s>>>(n_chunks, cp.per, std::max<int64_t>(nnz, 1), chunk_w,
                                                                 sig, boff, list_sig, list_w, h);
        }
    }
    const uint32_t tiles = m > kZetaBits ? 1u << (m - kZetaBits) : 1u;
    const bool dense = route == MPT_ROUTE_DENSE || (route == MPT_ROUTE_AUTO && dense_route_pays(m, nnz));
    if (!dense) {
        LaunchScope ls("weights_tile", 8.0 * (double)(1ull << m), s);
        k_weights_tile<<<std::min(tiles, 1024u), kZetaThreads, 0, s>>>(m, (uint32_t)std::max<int64_t>(nnz, 1), tiles,
                                                                      list_sig, list_w, h, W);
    } else {
        // long list: scatter into a zeroed table, then the zeta passes
        const int64_t n = (int64_t)1 << m;
        const uint32_t cap = (uint32_t)std::max<int64_t>(nnz, 1);
        LaunchScope ls("weights_dense", 8.0 * (double)n, s);
        k_dense_zero<<<grid_for(n, 256, 16384), 256, 0, s>>>(n, W);
        k_dense_scatter<<<(uint32_t)std::min<int64_t>((cap + kScatterSlice - 1) / kScatterSlice, 1024),
                          kScatterThreads, 0, s>>>(cap, list_sig, list_w, h, W);
        const int64_t waves = (n + (1 << kLowPassBits) - 1) >> kLowPassBits;
        k_dense_zeta_low<<<(uint32_t)((waves * kWave + kDenseThreads - 1) / kDenseThreads), kDenseThreads, 0, s>>>(n, W);
        if (m > kLowPassBits) {
            const int hb = m - kLowPassBits, passes = (hb + kHighPassMax - 1) / kHighPassMax;
            for (int p = 0, j = kLowPassBits; p < passes; ++p) {
                const int K = hb / passes + (p < hb % passes ? 1 : 0);
                dense_zeta_high(m, j, K, W, s);
                j += K;
            }
        }
    }
    k_check_total<<<1, 64, 0, s>>>(m, W, h);
    MPT_HIP_TRY(hipGetLastError());
    return read_errors(h, s, total);
}

int solve(int m, const int64_t *W, int64_t *C, uint32_t *split, int64_t *opt_cost, void *workspace,
          size_t workspace_bytes, hipStream_t s, int64_t total, int64_t chunk_pairs) {
    mptlib::Range range("mpt solve_exact");
    int rc = check_common(m, 0, 0);
    if (rc) return rc;
    if (!W || !C || !split) return fail(MPT_E_INVALID, "W, C and split must not be NULL");
    if (chunk_pairs < 0) return fail(MPT_E_INVALID, "chunk_pairs = %lld is negative", (long long)chunk_pairs);
    const WsLayout L = ws_layout(m, 0, chunk_pairs);
    if ((rc = check_ws(workspace, workspace_bytes, L.total))) return rc;
    char *ws = (char *)workspace;
    int64_t *part_v = (int64_t *)(ws + L.part_v);
    uint32_t *part_a = (uint32_t *)(ws + L.part_a);
    const int64_t n = (int64_t)1 << m;
    if (m >= kRbMinM) {
        // packed keys need every cost below 2^(62-m): sum_i w(R_i) picks the
        // representation. Unknown (< 0): read it back from W.
        if (total < 0) {
            WsHeader *h = (WsHeader *)ws;
            rb::k_request_total<<<1, 64, 0, s>>>(m, W, h);
            MPT_HIP_TRY(hipMemcpyAsync(&total, &h->total, sizeof total, hipMemcpyDeviceToHost, s));
            MPT_HIP_TRY(hipStreamSynchronize(s));
        }
        // doubles while 2 C' < 2^52 (Key<double>); below 2^62 keys fit uint64
        if (total < ((int64_t)1 << (61 - m))) {
            // narrow cross-pair keys while every C(A) + C(B) stays below 2^20 - 1
            // (then 2 C' < 2^52 too, for any m up to MPT_MAX_M)
            static_assert(rb::kNarrowTotal <= ((int64_t)1 << (51 - MPT_MAX_M)), "narrow keys imply double keys");
            if (total < rb::kNarrowTotal - 1)
                rc = solve_rb<double, true>(m, W, C, split, ws, L, chunk_pairs, s);
            else if (total < ((int64_t)1 << (51 - m)))
                rc = solve_rb<double, false>(m, W, C, split, ws, L, chunk_pairs, s);
            else
                rc = solve_rb<uint64_t, false>(m, W, C, split, ws, L, chunk_pairs, s);
            if (rc) return rc;
            if (opt_cost) {
                MPT_HIP_TRY(hipMemcpyAsync(opt_cost, C + (n - 1), sizeof(int64_t), hipMemcpyDeviceToHost, s));
                MPT_HIP_TRY(hipStreamSynchronize(s));
            }
            return MPT_OK;
        }
    }
    {
        LaunchScope ls("dp_init", 8.0 * n, s);
        k_dp_init<<<grid_for(n, 256, 16384), 256, 0, s>>>(m, W, C, split);
    }
    for (int p = 2; p <= m; ++p) {
        LayerPlan P = plan_layer(m, p);
        const double pairs = (double)P.n_sets * (double)((1ull << (p - 1)) - 1);
        if (P.kind == KIND_LANE) {
            LaunchScope ls("dp_lane", pairs, s);
            k_dp_lane<<<(P.n_sets + 255) / 256, 256, 0, s>>>(m, p, P.n_sets, W, C, split);
        } else {
            {
                LaunchScope ls("dp_wave", pairs, s);
                k_dp_wave<<<std::min((P.n_tasks + 3) / 4, kMaxGrid), 256, 0, s>>>(
                    m, p, P.seg_bits, P.n_tasks, P.seg_log, W, C, split, part_v, part_a);
            }
            if (P.seg_log > 0) {
                LaunchScope ls("dp_reduce", (double)P.n_tasks, s);
                k_dp_reduce<<<std::min((P.n_sets + 3) / 4, kMaxGrid), 256, 0, s>>>(m, p, P.n_sets, P.seg_log, W, C,
                                                                                  split, part_v, part_a);
            }
        }
        MPT_HIP_TRY(hipGetLastError());
    }
    MPT_HIP_TRY(hipGetLastError());
    if (opt_cost) {
        MPT_HIP_TRY(hipMemcpyAsync(opt_cost, C + (n - 1), sizeof(int64_t), hipMemcpyDeviceToHost, s));
        MPT_HIP_TRY(hipStreamSynchronize(s));
    }
    return MPT_OK;
}

int extract(int m, int64_t n_chunks, int64_t nnz, const int64_t *req_off, const int32_t *req_chunks,
            const uint32_t *sig, const uint32_t *split, int32_t *order_chunks, void *workspace,
            size_t workspace_bytes, hipStream_t s, bool validate) {
    mptlib::Range range("mpt extract_orders");
    int rc = check_common(m, n_chunks, nnz);
    if (rc) return rc;
    if (!req_off || !split) return fail(MPT_E_INVALID, "req_off and split must not be NULL");
    if (nnz > 0 && (!req_chunks || !order_chunks || !sig))
        return fail(MPT_E_INVALID, "req_chunks, sig and order_chunks must not be NULL");
    const WsLayout L = ws_layout(m, nnz, 0);
    if ((rc = check_ws(workspace, workspace_bytes, L.extract_end))) return rc;
    char *ws = (char *)workspace;
    WsHeader *h = (WsHeader *)ws;
    if (validate) {
        k_header_init<<<1, 64, 0, s>>>(h);
        k_check_offsets<<<1, 64, 0, s>>>(m, nnz, req_off, h);
    }
    {
        LaunchScope ls("extract", (double)nnz, s);
        uint64_t *keys = (uint64_t *)(ws + L.keys);
        const int64_t nk = (int64_t)extract_keys(nnz);
        k_fill_u64<<<grid_for(nk - nnz, 256), 256, 0, s>>>(keys, nnz, nk, ~0ull);
        k_extract<<<m, 256, 0, s>>>(m, n_chunks, nnz, req_off, req_chunks, sig, split, keys, h);
        MPT_HIP_TRY(hipGetLastError());
        // offsets and the hierarchy are checked before the sort (inputs that
        // the library produced itself need no check)
        if (validate && (rc = read_errors(h, s))) return rc;
        if (nnz > 0) {
            if ((rc = mptlib::sort_keys(keys, nk, s))) return rc;
            k_extract_out<<<grid_for(nnz, 256), 256, 0, s>>>(nnz, keys, order_chunks);
        }
    }
    MPT_HIP_TRY(hipGetLastError());
    return MPT_OK;
}

}  // namespace mptcore

// ===========================================================================
// C ABI

extern "C" size_t mpt_workspace_bytes(int m, int64_t nnz) {
    try {
        return mptcore::workspace_bytes(m, nnz, 0);
    } catch (...) {
        return 0;
    }
}

extern "C" const char *mpt_status_string(int status) {
    switch (status) {
        case MPT_OK: return "ok";
        case MPT_E_INVALID: return "invalid argument";
        case MPT_E_RANGE: return "chunk id out of range";
        case MPT_E_DUP: return "chunk repeated inside a request";
        case MPT_E_WEIGHT: return "chunk weight out of range";
        case MPT_E_OVERFLOW: return "costs would overflow int64";
        case MPT_E_WORKSPACE: return "workspace too small or misaligned";
        case MPT_E_STATE: return "call out of order for the context's state";
        case MPT_E_DEVICE: return "HIP runtime error";
        case MPT_E_INTERNAL: return "internal error";
        default: return "unknown status";
    }
}

extern "C" const char *mpt_last_error(void) { return mptlib::error_text(); }

extern "C" int mpt_build_weights(int m, int64_t n_chunks, int64_t nnz, const int64_t *chunk_w,
                                 const int64_t *req_off, const int32_t *req_chunks, uint32_t *sig,
                                 int64_t *W, void *workspace, size_t workspace_bytes, void *stream) {
    mptlib::clear_error();
    return mptlib::guarded(__func__, [&]() -> int {
        return mptcore::build(m, n_chunks, nnz, chunk_w, req_off, req_chunks, sig, W, workspace, workspace_bytes,
                              (hipStream_t)stream, nullptr, MPT_ROUTE_AUTO);
    });
}

extern "C" int mpt_solve_exact(int m, const int64_t *W, int64_t *C, uint32_t *split, int64_t *opt_cost,
                               void *workspace, size_t workspace_bytes, void *stream) {
    mptlib::clear_error();
    return mptlib::guarded(__func__, [&]() -> int {
        return mptcore::solve(m, W, C, split, opt_cost, workspace, workspace_bytes, (hipStream_t)stream, -1, 0);
    });
}

extern "C" int mpt_extract_orders(int m, int64_t n_chunks, int64_t nnz, const int64_t *req_off,
                                  const int32_t *req_chunks, const uint32_t *sig, const uint32_t *split,
                                  int32_t *order_chunks, void *workspace, size_t workspace_bytes, void *stream) {
    mptlib::clear_error();
    return mptlib::guarded(__func__, [&]() -> int {
        return mptcore::extract(m, n_chunks, nnz, req_off, req_chunks, sig, split, order_chunks, workspace,
                                workspace_bytes, (hipStream_t)stream, true);
    });
}

// ---------------------------------------------------------------------------
// The solve without a caller workspace: its scratch is a file-scope device
// array of MPT_NOALLOC_SCRATCH_BYTES, one per device the library runs on,
// held until the process ends. Host code never passes the array's name to a
// kernel: on each device, the first call looks up the array's device address
// with hipGetSymbolAddress (that device current) and keeps it.

static __device__ __align__(256) unsigned char scratch[MPT_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

int scratch_address(void **out) {
    int dev = -1;
    MPT_HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return fail(MPT_E_DEVICE, "device %d outside [0, %d)", dev, kMaxDevices);
    std::lock_guard<std::mutex> g(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        MPT_HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p || ((uintptr_t)p & 255u)) return fail(MPT_E_DEVICE, "scratch array has no aligned device address");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return MPT_OK;
}

}  // namespace

extern "C" int mpt_solve_exact_noalloc(int m, const int64_t *W, int64_t *C, uint32_t *split, int64_t *opt_cost,
                                       void *stream) {
    mptlib::clear_error();
    return mptlib::guarded(__func__, [&]() -> int {
        if (m < 1 || m > MPT_NOALLOC_MAX_M)
            return fail(MPT_E_INVALID, "m = %d outside [1, %d] (MPT_NOALLOC_MAX_M)", m, MPT_NOALLOC_MAX_M);
        const size_t need = mptcore::workspace_bytes(m, 0, 0);
        if (need == 0 || need > sizeof(scratch))
            return fail(MPT_E_INTERNAL, "m = %d needs %zu bytes of scratch, the array holds %zu", m, need,
                        sizeof(scratch));
        void *ws = nullptr;
        int rc = scratch_address(&ws);
        if (rc) return rc;
        return mptcore::solve(m, W, C, split, opt_cost, ws, sizeof(scratch), (hipStream_t)stream, -1, 0);
    });
}

// ---------------------------------------------------------------------------
namespace mptlib {

thread_local std::string t_last_error;

int fail(int status, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    t_last_error = buf;
    return status;
}

void clear_error() { t_last_error.clear(); }
const char *error_text() { return t_last_error.c_str(); }

// --- event profiler ---------------------------------------------------------
struct ProfRecord { std::string name; double work; hipEvent_t a, b; };
struct Profiler {
    std::mutex mu;
    bool on = false;
    std::string prefix;      // record only launches whose label starts with it
    std::vector<ProfRecord> recs;
} g_prof;

LaunchScope::LaunchScope(const char *n, double wk, hipStream_t st) : s_(st), name_(n), work_(wk) {
    std::lock_guard<std::mutex> g(g_prof.mu);
    if (!g_prof.on || std::strncmp(n, g_prof.prefix.c_str(), g_prof.prefix.size()) != 0) return;
    if (hipEventCreate(&a_) != hipSuccess || hipEventCreate(&b_) != hipSuccess) return;
    active_ = hipEventRecord(a_, s_) == hipSuccess;
}

LaunchScope::~LaunchScope() {
    if (!active_) return;
    std::lock_guard<std::mutex> g(g_prof.mu);
    if (hipEventRecord(b_, s_) == hipSuccess) g_prof.recs.push_back({name_, work_, a_, b_});
}

}  // namespace mptlib

using mptlib::g_prof;
using mptlib::ProfRecord;

extern "C" int mpt_profile_begin(void) { return mpt_profile_begin_prefix(""); }

extern "C" int mpt_profile_begin_prefix(const char *prefix) {
    std::lock_guard<std::mutex> g(g_prof.mu);
    for (auto &r : g_prof.recs) { (void)hipEventDestroy(r.a); (void)hipEventDestroy(r.b); }
    g_prof.recs.clear();
    g_prof.prefix = prefix ? prefix : "";
    g_prof.on = true;
    return MPT_OK;
}

extern "C" int mpt_profile_end(mpt_profile_row *rows, int max_entries) {
    std::vector<ProfRecord> recs;
    {
        std::lock_guard<std::mutex> g(g_prof.mu);
        g_prof.on = false;
        recs.swap(g_prof.recs);
    }
    std::vector<mpt_profile_row> agg;
    int status = MPT_OK;
    for (auto &r : recs) {
        float ms = 0.f;
        if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess)
            status = fail(MPT_E_DEVICE, "profiling event failed");
        (void)hipEventDestroy(r.a);
        (void)hipEventDestroy(r.b);
        auto it = std::find_if(agg.begin(), agg.end(), [&](const mpt_profile_row &x) { return r.name == x.kernel; });
        if (it == agg.end()) {
            mpt_profile_row row{};
            snprintf(row.kernel, sizeof row.kernel, "%s", r.name.c_str());
            agg.push_back(row);
            it = agg.end() - 1;
        }
        it->launches += 1;
        it->total_ms += ms;
        it->work += r.work;
    }
    if (status != MPT_OK) return status;
    for (int i = 0; i < (int)agg.size() && i < max_entries; ++i) rows[i] = agg[i];
    return (int)agg.size();
}
