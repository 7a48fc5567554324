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
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "mpt.h"

namespace {

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
    int64_t pad[30];
};
static_assert(sizeof(WsHeader) == 256, "header is one 256-byte block");

inline size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

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
    if (threadIdx.x == 0) { h->err = 0; h->n_list = 0; h->zero_weight = 0; }
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
// (S_x, w(x)) list; the others only reach W(empty) and are summed apart.
__global__ void k_compact(int64_t n_chunks, int64_t cap, const int64_t *w, const uint32_t *sig,
                          uint32_t *list_sig, int64_t *list_w, WsHeader *h) {
    for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < n_chunks; x += (int64_t)gridDim.x * blockDim.x) {
        int64_t wx = w[x];
        if (wx <= 0 || wx > MPT_MAX_CHUNK_WEIGHT) { atomicOr(&h->err, ERR_WEIGHT); continue; }
        uint32_t s = sig[x];
        if (s == 0) {
            atomicAdd((unsigned long long *)&h->zero_weight, (unsigned long long)wx);
        } else {
            uint32_t idx = atomicAdd(&h->n_list, 1u);
            if ((int64_t)idx < cap) { list_sig[idx] = s; list_w[idx] = wx; }
            else atomicOr(&h->err, ERR_INVALID);
        }
    }
}

// W table, one workgroup per tile of 2^b consecutive subsets that share the
// high bits H = tile id. A chunk reaches W(H|L) iff H|L is inside S_x, i.e.
// iff S_x's high part contains H and its low part contains L. So the tile
// keeps f(L) = sum of w(x) over chunks whose high part contains H and whose
// low part equals L, and a superset-sum (zeta) over the b low bits turns f
// into W. The zeta over the high bits is thereby done on the sparse list,
// and the dense table is written exactly once.
constexpr int kZetaBits = 13;             // 2^13 int64 = 64 KiB of LDS per tile
constexpr int kZetaThreads = 512;

__global__ __launch_bounds__(kZetaThreads) void k_weights_tile(
        int m, int b, uint32_t cap, const uint32_t *list_sig, const int64_t *list_w, const WsHeader *h,
        int64_t *W) {
    __shared__ int64_t tile[1 << kZetaBits];
    const int n = 1 << b;
    const uint32_t hi = blockIdx.x;                 // high part H of every subset in this tile
    const uint32_t lowmask = (uint32_t)n - 1u;
    for (int e = threadIdx.x; e < n; e += blockDim.x) tile[e] = 0;
    __syncthreads();
    const uint32_t cnt = min(h->n_list, cap);
    for (uint32_t j = threadIdx.x; j < cnt; j += blockDim.x) {
        uint32_t s = list_sig[j];
        uint32_t shi = s >> b;
        if ((shi & hi) == hi)
            atomicAdd((unsigned long long *)&tile[s & lowmask], (unsigned long long)list_w[j]);
    }
    if (hi == 0 && threadIdx.x == 0)
        atomicAdd((unsigned long long *)&tile[0], (unsigned long long)h->zero_weight);
    __syncthreads();
    // superset sums over the low bits, three bits per LDS round trip
    for (int j = 0; j < b; j += 3) {
        const int r = min(3, b - j);
        const int g = 1 << r;
        const int ngroups = n >> r;
        for (int q = threadIdx.x; q < ngroups; q += blockDim.x) {
            // group q: the 2^r elements base + k * 2^j, bits j..j+r-1 of base clear
            const int base = ((q >> j) << (j + r)) | (q & ((1 << j) - 1));
            int64_t v[8];
#pragma unroll
            for (int k = 0; k < 8; ++k)
                if (k < g) v[k] = tile[base + (k << j)];
#pragma unroll
            for (int t = 0; t < 3; ++t) {
                if (t < r) {
#pragma unroll
                    for (int k = 0; k < 8; ++k)
                        if (k < g && !((k >> t) & 1)) v[k] += v[k | (1 << t)];
                }
            }
#pragma unroll
            for (int k = 0; k < 8; ++k)
                if (k < g) tile[base + (k << j)] = v[k];
        }
        __syncthreads();
    }
    int64_t *out = W + ((int64_t)hi << b);
    for (int e = threadIdx.x; e < n; e += blockDim.x) out[e] = tile[e];
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
    const uint32_t task = lb * (blockDim.x / kWave) + wave;
    if (task >= n_tasks) return;
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

// second stage for split layers: one wave per subset
__global__ __launch_bounds__(256) void k_dp_reduce(int m, int p, uint32_t n_sets, int seg_log,
                                                   const int64_t *__restrict__ W, int64_t *__restrict__ C,
                                                   uint32_t *__restrict__ split, const int64_t *__restrict__ part_v,
                                                   const uint32_t *__restrict__ part_a) {
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const uint32_t lane = threadIdx.x % kWave;
    const uint32_t set_rank = blockIdx.x * (blockDim.x / kWave) + wave;
    if (set_rank >= n_sets) return;
    const uint32_t nseg = 1u << seg_log;
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

// ---------------------------------------------------------------------------
// phase 3: one workgroup per request i. Chunk x of R_i is emitted at the
// first node of i's root-to-leaf path that lies inside S_x; inside a node
// chunks go in ascending id. The output slot of x is its rank under the key
// (depth, id); keys are distinct because ids are distinct within R_i.
__global__ __launch_bounds__(256) void k_extract(int m, int64_t n_chunks, int64_t nnz, const int64_t *req_off,
                                                 const int32_t *req_chunks, const uint32_t *sig,
                                                 const uint32_t *split, uint64_t *keys, int32_t *order_chunks,
                                                 WsHeader *h) {
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
            key = ((uint64_t)d << 32) | (uint32_t)x;
        }
        keys[j] = key;
    }
    __syncthreads();
    for (int64_t j = lo + threadIdx.x; j < hi; j += blockDim.x) {
        const uint64_t kj = keys[j];
        int64_t rank = 0;
        for (int64_t t = lo; t < hi; ++t) rank += keys[t] < kj;
        order_chunks[lo + rank] = (int32_t)(kj & 0xffffffffu);
    }
}

// ---------------------------------------------------------------------------
// host side

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

#define HIP_TRY(expr)                                                                      \
    do {                                                                                   \
        hipError_t e_ = (expr);                                                            \
        if (e_ != hipSuccess)                                                              \
            return fail(MPT_E_DEVICE, "%s: %s (%s:%d)", #expr, hipGetErrorString(e_),     \
                        __FILE__, __LINE__);                                               \
    } while (0)

// --- event profiler ---------------------------------------------------------
struct ProfRecord { std::string name; double work; hipEvent_t a, b; };
struct Profiler {
    std::mutex mu;
    bool on = false;
    std::vector<ProfRecord> recs;
} g_prof;

struct LaunchScope {
    hipStream_t s;
    bool active = false;
    hipEvent_t a{}, b{};
    const char *name;
    double work;
    LaunchScope(const char *n, double wk, hipStream_t st) : s(st), name(n), work(wk) {
        std::lock_guard<std::mutex> g(g_prof.mu);
        if (!g_prof.on) return;
        if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) return;
        active = hipEventRecord(a, s) == hipSuccess;
    }
    ~LaunchScope() {
        if (!active) return;
        std::lock_guard<std::mutex> g(g_prof.mu);
        if (hipEventRecord(b, s) == hipSuccess) g_prof.recs.push_back({name, work, a, b});
    }
};

inline int grid_for(int64_t n, int threads, int cap = 8192) {
    int64_t g = (n + threads - 1) / threads;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (int)g;
}

// layer plan of the DP: which kernel and how many segments per subset
struct LayerPlan { int p; uint32_t n_sets; int kind; int seg_bits; int seg_log; uint32_t n_tasks; };
enum { KIND_LANE = 0, KIND_WAVE = 1 };
constexpr uint32_t kTargetWaves = 32768;   // enough waves to fill 256 CUs several times over

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

struct WsLayout {
    size_t list_sig, list_w, part_v, part_a, keys, total;
};

WsLayout ws_layout(int m, int64_t nnz) {
    WsLayout L{};
    const size_t nz = (size_t)std::max<int64_t>(nnz, 1);
    const size_t P = std::max<size_t>(dp_partial_entries(m), 1);
    size_t off = sizeof(WsHeader);
    // build-phase list, DP partials and extraction keys are never live at
    // the same time, so they share the region after the header
    L.list_sig = off;
    L.list_w = off + align256(nz * 4);
    size_t build_end = L.list_w + align256(nz * 8);
    L.part_v = off;
    L.part_a = off + align256(P * 8);
    size_t dp_end = L.part_a + align256(P * 4);
    L.keys = off;
    size_t ex_end = L.keys + align256(nz * 8);
    L.total = std::max(build_end, std::max(dp_end, ex_end));
    return L;
}

int check_ws(int m, int64_t nnz, void *ws, size_t bytes) {
    if (!ws) return fail(MPT_E_WORKSPACE, "workspace is NULL");
    if (((uintptr_t)ws & 255u) != 0) return fail(MPT_E_WORKSPACE, "workspace is not 256-byte aligned");
    size_t need = ws_layout(m, nnz).total;
    if (bytes < need) return fail(MPT_E_WORKSPACE, "workspace has %zu bytes, needs %zu", bytes, need);
    return MPT_OK;
}

int read_errors(WsHeader *h, hipStream_t s) {
    uint32_t err = 0;
    HIP_TRY(hipMemcpyAsync(&err, &h->err, sizeof err, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (err & ERR_INVALID) return fail(MPT_E_INVALID, "req_off is not a CSR offset array of length m+1 ending at nnz, or split is not a hierarchy");
    if (err & ERR_RANGE) return fail(MPT_E_RANGE, "a chunk id is outside [0, n_chunks)");
    if (err & ERR_DUP) return fail(MPT_E_DUP, "a chunk is repeated inside one request");
    if (err & ERR_WEIGHT) return fail(MPT_E_WEIGHT, "a chunk weight is <= 0 or > 2^32");
    if (err & ERR_OVERFLOW) return fail(MPT_E_OVERFLOW, "sum of request weights reaches 2^61");
    return MPT_OK;
}

int check_common(int m, int64_t n_chunks, int64_t nnz) {
    if (m < 1 || m > MPT_MAX_M) return fail(MPT_E_INVALID, "m = %d outside [1, %d]", m, MPT_MAX_M);
    if (n_chunks < 0 || n_chunks > MPT_MAX_CHUNKS) return fail(MPT_E_INVALID, "n_chunks = %lld out of range", (long long)n_chunks);
    if (nnz < 0 || nnz > (int64_t)INT32_MAX) return fail(MPT_E_INVALID, "nnz = %lld out of range", (long long)nnz);
    return MPT_OK;
}

}  // namespace

// ===========================================================================
// C ABI

extern "C" size_t mpt_workspace_bytes(int m, int64_t nnz) {
    if (m < 1 || m > MPT_MAX_M || nnz < 0) return 0;
    return ws_layout(m, nnz).total;
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
        case MPT_E_DEVICE: return "HIP runtime error";
        default: return "unknown status";
    }
}

extern "C" const char *mpt_last_error(void) { return t_last_error.c_str(); }

extern "C" int mpt_build_weights(int m, int64_t n_chunks, int64_t nnz, const int64_t *chunk_w,
                                 const int64_t *req_off, const int32_t *req_chunks, uint32_t *sig,
                                 int64_t *W, void *workspace, size_t workspace_bytes, void *stream) {
    t_last_error.clear();
    int rc = check_common(m, n_chunks, nnz);
    if (rc) return rc;
    if (!req_off || !W) return fail(MPT_E_INVALID, "req_off and W must not be NULL");
    if (n_chunks > 0 && (!chunk_w || !sig)) return fail(MPT_E_INVALID, "chunk_w and sig must not be NULL");
    if (nnz > 0 && !req_chunks) return fail(MPT_E_INVALID, "req_chunks must not be NULL");
    if ((rc = check_ws(m, nnz, workspace, workspace_bytes))) return rc;
    hipStream_t s = (hipStream_t)stream;
    char *ws = (char *)workspace;
    WsHeader *h = (WsHeader *)ws;
    WsLayout L = ws_layout(m, nnz);
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
            k_compact<<<grid_for(n_chunks, 256), 256, 0, s>>>(n_chunks, std::max<int64_t>(nnz, 1), chunk_w, sig,
                                                              list_sig, list_w, h);
        }
    }
    const int b = std::min(m, kZetaBits);
    {
        LaunchScope ls("weights_tile", 8.0 * (double)(1ull << m), s);
        k_weights_tile<<<1u << (m - b), kZetaThreads, 0, s>>>(m, b, (uint32_t)std::max<int64_t>(nnz, 1), list_sig,
                                                              list_w, h, W);
    }
    k_check_total<<<1, 64, 0, s>>>(m, W, h);
    HIP_TRY(hipGetLastError());
    return read_errors(h, s);
}

extern "C" int mpt_solve_exact(int m, const int64_t *W, int64_t *C, uint32_t *split, int64_t *opt_cost,
                               void *workspace, size_t workspace_bytes, void *stream) {
    t_last_error.clear();
    int rc = check_common(m, 0, 0);
    if (rc) return rc;
    if (!W || !C || !split) return fail(MPT_E_INVALID, "W, C and split must not be NULL");
    if ((rc = check_ws(m, 0, workspace, workspace_bytes))) return rc;
    hipStream_t s = (hipStream_t)stream;
    char *ws = (char *)workspace;
    WsLayout L = ws_layout(m, 0);
    int64_t *part_v = (int64_t *)(ws + L.part_v);
    uint32_t *part_a = (uint32_t *)(ws + L.part_a);
    const int64_t n = (int64_t)1 << m;
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
                k_dp_wave<<<(P.n_tasks + 3) / 4, 256, 0, s>>>(m, p, P.seg_bits, P.n_tasks, P.seg_log, W, C, split,
                                                               part_v, part_a);
            }
            if (P.seg_log > 0) {
                LaunchScope ls("dp_reduce", (double)P.n_tasks, s);
                k_dp_reduce<<<(P.n_sets + 3) / 4, 256, 0, s>>>(m, p, P.n_sets, P.seg_log, W, C, split, part_v,
                                                                 part_a);
            }
        }
        HIP_TRY(hipGetLastError());
    }
    HIP_TRY(hipGetLastError());
    if (opt_cost) {
        HIP_TRY(hipMemcpyAsync(opt_cost, C + (n - 1), sizeof(int64_t), hipMemcpyDeviceToHost, s));
        HIP_TRY(hipStreamSynchronize(s));
    }
    return MPT_OK;
}

extern "C" int mpt_extract_orders(int m, int64_t n_chunks, int64_t nnz, const int64_t *req_off,
                                  const int32_t *req_chunks, const uint32_t *sig, const uint32_t *split,
                                  int32_t *order_chunks, void *workspace, size_t workspace_bytes, void *stream) {
    t_last_error.clear();
    int rc = check_common(m, n_chunks, nnz);
    if (rc) return rc;
    if (!req_off || !split) return fail(MPT_E_INVALID, "req_off and split must not be NULL");
    if (nnz > 0 && (!req_chunks || !order_chunks || !sig))
        return fail(MPT_E_INVALID, "req_chunks, sig and order_chunks must not be NULL");
    if ((rc = check_ws(m, nnz, workspace, workspace_bytes))) return rc;
    hipStream_t s = (hipStream_t)stream;
    char *ws = (char *)workspace;
    WsHeader *h = (WsHeader *)ws;
    WsLayout L = ws_layout(m, nnz);
    k_header_init<<<1, 64, 0, s>>>(h);
    k_check_offsets<<<1, 64, 0, s>>>(m, nnz, req_off, h);
    {
        LaunchScope ls("extract", (double)nnz, s);
        k_extract<<<m, 256, 0, s>>>(m, n_chunks, nnz, req_off, req_chunks, sig, split, (uint64_t *)(ws + L.keys),
                                    order_chunks, h);
    }
    HIP_TRY(hipGetLastError());
    return read_errors(h, s);
}

extern "C" int mpt_profile_begin(void) {
    std::lock_guard<std::mutex> g(g_prof.mu);
    for (auto &r : g_prof.recs) { (void)hipEventDestroy(r.a); (void)hipEventDestroy(r.b); }
    g_prof.recs.clear();
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
