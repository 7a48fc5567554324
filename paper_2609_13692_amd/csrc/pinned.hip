// libmpt.so, Section 7.1 of "Prefix Sharing Is a Sorting Problem": the
// quality-preserving pinned variant. The top-t chunks of every request in
// relevance order (its input order) stay at the end of its sequence, most
// relevant last; the rest (the free part) is laid out by the exact DP or the
// agglomerative greedy. Requests whose free parts are equal sets take one
// free sequence, so that their pinned suffixes can share trie nodes.
//   mpt_pinned_split     the distinct free sets (sorted, numbered by their
//                        first request) and each request's set index
//   mpt_pinned_assemble  free sequence of the request's set ++ pinned suffix
// Between the two, the caller lays out the distinct sets with the exact or
// greedy entry points.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "bitonic.h"
#include "common.h"
#include "mpt.h"
#include "seqsort.h"

namespace {

using mptlib::align256;
using mptlib::fail;
using mptlib::grid_for;
using mptlib::kSeqSortTile;
using mptlib::kSortTile;
using mptlib::LaunchScope;
using mptlib::sort_keys;
using mptlib::sort_requests;

constexpr int kWave = 64;

enum : uint32_t { PERR_INVALID = 1u, PERR_RANGE = 2u };

struct PHeader {
    uint32_t err;
    int32_t n_distinct;
    int64_t pad[31];
};
static_assert(sizeof(PHeader) == 256, "header is one 256-byte block");

inline int64_t pow2_at_least(int64_t n) {
    int64_t p = 1;
    while (p < n) p <<= 1;
    return p;
}

struct PLayout {
    size_t keys, rf_off, rf_chunks, ord, gstart, lead, rep, roff, total;
    int64_t kpad, mpad;
};

PLayout p_layout(int m, int64_t nnz) {
    PLayout L{};
    const size_t mm = (size_t)m, nz = (size_t)std::max<int64_t>(nnz, 1);
    L.kpad = std::max<int64_t>(pow2_at_least(std::max<int64_t>(nnz, 1)), kSortTile);
    L.mpad = std::max<int64_t>(pow2_at_least(m), kSeqSortTile);
    size_t o = align256(sizeof(PHeader));
    auto take = [&](size_t bytes) { size_t at = o; o = align256(o + std::max<size_t>(bytes, 1)); return at; };
    L.keys = take(8 * (size_t)L.kpad);
    L.rf_off = take(8 * (mm + 1));
    L.rf_chunks = take(4 * nz);
    L.ord = take(4 * (size_t)L.mpad);
    L.gstart = take(4 * mm);
    L.lead = take(4 * mm);
    L.rep = take(8 * (mm + 1));
    L.roff = take(8 * (mm + 1));
    L.total = o;
    return L;
}

__global__ void k_p_header(PHeader *h) {
    if (threadIdx.x == 0) { h->err = 0; h->n_distinct = 0; }
}

__global__ void k_p_check(int m, int64_t n_chunks, int64_t nnz, const int64_t *off, const int32_t *chunks, PHeader *h) {
    bool ok = true;
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < m; i += gridDim.x * blockDim.x)
        ok = ok && off[i] <= off[i + 1];
    if (blockIdx.x == 0 && threadIdx.x == 0) ok = ok && off[0] == 0 && off[m] == nnz;
    if (!ok) atomicOr(&h->err, PERR_INVALID);
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < nnz; j += (int64_t)gridDim.x * blockDim.x)
        if (chunks[j] < 0 || (int64_t)chunks[j] >= n_chunks) atomicOr(&h->err, PERR_RANGE);
}

// free-part length of every request (into cnt[i + 1], for the scan)
__global__ void k_p_counts(int m, int t, const int64_t *off, int64_t *cnt) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < m; i += gridDim.x * blockDim.x) {
        const int64_t len = off[i + 1] - off[i];
        cnt[i + 1] = len - std::min<int64_t>(t, len);
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) cnt[0] = 0;
}

// in-place inclusive scan of a[1 .. n] (one workgroup of 1024)
__global__ __launch_bounds__(1024) void k_p_scan(int n, int64_t *a) {
    __shared__ int64_t sw[16];
    __shared__ int64_t carry;
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (int b0 = 1; b0 <= n; b0 += blockDim.x) {
        const int i = b0 + threadIdx.x;
        int64_t x = i <= n ? a[i] : 0;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const int64_t y = __shfl_up(x, o, kWave);
            if (lane >= o) x += y;
        }
        if (lane == kWave - 1) sw[wid] = x;
        __syncthreads();
        int64_t before = carry;
        for (int k = 0; k < wid; ++k) before += sw[k];
        if (i <= n) a[i] = before + x;
        __syncthreads();
        if (threadIdx.x == blockDim.x - 1) carry = before + x;
        __syncthreads();
    }
}

// in-place inclusive max-scan of a[0 .. n) (one workgroup of 1024)
__global__ __launch_bounds__(1024) void k_p_max_scan(int n, int32_t *a) {
    __shared__ int32_t sw[16];
    __shared__ int32_t carry;
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    if (threadIdx.x == 0) carry = -1;
    __syncthreads();
    for (int b0 = 0; b0 < n; b0 += blockDim.x) {
        const int i = b0 + threadIdx.x;
        int32_t x = i < n ? a[i] : -1;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const int32_t y = __shfl_up(x, o, kWave);
            if (lane >= o) x = max(x, y);
        }
        if (lane == kWave - 1) sw[wid] = x;
        __syncthreads();
        int32_t before = carry;
        for (int k = 0; k < wid; ++k) before = max(before, sw[k]);
        if (i < n) a[i] = max(before, x);
        __syncthreads();
        if (threadIdx.x == blockDim.x - 1) carry = max(before, x);
        __syncthreads();
    }
}

// (request, chunk) keys of the free slots; pinned slots are padding
__global__ void k_p_keys(int m, int t, int64_t nnz, int64_t npad, const int64_t *off, const int32_t *chunks,
                         uint64_t *keys) {
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < npad; j += (int64_t)gridDim.x * blockDim.x) {
        if (j >= nnz) { keys[j] = ~0ull; continue; }
        int lo = 0, hi = m - 1;                 // request of slot j
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (off[mid] <= j) lo = mid; else hi = mid - 1;
        }
        keys[j] = (j - off[lo] >= t) ? (((uint64_t)lo << 32) | (uint32_t)chunks[j]) : ~0ull;
    }
}

__global__ void k_p_free_chunks(int m, const int64_t *rf_off, const uint64_t *keys, int32_t *rf_chunks) {
    const int64_t n = rf_off[m];
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x)
        rf_chunks[e] = (int32_t)(keys[e] & 0xffffffffu);
}

// sorted position s starts a group of equal free sets (the first member is
// the smallest request of the group: equal sequences sort by index)
__global__ void k_p_group_starts(int m, const int32_t *ord, const int64_t *rf_off, const int32_t *rf_chunks,
                                 int32_t *gstart) {
    for (int s = blockIdx.x * blockDim.x + threadIdx.x; s < m; s += gridDim.x * blockDim.x) {
        bool fresh = s == 0;
        if (!fresh) {
            const int a = ord[s - 1], b = ord[s];
            const int64_t la = rf_off[a + 1] - rf_off[a], lb = rf_off[b + 1] - rf_off[b];
            fresh = la != lb;
            for (int64_t j = 0; j < la && !fresh; ++j) fresh = rf_chunks[rf_off[a] + j] != rf_chunks[rf_off[b] + j];
        }
        gstart[s] = fresh ? s : -1;
    }
}

// leader of every request; representatives (leaders of themselves) and
// their free lengths, indexed by request, for the scans
__global__ void k_p_leaders(int m, const int32_t *ord, const int32_t *gstart, const int64_t *rf_off, int32_t *lead,
                            int64_t *rep, int64_t *roff) {
    for (int s = blockIdx.x * blockDim.x + threadIdx.x; s < m; s += gridDim.x * blockDim.x) {
        const int i = ord[s];
        const int l = ord[gstart[s]];
        lead[i] = l;
        const bool is_rep = l == i;
        rep[i + 1] = is_rep ? 1 : 0;
        roff[i + 1] = is_rep ? rf_off[i + 1] - rf_off[i] : 0;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) { rep[0] = 0; roff[0] = 0; }
}

// distinct sets in order of their representative: offsets, chunks, and the
// set index of every request
__global__ void k_p_distinct(int m, const int32_t *lead, const int64_t *rep, const int64_t *roff,
                             const int64_t *rf_off, const int32_t *rf_chunks, int32_t *dmap, int64_t *free_off,
                             int32_t *free_chunks, PHeader *h) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < m; i += gridDim.x * blockDim.x) {
        dmap[i] = (int32_t)rep[lead[i]];
        if (lead[i] == i) {
            const int64_t d = rep[i], at = roff[i], len = rf_off[i + 1] - rf_off[i];
            free_off[d] = at;
            for (int64_t j = 0; j < len; ++j) free_chunks[at + j] = rf_chunks[rf_off[i] + j];
        }
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        free_off[rep[m]] = roff[m];
        h->n_distinct = (int32_t)rep[m];
    }
}

// free sequence of the request's set, then the pinned suffix (most relevant last)
__global__ void k_p_assemble(int m, int t, int n_distinct, const int64_t *off, const int32_t *chunks,
                             const int32_t *dmap, const int64_t *free_off, const int32_t *free_layout, int32_t *seqs,
                             PHeader *h) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < m; i += gridDim.x * blockDim.x) {
        const int d = dmap[i];
        if (d < 0 || d >= n_distinct) { atomicOr(&h->err, PERR_INVALID); continue; }
        const int64_t len = off[i + 1] - off[i], tp = std::min<int64_t>(t, len);
        const int64_t f = free_off[d + 1] - free_off[d];
        if (f != len - tp || free_off[d] < 0) { atomicOr(&h->err, PERR_INVALID); continue; }
        int32_t *dst = seqs + off[i];
        for (int64_t q = 0; q < f; ++q) dst[q] = free_layout[free_off[d] + q];
        for (int64_t q = 0; q < tp; ++q) dst[f + q] = chunks[off[i] + tp - 1 - q];
    }
}

int p_check_ws(const PLayout &L, void *ws, size_t bytes) {
    if (!ws) return fail(MPT_E_WORKSPACE, "workspace is NULL");
    if (((uintptr_t)ws & 255u) != 0) return fail(MPT_E_WORKSPACE, "workspace is not 256-byte aligned");
    if (bytes < L.total) return fail(MPT_E_WORKSPACE, "workspace has %zu bytes, needs %zu", bytes, L.total);
    return MPT_OK;
}

int p_read(PHeader *h, hipStream_t s, int *n_distinct) {
    PHeader hh;
    MPT_HIP_TRY(hipMemcpyAsync(&hh, h, sizeof hh, hipMemcpyDeviceToHost, s));
    MPT_HIP_TRY(hipStreamSynchronize(s));
    if (hh.err & PERR_INVALID) return fail(MPT_E_INVALID, "offsets are not CSR, or the set map does not match the free layout");
    if (hh.err & PERR_RANGE) return fail(MPT_E_RANGE, "a chunk id is outside [0, n_chunks)");
    if (n_distinct) *n_distinct = hh.n_distinct;
    return MPT_OK;
}

}  // namespace

extern "C" size_t mpt_pinned_workspace_bytes(int m, int64_t nnz) {
    if (m < 1 || m > MPT_LAYOUT_MAX_M || nnz < 0) return 0;
    return p_layout(m, nnz).total;
}

extern "C" int mpt_pinned_split(int m, int64_t n_chunks, int64_t nnz, const int64_t *req_off,
                                const int32_t *req_chunks, int t, int32_t *dmap, int64_t *free_off,
                                int32_t *free_chunks, int *n_distinct, void *workspace, size_t workspace_bytes,
                                void *stream) {
    mptlib::clear_error();
    if (m < 1 || m > MPT_LAYOUT_MAX_M) return fail(MPT_E_INVALID, "m = %d outside [1, %d]", m, MPT_LAYOUT_MAX_M);
    if (n_chunks < 0 || n_chunks > MPT_MAX_CHUNKS || nnz < 0 || nnz > (int64_t)INT32_MAX)
        return fail(MPT_E_INVALID, "n_chunks or nnz out of range");
    if (t < 0) return fail(MPT_E_INVALID, "t = %d is negative", t);
    if (!req_off || !dmap || !free_off || !n_distinct || (nnz > 0 && (!req_chunks || !free_chunks)))
        return fail(MPT_E_INVALID, "req_off, req_chunks, dmap, free_off, free_chunks and n_distinct must not be NULL");
    const PLayout L = p_layout(m, nnz);
    int rc = p_check_ws(L, workspace, workspace_bytes);
    if (rc) return rc;
    hipStream_t s = (hipStream_t)stream;
    char *ws = (char *)workspace;
    PHeader *h = (PHeader *)ws;
    k_p_header<<<1, 64, 0, s>>>(h);
    k_p_check<<<grid_for(std::max<int64_t>(nnz, m), 256), 256, 0, s>>>(m, n_chunks, nnz, req_off, req_chunks, h);
    MPT_HIP_TRY(hipGetLastError());
    if ((rc = p_read(h, s, nullptr))) return rc;
    uint64_t *keys = (uint64_t *)(ws + L.keys);
    int64_t *rf_off = (int64_t *)(ws + L.rf_off), *rep = (int64_t *)(ws + L.rep), *roff = (int64_t *)(ws + L.roff);
    int32_t *rf_chunks = (int32_t *)(ws + L.rf_chunks), *ord = (int32_t *)(ws + L.ord);
    int32_t *gstart = (int32_t *)(ws + L.gstart), *lead = (int32_t *)(ws + L.lead);
    {
        LaunchScope ls("p_split", (double)nnz, s);
        k_p_counts<<<grid_for(m, 256), 256, 0, s>>>(m, t, req_off, rf_off);
        k_p_scan<<<1, 1024, 0, s>>>(m, rf_off);
        k_p_keys<<<grid_for(L.kpad, 256), 256, 0, s>>>(m, t, nnz, L.kpad, req_off, req_chunks, keys);
        if ((rc = sort_keys(keys, L.kpad, s))) return rc;
        k_p_free_chunks<<<grid_for(std::max<int64_t>(nnz, 1), 256), 256, 0, s>>>(m, rf_off, keys, rf_chunks);
        // (gstart, written after the sort, is its scratch)
        if ((rc = sort_requests(ord, gstart, m, L.mpad, rf_off, rf_chunks, s))) return rc;
        k_p_group_starts<<<grid_for(m, 256), 256, 0, s>>>(m, ord, rf_off, rf_chunks, gstart);
        k_p_max_scan<<<1, 1024, 0, s>>>(m, gstart);
        k_p_leaders<<<grid_for(m, 256), 256, 0, s>>>(m, ord, gstart, rf_off, lead, rep, roff);
        // exclusive positions: rep[i] = number of representatives before i
        k_p_scan<<<1, 1024, 0, s>>>(m, rep);
        k_p_scan<<<1, 1024, 0, s>>>(m, roff);
        k_p_distinct<<<grid_for(m, 256), 256, 0, s>>>(m, lead, rep, roff, rf_off, rf_chunks, dmap, free_off,
                                                      free_chunks, h);
    }
    MPT_HIP_TRY(hipGetLastError());
    return p_read(h, s, n_distinct);
}

extern "C" int mpt_pinned_assemble(int m, int64_t nnz, const int64_t *req_off, const int32_t *req_chunks, int t,
                                   const int32_t *dmap, int n_distinct, const int64_t *free_off,
                                   const int32_t *free_layout, int32_t *seqs, void *workspace,
                                   size_t workspace_bytes, void *stream) {
    mptlib::clear_error();
    if (m < 1 || m > MPT_LAYOUT_MAX_M) return fail(MPT_E_INVALID, "m = %d outside [1, %d]", m, MPT_LAYOUT_MAX_M);
    if (nnz < 0 || t < 0 || n_distinct < 1 || n_distinct > m) return fail(MPT_E_INVALID, "nnz, t or n_distinct out of range");
    if (!req_off || !dmap || !free_off || (nnz > 0 && (!req_chunks || !seqs || !free_layout)))
        return fail(MPT_E_INVALID, "array arguments must not be NULL");
    if (!workspace || ((uintptr_t)workspace & 255u) || workspace_bytes < sizeof(PHeader))
        return fail(MPT_E_WORKSPACE, "workspace missing, misaligned or smaller than 256 bytes");
    hipStream_t s = (hipStream_t)stream;
    PHeader *h = (PHeader *)workspace;
    k_p_header<<<1, 64, 0, s>>>(h);
    {
        LaunchScope ls("p_assemble", (double)nnz, s);
        k_p_assemble<<<grid_for(m, 256), 256, 0, s>>>(m, t, n_distinct, req_off, req_chunks, dmap, free_off,
                                                      free_layout, seqs, h);
    }
    MPT_HIP_TRY(hipGetLastError());
    return p_read(h, s, nullptr);
}
