// Lexicographic sort of requests by their chunk sequences (a CSR of
// sequences: off[m+1], seqs[off[m]]): a bitonic sort of request indices with
// a comparator that reads the sequences; a proper prefix sorts first, equal
// sequences by request index. Tiles of kSeqSortTile indices are sorted in
// LDS, with the first kSeqLdsDepth chunks and the length of every request of
// the tile staged there, so that a comparison reads global memory only when
// two sequences agree on all the staged chunks. Shared by the library's
// source files.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "common.h"

namespace mptlib {

constexpr int kSeqSortTile = 1024;            // requests sorted in LDS per workgroup
constexpr int kSeqLdsDepth = 8;               // leading chunks of each request staged in LDS
constexpr int kSeqLdsStride = kSeqLdsDepth + 1;   // padded row: rows of nearby slots in distinct banks

// a < b: sequence order, a proper prefix first, equal sequences by index;
// index -1 is padding and sorts last
__device__ inline bool seq_less(int a, int b, const int64_t *off, const int32_t *seqs) {
    if (b < 0) return a >= 0;
    if (a < 0) return false;
    const int64_t la = off[a + 1] - off[a], lb = off[b + 1] - off[b];
    const int32_t *sa = seqs + off[a], *sb = seqs + off[b];
    const int64_t n = la < lb ? la : lb;
    for (int64_t j = 0; j < n; ++j)
        if (sa[j] != sb[j]) return sa[j] < sb[j];
    if (la != lb) return la < lb;
    return a < b;
}

// the same order from chunk kSeqLdsDepth on (the first kSeqLdsDepth chunks
// are equal and both sequences are longer)
__device__ inline bool seq_less_tail(int a, int b, const int64_t *off, const int32_t *seqs) {
    const int64_t la = off[a + 1] - off[a], lb = off[b + 1] - off[b];
    const int32_t *sa = seqs + off[a], *sb = seqs + off[b];
    const int64_t n = la < lb ? la : lb;
    for (int64_t j = kSeqLdsDepth; j < n; ++j)
        if (sa[j] != sb[j]) return sa[j] < sb[j];
    if (la != lb) return la < lb;
    return a < b;
}

// a tile's requests in LDS: ids (-1: padding), lengths, leading chunks
struct SeqTile {
    int32_t id[kSeqSortTile];
    int64_t len[kSeqSortTile];
    int32_t c[kSeqSortTile * kSeqLdsStride];
    int32_t t[kSeqSortTile];                  // the tile's order, as slots of the arrays above
};

__device__ inline void seq_tile_load(SeqTile &T, const int32_t *ord, int64_t base, const int64_t *off,
                                     const int32_t *seqs) {
    for (int e = threadIdx.x; e < kSeqSortTile; e += blockDim.x) {
        const int a = ord[base + e];
        T.id[e] = a;
        T.t[e] = e;
        int64_t la = 0;
        if (a >= 0) la = off[a + 1] - off[a];
        T.len[e] = la;
        const int32_t *sa = a >= 0 ? seqs + off[a] : nullptr;
#pragma unroll
        for (int j = 0; j < kSeqLdsDepth; ++j) T.c[e * kSeqLdsStride + j] = j < la ? sa[j] : 0;
    }
}

// seq_less on two slots of the tile
__device__ inline bool seq_less_slot(const SeqTile &T, int x, int y, const int64_t *off, const int32_t *seqs) {
    const int a = T.id[x], b = T.id[y];
    if (b < 0) return a >= 0;
    if (a < 0) return false;
    const int64_t la = T.len[x], lb = T.len[y];
    const int64_t n = la < lb ? la : lb;
    const int64_t nl = n < kSeqLdsDepth ? n : kSeqLdsDepth;
    for (int64_t j = 0; j < nl; ++j) {
        const int32_t u = T.c[x * kSeqLdsStride + j], v = T.c[y * kSeqLdsStride + j];
        if (u != v) return u < v;
    }
    if (n > kSeqLdsDepth) return seq_less_tail(a, b, off, seqs);
    if (la != lb) return la < lb;
    return a < b;
}

static __global__ void k_l_ord_init(int m, int64_t mpad, int32_t *ord) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < mpad; i += (int64_t)gridDim.x * blockDim.x)
        ord[i] = i < m ? (int32_t)i : -1;
}

// all stages with k <= kSeqSortTile inside one tile of request indices
static __global__ __launch_bounds__(256) void k_l_seq_sort_tile(int32_t *ord, const int64_t *off, const int32_t *seqs) {
    __shared__ SeqTile T;
    const int64_t base = (int64_t)blockIdx.x * kSeqSortTile;
    seq_tile_load(T, ord, base, off, seqs);
    __syncthreads();
    for (int k = 2; k <= kSeqSortTile; k <<= 1)
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int p = threadIdx.x; p < kSeqSortTile / 2; p += blockDim.x) {
                const int i = ((p & ~(j - 1)) << 1) | (p & (j - 1)), l = i + j;    // j: a power of two
                const bool up = ((base + i) & k) == 0;
                const int x = T.t[i], y = T.t[l];
                if (seq_less_slot(T, y, x, off, seqs) == up) { T.t[i] = y; T.t[l] = x; }
            }
            __syncthreads();
        }
    for (int e = threadIdx.x; e < kSeqSortTile; e += blockDim.x) ord[base + e] = T.id[T.t[e]];
}

static __global__ void k_l_seq_sort_global(int32_t *ord, int64_t n, int64_t k, int64_t j, const int64_t *off,
                                    const int32_t *seqs) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n / 2; p += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = ((p & ~(j - 1)) << 1) | (p & (j - 1)), l = i + j;    // j: a power of two
        const bool up = (i & k) == 0;
        const int a = ord[i], b = ord[l];
        if (seq_less(b, a, off, seqs) == up) { ord[i] = b; ord[l] = a; }
    }
}

static __global__ __launch_bounds__(256) void k_l_seq_sort_tile_merge(int32_t *ord, int64_t k, const int64_t *off,
                                                               const int32_t *seqs) {
    __shared__ SeqTile T;
    const int64_t base = (int64_t)blockIdx.x * kSeqSortTile;
    seq_tile_load(T, ord, base, off, seqs);
    __syncthreads();
    const bool up = (base & k) == 0;
    for (int j = kSeqSortTile >> 1; j > 0; j >>= 1) {
        for (int p = threadIdx.x; p < kSeqSortTile / 2; p += blockDim.x) {
            const int i = ((p & ~(j - 1)) << 1) | (p & (j - 1)), l = i + j;    // j: a power of two
            const int x = T.t[i], y = T.t[l];
            if (seq_less_slot(T, y, x, off, seqs) == up) { T.t[i] = y; T.t[l] = x; }
        }
        __syncthreads();
    }
    for (int e = threadIdx.x; e < kSeqSortTile; e += blockDim.x) ord[base + e] = T.id[T.t[e]];
}

// Up to kSeqRankMax requests the order comes from ranks instead: the
// position of request i is the number of requests before it in seq_less
// order (a strict total order, so the ranks are a permutation), counted
// over all pairs. Workgroup (x, y) takes 256 requests i, one per thread,
// against 64 requests j staged in LDS. Every request's first kSeqLdsDepth
// chunks are packed as four 64-bit words of two biased chunks (chunk + 1,
// 0 past the end; chunk ids are validated to lie in [0, n_chunks)), so that
// the word order is the sequence order on those chunks with a proper prefix
// first; sequences equal there are ordered by length, or by index, or, when
// both go on past them, by seq_less_tail. m^2 comparisons with no
// dependent stages: at m = 4096 a few µs, where the bitonic sort's 55
// dependent stages of four workgroups took about 0.13 ms.
constexpr int kSeqRankMax = 16384;
constexpr int kSeqRankTile = 256;         // requests i per workgroup, one per thread
constexpr int kSeqRankTileY = 64;         // requests j per workgroup, staged in LDS
constexpr int kSeqWords = kSeqLdsDepth / 2;
static_assert(kSeqLdsDepth % 2 == 0, "chunks pair up into 64-bit words");

__device__ inline void seq_words(int a, const int64_t *off, const int32_t *seqs, uint64_t (&w)[kSeqWords], int64_t &len) {
    len = off[a + 1] - off[a];
    const int32_t *sa = seqs + off[a];
    uint32_t b[kSeqLdsDepth];
#pragma unroll
    for (int j = 0; j < kSeqLdsDepth; ++j) b[j] = j < len ? (uint32_t)sa[j] + 1u : 0u;
#pragma unroll
    for (int q = 0; q < kSeqWords; ++q) w[q] = ((uint64_t)b[2 * q] << 32) | b[2 * q + 1];
}

static __global__ void k_l_rank_zero(int m, int32_t *rank) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < m; i += gridDim.x * blockDim.x) rank[i] = 0;
}

// (the j side's words of one request are adjacent in LDS: every thread
// reads the same j, so two 16-byte broadcast reads)
static __global__ __launch_bounds__(kSeqRankTile) void k_l_seq_rank(int m, const int64_t *off, const int32_t *seqs,
                                                                    int32_t *rank) {
    __shared__ uint64_t yw[kSeqRankTileY][kSeqWords];
    __shared__ int64_t ylen[kSeqRankTileY];
    const int j0 = blockIdx.y * kSeqRankTileY;
    const int ny = min(kSeqRankTileY, m - j0);
    if ((int)threadIdx.x < ny) {
        uint64_t w[kSeqWords];
        int64_t len;
        seq_words(j0 + (int)threadIdx.x, off, seqs, w, len);
#pragma unroll
        for (int q = 0; q < kSeqWords; ++q) yw[threadIdx.x][q] = w[q];
        ylen[threadIdx.x] = len;
    }
    const int i = blockIdx.x * kSeqRankTile + (int)threadIdx.x;
    uint64_t xw[kSeqWords] = {};
    int64_t xlen = 0;
    if (i < m) seq_words(i, off, seqs, xw, xlen);
    __syncthreads();
    if (i >= m) return;
    int count = 0;
#pragma unroll 8
    for (int jj = 0; jj < ny; ++jj) {
        bool lt = false, eq = true;
#pragma unroll
        for (int q = 0; q < kSeqWords; ++q) {
            const uint64_t a = yw[jj][q];
            lt = lt || (eq && a < xw[q]);
            eq = eq && a == xw[q];
        }
        if (eq) {
            const int j = j0 + jj;
            const int64_t la = ylen[jj];
            if (la > kSeqLdsDepth && xlen > kSeqLdsDepth) lt = seq_less_tail(j, i, off, seqs);
            else lt = la < xlen || (la == xlen && j < i);
        }
        count += lt ? 1 : 0;
    }
    if (count) atomicAdd(&rank[i], count);
}

// ord[rank[i]] = i, then -1 up to n
static __global__ void k_l_rank_scatter(int m, int64_t n, const int32_t *rank, int32_t *ord) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n; p += (int64_t)gridDim.x * blockDim.x) {
        if (p < m) ord[rank[p]] = (int32_t)p;
        else ord[p] = -1;
    }
}

// ord[0 .. n) gets the request ids 0 .. m-1 in order, then -1 (padding);
// n is a power of two, at least kSeqSortTile; rank (m entries) is scratch
// (on return, m <= kSeqRankMax: the position of each request)
inline int sort_requests(int32_t *ord, int32_t *rank, int m, int64_t n, const int64_t *off, const int32_t *seqs,
                         hipStream_t s) {
    if (m <= kSeqRankMax) {
        const unsigned tx = (unsigned)((m + kSeqRankTile - 1) / kSeqRankTile);
        const unsigned ty = (unsigned)((m + kSeqRankTileY - 1) / kSeqRankTileY);
        k_l_rank_zero<<<grid_for(m, 256), 256, 0, s>>>(m, rank);
        k_l_seq_rank<<<dim3(tx, ty), kSeqRankTile, 0, s>>>(m, off, seqs, rank);
        k_l_rank_scatter<<<grid_for(n, 256), 256, 0, s>>>(m, n, rank, ord);
        MPT_HIP_TRY(hipGetLastError());
        return MPT_OK;
    }
    const int tiles = (int)(n / kSeqSortTile);
    k_l_ord_init<<<grid_for(n, 256), 256, 0, s>>>(m, n, ord);
    k_l_seq_sort_tile<<<tiles, 256, 0, s>>>(ord, off, seqs);
    for (int64_t k = 2 * kSeqSortTile; k <= n; k <<= 1) {
        for (int64_t j = k >> 1; j >= kSeqSortTile; j >>= 1)
            k_l_seq_sort_global<<<grid_for(n / 2, 256, 16384), 256, 0, s>>>(ord, n, k, j, off, seqs);
        k_l_seq_sort_tile_merge<<<tiles, 256, 0, s>>>(ord, k, off, seqs);
    }
    MPT_HIP_TRY(hipGetLastError());
    return MPT_OK;
}

}  // namespace mptlib
