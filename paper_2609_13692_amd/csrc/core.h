// The three phases of the exact solver (mpt.hip), shared by the exported
// stateless calls and the context layer (ctx.hip). Arguments as in
// include/mpt.h; all arrays are device memory.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace mptcore {

// Workspace bytes of the three phases; chunk_pairs as for solve() (0 = the
// library's level plan). 0 for sizes out of range.
size_t workspace_bytes(int m, int64_t nnz, int64_t chunk_pairs);

// W table and demand sets; *total (nullable) receives sum_i w(R_i). route:
// MPT_ROUTE_AUTO, MPT_ROUTE_LIST or MPT_ROUTE_DENSE.
int build(int m, int64_t n_chunks, int64_t nnz, const int64_t *chunk_w, const int64_t *req_off,
          const int32_t *req_chunks, uint32_t *sig, int64_t *W, void *workspace, size_t workspace_bytes,
          hipStream_t s, int64_t *total, int route);

// The Section 3.1 DP. total: sum_i w(R_i) of the instance that W belongs to,
// or < 0 to read it back from W (one stream synchronisation). chunk_pairs > 0
// overrides the level plan (cross pairs in chunks of at most that many pairs).
int solve(int m, const int64_t *W, int64_t *C, uint32_t *split, int64_t *opt_cost, void *workspace,
          size_t workspace_bytes, hipStream_t s, int64_t total, int64_t chunk_pairs);

// Orders read off the hierarchy. validate = false skips the offset and
// hierarchy checks (and their synchronisation) for inputs the library made.
int extract(int m, int64_t n_chunks, int64_t nnz, const int64_t *req_off, const int32_t *req_chunks,
            const uint32_t *sig, const uint32_t *split, int32_t *order_chunks, void *workspace,
            size_t workspace_bytes, hipStream_t s, bool validate);

}  // namespace mptcore
