// The context layer of libmpt.so (include/mpt.h): one instance on one device,
// the three phases of the exact solver in order (Section 2's problem,
// Theorem 1 and the Section 3.1 recurrence), over one caller-owned workspace
// that holds the copied instance, the W, C and split tables, the demand sets,
// the orders and the phases' own scratch. Host code only; the kernels are
// those of mpt.hip (through core.h).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <new>

#include "common.h"
#include "core.h"
#include "mpt.h"

using mptlib::align256;
using mptlib::fail;

namespace {

enum State { CREATED = 0, BUILT = 1, SOLVED = 2, EXTRACTED = 3 };

// byte offsets of the context's arrays inside its workspace
struct CtxLayout {
    size_t req_off, req_chunks, chunk_w, sig, W, C, split, orders, core, core_bytes, total;
};

CtxLayout ctx_layout(int m, int64_t n_chunks, int64_t nnz, int64_t chunk_pairs) {
    CtxLayout L{};
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off += align256(bytes > 0 ? bytes : 1);
        return at;
    };
    L.req_off = take(8 * (size_t)(m + 1));
    L.req_chunks = take(4 * (size_t)nnz);
    L.chunk_w = take(8 * (size_t)n_chunks);
    L.sig = take(4 * (size_t)n_chunks);
    L.W = take((size_t)8 << m);
    L.C = take((size_t)8 << m);
    L.split = take((size_t)4 << m);
    L.orders = take(4 * (size_t)nnz);
    L.core_bytes = mptcore::workspace_bytes(m, nnz, chunk_pairs);
    L.core = take(L.core_bytes);
    L.total = L.core_bytes ? off : 0;
    return L;
}

bool sizes_ok(int m, int64_t n_chunks, int64_t nnz) {
    return m >= 1 && m <= MPT_MAX_M && n_chunks >= 0 && n_chunks <= MPT_MAX_CHUNKS && nnz >= 0 &&
           nnz <= (int64_t)INT32_MAX;
}

// makes the context's device current for one call, restores the caller's
class DeviceScope {
  public:
    explicit DeviceScope(int dev) {
        ok_ = hipGetDevice(&prev_) == hipSuccess;
        if (ok_ && prev_ != dev) ok_ = hipSetDevice(dev) == hipSuccess;
        if (!ok_) prev_ = -1;
    }
    ~DeviceScope() {
        if (prev_ >= 0) (void)hipSetDevice(prev_);
    }
    bool ok() const { return ok_; }
    DeviceScope(const DeviceScope &) = delete;
    DeviceScope &operator=(const DeviceScope &) = delete;

  private:
    int prev_ = -1;
    bool ok_ = false;
};

}  // namespace

struct mpt_ctx {
    int device = 0;
    hipStream_t stream = nullptr;
    char *ws = nullptr;
    size_t ws_bytes = 0;
    int64_t chunk_pairs = 0;
    int route = MPT_ROUTE_AUTO;
    State state = CREATED;
    int m = 0;
    int64_t n_chunks = 0, nnz = 0, total = 0;
    CtxLayout lay{};

    template <class T>
    T *at(size_t off) const { return reinterpret_cast<T *>(ws + off); }
};

namespace {

int table_info(const mpt_ctx *c, int which, size_t *off, size_t *bytes) {
    const size_t n = (size_t)1 << c->m;
    State need = BUILT;
    switch (which) {
        case MPT_TABLE_W: *off = c->lay.W; *bytes = 8 * n; break;
        case MPT_TABLE_SIG: *off = c->lay.sig; *bytes = 4 * (size_t)c->n_chunks; break;
        case MPT_TABLE_C: *off = c->lay.C; *bytes = 8 * n; need = SOLVED; break;
        case MPT_TABLE_SPLIT: *off = c->lay.split; *bytes = 4 * n; need = SOLVED; break;
        case MPT_TABLE_ORDERS: *off = c->lay.orders; *bytes = 4 * (size_t)c->nnz; need = EXTRACTED; break;
        default: return fail(MPT_E_INVALID, "unknown table %d", which);
    }
    if (c->state < need)
        return fail(MPT_E_STATE, "table %d is written by a phase that has not run since the last build", which);
    return MPT_OK;
}

}  // namespace

extern "C" int mpt_create(mpt_ctx **out, int hip_device, void *hip_stream) {
    mptlib::clear_error();
    return mptlib::guarded(__func__, [&]() -> int {
        if (!out) return fail(MPT_E_INVALID, "out must not be NULL");
        *out = nullptr;
        int n = 0;
        MPT_HIP_TRY(hipGetDeviceCount(&n));
        if (hip_device < 0 || hip_device >= n)
            return fail(MPT_E_INVALID, "hip_device = %d outside [0, %d)", hip_device, n);
        if (hip_stream) {
            hipDevice_t d = -1;
            MPT_HIP_TRY(hipStreamGetDevice((hipStream_t)hip_stream, &d));
            if (d != hip_device) return fail(MPT_E_INVALID, "the stream belongs to device %d, not %d", d, hip_device);
        }
        mpt_ctx *c = new (std::nothrow) mpt_ctx();
        if (!c) return fail(MPT_E_INTERNAL, "out of host memory");
        c->device = hip_device;
        c->stream = (hipStream_t)hip_stream;
        *out = c;
        return MPT_OK;
    });
}

extern "C" void mpt_destroy(mpt_ctx *ctx) { delete ctx; }

extern "C" int mpt_set_option(mpt_ctx *ctx, int option, int64_t value) {
    mptlib::clear_error();
    if (!ctx) return fail(MPT_E_INVALID, "ctx must not be NULL");
    if (option == MPT_OPT_CHUNK_PAIRS) {
        if (value < 0) return fail(MPT_E_INVALID, "MPT_OPT_CHUNK_PAIRS = %lld is negative", (long long)value);
        ctx->chunk_pairs = value;
    } else if (option == MPT_OPT_WEIGHT_ROUTE) {
        if (value != MPT_ROUTE_AUTO && value != MPT_ROUTE_LIST && value != MPT_ROUTE_DENSE)
            return fail(MPT_E_INVALID, "MPT_OPT_WEIGHT_ROUTE = %lld is not a route", (long long)value);
        ctx->route = (int)value;
    } else {
        return fail(MPT_E_INVALID, "unknown option %d", option);
    }
    ctx->state = CREATED;
    return MPT_OK;
}

extern "C" size_t mpt_ctx_workspace_bytes(const mpt_ctx *ctx, int m, int64_t n_chunks, int64_t nnz) {
    try {
        if (!sizes_ok(m, n_chunks, nnz)) return 0;
        return ctx_layout(m, n_chunks, nnz, ctx ? ctx->chunk_pairs : 0).total;
    } catch (...) {
        return 0;
    }
}

extern "C" int mpt_set_workspace(mpt_ctx *ctx, void *dev_ptr, size_t bytes) {
    mptlib::clear_error();
    if (!ctx) return fail(MPT_E_INVALID, "ctx must not be NULL");
    if (dev_ptr && ((uintptr_t)dev_ptr & 255u)) return fail(MPT_E_WORKSPACE, "workspace is not 256-byte aligned");
    ctx->ws = (char *)dev_ptr;
    ctx->ws_bytes = dev_ptr ? bytes : 0;
    ctx->state = CREATED;
    return MPT_OK;
}

extern "C" int mpt_ctx_build_weights(mpt_ctx *ctx, int m, int64_t n_chunks, int64_t nnz, const int64_t *chunk_w,
                                     const int64_t *req_off, const int32_t *req_chunks) {
    mptlib::clear_error();
    if (!ctx) return fail(MPT_E_INVALID, "ctx must not be NULL");
    ctx->state = CREATED;
    return mptlib::guarded(__func__, [&]() -> int {
        if (!sizes_ok(m, n_chunks, nnz))
            return fail(MPT_E_INVALID, "sizes out of range: m = %d, n_chunks = %lld, nnz = %lld", m,
                        (long long)n_chunks, (long long)nnz);
        if (!req_off) return fail(MPT_E_INVALID, "req_off must not be NULL");
        if (n_chunks > 0 && !chunk_w) return fail(MPT_E_INVALID, "chunk_w must not be NULL");
        if (nnz > 0 && !req_chunks) return fail(MPT_E_INVALID, "req_chunks must not be NULL");
        const CtxLayout L = ctx_layout(m, n_chunks, nnz, ctx->chunk_pairs);
        if (!ctx->ws) return fail(MPT_E_WORKSPACE, "no workspace: call mpt_set_workspace first");
        if (ctx->ws_bytes < L.total)
            return fail(MPT_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ctx->ws_bytes, L.total);
        DeviceScope dev(ctx->device);
        if (!dev.ok()) return fail(MPT_E_DEVICE, "cannot make device %d current", ctx->device);
        ctx->lay = L;
        ctx->m = m;
        ctx->n_chunks = n_chunks;
        ctx->nnz = nnz;
        hipStream_t s = ctx->stream;
        MPT_HIP_TRY(hipMemcpyAsync(ctx->at<void>(L.req_off), req_off, 8 * (size_t)(m + 1), hipMemcpyDefault, s));
        if (nnz > 0)
            MPT_HIP_TRY(hipMemcpyAsync(ctx->at<void>(L.req_chunks), req_chunks, 4 * (size_t)nnz, hipMemcpyDefault, s));
        if (n_chunks > 0)
            MPT_HIP_TRY(hipMemcpyAsync(ctx->at<void>(L.chunk_w), chunk_w, 8 * (size_t)n_chunks, hipMemcpyDefault, s));
        int64_t total = 0;
        const int rc = mptcore::build(m, n_chunks, nnz, ctx->at<int64_t>(L.chunk_w), ctx->at<int64_t>(L.req_off),
                                      ctx->at<int32_t>(L.req_chunks), ctx->at<uint32_t>(L.sig), ctx->at<int64_t>(L.W),
                                      ctx->ws + L.core, L.core_bytes, s, &total, ctx->route);
        if (rc) return rc;
        ctx->total = total;
        ctx->state = BUILT;
        return MPT_OK;
    });
}

extern "C" int mpt_ctx_solve_exact(mpt_ctx *ctx, int64_t *opt_cost, int64_t *savings, uint32_t *split_host) {
    mptlib::clear_error();
    if (!ctx) return fail(MPT_E_INVALID, "ctx must not be NULL");
    if (ctx->state < BUILT) return fail(MPT_E_STATE, "mpt_ctx_solve_exact needs a built instance (mpt_ctx_build_weights)");
    return mptlib::guarded(__func__, [&]() -> int {
        DeviceScope dev(ctx->device);
        if (!dev.ok()) return fail(MPT_E_DEVICE, "cannot make device %d current", ctx->device);
        const CtxLayout &L = ctx->lay;
        hipStream_t s = ctx->stream;
        ctx->state = BUILT;
        int64_t opt = 0;
        const bool want_opt = opt_cost || savings;
        int rc = mptcore::solve(ctx->m, ctx->at<int64_t>(L.W), ctx->at<int64_t>(L.C), ctx->at<uint32_t>(L.split),
                                want_opt ? &opt : nullptr, ctx->ws + L.core, L.core_bytes, s, ctx->total,
                                ctx->chunk_pairs);
        if (rc) return rc;
        if (split_host) {
            MPT_HIP_TRY(hipMemcpyAsync(split_host, ctx->at<void>(L.split), (size_t)4 << ctx->m, hipMemcpyDeviceToHost, s));
            MPT_HIP_TRY(hipStreamSynchronize(s));
        }
        if (opt_cost) *opt_cost = opt;
        if (savings) *savings = ctx->total - opt;
        ctx->state = SOLVED;
        return MPT_OK;
    });
}

extern "C" int mpt_ctx_optimum(const mpt_ctx *ctx, int64_t *opt_cost, int64_t *savings) {
    mptlib::clear_error();
    if (!ctx) return fail(MPT_E_INVALID, "ctx must not be NULL");
    if (ctx->state < SOLVED) return fail(MPT_E_STATE, "mpt_ctx_optimum needs a solved instance (mpt_ctx_solve_exact)");
    return mptlib::guarded(__func__, [&]() -> int {
        if (!opt_cost && !savings) return MPT_OK;
        DeviceScope dev(ctx->device);
        if (!dev.ok()) return fail(MPT_E_DEVICE, "cannot make device %d current", ctx->device);
        int64_t opt = 0;
        const int64_t *C = ctx->at<int64_t>(ctx->lay.C);
        MPT_HIP_TRY(hipMemcpyAsync(&opt, C + (((int64_t)1 << ctx->m) - 1), sizeof opt, hipMemcpyDeviceToHost,
                                   ctx->stream));
        MPT_HIP_TRY(hipStreamSynchronize(ctx->stream));
        if (opt_cost) *opt_cost = opt;
        if (savings) *savings = ctx->total - opt;
        return MPT_OK;
    });
}

extern "C" int mpt_ctx_extract_orders(mpt_ctx *ctx, int32_t *order_chunks_host) {
    mptlib::clear_error();
    if (!ctx) return fail(MPT_E_INVALID, "ctx must not be NULL");
    if (ctx->state < SOLVED) return fail(MPT_E_STATE, "mpt_ctx_extract_orders needs a solved instance (mpt_ctx_solve_exact)");
    return mptlib::guarded(__func__, [&]() -> int {
        DeviceScope dev(ctx->device);
        if (!dev.ok()) return fail(MPT_E_DEVICE, "cannot make device %d current", ctx->device);
        const CtxLayout &L = ctx->lay;
        hipStream_t s = ctx->stream;
        ctx->state = SOLVED;
        // offsets and chunk ids were validated by the build, split made by the solve
        int rc = mptcore::extract(ctx->m, ctx->n_chunks, ctx->nnz, ctx->at<int64_t>(L.req_off),
                                  ctx->at<int32_t>(L.req_chunks), ctx->at<uint32_t>(L.sig),
                                  ctx->at<uint32_t>(L.split), ctx->at<int32_t>(L.orders), ctx->ws + L.core,
                                  L.core_bytes, s, false);
        if (rc) return rc;
        if (order_chunks_host && ctx->nnz > 0) {
            MPT_HIP_TRY(hipMemcpyAsync(order_chunks_host, ctx->at<void>(L.orders), 4 * (size_t)ctx->nnz,
                                       hipMemcpyDeviceToHost, s));
            MPT_HIP_TRY(hipStreamSynchronize(s));
        }
        ctx->state = EXTRACTED;
        return MPT_OK;
    });
}

extern "C" int mpt_copy_table(const mpt_ctx *ctx, int which, void *host_dst, size_t bytes) {
    mptlib::clear_error();
    if (!ctx) return fail(MPT_E_INVALID, "ctx must not be NULL");
    return mptlib::guarded(__func__, [&]() -> int {
        size_t off = 0, need = 0;
        int rc = table_info(ctx, which, &off, &need);
        if (rc) return rc;
        if (need == 0) return MPT_OK;
        if (!host_dst) return fail(MPT_E_INVALID, "host_dst must not be NULL");
        if (bytes < need) return fail(MPT_E_INVALID, "table %d has %zu bytes, host_dst only %zu", which, need, bytes);
        DeviceScope dev(ctx->device);
        if (!dev.ok()) return fail(MPT_E_DEVICE, "cannot make device %d current", ctx->device);
        MPT_HIP_TRY(hipMemcpyAsync(host_dst, ctx->ws + off, need, hipMemcpyDeviceToHost, ctx->stream));
        MPT_HIP_TRY(hipStreamSynchronize(ctx->stream));
        return MPT_OK;
    });
}

extern "C" int mpt_table_device(const mpt_ctx *ctx, int which, const void **dev_ptr, size_t *bytes) {
    mptlib::clear_error();
    if (!ctx || !dev_ptr || !bytes) return fail(MPT_E_INVALID, "ctx, dev_ptr and bytes must not be NULL");
    size_t off = 0, need = 0;
    int rc = table_info(ctx, which, &off, &need);
    if (rc) return rc;
    *dev_ptr = ctx->ws + off;
    *bytes = need;
    return MPT_OK;
}
