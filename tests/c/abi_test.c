/*
 * abi_test.c -- a C11 program against the C ABI of libmpt.so (include/mpt.h),
 * compiled as C by hipcc and linked against the library: the header must be
 * plain C, and every call is made the way a C caller makes it.
 *
 *   abi_test host          argument checks that need no GPU
 *   abi_test run IN OUT    solves the instance in IN through the context
 *                          layer (and W through the stateless call), checks
 *                          the state machine on the way, writes OUT
 *
 * IN (text): m n_chunks nnz, then n_chunks weights, m + 1 request offsets
 * and nnz chunk ids. OUT (text): OPT_free and the savings, then the W, C and
 * split tables (2^m entries each) and the orders (nnz entries).
 * Exit status 0 when every check passed; the failing check is printed.
 */
#include <hip/hip_runtime_api.h>
#include <inttypes.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "mpt.h"

static int failures = 0;

#define CHECK(cond)                                                              \
    do {                                                                         \
        if (!(cond)) {                                                           \
            fprintf(stderr, "FAIL %s:%d: %s (last error: %s)\n", __FILE__, __LINE__, \
                    #cond, mpt_last_error());                                    \
            ++failures;                                                          \
        }                                                                        \
    } while (0)

static int host_checks(void) {
    static const int codes[] = {MPT_OK, MPT_E_INVALID, MPT_E_RANGE, MPT_E_DUP, MPT_E_WEIGHT, MPT_E_OVERFLOW,
                                MPT_E_WORKSPACE, MPT_E_STATE, MPT_E_DEVICE, MPT_E_INTERNAL};
    for (size_t i = 0; i < sizeof codes / sizeof codes[0]; ++i) {
        const char *t = mpt_status_string(codes[i]);
        CHECK(t != NULL && strcmp(t, "unknown status") != 0);
    }
    CHECK(strcmp(mpt_status_string(-1000), "unknown status") == 0);

    CHECK(mpt_workspace_bytes(0, 0) == 0);
    CHECK(mpt_workspace_bytes(MPT_MAX_M + 1, 0) == 0);
    CHECK(mpt_workspace_bytes(12, -1) == 0);
    size_t ws12 = mpt_workspace_bytes(12, 48);
    CHECK(ws12 >= 256 && ws12 % 256 == 0);
    CHECK(mpt_ctx_workspace_bytes(NULL, 12, 64, 48) >= ((size_t)20 << 12) + ws12);
    CHECK(mpt_ctx_workspace_bytes(NULL, MPT_MAX_M + 1, 64, 48) == 0);

    /* stateless calls reject bad sizes and NULL arrays before any device work */
    void *dummy = (void *)(uintptr_t)4096, *ws = (void *)(uintptr_t)(256 * 16);
    CHECK(mpt_build_weights(0, 1, 0, dummy, dummy, NULL, dummy, dummy, ws, 1u << 20, NULL) == MPT_E_INVALID);
    CHECK(strlen(mpt_last_error()) > 0);
    CHECK(mpt_solve_exact(MPT_MAX_M + 1, dummy, dummy, dummy, NULL, ws, 1u << 20, NULL) == MPT_E_INVALID);
    CHECK(mpt_solve_exact(4, NULL, dummy, dummy, NULL, ws, 1u << 20, NULL) == MPT_E_INVALID);
    CHECK(mpt_solve_exact(4, dummy, dummy, dummy, NULL, NULL, 1u << 20, NULL) == MPT_E_WORKSPACE);
    CHECK(mpt_extract_orders(3, 5, -2, dummy, dummy, dummy, dummy, dummy, ws, 1u << 20, NULL) == MPT_E_INVALID);

    /* the context layer rejects NULL contexts and bad options */
    CHECK(mpt_create(NULL, 0, NULL) == MPT_E_INVALID);
    mpt_destroy(NULL);
    CHECK(mpt_set_option(NULL, MPT_OPT_CHUNK_PAIRS, 1) == MPT_E_INVALID);
    CHECK(mpt_set_workspace(NULL, NULL, 0) == MPT_E_INVALID);
    CHECK(mpt_ctx_build_weights(NULL, 4, 1, 0, dummy, dummy, NULL) == MPT_E_INVALID);
    CHECK(mpt_ctx_solve_exact(NULL, NULL, NULL, NULL) == MPT_E_INVALID);
    CHECK(mpt_ctx_extract_orders(NULL, NULL) == MPT_E_INVALID);
    CHECK(mpt_copy_table(NULL, MPT_TABLE_W, dummy, 8) == MPT_E_INVALID);

    int n_dev = 0;
    if (hipGetDeviceCount(&n_dev) != hipSuccess || n_dev == 0) {
        mpt_ctx *c = (mpt_ctx *)dummy;
        CHECK(mpt_create(&c, 0, NULL) != MPT_OK && c == NULL);
    }
    return failures;
}

typedef struct {
    int m;
    int64_t n_chunks, nnz;
    int64_t *w, *off;
    int32_t *chunks;
} instance;

static int read_instance(const char *path, instance *in) {
    FILE *f = fopen(path, "r");
    if (!f) return -1;
    int ok = fscanf(f, "%d %" SCNd64 " %" SCNd64, &in->m, &in->n_chunks, &in->nnz) == 3;
    in->w = (int64_t *)malloc(sizeof(int64_t) * (size_t)(in->n_chunks + 1));
    in->off = (int64_t *)malloc(sizeof(int64_t) * (size_t)(in->m + 1));
    in->chunks = (int32_t *)malloc(sizeof(int32_t) * (size_t)(in->nnz + 1));
    for (int64_t i = 0; ok && i < in->n_chunks; ++i) ok = fscanf(f, "%" SCNd64, &in->w[i]) == 1;
    for (int i = 0; ok && i <= in->m; ++i) ok = fscanf(f, "%" SCNd64, &in->off[i]) == 1;
    for (int64_t i = 0; ok && i < in->nnz; ++i) ok = fscanf(f, "%" SCNd32, &in->chunks[i]) == 1;
    fclose(f);
    return ok ? 0 : -1;
}

#define HIP_OK(expr)                                                       \
    do {                                                                   \
        hipError_t e_ = (expr);                                            \
        if (e_ != hipSuccess) {                                            \
            fprintf(stderr, "HIP %s: %s\n", #expr, hipGetErrorString(e_)); \
            return 2;                                                      \
        }                                                                  \
    } while (0)

static int run(const char *in_path, const char *out_path) {
    instance in;
    if (read_instance(in_path, &in)) {
        fprintf(stderr, "cannot read %s\n", in_path);
        return 2;
    }
    const int m = in.m;
    const size_t n = (size_t)1 << m;
    fprintf(stderr, "[abi_test] m=%d n_chunks=%" PRId64 " nnz=%" PRId64 "\n", m, in.n_chunks, in.nnz);

    mpt_ctx *ctx = NULL;
    CHECK(mpt_create(&ctx, 0, NULL) == MPT_OK && ctx != NULL);
    if (!ctx) return 1;
    const size_t bytes = mpt_ctx_workspace_bytes(ctx, m, in.n_chunks, in.nnz);
    CHECK(bytes > 0);
    void *ws = NULL;
    HIP_OK(hipMalloc(&ws, bytes));

    /* out of order: no workspace, then no instance, then no solve */
    CHECK(mpt_ctx_build_weights(ctx, m, in.n_chunks, in.nnz, in.w, in.off, in.chunks) == MPT_E_WORKSPACE);
    CHECK(mpt_set_workspace(ctx, ws, bytes) == MPT_OK);
    CHECK(mpt_ctx_solve_exact(ctx, NULL, NULL, NULL) == MPT_E_STATE);
    CHECK(mpt_ctx_build_weights(ctx, m, in.n_chunks, in.nnz, in.w, in.off, in.chunks) == MPT_OK);
    CHECK(mpt_ctx_extract_orders(ctx, NULL) == MPT_E_STATE);

    int64_t opt = -1, sav = -1;
    uint32_t *split_host = (uint32_t *)malloc(4 * n);
    int64_t *W = (int64_t *)malloc(8 * n), *C = (int64_t *)malloc(8 * n);
    uint32_t *split = (uint32_t *)malloc(4 * n);
    int32_t *orders = (int32_t *)malloc(4 * (size_t)(in.nnz + 1));
    CHECK(mpt_ctx_solve_exact(ctx, &opt, &sav, split_host) == MPT_OK);
    int64_t total = 0;
    for (int64_t j = 0; j < in.nnz; ++j) total += in.w[in.chunks[j]];
    CHECK(opt >= 0 && sav == total - opt);
    CHECK(mpt_ctx_extract_orders(ctx, orders) == MPT_OK);
    CHECK(mpt_copy_table(ctx, MPT_TABLE_W, W, 8 * n) == MPT_OK);
    CHECK(mpt_copy_table(ctx, MPT_TABLE_C, C, 8 * n) == MPT_OK);
    CHECK(mpt_copy_table(ctx, MPT_TABLE_SPLIT, split, 4 * n) == MPT_OK);
    CHECK(mpt_copy_table(ctx, MPT_TABLE_SPLIT, split, 4 * n - 1) == MPT_E_INVALID);
    CHECK(memcmp(split, split_host, 4 * n) == 0);
    CHECK(C[n - 1] == opt && C[0] == MPT_COST_SENTINEL);

    /* the stateless build on device copies of the inputs gives the same W */
    int64_t *d_w = NULL, *d_off = NULL, *d_W = NULL;
    int32_t *d_ch = NULL;
    uint32_t *d_sig = NULL;
    void *d_ws = NULL;
    const size_t sws = mpt_workspace_bytes(m, in.nnz);
    HIP_OK(hipMalloc((void **)&d_w, 8 * (size_t)(in.n_chunks + 1)));
    HIP_OK(hipMalloc((void **)&d_off, 8 * (size_t)(m + 1)));
    HIP_OK(hipMalloc((void **)&d_ch, 4 * (size_t)(in.nnz + 1)));
    HIP_OK(hipMalloc((void **)&d_sig, 4 * (size_t)(in.n_chunks + 1)));
    HIP_OK(hipMalloc((void **)&d_W, 8 * n));
    HIP_OK(hipMalloc(&d_ws, sws));
    HIP_OK(hipMemcpy(d_w, in.w, 8 * (size_t)in.n_chunks, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(d_off, in.off, 8 * (size_t)(m + 1), hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(d_ch, in.chunks, 4 * (size_t)in.nnz, hipMemcpyHostToDevice));
    CHECK(mpt_build_weights(m, in.n_chunks, in.nnz, d_w, d_off, d_ch, d_sig, d_W, d_ws, sws, NULL) == MPT_OK);
    int64_t *W2 = (int64_t *)malloc(8 * n);
    HIP_OK(hipMemcpy(W2, d_W, 8 * n, hipMemcpyDeviceToHost));
    CHECK(memcmp(W, W2, 8 * n) == 0);

    FILE *f = fopen(out_path, "w");
    if (!f) return 2;
    fprintf(f, "%" PRId64 " %" PRId64 "\n", opt, sav);
    for (size_t s = 0; s < n; ++s) fprintf(f, "%" PRId64 "\n", W[s]);
    for (size_t s = 0; s < n; ++s) fprintf(f, "%" PRId64 "\n", C[s]);
    for (size_t s = 0; s < n; ++s) fprintf(f, "%" PRIu32 "\n", split[s]);
    for (int64_t j = 0; j < in.nnz; ++j) fprintf(f, "%" PRId32 "\n", orders[j]);
    fclose(f);

    HIP_OK(hipFree(d_w));
    HIP_OK(hipFree(d_off));
    HIP_OK(hipFree(d_ch));
    HIP_OK(hipFree(d_sig));
    HIP_OK(hipFree(d_W));
    HIP_OK(hipFree(d_ws));
    mpt_destroy(ctx);
    HIP_OK(hipFree(ws));
    free(W);
    free(W2);
    free(C);
    free(split);
    free(split_host);
    free(orders);
    free(in.w);
    free(in.off);
    free(in.chunks);
    return failures ? 1 : 0;
}

int main(int argc, char **argv) {
    if (argc == 2 && strcmp(argv[1], "host") == 0) return host_checks() ? 1 : 0;
    if (argc == 4 && strcmp(argv[1], "run") == 0) return run(argv[2], argv[3]);
    fprintf(stderr, "usage: abi_test host | abi_test run IN OUT\n");
    return 2;
}
