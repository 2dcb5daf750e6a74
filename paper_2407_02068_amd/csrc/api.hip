// api.hip -- the C ABI of liblpv (include/lpv.h): argument checks, the packed
// weight handle, device memory and kernel dispatch.
//
// Every check runs before the first HIP call, so a rejected call touches no
// device state (and the checks can be exercised on a machine without a GPU).
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <cmath>
#include <new>

#include <mutex>
#include "lpv_internal.h"

namespace {

thread_local char g_err[512];

lpv_status fail(lpv_status s, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return s;
}

lpv_status hip_fail(hipError_t e, const char* what)
{
    return fail(LPV_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

int elem_size(int dt)
{
    switch (dt) {
    case LPV_F32: return 4;
    case LPV_F16: return 2;
    case LPV_BF16: return 2;
    default: return 0;
    }
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

constexpr int64_t MAX_DIM = 65536;  // N and K (schedule tables are sized for it)
// K of the 16-bit kernels: one schedule group's walk (one 16-byte entry per
// 32 reduction columns, padded to an even count) must fit the kernel's 32 KB
// LDS table beside the group's descriptor and 1 KB of bias
constexpr int64_t MAX_K16 = 63424;
// Leading dimensions of X and W: the kernels address a 256-row tile of either
// with 32-bit byte offsets.
constexpr int64_t MAX_LD = (int64_t)1 << 22;
constexpr int64_t MAX_M = (int64_t)1 << 31;

// Device allocations fail on purpose when LPV_FAULT_INJECT=alloc (tests of
// the error path).
bool inject_alloc_failure()
{
    const char* v = getenv("LPV_FAULT_INJECT");
    return v && strcmp(v, "alloc") == 0;
}

hipError_t dmalloc(void** p, size_t bytes)
{
    *p = nullptr;
    if (inject_alloc_failure())
        return hipErrorOutOfMemory;
    if (bytes == 0)
        return hipSuccess;
    return hipMalloc(p, bytes);
}

lpv_status check_block(int32_t b)
{
    return (b == 16 || b == 32 || b == 64) ? LPV_OK : LPV_ERR_BLOCK;
}

// Shared checks of the linear calls: X (M x K, ldx), Y (M x N, ldy), bias.
lpv_status check_linear(int es, int64_t N, int64_t K, const void* X, int64_t ldx, int64_t M,
                        const void* bias, const void* Y, int64_t ldy, int epi)
{
    if (M < 0 || M >= MAX_M)
        return fail(LPV_ERR_SHAPE, "M = %lld is out of range [0, 2^31)", (long long)M);
    if (epi != LPV_EPI_NONE && epi != LPV_EPI_GELU)
        return fail(LPV_ERR_INVALID_ARG, "unknown epilogue %d", epi);
    if (ldx < K)
        return fail(LPV_ERR_INVALID_ARG, "ldx = %lld < K = %lld", (long long)ldx, (long long)K);
    if (ldx > MAX_LD)
        return fail(LPV_ERR_INVALID_ARG, "ldx = %lld is above %lld", (long long)ldx,
                    (long long)MAX_LD);
    if (ldy < N)
        return fail(LPV_ERR_INVALID_ARG, "ldy = %lld < N = %lld", (long long)ldy, (long long)N);
    if ((ldx * es) % 16 || (ldy * es) % 16)
        return fail(LPV_ERR_INVALID_ARG, "ldx and ldy must be multiples of 16 bytes");
    if (M == 0)
        return LPV_OK;
    if (!X || !Y)
        return fail(LPV_ERR_INVALID_ARG, "X and Y must not be NULL when M > 0");
    if (!aligned16(X) || !aligned16(Y) || (bias && !aligned16(bias)))
        return fail(LPV_ERR_INVALID_ARG, "X, Y and bias must be 16-byte aligned");
    const uintptr_t x0 = (uintptr_t)X, x1 = x0 + (uintptr_t)(((M - 1) * ldx + K) * es);
    const uintptr_t y0 = (uintptr_t)Y, y1 = y0 + (uintptr_t)(((M - 1) * ldy + N) * es);
    if (x0 < y1 && y0 < x1)
        return fail(LPV_ERR_ALIAS, "X and Y overlap");
    return LPV_OK;
}

void free_handle(lpv_bsr* h)
{
    if (!h)
        return;
    void* bufs[] = {h->meta, h->col_idx, h->values, h->step_col, h->step_bits, h->step_tile,
                    h->walk, h->stream_vals, h->gradw_ws};
    for (void* p : bufs)
        if (p)
            (void)hipFree(p);
    delete[] h->gdesc_host;
    delete h;
}

}  // namespace

extern "C" {

const char* lpv_status_str(lpv_status s)
{
    switch (s) {
    case LPV_OK: return "LPV_OK";
    case LPV_ERR_INVALID_ARG: return "LPV_ERR_INVALID_ARG";
    case LPV_ERR_SHAPE: return "LPV_ERR_SHAPE";
    case LPV_ERR_DTYPE: return "LPV_ERR_DTYPE";
    case LPV_ERR_BLOCK: return "LPV_ERR_BLOCK";
    case LPV_ERR_ALIAS: return "LPV_ERR_ALIAS";
    case LPV_ERR_ALLOC: return "LPV_ERR_ALLOC";
    case LPV_ERR_HIP: return "LPV_ERR_HIP";
    default: return "LPV_ERR_UNKNOWN";
    }
}

const char* lpv_last_error(void) { return g_err; }

lpv_status lpv_bsr_pack(const void* W, int64_t ldw, int64_t N, int64_t K, lpv_dtype dt,
                        int32_t b_r, int32_t b_c, const uint8_t* mask, void* stream,
                        lpv_bsr** out)
{
    g_err[0] = 0;
    if (!out)
        return fail(LPV_ERR_INVALID_ARG, "out must not be NULL");
    *out = nullptr;
    const int es = elem_size(dt);
    if (!es)
        return fail(LPV_ERR_DTYPE, "unknown element type %d", (int)dt);
    if (check_block(b_r) || check_block(b_c))
        return fail(LPV_ERR_BLOCK, "block %dx%d: each side must be 16, 32 or 64", b_r, b_c);
    if (N <= 0 || K <= 0 || N > MAX_DIM || K > MAX_DIM)
        return fail(LPV_ERR_SHAPE, "weight %lldx%lld: each side must be in [1, %lld]",
                    (long long)N, (long long)K, (long long)MAX_DIM);
    if (N % b_r || K % b_c)
        return fail(LPV_ERR_SHAPE, "block %dx%d does not divide weight %lldx%lld", b_r, b_c,
                    (long long)N, (long long)K);
    if (es == 2 && K > MAX_K16)
        return fail(LPV_ERR_SHAPE, "K = %lld: the 16-bit kernels take K <= %lld", (long long)K,
                    (long long)MAX_K16);
    if (!W || !mask)
        return fail(LPV_ERR_INVALID_ARG, "W and mask must not be NULL");
    if (ldw < K || (ldw * es) % 16 || !aligned16(W))
        return fail(LPV_ERR_INVALID_ARG, "W must be 16-byte aligned with ldw >= K and ldw a "
                                         "multiple of 16 bytes");

    lpv_bsr* h = new (std::nothrow) lpv_bsr();
    if (!h)
        return fail(LPV_ERR_ALLOC, "host allocation failed");
    h->N = N;
    h->K = K;
    h->b_r = b_r;
    h->b_c = b_c;
    h->R = (int32_t)(N / b_r);
    h->C = (int32_t)(K / b_c);
    h->dtype = dt;
    h->n_tile_rows = (int32_t)((N + lpv::TILE - 1) / lpv::TILE);
    h->n_tile_cols = (int32_t)((K + lpv::TILE - 1) / lpv::TILE);
    h->n_groups = (h->n_tile_rows + lpv::GROUP_TILES - 1) / lpv::GROUP_TILES;
    hipStream_t s = (hipStream_t)stream;

    // one buffer for gdesc (16-byte entries first), row_ptr, group_order,
    // step_ptr, group_tile0 and the plan
    const size_t n_meta = 4 * (size_t)h->n_groups + (size_t)(h->R + 1) +
                          3 * (size_t)(h->n_groups + 1) + 4;
    void* meta = nullptr;
    hipError_t e = dmalloc(&meta, n_meta * sizeof(int32_t));
    if (e != hipSuccess) {
        free_handle(h);
        return e == hipErrorOutOfMemory ? fail(LPV_ERR_ALLOC, "device allocation failed")
                                        : hip_fail(e, "hipMalloc");
    }
    h->meta = meta;
    e = hipGetDevice(&h->device);
    if (e != hipSuccess) {
        free_handle(h);
        return hip_fail(e, "hipGetDevice");
    }
    h->gdesc = (int4*)meta;
    h->row_ptr = (int32_t*)(h->gdesc + h->n_groups);
    h->group_order = h->row_ptr + (h->R + 1);
    h->step_ptr = h->group_order + (h->n_groups + 1);
    h->group_tile0 = h->step_ptr + (h->n_groups + 1);
    lpv::Plan* plan_d = (lpv::Plan*)(h->group_tile0 + (h->n_groups + 1));

    lpv::PackArgs a = {};
    a.W = W;
    a.ldw = ldw;
    a.N = N;
    a.K = K;
    a.es = es;
    a.b_r = b_r;
    a.b_c = b_c;
    a.R = h->R;
    a.C = h->C;
    a.mask = mask;
    a.n_tile_rows = h->n_tile_rows;
    a.n_tile_cols = h->n_tile_cols;
    a.n_groups = h->n_groups;

    lpv::Plan plan = {};
    const bool mfma_path = dt != LPV_F32;
    if (mfma_path) {
        h->gdesc_host = new (std::nothrow) int4[h->n_groups];
        if (!h->gdesc_host) {
            free_handle(h);
            return fail(LPV_ERR_ALLOC, "host allocation failed");
        }
    }
    e = lpv::launch_pack_plan(a, h->row_ptr, h->step_ptr, h->group_tile0, h->group_order,
                              h->gdesc, plan_d, s);
    if (e == hipSuccess)
        e = hipMemcpyAsync(&plan, plan_d, sizeof plan, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess && mfma_path)
        e = hipMemcpyAsync(h->gdesc_host, h->gdesc, (size_t)h->n_groups * sizeof(int4),
                           hipMemcpyDeviceToHost, s);
    if (e == hipSuccess)
        e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
        free_handle(h);
        return hip_fail(e, "pack plan");
    }
    h->nnzb = plan.nnzb;
    h->n_steps = mfma_path ? plan.n_steps : 0;
    h->n_tiles = mfma_path ? plan.n_tiles : 0;
    h->n_walk = mfma_path ? plan.n_walk : 0;
    if (h->n_tiles >= ((int64_t)1 << 21)) {
        // the kernels address the tile stream with 32-bit byte offsets
        const long long nt = (long long)h->n_tiles;
        free_handle(h);
        return fail(LPV_ERR_SHAPE, "%lld kept 32 x 32 tiles: at most 2^21 - 1 are supported", nt);
    }

    const size_t blk = (size_t)b_r * b_c * es;
    e = dmalloc((void**)&h->col_idx, (size_t)h->nnzb * sizeof(int32_t));
    if (e == hipSuccess)
        e = dmalloc(&h->values, (size_t)h->nnzb * blk);
    if (e == hipSuccess && mfma_path) {
        e = dmalloc((void**)&h->step_col, (size_t)h->n_steps * sizeof(int32_t));
        if (e == hipSuccess)
            e = dmalloc((void**)&h->step_bits, (size_t)h->n_steps * sizeof(int32_t));
        if (e == hipSuccess)
            e = dmalloc((void**)&h->step_tile, (size_t)h->n_steps * sizeof(int32_t));
        if (e == hipSuccess)
            e = dmalloc((void**)&h->walk, (size_t)h->n_walk * sizeof(int2));
        if (e == hipSuccess)
            e = dmalloc(&h->stream_vals, (size_t)h->n_tiles * lpv::TILE * lpv::TILE * es);
    }
    if (e != hipSuccess) {
        free_handle(h);
        return e == hipErrorOutOfMemory ? fail(LPV_ERR_ALLOC, "device allocation failed")
                                        : hip_fail(e, "hipMalloc");
    }
    e = lpv::launch_pack_fill(a, h, s);
    if (e == hipSuccess)
        e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
        free_handle(h);
        return hip_fail(e, "pack fill");
    }
    *out = h;
    return LPV_OK;
}

lpv_status lpv_bsr_info_get(const lpv_bsr* h, lpv_bsr_info* out)
{
    if (!h || !out)
        return fail(LPV_ERR_INVALID_ARG, "handle and out must not be NULL");
    out->N = h->N;
    out->K = h->K;
    out->b_r = h->b_r;
    out->b_c = h->b_c;
    out->R = h->R;
    out->C = h->C;
    out->nnzb = h->nnzb;
    out->dtype = h->dtype;
    out->device = h->device;
    out->tile_rows = lpv::TILE;
    out->tile_cols = lpv::TILE;
    out->group_tiles = lpv::GROUP_TILES;
    out->n_groups = h->dtype == LPV_F32 ? 0 : h->n_groups;
    out->n_steps = h->n_steps;
    out->n_tiles = h->n_tiles;
    return LPV_OK;
}

lpv_status lpv_bsr_export(const lpv_bsr* h, int32_t* row_ptr, int32_t* col_idx, void* values,
                          void* stream)
{
    if (!h)
        return fail(LPV_ERR_INVALID_ARG, "handle must not be NULL");
    hipStream_t s = (hipStream_t)stream;
    const size_t blk = (size_t)h->b_r * h->b_c * elem_size(h->dtype);
    hipError_t e = hipSuccess;
    if (row_ptr)
        e = hipMemcpyAsync(row_ptr, h->row_ptr, (size_t)(h->R + 1) * sizeof(int32_t),
                           hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess && col_idx && h->nnzb)
        e = hipMemcpyAsync(col_idx, h->col_idx, (size_t)h->nnzb * sizeof(int32_t),
                           hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess && values && h->nnzb)
        e = hipMemcpyAsync(values, h->values, (size_t)h->nnzb * blk, hipMemcpyDeviceToDevice, s);
    return e == hipSuccess ? LPV_OK : hip_fail(e, "export copy");
}

lpv_status lpv_bsr_schedule_export(const lpv_bsr* h, int32_t* group_order, int32_t* step_ptr,
                                   int32_t* step_col, int32_t* step_bits, int32_t* step_tile,
                                   void* stream)
{
    if (!h)
        return fail(LPV_ERR_INVALID_ARG, "handle must not be NULL");
    if (h->dtype == LPV_F32)
        return fail(LPV_ERR_DTYPE, "fp32 handles walk the BSR arrays and carry no tile schedule");
    hipStream_t s = (hipStream_t)stream;
    hipError_t e = hipSuccess;
    const size_t ng = (size_t)h->n_groups, ns = (size_t)h->n_steps;
    struct {
        void* dst;
        const void* src;
        size_t n;
    } cp[] = {{group_order, h->group_order, ng},
              {step_ptr, h->step_ptr, ng + 1},
              {step_col, h->step_col, ns},
              {step_bits, h->step_bits, ns},
              {step_tile, h->step_tile, ns}};
    for (auto& c : cp)
        if (e == hipSuccess && c.dst && c.n)
            e = hipMemcpyAsync(c.dst, c.src, c.n * sizeof(int32_t), hipMemcpyDeviceToDevice, s);
    return e == hipSuccess ? LPV_OK : hip_fail(e, "schedule copy");
}

lpv_status lpv_bsr_unpack(const lpv_bsr* h, void* W_out, int64_t ldw, void* stream)
{
    if (!h)
        return fail(LPV_ERR_INVALID_ARG, "handle must not be NULL");
    const int es = elem_size(h->dtype);
    if (!W_out || ldw < h->K || (ldw * es) % 16 || !aligned16(W_out))
        return fail(LPV_ERR_INVALID_ARG, "W_out must be 16-byte aligned with ldw >= K and ldw a "
                                         "multiple of 16 bytes");
    hipError_t e = lpv::launch_unpack(h, W_out, ldw, (hipStream_t)stream);
    return e == hipSuccess ? LPV_OK : hip_fail(e, "unpack launch");
}

lpv_status lpv_bsr_linear(const lpv_bsr* h, const void* X, int64_t ldx, int64_t M,
                          const void* bias, void* Y, int64_t ldy, lpv_epilogue epi, void* stream)
{
    if (!h)
        return fail(LPV_ERR_INVALID_ARG, "handle must not be NULL");
    lpv_status st = check_linear(elem_size(h->dtype), h->N, h->K, X, ldx, M, bias, Y, ldy, epi);
    if (st != LPV_OK || M == 0)
        return st;
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return hip_fail(e, "hipGetDevice");
    if (dev != h->device)
        return fail(LPV_ERR_INVALID_ARG, "handle lives on device %d, current device is %d",
                    h->device, dev);
    lpv::LinearCall c = {X, ldx, M, bias, Y, ldy, epi == LPV_EPI_GELU};
    e = lpv::launch_bsr_linear(h, c, (hipStream_t)stream);
    return e == hipSuccess ? LPV_OK : hip_fail(e, "bsr_linear launch");
}

lpv_status lpv_dense_linear(const void* W, int64_t ldw, int64_t N, int64_t K, lpv_dtype dt,
                            const void* X, int64_t ldx, int64_t M, const void* bias, void* Y,
                            int64_t ldy, lpv_epilogue epi, void* stream)
{
    const int es = elem_size(dt);
    if (!es)
        return fail(LPV_ERR_DTYPE, "unknown element type %d", (int)dt);
    if (N <= 0 || K <= 0 || N > MAX_DIM || K > MAX_DIM || N % 16 || K % 16)
        return fail(LPV_ERR_SHAPE, "weight %lldx%lld: sides must be multiples of 16 in [16, %lld]",
                    (long long)N, (long long)K, (long long)MAX_DIM);
    if (es == 2 && K > MAX_K16)
        return fail(LPV_ERR_SHAPE, "K = %lld: the 16-bit kernels take K <= %lld", (long long)K,
                    (long long)MAX_K16);
    if (!W || ldw < K || ldw > MAX_LD || (ldw * es) % 16 || !aligned16(W))
        return fail(LPV_ERR_INVALID_ARG, "W must be non-NULL, 16-byte aligned, K <= ldw <= 2^22 "
                                         "and ldw a multiple of 16 bytes");
    lpv_status st = check_linear(es, N, K, X, ldx, M, bias, Y, ldy, epi);
    if (st != LPV_OK || M == 0)
        return st;
    lpv::LinearCall c = {X, ldx, M, bias, Y, ldy, epi == LPV_EPI_GELU};
    hipError_t e = lpv::launch_dense_linear(W, ldw, N, K, dt, c, (hipStream_t)stream);
    return e == hipSuccess ? LPV_OK : hip_fail(e, "dense_linear launch");
}

lpv_status lpv_mask_topk(const void* W, int64_t ldw, int64_t N, int64_t K, lpv_dtype dt,
                         int32_t b_r, int32_t b_c, const void* G, int64_t ldg,
                         int32_t sparsity_pct, uint8_t* mask, double* scores, void* stream)
{
    g_err[0] = 0;
    const int es = elem_size(dt);
    if (!es)
        return fail(LPV_ERR_DTYPE, "unknown element type %d", (int)dt);
    if (check_block(b_r) || check_block(b_c))
        return fail(LPV_ERR_BLOCK, "block %dx%d: each side must be 16, 32 or 64", b_r, b_c);
    if (N <= 0 || K <= 0 || N > MAX_DIM || K > MAX_DIM)
        return fail(LPV_ERR_SHAPE, "weight %lldx%lld: each side must be in [1, %lld]",
                    (long long)N, (long long)K, (long long)MAX_DIM);
    if (N % b_r || K % b_c)
        return fail(LPV_ERR_SHAPE, "block %dx%d does not divide weight %lldx%lld", b_r, b_c,
                    (long long)N, (long long)K);
    if (sparsity_pct < 0 || sparsity_pct > 100)
        return fail(LPV_ERR_INVALID_ARG, "sparsity %d%% is outside [0, 100]", sparsity_pct);
    if (!W || !mask || !scores)
        return fail(LPV_ERR_INVALID_ARG, "W, mask and scores must not be NULL");
    if (ldw < K || (G && ldg < K))
        return fail(LPV_ERR_INVALID_ARG, "ldw and ldg must be >= K");
    if ((uintptr_t)W % es || (G && (uintptr_t)G % es) || (uintptr_t)scores % 8)
        return fail(LPV_ERR_INVALID_ARG, "W and G must be aligned to their element size, scores "
                                         "to 8 bytes");
    const int64_t nb = (N / b_r) * (K / b_c);
    lpv::MaskCall m = {W, ldw, G, ldg, N, K, (int)dt, b_r, b_c,
                       ((100 - (int64_t)sparsity_pct) * nb + 99) / 100, mask, scores};
    hipError_t e = lpv::launch_mask_topk(m, (hipStream_t)stream);
    return e == hipSuccess ? LPV_OK : hip_fail(e, "mask_topk launch");
}

lpv_status lpv_bsr_transpose(const lpv_bsr* h, void* stream, lpv_bsr** out)
{
    g_err[0] = 0;
    if (!out)
        return fail(LPV_ERR_INVALID_ARG, "out must not be NULL");
    *out = nullptr;
    if (!h)
        return fail(LPV_ERR_INVALID_ARG, "handle must not be NULL");
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return hip_fail(e, "hipGetDevice");
    if (dev != h->device)
        return fail(LPV_ERR_INVALID_ARG, "handle lives on device %d, current device is %d",
                    h->device, dev);
    hipStream_t s = (hipStream_t)stream;
    const int es = elem_size(h->dtype);
    // the pruned weight transposed (K x N, row stride N) and the transposed
    // mask (C x R), built on the device and packed like any weight
    void* WT = nullptr;
    void* mT = nullptr;
    e = dmalloc(&WT, (size_t)(h->K * h->N) * es);
    if (e == hipSuccess)
        e = dmalloc(&mT, (size_t)h->R * h->C);
    if (e != hipSuccess) {
        (void)hipFree(WT);
        return e == hipErrorOutOfMemory ? fail(LPV_ERR_ALLOC, "device allocation failed")
                                        : hip_fail(e, "hipMalloc");
    }
    e = hipMemsetAsync(WT, 0, (size_t)(h->K * h->N) * es, s);
    if (e == hipSuccess)
        e = hipMemsetAsync(mT, 0, (size_t)h->R * h->C, s);
    if (e == hipSuccess)
        e = lpv::launch_transpose_blocks(h, WT, h->N, (uint8_t*)mT, s);
    lpv_status st = e == hipSuccess ? LPV_OK : hip_fail(e, "transpose launch");
    if (st == LPV_OK)
        st = lpv_bsr_pack(WT, h->N, h->K, h->N, (lpv_dtype)h->dtype, h->b_c, h->b_r,
                          (const uint8_t*)mT, stream, out);
    const hipError_t es2 = hipStreamSynchronize(s);  // before the buffers are freed
    (void)hipFree(WT);
    (void)hipFree(mT);
    if (st == LPV_OK && es2 != hipSuccess) {
        lpv_bsr_destroy(*out);
        *out = nullptr;
        return hip_fail(es2, "transpose");
    }
    return st;
}

lpv_status lpv_bsr_grad_w(const lpv_bsr* h, const void* G, int64_t ldg, const void* X,
                          int64_t ldx, int64_t M, void* dW, void* stream)
{
    if (!h)
        return fail(LPV_ERR_INVALID_ARG, "handle must not be NULL");
    const int es = elem_size(h->dtype);
    if (M < 0 || M >= MAX_M)
        return fail(LPV_ERR_SHAPE, "M = %lld is out of range [0, 2^31)", (long long)M);
    if (ldg < h->N || ldx < h->K)
        return fail(LPV_ERR_INVALID_ARG, "ldg must be >= N and ldx >= K");
    if (ldg > MAX_LD || ldx > MAX_LD)
        return fail(LPV_ERR_INVALID_ARG, "ldg and ldx must be at most %lld", (long long)MAX_LD);
    if ((ldg * es) % 16 || (ldx * es) % 16)
        return fail(LPV_ERR_INVALID_ARG, "ldg and ldx must be multiples of 16 bytes");
    if (h->nnzb > 0 && (!dW || (uintptr_t)dW % es))
        return fail(LPV_ERR_INVALID_ARG, "dW must be non-NULL and aligned to its element size");
    if (M > 0 && (!G || !X || !aligned16(G) || !aligned16(X)))
        return fail(LPV_ERR_INVALID_ARG, "G and X must be non-NULL and 16-byte aligned");
    if (M > 0 && h->nnzb > 0) {
        const uintptr_t w0 = (uintptr_t)dW,
                        w1 = w0 + (uintptr_t)(h->nnzb * h->b_r * h->b_c * es);
        const uintptr_t g0 = (uintptr_t)G, g1 = g0 + (uintptr_t)(((M - 1) * ldg + h->N) * es);
        const uintptr_t x0 = (uintptr_t)X, x1 = x0 + (uintptr_t)(((M - 1) * ldx + h->K) * es);
        if ((w0 < g1 && g0 < w1) || (w0 < x1 && x0 < w1))
            return fail(LPV_ERR_ALIAS, "dW overlaps G or X");
    }
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return hip_fail(e, "hipGetDevice");
    if (dev != h->device)
        return fail(LPV_ERR_INVALID_ARG, "handle lives on device %d, current device is %d",
                    h->device, dev);
    // the handle's workspace, allocated on its first weight-gradient call
    // (its size does not depend on M)
    const size_t need = lpv::grad_w_workspace_bytes(h);
    if (M > 0 && need > h->gradw_ws_bytes) {
        static std::mutex ws_mutex;
        std::lock_guard<std::mutex> lock(ws_mutex);
        if (need > h->gradw_ws_bytes) {
            if (h->gradw_ws) {
                e = hipDeviceSynchronize();  // (the size is fixed per handle: not reached)
                if (e != hipSuccess)
                    return hip_fail(e, "hipDeviceSynchronize");
                (void)hipFree(h->gradw_ws);
                h->gradw_ws = nullptr;
                h->gradw_ws_bytes = 0;
            }
            void* p = nullptr;
            e = dmalloc(&p, need);
            if (e != hipSuccess)
                return e == hipErrorOutOfMemory ? fail(LPV_ERR_ALLOC, "workspace allocation failed")
                                                : hip_fail(e, "hipMalloc");
            h->gradw_ws = p;
            h->gradw_ws_bytes = need;
        }
    }
    lpv::GradWCall c = {G, ldg, X, ldx, M, dW, (float*)h->gradw_ws};
    e = lpv::launch_grad_w(h, c, (hipStream_t)stream);
    if (e == hipErrorOutOfMemory)
        return fail(LPV_ERR_ALLOC, "workspace allocation failed");
    return e == hipSuccess ? LPV_OK : hip_fail(e, "grad_w launch");
}

namespace {

// Shared checks of the two bias-gradient calls.
lpv_status check_bias_grad(const void* G, int64_t ldg, int64_t M, int64_t N, lpv_dtype dt,
                           void* db)
{
    const int es = elem_size(dt);
    if (!es)
        return fail(LPV_ERR_DTYPE, "unknown element type %d", (int)dt);
    if (N <= 0 || N > MAX_DIM)
        return fail(LPV_ERR_SHAPE, "N = %lld is out of range [1, %lld]", (long long)N,
                    (long long)MAX_DIM);
    if (M < 0 || M >= MAX_M)
        return fail(LPV_ERR_SHAPE, "M = %lld is out of range [0, 2^31)", (long long)M);
    if (ldg < N || ldg > MAX_LD || (ldg * es) % 16)
        return fail(LPV_ERR_INVALID_ARG, "ldg must be in [N, 2^22] and a multiple of 16 bytes");
    if (!db || (uintptr_t)db % es)
        return fail(LPV_ERR_INVALID_ARG, "db must be non-NULL and aligned to its element size");
    if (M > 0 && (!G || !aligned16(G)))
        return fail(LPV_ERR_INVALID_ARG, "G must be non-NULL and 16-byte aligned");
    return LPV_OK;
}

}  // namespace

lpv_status lpv_bias_grad(const void* G, int64_t ldg, int64_t M, int64_t N, lpv_dtype dt,
                         void* db, void* stream)
{
    const lpv_status st = check_bias_grad(G, ldg, M, N, dt, db);
    if (st != LPV_OK)
        return st;
    hipError_t e = lpv::launch_bias_grad(G, ldg, M, N, dt, db, (hipStream_t)stream);
    if (e == hipErrorOutOfMemory)
        return fail(LPV_ERR_ALLOC, "workspace allocation failed");
    return e == hipSuccess ? LPV_OK : hip_fail(e, "bias_grad launch");
}

lpv_status lpv_bias_grad_noalloc(const void* G, int64_t ldg, int64_t M, int64_t N, lpv_dtype dt,
                                 void* db, void* stream)
{
    const lpv_status st = check_bias_grad(G, ldg, M, N, dt, db);
    if (st != LPV_OK)
        return st;
    if (N > lpv::BIAS_NOALLOC_SCRATCH_FLOATS)
        return fail(LPV_ERR_SHAPE, "N = %lld is above the %lld columns the fixed scratch holds",
                    (long long)N, (long long)lpv::BIAS_NOALLOC_SCRATCH_FLOATS);
    const hipError_t e = lpv::launch_bias_grad_noalloc(G, ldg, M, N, dt, db, (hipStream_t)stream);
    return e == hipSuccess ? LPV_OK : hip_fail(e, "bias_grad_noalloc launch");
}

}  // extern "C"

namespace {

lpv_status delta_curve_impl(const void* W, int64_t ldw, int64_t N, int64_t K, lpv_dtype dt,
                            int32_t b_r, int32_t b_c, const void* grad, int64_t ldg,
                            const void* samples, int64_t lds, int64_t sample_stride,
                            int64_t n_samples, double kappa, const int32_t* pcts,
                            int32_t n_points, double* delta, void* ws, size_t ws_bytes,
                            void* stream)
{
    g_err[0] = 0;
    const int es = elem_size(dt);
    if (!es)
        return fail(LPV_ERR_DTYPE, "unknown element type %d", (int)dt);
    if (check_block(b_r) || check_block(b_c))
        return fail(LPV_ERR_BLOCK, "block %dx%d: each side must be 16, 32 or 64", b_r, b_c);
    if (N <= 0 || K <= 0 || N > MAX_DIM || K > MAX_DIM)
        return fail(LPV_ERR_SHAPE, "weight %lldx%lld: each side must be in [1, %lld]",
                    (long long)N, (long long)K, (long long)MAX_DIM);
    if (N % b_r || K % b_c)
        return fail(LPV_ERR_SHAPE, "block %dx%d does not divide weight %lldx%lld", b_r, b_c,
                    (long long)N, (long long)K);
    if ((N / b_r) * (K / b_c) > lpv::DELTA_MAX_BLOCKS)
        return fail(LPV_ERR_SHAPE, "%lld blocks: at most %lld are supported",
                    (long long)((N / b_r) * (K / b_c)), (long long)lpv::DELTA_MAX_BLOCKS);
    if (n_samples < 0 || n_samples > 65000)  // one grid row per vector
        return fail(LPV_ERR_SHAPE, "n_samples = %lld is out of range [0, 65000]",
                    (long long)n_samples);
    if (n_points < 1 || n_points > lpv::DELTA_MAX_POINTS || !pcts)
        return fail(LPV_ERR_INVALID_ARG, "1 to %d sparsity points are needed",
                    lpv::DELTA_MAX_POINTS);
    for (int i = 0; i < n_points; ++i)
        if (pcts[i] < 0 || pcts[i] > 100 || (i > 0 && pcts[i] < pcts[i - 1]))
            return fail(LPV_ERR_INVALID_ARG, "sparsity points must ascend within [0, 100]");
    if (!(kappa == kappa) || kappa > 1e300 || kappa < -1e300)
        return fail(LPV_ERR_INVALID_ARG, "kappa must be finite");
    if (!W || !grad || !delta || (n_samples > 0 && !samples))
        return fail(LPV_ERR_INVALID_ARG, "W, grad, delta (and samples) must not be NULL");
    if (!aligned16(W) || !aligned16(grad) || (n_samples > 0 && !aligned16(samples)) ||
        (uintptr_t)delta % 8)
        return fail(LPV_ERR_INVALID_ARG, "W, grad and samples must be 16-byte aligned, delta 8");
    if (ldw < K || ldg < K || (n_samples > 0 && lds < K) || ldw > MAX_LD || ldg > MAX_LD ||
        lds > MAX_LD || (ldw * es) % 16 || (ldg * es) % 16 || (n_samples > 0 && (lds * es) % 16))
        return fail(LPV_ERR_INVALID_ARG, "ldw, ldg, lds must be in [K, 2^22] and multiples of 16 "
                                         "bytes");
    if (n_samples > 0 && (sample_stride < (N - 1) * lds + K || (sample_stride * es) % 16))
        return fail(LPV_ERR_INVALID_ARG, "sample_stride must cover one sample and be a multiple "
                                         "of 16 bytes");
    lpv::DeltaCall c = {};
    c.W = W;
    c.ldw = ldw;
    c.N = N;
    c.K = K;
    c.dtype = dt;
    c.b_r = b_r;
    c.b_c = b_c;
    c.grad = grad;
    c.ldg = ldg;
    c.samples = samples;
    c.lds = lds;
    c.stride = sample_stride;
    c.n_samples = n_samples;
    c.kappa = kappa;
    c.n_points = n_points;
    const int64_t nb = (N / b_r) * (K / b_c);
    for (int i = 0; i < n_points; ++i)
        c.keep[i] = (int32_t)(((100 - (int64_t)pcts[i]) * nb + 99) / 100);
    c.delta = delta;
    if (ws) {
        const size_t need = lpv::delta_workspace_bytes(N, K, b_r, b_c, n_samples, n_points);
        if (ws_bytes < need || (uintptr_t)ws % 16)
            return fail(LPV_ERR_INVALID_ARG, "workspace: %zu bytes 16-byte aligned are needed",
                        need);
    }
    c.ws = ws;
    c.ws_bytes = ws_bytes;
    hipError_t e = lpv::launch_delta_curve(c, (hipStream_t)stream);
    if (e == hipErrorOutOfMemory)
        return fail(LPV_ERR_ALLOC, "workspace allocation failed");
    return e == hipSuccess ? LPV_OK : hip_fail(e, "delta_curve launch");
}

}  // namespace

extern "C" {

lpv_status lpv_delta_curve(const void* W, int64_t ldw, int64_t N, int64_t K, lpv_dtype dt,
                           int32_t b_r, int32_t b_c, const void* grad, int64_t ldg,
                           const void* samples, int64_t lds, int64_t sample_stride,
                           int64_t n_samples, double kappa, const int32_t* pcts, int32_t n_points,
                           double* delta, void* stream)
{
    return delta_curve_impl(W, ldw, N, K, dt, b_r, b_c, grad, ldg, samples, lds, sample_stride,
                            n_samples, kappa, pcts, n_points, delta, nullptr, 0, stream);
}

lpv_status lpv_delta_curve_ws(const void* W, int64_t ldw, int64_t N, int64_t K, lpv_dtype dt,
                              int32_t b_r, int32_t b_c, const void* grad, int64_t ldg,
                              const void* samples, int64_t lds, int64_t sample_stride,
                              int64_t n_samples, double kappa, const int32_t* pcts,
                              int32_t n_points, double* delta, void* workspace,
                              size_t workspace_bytes, void* stream)
{
    if (!workspace)
        return fail(LPV_ERR_INVALID_ARG, "workspace must not be NULL");
    return delta_curve_impl(W, ldw, N, K, dt, b_r, b_c, grad, ldg, samples, lds, sample_stride,
                            n_samples, kappa, pcts, n_points, delta, workspace, workspace_bytes,
                            stream);
}

lpv_status lpv_delta_curve_workspace_size(int64_t N, int64_t K, int32_t b_r, int32_t b_c,
                                          int64_t n_samples, int32_t n_points, size_t* bytes)
{
    if (!bytes)
        return fail(LPV_ERR_INVALID_ARG, "bytes must not be NULL");
    if (check_block(b_r) || check_block(b_c))
        return fail(LPV_ERR_BLOCK, "block %dx%d: each side must be 16, 32 or 64", b_r, b_c);
    if (N <= 0 || K <= 0 || N > MAX_DIM || K > MAX_DIM || N % b_r || K % b_c ||
        (N / b_r) * (K / b_c) > lpv::DELTA_MAX_BLOCKS)
        return fail(LPV_ERR_SHAPE, "weight %lldx%lld with %dx%d blocks", (long long)N,
                    (long long)K, b_r, b_c);
    if (n_samples < 0 || n_samples > 65000 || n_points < 1 || n_points > lpv::DELTA_MAX_POINTS)
        return fail(LPV_ERR_INVALID_ARG, "n_samples in [0, 65000], n_points in [1, %d]",
                    lpv::DELTA_MAX_POINTS);
    *bytes = lpv::delta_workspace_bytes(N, K, b_r, b_c, n_samples, n_points);
    return LPV_OK;
}

void lpv_bsr_destroy(lpv_bsr* h)
{
    free_handle(h);
}

}  // extern "C"

lpv_status lpv_add_layernorm(const void* x, const void* y, int64_t M, int64_t D, lpv_dtype dt,
                             const void* gamma, const void* beta, double eps, void* S, void* out,
                             void* stream)
{
    if (dt != LPV_BF16 && dt != LPV_F16)
        return fail(LPV_ERR_DTYPE, "add_layernorm takes 16-bit element types only (got %d)", (int)dt);
    if (D < 4 || D > lpv::LN_MAX_D || D % 4)
        return fail(LPV_ERR_SHAPE, "D = %lld must be a multiple of 4 in [4, %d]", (long long)D,
                    lpv::LN_MAX_D);
    if (M < 0 || M >= MAX_M)
        return fail(LPV_ERR_SHAPE, "M = %lld is out of range [0, 2^31)", (long long)M);
    if (!(eps >= 0.0) || !std::isfinite(eps))
        return fail(LPV_ERR_INVALID_ARG, "eps must be finite and >= 0");
    auto a8 = [](const void* p) { return ((uintptr_t)p & 7u) == 0; };
    if (!gamma || !beta || !a8(gamma) || !a8(beta))
        return fail(LPV_ERR_INVALID_ARG, "gamma and beta must be non-NULL and 8-byte aligned");
    if (M > 0 && (!x || !out || !a8(x) || !a8(out) || (y && !a8(y)) || (S && !a8(S))))
        return fail(LPV_ERR_INVALID_ARG, "x, y, S and out must be 8-byte aligned (x, out non-NULL)");
    hipError_t e = lpv::launch_add_layernorm(x, y, M, (int32_t)D, dt, gamma, beta, (float)eps, S,
                                             out, (hipStream_t)stream);
    return e == hipSuccess ? LPV_OK : hip_fail(e, "add_layernorm launch");
}

lpv_status lpv_attention(const void* qkv, int64_t n_seq, int32_t T, int32_t H, int32_t hd,
                         lpv_dtype dt, void* out, void* stream)
{
    if (dt != LPV_BF16 && dt != LPV_F16)
        return fail(LPV_ERR_DTYPE, "attention takes 16-bit element types only (got %d)", (int)dt);
    if (hd != lpv::ATT_HD)
        return fail(LPV_ERR_SHAPE, "head dimension %d is not supported (only %d)", hd, lpv::ATT_HD);
    if (T < 1 || T > lpv::ATT_MAX_T)
        return fail(LPV_ERR_SHAPE, "T = %d is out of range [1, %d]", T, lpv::ATT_MAX_T);
    if (H < 1 || H > 64)
        return fail(LPV_ERR_SHAPE, "H = %d is out of range [1, 64]", H);
    if (n_seq < 0 || n_seq * T >= MAX_M || n_seq * H >= MAX_M)
        return fail(LPV_ERR_SHAPE, "n_seq = %lld is out of range", (long long)n_seq);
    if (n_seq > 0) {
        if (!qkv || !out || !aligned16(qkv) || !aligned16(out))
            return fail(LPV_ERR_INVALID_ARG, "qkv and out must be non-NULL and 16-byte aligned");
        const uintptr_t q0 = (uintptr_t)qkv, q1 = q0 + (uintptr_t)(n_seq * T * 3 * H * hd * 2);
        const uintptr_t o0 = (uintptr_t)out, o1 = o0 + (uintptr_t)(n_seq * T * H * hd * 2);
        if (o0 < q1 && q0 < o1)
            return fail(LPV_ERR_ALIAS, "out must not overlap qkv");
    }
    hipError_t e = lpv::launch_attention(qkv, n_seq, T, H, dt, out, (hipStream_t)stream);
    return e == hipSuccess ? LPV_OK : hip_fail(e, "attention launch");
}
