/*
 * lpv.h -- C ABI of liblpv, a block-sparse linear layer for AMD MI355X (gfx950).
 *
 * The layer is the one that block-structured pruning of vision transformers
 * (LPViT, arXiv 2407.02068) makes cheaper:
 *
 *     Y = g(X * W~^T + b)
 *
 * X is the dense token-by-channel activation (M tokens x K input features), W is
 * a linear weight in the nn.Linear layout (N output features x K input
 * features), b the bias and g the identity or GELU.  W~ is W with whole blocks
 * removed: the weight is cut into a grid of b_r x b_c blocks, a binary block
 * mask keeps or drops each block, and W~[n][k] = W[n][k] when the block
 * (n / b_r, k / b_c) is kept and 0 otherwise (the paper's masked weight, Sec.
 * 3.1).  The work of the layer is proportional to the number of kept blocks
 * times the number of token tiles (the per-matmul cost model of Sec. 3.4).
 *
 * Conventions shared by every call
 * --------------------------------
 * - Pointers named as device pointers are HIP device memory of the current
 *   device; the caller owns them.  The library keeps no caller pointer after a
 *   call returns.
 * - Matrices are row-major with a leading dimension in ELEMENTS (ldx, ldw,
 *   ldy).  Device pointers must be 16-byte aligned and ld * element size must be
 *   a multiple of 16 bytes; otherwise LPV_ERR_INVALID_ARG.
 * - X, W, bias and Y share one element type (lpv_dtype).  Arithmetic inside
 *   the kernels is float32 (bf16/fp16 inputs go to the matrix cores with float32
 *   accumulation); the result is rounded once, to nearest even, to the element
 *   type.
 * - `stream` is a hipStream_t (NULL = the default stream).  Every call only
 *   enqueues work on it and returns, except lpv_bsr_pack, which waits once for
 *   its own work (see there).
 * - Every argument is checked before any HIP call; a bad argument returns a
 *   negative lpv_status and changes nothing.  lpv_last_error() then gives a
 *   message for the calling thread.  No exception crosses the ABI.
 * - Block sides b_r and b_c are each 16, 32 or 64 (the block shapes of the
 *   paper's experiments, Tables 2 and 4); they must divide N and K exactly (the
 *   block-score grid of Sec. 3.1 has N/b_r x K/b_c entries), else
 *   LPV_ERR_SHAPE.  Non-finite values in X are outside the contract.
 */
#ifndef LPV_H
#define LPV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    LPV_OK = 0,
    LPV_ERR_INVALID_ARG = -1, /* null pointer, bad leading dimension, misalignment */
    LPV_ERR_SHAPE = -2,       /* sizes out of range or not divisible by the block */
    LPV_ERR_DTYPE = -3,       /* unknown element type */
    LPV_ERR_BLOCK = -4,       /* block side not in {16, 32, 64} */
    LPV_ERR_ALIAS = -5,       /* X and Y overlap */
    LPV_ERR_ALLOC = -6,       /* device or host allocation failed */
    LPV_ERR_HIP = -7          /* a HIP runtime call failed; see lpv_last_error() */
} lpv_status;

typedef enum { LPV_F32 = 0, LPV_F16 = 1, LPV_BF16 = 2 } lpv_dtype;

typedef enum { LPV_EPI_NONE = 0, LPV_EPI_GELU = 1 } lpv_epilogue;

/* A packed block-sparse weight.  Opaque; owns its device buffers; immutable
 * after lpv_bsr_pack returns, so calls on different streams may share it. */
typedef struct lpv_bsr lpv_bsr;

typedef struct {
    int64_t N, K;         /* weight shape: output x input features */
    int32_t b_r, b_c;     /* block shape */
    int32_t R, C;         /* block grid: N / b_r x K / b_c */
    int64_t nnzb;         /* kept blocks */
    int32_t dtype;        /* lpv_dtype */
    int32_t device;       /* HIP device the buffers live on */
    /* tile schedule (see lpv_bsr_schedule_export) */
    int32_t tile_rows;    /* output rows per schedule tile (32) */
    int32_t tile_cols;    /* reduction columns per schedule tile (32) */
    int32_t group_tiles;  /* tile rows per group */
    int32_t n_groups;     /* groups of tile rows */
    int64_t n_steps;      /* (group, tile column) pairs with work */
    int64_t n_tiles;      /* kept (tile row, tile column) pairs */
} lpv_bsr_info;

/*
 * lpv_bsr_pack -- mask -> BSR (block compressed sparse row), on the GPU.
 *
 * Paper: the pruned weight W~ = W (.) M over b_r x b_c blocks (Sec. 3.1); the
 * kept-block count is the block count of the cost model (Sec. 3.4).
 *
 * W     device, N x K, row stride ldw >= K, element type dt.
 * mask  device, uint8, R x C = (N / b_r) x (K / b_c), row-major; nonzero keeps
 *       the block.
 * out   host; receives a new handle (NULL on failure).
 *
 * The handle holds the canonical BSR arrays: row_ptr[R + 1] (row_ptr[0] = 0,
 * row_ptr[r + 1] - row_ptr[r] = kept blocks of block-row r), col_idx[nnzb]
 * (ascending within a block-row) and values[nnzb][b_r][b_c] (raw element bits
 * of each kept block, row-major), plus the tile schedule and an internal copy
 * of the kept values in matrix-core operand order.  Dropped blocks are never
 * read by lpv_bsr_linear, so NaN or Inf in them cannot reach Y.
 *
 * Allocates device memory (freed by lpv_bsr_destroy) and waits once on
 * `stream` to learn the kept count.  W and mask may be freed afterwards.
 * N, K <= 65536.  bf16 / fp16: at most 2^21 - 1 kept 32 x 32 tiles (the
 * kernels address the tile copy with 32-bit byte offsets) and K <= 63424 (a
 * group's walk, one entry per 32 reduction columns, must fit the kernel's LDS
 * table); SHAPE otherwise.
 * Errors: INVALID_ARG, SHAPE, DTYPE, BLOCK, ALLOC, HIP.
 */
lpv_status lpv_bsr_pack(const void* W, int64_t ldw, int64_t N, int64_t K, lpv_dtype dt,
                        int32_t b_r, int32_t b_c, const uint8_t* mask, void* stream,
                        lpv_bsr** out);

/* Shape, kept count and schedule sizes of a handle (host struct).  nnzb is the
 * kept-block count of Sec. 3.4 (ceil((1 - alpha) R C) for a top-k mask). */
lpv_status lpv_bsr_info_get(const lpv_bsr* h, lpv_bsr_info* out);

/*
 * lpv_bsr_export -- copy the canonical BSR arrays (described at lpv_bsr_pack):
 * the kept blocks of the masked weight of Sec. 3.1, by block row, into caller
 * device buffers: row_ptr int32[R + 1], col_idx int32[nnzb],
 * values [nnzb][b_r][b_c] of the handle's element type.  Any of the three may
 * be NULL to skip it.  Asynchronous on `stream`.
 */
lpv_status lpv_bsr_export(const lpv_bsr* h, int32_t* row_ptr, int32_t* col_idx, void* values,
                          void* stream);

/*
 * lpv_bsr_schedule_export -- copy the tile schedule into caller device buffers
 * (each may be NULL).  The schedule counts the work of each output group in
 * kept tiles, the unit of the cost model of Sec. 3.4 (token tiles times kept
 * blocks):
 *   group_order int32[n_groups]      groups in launch order (most work first);
 *   step_ptr    int32[n_groups + 1]  steps of group g are [step_ptr[g], step_ptr[g+1]);
 *   step_col    int32[n_steps]       tile column of each step, ascending per group;
 *   step_bits   int32[n_steps]       bit j set when tile row g*group_tiles + j keeps
 *                                    tile (row, step_col);
 *   step_tile   int32[n_steps]       index of the step's first kept tile in the
 *                                    operand-order value stream (prefix sum of
 *                                    popcount(step_bits)).
 * A tile is tile_rows x tile_cols elements of W; it is kept when any element of
 * it lies in a kept block.  Asynchronous on `stream`.
 */
lpv_status lpv_bsr_schedule_export(const lpv_bsr* h, int32_t* group_order, int32_t* step_ptr,
                                   int32_t* step_col, int32_t* step_bits, int32_t* step_tile,
                                   void* stream);

/*
 * lpv_bsr_unpack -- the pruned dense weight W~ = W (.) M of Sec. 3.1 (N x K,
 * row stride ldw >= K) into a caller device buffer; dropped blocks become
 * +0.0.  Asynchronous.
 */
lpv_status lpv_bsr_unpack(const lpv_bsr* h, void* W_out, int64_t ldw, void* stream);

/*
 * lpv_bsr_linear -- Y = g(X * W~^T + b), the block-sparse hot path.
 *
 * X     device, M x K, row stride K <= ldx <= 2^22 (the kernels address a
 *       256-token slice of X with 32-bit byte offsets).
 * bias  device, N elements, or NULL for no bias.
 * Y     device, M x N, row stride ldy >= N; must not overlap X.
 * epi   LPV_EPI_NONE or LPV_EPI_GELU (x Phi(x) with the error function, after
 *       the bias, in float32 to 5e-6 relative).
 *
 * The product of the input with the block-sparse weight of Sec. 3.4: each
 * token tile times each group of output tile rows walks only the kept tiles
 * of its rows, on the matrix cores for bf16/fp16.  M = 0 is a no-op.
 * One kernel launch per run of output groups whose per-launch tables fit in
 * LDS (a single launch for ViT-sized layers), no allocation, no host
 * synchronisation.
 * Errors: INVALID_ARG, SHAPE, ALIAS, HIP.
 */
lpv_status lpv_bsr_linear(const lpv_bsr* h, const void* X, int64_t ldx, int64_t M,
                          const void* bias, void* Y, int64_t ldy, lpv_epilogue epi,
                          void* stream);

/*
 * lpv_dense_linear -- Y = g(X * W^T + b) with a dense W (N x K, row stride
 * K <= ldw <= 2^22), through the library's own matrix-core kernel: the
 * unpruned layer, the counterpart of the "Dense" rows of Tab. 2 and Tab. 4,
 * and the reference point for the speed-up of the block-sparse path.  Same
 * conventions as lpv_bsr_linear; N and K must be multiples of 16 and at most
 * 65536, K at most 63424 for bf16 / fp16 (SHAPE otherwise).
 */
lpv_status lpv_dense_linear(const void* W, int64_t ldw, int64_t N, int64_t K, lpv_dtype dt,
                            const void* X, int64_t ldx, int64_t M, const void* bias, void* Y,
                            int64_t ldy, lpv_epilogue epi, void* stream);

/*
 * lpv_mask_topk -- the block mask of a weight (Sec. 3.1): score every b_r x b_c
 * block, keep the ceil((100 - sparsity_pct) R C / 100) best-ranked (Sec. 3.4's
 * kept-block count at an integer percentage), drop the rest.
 *
 * W       device, N x K, row stride ldw >= K, element type dt.
 * G       device, N x K (row stride ldg >= K), dt: the loss gradient dL/dW.
 *         Given, a block's score is the mean of |W * G| over its elements (the
 *         paper's 2-D average pool of the first-order Taylor score); NULL, it
 *         is the block's sum of squares W^2 (ranks like the L2 norm).
 * mask    device, R x C uint8, row-major (R = N / b_r, C = K / b_c): 1 keeps
 *         the block.  It is the input of lpv_bsr_pack.
 * scores  device, R x C float64, receives the block scores (also the
 *         selection's workspace).
 *
 * A score is summed in float64 over the block's elements in row-major order,
 * one addition after the other, so its value is reproducible bit for bit.
 * Ranking: larger score first, equal scores by lower row-major block index.
 * NaN in W or G is outside the contract.  Two kernel launches on `stream`, no
 * allocation, no host synchronisation.  b_r, b_c in {16, 32, 64}.
 * Errors: INVALID_ARG, SHAPE, DTYPE, BLOCK, HIP.
 */
lpv_status lpv_mask_topk(const void* W, int64_t ldw, int64_t N, int64_t K, lpv_dtype dt,
                         int32_t b_r, int32_t b_c, const void* G, int64_t ldg,
                         int32_t sparsity_pct, uint8_t* mask, double* scores, void* stream);

/*
 * Backward of the layer, for finetuning the pruned model (Fig. 1, Sec. 4).
 * The mask stays fixed: a dropped block neither passes a gradient to the
 * input nor receives one.  G is the gradient at the pre-activation
 * Z = X W~^T + b (M x N): with the GELU epilogue the caller multiplies dL/dY
 * by GELU'(Z) element-wise first.  The three results follow from the chain
 * rule: dX = G W~, dW = G^T X on the kept blocks, db = sum over tokens of G.
 */

/*
 * lpv_bsr_transpose -- a new handle holding W~^T (K x N, blocks b_c x b_r) of
 * the handle h, so that the input gradient is the forward call on it:
 *   lpv_bsr_linear(ht, G, ldg, M, NULL, dX, lddx, LPV_EPI_NONE, stream)
 * computes dX = G W~ (M x K).  Its BSR arrays are those lpv_bsr_pack gives for
 * the transposed weight and mask.  Device work on `stream`, synchronised
 * before returning (like lpv_bsr_pack); temporary device memory of K N
 * elements is allocated and freed.  *out receives the handle (release it with
 * lpv_bsr_destroy), NULL on failure.
 * Errors: INVALID_ARG, SHAPE (K N too large for pack), ALLOC, HIP.
 */
lpv_status lpv_bsr_transpose(const lpv_bsr* h, void* stream, lpv_bsr** out);

/*
 * lpv_bsr_grad_w -- the weight gradient on the kept blocks:
 *   dW[n][k] = sum over m of G[m][n] X[m][k]   for (n, k) in a kept block.
 * G       device, M x N (row stride ldg >= N), the handle's element type.
 * X       device, M x K (row stride ldx >= K), same type: the layer's input.
 * dW      device, nnzb x b_r x b_c elements of the handle's type, written in
 *         the BSR value order of lpv_bsr_export (block-rows ascending, kept
 *         columns ascending, each block row-major).
 * Sums run in float32 over fixed token chunks added in a fixed order, one
 * rounding at the end.  16-bit types use the matrix cores; fp32 handles a
 * plain kernel.  The partial sums of the kept tiles per token chunk live in a
 * workspace the handle owns: allocated on the handle's first 16-bit call
 * (chunks x kept tiles x 4 KiB, the chunk count fixed per handle by the
 * device's compute-unit count) and freed by lpv_bsr_destroy, so later calls
 * allocate nothing.  Calls on one handle that overlap in time (different
 * streams) race on it and are not allowed; calls in one stream's order are
 * fine.  M = 0 writes zeros.  G, X 16-byte aligned, ldg and ldx multiples of
 * 16 bytes and at most 2^22 elements, M < 2^31.  No host synchronisation.
 * Errors: INVALID_ARG, SHAPE, ALLOC (first call only), HIP.
 */
lpv_status lpv_bsr_grad_w(const lpv_bsr* h, const void* G, int64_t ldg, const void* X,
                          int64_t ldx, int64_t M, void* dW, void* stream);

/*
 * lpv_bias_grad -- db[n] = sum over m of G[m][n] (N elements of type dt).
 * G device, M x N, row stride ldg >= N, 16-byte aligned, ldg a multiple of 16
 * bytes.  float32 sums over fixed token chunks added in order, one rounding.
 * Allocates and frees a stream-ordered workspace; no host synchronisation.
 * M = 0 gives zeros.
 * Errors: INVALID_ARG, SHAPE, DTYPE, ALLOC, HIP.
 */
lpv_status lpv_bias_grad(const void* G, int64_t ldg, int64_t M, int64_t N, lpv_dtype dt,
                         void* db, void* stream);

/*
 * lpv_bias_grad_noalloc -- lpv_bias_grad for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving or training
 * loops, harnesses that forbid hipMalloc).  Same arguments, checks and result
 * as lpv_bias_grad (the token chunking may differ, so the float32 sums may
 * round differently, within the same bound); it calls no allocation routine.
 * Its partial sums live in a fixed scratch array of 2^20 float32 (4 MiB) that
 * each device the call runs on holds until the process ends; the chunk count
 * is capped so that chunks x N fits (N up to 2^20; SHAPE above).  Every call
 * on one device shares that array: calls that overlap in time on one device
 * (different streams, threads) race and are not allowed.  Nothing in the
 * array needs clearing between calls: each call writes every partial it reads.
 * Errors: INVALID_ARG, SHAPE, DTYPE, HIP.
 */
lpv_status lpv_bias_grad_noalloc(const void* G, int64_t ldg, int64_t M, int64_t N, lpv_dtype dt,
                                 void* db, void* stream);

/*
 * lpv_delta_curve -- the delta curve of one layer (Sec. 3.3): the second-order
 * Taylor term of pruning it at ratio alpha,
 *   delta(alpha) = grad . dW + 1/2 dW^T H dW,  H = kappa I + (1/n) sum_s g_s g_s^T
 * (the empirical Fisher over n calibration samples), at each sparsity
 * percentage pcts[i] (alpha = pcts[i] / 100).  dW = -W on the blocks dropped at
 * that percentage: those outside the top ceil((100 - p) R C / 100) by the
 * Taylor score mean |W grad| per block (lpv_mask_topk's ranking with G = grad;
 * ties to the lower row-major index), so the dropped sets are nested.
 *
 * W        device, N x K (row stride ldw), element type dt.
 * grad     device, N x K (row stride ldg), dt: the layer's loss gradient.
 * samples  device, n_samples per-sample gradients, each N x K with row stride
 *          lds, sample s at samples + s * sample_stride elements; dt.
 * pcts     host, n_points (1..128) sparsity percentages, non-decreasing in
 *          [0, 100].
 * delta    device, n_points float64, receives the curve.
 *
 * The curve is built with the paper's incremental update over the ratio
 * steps: float64 dot products of every per-sample gradient (and of grad, and W)
 * with -W over every block, then the steps in rank order.  All sums run in a
 * fixed order.  At most 2^17 blocks, n_samples <= 65000.  Allocates and frees a
 * stream-ordered workspace; no host synchronisation.
 * Errors: INVALID_ARG, SHAPE, DTYPE, BLOCK, ALLOC, HIP.
 */
lpv_status lpv_delta_curve(const void* W, int64_t ldw, int64_t N, int64_t K, lpv_dtype dt,
                           int32_t b_r, int32_t b_c, const void* grad, int64_t ldg,
                           const void* samples, int64_t lds, int64_t sample_stride,
                           int64_t n_samples, double kappa, const int32_t* pcts, int32_t n_points,
                           double* delta, void* stream);

/*
 * lpv_delta_curve_ws -- lpv_delta_curve with a workspace the caller owns, for
 * the same curve (Sec. 3.3) computed over and over (one call per layer and
 * calibration batch) without an allocation per call.  Same arguments, checks
 * and result as lpv_delta_curve, plus:
 * workspace        device, at least the bytes lpv_delta_curve_workspace_size
 *                  gives for the same shape, 16-byte aligned, non-NULL; owned
 *                  by the caller, who must not reuse it before the call's work
 *                  on the stream has finished.  Its contents need no clearing.
 * workspace_bytes  its size; too small is INVALID_ARG.
 * Allocates nothing.
 * Errors: INVALID_ARG, SHAPE, DTYPE, BLOCK, HIP.
 */
lpv_status lpv_delta_curve_ws(const void* W, int64_t ldw, int64_t N, int64_t K, lpv_dtype dt,
                              int32_t b_r, int32_t b_c, const void* grad, int64_t ldg,
                              const void* samples, int64_t lds, int64_t sample_stride,
                              int64_t n_samples, double kappa, const int32_t* pcts,
                              int32_t n_points, double* delta, void* workspace,
                              size_t workspace_bytes, void* stream);

/*
 * lpv_delta_curve_workspace_size -- the workspace lpv_delta_curve_ws needs for
 * an N x K weight in b_r x b_c blocks, n_samples per-sample gradients and
 * n_points sparsity points (float64 block scores and dot products, the rank
 * tables).  Host only; writes *bytes.
 * Errors: INVALID_ARG (NULL bytes, n_samples or n_points out of range), BLOCK,
 * SHAPE.
 */
lpv_status lpv_delta_curve_workspace_size(int64_t N, int64_t K, int32_t b_r, int32_t b_c,
                                          int64_t n_samples, int32_t n_points, size_t* bytes);

/* Release a handle and its device buffers.  NULL-safe.  The caller must make
 * sure no enqueued work still uses it. */
void lpv_bsr_destroy(lpv_bsr* h);

/* Static name of a status code. */
const char* lpv_status_str(lpv_status s);

/* Detail of the calling thread's last failed call ("" if none). */
const char* lpv_last_error(void);

/* ------------------------------------------------------------------------
 * The encoder block around the pruned layers.  The paper prunes the linear
 * layers of DeiT / Swin encoder blocks (Sec. 4) and measures whole models
 * (Tab. 2); these two calls are the rest of a pre-norm block (LN -> qkv ->
 * attention -> proj -> residual -> LN -> fc1 + GELU -> fc2 -> residual), so
 * the block can run on the GPU with the block-sparse layers in place.  16-bit
 * element types only (DTYPE otherwise).
 * ------------------------------------------------------------------------ */

/*
 * lpv_add_layernorm -- per row of M rows of D elements (row-major, rows
 * contiguous): s = x + y (y may be NULL: s = x), and
 *   out = (s - mean(s)) / sqrt(var(s) + eps) * gamma + beta,
 * var the biased variance over the row.  s is formed, and the statistics
 * taken, in float32; s is written, rounded, to S when S is not NULL.
 * x, y, S, out: device, M x D, 8-byte aligned; S and out may alias x or y.
 * gamma, beta: device, D elements, 8-byte aligned.  4 <= D <= 2048, D a
 * multiple of 4; 0 <= M < 2^31; eps finite and >= 0.  No host
 * synchronisation, no allocation.
 * Errors: INVALID_ARG, SHAPE, DTYPE, HIP.
 */
lpv_status lpv_add_layernorm(const void* x, const void* y, int64_t M, int64_t D, lpv_dtype dt,
                             const void* gamma, const void* beta, double eps, void* S, void* out,
                             void* stream);

/*
 * lpv_attention -- multi-head self-attention of n_seq sequences of T tokens:
 * for every sequence and head h, out_h = softmax(Q_h K_h^T / sqrt(hd)) V_h.
 * qkv: device, (n_seq T) x (3 H hd) row-major, the qkv layer's output: row t
 *      holds q, then k, then v, each H heads of hd contiguous elements.
 * out: device, (n_seq T) x (H hd), head h in columns h hd .. h hd + hd - 1;
 *      must not overlap qkv.
 * Float32 scores and accumulation (matrix cores); the softmax weights are
 * rounded once to the element type and the output divided by their sum.
 * hd = 64; 1 <= T <= 512; 1 <= H <= 64; n_seq >= 0 with n_seq T and n_seq H
 * below 2^31.  qkv and out 16-byte aligned.  No host synchronisation, no
 * allocation.
 * Errors: INVALID_ARG, SHAPE, DTYPE, ALIAS (out overlaps qkv), HIP.
 */
lpv_status lpv_attention(const void* qkv, int64_t n_seq, int32_t T, int32_t H, int32_t hd,
                         lpv_dtype dt, void* out, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* LPV_H */
