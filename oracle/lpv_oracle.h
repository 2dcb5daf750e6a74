/*
 * lpv_oracle.h -- the float64 CPU oracle's own interface (test infrastructure
 * only; see lpv_oracle.c).  It is independent of the library's include/lpv.h:
 * the two declare no common type, constant or function.
 */
#ifndef LPV_ORACLE_H
#define LPV_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { LPVO_F32 = 0, LPVO_F16 = 1, LPVO_BF16 = 2 };

/* Bytes per element of an element type, 0 for an unknown type. */
int lpvo_elem_size(int dtype);

/* Exact decode of n elements to float64.  Returns 0, or -1 on a bad argument. */
int lpvo_decode(int dtype, const void* src, int64_t n, double* dst);

/* Plain BSR pack of W (N x K, row stride ldw elements) under the row-major
 * block mask (N/b_r x K/b_c).  row_ptr, col_idx and values may each be NULL to
 * skip that output.  Returns the kept-block count, or -1 on a bad argument
 * (including block sizes that do not divide N or K). */
int64_t lpvo_pack(int dtype, const void* W, int64_t ldw, int64_t N, int64_t K,
                  int b_r, int b_c, const uint8_t* mask,
                  int32_t* row_ptr, int32_t* col_idx, void* values);

/* Inverse of lpvo_pack: writes the pruned dense weight, +0.0 in dropped
 * blocks.  Returns 0, or -1 on a bad argument. */
int lpvo_unpack(int dtype, int64_t N, int64_t K, int b_r, int b_c,
                const int32_t* row_ptr, const int32_t* col_idx, const void* values,
                void* W_out, int64_t ldw);

/* GELU with the exact error function, float64. */
double lpvo_gelu(double v);

/* Y (float64, M x N, row stride ldy) = g(X W~^T + b); X is M x K (row stride
 * ldx), W is N x K (row stride ldw), bias has N elements or is NULL, all of
 * element type dtype.  gelu != 0 selects g = GELU.  Rows of Y are split over
 * nthreads host threads.  Returns 0, -1 on a bad argument, -2 when host memory
 * runs out. */
int lpvo_linear(int dtype, const void* X, int64_t ldx, int64_t M,
                const void* W, int64_t ldw, int64_t N, int64_t K,
                int b_r, int b_c, const uint8_t* mask, const void* bias,
                int gelu, double* Y, int64_t ldy, int nthreads);

/* Block scores (R x C float64, row-major): with G, the mean of |W * G| over
 * each block (the average-pooled first-order Taylor score); without G (NULL),
 * the sum of squares of the block's elements.  Elements are visited row by row
 * within the block and summed one after the other.  Returns 0, or -1 on a bad
 * argument. */
int lpvo_block_scores(int dtype, const void* W, int64_t ldw, const void* G, int64_t ldg,
                      int64_t N, int64_t K, int b_r, int b_c, double* scores);

/* Blocks kept at an integer sparsity percentage: ceil((100 - p) n / 100).
 * Returns -1 on a bad argument. */
int64_t lpvo_keep_count(int64_t n_blocks, int sparsity_pct);

/* Mask of the n_keep highest scores (ties: the lower index first).  Returns 0,
 * -1 on a bad argument (NaN scores included), -2 when host memory runs out. */
int lpvo_mask_topk(const double* scores, int64_t n_blocks, int64_t n_keep, uint8_t* mask);

/* Backward of the layer for G = dL/dZ at the pre-activation Z = X W~^T + b
 * (M x N, row stride ldg), in float64, the mask held fixed:
 *   lpvo_grad_x: dX (M x K, row stride lddx) = G W~, summed over n ascending;
 *     rows split over nthreads host threads.  Returns 0, -1 on a bad argument,
 *     -2 when host memory runs out.
 *   lpvo_grad_w: dW restricted to the kept blocks, G^T X summed over m
 *     ascending, written block by block in lpvo_pack's order (nnzb x b_r x b_c;
 *     dW may be NULL to count).  Returns the kept-block count, -1 or -2.
 *   lpvo_grad_bias: db[n] = sum over m ascending of G[m][n].  Returns 0 or -1. */
int lpvo_grad_x(int dtype, const void* G, int64_t ldg, int64_t M, const void* W, int64_t ldw,
                int64_t N, int64_t K, int b_r, int b_c, const uint8_t* mask, double* dX,
                int64_t lddx, int nthreads);
int64_t lpvo_grad_w(int dtype, const void* G, int64_t ldg, const void* X, int64_t ldx, int64_t M,
                    int64_t N, int64_t K, int b_r, int b_c, const uint8_t* mask, double* dW);
int lpvo_grad_bias(int dtype, const void* G, int64_t ldg, int64_t M, int64_t N, double* db);

/* The delta curve (second-order Taylor term of pruning against the pruning
 * ratio, empirical-Fisher Hessian kappa I + (1/n) sum g g^T) at each sparsity
 * percentage pcts[i] (0..100): delta[i] = grad . dW + 1/2 (kappa |dW|^2 +
 * (1/n) sum_s (g_s . dW)^2), dW = -W on the blocks dropped at that percentage
 * by the gradient's Taylor score.  grad: N x K (row stride K); samples:
 * n_samples x N x K, contiguous.  Returns 0, -1 on a bad argument, -2 when
 * host memory runs out. */
int lpvo_delta_curve(int dtype, const void* W, int64_t ldw, int64_t N, int64_t K, int b_r, int b_c,
                     const void* grad, const void* samples, int64_t n_samples, double kappa,
                     const int32_t* pcts, int n_points, double* delta);

#ifdef __cplusplus
}
#endif
#endif
