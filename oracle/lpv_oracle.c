/*
 * lpv_oracle.c -- float64 CPU oracle for the block-sparse linear layer of
 * LPViT (arXiv 2407.02068).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plain definition that the
 * GPU library is checked against.  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load it.  It shares no source, header,
 * table or helper with the HIP library, and it includes nothing from it.
 *
 * What it computes (paper, Sec. 3.1, the masked-weight formula):
 *   A weight W (H x W in the paper, N x K here: output features x input
 *   features, the nn.Linear layout) is cut into a grid of fixed (B_h, B_w)
 *   blocks; a binary block mask M keeps or drops each block, and the pruned
 *   weight is W~[i][j] = W[i][j] * M[ceil(i/B_h)][ceil(j/B_w)] (1-based).  With
 *   0-based indices the block of element (n, k) is (n / b_r, k / b_c), where
 *   b_r = B_h runs along output features and b_c = B_w along the reduction.
 *   The grid S' has H/B_h x W/B_w entries, so the block sizes must divide the
 *   weight's sides exactly (same passage); other shapes are rejected.
 *
 *   Pruning is applied here by SELECTION: a dropped element is replaced by
 *   0.0, it is not multiplied by 0.  A NaN or Inf stored in a dropped block
 *   therefore never reaches the output.
 *
 *   The linear layer is Y = X * W~^T + b over tokens m (rows of X), with an
 *   optional exact-erf GELU after the bias, all in float64:
 *     Y[m][n] = g( sum_{k=0}^{K-1} X[m][k] * W~[n][k] + b[n] ),
 *   g = identity or g(v) = v/2 * (1 + erf(v / sqrt 2)).
 *   The sum runs over k in ascending order.  Nothing is rounded to a narrower
 *   type: the float64 result is returned as is.
 *
 *   The BSR (block compressed sparse row) arrays that the library's pack call
 *   must reproduce bit for bit are, in the oracle's own plain form:
 *     row_ptr[0] = 0, row_ptr[r+1] = row_ptr[r] + (number of kept blocks in
 *       block-row r);
 *     col_idx[row_ptr[r] .. row_ptr[r+1]) = the kept block columns of block-row
 *       r in ascending order;
 *     values[p] = the raw element bits of kept block p, b_r rows of b_c
 *       elements, row-major.
 *   The kept count of a weight is the paper's per-matmul block count in its
 *   power model (Sec. 3.4): the number of blocks that survive pruning.
 *
 * Element types: 0 = fp32, 1 = fp16 (IEEE binary16), 2 = bf16.  Inputs are
 * decoded exactly to float64 by the decoders below, written from the IEEE 754
 * definitions of the formats.
 *
 * Build: gcc -O2 -ffp-contract=off -fno-fast-math -fPIC -shared -pthread
 *        lpv_oracle.c -o liblpv_oracle.so -lm
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "lpv_oracle.h"

/* ------------------------------------------------------------------------ */
/* Exact decoders                                                            */
/* ------------------------------------------------------------------------ */

/* bf16 is the upper half of an IEEE binary32: append 16 zero bits. */
static double dec_bf16(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* IEEE binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits. */
static double dec_f16(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int f = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24); /* subnormal: f * 2^-14 / 2^10 */
    else if (e == 31)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + f), e - 25); /* (1 + f/2^10) * 2^(e-15) */
    return sign ? -v : v;
}

static double dec_f32(uint32_t u)
{
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

int lpvo_elem_size(int dtype)
{
    switch (dtype) {
    case LPVO_F32: return 4;
    case LPVO_F16: return 2;
    case LPVO_BF16: return 2;
    default: return 0;
    }
}

static double dec_one(int dtype, const void* base, int64_t idx)
{
    if (dtype == LPVO_F32) {
        uint32_t u;
        memcpy(&u, (const char*)base + 4 * idx, 4);
        return dec_f32(u);
    }
    uint16_t h;
    memcpy(&h, (const char*)base + 2 * idx, 2);
    return dtype == LPVO_F16 ? dec_f16(h) : dec_bf16(h);
}

int lpvo_decode(int dtype, const void* src, int64_t n, double* dst)
{
    if (!lpvo_elem_size(dtype) || n < 0 || (n > 0 && (!src || !dst)))
        return -1;
    for (int64_t i = 0; i < n; ++i)
        dst[i] = dec_one(dtype, src, i);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Block grid and BSR pack / unpack (Sec. 3.1)                               */
/* ------------------------------------------------------------------------ */

static int grid_ok(int64_t N, int64_t K, int b_r, int b_c)
{
    return N >= 0 && K >= 0 && b_r > 0 && b_c > 0 && N % b_r == 0 && K % b_c == 0;
}

int64_t lpvo_pack(int dtype, const void* W, int64_t ldw, int64_t N, int64_t K,
                  int b_r, int b_c, const uint8_t* mask,
                  int32_t* row_ptr, int32_t* col_idx, void* values)
{
    int es = lpvo_elem_size(dtype);
    if (!es || !grid_ok(N, K, b_r, b_c) || ldw < K || !mask)
        return -1;
    int64_t R = N / b_r, C = K / b_c;
    int64_t p = 0;
    if (row_ptr)
        row_ptr[0] = 0;
    for (int64_t r = 0; r < R; ++r) {
        for (int64_t c = 0; c < C; ++c) {
            if (!mask[r * C + c])
                continue;
            if (col_idx)
                col_idx[p] = (int32_t)c;
            if (values) {
                /* block p holds rows r*b_r.. and columns c*b_c.. of W */
                char* dst = (char*)values + p * (int64_t)b_r * b_c * es;
                for (int i = 0; i < b_r; ++i) {
                    const char* src = (const char*)W + ((r * b_r + i) * ldw + c * b_c) * es;
                    memcpy(dst + (int64_t)i * b_c * es, src, (size_t)b_c * es);
                }
            }
            ++p;
        }
        if (row_ptr)
            row_ptr[r + 1] = (int32_t)p;
    }
    return p;
}

int lpvo_unpack(int dtype, int64_t N, int64_t K, int b_r, int b_c,
                const int32_t* row_ptr, const int32_t* col_idx, const void* values,
                void* W_out, int64_t ldw)
{
    int es = lpvo_elem_size(dtype);
    if (!es || !grid_ok(N, K, b_r, b_c) || ldw < K || !row_ptr || !W_out)
        return -1;
    int64_t R = N / b_r, C = K / b_c;
    /* every element starts as +0.0, which is all-zero bits in all three formats */
    for (int64_t n = 0; n < N; ++n)
        memset((char*)W_out + n * ldw * es, 0, (size_t)K * es);
    for (int64_t r = 0; r < R; ++r) {
        for (int64_t p = row_ptr[r]; p < row_ptr[r + 1]; ++p) {
            int64_t c = col_idx[p];
            if (c < 0 || c >= C)
                return -1;
            const char* src = (const char*)values + p * (int64_t)b_r * b_c * es;
            for (int i = 0; i < b_r; ++i) {
                char* dst = (char*)W_out + ((r * b_r + i) * ldw + c * b_c) * es;
                memcpy(dst, src + (int64_t)i * b_c * es, (size_t)b_c * es);
            }
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Y = g(X W~^T + b) in float64                                              */
/* ------------------------------------------------------------------------ */

double lpvo_gelu(double v)
{
    /* GELU(v) = v * Phi(v), Phi the standard normal CDF written with erf */
    return 0.5 * v * (1.0 + erf(v / sqrt(2.0)));
}

struct linear_job {
    int dtype;
    const void* X;
    int64_t ldx;
    int64_t m_begin, m_end;
    const double* Wt; /* [K][N]: the expanded, pruned weight, transposed */
    const double* b;  /* [N] */
    int64_t N, K;
    int gelu;
    double* Y;
    int64_t ldy;
};

static void* linear_rows(void* arg)
{
    struct linear_job* j = (struct linear_job*)arg;
    double* x = (double*)malloc(sizeof(double) * (size_t)(j->K ? j->K : 1));
    double* acc = (double*)malloc(sizeof(double) * (size_t)(j->N ? j->N : 1));
    if (!x || !acc) {
        free(x);
        free(acc);
        return (void*)1;
    }
    for (int64_t m = j->m_begin; m < j->m_end; ++m) {
        for (int64_t k = 0; k < j->K; ++k)
            x[k] = dec_one(j->dtype, j->X, m * j->ldx + k);
        for (int64_t n = 0; n < j->N; ++n)
            acc[n] = 0.0;
        /* acc[n] = sum over k ascending of X[m][k] * W~[n][k] */
        for (int64_t k = 0; k < j->K; ++k) {
            const double xk = x[k];
            const double* wk = j->Wt + k * j->N;
            for (int64_t n = 0; n < j->N; ++n)
                acc[n] += xk * wk[n];
        }
        double* y = j->Y + m * j->ldy;
        for (int64_t n = 0; n < j->N; ++n) {
            double v = acc[n] + j->b[n];
            y[n] = j->gelu ? lpvo_gelu(v) : v;
        }
    }
    free(x);
    free(acc);
    return NULL;
}

int lpvo_linear(int dtype, const void* X, int64_t ldx, int64_t M,
                const void* W, int64_t ldw, int64_t N, int64_t K,
                int b_r, int b_c, const uint8_t* mask, const void* bias,
                int gelu, double* Y, int64_t ldy, int nthreads)
{
    if (!lpvo_elem_size(dtype) || !grid_ok(N, K, b_r, b_c) || M < 0 || ldx < K ||
        ldw < K || ldy < N || !mask || (M > 0 && (!X || !Y)) || (N * K > 0 && !W))
        return -1;
    if (M == 0 || N == 0)
        return 0;
    const int64_t C = K / b_c;
    double* Wt = (double*)malloc(sizeof(double) * (size_t)(K * N + 1));
    double* b = (double*)malloc(sizeof(double) * (size_t)N);
    if (!Wt || !b) {
        free(Wt);
        free(b);
        return -2;
    }
    /* Expand the block mask into the dense pruned weight, transposed. */
    for (int64_t n = 0; n < N; ++n)
        for (int64_t k = 0; k < K; ++k)
            Wt[k * N + n] = mask[(n / b_r) * C + (k / b_c)] ? dec_one(dtype, W, n * ldw + k) : 0.0;
    for (int64_t n = 0; n < N; ++n)
        b[n] = bias ? dec_one(dtype, bias, n) : 0.0;

    if (nthreads < 1)
        nthreads = 1;
    if (nthreads > M)
        nthreads = (int)M;
    struct linear_job* jobs = (struct linear_job*)calloc((size_t)nthreads, sizeof *jobs);
    pthread_t* tid = (pthread_t*)calloc((size_t)nthreads, sizeof *tid);
    char* running = (char*)calloc((size_t)nthreads, 1);
    int rc = 0;
    if (!jobs || !tid || !running) {
        rc = -2;
        goto out;
    }
    /* contiguous ranges of token rows, one per thread; each row is computed
       entirely by one thread, so the result does not depend on nthreads */
    for (int t = 0; t < nthreads; ++t) {
        jobs[t] = (struct linear_job){dtype, X, ldx, M * t / nthreads, M * (t + 1) / nthreads,
                                      Wt, b, N, K, gelu, Y, ldy};
    }
    for (int t = 1; t < nthreads; ++t)
        running[t] = pthread_create(&tid[t], NULL, linear_rows, &jobs[t]) == 0;
    for (int t = 0; t < nthreads; ++t)
        if (!running[t] && linear_rows(&jobs[t]))
            rc = -2;
    for (int t = 1; t < nthreads; ++t) {
        if (running[t]) {
            void* ret = NULL;
            pthread_join(tid[t], &ret);
            if (ret)
                rc = -2;
        }
    }
out:
    free(jobs);
    free(tid);
    free(running);
    free(Wt);
    free(b);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Block scores and the top-k block mask (Sec. 3.1, Sec. 3.4)                */
/* ------------------------------------------------------------------------ */

/*
 * The paper ranks the blocks of a weight by the 2-D average pool of the
 * first-order Taylor score of its elements, S = |W . grad_W f| (element-wise),
 * and drops the bottom-ranked ones for a pruning ratio alpha; the number of
 * blocks that survive is the ceiling of (1 - alpha) times the block count (the
 * block term of the power model, Sec. 3.4).
 *
 * Score of block (r, c), in float64, its elements visited row by row
 * (n = r b_r .. r b_r + b_r - 1, and within a row k = c b_c .. c b_c + b_c - 1)
 * and accumulated one after the other:
 *   G given:  S'[r][c] = (sum |W[n][k] * G[n][k]|) / (b_r b_c)
 *   G NULL:   S'[r][c] = sum W[n][k]^2   (no gradient: the block's squared L2
 *             norm, which ranks blocks like their L2 norm)
 * Every product of two decoded elements is exact in float64 (at most 24 + 24
 * significant bits) and b_r b_c is a power of two, so the result depends only
 * on the fixed summation order.
 */
int lpvo_block_scores(int dtype, const void* W, int64_t ldw, const void* G, int64_t ldg,
                      int64_t N, int64_t K, int b_r, int b_c, double* scores)
{
    if (!lpvo_elem_size(dtype) || !grid_ok(N, K, b_r, b_c) || ldw < K || (G && ldg < K) ||
        ((N > 0 && K > 0) && (!W || !scores)))
        return -1;
    const int64_t R = N / b_r, C = K / b_c;
    for (int64_t r = 0; r < R; ++r) {
        for (int64_t c = 0; c < C; ++c) {
            double s = 0.0;
            for (int64_t n = r * b_r; n < (r + 1) * b_r; ++n) {
                for (int64_t k = c * b_c; k < (c + 1) * b_c; ++k) {
                    const double w = dec_one(dtype, W, n * ldw + k);
                    if (G)
                        s += fabs(w * dec_one(dtype, G, n * ldg + k));
                    else
                        s += w * w;
                }
            }
            scores[r * C + c] = G ? s / (double)(b_r * b_c) : s;
        }
    }
    return 0;
}

/* ceil((100 - p) / 100 * n_blocks) for an integer percentage p, exactly. */
int64_t lpvo_keep_count(int64_t n_blocks, int sparsity_pct)
{
    if (n_blocks < 0 || sparsity_pct < 0 || sparsity_pct > 100)
        return -1;
    return ((100 - (int64_t)sparsity_pct) * n_blocks + 99) / 100;
}

/* Block i ranks before block j if its score is larger, or the scores are
 * equal and i is the lower row-major index. */
static const double* g_rank_scores;

static int rank_cmp(const void* a, const void* b)
{
    const int64_t i = *(const int64_t*)a, j = *(const int64_t*)b;
    const double si = g_rank_scores[i], sj = g_rank_scores[j];
    if (si > sj)
        return -1;
    if (si < sj)
        return 1;
    return i < j ? -1 : (i > j ? 1 : 0);
}

/* mask[i] = 1 for the n_keep best-ranked of n_blocks scores, 0 otherwise.
 * NaN scores are outside the contract (rejected).  Not thread-safe (qsort
 * comparator state). */
int lpvo_mask_topk(const double* scores, int64_t n_blocks, int64_t n_keep, uint8_t* mask)
{
    if (n_blocks < 0 || n_keep < 0 || n_keep > n_blocks || (n_blocks > 0 && (!scores || !mask)))
        return -1;
    for (int64_t i = 0; i < n_blocks; ++i)
        if (scores[i] != scores[i])
            return -1;
    int64_t* order = (int64_t*)malloc((size_t)(n_blocks > 0 ? n_blocks : 1) * sizeof(int64_t));
    if (!order)
        return -2;
    for (int64_t i = 0; i < n_blocks; ++i)
        order[i] = i;
    g_rank_scores = scores;
    qsort(order, (size_t)n_blocks, sizeof(int64_t), rank_cmp);
    memset(mask, 0, (size_t)n_blocks);
    for (int64_t i = 0; i < n_keep; ++i)
        mask[order[i]] = 1;
    free(order);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Backward of the block-sparse linear layer (finetuning, Sec. 3.1 / Fig. 1)  */
/* ------------------------------------------------------------------------ */

/*
 * After pruning, the paper finetunes the pruned model.  The block mask stays
 * fixed while finetuning: a dropped block is absent from the layer, so it
 * neither passes a gradient to the input nor receives one.  For the
 * pre-activation Z = X W~^T + b and its gradient G = dL/dZ (M x N; with the
 * GELU epilogue the caller first multiplies dL/dY by g'(Z) element-wise), the
 * chain rule gives, in float64:
 *   dX[m][k] = sum_{n=0}^{N-1} G[m][n] * W~[n][k]       (n ascending)
 *   dW[n][k] = sum_{m=0}^{M-1} G[m][n] * X[m][k]        (m ascending), only for
 *              (n, k) in a kept block, returned block by block in the BSR order
 *              of lpvo_pack (block-rows ascending, kept columns ascending, each
 *              block b_r rows of b_c values)
 *   db[n]    = sum_{m=0}^{M-1} G[m][n]                  (m ascending)
 */

struct gradx_job {
    int dtype;
    const void* G;
    int64_t ldg;
    int64_t m_begin, m_end;
    const double* Wd; /* [N][K]: the expanded, pruned weight */
    int64_t N, K;
    double* dX;
    int64_t lddx;
};

static void* gradx_rows(void* arg)
{
    struct gradx_job* j = (struct gradx_job*)arg;
    for (int64_t m = j->m_begin; m < j->m_end; ++m) {
        double* out = j->dX + m * j->lddx;
        for (int64_t k = 0; k < j->K; ++k)
            out[k] = 0.0;
        /* out[k] = sum over n ascending of G[m][n] * W~[n][k] */
        for (int64_t n = 0; n < j->N; ++n) {
            const double g = dec_one(j->dtype, j->G, m * j->ldg + n);
            const double* wn = j->Wd + n * j->K;
            for (int64_t k = 0; k < j->K; ++k)
                out[k] += g * wn[k];
        }
    }
    return NULL;
}

int lpvo_grad_x(int dtype, const void* G, int64_t ldg, int64_t M, const void* W, int64_t ldw,
                int64_t N, int64_t K, int b_r, int b_c, const uint8_t* mask, double* dX,
                int64_t lddx, int nthreads)
{
    if (!lpvo_elem_size(dtype) || !grid_ok(N, K, b_r, b_c) || M < 0 || ldg < N || ldw < K ||
        lddx < K || !mask || (M > 0 && (!G || !dX)) || (N * K > 0 && !W))
        return -1;
    if (M == 0 || K == 0)
        return 0;
    const int64_t C = K / b_c;
    double* Wd = (double*)malloc(sizeof(double) * (size_t)(N * K + 1));
    if (!Wd)
        return -2;
    for (int64_t n = 0; n < N; ++n)
        for (int64_t k = 0; k < K; ++k)
            Wd[n * K + k] = mask[(n / b_r) * C + (k / b_c)] ? dec_one(dtype, W, n * ldw + k) : 0.0;
    if (nthreads < 1)
        nthreads = 1;
    if (nthreads > M)
        nthreads = (int)M;
    struct gradx_job* jobs = (struct gradx_job*)calloc((size_t)nthreads, sizeof *jobs);
    pthread_t* tid = (pthread_t*)calloc((size_t)nthreads, sizeof *tid);
    char* running = (char*)calloc((size_t)nthreads, 1);
    int rc = 0;
    if (!jobs || !tid || !running) {
        rc = -2;
        goto out;
    }
    for (int t = 0; t < nthreads; ++t)
        jobs[t] = (struct gradx_job){dtype, G, ldg, M * t / nthreads, M * (t + 1) / nthreads,
                                     Wd, N, K, dX, lddx};
    for (int t = 1; t < nthreads; ++t)
        running[t] = pthread_create(&tid[t], NULL, gradx_rows, &jobs[t]) == 0;
    for (int t = 0; t < nthreads; ++t)
        if (!running[t])
            gradx_rows(&jobs[t]);
    for (int t = 1; t < nthreads; ++t)
        if (running[t])
            pthread_join(tid[t], NULL);
out:
    free(jobs);
    free(tid);
    free(running);
    free(Wd);
    return rc;
}

int64_t lpvo_grad_w(int dtype, const void* G, int64_t ldg, const void* X, int64_t ldx, int64_t M,
                    int64_t N, int64_t K, int b_r, int b_c, const uint8_t* mask, double* dW)
{
    if (!lpvo_elem_size(dtype) || !grid_ok(N, K, b_r, b_c) || M < 0 || ldg < N || ldx < K ||
        !mask || (M > 0 && (!G || !X)))
        return -1;
    const int64_t R = N / b_r, C = K / b_c;
    int64_t p = 0; /* kept blocks so far, in BSR order */
    double* g = (double*)malloc(sizeof(double) * (size_t)(b_r > 0 ? b_r : 1));
    double* x = (double*)malloc(sizeof(double) * (size_t)(b_c > 0 ? b_c : 1));
    if (!g || !x) {
        free(g);
        free(x);
        return -2;
    }
    for (int64_t r = 0; r < R; ++r) {
        for (int64_t c = 0; c < C; ++c) {
            if (!mask[r * C + c])
                continue;
            if (dW) {
                double* out = dW + p * b_r * b_c;
                for (int64_t e = 0; e < (int64_t)b_r * b_c; ++e)
                    out[e] = 0.0;
                /* every element: sum over m ascending of G[m][n] * X[m][k] */
                for (int64_t m = 0; m < M; ++m) {
                    for (int i = 0; i < b_r; ++i)
                        g[i] = dec_one(dtype, G, m * ldg + r * b_r + i);
                    for (int j = 0; j < b_c; ++j)
                        x[j] = dec_one(dtype, X, m * ldx + c * b_c + j);
                    for (int i = 0; i < b_r; ++i)
                        for (int j = 0; j < b_c; ++j)
                            out[i * b_c + j] += g[i] * x[j];
                }
            }
            ++p;
        }
    }
    free(g);
    free(x);
    return p;
}

int lpvo_grad_bias(int dtype, const void* G, int64_t ldg, int64_t M, int64_t N, double* db)
{
    if (!lpvo_elem_size(dtype) || M < 0 || N < 0 || ldg < N || (N > 0 && !db) ||
        (M > 0 && N > 0 && !G))
        return -1;
    for (int64_t n = 0; n < N; ++n) {
        double s = 0.0;
        for (int64_t m = 0; m < M; ++m)
            s += dec_one(dtype, G, m * ldg + n);
        db[n] = s;
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* The delta curve of a layer (Sec. 3.3, the empirical-Fisher Hessian)       */
/* ------------------------------------------------------------------------ */

/*
 * The paper collects, per layer, the second-order Taylor term of the output
 * distortion against the pruning ratio alpha:
 *   delta(alpha) = grad^T dW(alpha) + 1/2 dW(alpha)^T H dW(alpha),
 * with the Hessian approximated by the empirical Fisher over N calibration
 * samples, H = kappa I + (1/N) sum_n g_n g_n^T (g_n: the per-sample gradient of
 * the layer's weight, flattened).  dW(alpha) is the weight change of pruning at
 * ratio alpha: -W[e] for every element e of a dropped block, 0 elsewhere.  The
 * blocks dropped at a sparsity percentage p (alpha = p / 100) are those outside
 * the top ceil((100 - p) R C / 100) by the Sec. 3.1 score with the gradient
 * (mean |W grad| per block; ties to the lower index), exactly as
 * lpvo_block_scores + lpvo_keep_count + lpvo_mask_topk give them.
 *
 * This function is the direct definition at every requested percentage:
 *   delta = sum_e grad[e] dW[e]
 *         + 1/2 ( kappa sum_e dW[e]^2 + (1/N) sum_n (sum_e g_n[e] dW[e])^2 ),
 * each sum over e in row-major order, n ascending, in float64.
 */
int lpvo_delta_curve(int dtype, const void* W, int64_t ldw, int64_t N, int64_t K, int b_r, int b_c,
                     const void* grad, const void* samples, int64_t n_samples, double kappa,
                     const int32_t* pcts, int n_points, double* delta)
{
    if (!lpvo_elem_size(dtype) || !grid_ok(N, K, b_r, b_c) || ldw < K || !W || !grad ||
        n_samples < 0 || (n_samples > 0 && !samples) || n_points < 0 || (n_points > 0 && (!pcts || !delta)))
        return -1;
    for (int i = 0; i < n_points; ++i)
        if (pcts[i] < 0 || pcts[i] > 100)
            return -1;
    const int64_t R = N / b_r, C = K / b_c, nb = R * C, D = N * K;
    double* scores = (double*)malloc(sizeof(double) * (size_t)(nb + 1));
    uint8_t* mask = (uint8_t*)malloc((size_t)nb + 1);
    double* dw = (double*)malloc(sizeof(double) * (size_t)(D + 1));
    int rc = 0;
    if (!scores || !mask || !dw) {
        rc = -2;
        goto out;
    }
    /* the gradient is N x K with row stride K (grad) */
    if (lpvo_block_scores(dtype, W, ldw, grad, K, N, K, b_r, b_c, scores)) {
        rc = -1;
        goto out;
    }
    for (int i = 0; i < n_points; ++i) {
        const int64_t keep = lpvo_keep_count(nb, pcts[i]);
        rc = lpvo_mask_topk(scores, nb, keep, mask);
        if (rc)
            goto out;
        for (int64_t n = 0; n < N; ++n)
            for (int64_t k = 0; k < K; ++k)
                dw[n * K + k] = mask[(n / b_r) * C + (k / b_c)] ? 0.0 : -dec_one(dtype, W, n * ldw + k);
        double lin = 0.0, sq = 0.0, fisher = 0.0;
        for (int64_t e = 0; e < D; ++e) {
            lin += dec_one(dtype, grad, e) * dw[e];
            sq += dw[e] * dw[e];
        }
        for (int64_t s = 0; s < n_samples; ++s) {
            double p = 0.0;
            for (int64_t e = 0; e < D; ++e)
                p += dec_one(dtype, samples, s * D + e) * dw[e];
            fisher += p * p;
        }
        delta[i] = lin + 0.5 * (kappa * sq + (n_samples > 0 ? fisher / (double)n_samples : 0.0));
    }
out:
    free(scores);
    free(mask);
    free(dw);
    return rc;
}
