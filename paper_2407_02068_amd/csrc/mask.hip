// mask.hip -- the block mask of a weight on the GPU: block scores, then the
// top-k blocks (gfx950).
//
// Paper, Sec. 3.1: the blocks of a weight are ranked by the 2-D average pool
// of the first-order Taylor score |W * grad_W f| of their elements, and the
// bottom-ranked ones are dropped; Sec. 3.4: ceil((1 - alpha) R C) blocks
// survive.  Without a gradient the score is the block's sum of squares (it
// ranks like the block's L2 norm).
//
// A score is an integer-deciding quantity (it picks the kept set), so it is
// computed exactly as specified: in float64, the block's elements row by row,
// one addition after the other, with no contraction into fused multiply-adds.
// Every product of two decoded elements is exact in float64 and the average's
// divisor is a power of two, so the value depends only on that order.
//
// Scores are non-negative (+0.0 at least), so their IEEE bit patterns order
// like their values; the selection works on those 64-bit keys.
#include "lpv_device.h"
#include "lpv_internal.h"

namespace lpv {
namespace {

template <int DT> __device__ inline double load_f64(const char* base, int64_t idx)
{
    if (DT == LPV_F32)
        return (double)((const float*)base)[idx];
    const uint16_t bits = ((const uint16_t*)base)[idx];
    if (DT == LPV_BF16)
        return (double)__uint_as_float((uint32_t)bits << 16);
    return (double)(float)__builtin_bit_cast(_Float16, bits);
}

// 8 consecutive elements (16-byte aligned) decoded to float64, from 16-byte loads.
template <int DT> __device__ inline void load8_f64(const char* base, int64_t idx, double* out)
{
    if (DT == LPV_F32) {
        const float4 a = *(const float4*)(base + idx * 4), b = *(const float4*)(base + idx * 4 + 16);
        out[0] = a.x, out[1] = a.y, out[2] = a.z, out[3] = a.w;
        out[4] = b.x, out[5] = b.y, out[6] = b.z, out[7] = b.w;
    } else {
        const uint4 u = *(const uint4*)(base + idx * 2);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint16_t lo = (uint16_t)(w[j] & 0xffffu), hi = (uint16_t)(w[j] >> 16);
            if (DT == LPV_BF16) {
                out[2 * j] = (double)__uint_as_float((uint32_t)lo << 16);
                out[2 * j + 1] = (double)__uint_as_float((uint32_t)hi << 16);
            } else {
                out[2 * j] = (double)(float)__builtin_bit_cast(_Float16, lo);
                out[2 * j + 1] = (double)(float)__builtin_bit_cast(_Float16, hi);
            }
        }
    }
}

// One thread per block (r, c) = blockIdx.x * 256 + threadIdx.x (row-major).
// VEC: the block's rows are read 16 bytes at a time (W and G 16-byte aligned,
// row strides multiples of 16 bytes); the elements are still added one after
// the other in row-major order, so the score is the same bit for bit.
template <int DT, bool TAYLOR, bool VEC>
__global__ __launch_bounds__(256) void k_block_scores(const char* __restrict__ W, int64_t ldw,
                                                      const char* __restrict__ G, int64_t ldg,
                                                      int64_t R, int64_t C, int32_t b_r,
                                                      int32_t b_c, double* __restrict__ scores)
{
#pragma clang fp contract(off)
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= R * C)
        return;
    const int64_t r = i / C, c = i - r * C;
    double s = 0.0;
    for (int32_t a = 0; a < b_r; ++a) {
        const int64_t n = r * b_r + a;
        if (VEC) {
            for (int32_t b = 0; b < b_c; b += 8) {
                const int64_t k = c * b_c + b;
                double w[8], g[8];
                load8_f64<DT>(W, n * ldw + k, w);
                if (TAYLOR)
                    load8_f64<DT>(G, n * ldg + k, g);
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    if (TAYLOR) {
                        const double p = w[j] * g[j];
                        s = s + (p < 0.0 ? -p : p);
                    } else {
                        s = s + w[j] * w[j];
                    }
                }
            }
        } else {
            for (int32_t b = 0; b < b_c; ++b) {
                const int64_t k = c * b_c + b;
                const double w = load_f64<DT>(W, n * ldw + k);
                if (TAYLOR) {
                    const double p = w * load_f64<DT>(G, n * ldg + k);
                    s = s + (p < 0.0 ? -p : p);
                } else {
                    s = s + w * w;
                }
            }
        }
    }
    scores[i] = TAYLOR ? s / (double)(b_r * b_c) : s;
}

constexpr int SEL_THREADS = 1024;

__device__ inline uint64_t key_of(double v) { return (uint64_t)__double_as_longlong(v); }

// Block-wide sum of one value per thread (all threads call it).
__device__ inline int64_t block_sum(int64_t v, int64_t* s_part)
{
    for (int o = 32; o > 0; o >>= 1)
        v += __shfl_xor(v, o, 64);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    __syncthreads();
    if (lane == 0)
        s_part[wave] = v;
    __syncthreads();
    int64_t t = 0;
    for (int w = 0; w < SEL_THREADS / 64; ++w)
        t += s_part[w];
    return t;
}

// One workgroup: mask[i] = 1 for the n_keep best-ranked scores (larger first,
// equal scores by lower index).  T, the n_keep-th largest key, is found bit by
// bit from the top: the largest T with at least n_keep keys >= T.  Then every
// key > T is kept, and of the keys == T the (n_keep - #keys > T) lowest indices.
__global__ __launch_bounds__(SEL_THREADS) void k_mask_topk(const double* __restrict__ scores,
                                                           int64_t n, int64_t n_keep,
                                                           uint8_t* __restrict__ mask)
{
    __shared__ int64_t s_part[SEL_THREADS / 64];
    __shared__ int64_t s_scan[SEL_THREADS];
    const int tid = threadIdx.x;
    if (n_keep <= 0) {
        for (int64_t i = tid; i < n; i += SEL_THREADS)
            mask[i] = 0;
        return;
    }
    uint64_t T = 0;
    for (int bit = 63; bit >= 0; --bit) {
        const uint64_t cand = T | ((uint64_t)1 << bit);
        int64_t cnt = 0;
        for (int64_t i = tid; i < n; i += SEL_THREADS)
            cnt += key_of(scores[i]) >= cand;
        if (block_sum(cnt, s_part) >= n_keep)
            T = cand;
    }
    int64_t above = 0;
    for (int64_t i = tid; i < n; i += SEL_THREADS)
        above += key_of(scores[i]) > T;
    const int64_t need = n_keep - block_sum(above, s_part);  // >= 1 keys equal to T
    // ties in index order: chunks of SEL_THREADS, inclusive scan of the flags
    int64_t taken = 0;
    for (int64_t base = 0; base < n; base += SEL_THREADS) {
        const int64_t i = base + tid;
        const uint64_t k = i < n ? key_of(scores[i]) : 0;
        const int tie = i < n && k == T;
        __syncthreads();
        s_scan[tid] = tie;
        __syncthreads();
        for (int o = 1; o < SEL_THREADS; o <<= 1) {
            const int64_t v = tid >= o ? s_scan[tid - o] : 0;
            __syncthreads();
            s_scan[tid] += v;
            __syncthreads();
        }
        if (i < n)
            mask[i] = k > T || (tie && taken + s_scan[tid] <= need);
        taken += s_scan[SEL_THREADS - 1];
    }
}

}  // namespace

hipError_t launch_block_scores(const MaskCall& m, hipStream_t s)
{
    const int64_t R = m.N / m.b_r, C = m.K / m.b_c, nb = R * C;
    if (nb > 0) {
        const dim3 grid((unsigned)((nb + 255) / 256)), block(256);
        const int es = m.dtype == LPV_F32 ? 4 : 2;
        const bool vec = ((uintptr_t)m.W % 16) == 0 && (m.ldw * es) % 16 == 0 &&
                         (!m.G || (((uintptr_t)m.G % 16) == 0 && (m.ldg * es) % 16 == 0));
#define LPV_SCORES(DT_, TY_, V_)                                                                   \
    hipLaunchKernelGGL((k_block_scores<DT_, TY_, V_>), grid, block, 0, s, (const char*)m.W, m.ldw, \
                       (const char*)m.G, m.ldg, R, C, m.b_r, m.b_c, m.scores)
#define LPV_SCORES_DT(DT_)                   \
    do {                                     \
        if (m.G && vec)                      \
            LPV_SCORES(DT_, true, true);     \
        else if (m.G)                        \
            LPV_SCORES(DT_, true, false);    \
        else if (vec)                        \
            LPV_SCORES(DT_, false, true);    \
        else                                 \
            LPV_SCORES(DT_, false, false);   \
    } while (0)
        if (m.dtype == LPV_BF16)
            LPV_SCORES_DT(LPV_BF16);
        else if (m.dtype == LPV_F16)
            LPV_SCORES_DT(LPV_F16);
        else
            LPV_SCORES_DT(LPV_F32);
#undef LPV_SCORES_DT
#undef LPV_SCORES
    }
    return hipGetLastError();
}

hipError_t launch_mask_topk(const MaskCall& m, hipStream_t s)
{
    const int64_t nb = (m.N / m.b_r) * (m.K / m.b_c);
    const hipError_t e = launch_block_scores(m, s);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_mask_topk, dim3(1), dim3(SEL_THREADS), 0, s, (const double*)m.scores, nb,
                       m.n_keep, m.mask);
    return hipGetLastError();
}

}  // namespace lpv
