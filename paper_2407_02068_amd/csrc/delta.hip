// delta.hip -- the delta curve of a layer on the GPU (gfx950).
//
// Paper, Sec. 3.3 (empirical complexity): the second-order Taylor term of the
// output distortion when a layer is pruned at ratio alpha,
//   delta(alpha) = grad^T dW(alpha) + 1/2 dW(alpha)^T H dW(alpha),
// with the empirical Fisher H = kappa I + (1/N) sum_n g_n g_n^T.  As alpha
// rises, the dropped blocks grow by a set d (blocks ranked by the Sec. 3.1
// Taylor score, lowest first), and the paper's update is
//   delta_k - delta_{k-1} = grad' . d + (d/2 + dW_{k-1})^T H' d.
// Blocks are disjoint, so with b_n = g_n . d and a_n = g_n . dW_{k-1} this is
//   grad . d + kappa |d|^2 / 2 + (1/N) sum_n (b_n / 2 + a_n) b_n,
// and a_n grows by b_n.  Everything reduces to dot products of each vector
// (per-sample gradients, grad, and W itself for |d|^2) with -W over every
// block: one pass over the per-sample gradients, which bounds the time (HBM).
//
//   k_block_rank   rank of each block by (-score, index) and its inverse
//   k_delta_dots   float64 block dot products, one workgroup per (block-row,
//                  vector)
//   k_delta_curve  one workgroup: the ratio steps in rank order, the update
// All sums run in a fixed order (float64), so results do not depend on timing.
#include "lpv_device.h"
#include "lpv_internal.h"

namespace lpv {
namespace {

// rank[b] = #{b' : score(b') > score(b), or equal and b' < b}; perm[rank[b]] = b.
// Scores are non-negative, so their bit patterns order like their values.
// One thread per block, the keys staged through LDS 1024 at a time.
__global__ __launch_bounds__(256) void k_block_rank(const double* __restrict__ scores, int64_t nb,
                                                    int32_t* __restrict__ perm)
{
    __shared__ uint64_t s_key[1024];
    const int64_t b = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const uint64_t key = b < nb ? (uint64_t)__double_as_longlong(scores[b]) : 0;
    int64_t rank = 0;
    for (int64_t base = 0; base < nb; base += 1024) {
        __syncthreads();
        for (int i = threadIdx.x; i < 1024; i += 256)
            s_key[i] = base + i < nb ? (uint64_t)__double_as_longlong(scores[base + i]) : 0;
        __syncthreads();
        const int n = (int)min((int64_t)1024, nb - base);
        for (int i = 0; i < n; ++i) {
            const uint64_t k2 = s_key[i];
            rank += (k2 > key) || (k2 == key && base + i < b);
        }
    }
    if (b < nb)
        perm[rank] = (int32_t)b;
}

// The 8 elements at idx .. idx + 7 (idx a multiple of 8, 16-byte aligned) in
// float64, from 16-byte loads.
template <int DT> __device__ inline void load8(const char* base, int64_t idx, double* out)
{
    if constexpr (DT == LPV_F32) {
        const float4 a = *(const float4*)(base + idx * 4), b = *(const float4*)(base + idx * 4 + 16);
        out[0] = a.x, out[1] = a.y, out[2] = a.z, out[3] = a.w;
        out[4] = b.x, out[5] = b.y, out[6] = b.z, out[7] = b.w;
    } else {
        const uint4 u = *(const uint4*)(base + idx * 2);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            out[2 * i] = (double)Elem<DT>::to_f32((uint16_t)(w[i] & 0xffffu));
            out[2 * i + 1] = (double)Elem<DT>::to_f32((uint16_t)(w[i] >> 16));
        }
    }
}

// dots[v][r C + c] = sum over block (r, c) of x_v[e] * (-W[e]), float64:
// x_v = sample v (v < n_samples), grad (v = n_samples), W (v = n_samples + 1).
// Workgroup (block-row r, vector v).  The block-row's 8-element column chunks
// (nch = K / 8) are spread over the threads; when nch < 256 the rows are split
// into G = 256 / nch interleaved groups as well.  Thread (g, q) sums chunk q
// over rows g, g + G, ... (ascending); a block's sum then adds its chunks' sums
// group by group, in column order.
template <int DT>
__global__ __launch_bounds__(256) void k_delta_dots(const DeltaCall c, int32_t C,
                                                    double* __restrict__ dots)
{
    extern __shared__ double s_part[];  // G x nch chunk sums
    constexpr int ES = DT == LPV_F32 ? 4 : 2;
    const int r = blockIdx.x;
    const int64_t v = blockIdx.y;
    const char* x;
    int64_t ldx;
    if (v < c.n_samples) {
        x = (const char*)c.samples + v * c.stride * ES;
        ldx = c.lds;
    } else if (v == c.n_samples) {
        x = (const char*)c.grad;
        ldx = c.ldg;
    } else {
        x = (const char*)c.W;
        ldx = c.ldw;
    }
    const char* w = (const char*)c.W;
    const int nch = (int)(c.K / 8);
    const int G = nch >= 256 ? 1 : 256 / nch;
    for (int t = threadIdx.x; t < G * nch; t += 256) {
        const int g = t / nch, q = t - g * nch;
        double acc = 0.0;
#pragma unroll 4
        for (int i = g; i < c.b_r; i += G) {
            const int64_t row = (int64_t)r * c.b_r + i;
            double xv[8], wv[8];
            load8<DT>(x, row * ldx + (int64_t)q * 8, xv);
            load8<DT>(w, row * c.ldw + (int64_t)q * 8, wv);
#pragma unroll
            for (int j = 0; j < 8; ++j)
                acc += xv[j] * -wv[j];
        }
        s_part[t] = acc;
    }
    __syncthreads();
    const int per = c.b_c / 8;
    for (int cc = threadIdx.x; cc < C; cc += 256) {
        double s = 0.0;
        for (int g = 0; g < G; ++g)
            for (int q = 0; q < per; ++q)
                s += s_part[g * nch + cc * per + q];
        dots[v * ((int64_t)(c.N / c.b_r) * C) + (int64_t)r * C + cc] = s;
    }
}

// One workgroup.  Step k of the curve drops the blocks of rank
// [keep[k], keep[k - 1]) (keep[-1] = all blocks), in rank order.  Thread v
// (a vector) walks the steps: its step sum B_k; samples keep a_v and write
// (B_k / 2 + a_v) B_k, grad and W their step sums.  Then thread 0 adds, step by
// step, grad . d + kappa |d|^2 / 2 + (1/N) sum_v (in order) of the samples'
// terms.
__global__ __launch_bounds__(1024) void k_delta_curve(const DeltaCall c, int64_t nb,
                                                      const double* __restrict__ dots,
                                                      const int32_t* __restrict__ perm,
                                                      double* __restrict__ q)
{
    const int64_t nv = c.n_samples + 2;
    for (int64_t v = threadIdx.x; v < nv; v += 1024) {
        const double* dv = dots + v * nb;
        double a = 0.0;
        int64_t hi = nb;
        for (int k = 0; k < c.n_points; ++k) {
            const int64_t lo = c.keep[k];
            double bsum = 0.0;
            for (int64_t rk = lo; rk < hi; ++rk)
                bsum += dv[perm[rk]];
            hi = lo;
            if (v < c.n_samples) {
                q[(int64_t)k * nv + v] = (0.5 * bsum + a) * bsum;
                a += bsum;
            } else {
                q[(int64_t)k * nv + v] = bsum;
            }
        }
    }
    __syncthreads();  // the step terms in q are visible to thread 0
    if (threadIdx.x == 0) {
        double delta = 0.0;
        for (int k = 0; k < c.n_points; ++k) {
            const double* qk = q + (int64_t)k * nv;
            double f = 0.0;
            for (int64_t v = 0; v < c.n_samples; ++v)
                f += qk[v];
            // grad . d, then |d|^2 = -(W . (-W)) over the step
            const double lin = qk[c.n_samples], sq = -qk[c.n_samples + 1];
            delta += lin + 0.5 * c.kappa * sq + (c.n_samples > 0 ? f / (double)c.n_samples : 0.0);
            c.delta[k] = delta;
        }
    }
}

}  // namespace

hipError_t launch_delta_curve(const DeltaCall& c, hipStream_t s)
{
    const int32_t R = (int32_t)(c.N / c.b_r), C = (int32_t)(c.K / c.b_c);
    const int64_t nb = (int64_t)R * C, nv = c.n_samples + 2;
    // workspace: scores (nb), dots (nv x nb), step terms (points x nv), perm (nb)
    const size_t bytes = (size_t)(nb + nv * nb + (int64_t)c.n_points * nv) * sizeof(double) +
                         (size_t)nb * sizeof(int32_t);
    char* ws = nullptr;
    hipError_t e = hipMallocAsync((void**)&ws, bytes, s);
    if (e != hipSuccess)
        return e;
    double* scores = (double*)ws;
    double* dots = scores + nb;
    double* q = dots + nv * nb;
    int32_t* perm = (int32_t*)(q + (int64_t)c.n_points * nv);
    MaskCall m = {c.W, c.ldw, c.grad, c.ldg, c.N, c.K, c.dtype, c.b_r, c.b_c, 0, nullptr, scores};
    e = launch_block_scores(m, s);
    if (e == hipSuccess) {
        hipLaunchKernelGGL(k_block_rank, dim3((unsigned)((nb + 255) / 256)), dim3(256), 0, s,
                           (const double*)scores, nb, perm);
        e = hipGetLastError();
    }
    if (e == hipSuccess) {
        const dim3 grid((unsigned)R, (unsigned)nv);
        const int64_t nch = c.K / 8;
        const size_t lds = (size_t)(nch >= 256 ? nch : 256 / nch * nch) * sizeof(double);
        if (c.dtype == LPV_BF16)
            hipLaunchKernelGGL(k_delta_dots<LPV_BF16>, grid, dim3(256), lds, s, c, C, dots);
        else if (c.dtype == LPV_F16)
            hipLaunchKernelGGL(k_delta_dots<LPV_F16>, grid, dim3(256), lds, s, c, C, dots);
        else
            hipLaunchKernelGGL(k_delta_dots<LPV_F32>, grid, dim3(256), lds, s, c, C, dots);
        e = hipGetLastError();
    }
    if (e == hipSuccess) {
        hipLaunchKernelGGL(k_delta_curve, dim3(1), dim3(1024), 0, s, c, nb, (const double*)dots,
                           (const int32_t*)perm, q);
        e = hipGetLastError();
    }
    const hipError_t ef = hipFreeAsync(ws, s);
    return e != hipSuccess ? e : ef;
}

}  // namespace lpv
