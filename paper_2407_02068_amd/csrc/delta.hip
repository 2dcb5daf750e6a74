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
//   k_rank         rank of each block by (-score, index) and its inverse
//   k_delta_dots   float64 block dot products, one workgroup per (block-row,
//                  vector)
//   k_delta_steps  each vector's sum over each ratio step's blocks
//   k_delta_finish one workgroup: the update, step by step
// All sums run in a fixed order (float64), so results do not depend on timing.
#include "lpv_device.h"
#include "lpv_internal.h"

namespace lpv {
namespace {

// rank[b] = #{b' : score(b') > score(b), or equal and b' < b}; perm[rank[b]] = b.
// Scores are non-negative, so their bit patterns order like their values.
// Workgroup: 64 blocks (lane l: block 64 x + l) times RANK_WAVES waves; wave w
// counts the keys ahead of its lane's block in the w-th part of the key range
// (each key read once per wave, a wave-uniform load); the parts' integer
// counts are added in LDS (exact in any order) and the permutation written.
constexpr int RANK_WAVES = 16;

__global__ __launch_bounds__(64 * RANK_WAVES) void k_rank(const double* __restrict__ scores,
                                                          int64_t nb, int32_t* __restrict__ perm)
{
    __shared__ int32_t s_cnt[RANK_WAVES][64];
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int64_t b = (int64_t)blockIdx.x * 64 + lane;
    const uint64_t* keys = (const uint64_t*)scores;
    const uint64_t key = keys[min(b, nb - 1)];
    const int64_t per = (nb + RANK_WAVES - 1) / RANK_WAVES;
    const int64_t k0 = min(nb, (int64_t)w * per), k1 = min(nb, k0 + per);
    int32_t r = 0;
#pragma unroll 8
    for (int64_t i = k0; i < k1; ++i) {
        const uint64_t k2 = keys[i];
        r += (k2 > key) || (k2 == key && i < b);
    }
    s_cnt[w][lane] = r;
    __syncthreads();
    if (w == 0 && b < nb) {
        int32_t rank = 0;
#pragma unroll
        for (int j = 0; j < RANK_WAVES; ++j)
            rank += s_cnt[j][lane];
        perm[rank] = (int32_t)b;
    }
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
// Workgroup (block-row r, vectors VPW y .. VPW y + VPW - 1): each W chunk is
// loaded once for its VPW vectors.  The block-row's 8-element column chunks
// (nch = K / 8) are spread over the threads; when nch < 256 the rows are split
// into G = 256 / nch interleaved groups as well.  Thread (g, q) sums chunk q
// over rows g, g + G, ... (ascending); a block's sum then adds its chunks' sums
// group by group, in column order.
template <int DT, int VPW>
__global__ __launch_bounds__(256) void k_delta_dots(const DeltaCall c, int32_t C,
                                                    double* __restrict__ dots)
{
    extern __shared__ double s_part[];  // VPW x G x nch chunk sums
    constexpr int ES = DT == LPV_F32 ? 4 : 2;
    const int r = blockIdx.x;
    const int64_t nv = c.n_samples + 2, v0 = (int64_t)blockIdx.y * VPW;
    const int nvv = (int)min((int64_t)VPW, nv - v0);
    const char* xs[VPW];
    int64_t lx[VPW];
#pragma unroll
    for (int u = 0; u < VPW; ++u) {
        const int64_t v = min(v0 + u, nv - 1);
        if (v < c.n_samples) {
            xs[u] = (const char*)c.samples + v * c.stride * ES;
            lx[u] = c.lds;
        } else if (v == c.n_samples) {
            xs[u] = (const char*)c.grad;
            lx[u] = c.ldg;
        } else {
            xs[u] = (const char*)c.W;
            lx[u] = c.ldw;
        }
    }
    const char* w = (const char*)c.W;
    const int nch = (int)(c.K / 8);
    const int G = nch >= 256 ? 1 : 256 / nch;
    for (int t = threadIdx.x; t < G * nch; t += 256) {
        const int g = t / nch, q = t - g * nch;
        double acc[VPW];
#pragma unroll
        for (int u = 0; u < VPW; ++u)
            acc[u] = 0.0;
#pragma unroll 2
        for (int i = g; i < c.b_r; i += G) {
            const int64_t row = (int64_t)r * c.b_r + i;
            double wv[8];
            load8<DT>(w, row * c.ldw + (int64_t)q * 8, wv);
#pragma unroll
            for (int u = 0; u < VPW; ++u) {
                if (u < nvv) {
                    double xv[8];
                    load8<DT>(xs[u], row * lx[u] + (int64_t)q * 8, xv);
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        acc[u] += xv[j] * -wv[j];
                }
            }
        }
#pragma unroll
        for (int u = 0; u < VPW; ++u)
            s_part[u * G * nch + t] = acc[u];
    }
    __syncthreads();
    const int per = c.b_c / 8;
    for (int i = threadIdx.x; i < nvv * C; i += 256) {
        const int u = i / C, cc = i - u * C;
        const double* sp = s_part + u * G * nch;
        double s = 0.0;
        for (int g = 0; g < G; ++g)
            for (int q = 0; q < per; ++q)
                s += sp[g * nch + cc * per + q];
        dots[(v0 + u) * ((int64_t)(c.N / c.b_r) * C) + (int64_t)r * C + cc] = s;
    }
}

// Step sums: step k drops the blocks of rank [keep[k], keep[k - 1])
// (keep[-1] = all blocks).  One wave per (vector v, step k): lane l adds the
// step's blocks of rank lo + l, lo + l + 64, ... in order, then a fixed
// butterfly adds the lanes.  bsum[k][v] = the step's sum of dots[v].
__global__ __launch_bounds__(256) void k_delta_steps(const DeltaCall c, int64_t nb,
                                                     const double* __restrict__ dots,
                                                     const int32_t* __restrict__ perm,
                                                     double* __restrict__ bsum)
{
    const int64_t nv = c.n_samples + 2;
    const int64_t idx = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (idx >= nv * c.n_points)
        return;  // whole waves
    const int lane = threadIdx.x & 63;
    const int64_t v = idx / c.n_points;
    const int k = (int)(idx - v * c.n_points);
    const int64_t lo = c.keep[k], hi = k > 0 ? c.keep[k - 1] : nb;
    const double* dv = dots + v * nb;
    double s = 0.0;
    for (int64_t rk = lo + lane; rk < hi; rk += 64)
        s += dv[perm[rk]];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        s += __shfl_xor(s, o, 64);
    if (lane == 0)
        bsum[(int64_t)k * nv + v] = s;
}

// One workgroup.  Sample v keeps a_v = g_v . dW_{k-1} and turns its step sums
// into (B_k / 2 + a_v) B_k (in place); then thread k adds the samples' terms
// in order; thread 0 adds, step by step, grad . d + kappa |d|^2 / 2 +
// (1/N) sum_v (...).  STAGED: the step sums and the step terms sit in LDS (one
// coalesced load first), so none of the serial loops waits on global memory.
template <bool STAGED>
__global__ __launch_bounds__(1024) void k_delta_finish(const DeltaCall c, double* __restrict__ bsum,
                                                       double* __restrict__ term)
{
    extern __shared__ double s_fin[];  // STAGED: step sums (n_points x nv), step terms
    const int64_t nv = c.n_samples + 2;
    double* q = bsum;
    double* tk = term;
    if (STAGED) {
        const int64_t n = (int64_t)c.n_points * nv;
        for (int64_t i = threadIdx.x; i < n; i += 1024)
            s_fin[i] = bsum[i];
        __syncthreads();
        q = s_fin;
        tk = s_fin + n;
    }
    // (the loads of each loop are independent of its running sums: unrolled,
    // they are issued ahead of the additions)
    for (int64_t v = threadIdx.x; v < c.n_samples; v += 1024) {
        double a = 0.0;
#pragma unroll 8
        for (int k = 0; k < c.n_points; ++k) {
            const double b = q[(int64_t)k * nv + v];
            q[(int64_t)k * nv + v] = (0.5 * b + a) * b;
            a += b;
        }
    }
    __syncthreads();
    for (int k = threadIdx.x; k < c.n_points; k += 1024) {
        const double* qk = q + (int64_t)k * nv;
        double f = 0.0;
#pragma unroll 16
        for (int64_t v = 0; v < c.n_samples; ++v)
            f += qk[v];
        // grad . d, and |d|^2 = -(W . (-W)) over the step
        tk[k] = qk[c.n_samples] + 0.5 * c.kappa * -qk[c.n_samples + 1] +
                (c.n_samples > 0 ? f / (double)c.n_samples : 0.0);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double delta = 0.0;
        for (int k = 0; k < c.n_points; ++k) {
            delta += tk[k];
            c.delta[k] = delta;
        }
    }
}

}  // namespace

size_t delta_workspace_bytes(int64_t N, int64_t K, int32_t b_r, int32_t b_c, int64_t n_samples,
                             int32_t n_points)
{
    const int64_t nb = (N / b_r) * (K / b_c), nv = n_samples + 2;
    // scores (nb), dots (nv x nb), step sums (points x nv), step terms
    // (points), perm (nb)
    return (size_t)(nb + nv * nb + (int64_t)n_points * nv + n_points) * sizeof(double) +
           (size_t)nb * sizeof(int32_t);
}

hipError_t launch_delta_curve(const DeltaCall& c, hipStream_t s)
{
    const int32_t R = (int32_t)(c.N / c.b_r), C = (int32_t)(c.K / c.b_c);
    const int64_t nb = (int64_t)R * C, nv = c.n_samples + 2;
    const size_t bytes = delta_workspace_bytes(c.N, c.K, c.b_r, c.b_c, c.n_samples, c.n_points);
    // the caller's workspace, else one allocated (and freed) on the stream
    char* ws = (char*)c.ws;
    const bool own = ws == nullptr;
    hipError_t e = hipSuccess;
    if (own) {
        e = hipMallocAsync((void**)&ws, bytes, s);
        if (e != hipSuccess)
            return e;
    } else if (c.ws_bytes < bytes) {
        return hipErrorInvalidValue;
    }
    double* scores = (double*)ws;
    double* dots = scores + nb;
    double* q = dots + nv * nb;
    double* term = q + (int64_t)c.n_points * nv;
    int32_t* perm = (int32_t*)(term + c.n_points);
    MaskCall m = {c.W, c.ldw, c.grad, c.ldg, c.N, c.K, c.dtype, c.b_r, c.b_c, 0, nullptr, scores};
    e = launch_block_scores(m, s);
    if (e == hipSuccess) {
        hipLaunchKernelGGL(k_rank, dim3((unsigned)((nb + 63) / 64)), dim3(64 * RANK_WAVES), 0, s,
                           (const double*)scores, nb, perm);
        e = hipGetLastError();
    }
    if (e == hipSuccess) {
        const int64_t nch = c.K / 8;
        const int64_t part = (nch >= 256 ? nch : 256 / nch * nch) * (int64_t)sizeof(double);
        // vectors per workgroup: 4 while their chunk sums fit 64 KB of LDS
        const int vpw = part * 4 <= 65536 ? 4 : 1;
        const dim3 grid((unsigned)R, (unsigned)((nv + vpw - 1) / vpw));
        const size_t lds = (size_t)(part * vpw);
#define LPV_DOTS(DT_)                                                                         \
    do {                                                                                      \
        if (vpw == 4)                                                                         \
            hipLaunchKernelGGL((k_delta_dots<DT_, 4>), grid, dim3(256), lds, s, c, C, dots); \
        else                                                                                  \
            hipLaunchKernelGGL((k_delta_dots<DT_, 1>), grid, dim3(256), lds, s, c, C, dots); \
    } while (0)
        if (c.dtype == LPV_BF16)
            LPV_DOTS(LPV_BF16);
        else if (c.dtype == LPV_F16)
            LPV_DOTS(LPV_F16);
        else
            LPV_DOTS(LPV_F32);
#undef LPV_DOTS
        e = hipGetLastError();
    }
    if (e == hipSuccess) {
        const int64_t waves = nv * c.n_points;
        hipLaunchKernelGGL(k_delta_steps, dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s, c, nb,
                           (const double*)dots, (const int32_t*)perm, q);
        e = hipGetLastError();
        if (e == hipSuccess) {
            const size_t fin = (size_t)((int64_t)c.n_points * nv + c.n_points) * sizeof(double);
            if (fin <= 65536)
                hipLaunchKernelGGL(k_delta_finish<true>, dim3(1), dim3(1024), fin, s, c, q, term);
            else
                hipLaunchKernelGGL(k_delta_finish<false>, dim3(1), dim3(1024), 0, s, c, q, term);
            e = hipGetLastError();
        }
    }
    const hipError_t ef = own ? hipFreeAsync(ws, s) : hipSuccess;
    return e != hipSuccess ? e : ef;
}

}  // namespace lpv
