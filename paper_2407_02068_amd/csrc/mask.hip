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

// The same scores with the loads taken off the additions' path: a workgroup
// takes NB consecutive blocks of one block row; all its threads load them
// with 16-byte reads and write every element's term (|w g| or w w, exact in
// float64) to LDS; then thread j adds up block j's terms from LDS, one after
// the other in the same row-major order (the same value bit for bit).  A
// block's terms sit at a stride of its size plus 16 bytes, so the adding
// threads' 16-byte reads fall in distinct banks.
constexpr int SC_THREADS = 256;
constexpr int SC_LDS = 131072;  // bytes of float64 terms per workgroup

template <int DT, bool TAYLOR>
__global__ __launch_bounds__(SC_THREADS) void k_block_scores_lds(const char* __restrict__ W,
                                                                 int64_t ldw,
                                                                 const char* __restrict__ G,
                                                                 int64_t ldg, int64_t C,
                                                                 int32_t b_r, int32_t b_c,
                                                                 int32_t nb,
                                                                 double* __restrict__ scores)
{
#pragma clang fp contract(off)
    // at most SC_LDS bytes of terms and 16 bytes of padding per block
    // (blocks of at least 256 elements: at most SC_LDS / 2048 blocks)
    __shared__ double2 terms[(SC_LDS + 16 * (SC_LDS / 2048)) / 16];
    const int64_t n_chunks = (C + nb - 1) / nb;
    const int64_t r = blockIdx.x / n_chunks, c0 = (blockIdx.x - r * n_chunks) * nb;
    const int nbk = (int)min((int64_t)nb, C - c0);  // blocks of this workgroup
    const int n_el = b_r * b_c;
    const int stride = n_el / 2 + 1;                  // double2 units per block
    const int u_row = b_c / 8;                        // 8-element units per block row
    const int units = nbk * b_r * u_row;
    for (int i = threadIdx.x; i < units; i += SC_THREADS) {
        const int q = i % u_row, t = i / u_row, j = t % nbk, a = t / nbk;
        const int64_t n = r * b_r + a, k = (c0 + j) * b_c + 8 * q;
        double w[8], g[8];
        load8_f64<DT>(W, n * ldw + k, w);
        if (TAYLOR)
            load8_f64<DT>(G, n * ldg + k, g);
        double2* dst = terms + j * stride + (a * b_c + 8 * q) / 2;
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
            double t0, t1;
            if (TAYLOR) {
                const double p0 = w[e] * g[e], p1 = w[e + 1] * g[e + 1];
                t0 = p0 < 0.0 ? -p0 : p0;
                t1 = p1 < 0.0 ? -p1 : p1;
            } else {
                t0 = w[e] * w[e];
                t1 = w[e + 1] * w[e + 1];
            }
            dst[e / 2] = double2{t0, t1};
        }
    }
    __syncthreads();
    const int j = threadIdx.x;
    if (j >= nbk)
        return;
    const double2* src = terms + j * stride;
    double s = 0.0;
    for (int e = 0; e < n_el / 2; e += 4) {  // n_el is a multiple of 8
        const double2 v0 = src[e], v1 = src[e + 1], v2 = src[e + 2], v3 = src[e + 3];
        s = s + v0.x;
        s = s + v0.y;
        s = s + v1.x;
        s = s + v1.y;
        s = s + v2.x;
        s = s + v2.y;
        s = s + v3.x;
        s = s + v3.y;
    }
    scores[r * C + c0 + j] = TAYLOR ? s / (double)n_el : s;
}

constexpr int SEL_THREADS = 1024;

__device__ inline uint64_t key_of(double v) { return (uint64_t)__double_as_longlong(v); }

// One workgroup: mask[i] = 1 for the n_keep best-ranked scores (larger first,
// equal scores by lower index).  T, the n_keep-th largest key, is found one
// byte at a time from the top (a radix select): among the keys that match the
// bytes found so far, an LDS histogram of the next byte gives the byte of T
// and how many keys above it drop out.  Then every key > T is kept, and of the
// keys == T the (n_keep - #keys > T) lowest indices (wave ballots give each
// tie its rank in index order).  Up to SEL_REG keys per thread stay in
// registers; more are read again from global memory in every pass.
constexpr int SEL_REG = 8;

__global__ __launch_bounds__(SEL_THREADS) void k_mask_topk(const double* __restrict__ scores,
                                                           int64_t n, int64_t n_keep,
                                                           uint8_t* __restrict__ mask)
{
    __shared__ int64_t s_part[SEL_THREADS / 64];
    __shared__ uint32_t s_hist[256];
    __shared__ uint32_t s_sel[2];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (n_keep <= 0) {
        for (int64_t i = tid; i < n; i += SEL_THREADS)
            mask[i] = 0;
        return;
    }
    const bool in_reg = n <= (int64_t)SEL_REG * SEL_THREADS;
    uint64_t kr[SEL_REG];
#pragma unroll
    for (int q = 0; q < SEL_REG; ++q) {
        const int64_t i = (int64_t)q * SEL_THREADS + tid;
        kr[q] = in_reg && i < n ? key_of(scores[i]) : 0;
    }
    uint64_t prefix = 0, pmask = 0;
    int64_t remaining = n_keep;  // rank of T among the keys matching the prefix
    for (int byte = 7; byte >= 0; --byte) {
        const int sh = 8 * byte;
        for (int i = tid; i < 256; i += SEL_THREADS)
            s_hist[i] = 0;
        __syncthreads();
        if (in_reg) {
#pragma unroll
            for (int q = 0; q < SEL_REG; ++q) {
                const int64_t i = (int64_t)q * SEL_THREADS + tid;
                if (i < n && (kr[q] & pmask) == prefix)
                    atomicAdd(&s_hist[(kr[q] >> sh) & 255], 1u);
            }
        } else {
            for (int64_t i = tid; i < n; i += SEL_THREADS) {
                const uint64_t k = key_of(scores[i]);
                if ((k & pmask) == prefix)
                    atomicAdd(&s_hist[(k >> sh) & 255], 1u);
            }
        }
        __syncthreads();
        if (wave == 0) {
            // the byte value v with (# above v) < remaining <= (# at or above
            // v): lane L holds bins 4L .. 4L + 3 and the suffix sum S_L of the
            // bins from 4L up; the lane with S_{L+1} < remaining <= S_L scans
            // its four
            const uint32_t h0 = s_hist[4 * lane], h1 = s_hist[4 * lane + 1],
                           h2 = s_hist[4 * lane + 2], h3 = s_hist[4 * lane + 3];
            uint32_t suf = h0 + h1 + h2 + h3;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const uint32_t t = __shfl_down(suf, o, 64);
                if (lane + o < 64)
                    suf += t;
            }
            uint32_t up = __shfl_down(suf, 1, 64);  // S_{L+1}
            if (lane == 63)
                up = 0;
            if (up < (uint64_t)remaining && suf >= (uint64_t)remaining) {
                uint32_t above = up;
                int v = 4 * lane + 3;
                const uint32_t hv[4] = {h0, h1, h2, h3};
                for (int b = 3; b > 0; --b, --v) {
                    if (above + hv[b] >= (uint64_t)remaining)
                        break;
                    above += hv[b];
                }
                s_sel[0] = (uint32_t)v;
                s_sel[1] = above;
            }
        }
        __syncthreads();
        prefix |= (uint64_t)s_sel[0] << sh;
        pmask |= (uint64_t)255 << sh;
        remaining -= s_sel[1];
        __syncthreads();  // s_hist and s_sel are rewritten by the next pass
    }
    const uint64_t T = prefix;
    const int64_t need = remaining;  // >= 1 keys equal to T
    // ties in index order: per chunk of SEL_THREADS indices, each tie's rank
    // from a ballot within its wave and the wave totals before it
    int64_t taken = 0;
    for (int64_t base = 0; base < n; base += SEL_THREADS) {
        const int64_t i = base + tid;
        const int q = (int)(base / SEL_THREADS);
        const uint64_t k = i < n ? (in_reg && q < SEL_REG ? kr[q] : key_of(scores[i])) : 0;
        const bool tie = i < n && k == T;
        const uint64_t bal = __ballot(tie);
        const int64_t before_in_wave = __popcll(bal & (((uint64_t)1 << lane) - 1));
        if (lane == 0)
            s_part[wave] = __popcll(bal);
        __syncthreads();
        int64_t before = taken + before_in_wave, total = 0;
        for (int w = 0; w < SEL_THREADS / 64; ++w) {
            if (w < wave)
                before += s_part[w];
            total += s_part[w];
        }
        if (i < n)
            mask[i] = k > T || (tie && before < need);
        taken += total;
        __syncthreads();  // s_part is rewritten by the next chunk
    }
}

}  // namespace

hipError_t launch_block_scores(const MaskCall& m, hipStream_t s)
{
    const int64_t R = m.N / m.b_r, C = m.K / m.b_c, nb = R * C;
    const int es = m.dtype == LPV_F32 ? 4 : 2;
    const bool vec = ((uintptr_t)m.W % 16) == 0 && (m.ldw * es) % 16 == 0 &&
                     (!m.G || (((uintptr_t)m.G % 16) == 0 && (m.ldg * es) % 16 == 0));
    if (nb > 0 && vec) {
        // blocks per workgroup: as many as fit SC_LDS bytes of float64 terms
        // (at least one), at most one per thread
        const int bytes = m.b_r * m.b_c * 8;
        const int nbw = (int)min(min((int64_t)max(1, SC_LDS / bytes), (int64_t)SC_THREADS), C);
        const int64_t n_wg = R * ((C + nbw - 1) / nbw);
        const dim3 grid((unsigned)n_wg), block(SC_THREADS);
#define LPV_SCORES2(DT_, TY_)                                                                       \
    hipLaunchKernelGGL((k_block_scores_lds<DT_, TY_>), grid, block, 0, s, (const char*)m.W, m.ldw, \
                       (const char*)m.G, m.ldg, C, m.b_r, m.b_c, nbw, m.scores)
        if (m.dtype == LPV_BF16) {
            if (m.G)
                LPV_SCORES2(LPV_BF16, true);
            else
                LPV_SCORES2(LPV_BF16, false);
        } else if (m.dtype == LPV_F16) {
            if (m.G)
                LPV_SCORES2(LPV_F16, true);
            else
                LPV_SCORES2(LPV_F16, false);
        } else {
            if (m.G)
                LPV_SCORES2(LPV_F32, true);
            else
                LPV_SCORES2(LPV_F32, false);
        }
#undef LPV_SCORES2
        return hipGetLastError();
    }
    if (nb > 0) {
        const dim3 grid((unsigned)((nb + 255) / 256)), block(256);
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
