// encoder.hip -- the rest of a ViT encoder block around the pruned linear
// layers (gfx950): the residual sum with layer normalisation, and multi-head
// self-attention on the matrix cores.
//
// The paper prunes the linear layers of DeiT and Swin encoder blocks (Sec. 4)
// and reports whole-model speed and power (Tab. 2).  Between those layers sits
// the standard pre-norm block: LN -> qkv -> attention -> proj -> residual ->
// LN -> fc1 + GELU -> fc2 -> residual.  These kernels let the block run end to
// end on the GPU with the block-sparse layers in place.
#include <math.h>

#include "lpv_device.h"
#include "lpv_internal.h"

namespace lpv {
namespace {

// ---------------------------------------------------------------- residual + layer norm

constexpr int LN_CHUNKS = LN_MAX_D / 256;  // 4 elements per lane per 256 columns

// One wave per row: s = x + y in float32 (y may be absent), then
// out = (s - mean) / sqrt(var + eps) * gamma + beta with mean and the biased
// variance taken over the row in two passes over registers; s (rounded) is
// written to S when asked.  Every lane reads its elements before it writes
// them, so S and out may alias x or y.
template <int DT>
__global__ __launch_bounds__(256) void k_add_layernorm(const uint16_t* x, const uint16_t* y,
                                                       int64_t M, int32_t D,
                                                       const uint16_t* __restrict__ gamma,
                                                       const uint16_t* __restrict__ beta,
                                                       float eps, uint16_t* S, uint16_t* out)
{
    using E = Elem<DT>;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= M)
        return;
    float v[LN_CHUNKS][4];
    float sum = 0.0f;
#pragma unroll
    for (int i = 0; i < LN_CHUNKS; ++i) {
        const int c = 256 * i + 4 * lane;
        if (c < D) {
            const uint2 xv = *(const uint2*)(x + row * D + c);
            const uint16_t* xe = (const uint16_t*)&xv;
            uint2 yv = {0u, 0u};
            if (y)
                yv = *(const uint2*)(y + row * D + c);
            const uint16_t* ye = (const uint16_t*)&yv;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                v[i][j] = E::to_f32(xe[j]) + (y ? E::to_f32(ye[j]) : 0.0f);
                sum += v[i][j];
            }
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        sum += __shfl_xor(sum, o, 64);
    const float mean = sum / (float)D;
    float sq = 0.0f;
#pragma unroll
    for (int i = 0; i < LN_CHUNKS; ++i)
        if (256 * i + 4 * lane < D)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                sq += (v[i][j] - mean) * (v[i][j] - mean);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        sq += __shfl_xor(sq, o, 64);
    const float rstd = 1.0f / sqrtf(sq / (float)D + eps);
#pragma unroll
    for (int i = 0; i < LN_CHUNKS; ++i) {
        const int c = 256 * i + 4 * lane;
        if (c < D) {
            const uint2 gv = *(const uint2*)(gamma + c), bv = *(const uint2*)(beta + c);
            const uint16_t* ge = (const uint16_t*)&gv;
            const uint16_t* be = (const uint16_t*)&bv;
            float r[4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                r[j] = (v[i][j] - mean) * rstd * E::to_f32(ge[j]) + E::to_f32(be[j]);
            if (S)
                *(uint2*)(S + row * D + c) =
                    uint2{pack2<DT>(v[i][0], v[i][1]), pack2<DT>(v[i][2], v[i][3])};
            *(uint2*)(out + row * D + c) = uint2{pack2<DT>(r[0], r[1]), pack2<DT>(r[2], r[3])};
        }
    }
}

// ---------------------------------------------------------------- attention

// One workgroup per (sequence, head), 4 waves; wave w takes the 32-query tiles
// w, w + 4, ...  With Q and K both token-major, S^T = K Q^T comes from the
// matrix cores straight from global memory (lane: key or query l % 32, 8
// consecutive head dimensions).  Its accumulator gives lane l query l % 32 and,
// in register r, key 8 (r / 4) + 4 (l / 32) + r % 4 of the 32-key tile: a row
// of softmax lives in two lanes (l and l ^ 32), so the online softmax (running
// maximum m, running sum l, rescale by 2^(m_old - m_new)) needs one lane swap.
// The weights P^T, rounded once, are already the B operand of O^T = V^T P^T
// when the k slots of the two 16-key steps are read as those keys; V^T (A
// operand: lane = head dimension, 8 keys in two runs of 4) is staged once per
// workgroup in LDS, transposed, zero past the last token.  O^T's accumulator
// again holds one query per lane, so the rescale and the final 1 / l are
// per lane.  The weights summed into l are the rounded ones, so the output is
// exactly a weighted mean of V with those weights.
template <int DT>
__global__ __launch_bounds__(256) void k_attention(const uint16_t* __restrict__ qkv, int32_t T,
                                                   int32_t H, uint16_t* __restrict__ out)
{
    using E = Elem<DT>;
    using F = typename E::frag;
    extern __shared__ uint16_t vt[];  // [64][Tp]
    const int seq = blockIdx.x / H, h = blockIdx.x - seq * H;
    const int n_kt = (T + 31) / 32, Tp = 32 * n_kt + 4;  // + 4: rows start 8 bytes apart in banks
    const int64_t ld = 3 * (int64_t)H * ATT_HD, ldo = (int64_t)H * ATT_HD;
    const uint16_t* base = qkv + (int64_t)seq * T * ld;

    for (int i = threadIdx.x; i < n_kt * 32 * 8; i += 256) {
        const int s = i >> 3, c = i & 7;
        uint4 v = {0u, 0u, 0u, 0u};
        if (s < T)
            v = *(const uint4*)(base + s * ld + 2 * ldo + h * ATT_HD + 8 * c);
        const uint16_t* e = (const uint16_t*)&v;
#pragma unroll
        for (int j = 0; j < 8; ++j)
            vt[(8 * c + j) * Tp + s] = e[j];
    }
    __syncthreads();

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int l32 = lane & 31, half = lane >> 5;
    const float scale = 0.125f * 1.44269504088896340736f;  // 1 / sqrt(64), in base 2
    for (int qt = wave; qt < n_kt; qt += 4) {
        const int q = qt * 32 + l32;
        const uint16_t* qrow = base + (int64_t)min(q, T - 1) * ld + h * ATT_HD + 8 * half;
        F qf[4];
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
            qf[ks] = as_frag<F>(*(const uint4*)(qrow + 16 * ks));
        f32x16 o[2] = {f32x16{}, f32x16{}};
        float m = -INFINITY, l = 0.0f;
        for (int kt = 0; kt < n_kt; ++kt) {
            const uint16_t* krow =
                base + (int64_t)min(kt * 32 + l32, T - 1) * ld + ldo + h * ATT_HD + 8 * half;
            F kf[4];
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
                kf[ks] = as_frag<F>(*(const uint4*)(krow + 16 * ks));
            f32x16 s = {};
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
                s = E::mma(kf[ks], qf[ks], s);
            float mt = -INFINITY;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int key = kt * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
                s[r] = key < T ? s[r] * scale : -INFINITY;
                mt = fmaxf(mt, s[r]);
            }
            mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
            const float mn = fmaxf(m, mt);  // finite: every tile has a key
            const float alpha = exp2f(m - mn);
            uint32_t pb[8];
            float ps = 0.0f;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                pb[j] = pack2<DT>(exp2f(s[2 * j] - mn), exp2f(s[2 * j + 1] - mn));
                ps += E::to_f32((uint16_t)(pb[j] & 0xffffu)) + E::to_f32((uint16_t)(pb[j] >> 16));
            }
            ps += __shfl_xor(ps, 32, 64);
            l = l * alpha + ps;
            m = mn;
            o[0] *= alpha;
            o[1] *= alpha;
#pragma unroll
            for (int st = 0; st < 2; ++st) {
                const F pf = as_frag<F>(uint4{pb[4 * st], pb[4 * st + 1], pb[4 * st + 2], pb[4 * st + 3]});
#pragma unroll
                for (int dt = 0; dt < 2; ++dt) {
                    const uint16_t* vp = vt + (32 * dt + l32) * Tp + kt * 32 + 16 * st + 4 * half;
                    const uint2 lo = *(const uint2*)vp, hi = *(const uint2*)(vp + 8);
                    o[dt] = E::mma(as_frag<F>(uint4{lo.x, lo.y, hi.x, hi.y}), pf, o[dt]);
                }
            }
        }
        if (q < T) {
            const float inv = 1.0f / l;
            uint16_t* orow = out + ((int64_t)seq * T + q) * ldo + h * ATT_HD;
#pragma unroll
            for (int dt = 0; dt < 2; ++dt)
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    *(uint2*)(orow + 32 * dt + 8 * g + 4 * half) =
                        uint2{pack2<DT>(o[dt][4 * g] * inv, o[dt][4 * g + 1] * inv),
                              pack2<DT>(o[dt][4 * g + 2] * inv, o[dt][4 * g + 3] * inv)};
        }
    }
}

}  // namespace

hipError_t launch_add_layernorm(const void* x, const void* y, int64_t M, int32_t D, int dtype,
                                const void* gamma, const void* beta, float eps, void* S, void* out,
                                hipStream_t s)
{
    if (M == 0)
        return hipSuccess;
    const dim3 grid((unsigned)((M + 3) / 4)), block(256);
    if (dtype == LPV_BF16)
        hipLaunchKernelGGL(k_add_layernorm<LPV_BF16>, grid, block, 0, s, (const uint16_t*)x,
                           (const uint16_t*)y, M, D, (const uint16_t*)gamma, (const uint16_t*)beta,
                           eps, (uint16_t*)S, (uint16_t*)out);
    else
        hipLaunchKernelGGL(k_add_layernorm<LPV_F16>, grid, block, 0, s, (const uint16_t*)x,
                           (const uint16_t*)y, M, D, (const uint16_t*)gamma, (const uint16_t*)beta,
                           eps, (uint16_t*)S, (uint16_t*)out);
    return hipGetLastError();
}

hipError_t launch_attention(const void* qkv, int64_t n_seq, int32_t T, int32_t H, int dtype,
                            void* out, hipStream_t s)
{
    if (n_seq == 0)
        return hipSuccess;
    const int n_kt = (T + 31) / 32;
    const size_t lds = (size_t)ATT_HD * (32 * n_kt + 4) * 2;
    const dim3 grid((unsigned)(n_seq * H)), block(256);
    // dynamic LDS beyond 64 KB (T > 480) must be allowed per kernel; the
    // setting is idempotent, so a race between threads is harmless
    static bool allowed[2] = {false, false};
    const int ix = dtype == LPV_BF16 ? 1 : 0;
    if (!allowed[ix]) {
        const int max_lds = ATT_HD * (ATT_MAX_T + 4) * 2;
        const hipError_t e =
            dtype == LPV_BF16
                ? hipFuncSetAttribute((const void*)k_attention<LPV_BF16>,
                                      hipFuncAttributeMaxDynamicSharedMemorySize, max_lds)
                : hipFuncSetAttribute((const void*)k_attention<LPV_F16>,
                                      hipFuncAttributeMaxDynamicSharedMemorySize, max_lds);
        if (e != hipSuccess)
            return e;
        allowed[ix] = true;
    }
    if (dtype == LPV_BF16)
        hipLaunchKernelGGL(k_attention<LPV_BF16>, grid, block, lds, s, (const uint16_t*)qkv, T, H,
                           (uint16_t*)out);
    else
        hipLaunchKernelGGL(k_attention<LPV_F16>, grid, block, lds, s, (const uint16_t*)qkv, T, H,
                           (uint16_t*)out);
    return hipGetLastError();
}

}  // namespace lpv
