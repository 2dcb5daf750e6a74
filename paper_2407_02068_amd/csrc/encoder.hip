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

// One workgroup per (sequence, head), 8 waves.  K and V of the head are staged
// once in LDS, row-major (row = token, 64 elements and 16 bytes of padding:
// 144-byte rows put 16 consecutive rows of one 16-byte column in distinct
// banks), zero past the last token; wave w takes the 32-query tiles w, w + 8,
// ...  S^T = K Q^T on the matrix cores (lane: key or query l % 32, 8
// consecutive head dimensions; K from LDS, Q from global memory once per
// tile).  Its accumulator gives lane l query l % 32 and, in register r, key
// 8 (r / 4) + 4 (l / 32) + r % 4 of the 32-key tile: a row of softmax lives
// in two lanes (l and l ^ 32), so the online softmax (running maximum m,
// running sum l, rescale by 2^(m_old - m_new)) needs one lane swap.  The
// weights P^T, rounded once, are already the B operand of O^T = V^T P^T when
// the k slots of the two 16-key steps are read as those keys; the V^T operand
// (lane = head dimension, 8 keys in two runs of 4) comes from the row-major V
// by transposing LDS reads (ds_read_b64_tr_b16: within 16 lanes, lane j
// reads key t0 + j / 4 at dimensions c0 + 4 (j % 4) .. + 3, and lane i
// receives keys t0 .. t0 + 3 of dimension c0 + i).  O^T's accumulator again
// holds one query per lane, so the rescale and the final 1 / l are per lane.
// The weights summed into l are the rounded ones, so the output is exactly a
// weighted mean of V with those weights.
constexpr int ATT_NT = 512;
constexpr int ATT_RS = ATT_HD * 2 + 16;  // bytes per staged row
static_assert(2 * ((ATT_MAX_T + 31) / 32 * 32) * ATT_RS <= 163840, "K and V of a head fit in LDS");

typedef short att_v4s __attribute__((ext_vector_type(4)));

__device__ inline uint2 att_tr_read(uint32_t addr)
{
    return __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                         (__attribute__((address_space(3))) att_v4s*)(uintptr_t)addr));
}

typedef unsigned int att_u4 __attribute__((ext_vector_type(4)));

// c + the two 16-bit values packed in p (one dot product with (1, 1): the
// products are exact, the sum is float32)
template <int DT> __device__ inline float att_add2(uint32_t p, float c)
{
    if (DT == LPV_BF16)
        return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, p),
                                               __builtin_bit_cast(bf16x2, 0x3f803f80u), c, false);
    return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, p), __builtin_bit_cast(f16x2, 0x3c003c00u),
                                  c, false);
}

__device__ inline uint4 att_read16(uint32_t addr)
{
    return __builtin_bit_cast(uint4, *(const __attribute__((address_space(3))) att_u4*)(uintptr_t)addr);
}

template <int DT>
__global__ __launch_bounds__(ATT_NT) void k_attention(const uint16_t* __restrict__ qkv, int32_t T,
                                                      int32_t H, uint16_t* __restrict__ out)
{
    using E = Elem<DT>;
    using F = typename E::frag;
    extern __shared__ uint4 att_lds[];  // K rows, then V rows
    const int seq = blockIdx.x / H, h = blockIdx.x - seq * H;
    const int n_kt = (T + 31) / 32, Tp = 32 * n_kt;
    const int64_t ld = 3 * (int64_t)H * ATT_HD, ldo = (int64_t)H * ATT_HD;
    const uint16_t* base = qkv + (int64_t)seq * T * ld;
    char* kl = (char*)att_lds;
    char* vl = kl + Tp * ATT_RS;

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int l32 = lane & 31, half = lane >> 5;
    // the Q fragments of this wave's first query tile, loaded while K and V
    // are staged (lane: query l % 32, dimensions 8 half + 16 ks)
    F qf[4];
    auto load_q = [&](int qt) {
        const uint16_t* qrow =
            base + (int64_t)min(qt * 32 + l32, T - 1) * ld + h * ATT_HD + 8 * half;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
            qf[ks] = as_frag<F>(*(const uint4*)(qrow + 16 * ks));
    };
    if (wave < n_kt)
        load_q(wave);
    // staging: 16-byte chunk c (0..7) of row s of K and V; every load of a
    // batch is issued before the first LDS write
    constexpr int SB = 4;
    for (int i0 = threadIdx.x; i0 < Tp * 8; i0 += SB * ATT_NT) {
        uint4 kv[SB], vv[SB];
#pragma unroll
        for (int b = 0; b < SB; ++b) {
            const int i = i0 + b * ATT_NT, s = i >> 3, c = i & 7;
            kv[b] = uint4{0u, 0u, 0u, 0u};
            vv[b] = uint4{0u, 0u, 0u, 0u};
            if (s < T) {
                const uint16_t* row = base + (int64_t)s * ld + h * ATT_HD + 8 * c;
                kv[b] = *(const uint4*)(row + ldo);
                vv[b] = *(const uint4*)(row + 2 * ldo);
            }
        }
#pragma unroll
        for (int b = 0; b < SB; ++b) {
            const int i = i0 + b * ATT_NT, s = i >> 3, c = i & 7;
            if (i < Tp * 8) {
                *(uint4*)(kl + s * ATT_RS + 16 * c) = kv[b];
                *(uint4*)(vl + s * ATT_RS + 16 * c) = vv[b];
            }
        }
    }
    __syncthreads();

    // this lane's K fragment (key l32 of a tile, dimensions 8 half + 16 ks)
    const uint32_t ka = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)kl +
                        l32 * ATT_RS + half * 16;
    // this lane's transposing V read: 16-lane group g = lane / 16 takes
    // dimensions 16 (g % 2) + 0..15 (of 32 dt + ..) and keys 4 (g / 2) + 0..3
    // (of the 16-key step; + 8 for the second run)
    const int g = lane >> 4, jj = lane & 15;
    const uint32_t va = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)vl +
                        ((jj >> 2) + 4 * (g >> 1)) * ATT_RS + (16 * (g & 1) + 4 * (jj & 3)) * 2;
    const float scale = 0.125f * 1.44269504088896340736f;  // 1 / sqrt(64), in base 2
    for (int qt = wave; qt < n_kt; qt += ATT_NT / 64) {
        const int q = qt * 32 + l32;
        if (qt != wave)
            load_q(qt);
        f32x16 o[2] = {f32x16{}, f32x16{}};
        float m = -INFINITY, l = 0.0f;  // running maximum of the unscaled scores, sum
        for (int kt = 0; kt < n_kt; ++kt) {
            const uint32_t kt_off = (uint32_t)kt * 32 * ATT_RS;
            f32x16 s = {};
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
                s = E::mma(as_frag<F>(att_read16(ka + kt_off + 32 * ks)), qf[ks], s);
            if (kt == n_kt - 1 && T % 32) {  // the last tile: keys past T drop out
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if (kt * 32 + 8 * (r >> 2) + 4 * half + (r & 3) >= T)
                        s[r] = -INFINITY;
            }
            float mt = s[0];
#pragma unroll
            for (int r = 1; r < 16; ++r)
                mt = fmaxf(mt, s[r]);
            mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
            const float mn = fmaxf(m, mt);  // finite: every tile has a key
            // weights 2^((s - mn) scale): the scale is positive, so the maximum
            // of the scaled scores is the scaled maximum (arguments <= 0; the
            // hardware exp2 flushes results below 2^-126 to zero)
            const float nms = -mn * scale;
            const float alpha = __builtin_amdgcn_exp2f((m - mn) * scale);
            uint32_t pb[8];
            float ps = 0.0f;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                pb[j] = pack2<DT>(__builtin_amdgcn_exp2f(fmaf(s[2 * j], scale, nms)),
                                  __builtin_amdgcn_exp2f(fmaf(s[2 * j + 1], scale, nms)));
                ps = att_add2<DT>(pb[j], ps);
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
                    const uint32_t vp = va + kt_off + (uint32_t)(16 * st) * ATT_RS + 64 * dt;
                    const uint2 lo = att_tr_read(vp), hi = att_tr_read(vp + 8 * ATT_RS);
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
                for (int gg = 0; gg < 4; ++gg)
                    *(uint2*)(orow + 32 * dt + 8 * gg + 4 * half) =
                        uint2{pack2<DT>(o[dt][4 * gg] * inv, o[dt][4 * gg + 1] * inv),
                              pack2<DT>(o[dt][4 * gg + 2] * inv, o[dt][4 * gg + 3] * inv)};
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
    const size_t lds = (size_t)2 * 32 * n_kt * ATT_RS;
    const dim3 grid((unsigned)(n_seq * H)), block(ATT_NT);
    // dynamic LDS beyond 64 KB (T > 224) must be allowed per kernel; the
    // setting is idempotent, so a race between threads is harmless
    static bool allowed[2] = {false, false};
    const int ix = dtype == LPV_BF16 ? 1 : 0;
    if (!allowed[ix]) {
        const int max_lds = 2 * ((ATT_MAX_T + 31) / 32 * 32) * ATT_RS;
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
