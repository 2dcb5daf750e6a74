// linear.hip -- Y = g(X W~^T + b): the block-sparse hot path and the dense
// reference path.
//
// bf16 / fp16 (matrix cores).  A workgroup of 4 waves owns one tile of BM = 256
// tokens times one group of GROUP_TILES x 32 output rows.  It walks the
// group's steps (the 32-wide reduction columns where any of its rows keeps a
// tile; pruned columns are never touched):
//   1. the X slice [256 tokens x 32 columns] and the step's kept W tiles are
//      loaded from HBM with 16-byte coalesced loads and staged in LDS (double
//      buffered: step s+1 is in flight while step s computes);
//   2. each wave takes 64 tokens and, for every kept tile of the step, issues
//      v_mfma_f32_32x32x16 (bf16 or fp16 in, float32 accumulate) into its
//      accumulator for that tile row.
// The work per workgroup is therefore proportional to the kept tiles, the
// quantity the paper's cost model counts (Sec. 3.4).  The epilogue adds the
// bias, applies GELU if asked, rounds once to the element type and stores Y
// through LDS so every row segment goes out as full 128-byte lines.
//
// MFMA operand roles: A = a W tile (rows = output features), B = X slice
// transposed (columns = tokens), so D[n][token]; lane l then holds token l % 32
// and, per group of 4 accumulator registers, 4 consecutive output features.
//
// The dense path is the same kernel with every tile kept and W read straight
// from its row-major layout.  fp32 runs a plain VALU kernel over the canonical
// BSR arrays (it serves the small fp32 configuration only).
#include "lpv_device.h"
#include "lpv_internal.h"

namespace lpv {
namespace {

constexpr int NT = 256;       // threads per workgroup (4 waves)
constexpr int XROW = 5;       // uint4 per staged X row: 64 bytes of data + 16 bytes pad
constexpr int TILE_U4 = 128;  // uint4 per 32x32 16-bit tile
constexpr int EROW = 9;       // uint4 per epilogue row: 128 bytes + 16 bytes pad

struct Args {
    const char* X;
    int64_t ldx, M, K, N;
    // sparse operand stream and schedule
    const uint4* stream;
    const int32_t* step_ptr;
    const int32_t* step_col;
    const int32_t* step_bits;
    const int32_t* step_tile;
    const int32_t* group_order;
    // dense weight
    const char* W;
    int64_t ldw;
    int32_t n_groups, n_tile_rows, n_tile_cols, n_mtiles;
    const char* bias;
    char* Y;
    int64_t ldy;
};

constexpr int G = GROUP_TILES;
constexpr int SMEM_MAIN = 2 * BM * XROW + 2 * G * TILE_U4;
constexpr int SMEM_EPI = 4 * 64 * EROW;
constexpr int SMEM_U4 = SMEM_MAIN > SMEM_EPI ? SMEM_MAIN : SMEM_EPI;

template <int DT, bool GELU, bool DENSE>
__global__ __launch_bounds__(NT, 2) void k_linear16(Args a)
{
    using E = Elem<DT>;
    using F = typename E::frag;
    __shared__ uint4 smem[SMEM_U4];
    uint4* xs = smem;                 // [2][BM * XROW]
    uint4* ws = smem + 2 * BM * XROW; // [2][G * TILE_U4]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

    // Work item of this workgroup.  Consecutive workgroups go to different
    // XCDs (round robin over 8), so hand each XCD a contiguous run of items:
    // the groups of one token tile then share that XCD's L2 for their X reads.
    const int n_items = a.n_mtiles * a.n_groups;
    const int per_xcd = (int)(gridDim.x >> 3);
    const int item = (int)(blockIdx.x & 7) * per_xcd + (int)(blockIdx.x >> 3);
    if (item >= n_items)
        return;
    const int mt = item / a.n_groups;
    const int gs = item - mt * a.n_groups;
    const int g = DENSE ? gs : a.group_order[gs];
    const int s_begin = DENSE ? 0 : a.step_ptr[g];
    const int s_end = DENSE ? a.n_tile_cols : a.step_ptr[g + 1];
    const int64_t m0 = (int64_t)mt * BM;
    const int row0 = g * G;
    const int rows_valid = min(G, a.n_tile_rows - row0);

    f32x16 acc[2][G];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int j = 0; j < G; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                acc[t][j][v] = 0.0f;

    // ---- global -> registers for one step
    uint4 xr[4];
    uint4 wr[G / 2];
    int bits_next = 0;
    auto fetch = [&](int s) {
        const int col = DENSE ? s : a.step_col[s];
        const int bits = DENSE ? ((1 << rows_valid) - 1) : a.step_bits[s];
        bits_next = bits;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int idx = i * NT + tid;
            const int r = idx >> 2, ch = idx & 3;
            const int64_t m = m0 + r;
            const int64_t k = (int64_t)col * TILE + ch * 8;
            xr[i] = make_uint4(0, 0, 0, 0);
            if (m < a.M && k < a.K)
                xr[i] = *(const uint4*)(a.X + (m * a.ldx + k) * 2);
        }
        if (DENSE) {
#pragma unroll
            for (int i = 0; i < G / 2; ++i) {
                const int idx = i * NT + tid;
                const int rr = idx >> 2, ch = idx & 3;
                const int64_t n = (int64_t)row0 * TILE + rr;
                const int64_t k = (int64_t)col * TILE + ch * 8;
                wr[i] = make_uint4(0, 0, 0, 0);
                if (n < a.N && k < a.K)
                    wr[i] = *(const uint4*)(a.W + (n * a.ldw + k) * 2);
            }
        } else {
            const int nk = __popc(bits);
            const uint4* src = a.stream + (int64_t)a.step_tile[s] * TILE_U4;
#pragma unroll
            for (int i = 0; i < G / 2; ++i) {
                const int idx = i * NT + tid;
                if (idx < nk * TILE_U4)
                    wr[i] = src[idx];
            }
        }
    };
    // ---- registers -> LDS buffer
    auto commit = [&](int buf) {
        uint4* xb = xs + buf * BM * XROW;
        uint4* wb = ws + buf * G * TILE_U4;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int idx = i * NT + tid;
            xb[(idx >> 2) * XROW + (idx & 3)] = xr[i];
        }
        if (DENSE) {
            // row rr, 16-byte chunk ch of the group's W rows -> operand order
#pragma unroll
            for (int i = 0; i < G / 2; ++i) {
                const int idx = i * NT + tid;
                const int rr = idx >> 2, ch = idx & 3;
                const int j = rr >> 5, l = (rr & 31) + 32 * (ch & 1), ks = ch >> 1;
                wb[j * TILE_U4 + ks * 64 + l] = wr[i];
            }
        } else {
            const int nk = __popc(bits_next);
#pragma unroll
            for (int i = 0; i < G / 2; ++i) {
                const int idx = i * NT + tid;
                if (idx < nk * TILE_U4)
                    wb[idx] = wr[i];
            }
        }
    };
    // ---- LDS -> matrix cores
    auto compute = [&](int buf, int bits) {
        const uint4* xb = xs + buf * BM * XROW;
        const uint4* wb = ws + buf * G * TILE_U4;
        F xa[2][2];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const int r = wave * 64 + t * 32 + (lane & 31);
                xa[t][ks] = as_frag<F>(xb[r * XROW + ks * 2 + (lane >> 5)]);
            }
        int idx = 0;
#pragma unroll
        for (int j = 0; j < G; ++j) {
            if (bits & (1 << j)) {
                const F w0 = as_frag<F>(wb[idx * TILE_U4 + lane]);
                const F w1 = as_frag<F>(wb[idx * TILE_U4 + 64 + lane]);
                acc[0][j] = E::mma(w0, xa[0][0], acc[0][j]);
                acc[1][j] = E::mma(w0, xa[1][0], acc[1][j]);
                acc[0][j] = E::mma(w1, xa[0][1], acc[0][j]);
                acc[1][j] = E::mma(w1, xa[1][1], acc[1][j]);
                ++idx;
            }
        }
    };

    if (s_begin < s_end) {
        fetch(s_begin);
        commit(0);
    }
    __syncthreads();
    for (int s = s_begin; s < s_end; ++s) {
        const int buf = (s - s_begin) & 1;
        const int bits = bits_next;
        if (s + 1 < s_end)
            fetch(s + 1);
        compute(buf, bits);
        if (s + 1 < s_end)
            commit(buf ^ 1);
        __syncthreads();
    }

    // ---- epilogue: bias, GELU, one rounding, transpose through LDS, store
    uint4* eb = smem + wave * 64 * EROW;
    uint2* eb2 = (uint2*)eb;
#pragma unroll
    for (int jp = 0; jp < G; jp += 2) {
        if (jp >= rows_valid)
            break;
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
            const int j = jp + jj;
            const int64_t n_tile = (int64_t)(row0 + j) * TILE;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int n_off = 8 * q + 4 * (lane >> 5);
                float b[4] = {0.f, 0.f, 0.f, 0.f};
                if (a.bias && n_tile + n_off < a.N) {
                    const uint2 bb = *(const uint2*)(a.bias + (n_tile + n_off) * 2);
                    b[0] = E::to_f32(bb.x & 0xffff);
                    b[1] = E::to_f32(bb.x >> 16);
                    b[2] = E::to_f32(bb.y & 0xffff);
                    b[3] = E::to_f32(bb.y >> 16);
                }
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    float v[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        v[e] = acc[t][j][4 * q + e] + b[e];
                        if (GELU)
                            v[e] = gelu_erf(v[e]);
                    }
                    uint2 o;
                    o.x = (uint32_t)E::from_f32(v[0]) | ((uint32_t)E::from_f32(v[1]) << 16);
                    o.y = (uint32_t)E::from_f32(v[2]) | ((uint32_t)E::from_f32(v[3]) << 16);
                    const int row = t * 32 + (lane & 31);
                    eb2[row * (EROW * 2) + (jj * 32 + n_off) / 4] = o;
                }
            }
        }
        __syncthreads();
        const bool second = jp + 1 < rows_valid;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int row = i * 8 + (lane >> 3), ch = lane & 7;
            const int64_t m = m0 + wave * 64 + row;
            const int64_t n = (int64_t)(row0 + jp) * TILE + ch * 8;
            if (m < a.M && n < a.N && (ch < 4 || second))
                *(uint4*)(a.Y + (m * a.ldy + n) * 2) = eb[row * EROW + ch];
        }
        __syncthreads();
    }
}

// fp32: 64 tokens x 16 outputs per workgroup; thread = one token x 4 outputs.
// Sparse: the 16 outputs lie in one block-row (b_r >= 16), whose kept blocks
// are walked through row_ptr / col_idx.  Dense: every column.
template <bool GELU, bool DENSE>
__global__ __launch_bounds__(256) void k_linear_f32(const float* __restrict__ X, int64_t ldx,
                                                    int64_t M, int64_t K, int64_t N,
                                                    const float* __restrict__ values,
                                                    const int32_t* __restrict__ row_ptr,
                                                    const int32_t* __restrict__ col_idx,
                                                    int32_t b_r, int32_t b_c,
                                                    const float* __restrict__ W, int64_t ldw,
                                                    const float* __restrict__ bias,
                                                    float* __restrict__ Y, int64_t ldy)
{
    const int64_t m = (int64_t)blockIdx.x * 64 + (threadIdx.x & 63);
    const int64_t n0 = (int64_t)blockIdx.y * 16 + (threadIdx.x >> 6) * 4;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    const bool live = m < M;
    const int64_t mm = live ? m : 0;
    if (DENSE) {
        for (int64_t k = 0; k < K; ++k) {
            const float x = X[mm * ldx + k];
#pragma unroll
            for (int o = 0; o < 4; ++o)
                acc[o] = fmaf(x, W[(n0 + o) * ldw + k], acc[o]);
        }
    } else {
        const int r = (int)(n0 / b_r);
        const int64_t i0 = n0 - (int64_t)r * b_r;
        for (int p = row_ptr[r]; p < row_ptr[r + 1]; ++p) {
            const int64_t kc = (int64_t)col_idx[p] * b_c;
            const float* blk = values + (int64_t)p * b_r * b_c;
            for (int kk = 0; kk < b_c; ++kk) {
                const float x = X[mm * ldx + kc + kk];
#pragma unroll
                for (int o = 0; o < 4; ++o)
                    acc[o] = fmaf(x, blk[(i0 + o) * b_c + kk], acc[o]);
            }
        }
    }
    if (!live)
        return;
#pragma unroll
    for (int o = 0; o < 4; ++o) {
        float v = acc[o] + (bias ? bias[n0 + o] : 0.0f);
        if (GELU)
            v = gelu_erf(v);
        Y[m * ldy + n0 + o] = v;
    }
}

inline unsigned grid_items(int64_t n_items) { return (unsigned)(((n_items + 7) / 8) * 8); }

template <bool DENSE>
hipError_t launch16(int dtype, bool gelu, const Args& a, hipStream_t s)
{
    const dim3 grid(grid_items((int64_t)a.n_mtiles * a.n_groups)), block(NT);
    if (dtype == LPV_BF16) {
        if (gelu)
            hipLaunchKernelGGL((k_linear16<LPV_BF16, true, DENSE>), grid, block, 0, s, a);
        else
            hipLaunchKernelGGL((k_linear16<LPV_BF16, false, DENSE>), grid, block, 0, s, a);
    } else {
        if (gelu)
            hipLaunchKernelGGL((k_linear16<LPV_F16, true, DENSE>), grid, block, 0, s, a);
        else
            hipLaunchKernelGGL((k_linear16<LPV_F16, false, DENSE>), grid, block, 0, s, a);
    }
    return hipGetLastError();
}

Args base_args(const LinearCall& c, int64_t N, int64_t K)
{
    Args a = {};
    a.X = (const char*)c.X;
    a.ldx = c.ldx;
    a.M = c.M;
    a.K = K;
    a.N = N;
    a.bias = (const char*)c.bias;
    a.Y = (char*)c.Y;
    a.ldy = c.ldy;
    a.n_tile_rows = (int32_t)((N + TILE - 1) / TILE);
    a.n_tile_cols = (int32_t)((K + TILE - 1) / TILE);
    a.n_groups = (a.n_tile_rows + G - 1) / G;
    a.n_mtiles = (int32_t)((c.M + BM - 1) / BM);
    return a;
}

template <bool DENSE>
hipError_t launch_f32(bool gelu, const float* X, int64_t ldx, int64_t M, int64_t K, int64_t N,
                      const lpv_bsr* h, const float* W, int64_t ldw, const float* bias, float* Y,
                      int64_t ldy, hipStream_t s)
{
    const dim3 grid((unsigned)((M + 63) / 64), (unsigned)(N / 16)), block(256);
    const float* vals = h ? (const float*)h->values : nullptr;
    const int32_t* rp = h ? h->row_ptr : nullptr;
    const int32_t* ci = h ? h->col_idx : nullptr;
    const int32_t b_r = h ? h->b_r : 16, b_c = h ? h->b_c : 16;
    if (gelu)
        hipLaunchKernelGGL((k_linear_f32<true, DENSE>), grid, block, 0, s, X, ldx, M, K, N, vals,
                           rp, ci, b_r, b_c, W, ldw, bias, Y, ldy);
    else
        hipLaunchKernelGGL((k_linear_f32<false, DENSE>), grid, block, 0, s, X, ldx, M, K, N, vals,
                           rp, ci, b_r, b_c, W, ldw, bias, Y, ldy);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_bsr_linear(const lpv_bsr* h, const LinearCall& c, hipStream_t s)
{
    if (h->dtype == LPV_F32)
        return launch_f32<false>(c.gelu != 0, (const float*)c.X, c.ldx, c.M, h->K, h->N, h, nullptr,
                                 0, (const float*)c.bias, (float*)c.Y, c.ldy, s);
    Args a = base_args(c, h->N, h->K);
    a.stream = (const uint4*)h->stream_vals;
    a.step_ptr = h->step_ptr;
    a.step_col = h->step_col;
    a.step_bits = h->step_bits;
    a.step_tile = h->step_tile;
    a.group_order = h->group_order;
    return launch16<false>(h->dtype, c.gelu != 0, a, s);
}

hipError_t launch_dense_linear(const void* W, int64_t ldw, int64_t N, int64_t K, int dtype,
                               const LinearCall& c, hipStream_t s)
{
    if (dtype == LPV_F32)
        return launch_f32<true>(c.gelu != 0, (const float*)c.X, c.ldx, c.M, K, N, nullptr,
                                (const float*)W, ldw, (const float*)c.bias, (float*)c.Y, c.ldy, s);
    Args a = base_args(c, N, K);
    a.W = (const char*)W;
    a.ldw = ldw;
    return launch16<true>(dtype, c.gelu != 0, a, s);
}

}  // namespace lpv
