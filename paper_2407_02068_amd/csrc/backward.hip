// backward.hip -- backward of the block-sparse linear layer, for finetuning
// the pruned model (gfx950).
//
// Paper, Fig. 1 and Sec. 4: after block pruning the model is finetuned.  The
// mask stays fixed: a dropped block is absent from the layer, so it neither
// passes a gradient to the input nor receives one.  For the pre-activation
// Z = X W~^T + b and G = dL/dZ (M x N):
//   dX = G W~         the forward kernel run on the handle of W~^T, which
//                     k_transpose_blocks + pack build (lpv_bsr_transpose)
//   dW = G^T X        on the kept blocks only: k_gradw_tiles (matrix cores)
//                     and k_gradw_reduce, or k_gradw_plain for fp32 handles
//   db = sum_m G[m]   k_bias_partial + k_bias_reduce
// Every sum is taken in a fixed order, so results do not depend on timing.
#include <mutex>

#include <type_traits>

#include "lpv_device.h"
#include "lpv_internal.h"

namespace lpv {
namespace {

static __device__ uint4 g_zero_line[1];

// ---------------------------------------------------------------- transpose

// One workgroup per block-row r: every kept block (r, c) of the handle is
// written transposed into the dense K x N buffer WT (block (c, r) of W~^T),
// and maskT[c][r] is set.  Everything else in WT and maskT is left as the
// caller cleared it.
__global__ __launch_bounds__(256) void k_transpose_blocks(int32_t b_r, int32_t b_c, int32_t R,
                                                          int32_t es, const int32_t* __restrict__ row_ptr,
                                                          const int32_t* __restrict__ col_idx,
                                                          const char* __restrict__ values,
                                                          char* __restrict__ WT, int64_t ldwt,
                                                          uint8_t* __restrict__ maskT)
{
    const int r = blockIdx.x;
    const int p0 = row_ptr[r], p1 = row_ptr[r + 1];
    const int nb = b_r * b_c;
    for (int p = p0; p < p1; ++p) {
        const int c = col_idx[p];
        if (threadIdx.x == 0)
            maskT[(int64_t)c * R + r] = 1;
        for (int e = threadIdx.x; e < nb; e += 256) {
            const int i = e / b_c, j = e - i * b_c;  // W~[r b_r + i][c b_c + j]
            const char* src = values + ((int64_t)p * nb + e) * es;
            char* dst = WT + (((int64_t)c * b_c + j) * ldwt + (int64_t)r * b_r + i) * es;
            if (es == 4)
                *(uint32_t*)dst = *(const uint32_t*)src;
            else
                *(uint16_t*)dst = *(const uint16_t*)src;
        }
    }
}

// ---------------------------------------------------------------- element access

template <int DT> __device__ inline float load_elem(const char* base, int64_t idx)
{
    if constexpr (DT == LPV_F32)
        return ((const float*)base)[idx];
    else
        return Elem<DT>::to_f32(((const uint16_t*)base)[idx]);
}

template <int DT> __device__ inline void store_elem(char* base, int64_t idx, float v)
{
    if constexpr (DT == LPV_F32)
        ((float*)base)[idx] = v;
    else
        ((uint16_t*)base)[idx] = Elem<DT>::from_f32(v);
}

// ---------------------------------------------------------------- bias gradient

typedef uint32_t v4u __attribute__((ext_vector_type(4)));

// part[chunk][n] = sum over the chunk's token rows (ascending) of G[m][n], in
// float32.  Thread: 16 bytes of columns; grid (column blocks, chunks).
template <int DT>
__global__ __launch_bounds__(256) void k_bias_partial(const char* __restrict__ G, int64_t ldg,
                                                      int64_t M, int64_t N, int64_t rows,
                                                      float* __restrict__ part)
{
    constexpr int ES = DT == LPV_F32 ? 4 : 2, V = 16 / ES;
    const int64_t n0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * V;
    const int64_t m0 = (int64_t)blockIdx.y * rows, m1 = min(M, m0 + rows);
    if (n0 >= N)
        return;
    float acc[V];
#pragma unroll
    for (int i = 0; i < V; ++i)
        acc[i] = 0.0f;
    const bool full = n0 + V <= N;
    int64_t m = m0;
    if (full) {
        // 8 rows' loads in flight, then their sums in row order
        for (; m + 8 <= m1; m += 8) {
            v4u v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                v[u] = __builtin_nontemporal_load((const v4u*)(G + ((m + u) * ldg + n0) * ES));
#pragma unroll
            for (int u = 0; u < 8; ++u)
#pragma unroll
                for (int i = 0; i < V; ++i)
                    acc[i] += load_elem<DT>((const char*)&v[u], i);
        }
    }
    for (; m < m1; ++m) {
        if (full) {
            const uint4 v = *(const uint4*)(G + (m * ldg + n0) * ES);
#pragma unroll
            for (int i = 0; i < V; ++i)
                acc[i] += load_elem<DT>((const char*)&v, i);
        } else {
            for (int i = 0; i < V; ++i)
                if (n0 + i < N)
                    acc[i] += load_elem<DT>(G, m * ldg + n0 + i);
        }
    }
#pragma unroll
    for (int i = 0; i < V; ++i)
        if (n0 + i < N)
            part[blockIdx.y * N + n0 + i] = acc[i];
}

// db[n] from the chunks' partial sums in a fixed order: workgroup = 32
// columns; lane group l (0..7) adds chunks l, l + 8, ... in order, then the 8
// sums are added in order of l; one rounding.
template <int DT>
__global__ __launch_bounds__(256) void k_bias_reduce(const float* __restrict__ part, int n_chunks,
                                                     int64_t N, char* __restrict__ db)
{
    __shared__ float s_sum[8][32];
    const int col = threadIdx.x & 31, l = threadIdx.x >> 5;
    const int64_t n = (int64_t)blockIdx.x * 32 + col;
    float s = 0.0f;
    if (n < N)
        for (int c = l; c < n_chunks; c += 8)
            s += part[(int64_t)c * N + n];
    s_sum[l][col] = s;
    __syncthreads();
    if (l == 0 && n < N) {
        float t = 0.0f;
        for (int i = 0; i < 8; ++i)
            t += s_sum[i][col];
        store_elem<DT>(db, n, t);
    }
}

// ---------------------------------------------------------------- weight gradient, fp32

// Block-row of kept block p (row_ptr is ascending).
__device__ inline int block_row(const int32_t* row_ptr, int R, int64_t p)
{
    int lo = 0, hi = R;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (row_ptr[mid] <= p)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

// One workgroup per kept block; each thread sums whole elements over all
// tokens, ascending.  For fp32 handles (small layers).
template <int DT>
__global__ __launch_bounds__(256) void k_gradw_plain(int32_t b_r, int32_t b_c, int32_t R,
                                                     const int32_t* __restrict__ row_ptr,
                                                     const int32_t* __restrict__ col_idx,
                                                     const char* __restrict__ G, int64_t ldg,
                                                     const char* __restrict__ X, int64_t ldx,
                                                     int64_t M, char* __restrict__ out)
{
    const int64_t p = blockIdx.x;
    const int r = block_row(row_ptr, R, p), c = col_idx[p];
    const int nb = b_r * b_c;
    for (int e = threadIdx.x; e < nb; e += 256) {
        const int i = e / b_c, j = e - i * b_c;
        const int64_t n = (int64_t)r * b_r + i, k = (int64_t)c * b_c + j;
        float acc = 0.0f;
        for (int64_t m = 0; m < M; ++m)
            acc += load_elem<DT>(G, m * ldg + n) * load_elem<DT>(X, m * ldx + k);
        store_elem<DT>(out, p * nb + e, acc);
    }
}

// ---------------------------------------------------------------- weight gradient, 16-bit

// A workgroup takes a *window* -- one schedule group (8 tile rows, 256
// outputs n) times 8 tile columns (256 inputs k) -- and a chunk of tokens, and
// computes for every kept 32 x 32 tile of the window the partial product
// G[chunk, tile rows]^T X[chunk, tile columns] with the matrix cores.  Tokens
// are the reduction: they stream through a 2-stage LDS ring, 64 per stage
// (G: 64 x 256 and X: 64 x 256 elements, 32 KB each, rows of 512 bytes whose
// 64-byte segments are XOR-swizzled by the row).  The MFMA operands need 8
// consecutive tokens per lane; ds_read_b64_tr_b16 gathers them from the
// token-major rows: within each 16-lane group, lane i receives element i % 4
// of the 8-byte pieces read by lanes i / 4 + 4 q (q = 0..3), so when lane j
// reads row t0 + j / 4 at column c0 + 4 (j % 4), lane i holds rows t0 .. t0 + 3
// of column c0 + i.
//
// Wave w takes one tile row of the window (its kept tiles, at most 8): the
// row's G fragment is read once per k-step and each kept tile's X fragment
// into registers of its own.  The rows are paired on the SIMDs by kept count
// (largest with smallest), so every SIMD carries about the same number of
// products.
// Partials go to ws[chunk][tile row][tile col][1024] in accumulator order
// (lane-major float4 runs); k_gradw_reduce adds the chunks in order.
constexpr int GW_NT = 512;
constexpr int GW_TOK = 64;                   // tokens per step
constexpr int GW_KS = GW_TOK / 16;           // matrix-core k-steps per step
constexpr int GW_XOFF = GW_TOK * 512;        // bytes of a stage's G part (then X)
constexpr int GW_STAGE = 2 * GW_XOFF;        // one stage: 64 KB
constexpr int GW_NSTG = 2;
constexpr int GW_DMA = GW_TOK / 16;          // DMA instructions per wave and part

struct GradWDims {
    int64_t M, ldg, ldx, N, K;
    int32_t n_tile_rows, n_tile_cols, n_groups, n_wcols;
    int64_t chunk_rows;
    int32_t n_chunks;
    int32_t per_xcd;  // items per XCD (the grid is 8 per_xcd workgroups)
};

__device__ inline int gw_swz(int row) { return (row & 3) | ((row >> 1) & 4); }

__device__ inline uint32_t lds_u32(const void* p)
{
    return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) char*)p);
}

// 16 bytes per lane from a per-lane global address into LDS at M0 + 16 lane.
__device__ inline void gw_dma(const void* src, uint32_t m0)
{
    asm volatile(
        "s_nop 0\n"
        "global_load_lds_dwordx4 %0, off"
        :
        : "v"(src), "{m0}"(m0)
        : "memory");
}

// The same from a wave-uniform base (saddr) and a per-lane 32-bit offset.
__device__ inline void gw_dma_off(const char* base, uint32_t off, uint32_t m0)
{
    asm volatile(
        "s_nop 0\n"
        "global_load_lds_dwordx4 %0, %1"
        :
        : "v"(off), "s"(base), "{m0}"(m0)
        : "memory");
}

typedef short v4s __attribute__((ext_vector_type(4)));

__device__ inline v4s tr_read(uint32_t addr)
{
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) v4s*)(uintptr_t)addr);
}

template <int DT>
__global__ __launch_bounds__(GW_NT, 1) void k_gradw_tiles(const GradWDims d,
                                                          const int32_t* __restrict__ step_ptr,
                                                          const int32_t* __restrict__ step_col,
                                                          const int32_t* __restrict__ step_bits,
                                                          const char* __restrict__ G,
                                                          const char* __restrict__ X,
                                                          float* __restrict__ ws)
{
    using E = Elem<DT>;
    using F = typename E::frag;
    __shared__ uint4 smem[GW_NSTG * GW_STAGE / 16];
    __shared__ uint32_t s_mask[2];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // Items (chunk, window), chunk-major with window columns fastest, are
    // dealt to XCDs in contiguous runs (workgroup b runs on XCD b % 8): the
    // items that share a chunk's rows of G and X then mostly share one L2, and
    // a chunk whose items fall on two XCDs splits between groups, so that
    // each group's slice of G is still read by about one XCD.
    const int n_win = d.n_groups * d.n_wcols;
    const int item = (int)(blockIdx.x & 7) * d.per_xcd + (int)(blockIdx.x >> 3);
    if (item >= n_win * d.n_chunks)
        return;
    const int chunk = item / n_win, win = item - chunk * n_win;
    const int g = win / d.n_wcols, wc = win - g * d.n_wcols;
    const int64_t m_begin = (int64_t)chunk * d.chunk_rows;
    const int64_t m_end = min(d.M, m_begin + d.chunk_rows);

    // the window's kept tiles: bit 8 j + c for tile row j, tile column c
    if (tid < 64) {
        uint64_t bits = 0;
        const int s0 = step_ptr[g], s1 = step_ptr[g + 1];
        for (int s = s0 + lane; s < s1; s += 64) {
            const int c = step_col[s] - 8 * wc;
            if (c >= 0 && c < 8) {
                const int rb = step_bits[s];
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    if ((rb >> j) & 1)
                        bits |= (uint64_t)1 << (8 * j + c);
            }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            const uint32_t lo = __shfl_xor((uint32_t)bits, o, 64);
            const uint32_t hi = __shfl_xor((uint32_t)(bits >> 32), o, 64);
            bits |= (uint64_t)lo | ((uint64_t)hi << 32);
        }
        if (lane == 0) {
            s_mask[0] = (uint32_t)bits;
            s_mask[1] = (uint32_t)(bits >> 32);
        }
    }
    __syncthreads();
    const uint64_t wmask = (uint64_t)__builtin_amdgcn_readfirstlane(s_mask[0]) |
                           ((uint64_t)__builtin_amdgcn_readfirstlane(s_mask[1]) << 32);
    const int n_kept = __popcll(wmask);
    if (n_kept == 0 || m_begin >= m_end)
        return;  // uniform for the whole workgroup
    // This wave's tile row: rows ranked by kept count (descending, ties by
    // index); SIMD k (waves k and k + 4) takes the rows of rank k and 7 - k,
    // which balances the matrix-core work of the SIMDs.
    const int my_rank = wave < 4 ? wave : 11 - wave;
    int tj = 0;
    for (int j = 0; j < 8; ++j) {
        const int cj = __popc((uint32_t)(wmask >> (8 * j)) & 0xffu);
        int rank = 0;
        for (int i = 0; i < 8; ++i) {
            const int ci = __popc((uint32_t)(wmask >> (8 * i)) & 0xffu);
            rank += (ci > cj) || (ci == cj && i < j);
        }
        if (rank == my_rank)
            tj = j;
    }
    // (wave-uniform values, kept in scalar registers: every per-tile test
    // below is then one scalar compare and branch, not a lane mask)
    tj = __builtin_amdgcn_readfirstlane(tj);
    const uint32_t rowbits = __builtin_amdgcn_readfirstlane((uint32_t)(wmask >> (8 * tj)) & 0xffu);
    const int n_w = __builtin_amdgcn_readfirstlane(__popc(rowbits));
    int tc[8];  // the row's kept tile columns, ascending
    {
        uint32_t rest = rowbits;
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            tc[t] = __builtin_amdgcn_readfirstlane(rest ? __builtin_ctz(rest) : 0);
            rest &= rest - 1;
        }
    }

    // DMA: wave w fills rows 8w .. 8w + 7 of the G and the X part of a stage
    // (four 1 KB instructions each, two rows apiece); LDS chunk q (16 bytes)
    // of row r holds columns 32 (seg ^ swz(r)) + 8 (q % 4) .. + 7 with
    // seg = q / 4.
    const uint32_t smem0 = lds_u32(smem);
    int drow[GW_DMA];
    int64_t gcol[GW_DMA], xcol[GW_DMA];
    uint32_t gvo[GW_DMA], xvo[GW_DMA];  // byte offsets within a token step's rows
#pragma unroll
    for (int i = 0; i < GW_DMA; ++i) {
        drow[i] = (GW_TOK / 8) * wave + 2 * i + (lane >> 5);
        const int q = lane & 31;
        const int col = 32 * ((q >> 2) ^ gw_swz(drow[i])) + 8 * (q & 3);
        gcol[i] = min((int64_t)g * 256 + col, d.N - 8);  // past the edge: any valid
        xcol[i] = min((int64_t)wc * 256 + col, d.K - 8);  // columns (never kept)
        // (fit 32 bits: 64 rows of a leading dimension of at most 2^22)
        gvo[i] = (uint32_t)((drow[i] * d.ldg + gcol[i]) * 2);
        xvo[i] = (uint32_t)((drow[i] * d.ldx + xcol[i]) * 2);
    }
    const int64_t n_steps = (m_end - m_begin + GW_TOK - 1) / GW_TOK;
    const char* g0 = G + m_begin * d.ldg * 2;
    const char* x0 = X + m_begin * d.ldx * 2;
    const int64_t g_step = (int64_t)GW_TOK * d.ldg * 2, x_step = (int64_t)GW_TOK * d.ldx * 2;
    // issue the DMA of token step st into its stage: a step whose rows all
    // lie in the chunk from a wave-uniform row base and the fixed per-lane
    // offsets; the chunk's last, partial step row by row (rows past the chunk
    // read the zero line for G, and X rows past M repeat the last)
    auto dma_step = [&](int64_t st) {
        const uint32_t base = smem0 + (uint32_t)(st % GW_NSTG) * GW_STAGE +
                              (uint32_t)wave * (GW_TOK / 8) * 512;
        if (m_begin + (st + 1) * GW_TOK <= m_end) {
            const char* gb = g0 + st * g_step;
            const char* xb = x0 + st * x_step;
#pragma unroll
            for (int i = 0; i < GW_DMA; ++i) {
                gw_dma_off(gb, gvo[i], base + i * 1024);
                gw_dma_off(xb, xvo[i], base + GW_XOFF + i * 1024);
            }
            return;
        }
#pragma unroll
        for (int i = 0; i < GW_DMA; ++i) {
            const int64_t m = m_begin + st * GW_TOK + drow[i];
            const char* gs = m < m_end ? G + (m * d.ldg + gcol[i]) * 2 : (const char*)g_zero_line;
            const char* xs = X + (min(m, d.M - 1) * d.ldx + xcol[i]) * 2;
            gw_dma(gs, base + i * 1024);
            gw_dma(xs, base + GW_XOFF + i * 1024);
        }
    };

    // Transposed operand reads.  Fragment (k-step ks, half h) of lane (q16 =
    // lane / 16, j16 = lane % 16) is row 16 ks + 8 (q16 / 2) + 4 h + j16 / 4,
    // byte 32 (q16 % 2) + 8 (j16 % 4) of its 64-byte segment; the segment (the
    // tile row for G, the tile column for X) sits at (seg ^ swz(row)) 64, and
    // swz(row) = j16 / 4 + 4 (q16 / 2) is the same for all of the lane's rows.
    // So each fragment is a per-lane base (per kept tile, fixed for the whole
    // chunk) plus the stage and the constant 8192 ks + 2048 h.
    const int q16 = lane >> 4, j16 = lane & 15;
    const uint32_t sw = (uint32_t)((j16 >> 2) | ((q16 >> 1) << 2));
    const uint32_t r0 = (uint32_t)((8 * (q16 >> 1) + (j16 >> 2)) * 512 + 32 * (q16 & 1) + 8 * (j16 & 3));
    auto frag = [&](uint32_t addr, int ks) {
        const v4s lo4 = tr_read(addr + ks * 8192);
        const v4s hi4 = tr_read(addr + ks * 8192 + 2048);
        const v4s both[2] = {lo4, hi4};
        return __builtin_bit_cast(F, both);
    };

    // prologue: step 0
    dma_step(0);
    // the token steps, with the row's kept-tile count NW a compile-time
    // constant (one copy of the loop per count): no per-tile test in the loop
    auto steps = [&](auto nw_c) {
        constexpr int NW = decltype(nw_c)::value;
        constexpr int NA = NW > 0 ? NW : 1;
        const uint32_t ga = r0 + (((uint32_t)tj ^ sw) << 6);
        uint32_t xa[NA];
#pragma unroll
        for (int t = 0; t < NA; ++t)
            xa[t] = r0 + GW_XOFF + (((uint32_t)tc[t] ^ sw) << 6);
        f32x16 acc[NA];
#pragma unroll
        for (int t = 0; t < NA; ++t)
            acc[t] = f32x16{};
        for (int64_t st = 0; st < n_steps; ++st) {
            // step st's DMA (the wave's only one in flight) has landed; the
            // barrier publishes it to everyone and frees the stage of step
            // st - 1, which then receives step st + 1
            asm volatile("s_waitcnt vmcnt(0)\n s_barrier" ::: "memory");
            if (st + 1 < n_steps)
                dma_step(st + 1);
            const uint32_t stage = smem0 + (uint32_t)(st % GW_NSTG) * GW_STAGE;
            // one G fragment for the row and one X fragment per kept tile;
            // those of k-step ks + 1 are read before k-step ks's products
            F a[2], b[2][NA];
            a[0] = frag(stage + ga, 0);
#pragma unroll
            for (int t = 0; t < NW; ++t)
                b[0][t] = frag(stage + xa[t], 0);
#pragma unroll
            for (int ks = 0; ks < GW_KS; ++ks) {
                if (ks + 1 < GW_KS) {
                    a[(ks + 1) & 1] = frag(stage + ga, ks + 1);
#pragma unroll
                    for (int t = 0; t < NW; ++t)
                        b[(ks + 1) & 1][t] = frag(stage + xa[t], ks + 1);
                }
                // (the scheduler keeps the reads above ahead of the products)
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int t = 0; t < NW; ++t)
                    acc[t] = E::mma(a[ks & 1], b[ks & 1][t], acc[t]);
            }
        }
        // partials of this chunk
#pragma unroll
        for (int t = 0; t < NW; ++t) {
            const int64_t tile = (int64_t)(8 * g + tj) * d.n_tile_cols + (8 * wc + tc[t]);
            float* dst = ws + ((int64_t)chunk * d.n_tile_rows * d.n_tile_cols + tile) * 1024;
#pragma unroll
            for (int qq = 0; qq < 4; ++qq) {
                const float4 v = {acc[t][4 * qq], acc[t][4 * qq + 1], acc[t][4 * qq + 2],
                                  acc[t][4 * qq + 3]};
                *(float4*)(dst + qq * 256 + lane * 4) = v;
            }
        }
    };
    switch (n_w) {
    case 0: steps(std::integral_constant<int, 0>{}); break;
    case 1: steps(std::integral_constant<int, 1>{}); break;
    case 2: steps(std::integral_constant<int, 2>{}); break;
    case 3: steps(std::integral_constant<int, 3>{}); break;
    case 4: steps(std::integral_constant<int, 4>{}); break;
    case 5: steps(std::integral_constant<int, 5>{}); break;
    case 6: steps(std::integral_constant<int, 6>{}); break;
    case 7: steps(std::integral_constant<int, 7>{}); break;
    default: steps(std::integral_constant<int, 8>{}); break;
    }
}

// out[p][i][j] (BSR order) = the chunks' partials of element (n, k) =
// (r b_r + i, c b_c + j) added in chunk order, rounded once.  Accumulator
// order inside a 32 x 32 tile: element (nn, kk) is lane kk + 32 ((nn / 4) % 2),
// register 4 (nn / 8) + nn % 4.
template <int DT>
__global__ __launch_bounds__(256) void k_gradw_reduce(int32_t b_r, int32_t b_c, int32_t R,
                                                      const int32_t* __restrict__ row_ptr,
                                                      const int32_t* __restrict__ col_idx,
                                                      int64_t total, int32_t n_tile_cols,
                                                      int64_t chunk_stride, int32_t n_chunks,
                                                      const float* __restrict__ ws,
                                                      char* __restrict__ out)
{
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= total)
        return;
    const int nb = b_r * b_c;
    const int64_t p = idx / nb;
    const int e = (int)(idx - p * nb);
    const int r = block_row(row_ptr, R, p), c = col_idx[p];
    const int i = e / b_c, j = e - i * b_c;
    const int64_t n = (int64_t)r * b_r + i, k = (int64_t)c * b_c + j;
    const int nn = (int)(n & 31), kk = (int)(k & 31);
    const int64_t off = ((n >> 5) * n_tile_cols + (k >> 5)) * 1024 + (nn >> 3) * 256 +
                        (kk + 32 * ((nn >> 2) & 1)) * 4 + (nn & 3);
    float s = 0.0f;
    for (int ch = 0; ch < n_chunks; ++ch)
        s += ws[ch * chunk_stride + off];
    store_elem<DT>(out, idx, s);
}

int device_cus()
{
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
        return 256;
    return n;
}

}  // namespace

hipError_t launch_transpose_blocks(const lpv_bsr* h, void* WT, int64_t ldwt, uint8_t* maskT,
                                   hipStream_t s)
{
    const int es = h->dtype == LPV_F32 ? 4 : 2;
    if (h->R > 0)
        hipLaunchKernelGGL(k_transpose_blocks, dim3(h->R), dim3(256), 0, s, h->b_r, h->b_c, h->R,
                           es, (const int32_t*)h->row_ptr, (const int32_t*)h->col_idx,
                           (const char*)h->values, (char*)WT, ldwt, maskT);
    return hipGetLastError();
}

namespace {

// Token chunks of the bias gradient: about 512 workgroups (two per compute
// unit), at least 64 rows each, and at most max_chunks.
int64_t bias_chunks(int64_t M, int64_t N, int V, int64_t max_chunks, int64_t* rows)
{
    // (64-bit comparisons written out: the host min/max overloads of the HIP
    // headers may narrow to int)
    const int64_t bx = (N + 256 * V - 1) / (256 * V);
    int64_t n_chunks = (512 + bx - 1) / bx;
    if (n_chunks > max_chunks)
        n_chunks = max_chunks;
    if (n_chunks > (M + 63) / 64)
        n_chunks = (M + 63) / 64;
    if (n_chunks < 1)
        n_chunks = 1;
    *rows = (M + n_chunks - 1) / n_chunks;
    return M > 0 ? (M + *rows - 1) / *rows : 0;
}

// The two kernels of the bias gradient with the partial sums in `part`
// (n_chunks x N floats, every entry written before it is read).
hipError_t bias_grad_kernels(const void* G, int64_t ldg, int64_t M, int64_t N, int dtype,
                             void* db, float* part, int64_t n_chunks, int64_t rows, hipStream_t s)
{
    const int V = dtype == LPV_F32 ? 4 : 8;
    const int64_t bx = (N + 256 * V - 1) / (256 * V);
    if (n_chunks > 0) {
#define LPV_BIAS(DT_)                                                                            \
    hipLaunchKernelGGL(k_bias_partial<DT_>, dim3((unsigned)bx, (unsigned)n_chunks), dim3(256), 0, \
                       s, (const char*)G, ldg, M, N, rows, part)
        if (dtype == LPV_BF16)
            LPV_BIAS(LPV_BF16);
        else if (dtype == LPV_F16)
            LPV_BIAS(LPV_F16);
        else
            LPV_BIAS(LPV_F32);
#undef LPV_BIAS
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
    }
    const dim3 grid((unsigned)((N + 31) / 32));
    if (dtype == LPV_BF16)
        hipLaunchKernelGGL(k_bias_reduce<LPV_BF16>, grid, dim3(256), 0, s, part, (int)n_chunks, N, (char*)db);
    else if (dtype == LPV_F16)
        hipLaunchKernelGGL(k_bias_reduce<LPV_F16>, grid, dim3(256), 0, s, part, (int)n_chunks, N, (char*)db);
    else
        hipLaunchKernelGGL(k_bias_reduce<LPV_F32>, grid, dim3(256), 0, s, part, (int)n_chunks, N, (char*)db);
    return hipGetLastError();
}

// Scratch of lpv_bias_grad_noalloc: the partial sums live in this file-scope
// device array instead of an allocation.  Host code never uses the array's
// name as an address: each device's address comes from hipGetSymbolAddress
// on that device's first call and is kept in scratch_ptr.
static __device__ __align__(256) float scratch[BIAS_NOALLOC_SCRATCH_FLOATS];

constexpr int MAX_DEVICES = 64;
float* scratch_ptr[MAX_DEVICES];
std::once_flag scratch_once[MAX_DEVICES];
hipError_t scratch_err[MAX_DEVICES];

}  // namespace

hipError_t launch_bias_grad(const void* G, int64_t ldg, int64_t M, int64_t N, int dtype, void* db,
                            hipStream_t s)
{
    int64_t rows = 0;
    const int64_t n_chunks = bias_chunks(M, N, dtype == LPV_F32 ? 4 : 8, (int64_t)1 << 40, &rows);
    float* part = nullptr;
    hipError_t e = hipMallocAsync((void**)&part, (size_t)(max(n_chunks, (int64_t)1) * N) * sizeof(float), s);
    if (e != hipSuccess)
        return e;
    e = bias_grad_kernels(G, ldg, M, N, dtype, db, part, n_chunks, rows, s);
    const hipError_t ef = hipFreeAsync(part, s);
    return e != hipSuccess ? e : ef;
}

hipError_t launch_bias_grad_noalloc(const void* G, int64_t ldg, int64_t M, int64_t N, int dtype,
                                    void* db, hipStream_t s)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= MAX_DEVICES)
        return hipErrorInvalidDevice;
    // once per device, with that device current (it is: hipGetDevice above)
    std::call_once(scratch_once[dev], [dev]() {
        void* p = nullptr;
        scratch_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        scratch_ptr[dev] = scratch_err[dev] == hipSuccess ? (float*)p : nullptr;
    });
    if (scratch_err[dev] != hipSuccess)
        return scratch_err[dev];
    int64_t rows = 0;
    const int64_t n_chunks = bias_chunks(M, N, dtype == LPV_F32 ? 4 : 8,
                                         BIAS_NOALLOC_SCRATCH_FLOATS / N, &rows);
    return bias_grad_kernels(G, ldg, M, N, dtype, db, scratch_ptr[dev], n_chunks, rows, s);
}

// Token chunks of the weight gradient: about one workgroup per compute unit
// over the (group, 8-column window) pairs, at most ceil(M / GW_TOK).
static int64_t grad_w_chunk_cap(const lpv_bsr* h)
{
    const int64_t n_win = (int64_t)h->n_groups * ((h->n_tile_cols + 7) / 8);
    return max((int64_t)1, (int64_t)device_cus() / n_win);
}

size_t grad_w_workspace_bytes(const lpv_bsr* h)
{
    if (h->dtype == LPV_F32 || h->nnzb == 0)
        return 0;
    return (size_t)(grad_w_chunk_cap(h) * (int64_t)h->n_tile_rows * h->n_tile_cols * 1024) *
           sizeof(float);
}

hipError_t launch_grad_w(const lpv_bsr* h, const GradWCall& c, hipStream_t s)
{
    if (h->nnzb == 0)
        return hipSuccess;
    const int64_t nb = (int64_t)h->b_r * h->b_c;
    const int64_t total = h->nnzb * nb;
    if (c.M == 0) {
        // no tokens: every kept-block gradient is zero
        return hipMemsetAsync(c.dW, 0, (size_t)total * (h->dtype == LPV_F32 ? 4 : 2), s);
    }
    if (h->dtype == LPV_F32) {
        hipLaunchKernelGGL(k_gradw_plain<LPV_F32>, dim3((unsigned)h->nnzb), dim3(256), 0, s, h->b_r,
                           h->b_c, h->R, (const int32_t*)h->row_ptr, (const int32_t*)h->col_idx,
                           (const char*)c.G, c.ldg, (const char*)c.X, c.ldx, c.M, (char*)c.dW);
        return hipGetLastError();
    }
    GradWDims d = {};
    d.M = c.M;
    d.ldg = c.ldg;
    d.ldx = c.ldx;
    d.N = h->N;
    d.K = h->K;
    d.n_tile_rows = h->n_tile_rows;
    d.n_tile_cols = h->n_tile_cols;
    d.n_groups = h->n_groups;
    d.n_wcols = (h->n_tile_cols + 7) / 8;
    const int64_t n_win = (int64_t)d.n_groups * d.n_wcols;
    // about one workgroup per compute unit; chunks of whole token steps
    int64_t n_chunks = grad_w_chunk_cap(h);
    n_chunks = min(n_chunks, (c.M + GW_TOK - 1) / GW_TOK);
    d.chunk_rows = ((c.M + n_chunks - 1) / n_chunks + GW_TOK - 1) / GW_TOK * GW_TOK;
    d.n_chunks = (int32_t)((c.M + d.chunk_rows - 1) / d.chunk_rows);
    const int64_t chunk_stride = (int64_t)d.n_tile_rows * d.n_tile_cols * 1024;
    float* ws = c.ws;  // the handle's workspace: n_chunks <= grad_w_chunk_cap(h)
    if (!ws)
        return hipErrorInvalidValue;
    hipError_t e = hipSuccess;
    d.per_xcd = (int32_t)((n_win * d.n_chunks + 7) / 8);
    const dim3 grid((unsigned)(8 * d.per_xcd)), block(GW_NT);
    const dim3 rgrid((unsigned)((total + 255) / 256));
    if (h->dtype == LPV_BF16) {
        hipLaunchKernelGGL(k_gradw_tiles<LPV_BF16>, grid, block, 0, s, d, (const int32_t*)h->step_ptr,
                           (const int32_t*)h->step_col, (const int32_t*)h->step_bits,
                           (const char*)c.G, (const char*)c.X, ws);
        e = hipGetLastError();
        if (e == hipSuccess)
            hipLaunchKernelGGL(k_gradw_reduce<LPV_BF16>, rgrid, dim3(256), 0, s, h->b_r, h->b_c,
                               h->R, (const int32_t*)h->row_ptr, (const int32_t*)h->col_idx,
                               total, d.n_tile_cols, chunk_stride, d.n_chunks, ws, (char*)c.dW);
    } else {
        hipLaunchKernelGGL(k_gradw_tiles<LPV_F16>, grid, block, 0, s, d, (const int32_t*)h->step_ptr,
                           (const int32_t*)h->step_col, (const int32_t*)h->step_bits,
                           (const char*)c.G, (const char*)c.X, ws);
        e = hipGetLastError();
        if (e == hipSuccess)
            hipLaunchKernelGGL(k_gradw_reduce<LPV_F16>, rgrid, dim3(256), 0, s, h->b_r, h->b_c,
                               h->R, (const int32_t*)h->row_ptr, (const int32_t*)h->col_idx,
                               total, d.n_tile_cols, chunk_stride, d.n_chunks, ws, (char*)c.dW);
    }
    if (e == hipSuccess)
        e = hipGetLastError();
    return e;
}

}  // namespace lpv
