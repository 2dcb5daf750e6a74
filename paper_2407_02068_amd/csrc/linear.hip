// linear.hip -- Y = g(X W~^T + b): the block-sparse hot path and the dense
// reference path.
//
// bf16 / fp16 (matrix cores).  The work is cut into items: one tile of BM = 256
// tokens times one group of GROUP_TILES = 8 tile rows (256 output features).
// An item walks its group's steps -- the 32-wide reduction columns where any
// of its rows keeps a tile; other columns are never touched -- so its work is
// proportional to the kept tiles, the quantity the paper's cost model counts
// (Sec. 3.4).
//
// One persistent workgroup of 8 waves per compute unit takes items in turn
// (consecutive items, which share a token tile, go to workgroups on the same
// XCD so the X slice is fetched from HBM once per XCD L2).  Its steps, across
// item boundaries, flow through a 4-slot LDS ring:
//   - gfx950 global->LDS DMA (global_load_lds_dwordx4) stages each step's X
//     slice [256 tokens x 32 columns] and kept W tiles, 3 steps ahead, with
//     16-byte coalesced loads and no registers in between; every wave issues
//     the same number of DMA instructions per step (rows or tiles past the
//     operands read a zero line), so a fixed vmcnt wait tells a wave that its
//     part of a step has landed, and one barrier per step tells everyone;
//   - wave (m, h) takes tokens [64m, 64m + 64) and tile rows [4h, 4h + 4) of
//     the group and issues v_mfma_f32_32x32x16 (bf16 / fp16 in, float32
//     accumulate) for each kept tile; the two waves of a SIMD cover both row
//     halves, so every SIMD gets the step's whole kept count.
// The epilogue adds the bias (scalar loads), applies GELU if asked, rounds once
// to the element type and stores Y straight from the accumulators, while the
// DMA of the next item's first steps is already in flight.
//
// MFMA operand roles: A = a W tile (rows = output features), B = X slice
// transposed (columns = tokens), so D[n][token]: lane l holds token l % 32 and,
// per group of 4 accumulator registers, 4 consecutive output features.
//
// The dense path is the same kernel with every tile kept and W read straight
// from its row-major layout.  fp32 runs a plain VALU kernel over the canonical
// BSR arrays (it serves the small fp32 configuration only).
#include "lpv_device.h"
#include "lpv_internal.h"

namespace lpv {
namespace {

constexpr int NT = 512;             // threads per workgroup: 8 waves
constexpr int G = GROUP_TILES;      // tile rows per item
constexpr int NS = 4;               // LDS ring slots
constexpr int D = NS - 1;           // DMA runs D steps ahead of the matrix cores
constexpr int XU4 = BM * 4;         // 16-byte chunks of one X slice (256 x 32 elements)
constexpr int WU4 = G * 128;        // 16-byte chunks of G W tiles (32 x 32 elements each)
constexpr int SLOT = XU4 + WU4;     // one ring slot: 32 KB
constexpr int NSTORE = 16;          // store instructions per wave per item
constexpr int EPI_U4 = 64 * 4;      // per-wave epilogue tile: 64 rows x 64 bytes
constexpr int LPS = 4;              // DMA instructions per wave per step (2 X + 2 W)
constexpr int WAIT_A = LPS * (D - 2);        // DMA still allowed in flight at a step's barrier
constexpr int WAIT_B = WAIT_A + NSTORE;      // ... when an item's stores were issued since

static_assert(XU4 == 2 * 8 * 64 && WU4 == 2 * 8 * 64, "2 X and 2 W DMA instructions per wave");
static_assert((NS * SLOT + 8 * EPI_U4) * 16 <= 163840, "LDS budget of one workgroup");

// A zero line for DMA lanes outside X (token or column tails), and a sink for
// store lanes outside Y: the instruction count of a wave never depends on
// where the operands end.
static __device__ uint4 g_zero[1];
static __device__ uint4 g_sink[64];

// Sizes of one call (the arrays are separate __restrict__ kernel arguments,
// so the schedule and bias reads can go through the scalar cache).
struct Dims {
    int64_t ldx, M, K, N, ldw, ldy;
    int32_t n_groups, n_tile_rows, n_tile_cols, n_items;
};

struct Args {
    Dims d;
    const char* X;
    const uint4* stream;       // sparse operand stream
    const int32_t* step_ptr;
    const int2* step_meta;
    const int32_t* group_order;
    const char* W;             // dense weight
    const char* bias;
    char* Y;
};

typedef __attribute__((address_space(3))) void* lds_ptr;

__device__ inline void dma16(const void* src, uint4* lds_wave_base)
{
    __builtin_amdgcn_global_load_lds(src, (lds_ptr)lds_wave_base, 16, 0, 0);
}

// s_waitcnt vmcnt(n) lgkmcnt(0) (gfx9 encoding; expcnt left alone)
template <int N> __device__ inline void wait_vm_lgkm0()
{
    static_assert(N < 64, "vmcnt is 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14));
}

// The same with a wave-uniform count: s_waitcnt only takes an immediate, so
// dispatch over the counts the ring can produce (larger ones wait for more,
// which is always safe).
__device__ inline void wait_vm_lgkm0_dyn(int n)
{
#define LPV_W(N)                  \
    case N:                       \
        wait_vm_lgkm0<N>();       \
        break;
    switch (n) {
        LPV_W(0) LPV_W(1) LPV_W(2) LPV_W(3) LPV_W(4) LPV_W(5) LPV_W(6) LPV_W(7) LPV_W(8)
        LPV_W(9) LPV_W(10) LPV_W(11) LPV_W(12) LPV_W(13) LPV_W(14) LPV_W(15) LPV_W(16)
        LPV_W(17) LPV_W(18) LPV_W(19) LPV_W(20) LPV_W(21) LPV_W(22) LPV_W(23) LPV_W(24)
        LPV_W(25) LPV_W(26) LPV_W(27) LPV_W(28)
    default:
        wait_vm_lgkm0<28>();
        break;
    }
#undef LPV_W
}

__device__ inline void barrier_step()
{
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// 16-byte LDS read issued from inline assembly: the compiler then does not
// treat it as a read of LDS that the in-flight DMA may be writing (it would
// otherwise drain all DMA before every read).  The ring protocol (vmcnt wait +
// barrier per step) is what orders these reads after the DMA that fills them,
// and lds_wait() below after the reads themselves.
typedef int v4i __attribute__((ext_vector_type(4)));

__device__ inline uint32_t lds_addr(const void* p)
{
    return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) char*)p);
}

template <int OFF> __device__ inline v4i lds_read16(uint32_t addr)
{
    v4i r;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
    return r;
}

__device__ inline void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

__device__ inline void lds_write8(uint32_t addr, uint2 v)
{
    asm volatile("ds_write_b64 %0, %1" : : "v"(addr), "v"(v) : "memory");
}

// After lds_wait(): tie a value read by lds_read16 to that point, so its uses
// cannot move above the wait.
__device__ inline void after_wait(v4i& a) { asm volatile("" : "+v"(a)); }

// X slice layout in LDS: chunk (row r, 16-byte column chunk ch) at r * 4 + (ch ^ swz(r)).
__device__ inline int xswz(int r) { return (r >> 1) & 3; }
// Epilogue tile layout (64 rows of 64 bytes): chunk c of row r at c ^ eswz(r).
__device__ inline int eswz(int r) { return (r >> 1) & 3; }

template <int DT, bool GELU, bool DENSE, bool KTAIL>
__global__ __launch_bounds__(NT, 1) void k_linear16(
    const Dims a, const char* __restrict__ X, const uint4* __restrict__ stream,
    const int32_t* __restrict__ step_ptr, const int2* __restrict__ step_meta,
    const int32_t* __restrict__ group_order, const char* __restrict__ W,
    const uint32_t* __restrict__ bias32, char* __restrict__ Y)
{
    using E = Elem<DT>;
    using F = typename E::frag;
    __shared__ uint4 smem[NS * SLOT + NT / 64 * EPI_U4];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave
    const int wm = wave & 3, wh = wave >> 2;

    // this workgroup's items: k * P + item_off, k = 0, 1, ...
    const int P = (int)gridDim.x;
    const int item_off = (int)(blockIdx.x & 7) * (P >> 3) + (int)(blockIdx.x >> 3);
    const int my_items = item_off < a.n_items ? (a.n_items - item_off + P - 1) / P : 0;
    if (my_items == 0)
        return;

    const char* zero = (const char*)g_zero;
    const int last_col = a.n_tile_cols - 1;
    const uint32_t smem0 = lds_addr(smem);

    // Per-lane constants of this wave's DMA instructions.  X: LDS chunk p of
    // the slice holds row p / 4, column chunk (p % 4) ^ swz(row).  W: chunk q
    // of the step's operand-order tiles (dense: tile q / 128, lane q % 64 of
    // k-step (q / 64) % 2).
    int xrow[2], xcol[2], wrow[2], wcol[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int p = (wave * 2 + i) * 64 + lane;
        xrow[i] = p >> 2;
        xcol[i] = ((p & 3) ^ xswz(p >> 2)) * 8;
        wrow[i] = (p >> 7) * TILE + (p & 31);
        wcol[i] = ((p >> 6) & 1) * 16 + ((p >> 5) & 1) * 8;
    }

    auto group_of = [&](int k, int& g, int& mt) {
        const int it = k * P + item_off;
        mt = it / a.n_groups;
        const int gs = it - mt * a.n_groups;
        g = DENSE ? gs : group_order[gs];
    };
    auto steps_of = [&](int g, int& s0, int& s1) {
        if (DENSE) {
            s0 = 0;
            s1 = a.n_tile_cols;
        } else {
            s0 = step_ptr[g];
            s1 = step_ptr[g + 1];
        }
    };

    // ---- producer: the DMA cursor runs D steps ahead, across items.  Every
    // wave issues exactly 2 X and 2 W DMA instructions per step: X rows past M
    // repeat row M - 1 (their outputs are never stored); W chunks past the
    // step's kept tiles fetch the tiles that follow (the stream is padded), and
    // land in slot space nobody reads.
    int pk = -1, ps = 0, ps_end = 0;
    const char* xsrc[2];  // X[min(m0 + row, M - 1)][col chunk] at column tile 0
    const char* wsrc[2];  // dense: W[min(g * 256 + row, N - 1)][col chunk]
    auto next_item = [&]() {
        while (++pk < my_items) {
            int g, mt;
            group_of(pk, g, mt);
            steps_of(g, ps, ps_end);
            if (ps < ps_end) {
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    const int64_t m = min((int64_t)mt * BM + xrow[i], a.M - 1);
                    xsrc[i] = X + (m * a.ldx + xcol[i]) * 2;
                    const int64_t n = min((int64_t)g * G * TILE + wrow[i], a.N - 1);
                    wsrc[i] = DENSE ? W + (n * a.ldw + wcol[i]) * 2 : zero;
                }
                return;
            }
        }
    };
    // The DMA of one step: sources and LDS destinations of this wave's 4
    // instructions.  `meta` is step_meta[ps], loaded by the caller ahead of
    // time (sparse only).
    struct Dma {
        const char* src[4];
        uint4* dst[4];
    };
    auto dma_prep = [&](int slot, int2 meta, Dma& d) {
        uint4* xdst = smem + slot * SLOT + wave * 128;
        uint4* wdst = smem + slot * SLOT + XU4 + wave * 128;
        d.dst[0] = xdst;
        d.dst[1] = xdst + 64;
        d.dst[2] = wdst;
        d.dst[3] = wdst + 64;
        if (pk < my_items) {
            const int col = DENSE ? ps : (meta.x & 0xffff);
            const int64_t coff = (int64_t)col * TILE * 2;  // bytes to column tile col
            d.src[0] = xsrc[0] + coff;
            d.src[1] = xsrc[1] + coff;
            if (DENSE) {
                d.src[2] = wsrc[0] + coff;
                d.src[3] = wsrc[1] + coff;
            } else {
                const char* tiles = (const char*)stream + (int64_t)meta.y * 2048 + wave * 2048;
                d.src[2] = tiles + lane * 16;
                d.src[3] = tiles + 1024 + lane * 16;
            }
            if (KTAIL && col == last_col) {  // columns past K read the zero line
                if (col * TILE + xcol[0] >= a.K) d.src[0] = zero;
                if (col * TILE + xcol[1] >= a.K) d.src[1] = zero;
                if (DENSE && col * TILE + wcol[0] >= a.K) d.src[2] = zero;
                if (DENSE && col * TILE + wcol[1] >= a.K) d.src[3] = zero;
            }
        } else {
            // past the last step: the same instruction count, into a free slot
#pragma unroll
            for (int i = 0; i < 4; ++i)
                d.src[i] = zero;
        }
    };
    auto dma_advance = [&]() {
        if (pk < my_items && ++ps >= ps_end)
            next_item();
    };
    auto produce = [&](int slot, int2 meta) {
        Dma d;
        dma_prep(slot, meta, d);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            dma16(d.src[i], d.dst[i]);
        dma_advance();
    };

    next_item();
    int2 pmeta = make_int2(0, 0);  // step_meta at the producer cursor
#pragma unroll
    for (int i = 0; i < D; ++i) {
        if (!DENSE)
            pmeta = pk < my_items ? step_meta[ps] : make_int2(0, 0);
        produce(i, pmeta);
    }
    if (!DENSE)
        pmeta = pk < my_items ? step_meta[ps] : make_int2(0, 0);

    // LDS read addresses of this lane (slot 0; u = 1 is +2048 bytes, W ks = 1 is +1024)
    uint32_t xa_addr[2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        const int r = wm * 64 + (lane & 31);
        const int ch = ks * 2 + (lane >> 5);
        xa_addr[ks] = smem0 + (r * 4 + (ch ^ xswz(r))) * 16;
    }
    const uint32_t wa_addr = smem0 + XU4 * 16 + lane * 16;
    const uint32_t ebase = smem0 + NS * SLOT * 16 + wave * (EPI_U4 * 16);

    // Step 0 has landed everywhere before anyone reads it.
    wait_vm_lgkm0<LPS * (D - 1)>();
    barrier_step();

    f32x16 acc[2][4];
    int t = 0;     // steps consumed
    int e = -16;   // last step of the last item written out
    for (int ck = 0; ck < my_items; ++ck) {
        int g, mt, s0, s1;
        group_of(ck, g, mt);
        steps_of(g, s0, s1);
        const int rows = (1 << min(G, a.n_tile_rows - g * G)) - 1;
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    acc[u][j][v] = 0.0f;

        // One step.  The two waves of a SIMD take turns: group A (row half 0)
        // reads its operands after the step's barrier and then runs the matrix
        // cores; group B (row half 1) reads before the barrier and computes
        // after it, so one wave's LDS reads overlap the other's MFMAs.  Before
        // the barrier of step u every wave has waited for its DMA of step
        // u + 1 (group B reads that step before the next barrier); after it,
        // the slot of step u - 1 is free and is refilled with step u + D.  The
        // wait also covers an epilogue's stores when one was issued after that
        // DMA.  Metadata of the next step is loaded a step ahead.
        int bits = DENSE ? rows : (s0 < s1 ? (step_meta[s0].x >> 16) : 0);
        auto step = [&](int s) {
            const int cur = bits;
            if (!DENSE)
                bits = s + 1 < s1 ? (step_meta[s + 1].x >> 16) : 0;
            const uint32_t slot_off = (uint32_t)(t & (NS - 1)) * (SLOT * 16);
            const int bh = (cur >> (4 * wh)) & 15;
            v4i xa[2][2], wf[4][2];
            auto read_ops = [&]() {
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    xa[0][ks] = lds_read16<0>(xa_addr[ks] + slot_off);
                    xa[1][ks] = lds_read16<2048>(xa_addr[ks] + slot_off);
                }
                uint32_t wa = wa_addr + slot_off + (wh ? __popc(cur & 15) * 2048 : 0);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (bh & (1 << j)) {
                        wf[j][0] = lds_read16<0>(wa);
                        wf[j][1] = lds_read16<1024>(wa);
                        wa += 2048;
                    }
                }
            };
            auto sync = [&]() {
                if (e >= t - 2)
                    wait_vm_lgkm0<WAIT_B>();
                else
                    wait_vm_lgkm0<WAIT_A>();
                barrier_step();
            };
            Dma dm;
            if (wh == 0) {
                sync();
                read_ops();
                dma_prep((t + D) & (NS - 1), pmeta, dm);
                lds_wait();
            } else {
                read_ops();
                lds_wait();
                sync();
                dma_prep((t + D) & (NS - 1), pmeta, dm);
            }
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int ks = 0; ks < 2; ++ks)
                    after_wait(xa[u][ks]);
            // the refill of the freed slot goes out one instruction at a time
            // between the matrix-core instructions
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                dma16(dm.src[j], dm.dst[j]);
                if (bh & (1 << j)) {
                    after_wait(wf[j][0]);
                    after_wait(wf[j][1]);
                    const F w0 = __builtin_bit_cast(F, wf[j][0]);
                    const F w1 = __builtin_bit_cast(F, wf[j][1]);
                    acc[0][j] = E::mma(w0, __builtin_bit_cast(F, xa[0][0]), acc[0][j]);
                    acc[1][j] = E::mma(w0, __builtin_bit_cast(F, xa[1][0]), acc[1][j]);
                    acc[0][j] = E::mma(w1, __builtin_bit_cast(F, xa[0][1]), acc[0][j]);
                    acc[1][j] = E::mma(w1, __builtin_bit_cast(F, xa[1][1]), acc[1][j]);
                }
            }
            dma_advance();
            if (!DENSE)
                pmeta = pk < my_items ? step_meta[ps] : make_int2(0, 0);
            ++t;
        };
        for (int s = s0; s < s1; ++s)
            step(s);
        e = t - 1;

        // ---- epilogue: bias, GELU, one rounding; each wave transposes one
        // 64 x 32 tile at a time through its own 4 KB of LDS, then stores 16
        // bytes per lane, 64 contiguous bytes per row: exactly NSTORE store
        // instructions per wave.  The stores are non-temporal: Y is not read
        // again, and keeping it out of L2 leaves L2 to X and the tile stream.
        const int h = lane >> 5;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t n_tile = (int64_t)(g * G + wh * 4 + j) * TILE;
            uint32_t bw[16];
#pragma unroll
            for (int d = 0; d < 16; ++d)
                bw[d] = 0u;
            if (bias32) {
                if (n_tile + TILE <= a.N) {
#pragma unroll
                    for (int d = 0; d < 16; ++d)
                        bw[d] = bias32[n_tile / 2 + d];
                } else if (n_tile < a.N) {  // ragged last tile row (N % 32 == 16)
#pragma unroll
                    for (int d = 0; d < 8; ++d)
                        bw[d] = bias32[n_tile / 2 + d];
                }
            }
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int r = u * 32 + (lane & 31);  // token row within the wave's 64
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const uint32_t d0 = h ? bw[4 * q + 2] : bw[4 * q];
                    const uint32_t d1 = h ? bw[4 * q + 3] : bw[4 * q + 1];
                    float v[4] = {acc[u][j][4 * q] + E::to_f32(d0 & 0xffff),
                                  acc[u][j][4 * q + 1] + E::to_f32(d0 >> 16),
                                  acc[u][j][4 * q + 2] + E::to_f32(d1 & 0xffff),
                                  acc[u][j][4 * q + 3] + E::to_f32(d1 >> 16)};
                    if (GELU) {
#pragma unroll
                        for (int x = 0; x < 4; ++x)
                            v[x] = gelu_erf(v[x]);
                    }
                    uint2 o;
                    o.x = (uint32_t)E::from_f32(v[0]) | ((uint32_t)E::from_f32(v[1]) << 16);
                    o.y = (uint32_t)E::from_f32(v[2]) | ((uint32_t)E::from_f32(v[3]) << 16);
                    // row r, outputs 8q + 4h .. + 3: 16-byte chunk q ^ eswz(r), half h
                    lds_write8(ebase + r * 64 + ((q ^ eswz(r)) * 16) + h * 8, o);
                }
            }
            v4i ov[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = i * 16 + (lane >> 2), c = lane & 3;
                ov[i] = lds_read16<0>(ebase + r * 64 + ((c ^ eswz(r)) * 16));
            }
            lds_wait();
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                after_wait(ov[i]);
                const int r = i * 16 + (lane >> 2), c = lane & 3;
                const int64_t m = (int64_t)mt * BM + wm * 64 + r;
                const int64_t n = n_tile + c * 8;
                uint4* dst = (m < a.M && n < a.N) ? (uint4*)(Y + (m * a.ldy + n) * 2) : &g_sink[lane];
                __builtin_nontemporal_store(ov[i], (v4i*)dst);
            }
        }
    }
    // no DMA may still be writing this workgroup's LDS when it ends
    __builtin_amdgcn_s_waitcnt(0);
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

inline int num_cus()
{
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
        n = 256;
    return n;
}

template <bool DENSE>
hipError_t launch16(int dtype, bool gelu, const Args& a, hipStream_t s)
{
    if (a.d.n_items <= 0)
        return hipSuccess;
    int P = num_cus() & ~7;
    const int need = (a.d.n_items + 7) / 8 * 8;
    if (P < 8)
        P = 8;
    if (P > need)
        P = need;
    const dim3 grid(P), block(NT);
    const bool ktail = (a.d.K % TILE) != 0;
#define LPV_LAUNCH1(DT_, GELU_, KT_)                                                              \
    hipLaunchKernelGGL((k_linear16<DT_, GELU_, DENSE, KT_>), grid, block, 0, s, a.d, a.X,         \
                       a.stream, a.step_ptr, a.step_meta, a.group_order, a.W,                     \
                       (const uint32_t*)a.bias, a.Y)
#define LPV_LAUNCH(DT_, GELU_)                                                                    \
    do {                                                                                          \
        if (ktail)                                                                                \
            LPV_LAUNCH1(DT_, GELU_, true);                                                        \
        else                                                                                      \
            LPV_LAUNCH1(DT_, GELU_, false);                                                       \
    } while (0)
    if (dtype == LPV_BF16) {
        if (gelu)
            LPV_LAUNCH(LPV_BF16, true);
        else
            LPV_LAUNCH(LPV_BF16, false);
    } else {
        if (gelu)
            LPV_LAUNCH(LPV_F16, true);
        else
            LPV_LAUNCH(LPV_F16, false);
    }
#undef LPV_LAUNCH
#undef LPV_LAUNCH1
    return hipGetLastError();
}

Args base_args(const LinearCall& c, int64_t N, int64_t K)
{
    Args a = {};
    a.d.ldx = c.ldx;
    a.d.M = c.M;
    a.d.K = K;
    a.d.N = N;
    a.d.ldy = c.ldy;
    a.d.n_tile_rows = (int32_t)((N + TILE - 1) / TILE);
    a.d.n_tile_cols = (int32_t)((K + TILE - 1) / TILE);
    a.d.n_groups = (a.d.n_tile_rows + G - 1) / G;
    a.d.n_items = (int32_t)((c.M + BM - 1) / BM) * a.d.n_groups;
    a.X = (const char*)c.X;
    a.bias = (const char*)c.bias;
    a.Y = (char*)c.Y;
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
    a.step_meta = h->step_meta;
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
    a.d.ldw = ldw;
    return launch16<true>(dtype, c.gelu != 0, a, s);
}

}  // namespace lpv
