// linear.hip -- Y = g(X W~^T + b): the block-sparse hot path and the dense
// reference path.
//
// bf16 / fp16 (matrix cores).  The work is cut into items: one tile of BM = 256
// tokens times one group of GROUP_TILES = 8 tile rows (256 output features).
// An item walks its group's steps -- the 32-wide reduction columns where any
// of its rows keeps a tile; other columns are never touched -- so its work is
// proportional to the kept tiles, the quantity the paper's cost model counts
// (Sec. 3.4); with 16-wide block columns (KH) the two 16-column halves of a
// tile are kept or dropped on their own, and only kept halves are loaded and
// multiplied.  The walk starts at a per-group column and wraps around, so the
// groups that work on one token tile at the same time read different X
// columns.
//
// One persistent workgroup of 8 waves per compute unit takes items in turn
// (consecutive items, which share a token tile, go to workgroups on the same
// XCD so the X slice is fetched from HBM once per XCD L2); the items of a
// short last round are cut in two halves of tile rows, each the last item of
// its own workgroup.  Its steps, across item boundaries, go in pairs through
// two LDS pair slots, one barrier per pair:
//   - gfx950 global->LDS DMA (global_load_lds_dwordx4) stages a pair's X
//     slices [256 tokens x 2 x 32 columns] (four instructions per wave) and
//     the pair's kept W tiles (tile j by wave j, two instructions per step),
//     one pair ahead, 16 bytes per lane with no registers in between;
//   - each step's row bits travel from the producer cursor to the consumer in
//     a 64-bit queue (12 bits per step in flight: the wave's own four rows,
//     per 16-column half with KH, and the item's end); the wait before each
//     pair's barrier (vmcnt(0)) covers the next pair's DMA and a finished item's
//     stores, and the barrier tells every wave that the pair landed and that
//     the pair slot read before it is free;
//   - wave (m, h) takes tokens [64m, 64m + 64) and tile rows [4h, 4h + 4) of
//     the group and issues v_mfma_f32_32x32x16 (bf16 / fp16 in, float32
//     accumulate) for each kept tile; the two waves of a SIMD cover both row
//     halves, so every SIMD gets the step's whole kept count.  Each half step
//     reads the next half step's fragments while its own go to the matrix
//     cores; with many groups per token tile (LATE) a pair's last k-step is
//     multiplied after the barrier, over the next pair's first reads.
// The step loop carries no division and no scalar load on its critical path:
// the per-group descriptors (group, first step, step count, first column
// walked) are built at pack time, item coordinates advance by constants, and
// the walk is read one 64-entry segment ahead.
// The epilogue adds the bias (the accumulators start at it), applies GELU if
// asked, rounds once to the element type and stores Y (16 bytes per lane,
// transposed through LDS).  The next item's first pair, whose DMA went out
// during this item's last pair, has landed by then; the stores leave after the
// next barrier, beside the DMA of the pair after it.
//
// MFMA operand roles: A = a W tile (rows = output features), B = X slice
// transposed (columns = tokens), so D[n][token]: lane l holds token l % 32 and,
// per group of 4 accumulator registers, 4 consecutive output features.
//
// The dense path is the same kernel with every tile kept and W read straight
// from its row-major layout into the same slice layout as X.  fp32 runs a plain
// VALU kernel over the canonical BSR arrays (it serves the small fp32
// configuration only).
#include "lpv_device.h"
#include "lpv_internal.h"

namespace lpv {
namespace {

constexpr int NT = 512;             // threads per workgroup: 8 waves
constexpr int G = GROUP_TILES;      // tile rows per item
// Steps go in pairs, one barrier per pair.  The LDS ring has two pair slots:
// after the barrier of pair (b, b + 1) each wave loads steps b + 2 and b + 3
// into the pair slot that held b - 2 and b - 1.  A pair slot holds the X of
// both steps interleaved -- row r of the 256 tokens as 128 bytes, the two
// 64-byte column slices side by side, so that 8 lanes of a DMA instruction
// fetch a whole 128-byte line when the two columns are adjacent -- and the W
// tiles of each step (dense W: the group's 256 rows, interleaved like X).
constexpr int NS = 4;               // steps in flight (two pair slots)
constexpr int XP_U4 = BM * 8;       // 16-byte chunks of a pair's X (256 x 64 elements): 32 KB
constexpr int WS_U4 = G * 128;      // 16-byte chunks of one step's W tiles (8 x 32 x 32): 16 KB
constexpr int PSLOT = XP_U4 + 2 * WS_U4;  // one pair slot: 64 KB
constexpr int TAB_U4 = 2048;        // per-call tables (walk, slot descriptors, bias): 32 KB

static_assert(XP_U4 == 8 * 4 * 64 && WS_U4 == 8 * 2 * 64, "4 X and 2 W DMA instructions per wave");
static_assert((2 * PSLOT + TAB_U4) * 16 <= 163840, "LDS budget of one workgroup");

// A zero line for DMA lanes past K, and a sink for store lanes outside Y.
static __device__ uint4 g_zero[1];
static __device__ uint4 g_sink[64];

struct Dims {
    int64_t ldx, M, K, N, ldw, ldy;
    int32_t n_tile_rows, n_tile_cols, n_groups;
    int32_t gs0, n_slots;   // this launch: launch slots [gs0, gs0 + n_slots) ...
    int32_t n_items;        // ... times every token tile
    int32_t xcd_tiles;      // item order: 1 = each XCD owns whole token tiles
    int32_t p_div, p_mod;   // from one item of a workgroup to its next: token
                            // tiles and launch slots to advance, ...
    int32_t mt_carry;       // ... and token tiles more when the slot wraps
    int32_t walk0, n_walk;  // this launch's slice of the walk array
    int32_t walk_off, bias_off;  // byte offsets of the walk and bias tables in LDS
};

__device__ inline uint32_t lds_addr(const void* p)
{
    return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) char*)p);
}

// Global -> LDS DMA of 16 bytes per lane to 1 KB at a wave-uniform LDS base.
// Issued from inline assembly: the compiler then neither drains this DMA
// before every LDS read of the wave (as it must for the builtin, which it
// knows writes LDS) nor counts it in its own vmcnt waits.  Every wait for it
// is explicit (the ring protocol: vmcnt wait + barrier per step); the memory
// clobber keeps the compiler's LDS reads in program order around it.
__device__ inline void dma16(const void* src, uint4* lds_wave_base)
{
    asm volatile(
        "s_nop 0\n"
        "global_load_lds_dwordx4 %0, off"
        :
        : "v"(src), "{m0}"(lds_addr(lds_wave_base))
        : "memory");
}

// The same from a wave-uniform base and a 32-bit per-lane byte offset (the
// saddr + voffset form: no 64-bit address per lane is kept live).
__device__ inline void dma16(const char* base, uint32_t off, uint4* lds_wave_base)
{
    asm volatile(
        "s_nop 0\n"
        "global_load_lds_dwordx4 %0, %1"
        :
        : "v"(off), "s"(base), "{m0}"(lds_addr(lds_wave_base))
        : "memory");
}

// The same with the instruction offset IMM, which the hardware adds to both
// the global and the LDS address (global: saddr + voff + IMM; LDS: M0 + IMM +
// 16 * lane).  Two DMAs 1 KB apart in LDS share one M0 value this way.
template <int IMM> __device__ inline void dma16i(const char* saddr, uint32_t voff, uint32_t m0)
{
    asm volatile(
        "s_nop 0\n"
        "global_load_lds_dwordx4 %0, %1 offset:%3"
        :
        : "v"(voff), "s"(saddr), "{m0}"(m0), "i"(IMM)
        : "memory");
}

typedef int v4i __attribute__((ext_vector_type(4)));

// 16-byte LDS read at a byte address (an ordinary load: the compiler places
// the lgkmcnt wait before the first use of the value).
template <int OFF> __device__ inline v4i lds_read16(uint32_t addr)
{
    return *(const __attribute__((address_space(3))) v4i*)(uintptr_t)(addr + OFF);
}

__device__ inline void lds_write16(uint32_t addr, v4i v)
{
    *(__attribute__((address_space(3))) v4i*)(uintptr_t)addr = v;
}

// Pair X (and dense W) layout in LDS: chunk ch (0..7: 16 bytes; 0..3 the first
// step's column tile, 4..7 the second's) of row r at r * 8 + (ch ^ swz(r)).
// A 16-byte read by 16 lanes (rows r .. r + 15 of one chunk) then touches 16
// different 16-byte bank groups (the LDS serves 256 bytes per clock).
__device__ inline int xswz(int r) { return (r >> 1) & 7; }

// Walk entry (LDS table): {col | bits << 16 | last step of the item << 24 |
// last entry of its segment << 25, first tile, start of the next segment in
// this grid's item order, group}.  With 16-wide block columns (KH) a kept
// tile's two 16-column halves are kept or dropped on their own: bits are then
// the rows that keep the first half, and the first-tile word carries the rows
// that keep the second half in its top byte.  A slot's walk is cut into segments of at
// most 64 entries; the producer holds one segment in VGPR lanes (lane i =
// entry i) and the next one prefetched, so a step costs two lane reads and no
// memory access.
constexpr int W_LAST = 1 << 24, W_SEG_END = 1 << 25;
constexpr int SEG = 64;
// Queue entry of one step in flight (12 bits, up to 5 in a 64-bit queue): the
// kept rows among the wave's four (bit j: row 4 h + j of the group) for the
// first k-step (bits 0..3) and, with 16-wide block columns, the second (bits
// 4..7; otherwise the first serves both), and the item's last step (bit 8).
constexpr int E_LAST = 1 << 8, E_BITS = 12, E_MASK = (1 << E_BITS) - 1;

template <int DT, bool GELU, bool DENSE, bool KTAIL, bool KH, bool LATE>
__global__ __launch_bounds__(NT, 1) void k_linear16(
    const Dims a, const char* __restrict__ X, const char* __restrict__ stream,
    const int4* __restrict__ gdesc, const int2* __restrict__ walk,
    const char* __restrict__ W, const char* __restrict__ bias, char* __restrict__ Y)
{
    static_assert(!(DENSE && KH), "the dense path keeps whole tiles");
    using E = Elem<DT>;
    using F = typename E::frag;
    __shared__ uint4 smem[2 * PSLOT + TAB_U4];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave
    const int wm = wave & 3, wh = wave >> 2;
    const int wsh = 4 * wh;  // this wave's rows in a group's row bits

    // This workgroup's items.  Items are (token tile, launch slot) pairs,
    // slot-minor; workgroup b runs on XCD x = b % 8 as its c = b / 8-th of
    // C = P / 8.  xcd_tiles: XCD x owns token tiles x, x + 8, ... with all their
    // slots and deals them to its C workgroups in turn (c, c + C, ...), so
    // the items of one token tile share that XCD's L2.  Otherwise item
    // x C + c + k P, k = 0, 1, ...: an XCD's workgroups take C consecutive items.
    //
    // The last round: after R = n_items / P whole rounds the items left over
    // (fewer than one per workgroup) would keep a few workgroups busy while
    // the rest of the chip idles.  When at most half of the workgroups (of the
    // XCD, in the XCD order) would get one, each is cut into its two halves of
    // tile rows (4 hh .. 4 hh + 3 of the group, hh = 0, 1), run as the last
    // item of two workgroups: the same steps, with the other half's row bits
    // cleared, so half the W and half the matrix-core work per SIMD (each
    // SIMD runs one wave of either half), and half the stores.
    const int P = (int)gridDim.x, C = P >> 3;
    const int xcd = (int)(blockIdx.x & 7), cu = (int)(blockIdx.x >> 3);
    const int R = a.n_items / P;
    int first_mt, first_slot, my_items;
    int h_mt = 0, h_slot = 0, hh = -1;  // the half item (row half hh), if any
    if (a.xcd_tiles) {
        const int n_mt = a.n_items / a.n_slots;
        const int n_local = xcd < n_mt ? (n_mt - xcd + 7) / 8 * a.n_slots : 0;
        my_items = cu < n_local ? (n_local - cu + C - 1) / C : 0;
        first_mt = xcd + 8 * (cu / a.n_slots);
        first_slot = cu % a.n_slots;
        const int tail = n_local - C * R;
        if (tail > 0 && 2 * tail <= C) {
            my_items = R;
            if (cu < 2 * tail) {
                const int li = C * R + cu / 2;
                h_mt = xcd + 8 * (li / a.n_slots);
                h_slot = li % a.n_slots;
                hh = cu & 1;
            }
        }
    } else {
        const int item_off = xcd * C + cu;
        my_items = item_off < a.n_items ? (a.n_items - item_off + P - 1) / P : 0;
        first_mt = item_off / a.n_slots;
        first_slot = item_off % a.n_slots;
        const int tail = a.n_items - P * R;
        if (tail > 0 && 2 * tail <= P) {
            my_items = R;
            if (item_off < 2 * tail) {
                const int i = P * R + item_off / 2;
                h_mt = i / a.n_slots;
                h_slot = i % a.n_slots;
                hh = item_off & 1;
            }
        }
    }
    const int n_full = my_items;  // whole items; the half item, if any, comes last
    if (hh >= 0) {
        if (n_full == 0) {
            first_mt = h_mt;
            first_slot = h_slot;
        }
        ++my_items;
    }
    if (my_items == 0)
        return;

    // ---- per-call tables in LDS: slot descriptors {group, first walk entry,
    // walk length}, walk entries, float32 bias of each slot's 256 outputs
    char* tab = (char*)(smem + 2 * PSLOT);
    int4* t_desc = (int4*)tab;
    int4* t_walk = (int4*)(tab + a.walk_off);
    float* t_bias = (float*)(tab + a.bias_off);
    const int ncol = a.n_tile_cols;
    auto rows_of = [&](int g) { return (1 << min(G, a.n_tile_rows - g * G)) - 1; };
    for (int i = tid; i < a.n_slots; i += NT) {
        int4 d;
        if (DENSE) {
            const int nw = (ncol + 1) & ~1;  // an even walk: a step with no tile pads it
            d = make_int4(a.gs0 + i, i * nw, nw, 0);
        } else {
            d = gdesc[a.gs0 + i];
            d.y -= a.walk0;
        }
        t_desc[i] = d;
    }
    __syncthreads();
    for (int i = tid; i < a.n_walk; i += NT) {
        int slot = 0;  // the slot whose walk holds entry i (few slots: linear search)
        while (slot + 1 < a.n_slots && t_desc[slot + 1].y <= i)
            ++slot;
        const int4 d = t_desc[slot];
        const int j = i - d.y;  // position in the slot's walk
        int2 e;
        if (DENSE) {
            // the walk starts at an even column: the pair's two columns then
            // share 128-byte lines of X
            int col = ((int)((int64_t)(a.gs0 + slot) * ncol / a.n_groups) & ~1) + j;
            if (col >= ncol)
                col -= ncol;
            e = make_int2(j < ncol ? col | (rows_of(d.x) << 16) : 0, 0);
            if (j == d.z - 1)
                e.x |= W_LAST;
        } else {
            e = walk[a.walk0 + i];
        }
        const bool seg_end = (j % SEG == SEG - 1) || (j == d.z - 1);
        int next = d.y + (j / SEG + 1) * SEG;  // the slot's next segment ...
        if (j / SEG + 1 >= (d.z + SEG - 1) / SEG) {  // ... or the next item's first
            int ns = slot + a.p_mod;
            if (ns >= a.n_slots)
                ns -= a.n_slots;
            next = t_desc[ns].y;
        }
        t_walk[i] = make_int4(e.x | (seg_end ? W_SEG_END : 0), e.y, next, d.x);
    }
    for (int i = tid; i < a.n_slots * G * TILE; i += NT) {
        const int64_t n = (int64_t)t_desc[i / (G * TILE)].x * G * TILE + i % (G * TILE);
        t_bias[i] = (bias && n < a.N) ? E::to_f32(((const uint16_t*)bias)[n]) : 0.0f;
    }
    __syncthreads();

    const char* zero = (const char*)g_zero;
    const uint32_t smem0 = lds_addr(smem);
    const uint32_t walk_lds = lds_addr(t_walk), desc_lds = lds_addr(t_desc), bias_lds = lds_addr(t_bias);

    // Per-lane constants of this wave's pair DMA (X, dense W): instruction i
    // fills rows 32 wave + 8 i .. + 7 (1 KB); lane l writes chunk position
    // l % 8 of row 32 wave + 8 i + l / 8, which holds chunk ch = (l % 8) ^
    // swz(row): columns (ch % 4) * 8 .. + 7 of the first (ch < 4) or second
    // step's column tile.
    int srow[4], scol[4];
    uint32_t sel2 = 0;  // bit i: instruction i's lane fetches from the second step
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        srow[i] = wave * 32 + i * 8 + (lane >> 3);
        const int ch = (lane & 7) ^ xswz(srow[i]);
        scol[i] = (ch & 3) * 8;
        sel2 |= (uint32_t)(ch >> 2) << i;
    }

    // ---- producer: item pk (slot p_slot of token tile p_mt), segment
    // entries in lanes (cur) and the next segment (nxt), position p_i
    int pk = 0;
    int p_mt = first_mt;
    int p_slot = first_slot;
    // X of the producer's item: a uniform base (first row of the token tile)
    // and per-lane byte offsets of row min(row, M - 1 - m0), column chunk.
    // Dense W: the same for the item's group of output rows (rows past N
    // repeat its last).  Instruction i uses the base minus i KB (see dma16i).
    const char* xbase;
    uint32_t xoff[4];
    const char* wibase = nullptr;
    uint32_t wioff[4] = {0, 0, 0, 0};
    auto set_x = [&]() {
        const int64_t m0 = (int64_t)p_mt * BM;
        xbase = X + m0 * a.ldx * 2;
        const int last_row = (int)min((int64_t)BM - 1, a.M - 1 - m0);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            xoff[i] = (uint32_t)((min(srow[i], last_row) * a.ldx + scol[i]) * 2);
        if (DENSE) {
            const int64_t n0 = (int64_t)t_desc[p_slot].x * G * TILE;
            wibase = W + n0 * a.ldw * 2;
            const int wlast = (int)min((int64_t)G * TILE - 1, a.N - 1 - n0);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                wioff[i] = (uint32_t)((min(srow[i], wlast) * a.ldw + scol[i]) * 2);
        }
    };
    set_x();
    const uint32_t loff = (uint32_t)lane * 16;  // sparse W: lane's chunk of a tile
    auto seg_read = [&](int start) {
        return lds_read16<0>(walk_lds + min(start + lane, a.n_walk - 1) * 16);
    };
    int p_i = 0;
    v4i cur = *(const v4i*)&t_walk[min(t_desc[p_slot].y + lane, a.n_walk - 1)];
    v4i nxt = *(const v4i*)&t_walk[min(__builtin_amdgcn_readlane(cur.z, 0) + lane, a.n_walk - 1)];

    // One step's DMA for this wave: the step's ring position (step & 3: pair
    // slot (step >> 1) & 1, half step & 1), whether it loads anything (n: 0
    // for a step that keeps no tile, 2 with X only, 4 with this wave's W
    // tile), the column tile and its byte offset in a row of X / dense W, and
    // (sparse) the byte offset of this wave's W tile in the tile stream.
    // KH: the halves of this wave's tile to load (hl: bit 0 the first 16
    // columns, bit 1 the second).
    struct Dma {
        int slot, n, col, hl;
        uint32_t xcol, woff;
    };
    bool x_stale = false;  // the item advanced: set_x() before the next pair
    // rows the producer's item keeps (none past the last item: the producer
    // then keeps walking, inside the table, and its steps load nothing)
    int p_rows = n_full == 0 ? 0xf << (4 * hh) : 0xff;
    auto p_prepare = [&](int slot, Dma& d) -> int {
        d.slot = slot;
        d.n = 0;
        d.hl = 0;
        d.woff = 0;
        const int ex = __builtin_amdgcn_readlane(cur.x, p_i);
        // row bits in 0..7, the item's last step in bit 8 (= E_LAST)
        const int es = (int)((uint32_t)ex >> 16);
        int lo_bits = es & 0xff, hi_bits = lo_bits, all_bits = lo_bits;
        int tile0 = 0;
        if (KH) {
            const int ey = __builtin_amdgcn_readlane(cur.y, p_i);
            hi_bits = (int)((uint32_t)ey >> 24);
            all_bits = lo_bits | hi_bits;
            tile0 = ey & 0xffffff;
        }
        // a half item keeps its own half's rows (the tile stream order, and so
        // a tile's rank, still counts every kept row of the step)
        const int bits = all_bits & p_rows;
        d.col = ex & 0xffff;
        d.xcol = (uint32_t)d.col * (TILE * 2);
        if (bits)  // a step that keeps no tile (walk padding) loads nothing
            d.n = 2;
        if (DENSE) {
            if (bits)
                d.n = 4;
        } else if ((bits >> wave) & 1) {  // row `wave` of the group is kept: its tile
            // (the stream holds fewer than 2^21 tiles: the offset fits 32 bits)
            const int rank = __popc(all_bits & ((1 << wave) - 1));
            d.woff = (uint32_t)((KH ? tile0 : __builtin_amdgcn_readlane(cur.y, p_i)) + rank) * 2048u;
            d.n = 4;
            if (KH)
                d.hl = ((lo_bits >> wave) & 1) | (((hi_bits >> wave) & 1) << 1);
        }
        // the queue entry (p_rows clears the other half's rows in a half item,
        // and every row past the last item)
        const int e_lo = ((KH ? lo_bits & p_rows : bits) >> wsh) & 15;
        const int e_hi = KH ? (((hi_bits & p_rows) >> wsh) & 15) << 4 : 0;
        const int e = e_lo | e_hi | (es & E_LAST);
        // advance: next entry of the segment, or the next segment (whose
        // successor is read now; every half step waits for LDS reads)
        if (__builtin_expect(ex & W_SEG_END, 0)) {
            cur = nxt;
            p_i = 0;
            nxt = seg_read(__builtin_amdgcn_readlane(cur.z, 0));
        } else {
            ++p_i;
        }
        if (__builtin_expect(ex & W_LAST, 0)) {
            if (++pk < my_items) {
                if (pk == n_full) {
                    // on to the half item: its walk replaces the prefetched one
                    p_rows = 0xf << (4 * hh);
                    p_slot = h_slot;
                    p_mt = h_mt;
                    cur = seg_read(t_desc[h_slot].y);
                    nxt = seg_read(__builtin_amdgcn_readlane(cur.z, 0));
                    p_i = 0;
                } else {
                    p_slot += a.p_mod;
                    p_mt += a.p_div;
                    if (p_slot >= a.n_slots) {
                        p_slot -= a.n_slots;
                        p_mt += a.mt_carry;
                    }
                }
                // (items have an even number of steps: the next pair is the
                // new item's first)
                x_stale = true;
            } else {
                p_rows = 0;
            }
        }
        return e;
    };
    auto x_fresh = [&]() {
        // (the previous pair's DMA, issued after its p_prepare, used the old
        // item's bases)
        if (x_stale) {
            set_x();
            x_stale = false;
        }
    };
    // The DMA of a pair of prepared steps (d0, d1) into their pair slot, in
    // two parts.  X: 4 instructions of one M0 value (none if neither step
    // keeps a tile); lanes past K read the zero line.  W: dense, the group's
    // 256 rows of both column tiles (4 instructions, laid out like X); sparse,
    // this wave's tile of each step that keeps it (2 instructions each).
    auto dma_x = [&](const Dma d0, const Dma d1) {
        if (d0.n == 0 && d1.n == 0)
            return;
        const int ps = (d0.slot >> 1) & 1;
        if (KTAIL && (d0.col == ncol - 1 || d1.col == ncol - 1)) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const bool second = (sel2 >> i) & 1;
                const int col = second ? d1.col : d0.col;
                uint4* dx = smem + ps * PSLOT + wave * 256 + i * 64;
                if (col * TILE + scol[i] >= a.K)
                    dma16(zero, dx);
                else
                    dma16(xbase, xoff[i] + (second ? d1.xcol : d0.xcol), dx);
            }
            return;
        }
        const uint32_t mx = smem0 + (uint32_t)ps * (PSLOT * 16) + (uint32_t)wave * 4096;
        uint32_t vo[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            vo[i] = ((sel2 >> i) & 1) ? d1.xcol : d0.xcol;
        dma16i<0>(xbase, xoff[0] + vo[0], mx);
        dma16i<1024>(xbase - 1024, xoff[1] + vo[1], mx);
        dma16i<2048>(xbase - 2048, xoff[2] + vo[2], mx);
        dma16i<3072>(xbase - 3072, xoff[3] + vo[3], mx);
    };
    auto dma_w = [&](const Dma d0, const Dma d1) {
        const int ps = (d0.slot >> 1) & 1;
        const uint32_t wa = smem0 + (uint32_t)(ps * PSLOT + XP_U4) * 16;
        if (DENSE) {
            if (d0.n == 0 && d1.n == 0)
                return;
            if (KTAIL && (d0.col == ncol - 1 || d1.col == ncol - 1)) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const bool second = (sel2 >> i) & 1;
                    const int col = second ? d1.col : d0.col;
                    uint4* dw = smem + ps * PSLOT + XP_U4 + wave * 256 + i * 64;
                    if (col * TILE + scol[i] >= a.K)
                        dma16(zero, dw);
                    else
                        dma16(wibase, wioff[i] + (second ? d1.xcol : d0.xcol), dw);
                }
                return;
            }
            const uint32_t mw = wa + (uint32_t)wave * 4096;
            uint32_t vo[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                vo[i] = ((sel2 >> i) & 1) ? d1.xcol : d0.xcol;
            dma16i<0>(wibase, wioff[0] + vo[0], mw);
            dma16i<1024>(wibase - 1024, wioff[1] + vo[1], mw);
            dma16i<2048>(wibase - 2048, wioff[2] + vo[2], mw);
            dma16i<3072>(wibase - 3072, wioff[3] + vo[3], mw);
        } else {
            // (KH: only the kept halves; a dropped half's LDS keeps stale data
            // that no matrix-core instruction reads)
            if (d0.n == 4) {
                const uint32_t mw = wa + (uint32_t)wave * 2048;
                if (!KH || (d0.hl & 1))
                    dma16i<0>(stream, loff + d0.woff, mw);
                if (!KH || (d0.hl & 2))
                    dma16i<1024>(stream, loff + d0.woff, mw);
            }
            if (d1.n == 4) {
                const uint32_t mw = wa + WS_U4 * 16 + (uint32_t)wave * 2048;
                if (!KH || (d1.hl & 1))
                    dma16i<0>(stream, loff + d1.woff, mw);
                if (!KH || (d1.hl & 2))
                    dma16i<1024>(stream, loff + d1.woff, mw);
            }
        }
    };

    // ---- prologue: the first pair of steps
    uint64_t q = 0;  // queue entries of steps t, t + 1, ... (E_BITS each)
    {
        Dma d0, d1;
        q |= (uint64_t)(uint32_t)p_prepare(0, d0);
        q |= (uint64_t)(uint32_t)p_prepare(1, d1) << E_BITS;
        dma_x(d0, d1);
        dma_w(d0, d1);
    }

    // LDS read addresses of this lane in pair slot 0, by (half of the pair s,
    // k-step ks); token half u = 1 is +4096 bytes (32 rows), dense tile row
    // 4h + j is +4096 j bytes (xswz(r + 32) = xswz(r))
    uint32_t xa_addr[2][2], wd_addr[2][2];
#pragma unroll
    for (int sh = 0; sh < 2; ++sh) {
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const int ch = sh * 4 + ks * 2 + (lane >> 5);
            const int r = wm * 64 + (lane & 31);
            xa_addr[sh][ks] = smem0 + (r * 8 + (ch ^ xswz(r))) * 16;
            const int rw = wh * 128 + (lane & 31);
            wd_addr[sh][ks] = smem0 + XP_U4 * 16 + (rw * 8 + (ch ^ xswz(rw))) * 16;
        }
    }
    const uint32_t wa_addr = smem0 + XP_U4 * 16 + wh * 4 * 2048 + lane * 16;  // this half's rows

    // Operands of one half step (one 16-column k-step of a column tile): this
    // wave's two X fragments (token halves) and its kept W fragments.
    struct Ops {
        v4i x[2], w[4];
    };
    // LDS reads of half step (t, ks)
    auto read_half = [&](Ops& o, int t, int ks) {
        const int sh = t & 1;
        const uint32_t ps_off = (uint32_t)((t >> 1) & 1) * (PSLOT * 16);
        o.x[0] = lds_read16<0>(xa_addr[sh][ks] + ps_off);
        o.x[1] = lds_read16<4096>(xa_addr[sh][ks] + ps_off);
        // four W fragments whatever the mask (no branch): rows 4h .. 4h + 3
        // of the group, at fixed offsets in both layouts
        if (DENSE) {
            o.w[0] = lds_read16<0 * 4096>(wd_addr[sh][ks] + ps_off);
            o.w[1] = lds_read16<1 * 4096>(wd_addr[sh][ks] + ps_off);
            o.w[2] = lds_read16<2 * 4096>(wd_addr[sh][ks] + ps_off);
            o.w[3] = lds_read16<3 * 4096>(wd_addr[sh][ks] + ps_off);
        } else {
            // row j of the group's tile lies at W position j of the step's W
            // area (a dropped row's position holds stale data and is never used)
            const uint32_t wa = wa_addr + ps_off + (uint32_t)sh * (WS_U4 * 16) + ks * 1024;
            o.w[0] = lds_read16<0 * 2048>(wa);
            o.w[1] = lds_read16<1 * 2048>(wa);
            o.w[2] = lds_read16<2 * 2048>(wa);
            o.w[3] = lds_read16<3 * 2048>(wa);
        }
    };

    // consumer cursor
    int ck = 0;
    int c_mt = first_mt;
    int c_slot = first_slot;

    // Accumulators start at the bias of their outputs: lane l, register 4 qq
    // + i of tile row j holds output 8 qq + 4 (l / 32) + i of that row.
    f32x16 acc[2][4];
    const int h = lane >> 5;
    auto init_acc = [&](int slot) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            f32x16 b;
#pragma unroll
            for (int qq = 0; qq < 4; ++qq) {
                const v4i v = lds_read16<0>(bias_lds + (slot * G * TILE + (wh * 4 + j) * 32 + 8 * qq + 4 * h) * 4);
                // (int) v[i], an rvalue: this compiler bit-casts a vector
                // element lvalue as if it were element 0
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    b[4 * qq + i] = __builtin_bit_cast(float, (int)v[i]);
            }
            acc[0][j] = b;
            acc[1][j] = b;
        }
    };

    Ops r0, r1;

    // first half of step t: the second half's operands are read, then (t,
    // k-step 0) goes to the matrix cores
    auto half_a = [&](int t, int bits) {
        int bh = bits;
        // opaque to the compiler: a kept-row test is then one scalar bit test
        // and branch, not a 64-bit mask kept for the other half step
        asm volatile("" : "+s"(bh));
        read_half(r1, t, 1);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (bh & (1 << j)) {
                const F wj = __builtin_bit_cast(F, r0.w[j]);
                acc[0][j] = E::mma(wj, __builtin_bit_cast(F, r0.x[0]), acc[0][j]);
                acc[1][j] = E::mma(wj, __builtin_bit_cast(F, r0.x[1]), acc[1][j]);
            }
        }
    };
    // second half of step t: (t, k-step 1), while the first half of step t + 1
    // is read if it belongs to the same pair
    auto half_b = [&](int t, int bits, bool pre) {
        int bh = bits;
        asm volatile("" : "+s"(bh));
        if (pre)
            read_half(r0, t + 1, 0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (bh & (1 << j)) {
                const F wj = __builtin_bit_cast(F, r1.w[j]);
                acc[0][j] = E::mma(wj, __builtin_bit_cast(F, r1.x[0]), acc[0][j]);
                acc[1][j] = E::mma(wj, __builtin_bit_cast(F, r1.x[1]), acc[1][j]);
            }
        }
    };
    // ---- epilogue of item ck (GELU, one rounding).  Per 32 x 32 tile, lane l
    // holds token l % 32 and outputs 8 q + 4 h + (0..3); swapping the q-even /
    // q-odd halves between lanes l and l + 32 leaves each lane 8 consecutive
    // outputs (16 bytes) of its token.  pack() does that right after the
    // item's last step; flush() runs after the next barrier, which frees the
    // slot of that step: the chunks pass through this wave's own 4 KB of the
    // slot (the parts its next DMA refills) so that every store writes 8 whole
    // 128-byte lines of Y (lanes 8 i .. 8 i + 7: one token's 64 consecutive
    // outputs).  Streaming (non-temporal) stores keep the output from evicting
    // X and W from the caches.  16 stores per wave and item.
    v4i pko[2][4][2];  // (token half u, tile row j, p2): outputs 32 j + 16 p2 + 8 h + 0..7
    int64_t f_mw = 0, f_nw = 0;  // the packed item's first token and output of this wave
    bool f_inside = true;        // ... and whether its whole tile lies inside Y
    bool f_skip = false;         // ... and whether it is a half item of the other half
    auto pack = [&]() {
        f_skip = ck == n_full && wh != hh;
        const v4i cd = lds_read16<0>(desc_lds + c_slot * 16);
        const int c_g = __builtin_amdgcn_readfirstlane(cd.x);
        f_mw = (int64_t)c_mt * BM + wm * 64;
        f_nw = (int64_t)c_g * G * TILE + wh * 128;
        f_inside = (int64_t)c_mt * BM + BM <= a.M && (int64_t)(c_g + 1) * G * TILE <= a.N;
#pragma unroll
        for (int u = 0; u < 2; ++u) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                uint32_t pk[4][2];
#pragma unroll
                for (int qq = 0; qq < 4; ++qq) {
                    float v[4] = {acc[u][j][4 * qq], acc[u][j][4 * qq + 1], acc[u][j][4 * qq + 2],
                                  acc[u][j][4 * qq + 3]};
                    if (GELU) {
#pragma unroll
                        for (int x = 0; x < 4; ++x)
                            v[x] = gelu_erf(v[x]);
                    }
                    pk[qq][0] = pack2<DT>(v[0], v[1]);
                    pk[qq][1] = pack2<DT>(v[2], v[3]);
                }
#pragma unroll
                for (int p2 = 0; p2 < 2; ++p2) {
                    // lanes < 32 keep q = 2 p2 and take it from lane + 32; lanes
                    // >= 32 keep q = 2 p2 + 1 and take it from lane - 32
                    const auto s0 = __builtin_amdgcn_permlane32_swap(pk[2 * p2][0], pk[2 * p2 + 1][0], false, false);
                    const auto s1 = __builtin_amdgcn_permlane32_swap(pk[2 * p2][1], pk[2 * p2 + 1][1], false, false);
                    pko[u][j][p2].x = (int)s0[0];
                    pko[u][j][p2].y = (int)s1[0];
                    pko[u][j][p2].z = (int)s0[1];
                    pko[u][j][p2].w = (int)s1[1];
                }
            }
        }
    };
    auto flush = [&](int sslot) {
        if (f_skip)
            return;
        const int64_t mw = f_mw, nw = f_nw;
        const bool inside = f_inside;
        // staging: token tau (0..31) of a round at region tau / 16 of this
        // wave's own W area of the pair slot (the part its next W DMA refills),
        // row tau % 16 of 128 bytes, 16-byte chunk k at k ^ ((tau / 2) % 8):
        // conflict-free both ways
        const uint32_t st0 = smem0 + (uint32_t)(sslot * PSLOT + XP_U4) * 16 +
                             (uint32_t)wave * (DENSE ? 4096 : 2048);
        const uint32_t st1 = st0 + (DENSE ? 2048 : WS_U4 * 16);
        const int b = lane & 31;
        const uint32_t wbase = (b < 16 ? st0 : st1) + (b & 15) * 128;
        const int wswz = (b >> 1) & 7;
        // four rounds (u, lam): tokens 32 u + 0..31, outputs 64 lam + 0..63;
        // a round's writes follow the previous round's reads (LDS keeps one
        // wave's accesses in order)
        v4i o[2][2][4];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
#pragma unroll
            for (int lam = 0; lam < 2; ++lam) {
#pragma unroll
                for (int jj = 0; jj < 2; ++jj)
#pragma unroll
                    for (int p2 = 0; p2 < 2; ++p2) {
                        const int k = jj * 4 + 2 * p2 + h;  // chunk of the 128-byte line
                        lds_write16(wbase + ((k ^ wswz) * 16), pko[u][2 * lam + jj][p2]);
                    }
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int tau = 8 * i + (lane >> 3), k = lane & 7;
                    o[u][lam][i] = lds_read16<0>((i < 2 ? st0 : st1) + (tau & 15) * 128 +
                                                 ((k ^ ((tau >> 1) & 7)) * 16));
                }
            }
        }
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int lam = 0; lam < 2; ++lam)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int tau = 8 * i + (lane >> 3), k = lane & 7;
                    const int64_t m = mw + 32 * u + tau, n = nw + 64 * lam + 8 * k;
                    v4i* dst = (v4i*)(Y + (m * a.ldy + n) * 2);
                    if (!inside && !(m < a.M && n < a.N))
                        dst = (v4i*)&g_sink[lane];
                    __builtin_nontemporal_store(o[u][lam][i], dst);
                }
    };

    // Barrier of pair (b, b + 1): every wave has waited for all of its DMA
    // (steps b and b + 1, and its stores) and finished with steps b - 2 and
    // b - 1; their pair slot is free afterwards.
    auto sync = [&]() { asm volatile("s_waitcnt vmcnt(0)\n s_barrier" ::: "memory"); };
    int t = 0;
    sync();  // the first pair has landed
    // One item per iteration (items have an even number of steps).  After its
    // last pair: pack(), the next barrier (which frees that pair's slot), the
    // X DMA of steps t + 2 and t + 3, the stores staged through this wave's W
    // area of the free pair slot (flush), then their W DMA and the next item's
    // accumulators.  The packed outputs and the accumulators are never live
    // together.
    bool have = false;  // pko holds an item not yet stored
    for (;;) {
        read_half(r0, t, 0);
        {
            Dma d0, d1;
            x_fresh();
            q |= (uint64_t)(uint32_t)p_prepare((t + 2) & (NS - 1), d0) << (2 * E_BITS);
            q |= (uint64_t)(uint32_t)p_prepare((t + 3) & (NS - 1), d1) << (3 * E_BITS);
            dma_x(d0, d1);
            if (have)
                flush(((t + 2) >> 1) & 1);
            dma_w(d0, d1);
        }
        init_acc(c_slot);
        for (;;) {  // the pairs of the item
            const int e0 = (int)(q & E_MASK), e1 = (int)((q >> E_BITS) & E_MASK);
            // rows of each step that keep the second k-step (KH: their own bits)
            const int h0 = KH ? (e0 >> 4) & 15 : e0 & 15;
            const int h1 = KH ? (e1 >> 4) & 15 : e1 & 15;
            half_a(t, e0 & 15);
            half_b(t, h0, true);
            half_a(t + 1, e1 & 15);
            q >>= 2 * E_BITS;
            t += 2;
            if (LATE) {
                // the last k-step's operands are in registers before the
                // barrier lets the pair slot be refilled; its products keep
                // the matrix cores busy while the next fragments are read and
                // the next DMA is prepared
                __builtin_amdgcn_s_waitcnt(0xc07f);
                sync();
                read_half(r0, t, 0);
                half_b(t - 1, h1, false);
                if (e1 & E_LAST)
                    break;
            } else {
                half_b(t - 1, h1, false);
                sync();
                if (e1 & E_LAST)
                    break;
                read_half(r0, t, 0);
            }
            Dma d0, d1;
            x_fresh();
            q |= (uint64_t)(uint32_t)p_prepare((t + 2) & (NS - 1), d0) << (2 * E_BITS);
            q |= (uint64_t)(uint32_t)p_prepare((t + 3) & (NS - 1), d1) << (3 * E_BITS);
            dma_x(d0, d1);
            dma_w(d0, d1);
        }
        pack();
        have = true;
        if (++ck >= my_items)
            break;
        if (ck == n_full) {
            c_slot = h_slot;
            c_mt = h_mt;
        } else {
            c_slot += a.p_mod;
            c_mt += a.p_div;
            if (c_slot >= a.n_slots) {
                c_slot -= a.n_slots;
                c_mt += a.mt_carry;
            }
        }
    }
    flush(((t - 1) >> 1) & 1);
    // no DMA or store of this workgroup may be in flight when it ends
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

// Arguments of one k_linear16 launch.
struct Args {
    Dims d;
    const char* X;
    const char* stream;       // sparse: kept tiles in operand order
    const int4* gdesc;        // sparse: launch slot descriptors
    const int4* gdesc_host;   // sparse: their host copy (walk lengths)
    const int2* walk;         // sparse: the slots' walks
    const char* W;            // dense weight
    const char* bias;
    char* Y;
    bool kh;                  // sparse, 16-wide block columns: tile halves walked on their own
};

template <bool DENSE>
hipError_t launch16(int dtype, bool gelu, Args a, hipStream_t s)
{
    const int64_t n_mt = (a.d.M + BM - 1) / BM;
    const bool ktail = (a.d.K % TILE) != 0;
    if (!DENSE && ktail && !a.kh)
        return hipErrorInvalidValue;  // (a block width of 32 or 64 divides K into whole tiles)
    const int P0 = max(num_cus() & ~7, 8);
    // Launches over consecutive launch slots whose tables fit the 32 KB of LDS
    // reserved for them: 16 B per slot descriptor and walk entry, 1 KB of float32 bias
    // per slot.
    for (int gs0 = 0; gs0 < a.d.n_groups;) {
        int ns = 0, nw = 0;
        while (gs0 + ns < a.d.n_groups) {
            const int len = DENSE ? (a.d.n_tile_cols + 1) & ~1 : a.gdesc_host[gs0 + ns].z;
            if ((ns + 1) * (16 + G * TILE * 4) + (nw + len) * 16 > TAB_U4 * 16)
                break;
            ++ns;
            nw += len;
        }
        if (ns == 0)
            return hipErrorInvalidValue;  // one group's walk alone does not fit
        Dims d = a.d;
        d.gs0 = gs0;
        d.n_slots = ns;
        const int64_t items = n_mt * ns;
        if (items > 0x7fffffff)
            return hipErrorInvalidValue;
        d.n_items = (int32_t)items;
        d.walk0 = DENSE ? 0 : a.gdesc_host[gs0].y;
        d.n_walk = nw;
        d.walk_off = ns * 16;
        d.bias_off = d.walk_off + nw * 16;
        int P = P0;
        const int need = (d.n_items + 7) / 8 * 8;
        if (P > need)
            P = need;
        // Each XCD owns whole token tiles (its L2 then holds a tile's X for
        // all the tile's items) unless that deals some workgroup more items
        // than the plain order does.
        const int C = P / 8;
        const int64_t plain_max = (items + P - 1) / P;
        const int64_t xcd_max = ((n_mt + 7) / 8 * ns + C - 1) / C;
        d.xcd_tiles = n_mt >= 8 && xcd_max <= plain_max;
        // Multiplying a pair's last k-step after its barrier fills the time
        // the next fragments take to arrive but issues the next DMA later:
        // it pays when a token tile's X is shared through L2 by many groups
        // and costs when the DMA lead is the bound (few groups, long K).
        const bool late = a.d.n_groups >= 6;
        if (d.xcd_tiles) {
            d.p_div = 8 * (C / ns);
            d.p_mod = C % ns;
            d.mt_carry = 8;
        } else {
            d.p_div = P / ns;
            d.p_mod = P % ns;
            d.mt_carry = 1;
        }
        const dim3 grid(P), block(NT);
#define LPV_LAUNCH2(DT_, GELU_, KT_, KH_, LATE_)                                                   \
    hipLaunchKernelGGL((k_linear16<DT_, GELU_, DENSE, KT_, KH_, LATE_>), grid, block, 0, s, d,    \
                       a.X, a.stream, a.gdesc, a.walk, a.W, a.bias, a.Y)
        // (the rare reduction-tail kernels come in one order only)
#define LPV_LAUNCH1(DT_, GELU_, KT_, KH_)                                                         \
    do {                                                                                          \
        if (!(KT_) && late)                                                                       \
            LPV_LAUNCH2(DT_, GELU_, KT_, KH_, !(KT_));                                            \
        else                                                                                      \
            LPV_LAUNCH2(DT_, GELU_, KT_, KH_, false);                                             \
    } while (0)
        // A reduction tail (K = 16 mod 32) only occurs with 16-wide block
        // columns, so the sparse tail kernels are the KH ones.
#define LPV_LAUNCH(DT_, GELU_)                                                                    \
    do {                                                                                          \
        if constexpr (DENSE) {                                                                    \
            if (ktail)                                                                            \
                LPV_LAUNCH1(DT_, GELU_, true, false);                                             \
            else                                                                                  \
                LPV_LAUNCH1(DT_, GELU_, false, false);                                            \
        } else {                                                                                  \
            if (!a.kh)                                                                            \
                LPV_LAUNCH1(DT_, GELU_, false, false);                                            \
            else if (ktail)                                                                       \
                LPV_LAUNCH1(DT_, GELU_, true, true);                                              \
            else                                                                                  \
                LPV_LAUNCH1(DT_, GELU_, false, true);                                             \
        }                                                                                         \
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
#undef LPV_LAUNCH2
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
        gs0 += ns;
    }
    return hipSuccess;
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
    a.stream = (const char*)h->stream_vals;
    a.gdesc = h->gdesc;
    a.gdesc_host = h->gdesc_host;
    a.walk = h->walk;
    a.kh = h->b_c == 16;
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
