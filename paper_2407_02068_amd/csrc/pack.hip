// pack.hip -- block mask -> BSR arrays and the tile schedule, on the GPU.
//
// The masked weight of the paper (Sec. 3.1) keeps or drops whole b_r x b_c
// blocks; the cost of the layer is the number of kept blocks times the number
// of token tiles (Sec. 3.4).  Packing therefore produces
//   - the canonical BSR arrays (row_ptr, col_idx ascending per row, raw block
//     values row-major), which are exported bit for bit;
//   - a schedule over 32 x 32 tiles of W: tile rows are grouped GROUP_TILES at a
//     time, and for each group the list of tile columns ("steps") that hold a
//     kept tile in any of its rows, with a bit per row;
//   - the kept tiles' values in matrix-core operand order, laid out group by
//     group and step by step, so the linear kernel streams them contiguously.
// Counts are wave-level ballots and reductions; offsets are workgroup prefix
// sums built from wave-level scans.
#include "lpv_device.h"
#include "lpv_internal.h"

namespace lpv {
namespace {

constexpr int PLAN_THREADS = 1024;
constexpr int PLAN_WAVES = PLAN_THREADS / 64;
constexpr int MAX_R = 4096;       // N <= 65536 with b_r >= 16
constexpr int MAX_GROUPS = 2048 / GROUP_TILES;  // N <= 65536: 2048 tile rows
constexpr int MAX_C = 4096;       // K <= 65536 with b_c >= 16

// Is tile (tr, tc) touched by a kept block?  A tile overlaps at most 2 x 2
// blocks (16-wide blocks) and at least part of one.
__device__ inline bool tile_kept(const PackArgs& a, int tr, int tc)
{
    const int r0 = tr * TILE / a.b_r, r1 = min((tr * TILE + TILE - 1) / a.b_r, a.R - 1);
    const int c0 = tc * TILE / a.b_c, c1 = min((tc * TILE + TILE - 1) / a.b_c, a.C - 1);
    bool kept = false;
    for (int r = r0; r <= r1; ++r)
        for (int c = c0; c <= c1; ++c)
            kept |= a.mask[(int64_t)r * a.C + c] != 0;
    return kept;
}

__device__ inline int tile_bits(const PackArgs& a, int g, int tc)
{
    int bits = 0;
#pragma unroll
    for (int j = 0; j < GROUP_TILES; ++j) {
        const int tr = g * GROUP_TILES + j;
        if (tr < a.n_tile_rows && tile_kept(a, tr, tc))
            bits |= 1 << j;
    }
    return bits;
}

// In-place exclusive prefix sum of arr[0..n) (LDS) by one workgroup of
// PLAN_THREADS threads; returns the total.  Wave scans, then a scan of the wave
// totals, chunk by chunk with a running carry.
__device__ int block_exclusive_scan(int* arr, int n, int* s_wave, int* s_carry)
{
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int carry = 0;
    for (int base = 0; base < n; base += PLAN_THREADS) {
        const int i = base + tid;
        const int v = i < n ? arr[i] : 0;
        const int inc = wave_inclusive_scan(v);
        if (lane == 63)
            s_wave[wave] = inc;
        __syncthreads();
        if (wave == 0) {
            const int w = lane < PLAN_WAVES ? s_wave[lane] : 0;
            const int winc = wave_inclusive_scan(w);
            if (lane < PLAN_WAVES)
                s_wave[lane] = winc - w;
        }
        __syncthreads();
        const int excl = carry + s_wave[wave] + inc - v;
        if (i < n)
            arr[i] = excl;
        if (tid == PLAN_THREADS - 1)
            *s_carry = excl + v;
        __syncthreads();
        carry = *s_carry;
        __syncthreads();
    }
    return carry;
}

__global__ __launch_bounds__(PLAN_THREADS) void k_pack_plan(PackArgs a, int32_t* row_ptr,
                                                            int32_t* step_ptr,
                                                            int32_t* group_tile0,
                                                            int32_t* group_order, int4* gdesc,
                                                            Plan* plan)
{
    __shared__ int s_cnt[MAX_R];
    __shared__ int s_gsteps[MAX_GROUPS];
    __shared__ int s_gtiles[MAX_GROUPS];
    __shared__ int s_cost[MAX_GROUPS];
    __shared__ int s_rank[MAX_GROUPS];
    __shared__ int s_walk[MAX_GROUPS];
    __shared__ int s_wave[PLAN_WAVES];
    __shared__ int s_carry;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

    // kept blocks per block-row: one wave per row, a ballot per 64 columns
    for (int r = wave; r < a.R; r += PLAN_WAVES) {
        int cnt = 0;
        for (int c0 = 0; c0 < a.C; c0 += 64) {
            const int c = c0 + lane;
            const bool kept = c < a.C && a.mask[(int64_t)r * a.C + c] != 0;
            cnt += __popcll(__ballot(kept));
        }
        if (lane == 0)
            s_cnt[r] = cnt;
    }
    // steps and kept tiles per group: one wave per group, a lane per tile column
    for (int g = wave; g < a.n_groups; g += PLAN_WAVES) {
        int ns = 0, nt = 0;
        for (int tc0 = 0; tc0 < a.n_tile_cols; tc0 += 64) {
            const int tc = tc0 + lane;
            const int bits = tc < a.n_tile_cols ? tile_bits(a, g, tc) : 0;
            ns += __popcll(__ballot(bits != 0));
            nt += wave_sum(__popc(bits));
        }
        if (lane == 0) {
            s_gsteps[g] = ns;
            s_gtiles[g] = nt;
            s_cost[g] = ns + nt;  // one X slice per step, one tile product per kept tile
        }
    }
    __syncthreads();

    const int nnzb = block_exclusive_scan(s_cnt, a.R, s_wave, &s_carry);
    const int n_steps = block_exclusive_scan(s_gsteps, a.n_groups, s_wave, &s_carry);
    const int n_tiles = block_exclusive_scan(s_gtiles, a.n_groups, s_wave, &s_carry);
    for (int r = tid; r < a.R; r += PLAN_THREADS)
        row_ptr[r] = s_cnt[r];
    for (int g = tid; g < a.n_groups; g += PLAN_THREADS) {
        step_ptr[g] = s_gsteps[g];
        group_tile0[g] = s_gtiles[g];
        // launch order: most work first, ties by group index (a stable rank)
        const int cg = s_cost[g];
        int rank = 0;
        for (int h = 0; h < a.n_groups; ++h) {
            const int ch = s_cost[h];
            rank += (ch > cg) || (ch == cg && h < g);
        }
        group_order[rank] = g;
        s_rank[g] = rank;
        // steps walked for launch slot `rank`, padded to an even count (the
        // kernel takes steps in pairs) with steps that keep no tile; an empty
        // group still produces its bias, from two such steps
        const int ns = (g + 1 < a.n_groups ? s_gsteps[g + 1] : n_steps) - s_gsteps[g];
        s_walk[rank] = (max(ns, 1) + 1) & ~1;
    }
    __syncthreads();
    // the launch slots' walks lie one after the other, in launch order
    const int n_walk = block_exclusive_scan(s_walk, a.n_groups, s_wave, &s_carry);
    for (int g = tid; g < a.n_groups; g += PLAN_THREADS) {
        const int rank = s_rank[g];
        const int ns = (g + 1 < a.n_groups ? s_gsteps[g + 1] : n_steps) - s_gsteps[g];
        // the walk of slot `rank` starts at column step rank * ns / n_groups,
        // rounded down to even (the kernel's pairs then tend to cover aligned
        // column pairs), and wraps: slots that run side by side on one token
        // tile read different X columns at a time
        gdesc[rank] = make_int4(g, s_walk[rank], (max(ns, 1) + 1) & ~1,
                                ns > 0 ? (int)((int64_t)rank * ns / a.n_groups) & ~1 : 0);
    }
    if (tid == 0) {
        row_ptr[a.R] = nnzb;
        step_ptr[a.n_groups] = n_steps;
        group_tile0[a.n_groups] = n_tiles;
        plan->nnzb = nnzb;
        plan->n_steps = n_steps;
        plan->n_tiles = n_tiles;
        plan->n_walk = n_walk;
    }
}

// One workgroup per block-row: the kept columns in ascending order (ballot +
// running offset), then a cooperative 16-byte copy of the kept blocks.
__global__ __launch_bounds__(256) void k_pack_compact(PackArgs a, const int32_t* __restrict__ row_ptr,
                                                      int32_t* __restrict__ col_idx,
                                                      char* __restrict__ values)
{
    __shared__ int s_cols[MAX_C];
    __shared__ int s_wcnt[4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int r = blockIdx.x;
    const int base = row_ptr[r];
    int running = 0;
    for (int c0 = 0; c0 < a.C; c0 += 256) {
        const int c = c0 + tid;
        const bool kept = c < a.C && a.mask[(int64_t)r * a.C + c] != 0;
        const uint64_t b = __ballot(kept);
        if (lane == 0)
            s_wcnt[wave] = __popcll(b);
        __syncthreads();
        int off = 0, total = 0;
        for (int w = 0; w < 4; ++w) {
            off += w < wave ? s_wcnt[w] : 0;
            total += s_wcnt[w];
        }
        if (kept) {
            const int pos = running + off + lanes_below(b);
            s_cols[pos] = c;
            col_idx[base + pos] = c;
        }
        running += total;
        __syncthreads();
    }
    const int cpr = a.b_c * a.es / 16;  // 16-byte chunks per block row
    const int per_block = a.b_r * cpr;
    const int total = running * per_block;
    for (int q = tid; q < total; q += 256) {
        const int i = q / per_block, rem = q - i * per_block;
        const int row = rem / cpr, ch = rem - row * cpr;
        const int c = s_cols[i];
        const char* src = (const char*)a.W +
                          (((int64_t)r * a.b_r + row) * a.ldw + (int64_t)c * a.b_c) * a.es + ch * 16;
        char* dst = values + ((int64_t)(base + i) * a.b_r * a.b_c + (int64_t)row * a.b_c) * a.es + ch * 16;
        *(uint4*)dst = *(const uint4*)src;
    }
}

// One wave per group: the group's steps in ascending tile column, with the
// row bits and the index of the first kept tile in the operand stream.
__global__ __launch_bounds__(64) void k_sched_fill(PackArgs a, const int32_t* __restrict__ step_ptr,
                                                   const int32_t* __restrict__ group_tile0,
                                                   int32_t* __restrict__ step_col,
                                                   int32_t* __restrict__ step_bits,
                                                   int32_t* __restrict__ step_tile)
{
    const int g = blockIdx.x;
    int s = step_ptr[g], t = group_tile0[g];
    for (int tc0 = 0; tc0 < a.n_tile_cols; tc0 += 64) {
        const int tc = tc0 + (int)threadIdx.x;
        const int bits = tc < a.n_tile_cols ? tile_bits(a, g, tc) : 0;
        const uint64_t b = __ballot(bits != 0);
        const int pc = __popc(bits);
        const int inc = wave_inclusive_scan(pc);
        if (bits) {
            const int pos = s + lanes_below(b);
            step_col[pos] = tc;
            step_bits[pos] = bits;
            step_tile[pos] = t + inc - pc;
        }
        s += __popcll(b);
        t += __shfl(inc, 63, 64);
    }
}

// One workgroup per step: copy the step's kept tiles into operand order.
// Within a tile, 16-byte chunk (ks, l) holds W[row0 + (l & 31)][col0 + 16 ks +
// 8 (l >> 5) .. + 8]: lane l's operand of the ks-th 32x32x16 instruction.
// Elements of dropped blocks inside a kept tile are zero (selected, never
// copied), as are rows / columns past the weight's edge.
__global__ __launch_bounds__(256) void k_stream_fill(PackArgs a, const int32_t* __restrict__ step_ptr,
                                                     const int32_t* __restrict__ step_col,
                                                     const int32_t* __restrict__ step_bits,
                                                     const int32_t* __restrict__ step_tile,
                                                     uint4* __restrict__ stream)
{
    const int st = blockIdx.x;
    // group of this step: the last g with step_ptr[g] <= st
    int lo = 0, hi = a.n_groups - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (step_ptr[mid] <= st)
            lo = mid;
        else
            hi = mid - 1;
    }
    const int g = lo;
    const int col = step_col[st], bits = step_bits[st], tile0 = step_tile[st];
    const int nk = __popc(bits);
    for (int q = threadIdx.x; q < nk * 128; q += 256) {
        const int jj = q >> 7, rem = q & 127, ks = rem >> 6, l = rem & 63;
        int j = 0;
        for (int seen = -1; j < GROUP_TILES; ++j) {
            seen += (bits >> j) & 1;
            if (seen == jj && ((bits >> j) & 1))
                break;
        }
        const int64_t n = (int64_t)(g * GROUP_TILES + j) * TILE + (l & 31);
        const int64_t k = (int64_t)col * TILE + ks * 16 + (l >> 5) * 8;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (n < a.N && k < a.K && a.mask[(n / a.b_r) * a.C + k / a.b_c] != 0)
            v = *(const uint4*)((const char*)a.W + (n * a.ldw + k) * a.es);
        stream[(int64_t)(tile0 + jj) * 128 + rem] = v;
    }
}

// Rows of group g whose tile at column tc keeps a block in the tile's 16-column
// half h (16-wide block columns: that half is block column 2 tc + h).
__device__ inline int half_bits(const PackArgs& a, int g, int tc, int h)
{
    const int c = 2 * tc + h;
    if (c >= a.C)
        return 0;
    int bits = 0;
    for (int j = 0; j < GROUP_TILES; ++j) {
        const int tr = g * GROUP_TILES + j;
        if (tr >= a.n_tile_rows)
            break;
        const int r0 = tr * TILE / a.b_r, r1 = min((tr * TILE + TILE - 1) / a.b_r, a.R - 1);
        for (int r = r0; r <= r1; ++r)
            if (a.mask[(int64_t)r * a.C + c] != 0)
                bits |= 1 << j;
    }
    return bits;
}

// One wave per launch slot: the slot's walk, the group's steps starting at its
// rotation and wrapping, as {col | bits << 16 | last << 24, first tile}, then
// steps with no tile up to the (even) walk length.  With 16-wide block columns
// bits are the rows that keep the tile's first 16 columns, and the rows that
// keep its second 16 go in the top byte of the first-tile word (fewer than
// 2^21 tiles), so that the linear kernel moves and multiplies only kept halves.
__global__ __launch_bounds__(64) void k_walk_fill(const PackArgs a, const int4* __restrict__ gdesc,
                                                  const int32_t* __restrict__ step_ptr,
                                                  const int32_t* __restrict__ step_col,
                                                  const int32_t* __restrict__ step_bits,
                                                  const int32_t* __restrict__ step_tile,
                                                  int2* __restrict__ walk)
{
    const int4 d = gdesc[blockIdx.x];  // group, first walk entry, walk length, rotation
    const int s0 = step_ptr[d.x], ns = step_ptr[d.x + 1] - s0;
    for (int i = threadIdx.x; i < d.z; i += 64) {
        const int last = (i == d.z - 1) ? 1 << 24 : 0;
        int2 e = make_int2(last, 0);
        if (i < ns) {
            int j = d.w + i;
            if (j >= ns)
                j -= ns;
            const int s = s0 + j;
            if (a.b_c == 16) {
                const int tc = step_col[s];
                e = make_int2(tc | (half_bits(a, d.x, tc, 0) << 16) | last,
                              step_tile[s] | (half_bits(a, d.x, tc, 1) << 24));
            } else {
                e = make_int2(step_col[s] | (step_bits[s] << 16) | last, step_tile[s]);
            }
        }
        walk[d.y + i] = e;
    }
}

// One workgroup per block-row: the pruned dense rows, +0.0 in dropped blocks.
__global__ __launch_bounds__(256) void k_unpack(int64_t K, int32_t b_r, int32_t b_c, int32_t C,
                                                int32_t es, const int32_t* __restrict__ row_ptr,
                                                const int32_t* __restrict__ col_idx,
                                                const char* __restrict__ values, char* __restrict__ out,
                                                int64_t ldw)
{
    __shared__ int s_map[MAX_C];
    const int r = blockIdx.x;
    const int base = row_ptr[r], end = row_ptr[r + 1];
    for (int c = threadIdx.x; c < C; c += 256)
        s_map[c] = -1;
    __syncthreads();
    for (int p = base + threadIdx.x; p < end; p += 256)
        s_map[col_idx[p]] = p;
    __syncthreads();
    const int64_t cpr = K * es / 16;  // 16-byte chunks per weight row
    const int64_t total = (int64_t)b_r * cpr;
    for (int64_t q = threadIdx.x; q < total; q += 256) {
        const int64_t row = q / cpr, ch = q - row * cpr;
        const int64_t k = ch * 16 / es;
        const int c = (int)(k / b_c);
        const int p = s_map[c];
        uint4 v = make_uint4(0, 0, 0, 0);
        if (p >= 0)
            v = *(const uint4*)(values + ((int64_t)p * b_r * b_c + row * b_c + (k - (int64_t)c * b_c)) * es);
        *(uint4*)(out + (((int64_t)r * b_r + row) * ldw) * es + ch * 16) = v;
    }
}

}  // namespace

hipError_t launch_pack_plan(const PackArgs& a, int32_t* row_ptr, int32_t* step_ptr,
                            int32_t* group_tile0, int32_t* group_order, int4* gdesc, Plan* plan,
                            hipStream_t s)
{
    if (a.R > MAX_R || a.C > MAX_C || a.n_groups > MAX_GROUPS)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_pack_plan, dim3(1), dim3(PLAN_THREADS), 0, s, a, row_ptr, step_ptr,
                       group_tile0, group_order, gdesc, plan);
    return hipGetLastError();
}

hipError_t launch_pack_fill(const PackArgs& a, const lpv_bsr* h, hipStream_t s)
{
    if (a.R > MAX_R || a.C > MAX_C)
        return hipErrorInvalidValue;
    if (h->nnzb > 0)
        hipLaunchKernelGGL(k_pack_compact, dim3(a.R), dim3(256), 0, s, a, h->row_ptr, h->col_idx,
                           (char*)h->values);
    hipError_t e = hipGetLastError();
    // fp32 handles carry no schedule; a matrix-core handle always has a walk
    // (one entry per empty group), even when no tile is kept
    if (e != hipSuccess || h->walk == nullptr)
        return e;
    if (a.n_groups > 0)
        hipLaunchKernelGGL(k_sched_fill, dim3(a.n_groups), dim3(64), 0, s, a, h->step_ptr,
                           h->group_tile0, h->step_col, h->step_bits, h->step_tile);
    if (h->n_steps > 0)
        hipLaunchKernelGGL(k_stream_fill, dim3((unsigned)h->n_steps), dim3(256), 0, s, a,
                           h->step_ptr, h->step_col, h->step_bits, h->step_tile,
                           (uint4*)h->stream_vals);
    if (a.n_groups > 0)
        hipLaunchKernelGGL(k_walk_fill, dim3(a.n_groups), dim3(64), 0, s, a, h->gdesc, h->step_ptr,
                           h->step_col, h->step_bits, h->step_tile, h->walk);
    return hipGetLastError();
}

hipError_t launch_unpack(const lpv_bsr* h, void* W_out, int64_t ldw, hipStream_t s)
{
    const int es = h->dtype == LPV_F32 ? 4 : 2;
    if (h->C > MAX_C)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_unpack, dim3(h->R), dim3(256), 0, s, h->K, h->b_r, h->b_c, h->C, es,
                       h->row_ptr, h->col_idx, (const char*)h->values, (char*)W_out, ldw);
    return hipGetLastError();
}

}  // namespace lpv
