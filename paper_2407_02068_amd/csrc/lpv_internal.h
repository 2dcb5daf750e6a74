// lpv_internal.h -- host-side internals of liblpv: the handle, the schedule
// constants and the kernel launchers (implemented in pack.hip / linear.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/lpv.h"

namespace lpv {

// Schedule tile: 32 output rows x 32 reduction columns, the operand shape of
// one pair of 32x32x16 matrix-core instructions.
constexpr int TILE = 32;
// Tile rows per group: a workgroup owns one token tile times one group.
constexpr int GROUP_TILES = 8;
// Tokens per workgroup.
constexpr int BM = 256;

struct Plan {  // sizes learnt on the device during pack
    int32_t nnzb, n_steps, n_tiles, n_walk;
};

}  // namespace lpv

struct lpv_bsr {
    int64_t N, K;
    int32_t b_r, b_c, R, C;
    int64_t nnzb;
    int32_t dtype;  // lpv_dtype
    int32_t device;
    void* meta;  // one allocation: gdesc, row_ptr, group_order, step_ptr, group_tile0, plan
    // canonical BSR
    int32_t* row_ptr;  // R + 1
    int32_t* col_idx;  // nnzb
    void* values;      // nnzb * b_r * b_c elements
    // tile schedule (16-bit element types only)
    int32_t n_tile_rows, n_tile_cols, n_groups;
    int64_t n_steps, n_tiles;
    int4* gdesc;           // n_groups: {group, first walk entry, walk length, rotation} per launch slot
    int4* gdesc_host;      // host copy of gdesc (sizes the linear kernel's launches)
    int32_t* group_order;  // n_groups
    int32_t* step_ptr;     // n_groups + 1
    int32_t* group_tile0;  // n_groups + 1, first stream tile of each group
    int32_t* step_col;     // n_steps
    int32_t* step_bits;    // n_steps
    int32_t* step_tile;    // n_steps
    int64_t n_walk;
    int2* walk;            // n_walk: the launch slots' walks, {col | bits << 16 | last << 24, tile}
    void* stream_vals;     // n_tiles * TILE * TILE elements, operand order
    // workspace of lpv_bsr_grad_w (per-chunk float32 partial sums of every
    // tile), allocated on the first call and kept until destroy
    mutable void* gradw_ws;
    mutable size_t gradw_ws_bytes;
};

namespace lpv {

struct PackArgs {
    const void* W;
    int64_t ldw, N, K;
    int32_t es;  // element size in bytes
    int32_t b_r, b_c, R, C;
    const uint8_t* mask;
    int32_t n_tile_rows, n_tile_cols, n_groups;
};

// pack.hip
hipError_t launch_pack_plan(const PackArgs& a, int32_t* row_ptr, int32_t* step_ptr,
                            int32_t* group_tile0, int32_t* group_order, int4* gdesc, Plan* plan,
                            hipStream_t s);
hipError_t launch_pack_fill(const PackArgs& a, const lpv_bsr* h, hipStream_t s);
hipError_t launch_unpack(const lpv_bsr* h, void* W_out, int64_t ldw, hipStream_t s);

// linear.hip
struct LinearCall {
    const void* X;
    int64_t ldx, M;
    const void* bias;
    void* Y;
    int64_t ldy;
    int gelu;
};
hipError_t launch_bsr_linear(const lpv_bsr* h, const LinearCall& c, hipStream_t s);
hipError_t launch_dense_linear(const void* W, int64_t ldw, int64_t N, int64_t K, int dtype,
                               const LinearCall& c, hipStream_t s);

// mask.hip
struct MaskCall {
    const void* W;
    int64_t ldw;
    const void* G;  // NULL: sum-of-squares scores
    int64_t ldg, N, K;
    int dtype;
    int32_t b_r, b_c;
    int64_t n_keep;
    uint8_t* mask;
    double* scores;
};
hipError_t launch_mask_topk(const MaskCall& m, hipStream_t s);
hipError_t launch_block_scores(const MaskCall& m, hipStream_t s);  // scores only

// delta.hip
constexpr int DELTA_MAX_POINTS = 128;
constexpr int64_t DELTA_MAX_BLOCKS = (int64_t)1 << 17;
struct DeltaCall {
    const void* W;  // N x K, row stride ldw
    int64_t ldw, N, K;
    int dtype;
    int32_t b_r, b_c;
    const void* grad;  // N x K, row stride ldg
    int64_t ldg;
    const void* samples;  // n_samples x (N x K, row stride lds), sample stride `stride`
    int64_t lds, stride, n_samples;
    double kappa;
    int32_t n_points;
    int32_t keep[DELTA_MAX_POINTS];  // kept blocks at each point, non-increasing
    double* delta;                   // n_points, device
    void* ws;                        // caller workspace, or NULL: allocated per call
    size_t ws_bytes;
};
size_t delta_workspace_bytes(int64_t N, int64_t K, int32_t b_r, int32_t b_c, int64_t n_samples,
                             int32_t n_points);
hipError_t launch_delta_curve(const DeltaCall& c, hipStream_t s);

// backward.hip
struct GradWCall {
    const void* G;  // M x N, row stride ldg
    int64_t ldg;
    const void* X;  // M x K, row stride ldx
    int64_t ldx, M;
    void* dW;  // nnzb x b_r x b_c, BSR order
    float* ws; // at least grad_w_workspace_bytes(h) bytes
};
// Bytes of the weight-gradient workspace of a handle (any M).
size_t grad_w_workspace_bytes(const lpv_bsr* h);
hipError_t launch_transpose_blocks(const lpv_bsr* h, void* WT, int64_t ldwt, uint8_t* maskT,
                                   hipStream_t s);
hipError_t launch_grad_w(const lpv_bsr* h, const GradWCall& c, hipStream_t s);
// Encoder block around the pruned layers (encoder.hip).
constexpr int LN_MAX_D = 2048;     // widest row of the layer norm
constexpr int ATT_HD = 64;         // head dimension of the attention kernel
constexpr int ATT_MAX_T = 512;     // longest sequence (K and V staged in LDS)
hipError_t launch_add_layernorm(const void* x, const void* y, int64_t M, int32_t D, int dtype,
                                const void* gamma, const void* beta, float eps, void* S, void* out,
                                hipStream_t s);
hipError_t launch_attention(const void* qkv, int64_t n_seq, int32_t T, int32_t H, int dtype,
                            void* out, hipStream_t s);
hipError_t launch_bias_grad(const void* G, int64_t ldg, int64_t M, int64_t N, int dtype, void* db,
                            hipStream_t s);
// The same with the partial sums in a fixed device array of this many floats
// (4 MiB per device, held until the process ends): no allocation.
constexpr int64_t BIAS_NOALLOC_SCRATCH_FLOATS = (int64_t)1 << 20;
hipError_t launch_bias_grad_noalloc(const void* G, int64_t ldg, int64_t M, int64_t N, int dtype,
                                    void* db, hipStream_t s);

}  // namespace lpv
