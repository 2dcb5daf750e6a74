"""Seeded synthetic inputs for the block-sparse linear layer.

This module is shared by the tests, the benchmark and the smoke check; it feeds
the GPU library and the float64 oracle alike and holds none of the layer's
arithmetic.  It only draws numbers, rounds them to the element type both sides
consume, and draws block masks.

The paper's inputs are DeiT activations and pruned ImageNet-trained weights;
neither is available, so synthetic tensors of the same shapes stand in for
them: X ~ N(0, 1) token activations (197 tokens per image, DeiT widths
192/384/768, MLP width 4x), W ~ N(0, 0.02) and bias ~ N(0, 0.02), masks drawn
as described per workload.

Element types are named ``"f32"``, ``"f16"`` and ``"bf16"``; arrays are numpy
float32, float16 and uint16 (bf16 bit patterns) respectively.

Seeds: ``SeedSequence([240702068, cfg_id, layer_id, tensor_id])`` with
tensor_id 0 = X, 1 = W, 2 = bias, 3 = mask, 4 = per-layer sparsity draws,
5 = Zipf row ranks.
"""
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

SEED_ROOT = 240702068
T_X, T_W, T_BIAS, T_MASK, T_SPARSITY, T_ZIPF, T_GRAD = range(7)
TOKENS_PER_IMAGE = 197  # 224x224 image, 16x16 patches, plus the class token


def rng(cfg_id: int, layer_id: int, tensor_id: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([SEED_ROOT, cfg_id, layer_id, tensor_id]))


# --------------------------------------------------------------------------
# rounding generated float32 values to the element type both sides consume
# --------------------------------------------------------------------------

def bf16_bits(a) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest, ties to even.

    Written from the IEEE definition: bf16 keeps the upper 16 bits of a
    binary32, so adding 0x7FFF plus the lowest kept bit and truncating rounds
    to nearest with ties to even.  NaNs stay (quiet) NaNs."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    rounded = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        rounded = np.where(nan, ((u >> 16) | 0x40).astype(np.uint16), rounded)
    return rounded.astype(np.uint16)


def bf16_to_f32(bits) -> np.ndarray:
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << 16).view(np.float32)


def quantize(a, dtype: str) -> np.ndarray:
    a = np.asarray(a, np.float32)
    if dtype == "f32":
        return np.ascontiguousarray(a)
    if dtype == "f16":
        return np.ascontiguousarray(a.astype(np.float16))
    if dtype == "bf16":
        return bf16_bits(a)
    raise ValueError("unknown element type %r" % (dtype,))


def to_f32(arr, dtype: str) -> np.ndarray:
    """float32 view of values already in ``dtype`` (exact: every f16/bf16
    value is a float32 value)."""
    if dtype == "bf16":
        return bf16_to_f32(arr)
    return np.asarray(arr, np.float32)


def elem_size(dtype: str) -> int:
    return {"f32": 4, "f16": 2, "bf16": 2}[dtype]


# --------------------------------------------------------------------------
# masks
# --------------------------------------------------------------------------

def n_keep(R: int, C: int, sparsity_pct: int) -> int:
    """Kept blocks of an R x C grid at an integer sparsity percentage: the
    ceiling of (1 - alpha) times the block count, as in the paper's per-matmul
    block count (Sec. 3.4), computed in integers."""
    if not 0 <= sparsity_pct <= 100:
        raise ValueError("sparsity must be a percentage")
    return ((100 - sparsity_pct) * R * C + 99) // 100


def mask_bernoulli(g: np.random.Generator, R: int, C: int, p_keep: float) -> np.ndarray:
    """Each block kept independently with probability p_keep."""
    return (g.random((R, C)) < p_keep).astype(np.uint8)


def mask_uniform(g: np.random.Generator, R: int, C: int, keep: int) -> np.ndarray:
    """Exactly ``keep`` blocks, chosen uniformly without replacement."""
    m = np.zeros(R * C, np.uint8)
    m[g.choice(R * C, size=keep, replace=False)] = 1
    return m.reshape(R, C)


def block_scores(W_f32: np.ndarray, b_r: int, b_c: int) -> np.ndarray:
    """Sum of squares of each block (float64): ranks blocks like their L2 norm."""
    N, K = W_f32.shape
    w = W_f32.astype(np.float64).reshape(N // b_r, b_r, K // b_c, b_c)
    return np.einsum("rick,rick->rc", w, w)


def mask_topk(scores: np.ndarray, keep: int) -> np.ndarray:
    """Keep the ``keep`` highest-scoring blocks; ties go to the lower
    row-major block index."""
    R, C = scores.shape
    flat = scores.reshape(-1)
    order = np.lexsort((np.arange(flat.size), -flat))
    m = np.zeros(flat.size, np.uint8)
    m[order[:keep]] = 1
    return m.reshape(R, C)


def zipf_counts(g_rank: np.random.Generator, R: int, C: int, keep: int, s: float = 1.0) -> np.ndarray:
    """Per-row kept counts that follow a Zipf law over a seeded permutation of
    the rows, capped at C per row (overflow water-filled onto the others), then
    floored with largest remainders (ties to the lower row)."""
    if not 0 <= keep <= R * C:
        raise ValueError("keep out of range")
    ranks = g_rank.permutation(R) + 1
    w = 1.0 / ranks.astype(np.float64) ** s
    target = np.zeros(R)
    free = np.ones(R, bool)
    left = float(keep)
    while left > 1e-9 and free.any():
        share = left * w * free / np.sum(w[free])
        room = C - target
        add = np.minimum(share, room)
        target += add
        left -= float(np.sum(add))
        free &= target < C - 1e-12
    cnt = np.floor(target + 1e-9).astype(np.int64)
    short = keep - int(cnt.sum())
    rem = target - cnt
    order = np.lexsort((np.arange(R), -rem))
    for r in order:
        if short <= 0:
            break
        if cnt[r] < C:
            cnt[r] += 1
            short -= 1
    assert int(cnt.sum()) == keep and cnt.max() <= C
    return cnt


def mask_zipf(g_rank: np.random.Generator, g_cols: np.random.Generator, R: int, C: int,
              keep: int, s: float = 1.0) -> np.ndarray:
    cnt = zipf_counts(g_rank, R, C, keep, s)
    m = np.zeros((R, C), np.uint8)
    for r in range(R):
        m[r, g_cols.choice(C, size=int(cnt[r]), replace=False)] = 1
    return m


# --------------------------------------------------------------------------
# workloads
# --------------------------------------------------------------------------

@dataclass
class Linear:
    """One block-sparse linear layer's inputs, already in element type ``dtype``."""
    name: str
    dtype: str
    b_r: int
    b_c: int
    W: np.ndarray            # N x K
    mask: np.ndarray         # uint8, N/b_r x K/b_c
    bias: Optional[np.ndarray]
    gelu: bool
    X: Optional[np.ndarray] = None  # M x K; None for layers fed by a previous one
    M: int = 0
    meta: dict = field(default_factory=dict)

    @property
    def N(self):
        return self.W.shape[0]

    @property
    def K(self):
        return self.W.shape[1]

    @property
    def nnzb(self):
        return int(self.mask.sum())

    def kept_flops(self, M=None):
        M = self.M if M is None else M
        return 2 * M * self.nnzb * self.b_r * self.b_c

    def dense_flops(self, M=None):
        M = self.M if M is None else M
        return 2 * M * self.N * self.K


def _weights(cfg, layer, N, K, dtype, bias=True):
    W = quantize(rng(cfg, layer, T_W).normal(0.0, 0.02, (N, K)).astype(np.float32), dtype)
    b = quantize(rng(cfg, layer, T_BIAS).normal(0.0, 0.02, N).astype(np.float32), dtype) if bias else None
    return W, b


def activations(cfg, layer, M, K, dtype):
    return quantize(rng(cfg, layer, T_X).standard_normal((M, K), dtype=np.float32), dtype)


def tiny_fc1(M=TOKENS_PER_IMAGE):
    """DeiT-Tiny fc1 of one image: fp32 X [197 x 192], W [768 x 192], 16x16
    blocks, each kept with probability 1/2, bias, no GELU."""
    cfg, dt, b = 0, "f32", 16
    W, bias = _weights(cfg, 0, 768, 192, dt)
    mask = mask_bernoulli(rng(cfg, 0, T_MASK), 768 // b, 192 // b, 0.5)
    return Linear("tiny_fc1", dt, b, b, W, mask, bias, False, activations(cfg, 0, M, 192, dt), M)


def s_fc1_gelu(M=64 * TOKENS_PER_IMAGE):
    """DeiT-S fc1 at batch 64: bf16 X [12608 x 384], W [1536 x 384], 32x32
    blocks, top half of the blocks by L2 norm, bias + GELU."""
    cfg, dt, b = 1, "bf16", 32
    W, bias = _weights(cfg, 0, 1536, 384, dt)
    R, C = 1536 // b, 384 // b
    mask = mask_topk(block_scores(to_f32(W, dt), b, b), n_keep(R, C, 50))
    return Linear("s_fc1_gelu", dt, b, b, W, mask, bias, True, activations(cfg, 0, M, 384, dt), M)


B_LAYER = (("qkv", 2304, 768, 40, False), ("proj", 768, 768, 50, False),
           ("fc1", 3072, 768, 60, True), ("fc2", 768, 3072, 70, False))


def b_layer(M=128 * TOKENS_PER_IMAGE, with_x=True):
    """The four linears of one DeiT-B encoder layer at batch 128, bf16, 32x32
    blocks, top-k masks by block L2 norm at 40/50/60/70% sparsity.  Each layer
    gets its own X of its own width (the attention between qkv and proj is
    outside this layer)."""
    cfg, dt, b = 2, "bf16", 32
    out = []
    for lid, (name, N, K, sp, gelu) in enumerate(B_LAYER):
        W, bias = _weights(cfg, lid, N, K, dt)
        mask = mask_topk(block_scores(to_f32(W, dt), b, b), n_keep(N // b, K // b, sp))
        X = activations(cfg, lid, M, K, dt) if with_x else None
        out.append(Linear("b_layer." + name, dt, b, b, W, mask, bias, gelu, X, M,
                          meta={"sparsity": sp}))
    return out


def b_stack(M=256 * TOKENS_PER_IMAGE, layers=12, zipf_s=1.0):
    """Full DeiT-B linear stack: ``layers`` x (qkv, proj, fc1+GELU, fc2), bf16,
    32x32 blocks, per-linear sparsity drawn uniformly in [30%, 80%] (integer
    percent), row-block keep counts Zipf-distributed (skewed rows).  Only the
    first linear gets an X; the chain feeds the next ones (qkv's V third feeds
    proj)."""
    cfg, dt, b = 3, "bf16", 32
    g_sp = rng(cfg, 0, T_SPARSITY)
    out = []
    for layer in range(layers):
        for j, (name, N, K, _, gelu) in enumerate(B_LAYER):
            lid = 4 * layer + j
            sp = int(g_sp.integers(30, 81))
            W, bias = _weights(cfg, lid, N, K, dt)
            R, C = N // b, K // b
            mask = mask_zipf(rng(cfg, lid, T_ZIPF), rng(cfg, lid, T_MASK), R, C,
                             n_keep(R, C, sp), zipf_s)
            X = activations(cfg, 0, M, 768, dt) if lid == 0 else None
            out.append(Linear("b_stack.%d.%s" % (layer, name), dt, b, b, W, mask, bias, gelu,
                              X, M, meta={"sparsity": sp, "layer": layer}))
    return out


FC1_SWEEP_BLOCKS = (16, 32, 64)
FC1_SWEEP_SPARSITY = (0, 25, 50, 75, 90)


def grad_output(cfg, layer, M, N, dtype):
    """The backward's input: a gradient at the layer's pre-activation, M x N,
    N(0, 1) rounded to the element type (no trained loss exists here)."""
    return quantize(rng(cfg, layer, T_GRAD).standard_normal((M, N), dtype=np.float32), dtype)


def b_fc1(block=32, sparsity=50, dtype="bf16", M=256 * TOKENS_PER_IMAGE, gelu=False, with_x=True):
    """DeiT-B fc1 at batch 256: X [50432 x 768] ~ N(0,1) -> 3072 outputs,
    W ~ N(0, 0.02), square blocks of side ``block``, exactly n_keep blocks kept
    uniformly at random, bias, GELU only if asked.  The default is the
    headline point: 32x32 blocks, 50% sparsity, bf16."""
    cfg = 4
    layer = 100 * FC1_SWEEP_BLOCKS.index(block) + sparsity if block in FC1_SWEEP_BLOCKS else block
    N, K = 3072, 768
    W, bias = _weights(cfg, layer, N, K, dtype)
    R, C = N // block, K // block
    mask = mask_uniform(rng(cfg, layer, T_MASK), R, C, n_keep(R, C, sparsity))
    X = activations(cfg, 0, M, K, dtype) if with_x else None
    return Linear("b_fc1.%dx%d.s%d.%s" % (block, block, sparsity, dtype), dtype, block, block,
                  W, mask, bias, gelu, X, M, meta={"sparsity": sparsity})


def custom(cfg_id, M, N, K, b_r, b_c, dtype, mask_kind="uniform", sparsity=50, gelu=False,
           bias=True, layer=0):
    """A free-form workload for edge cases: any shape, block and mask kind
    (``uniform``, ``bernoulli``, ``topk``, ``zipf``, ``all``, ``none``)."""
    W, b = _weights(cfg_id, layer, N, K, dtype, bias)
    R, C = N // b_r, K // b_c
    g = rng(cfg_id, layer, T_MASK)
    if mask_kind == "uniform":
        mask = mask_uniform(g, R, C, n_keep(R, C, sparsity))
    elif mask_kind == "bernoulli":
        mask = mask_bernoulli(g, R, C, 1.0 - sparsity / 100.0)
    elif mask_kind == "topk":
        mask = mask_topk(block_scores(to_f32(W, dtype), b_r, b_c), n_keep(R, C, sparsity))
    elif mask_kind == "zipf":
        mask = mask_zipf(rng(cfg_id, layer, T_ZIPF), g, R, C, n_keep(R, C, sparsity))
    elif mask_kind == "all":
        mask = np.ones((R, C), np.uint8)
    elif mask_kind == "none":
        mask = np.zeros((R, C), np.uint8)
    else:
        raise ValueError(mask_kind)
    X = activations(cfg_id, layer, M, K, dtype)
    return Linear("custom.%dx%dx%d.%dx%d.%s.%s" % (M, N, K, b_r, b_c, dtype, mask_kind), dtype,
                  b_r, b_c, W, mask, b, gelu, X, M, meta={"sparsity": sparsity})


def small_ints(g: np.random.Generator, shape, lo=-2, hi=2, dtype="bf16"):
    """Small integers in [lo, hi] in element type ``dtype``: products and
    short sums of them are exact in every format."""
    return quantize(g.integers(lo, hi + 1, size=shape).astype(np.float32), dtype)
