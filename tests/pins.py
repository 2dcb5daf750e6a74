"""Pins of the float64 oracle against facts fixed outside it.

Each ``pin_*`` takes an oracle binding (``oracle.Oracle``) and raises
AssertionError when the oracle disagrees with what the paper, the mathematics
or an independent library routine fixes.  ``test_oracle_pins.py`` runs them on
the real oracle; ``test_oracle_mutants.py`` runs them on copies of the oracle
with planted mistakes and requires every mistake to be caught.

Independent references used here: the hand-worked fixture under ``golden/``,
the standard normal table, ``scipy.sparse.bsr_matrix`` (BSR arrays),
``numpy.matmul`` / ``numpy.kron`` (dense products, mask expansion), integer
arithmetic in int64, torch's CPU bf16 conversion and numpy's float16, and
numpy's reshape-sum and lexsort (block scores, the top-k order); for the
backward, the forward oracle itself (each gradient is checked as the adjoint of
the pinned forward map) besides numpy products and int64 sums.
"""
import json
import math
import os

import numpy as np

import workloads as wl

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _expand(mask, b_r, b_c):
    return np.kron(np.asarray(mask, np.float64), np.ones((b_r, b_c))) != 0


def _pruned_f64(W, dtype, mask, b_r, b_c):
    """Pruned weight in float64 built with numpy (select, not multiply)."""
    return np.where(_expand(mask, b_r, b_c), wl.to_f32(W, dtype).astype(np.float64), 0.0)


def _rand_case(seed, N, K, b_r, b_c, dtype, M=None, p_keep=0.5):
    g = np.random.default_rng(seed)
    W = wl.quantize(g.normal(0, 1, (N, K)).astype(np.float32), dtype)
    mask = (g.random((N // b_r, K // b_c)) < p_keep).astype(np.uint8)
    bias = wl.quantize(g.normal(0, 1, N).astype(np.float32), dtype)
    X = wl.quantize(g.normal(0, 1, (M or 8, K)).astype(np.float32), dtype)
    return X, W, mask, bias


# ---------------------------------------------------------------- decoders

def pin_decode_bf16_vs_torch(orc):
    """Every bf16 bit pattern decodes to torch's own bf16 -> float64 value."""
    import torch
    bits = np.arange(1 << 16, dtype=np.uint16)
    got = orc.decode(bits, "bf16")
    ref = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    # signed zeros survive
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def pin_decode_f16_vs_numpy(orc):
    """Every binary16 bit pattern decodes to numpy's float16 -> float64 value."""
    bits = np.arange(1 << 16, dtype=np.uint16)
    h = bits.view(np.float16)
    got = orc.decode(h, "f16")
    ref = h.astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def pin_decode_f32(orc):
    g = np.random.default_rng(7)
    u = g.integers(0, 1 << 32, size=20000, dtype=np.uint64).astype(np.uint32)
    f = np.concatenate([u.view(np.float32), np.array([0.0, -0.0, np.inf, -np.inf, 1e-45, -3.4e38],
                                                     np.float32)])
    got = orc.decode(f, "f32")
    with np.errstate(invalid="ignore"):
        ref = f.astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


# ---------------------------------------------------------------- GELU

def pin_gelu_normal_table(orc):
    """GELU(v) = v * Phi(v) at the standard normal table's points, the odd
    part identity GELU(v) - GELU(-v) = v, and its limits."""
    from scipy.special import erf
    for p in _golden("gelu_normal_cdf.json")["points"]:
        v = p["v"]
        assert math.isclose(orc.gelu(v), v * p["Phi"], rel_tol=1e-15, abs_tol=1e-300)
    for v in np.linspace(-6, 6, 97):
        assert math.isclose(orc.gelu(v) - orc.gelu(-v), v, rel_tol=1e-13, abs_tol=1e-15)
        ref = 0.5 * v * (1.0 + erf(v / math.sqrt(2.0)))
        assert math.isclose(orc.gelu(v), ref, rel_tol=1e-14, abs_tol=1e-300)
    assert orc.gelu(0.0) == 0.0
    assert orc.gelu(12.0) == 12.0
    assert orc.gelu(-12.0) == 0.0 or abs(orc.gelu(-12.0)) < 1e-30


# ---------------------------------------------------------------- pack

def pin_hand_worked(orc):
    """The worked 4x4 example with 2x2 blocks (Sec. 3.1 / Sec. 3.4 fixture)."""
    g = _golden("hand_worked_4x4_2x2.json")
    W = np.array(g["W"], np.float32)
    mask = np.array(g["mask"], np.uint8)
    b_r, b_c = g["b_r"], g["b_c"]
    assert int(mask.sum()) == g["kept_blocks"] == math.ceil((1 - g["alpha"]) * mask.size)
    rp, ci, vals = orc.pack(W, "f32", b_r, b_c, mask)
    assert rp.tolist() == g["row_ptr"]
    assert ci.tolist() == g["col_idx"]
    assert vals.tolist() == g["values"]
    assert orc.unpack(rp, ci, vals, "f32", 4, 4, b_r, b_c).tolist() == g["W_pruned"]
    X = np.array(g["X"], np.float32)
    bias = np.array(g["bias"], np.float32)
    Y = orc.linear(X, W, "f32", b_r, b_c, mask, bias, nthreads=1)
    assert Y.tolist() == g["Y"]


PACK_SHAPES = ((16, 16), (16, 32), (32, 16), (32, 32), (64, 32), (32, 64), (64, 64))


def pin_pack_vs_scipy(orc):
    """row_ptr / col_idx / values equal scipy.sparse.bsr_matrix's indptr /
    indices / data of the pruned weight (no kept block is all zero here)."""
    import scipy.sparse as sp
    for i, (b_r, b_c) in enumerate(PACK_SHAPES):
        for dtype in ("f32", "f16", "bf16"):
            N, K = 2 * 64, 3 * 64
            g = np.random.default_rng(100 + i)
            W = wl.quantize((g.normal(0, 1, (N, K)) + 0.01).astype(np.float32), dtype)
            Wf = wl.to_f32(W, dtype)
            assert np.all(Wf != 0)
            mask = (g.random((N // b_r, K // b_c)) < 0.4).astype(np.uint8)
            mask[0, :] = 0  # an empty block-row
            mask[-1, :] = 1  # a full one
            rp, ci, vals = orc.pack(W, dtype, b_r, b_c, mask)
            ref = sp.bsr_matrix(np.where(_expand(mask, b_r, b_c), Wf, 0.0).astype(np.float32),
                                blocksize=(b_r, b_c))
            ref.sort_indices()
            assert np.array_equal(rp, ref.indptr)
            assert np.array_equal(ci, ref.indices)
            got = wl.to_f32(vals, dtype)
            assert got.shape == ref.data.shape
            assert np.array_equal(got, ref.data)
            assert len(ci) == int(mask.sum())


def pin_pack_roundtrip(orc):
    """unpack(pack(W, mask)) is the selected weight bit for bit, dropped
    blocks hold +0.0 even where W held NaN or Inf, and pack(unpack(P)) == P."""
    for i, (b_r, b_c) in enumerate(PACK_SHAPES):
        for dtype in ("f32", "f16", "bf16"):
            N, K = 128, 128
            g = np.random.default_rng(200 + i)
            W = wl.quantize(g.normal(0, 1, (N, K)).astype(np.float32), dtype)
            mask = (g.random((N // b_r, K // b_c)) < 0.5).astype(np.uint8)
            exp = _expand(mask, b_r, b_c)
            Wbad = W.copy()
            bad = wl.quantize(np.array([np.nan, np.inf], np.float32), dtype)
            Wbad[~exp] = bad[0]
            Wbad[~exp & (np.arange(K)[None, :] % 2 == 0)] = bad[1]
            rp, ci, vals = orc.pack(Wbad, dtype, b_r, b_c, mask)
            Wu = orc.unpack(rp, ci, vals, dtype, N, K, b_r, b_c)
            bits = lambda a: a.view(np.uint32 if a.dtype == np.float32 else np.uint16)
            assert np.array_equal(bits(Wu)[exp], bits(W)[exp])
            assert np.all(bits(Wu)[~exp] == 0)
            rp2, ci2, vals2 = orc.pack(Wu, dtype, b_r, b_c, mask)
            assert np.array_equal(rp, rp2) and np.array_equal(ci, ci2)
            assert np.array_equal(bits(vals), bits(vals2))


# ---------------------------------------------------------------- contraction

def pin_identity_recovers_weight(orc):
    """X = I_K gives Y = W~^T + b exactly: row m of Y is column m of the
    pruned weight.  N != K, so a transposed operand cannot pass."""
    for dtype, (b_r, b_c) in (("bf16", (32, 16)), ("f32", (16, 32)), ("f16", (64, 32))):
        N, K = 192, 128
        _, W, mask, bias = _rand_case(11, N, K, b_r, b_c, dtype)
        X = wl.quantize(np.eye(K, dtype=np.float32), dtype)
        Y = orc.linear(X, W, dtype, b_r, b_c, mask, bias, nthreads=3)
        Wp = _pruned_f64(W, dtype, mask, b_r, b_c)
        b = wl.to_f32(bias, dtype).astype(np.float64)
        assert np.array_equal(Y, Wp.T + b[None, :])


def pin_onehot_rows(orc):
    """A one-hot row e_k of X returns column k of the pruned weight scaled by
    the hot value (a power of two, so exact)."""
    dtype, b_r, b_c = "bf16", 16, 16
    N, K = 64, 96
    _, W, mask, _ = _rand_case(12, N, K, b_r, b_c, dtype)
    ks = [0, 15, 16, 47, 95]
    Xf = np.zeros((len(ks), K), np.float32)
    for i, k in enumerate(ks):
        Xf[i, k] = 4.0
    Y = orc.linear(wl.quantize(Xf, dtype), W, dtype, b_r, b_c, mask, None, nthreads=1)
    Wp = _pruned_f64(W, dtype, mask, b_r, b_c)
    for i, k in enumerate(ks):
        assert np.array_equal(Y[i], 4.0 * Wp[:, k])


def pin_all_kept_is_dense(orc):
    """With every block kept the layer is the dense product: numpy.matmul in
    float64 agrees to float64 rounding."""
    for dtype in ("f32", "bf16"):
        X, W, _, bias = _rand_case(13, 96, 160, 32, 32, dtype, M=37)
        mask = np.ones((3, 5), np.uint8)
        Y = orc.linear(X, W, dtype, 32, 32, mask, bias, nthreads=2)
        ref = (wl.to_f32(X, dtype).astype(np.float64) @ wl.to_f32(W, dtype).astype(np.float64).T
               + wl.to_f32(bias, dtype).astype(np.float64))
        assert np.max(np.abs(Y - ref)) <= 1e-12 * np.max(np.abs(ref))


def pin_none_kept_is_bias(orc):
    """With no block kept the output is the bias, or GELU(bias), exactly."""
    from scipy.special import erf
    X, W, _, bias = _rand_case(14, 64, 64, 16, 16, "bf16", M=9)
    mask = np.zeros((4, 4), np.uint8)
    b = wl.to_f32(bias, "bf16").astype(np.float64)
    Y = orc.linear(X, W, "bf16", 16, 16, mask, bias)
    assert np.array_equal(Y, np.broadcast_to(b, Y.shape))
    Yg = orc.linear(X, W, "bf16", 16, 16, mask, bias, gelu=True)
    ref = 0.5 * b * (1.0 + erf(b / math.sqrt(2.0)))
    assert np.allclose(Yg, np.broadcast_to(ref, Yg.shape), rtol=1e-14, atol=0)
    Y0 = orc.linear(X, W, "bf16", 16, 16, mask, None)
    assert np.all(Y0 == 0.0)


def pin_complement_additivity(orc):
    """Y(mask) + Y(not mask) - b = Y(all kept): every block is counted once."""
    X, W, mask, bias = _rand_case(15, 128, 96, 32, 16, "f16", M=21)
    full = np.ones_like(mask)
    b = wl.to_f32(bias, "f16").astype(np.float64)
    Ya = orc.linear(X, W, "f16", 32, 16, mask, bias)
    Yb = orc.linear(X, W, "f16", 32, 16, 1 - mask, bias)
    Yf = orc.linear(X, W, "f16", 32, 16, full, bias)
    assert np.max(np.abs(Ya + Yb - b - Yf)) <= 1e-12 * np.max(np.abs(Yf))


def pin_bruteforce_tiny(orc):
    """Tiny shapes of every block shape: direct summation over the kept
    blocks only, in pure Python, walking the mask block by block."""
    for i, (b_r, b_c) in enumerate(PACK_SHAPES):
        N, K, M = 2 * b_r, 2 * b_c, 3
        X, W, mask, bias = _rand_case(300 + i, N, K, b_r, b_c, "bf16", M=M, p_keep=0.6)
        Xf = wl.to_f32(X, "bf16").astype(np.float64).tolist()
        Wf = wl.to_f32(W, "bf16").astype(np.float64).tolist()
        bf = wl.to_f32(bias, "bf16").astype(np.float64).tolist()
        ref = [[bf[n] for n in range(N)] for _ in range(M)]
        for r in range(N // b_r):
            for c in range(K // b_c):
                if not mask[r][c]:
                    continue
                for m in range(M):
                    for i2 in range(b_r):
                        s = 0.0
                        for j2 in range(b_c):
                            s += Xf[m][c * b_c + j2] * Wf[r * b_r + i2][c * b_c + j2]
                        ref[m][r * b_r + i2] += s
        Y = orc.linear(X, W, "bf16", b_r, b_c, mask, bias, nthreads=1)
        ref = np.array(ref)
        assert np.max(np.abs(Y - ref)) <= 1e-12 * max(1.0, np.max(np.abs(ref)))


def pin_exact_integers(orc):
    """Small-integer inputs: the product is exact in float64 and must equal
    the int64 product of the selected weight."""
    g = np.random.default_rng(16)
    for dtype, (b_r, b_c) in (("bf16", (32, 32)), ("f16", (16, 64)), ("f32", (64, 16))):
        M, N, K = 33, 128, 192
        Xi = g.integers(-2, 3, size=(M, K))
        Wi = g.integers(-2, 3, size=(N, K))
        bi = g.integers(-4, 5, size=N)
        mask = (g.random((N // b_r, K // b_c)) < 0.5).astype(np.uint8)
        ref = Xi @ np.where(_expand(mask, b_r, b_c), Wi, 0).T + bi
        Y = orc.linear(wl.quantize(Xi, dtype), wl.quantize(Wi, dtype), dtype, b_r, b_c, mask,
                       wl.quantize(bi, dtype), nthreads=4)
        assert np.array_equal(Y, ref.astype(np.float64))


def pin_nonfinite_in_dropped_blocks(orc):
    """NaN / Inf stored in dropped blocks never reaches Y; a NaN in a kept
    block does (the oracle does not hide bad kept weights)."""
    X, W, mask, bias = _rand_case(17, 64, 64, 16, 16, "bf16", M=5)
    mask[1, 2] = 0
    mask[0, 0] = 1
    clean = orc.linear(X, W, "bf16", 16, 16, mask, bias)
    W2 = W.copy()
    exp = _expand(mask, 16, 16)
    W2[~exp] = wl.quantize(np.array([np.nan], np.float32), "bf16")[0]
    W2[16:32, 32:48] = wl.quantize(np.array([np.inf], np.float32), "bf16")[0]
    assert np.array_equal(orc.linear(X, W2, "bf16", 16, 16, mask, bias), clean)
    W3 = W.copy()
    W3[0, 0] = wl.quantize(np.array([np.nan], np.float32), "bf16")[0]
    Y3 = orc.linear(X, W3, "bf16", 16, 16, mask, bias)
    assert np.all(np.isnan(Y3[:, 0]))


def pin_thread_invariance(orc):
    X, W, mask, bias = _rand_case(18, 96, 64, 32, 32, "f32", M=50)
    Y1 = orc.linear(X, W, "f32", 32, 32, mask, bias, gelu=True, nthreads=1)
    Y7 = orc.linear(X, W, "f32", 32, 32, mask, bias, gelu=True, nthreads=7)
    assert np.array_equal(Y1, Y7)


def pin_rejects_bad_grids(orc):
    """Block sizes that do not divide the weight are rejected (the score grid
    has H/B_h x W/B_w entries, Sec. 3.1)."""
    W = np.zeros((48, 64), np.float32)
    for b_r, b_c in ((32, 32), (16, 48), (0, 16)):
        try:
            orc.pack(W, "f32", b_r, b_c, np.ones((max(1, 48 // max(b_r, 1)), 1), np.uint8))
        except ValueError:
            continue
        raise AssertionError("block %dx%d accepted for a 48x64 weight" % (b_r, b_c))
    m = np.ones(64, np.uint8)
    assert orc.lib.lpvo_pack(0, W.ctypes.data, 64, 48, 64, 32, 32, m.ctypes.data,
                             None, None, None) == -1
    assert orc.lib.lpvo_pack(0, W.ctypes.data, 64, 48, 64, 16, 16, m.ctypes.data,
                             None, None, None) == 12


# ---- block scores and the top-k mask (Sec. 3.1 ranking, Sec. 3.4 count) ----

def pin_scores_vs_numpy(orc):
    """Block scores equal numpy's block sums (reshape + sum, its own order)
    to 1e-12 relative, and exactly for integer-valued weights; the Taylor form
    is the mean of |W * G| (signs in both W and G)."""
    g = np.random.default_rng(31)
    for dtype, N, K, b_r, b_c in (("f32", 64, 96, 16, 32), ("bf16", 96, 64, 32, 16),
                                  ("f16", 128, 128, 64, 64)):
        W = wl.quantize(g.standard_normal((N, K)).astype(np.float32), dtype)
        G = wl.quantize(g.standard_normal((N, K)).astype(np.float32), dtype)
        w, gg = orc.decode(W, dtype), orc.decode(G, dtype)
        R, C = N // b_r, K // b_c
        l2 = (w * w).reshape(R, b_r, C, b_c).sum(axis=(1, 3))
        ty = np.abs(w * gg).reshape(R, b_r, C, b_c).mean(axis=(1, 3))
        np.testing.assert_allclose(orc.block_scores(W, dtype, b_r, b_c), l2, rtol=1e-12)
        np.testing.assert_allclose(orc.block_scores(W, dtype, b_r, b_c, G), ty, rtol=1e-12)
    Wi = g.integers(-8, 9, (64, 64)).astype(np.float32)
    Gi = g.integers(-8, 9, (64, 64)).astype(np.float32)
    l2 = (Wi.astype(np.float64) ** 2).reshape(4, 16, 4, 16).sum(axis=(1, 3))
    assert np.array_equal(orc.block_scores(Wi, "f32", 16, 16), l2)
    ty = np.abs(Wi.astype(np.float64) * Gi).reshape(4, 16, 4, 16).sum(axis=(1, 3)) / 256.0
    assert np.array_equal(orc.block_scores(Wi, "f32", 16, 16, Gi), ty)


def pin_scores_onehot_block(orc):
    """A weight that is zero except in block (r, c) scores zero everywhere but
    (r, c): the score grid is indexed (row-block, column-block)."""
    N, K, b_r, b_c = 96, 64, 32, 16
    for r, c in ((0, 3), (2, 1), (1, 0)):
        W = np.zeros((N, K), np.float32)
        W[r * b_r:(r + 1) * b_r, c * b_c:(c + 1) * b_c] = 0.5
        s = orc.block_scores(W, "f32", b_r, b_c)
        want = np.zeros((N // b_r, K // b_c))
        want[r, c] = 0.25 * b_r * b_c
        assert np.array_equal(s, want), (r, c)


def pin_keep_count_ceiling(orc):
    """ceil((1 - alpha) R C) (Sec. 3.4) at integer percentages."""
    cases = {(2304, 50): 1152, (2304, 25): 1728, (10, 33): 7, (3, 50): 2, (7, 0): 7,
             (7, 100): 0, (0, 50): 0, (9216, 90): 922, (576, 90): 58, (100, 1): 99}
    for (n, p), want in cases.items():
        assert orc.keep_count(n, p) == want, (n, p)


def pin_topk_vs_lexsort(orc):
    """The mask keeps the first n_keep of numpy's lexsort by (-score, index),
    for random scores with many exact ties."""
    g = np.random.default_rng(32)
    for R, C in ((1, 1), (3, 5), (12, 24), (48, 12)):
        s = g.integers(0, 6, (R, C)).astype(np.float64) * 0.25
        for keep in sorted({0, 1, R * C // 2, R * C - 1, R * C}):
            keep = max(0, keep)
            order = np.lexsort((np.arange(R * C), -s.reshape(-1)))
            want = np.zeros(R * C, np.uint8)
            want[order[:keep]] = 1
            assert np.array_equal(orc.mask_topk(s, keep).reshape(-1), want), (R, C, keep)


def pin_topk_ties_to_lower_index(orc):
    """Equal scores: the lower row-major indices are kept; strictly decreasing
    scores keep a prefix; the highest score is always kept."""
    s = np.full((4, 6), 2.0)
    m = orc.mask_topk(s, 10).reshape(-1)
    assert m[:10].all() and not m[10:].any()
    d = np.arange(24, 0, -1, dtype=np.float64).reshape(4, 6)
    assert np.array_equal(orc.mask_topk(d, 5).reshape(-1), (np.arange(24) < 5).astype(np.uint8))
    u = np.arange(24, dtype=np.float64).reshape(4, 6)
    assert orc.mask_topk(u, 1)[3, 5] == 1 and orc.mask_topk(u, 1).sum() == 1


# ---------------------------------------------------------------- backward

def _grad_case(seed, M, N, K, b_r, b_c, dtype="f32", integers=False):
    g = np.random.default_rng(seed)
    if integers:
        draw = lambda shape: g.integers(-3, 4, shape).astype(np.float32)
    else:
        draw = lambda shape: g.normal(0, 1, shape).astype(np.float32)
    G = wl.quantize(draw((M, N)), dtype)
    X = wl.quantize(draw((M, K)), dtype)
    W = wl.quantize(draw((N, K)), dtype)
    mask = (g.random((N // b_r, K // b_c)) < 0.5).astype(np.uint8)
    mask[0, 0] = 1
    return G, X, W, mask


def _close(a, b, rtol=1e-12):
    assert abs(a - b) <= rtol * max(1.0, abs(a), abs(b)), (a, b)


def pin_grad_x_adjoint_of_forward(orc):
    # <dX, V> = <G, V W~^T>: the input gradient is the adjoint of the forward
    # map, which is pinned on its own (the forward oracle runs with X = V)
    for (b_r, b_c) in [(16, 32), (32, 16)]:
        G, X, W, mask = _grad_case(71 + b_r, 9, 96, 64, b_r, b_c)
        V = np.random.default_rng(72).normal(0, 1, X.shape).astype(np.float32)
        dX = orc.grad_x(G, W, "f32", b_r, b_c, mask)
        Y = orc.linear(V, W, "f32", b_r, b_c, mask)
        _close(float((dX * V.astype(np.float64)).sum()), float((Y * G.astype(np.float64)).sum()))


def pin_grad_x_vs_numpy(orc):
    # dX = G W~ with numpy's product over the numpy-built pruned weight
    G, X, W, mask = _grad_case(73, 7, 64, 96, 32, 16, dtype="bf16")
    dX = orc.grad_x(G, W, "bf16", 32, 16, mask)
    ref = wl.to_f32(G, "bf16").astype(np.float64) @ _pruned_f64(W, "bf16", mask, 32, 16)
    assert np.allclose(dX, ref, rtol=1e-12, atol=1e-12)


def pin_grad_w_vs_numpy(orc):
    # the kept blocks of numpy's G^T X, in BSR order (rows, then kept columns)
    for (b_r, b_c) in [(16, 32), (32, 16)]:
        G, X, W, mask = _grad_case(74 + b_c, 11, 96, 64, b_r, b_c, dtype="f16")
        dW = orc.grad_w(G, X, "f16", b_r, b_c, mask)
        full = G.astype(np.float64).T @ X.astype(np.float64)
        ref = [full[r * b_r:(r + 1) * b_r, c * b_c:(c + 1) * b_c]
               for r in range(mask.shape[0]) for c in range(mask.shape[1]) if mask[r, c]]
        assert dW.shape == (len(ref), b_r, b_c)
        assert np.allclose(dW, np.array(ref), rtol=1e-12, atol=1e-12)


def pin_grad_w_adjoint_of_forward(orc):
    # <dW, U> over the kept blocks = <G, X U~^T>, the forward oracle with weight U
    G, X, W, mask = _grad_case(75, 13, 64, 96, 16, 32)
    U = np.random.default_rng(76).normal(0, 1, W.shape).astype(np.float32)
    dW = orc.grad_w(G, X, "f32", 16, 32, mask)
    _, _, Ub = orc.pack(U, "f32", 16, 32, mask)
    Y = orc.linear(X, U, "f32", 16, 32, mask)
    _close(float((dW * Ub.astype(np.float64)).sum()), float((Y * G.astype(np.float64)).sum()))


def pin_grad_bias_adjoint_and_exact(orc):
    # <db, u> = <G, Y> for the forward oracle with X = 0 and bias u (Y[m] = u);
    # with integer G every partial sum is exact, so db equals int64 sums
    G, X, W, mask = _grad_case(77, 10, 64, 32, 16, 16)
    u = np.random.default_rng(78).normal(0, 1, 64).astype(np.float32)
    db = orc.grad_bias(G, "f32")
    Y = orc.linear(np.zeros_like(X), W, "f32", 16, 16, mask, bias=u)
    _close(float((db * u.astype(np.float64)).sum()), float((Y * G.astype(np.float64)).sum()))
    Gi, _, _, _ = _grad_case(79, 33, 48, 16, 16, 16, integers=True)
    assert np.array_equal(orc.grad_bias(Gi, "f32"), Gi.astype(np.int64).sum(axis=0).astype(np.float64))


def pin_grad_exact_integers(orc):
    # small integers: every product and partial sum is exact, so both
    # gradients equal int64 arithmetic exactly
    G, X, W, mask = _grad_case(80, 17, 64, 96, 32, 16, integers=True)
    Wi = np.where(_expand(mask, 32, 16), W.astype(np.int64), 0)
    assert np.array_equal(orc.grad_x(G, W, "f32", 32, 16, mask),
                          (G.astype(np.int64) @ Wi).astype(np.float64))
    full = G.astype(np.int64).T @ X.astype(np.int64)
    dW = orc.grad_w(G, X, "f32", 32, 16, mask)
    k = 0
    for r in range(mask.shape[0]):
        for c in range(mask.shape[1]):
            if mask[r, c]:
                assert np.array_equal(dW[k], full[r * 32:(r + 1) * 32, c * 16:(c + 1) * 16])
                k += 1
    assert k == dW.shape[0]


# ---------------------------------------------------------------- delta curve

def _delta_case(seed, N, K, n_s, dtype="f32", integers=False):
    g = np.random.default_rng(seed)
    if integers:
        draw = lambda shape: g.integers(-3, 4, shape).astype(np.float32)
    else:
        draw = lambda shape: g.normal(0, 1, shape).astype(np.float32)
    return (wl.quantize(draw((N, K)), dtype), wl.quantize(draw((N, K)), dtype),
            wl.quantize(draw((n_s, N, K)), dtype))


def _dropped_numpy(W, grad, b_r, b_c, p):
    """Dropped-block mask with numpy alone: block means of |W grad|, ranked by
    (-score, row-major index), the top ceil((100 - p) R C / 100) kept."""
    N, K = W.shape
    R, C = N // b_r, K // b_c
    a = np.abs(W.astype(np.float64) * grad.astype(np.float64))
    sc = a.reshape(R, b_r, C, b_c).sum(axis=(1, 3)).ravel() / (b_r * b_c)
    keep = -((p - 100) * R * C // 100)  # integer ceiling of (100 - p) R C / 100
    order = np.lexsort((np.arange(R * C), -sc))
    kept = np.zeros(R * C, bool)
    kept[order[:keep]] = True
    return ~_expand(kept.reshape(R, C).astype(np.uint8), b_r, b_c)


def pin_delta_zero_without_pruning(orc):
    W, gr, S = _delta_case(81, 64, 32, 3)
    assert orc.delta_curve(W, "f32", 16, 16, gr, S, 0.5, [0])[0] == 0.0


def pin_delta_vs_dense_fisher(orc):
    # the explicit Hessian kappa I + (1/n) sum g g^T as a dense numpy matrix,
    # the dropped set from numpy's own block scores and lexsort
    for (b_r, b_c, integers) in [(16, 16, False), (16, 32, False), (32, 16, True)]:
        W, gr, S = _delta_case(82 + b_c, 64, 64, 4, integers=integers)
        pcts = [0, 10, 25, 50, 75, 90, 100]
        got = orc.delta_curve(W, "f32", b_r, b_c, gr, S, 0.25, pcts)
        Gs = S.reshape(4, -1).astype(np.float64)
        H = 0.25 * np.eye(Gs.shape[1]) + Gs.T @ Gs / 4
        for i, p in enumerate(pcts):
            dw = np.where(_dropped_numpy(W, gr, b_r, b_c, p), -W.astype(np.float64), 0.0).ravel()
            ref = gr.astype(np.float64).ravel() @ dw + 0.5 * dw @ H @ dw
            if integers:
                assert got[i] == ref, (p, got[i], ref)  # every term exact
            else:
                assert abs(got[i] - ref) <= 1e-10 * max(1.0, abs(ref)), (p, got[i], ref)


def pin_delta_incremental_update(orc):
    # the paper's update from one ratio to the next: with d the newly pruned
    # part and D the previous change, delta_k - delta_{k-1} =
    # grad' . d + (d / 2 + D)^T H' d, H' the Fisher restricted to d's support
    W, gr, S = _delta_case(85, 64, 96, 5)
    pcts = [0, 20, 40, 60, 80, 100]
    got = orc.delta_curve(W, "f32", 16, 32, gr, S, 0.1, pcts)
    Gs = S.reshape(5, -1).astype(np.float64)
    prev = np.zeros(W.size)
    acc = 0.0
    for i, p in enumerate(pcts):
        cur = np.where(_dropped_numpy(W, gr, 16, 32, p), -W.astype(np.float64), 0.0).ravel()
        d = cur - prev
        sup = d != 0
        # H' d: the columns of H on d's support (a D-vector)
        Hd = 0.1 * d + Gs.T @ (Gs[:, sup] @ d[sup]) / 5
        acc += gr.astype(np.float64).ravel()[sup] @ d[sup] + (0.5 * d + prev) @ Hd
        assert abs(got[i] - acc) <= 1e-9 * max(1.0, abs(acc)), (p, got[i], acc)
        prev = cur


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
