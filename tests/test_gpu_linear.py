"""GPU parity of lpv_bsr_linear and lpv_dense_linear against the float64
oracle, on the same seeded inputs.

Bar: infinity-norm relative error (max|y - r| / max|r|) <= 2e-2 (bf16),
5e-3 (fp16), 1e-5 (fp32), float32 accumulation, both over the whole result
and within every 32 x 32 output tile (gpu_util.assert_close).  Small-integer inputs make the result exact in every
format and order, and then the GPU must match the oracle bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from gpu_util import TOL, TORCH, assert_close, bits, dev, f64, host, say
from paper_2407_02068_amd import lpv

pytestmark = pytest.mark.gpu

SHAPES = ((16, 16), (16, 32), (32, 16), (32, 32), (64, 32), (32, 64), (64, 64))


def run_bsr(w, X=None, gelu=None):
    X = w.X if X is None else X
    h = lpv.bsr_pack(dev(w.W, w.dtype), dev(w.mask), w.b_r, w.b_c)
    b = None if w.bias is None else dev(w.bias, w.dtype)
    Y = lpv.bsr_linear(h, dev(X, w.dtype), b, epi="gelu" if (w.gelu if gelu is None else gelu) else None)
    torch.cuda.synchronize()
    return h, Y


def ref(w, X=None, gelu=None):
    X = w.X if X is None else X
    return oracle.linear(X, w.W, w.dtype, w.b_r, w.b_c, w.mask, w.bias,
                         gelu=w.gelu if gelu is None else gelu)


def test_tiny_fc1_fp32():
    w = wl.tiny_fc1()
    say("tiny_fc1", w.nnzb)
    _, Y = run_bsr(w)
    assert_close(f64(Y), ref(w), "f32", "tiny_fc1")


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("b_r,b_c", SHAPES)
@pytest.mark.parametrize("M", [1, 31, 300])
def test_parity_small(dtype, b_r, b_c, M):
    # N = 384: 12 tile rows, several groups; K = 320 / 384: 10-12 tile columns
    K = 384 if b_c == 64 else 320
    w = wl.custom(30 + b_r + b_c, M, 384, K, b_r, b_c, dtype, "uniform", 50,
                  gelu=(M == 300))
    say("parity", dtype, b_r, b_c, M, "nnzb", w.nnzb)
    _, Y = run_bsr(w)
    assert_close(f64(Y), ref(w), dtype, w.name)


@pytest.mark.parametrize("b_r,b_c", [(16, 16), (32, 32), (64, 64)])
def test_parity_fp32_blocks(b_r, b_c):
    w = wl.custom(40, 129, 192, 192, b_r, b_c, "f32", "bernoulli", 50, gelu=True)
    say("fp32", b_r, b_c)
    _, Y = run_bsr(w)
    assert_close(f64(Y), ref(w), "f32", w.name)


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("b_r,b_c", [(16, 16), (32, 32), (64, 32)])
def test_exact_small_integers(dtype, b_r, b_c):
    """Integer inputs: every partial sum is exact in float32 and the result is
    exact in the output type, so the order of accumulation cannot matter."""
    g = np.random.default_rng(50)
    M, N, K = 300, 256, 320
    Xf = g.integers(-1, 2, size=(M, K)) * (g.random((M, K)) < 0.2)
    Wf = g.integers(-2, 3, size=(N, K))
    bf = g.integers(-8, 9, size=N)
    mask = (g.random((N // b_r, K // b_c)) < 0.5).astype(np.uint8)
    w = wl.Linear("exact", dtype, b_r, b_c, wl.quantize(Wf, dtype), mask, wl.quantize(bf, dtype),
                  False, wl.quantize(Xf, dtype), M)
    r = ref(w)
    assert np.max(np.abs(r)) < 256  # exact in bf16
    say("exact", dtype, b_r, b_c)
    _, Y = run_bsr(w)
    assert np.array_equal(f64(Y), r)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_dense_path(dtype):
    w = wl.custom(60, 300, 384, 320, 32, 32, dtype, "all", 0, gelu=True)
    say("dense", dtype)
    Y = lpv.dense_linear(dev(w.W, dtype), dev(w.X, dtype), dev(w.bias, dtype), epi="gelu")
    torch.cuda.synchronize()
    assert_close(f64(Y), ref(w), dtype, "dense")
    # the block-sparse path with every block kept computes the same thing
    _, Ys = run_bsr(w)
    assert_close(f64(Ys), ref(w), dtype, "all-kept bsr")


def test_dense_fp32():
    w = wl.custom(61, 70, 64, 96, 32, 32, "f32", "all", 0)
    Y = lpv.dense_linear(dev(w.W, "f32"), dev(w.X, "f32"), dev(w.bias, "f32"))
    torch.cuda.synchronize()
    assert_close(f64(Y), ref(w), "f32", "dense fp32")


@pytest.mark.parametrize("gelu", [False, True])
def test_no_kept_block_gives_bias(gelu):
    w = wl.custom(62, 257, 256, 192, 32, 32, "bf16", "none", 100, gelu=gelu)
    say("none kept", gelu)
    h, Y = run_bsr(w)
    assert h.info["nnzb"] == 0
    r = ref(w)
    if gelu:
        assert_close(f64(Y), r, "bf16", "gelu(bias)")
    else:
        assert np.array_equal(f64(Y), r)  # bias is a bf16 value: exact
    w.bias = None
    _, Y0 = run_bsr(w)
    assert torch.count_nonzero(Y0).item() == 0


def test_nonfinite_dropped_blocks_do_not_leak():
    w = wl.custom(63, 200, 256, 256, 32, 32, "bf16", "uniform", 50)
    _, Y = run_bsr(w)
    exp = np.kron(w.mask, np.ones((32, 32), np.uint8)) == 0
    W2 = w.W.copy()
    W2[exp] = wl.quantize(np.array([np.nan], np.float32), "bf16")[0]
    W2[exp & (np.arange(256)[None, :] % 3 == 0)] = wl.quantize(np.array([np.inf], np.float32), "bf16")[0]
    w2 = wl.Linear("nan", "bf16", 32, 32, W2, w.mask, w.bias, False, w.X, w.M)
    _, Y2 = run_bsr(w2)
    assert torch.isfinite(Y2.float()).all()
    assert torch.equal(Y.view(torch.int16), Y2.view(torch.int16))


def test_deterministic_and_token_permutation():
    w = wl.custom(64, 700, 384, 320, 32, 32, "bf16", "zipf", 40, gelu=True)
    h, Y1 = run_bsr(w)
    b = dev(w.bias, "bf16")
    X = dev(w.X, "bf16")
    Y2 = lpv.bsr_linear(h, X, b, epi="gelu")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        Y3 = lpv.bsr_linear(h, X, b, epi="gelu")
    torch.cuda.synchronize()
    assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16))
    assert torch.equal(Y1.view(torch.int16), Y3.view(torch.int16))
    perm = torch.from_numpy(np.random.default_rng(5).permutation(700)).cuda()
    Yp = lpv.bsr_linear(h, X[perm].contiguous(), b, epi="gelu")
    torch.cuda.synchronize()
    assert torch.equal(Yp.view(torch.int16), Y1[perm].view(torch.int16))


@pytest.mark.parametrize("dtype,b_c,K", [("bf16", 32, 192), ("bf16", 16, 176), ("f32", 16, 192)])
def test_strided_views_and_guard_bands(dtype, b_c, K):
    """X read through a column slice of a wider buffer (ldx > K); Y written
    into the middle of a padded buffer (ldy > N) whose canaries must survive.
    Also with 16-wide block columns and a 16-column reduction tail (the
    half-tile walk and the zero line in place of X past K)."""
    w = wl.custom(65, 197, 256, K, 32, b_c, dtype, "uniform", 40)
    tt = TORCH[dtype]
    big = torch.zeros((w.M, 3 * w.K), dtype=tt, device="cuda")
    big[:, w.K:2 * w.K] = dev(w.X, dtype)
    Xv = big[:, w.K:2 * w.K]
    ldy = w.N + 64
    canary = torch.full((w.M + 2, ldy), -7.0, dtype=tt, device="cuda")
    Yv = canary[1:w.M + 1, :w.N]
    h = lpv.bsr_pack(dev(w.W, dtype), dev(w.mask), w.b_r, w.b_c)
    lpv.bsr_linear(h, Xv, dev(w.bias, dtype), Y=Yv)
    torch.cuda.synchronize()
    assert_close(f64(Yv), ref(w), dtype, "strided")
    c = canary.float().cpu()
    assert torch.all(c[0] == -7) and torch.all(c[-1] == -7) and torch.all(c[:, w.N:] == -7)


def test_m_zero_is_noop():
    w = wl.custom(66, 1, 64, 64, 32, 32, "bf16", "uniform", 50)
    h = lpv.bsr_pack(dev(w.W, "bf16"), dev(w.mask), 32, 32)
    Y = lpv.bsr_linear(h, torch.empty((0, 64), dtype=torch.bfloat16, device="cuda"))
    assert Y.shape == (0, 64)


def test_rejects_aliasing_and_wrong_device_layouts():
    w = wl.custom(67, 64, 64, 64, 32, 32, "bf16", "uniform", 50)
    h = lpv.bsr_pack(dev(w.W, "bf16"), dev(w.mask), 32, 32)
    buf = torch.zeros((64, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(lpv.LpvError) as e:
        lpv.bsr_linear(h, buf[:, :64], Y=buf[:, 64:])
    assert e.value.status == -5
    with pytest.raises(lpv.LpvError):
        lpv.bsr_linear(h, buf[:, 1:65])  # misaligned X


def _sampled_rows(M, n=64, seed=0):
    g = np.random.default_rng(seed)
    rows = set(range(min(n, M))) | set(range(max(0, M - n), M))
    rows |= set(g.choice(M, size=min(n, M), replace=False).tolist())
    return np.array(sorted(rows))


def _full_size(w, gelu=None, seed=0):
    """Full-size run (the benchmark's launch configuration), checked on
    sampled token rows (first, last including the tail, random)."""
    say("full size", w.name, "M", w.M, "nnzb", w.nnzb)
    _, Y = run_bsr(w, gelu=gelu)
    rows = _sampled_rows(w.M, seed=seed)
    r = ref(w, X=w.X[rows], gelu=gelu)
    y = f64(Y[torch.from_numpy(rows).cuda()])
    assert_close(y, r, w.dtype, w.name + " sampled")
    return Y


def test_full_headline_fc1():
    _full_size(wl.b_fc1())


def test_full_headline_fc1_fp16_gelu():
    _full_size(wl.b_fc1(dtype="f16", gelu=True))


def test_full_s_fc1_gelu():
    _full_size(wl.s_fc1_gelu())


def test_full_b_layer():
    for w in wl.b_layer():
        _full_size(w)


@pytest.mark.parametrize("block", [16, 64])
def test_full_fc1_other_blocks(block):
    _full_size(wl.b_fc1(block=block, sparsity=75))


def test_full_dense_headline_shape():
    w = wl.b_fc1(sparsity=0)
    say("dense full", w.name)
    Y = lpv.dense_linear(dev(w.W, "bf16"), dev(w.X, "bf16"), dev(w.bias, "bf16"))
    torch.cuda.synchronize()
    rows = _sampled_rows(w.M)
    r = oracle.linear(w.X[rows], w.W, "bf16", 32, 32, np.ones_like(w.mask), w.bias)
    assert_close(f64(Y[torch.from_numpy(rows).cuda()]), r, "bf16", "dense full sampled")


def test_chain_b_stack_links():
    """The DeiT-B stack (qkv -> V third -> proj -> fc1 + GELU -> fc2) with
    skewed (Zipf) masks, 2 layers at 2 images; each link is checked against
    the oracle fed the GPU's own input to that link."""
    layers = wl.b_stack(M=2 * 197, layers=2)
    X = dev(layers[0].X, "bf16")
    for w in layers:
        h = lpv.bsr_pack(dev(w.W, "bf16"), dev(w.mask), 32, 32)
        Xin = X[:, 1536:2304] if w.name.endswith("proj") else X
        Y = lpv.bsr_linear(h, Xin, dev(w.bias, "bf16"), epi="gelu" if w.gelu else None)
        torch.cuda.synchronize()
        xin = host(Xin.contiguous(), "bf16")
        r = oracle.linear(xin, w.W, "bf16", 32, 32, w.mask, w.bias, gelu=w.gelu)
        assert_close(f64(Y), r, "bf16", w.name)
        X = Y


# ---- 16-wide block columns: tiles walked by 16-column halves -------------------

def _half_mask(g, R, C, pattern):
    """Block masks over 16-wide block columns: kept blocks only in even block
    columns (every kept tile keeps its first 16 columns only), only in odd
    ones (second half only), or anywhere (all three kinds of kept tile)."""
    keep = g.random((R, C)) < (0.6 if pattern != "random" else 0.35)
    if pattern == "first":
        keep[:, 1::2] = False
    elif pattern == "second":
        keep[:, 0::2] = False
    return keep.astype(np.uint8)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("b_r", [16, 32])
@pytest.mark.parametrize("pattern", ["first", "second", "random"])
def test_half_kept_tiles(dtype, b_r, pattern):
    """16-wide block columns: a kept 32 x 32 tile may keep one 16-column half
    and drop the other, and the kernel then moves and multiplies the kept half
    only.  Integer inputs (exact in every order), K = 336 (a 16-column tail),
    M = 300, two output groups; the result must equal the oracle's bit for bit."""
    g = np.random.default_rng(90 + b_r + len(pattern))
    M, N, K = 300, 384, 336
    Xf = g.integers(-1, 2, size=(M, K)) * (g.random((M, K)) < 0.2)
    Wf = g.integers(-2, 3, size=(N, K))
    bf = g.integers(-8, 9, size=N)
    mask = _half_mask(g, N // b_r, K // 16, pattern)
    w = wl.Linear("half." + pattern, dtype, b_r, 16, wl.quantize(Wf, dtype), mask,
                  wl.quantize(bf, dtype), False, wl.quantize(Xf, dtype), M)
    r = ref(w)
    assert np.max(np.abs(r)) < 256  # exact in bf16
    say("half tiles", dtype, b_r, pattern, "nnzb", int(mask.sum()))
    _, Y = run_bsr(w)
    assert np.array_equal(f64(Y), r)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_whole_tiles_as_16x16_blocks(dtype):
    """A 32 x 32 block mask written as 16 x 16 blocks (each kept block as its
    four quarters) keeps the same tiles with both halves: the two handles must
    give the same output bits (GELU on, M = 300, DeiT-S fc1 shape)."""
    w = wl.custom(92, 300, 1536, 384, 32, 32, dtype, "uniform", 50, gelu=True)
    _, Y32 = run_bsr(w)
    w16 = wl.Linear(w.name + ".as16", dtype, 16, 16, w.W, np.kron(w.mask, np.ones((2, 2), np.uint8)),
                    w.bias, True, w.X, w.M)
    _, Y16 = run_bsr(w16)
    say("whole tiles as 16x16", dtype)
    assert torch.equal(Y32.view(torch.int16), Y16.view(torch.int16))
    assert_close(f64(Y16), ref(w), dtype, w16.name)


# ---- shapes and paths the headline shapes never reach ----------------------------

TAIL_SHAPES = ((80, 48, 16, 16), (48, 80, 16, 16), (208, 112, 16, 16), (80, 64, 16, 32),
               (64, 80, 32, 16))


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("N,K,b_r,b_c", TAIL_SHAPES)
def test_tails_of_16_wide_blocks(dtype, N, K, b_r, b_c):
    """N or K = 16 mod 32: the last 32-wide tile row / column is half outside
    the weight (partial tile rows: bias and stores past N masked; K tail: the
    zero line in place of X past K).  Sparse and dense, GELU on, M = 300 (a
    ragged second token tile)."""
    w = wl.custom(70 + N + K, 300, N, K, b_r, b_c, dtype, "uniform", 50, gelu=True)
    say("tails", dtype, "N=%d K=%d" % (N, K), (b_r, b_c), "nnzb", w.nnzb)
    _, Y = run_bsr(w)
    assert_close(f64(Y), ref(w), dtype, w.name)
    Yd = lpv.dense_linear(dev(w.W, dtype), dev(w.X, dtype), dev(w.bias, dtype), epi="gelu")
    torch.cuda.synchronize()
    r = oracle.linear(w.X, w.W, dtype, b_r, b_c, np.ones_like(w.mask), w.bias, gelu=True)
    assert_close(f64(Yd), r, dtype, "dense " + w.name)


def _table_bytes(w):
    """Per-launch table bytes of the block-sparse kernel if every group of 8
    tile rows (256 outputs) went into one launch: 16 B per slot descriptor,
    1 KB of float32 bias per group, 16 B per walk entry (the tile columns the
    group keeps a tile in, padded to an even count).  Square blocks of 16 or
    32 (a 32 x 32 tile is kept when any block it covers is)."""
    assert w.b_r == w.b_c and w.b_r in (16, 32)
    m = w.mask
    if w.b_r == 16:
        R, C = m.shape
        m = m.reshape(R // 2, 2, C // 2, 2).any(axis=(1, 3))
    total = 0
    for g0 in range(0, m.shape[0], 8):
        steps = int(m[g0:g0 + 8].any(axis=0).sum())
        total += 16 + 1024 + 16 * (steps + (steps & 1))
    return total


@pytest.mark.parametrize("N,K,block", [(8192, 768, 32), (4096, 3072, 32), (8192, 768, 16)])
def test_multi_launch_tables(N, K, block):
    """Layers wide enough that the kernel's per-launch tables (walk, slot
    descriptors, bias) exceed the 32 KB it keeps in LDS: the call is split into
    several launches over runs of output groups.  Sparse with GELU (also with
    16 x 16 blocks, whose walk entries carry per-half row bits), and dense."""
    w = wl.custom(75, 300, N, K, block, block, "bf16", "uniform", 50, gelu=True)
    assert _table_bytes(w) > 32 * 1024
    say("multi-launch", N, K, block, "nnzb", w.nnzb)
    _, Y = run_bsr(w)
    assert_close(f64(Y), ref(w), "bf16", w.name)
    if block == 16:
        return
    Yd = lpv.dense_linear(dev(w.W, "bf16"), dev(w.X, "bf16"), dev(w.bias, "bf16"), epi="gelu")
    torch.cuda.synchronize()
    r = oracle.linear(w.X, w.W, "bf16", 32, 32, np.ones_like(w.mask), w.bias, gelu=True)
    assert_close(f64(Yd), r, "bf16", "dense " + w.name)


@pytest.mark.parametrize("dense,block", [(False, 32), (False, 16), (True, 32)])
def test_last_round_split(dense, block):
    """38 token tiles x 12 output groups: with 256 compute units, 8 XCDs of 32
    workgroups, XCDs 0-5 own 5 token tiles (60 items: one whole round of 32
    and 28 left, too many to halve) and XCDs 6-7 own 4 (48 items: 16 left,
    each run as two half items).  Rows of tiles on both kinds of XCD are
    checked against the oracle, for the block-sparse launch (32 x 32 blocks,
    and 16 x 16 blocks, whose tiles are walked by 16-column halves) and the
    dense one."""
    w = wl.custom(78, 38 * 256, 3072, 768, block, block, "bf16", "uniform", 0 if dense else 50)
    say("last round split", "dense" if dense else "sparse", block, "M", w.M, "nnzb", w.nnzb)
    if dense:
        Y = lpv.dense_linear(dev(w.W, "bf16"), dev(w.X, "bf16"), dev(w.bias, "bf16"))
        torch.cuda.synchronize()
    else:
        _, Y = run_bsr(w)
    g = np.random.default_rng(79)
    rows = []
    for tile in (0, 6, 7, 14, 30, 31, 37):
        rows += [tile * 256, tile * 256 + 255] + (tile * 256 + g.choice(256, 14, replace=False)).tolist()
    rows = np.array(sorted(set(rows)))
    r = ref(w, X=w.X[rows])
    assert_close(f64(Y[torch.from_numpy(rows).cuda()]), r, "bf16", w.name + " sampled")


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_zipf_many_token_tiles(dtype):
    """Skewed (Zipf) row keep counts with more than 8 token tiles of 256, so the
    XCD-owned item order of the persistent kernel runs with uneven groups."""
    w = wl.custom(76, 8 * 256 + 77, 768, 384, 32, 32, dtype, "zipf", 40, gelu=True)
    say("zipf", dtype, "M", w.M, "nnzb", w.nnzb)
    _, Y = run_bsr(w)
    assert_close(f64(Y), ref(w), dtype, w.name)


def test_full_b_stack_links_sampled():
    """The first block of the DeiT-B stack at its full size (M = 50432, Zipf
    masks, per-linear sparsity), chained qkv -> V third -> proj -> fc1 + GELU ->
    fc2 on the GPU; each link checked on sampled token rows against the oracle
    fed the GPU's own input rows of that link."""
    layers = wl.b_stack(layers=1)
    X = dev(layers[0].X, "bf16")
    rows = _sampled_rows(layers[0].M, n=48, seed=3)
    rows_d = torch.from_numpy(rows).cuda()
    for w in layers:
        h = lpv.bsr_pack(dev(w.W, "bf16"), dev(w.mask), 32, 32)
        Xin = X[:, 1536:2304] if w.name.endswith("proj") else X
        say("full stack link", w.name, "sparsity", w.meta["sparsity"], "nnzb", w.nnzb)
        Y = lpv.bsr_linear(h, Xin, dev(w.bias, "bf16"), epi="gelu" if w.gelu else None)
        torch.cuda.synchronize()
        xin = host(Xin[rows_d].contiguous(), "bf16")
        r = oracle.linear(xin, w.W, "bf16", 32, 32, w.mask, w.bias, gelu=w.gelu)
        assert_close(f64(Y[rows_d]), r, "bf16", w.name + " sampled")
        h.close()
        X = Y


@pytest.mark.parametrize("dense", [False, True])
def test_largest_reduction(dense):
    """K = 63424, the largest the 16-bit kernels take: one group's walk (1982
    column tiles) fills the kernel's LDS table."""
    w = wl.custom(80, 97, 256, 63424, 32, 32, "bf16", "uniform", 0 if dense else 50, gelu=True)
    say("largest K", "dense" if dense else "sparse", "nnzb", w.nnzb)
    if dense:
        Y = lpv.dense_linear(dev(w.W, "bf16"), dev(w.X, "bf16"), dev(w.bias, "bf16"), epi="gelu")
        torch.cuda.synchronize()
    else:
        _, Y = run_bsr(w)
    assert_close(f64(Y), ref(w), "bf16", w.name)
