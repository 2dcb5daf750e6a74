"""GPU parity of lpv_delta_curve against the float64 oracle, which evaluates
the delta curve's definition directly at every ratio (the GPU takes the
paper's incremental update; both in float64, so they agree to rounding)."""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from gpu_util import dev, say
from paper_2407_02068_amd import lpv

pytestmark = pytest.mark.gpu

TOL = 1e-9  # infinity-norm relative error: float64 sums in another order


def inputs(seed, N, K, n_s, dtype):
    g = np.random.default_rng(seed)
    W = wl.quantize(g.normal(0, 0.02, (N, K)).astype(np.float32), dtype)
    grad = wl.quantize(g.normal(0, 1e-3, (N, K)).astype(np.float32), dtype)
    S = wl.quantize(g.normal(0, 1e-2, (n_s, N, K)).astype(np.float32), dtype)
    return W, grad, S


def check(W, grad, S, dtype, b_r, b_c, kappa, pcts, what=""):
    say("delta_curve", what, dtype, W.shape, (b_r, b_c), "n=%d" % S.shape[0], pcts)
    Sd = dev(S.reshape(S.shape[0], -1), dtype).reshape(S.shape) if S.shape[0] else \
        torch.empty((0,) + W.shape, dtype=dev(W, dtype).dtype, device="cuda")
    got = lpv.delta_curve(dev(W, dtype), dev(grad, dtype), Sd, b_r, b_c, kappa, pcts)
    torch.cuda.synchronize()
    got = got.cpu().numpy()
    ref = oracle.delta_curve(W, dtype, b_r, b_c, grad, S, kappa, pcts)
    scale = max(np.abs(ref).max(), 1e-300)
    err = np.abs(got - ref).max() / scale
    say("  rel err %.2e (max |delta| %.3e)" % (err, scale))
    assert err <= TOL
    return got, ref


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("b_r,b_c", [(32, 32), (16, 16), (64, 32), (16, 64)])
def test_delta_curve_matches_oracle(dtype, b_r, b_c):
    W, grad, S = inputs(101 + b_r + b_c, 256, 192, 5, dtype)
    check(W, grad, S, dtype, b_r, b_c, 0.05, list(range(0, 101, 10)))


@pytest.mark.parametrize("n_s", [0, 1, 33])
def test_delta_curve_sample_counts(n_s):
    W, grad, S = inputs(102, 128, 256, n_s, "bf16")
    check(W, grad, S, "bf16", 32, 32, 0.0, [0, 5, 50, 95, 100], "samples")


def test_delta_curve_points():
    W, grad, S = inputs(103, 192, 128, 4, "bf16")
    # one point, repeated points, a point at 100%, an uneven grid
    check(W, grad, S, "bf16", 16, 16, 0.2, [100], "one point")
    check(W, grad, S, "bf16", 16, 16, 0.2, [30, 30, 31, 99], "repeats")
    got, _ = check(W, grad, S, "bf16", 16, 16, 0.2, [0, 0], "zeros")
    assert np.all(got == 0.0)


def test_delta_curve_ties_in_the_ranking():
    # equal scores everywhere: blocks are dropped from the highest index down
    W = np.ones((128, 128), np.float32)
    grad = np.ones((128, 128), np.float32)
    g = np.random.default_rng(104)
    S = g.integers(-2, 3, (3, 128, 128)).astype(np.float32)
    check(W, grad, S, "f32", 32, 32, 0.5, [0, 25, 50, 75, 100], "ties")


def test_delta_curve_headline_layer():
    # DeiT-B fc1's weight with 8 per-sample gradients at a few ratios
    w = wl.b_fc1(with_x=False)
    g = np.random.default_rng(105)
    grad = wl.quantize(g.normal(0, 1e-3, w.W.shape).astype(np.float32), "bf16")
    S = wl.quantize(g.normal(0, 1e-2, (8,) + w.W.shape).astype(np.float32), "bf16")
    check(w.W, grad, S, "bf16", 32, 32, 1e-4, [0, 30, 50, 70], "b_fc1")


def test_delta_curve_widest_rows():
    # K = 65536, the widest weight: the block dot kernel's chunk sums fill
    # 64 KB of LDS
    W, grad, S = inputs(106, 16, 65536, 2, "bf16")
    check(W, grad, S, "bf16", 16, 16, 0.01, [0, 50, 100], "K = 65536")


def test_delta_curve_many_blocks():
    # 32768 blocks of 16 x 16: the ranking kernel's key range split over its
    # 16 waves, 512 workgroups
    W, grad, S = inputs(107, 2048, 4096, 1, "bf16")
    check(W, grad, S, "bf16", 16, 16, 0.01, [0, 33, 67, 100], "32768 blocks")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_delta_curve_caller_workspace(dtype):
    # lpv_delta_curve_ws with a caller-owned workspace gives the curve of
    # lpv_delta_curve bit for bit, on two calls in a row (the second smaller,
    # the workspace holding the first call's contents)
    pcts = list(range(0, 101, 5))
    W, grad, S = inputs(108, 256, 256, 7, dtype)
    W2, grad2, S2 = inputs(109, 128, 192, 3, dtype)
    nbytes = lpv.delta_curve_workspace_size(256, 256, 32, 32, 7, len(pcts))
    assert nbytes >= lpv.delta_curve_workspace_size(128, 192, 16, 32, 3, len(pcts))
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    for (w_, g_, s_, b_r, b_c) in ((W, grad, S, 32, 32), (W2, grad2, S2, 16, 32)):
        say("delta_curve workspace", dtype, w_.shape, (b_r, b_c), "n=%d" % s_.shape[0])
        Wd, Gd = dev(w_, dtype), dev(g_, dtype)
        Sd = dev(s_.reshape(s_.shape[0], -1), dtype).reshape(s_.shape)
        a = lpv.delta_curve(Wd, Gd, Sd, b_r, b_c, 0.1, pcts)
        b = lpv.delta_curve(Wd, Gd, Sd, b_r, b_c, 0.1, pcts, workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(a, b)
        ref = oracle.delta_curve(w_, dtype, b_r, b_c, g_, s_, 0.1, pcts)
        assert np.abs(b.cpu().numpy() - ref).max() <= TOL * max(np.abs(ref).max(), 1e-300)
    with pytest.raises(lpv.LpvError):
        lpv.delta_curve(Wd, Gd, Sd, 16, 32, 0.1, pcts, workspace=ws[:64])


def test_delta_curve_many_points_and_samples():
    # 128 points x 72 vectors of step sums (74 KB): more than the finishing
    # kernel stages in LDS, so it runs on global memory
    W, grad, S = inputs(110, 64, 128, 70, "bf16")
    pcts = sorted(np.random.default_rng(111).integers(0, 101, 128).tolist())
    check(W, grad, S, "bf16", 16, 16, 0.02, pcts, "128 points")


def test_delta_curve_queued_calls_on_a_side_stream():
    # three calls queued back to back on a non-default stream (no
    # synchronisation in between, each with its own stream-ordered
    # workspace), each against the oracle
    pcts = [0, 20, 40, 60, 80, 100]
    cases = [inputs(112 + i, 128, 192, 3 + i, "bf16") for i in range(3)]
    st = torch.cuda.Stream()
    outs = []
    with torch.cuda.stream(st):
        for (W, grad, S), (b_r, b_c) in zip(cases, ((32, 32), (16, 16), (32, 64))):
            Sd = dev(S.reshape(S.shape[0], -1), "bf16").reshape(S.shape)
            outs.append(lpv.delta_curve(dev(W, "bf16"), dev(grad, "bf16"), Sd, b_r, b_c, 0.1, pcts,
                                        stream=st))
    st.synchronize()
    for (W, grad, S), (b_r, b_c), got in zip(cases, ((32, 32), (16, 16), (32, 64)), outs):
        ref = oracle.delta_curve(W, "bf16", b_r, b_c, grad, S, 0.1, pcts)
        err = np.abs(got.cpu().numpy() - ref).max() / max(np.abs(ref).max(), 1e-300)
        say("delta_curve queued", (b_r, b_c), "rel err %.2e" % err)
        assert err <= TOL
