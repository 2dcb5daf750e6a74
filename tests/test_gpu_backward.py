"""GPU parity of the backward of the block-sparse layer against the float64
oracle: the transposed handle (bit for bit), dX through the forward kernel on
it, dW on the kept blocks and db."""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from gpu_util import TOL, assert_close, bits, dev, f64, host, say
from paper_2407_02068_amd import lpv

pytestmark = pytest.mark.gpu


def case(M, N, K, b_r, b_c, dtype, kind="uniform", sparsity=50, cfg=90):
    w = wl.custom(cfg, M, N, K, b_r, b_c, dtype, kind, sparsity)
    G = wl.grad_output(cfg, 0, M, N, dtype)
    return w, G


def check_all(w, G, what=""):
    dt = w.dtype
    say("backward", what, dt, "M=%d N=%d K=%d" % (w.M, w.N, w.K), (w.b_r, w.b_c),
        "nnzb=%d" % w.nnzb)
    h = lpv.bsr_pack(dev(w.W, dt), dev(w.mask), w.b_r, w.b_c)
    ht = lpv.bsr_transpose(h)
    Gd, Xd = dev(G, dt), dev(w.X, dt)
    dX = lpv.bsr_linear(ht, Gd)
    dW = lpv.grad_w(h, Gd, Xd)
    db = lpv.bias_grad(Gd)
    torch.cuda.synchronize()
    rx = oracle.grad_x(G, w.W, dt, w.b_r, w.b_c, w.mask)
    rw = oracle.grad_w(G, w.X, dt, w.b_r, w.b_c, w.mask)
    rb = oracle.grad_bias(G, dt)
    assert_close(f64(dX), rx, dt, "dX")
    if w.nnzb:
        assert_close(f64(dW), rw, dt, "dW (per block)", tile=(w.b_r, w.b_c))
    assert_close(f64(db), rb, dt, "db")
    h.close()
    ht.close()


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("b_r,b_c", [(32, 32), (16, 16), (64, 32), (16, 64)])
def test_transposed_handle_is_the_pack_of_the_transpose(dtype, b_r, b_c):
    w = wl.custom(91, 8, 384, 256, b_r, b_c, dtype, "bernoulli", 50)
    say("transpose", dtype, (b_r, b_c), "nnzb=%d" % w.nnzb)
    h = lpv.bsr_pack(dev(w.W, dtype), dev(w.mask), b_r, b_c)
    ht = lpv.bsr_transpose(h)
    row_ptr, col_idx, values = lpv.bsr_export(ht)
    torch.cuda.synchronize()
    # the oracle's pack of the pruned weight transposed, with the mask transposed
    rp, ci, vals = oracle.pack(w.W, dtype, b_r, b_c, w.mask)
    WT = np.ascontiguousarray(oracle.unpack(rp, ci, vals, dtype, w.N, w.K, b_r, b_c).T)
    ert, eci, evals = oracle.pack(WT, dtype, b_c, b_r, np.ascontiguousarray(w.mask.T))
    assert np.array_equal(row_ptr.cpu().numpy(), ert)
    assert np.array_equal(col_idx.cpu().numpy(), eci)
    assert np.array_equal(bits(host(values, dtype)), bits(evals))
    assert ht.info["N"] == w.K and ht.info["K"] == w.N and ht.info["nnzb"] == w.nnzb
    h.close()
    ht.close()


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("b_r,b_c", [(32, 32), (16, 16), (64, 32), (16, 64), (64, 64)])
def test_backward_matches_oracle(dtype, b_r, b_c):
    # several windows and token chunks, ragged token count
    w, G = case(1000, 512, 384, b_r, b_c, dtype)
    check_all(w, G, "blocks")


@pytest.mark.parametrize("M", [1, 31, 32, 33, 257])
def test_backward_ragged_tokens(M):
    w, G = case(M, 320, 288, 32, 32, "bf16", cfg=92)
    check_all(w, G, "ragged M")


@pytest.mark.parametrize("kind", ["all", "none", "bernoulli", "zipf"])
def test_backward_mask_kinds(kind):
    w, G = case(600, 256, 512, 32, 16, "bf16", kind, 60, cfg=93)
    check_all(w, G, kind)


def test_backward_fp32():
    w, G = case(197, 768, 192, 16, 16, "f32", "bernoulli", 50, cfg=94)
    check_all(w, G, "fp32 tiny")


def test_backward_m0():
    w, G = case(4, 256, 256, 32, 32, "bf16", cfg=95)
    h = lpv.bsr_pack(dev(w.W, "bf16"), dev(w.mask), 32, 32)
    G0 = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    X0 = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    say("backward M = 0")
    dW = lpv.grad_w(h, G0, X0, out=torch.full((w.nnzb, 32, 32), 7.0, dtype=torch.bfloat16,
                                               device="cuda"))
    db = lpv.bias_grad(G0, out=torch.full((256,), 7.0, dtype=torch.bfloat16, device="cuda"))
    torch.cuda.synchronize()
    assert not dW.float().abs().sum().item() and not db.float().abs().sum().item()
    h.close()


def test_backward_exact_on_small_integers():
    # integer G and X with short sums: every float32 partial sum is exact, so
    # dW and db equal the oracle bit for bit after the final rounding
    g = np.random.default_rng(96)
    w = wl.custom(96, 64, 256, 256, 32, 32, "bf16", "bernoulli", 50)
    w.X = wl.small_ints(g, (64, 256), dtype="bf16")
    G = wl.small_ints(g, (64, 256), dtype="bf16")
    h = lpv.bsr_pack(dev(w.W, "bf16"), dev(w.mask), 32, 32)
    say("backward small integers")
    dW = lpv.grad_w(h, dev(G, "bf16"), dev(w.X, "bf16"))
    db = lpv.bias_grad(dev(G, "bf16"))
    torch.cuda.synchronize()
    assert np.array_equal(f64(dW), oracle.grad_w(G, w.X, "bf16", 32, 32, w.mask))
    assert np.array_equal(f64(db), oracle.grad_bias(G, "bf16"))
    h.close()


def test_backward_headline_sampled():
    # DeiT-B fc1 at its full size: dW on sampled kept blocks, dX on sampled
    # token rows, db in full
    w = wl.b_fc1()
    G = wl.grad_output(4, 0, w.M, w.N, "bf16")
    say("backward headline", w.M, w.N, w.K)
    h = lpv.bsr_pack(dev(w.W, "bf16"), dev(w.mask), 32, 32)
    ht = lpv.bsr_transpose(h)
    Gd, Xd = dev(G, "bf16"), dev(w.X, "bf16")
    dX = lpv.bsr_linear(ht, Gd)
    dW = lpv.grad_w(h, Gd, Xd)
    db = lpv.bias_grad(Gd)
    torch.cuda.synchronize()
    g = np.random.default_rng(97)
    kept = np.argwhere(w.mask)  # BSR order = row-major over the mask
    pick = np.sort(g.choice(len(kept), 6, replace=False))
    sub = np.zeros_like(w.mask)
    for p in pick:
        sub[tuple(kept[p])] = 1
    rw = oracle.grad_w(G, w.X, "bf16", 32, 32, sub)
    assert_close(f64(dW[torch.as_tensor(pick, device="cuda")]), rw, "bf16", "dW sampled blocks",
                 tile=(32, 32))
    rows = np.sort(g.choice(w.M, 64, replace=False))
    rx = oracle.grad_x(np.ascontiguousarray(G[rows]), w.W, "bf16", 32, 32, w.mask)
    assert_close(f64(dX[torch.as_tensor(rows, device="cuda")]), rx, "bf16", "dX sampled rows")
    assert_close(f64(db), oracle.grad_bias(G, "bf16"), "bf16", "db")
    h.close()
    ht.close()


def test_grad_w_reuses_the_handle_workspace():
    # the handle's workspace is allocated by the first call and reused: three
    # calls in a row (large M, smaller ragged M, large M again) each match the
    # oracle, and the first and last agree bit for bit
    w, G = case(1100, 512, 384, 32, 32, "bf16", cfg=98)
    h = lpv.bsr_pack(dev(w.W, "bf16"), dev(w.mask), 32, 32)
    Gd, Xd = dev(G, "bf16"), dev(w.X, "bf16")
    say("grad_w workspace reuse M=1100, 333, 1100")
    d1 = lpv.grad_w(h, Gd, Xd)
    d2 = lpv.grad_w(h, Gd[:333].contiguous(), Xd[:333].contiguous())
    d3 = lpv.grad_w(h, Gd, Xd)
    torch.cuda.synchronize()
    assert_close(f64(d1), oracle.grad_w(G, w.X, "bf16", 32, 32, w.mask), "bf16", "dW 1",
                 tile=(32, 32))
    assert_close(f64(d2), oracle.grad_w(G[:333], w.X[:333], "bf16", 32, 32, w.mask), "bf16",
                 "dW 2", tile=(32, 32))
    assert torch.equal(d1.view(torch.int16), d3.view(torch.int16))
    h.close()
