"""GPU parity of the encoder-block kernels around the pruned layers (residual +
layer norm, multi-head attention) against the float64 oracle."""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from gpu_util import TOL, assert_close, dev, f64, host, say
from oracle import encoder as enc
from paper_2407_02068_amd import lpv
from paper_2407_02068_amd.encoder import deit_chain

pytestmark = pytest.mark.gpu

T_QKV, T_LNX, T_LNY, T_LNG = 40, 41, 42, 43


def rel(y, ref):
    return oracle.rel_err(y, ref)


def gen(cfg, tid, shape, dtype, std=1.0, mean=0.0):
    a = wl.quantize(wl.rng(cfg, 0, tid).normal(mean, std, shape).astype(np.float32), dtype)
    return a, oracle.decode(a, dtype).reshape(shape)


def run_attention(n_seq, T, H, dtype, q_scale=1.0, cfg=95):
    say("attention", dtype, "n_seq=%d T=%d H=%d q_scale=%g" % (n_seq, T, H, q_scale))
    a, ref_in = gen(cfg, T_QKV, (n_seq * T, 3 * H * 64), dtype)
    if q_scale != 1.0:  # sharper scores: scale the q third
        a = a.copy()
        a[:, :H * 64] = wl.quantize(ref_in[:, :H * 64].astype(np.float32) * q_scale, dtype)
        ref_in = oracle.decode(a, dtype).reshape(a.shape)
    out = lpv.attention(dev(a, dtype), n_seq, T, H)
    torch.cuda.synchronize()
    return f64(out), ref_in


@pytest.mark.parametrize("n_seq,T,H,dtype", [
    (2, 197, 12, "bf16"), (1, 1, 1, "bf16"), (3, 31, 2, "bf16"), (2, 32, 3, "f16"),
    (2, 33, 1, "bf16"), (1, 100, 4, "f16"), (1, 512, 2, "bf16"), (4, 64, 64, "bf16")])
def test_attention_matches_oracle(n_seq, T, H, dtype):
    y, x = run_attention(n_seq, T, H, dtype)
    ref = enc.attention(x, n_seq, T, H, 64)
    e = rel(y, ref)
    say("  rel err %.3g" % e)
    assert e <= TOL[dtype]


def test_attention_sharp_scores():
    # scores with a spread of ~8: the running maximum and rescaling matter
    y, x = run_attention(2, 197, 3, "bf16", q_scale=8.0)
    e = rel(y, enc.attention(x, 2, 197, 3, 64))
    say("  rel err %.3g" % e)
    assert e <= TOL["bf16"]


def test_attention_empty_batch():
    out = lpv.attention(torch.empty((0, 3 * 64), dtype=torch.bfloat16, device="cuda"), 0, 7, 1)
    torch.cuda.synchronize()
    assert out.shape == (0, 64)


def test_attention_deit_b_batch_sampled():
    # the DeiT-B shape at batch 256 (197 tokens, 12 heads), checked on 4 sequences
    n_seq, T, H = 256, 197, 12
    say("attention full size", n_seq, T, H)
    a, x = gen(96, T_QKV, (n_seq * T, 3 * H * 64), "bf16")
    out = lpv.attention(dev(a, "bf16"), n_seq, T, H)
    torch.cuda.synchronize()
    y = f64(out)
    for s in (0, 1, 137, 255):
        rows = slice(s * T, (s + 1) * T)
        e = rel(y[rows], enc.attention(x[rows], 1, T, H, 64))
        assert e <= TOL["bf16"], (s, e)


@pytest.mark.parametrize("M,D,dtype,with_y", [
    (300, 768, "bf16", True), (5, 4, "bf16", True), (3, 2048, "bf16", False),
    (64, 260, "f16", False), (17, 1024, "f16", True), (0, 768, "bf16", True)])
def test_add_layernorm_matches_oracle(M, D, dtype, with_y):
    say("add_layernorm", dtype, "M=%d D=%d y=%s" % (M, D, with_y))
    xa, x = gen(97, T_LNX, (M, D), dtype, std=2.0, mean=0.5)
    ya, y = gen(97, T_LNY, (M, D), dtype)
    ga, g = gen(97, T_LNG, (D,), dtype, std=0.2, mean=1.0)
    ba, b = gen(98, T_LNG, (D,), dtype, std=0.1)
    xd = dev(xa, dtype)
    yd = dev(ya, dtype) if with_y else None
    S = torch.empty_like(xd)
    out = lpv.add_layernorm(xd, yd, dev(ga, dtype), dev(ba, dtype), 1e-6, S=S)
    torch.cuda.synchronize()
    s_ref, o_ref = enc.add_layernorm(x, y if with_y else None, g, b, 1e-6)
    if M:
        assert rel(f64(S), s_ref) <= TOL[dtype]
        e = rel(f64(out), o_ref)
        say("  rel err %.3g" % e)
        assert e <= TOL[dtype]


def test_add_layernorm_in_place_residual():
    # S aliasing x: the residual stream updated in place
    M, D = 40, 768
    xa, x = gen(99, T_LNX, (M, D), "bf16")
    ya, y = gen(99, T_LNY, (M, D), "bf16")
    ones = torch.ones(D, dtype=torch.bfloat16, device="cuda")
    zeros = torch.zeros(D, dtype=torch.bfloat16, device="cuda")
    xd = dev(xa, "bf16")
    out = lpv.add_layernorm(xd, dev(ya, "bf16"), ones, zeros, 1e-6, S=xd)
    torch.cuda.synchronize()
    s_ref, o_ref = enc.add_layernorm(x, y, np.ones(D), np.zeros(D), 1e-6)
    assert rel(f64(xd), s_ref) <= TOL["bf16"]
    assert rel(f64(out), o_ref) <= TOL["bf16"]


def test_add_layernorm_deit_b_batch_sampled():
    M, D = 256 * 197, 768
    say("add_layernorm full size", M, D)
    xa, x = gen(100, T_LNX, (M, D), "bf16")
    ya, y = gen(100, T_LNY, (M, D), "bf16")
    ga, g = gen(100, T_LNG, (D,), "bf16", std=0.2, mean=1.0)
    ba, b = gen(101, T_LNG, (D,), "bf16", std=0.1)
    out = lpv.add_layernorm(dev(xa, "bf16"), dev(ya, "bf16"), dev(ga, "bf16"), dev(ba, "bf16"), 1e-6)
    torch.cuda.synchronize()
    rows = np.array([0, 1, 12345, M // 2, M - 1])
    _, o_ref = enc.add_layernorm(x[rows], y[rows], g, b, 1e-6)
    assert rel(f64(out)[rows], o_ref) <= TOL["bf16"]


# ---- the chained encoder (the composition bench.py times) -----------------------

def _check_chain(n_seq, blocks, seqs):
    """Run the DeiT-B encoder chain (block-sparse linears with the stack's
    Zipf masks and per-linear sparsity) and check every link on the token rows
    of sequences ``seqs`` against the oracle fed the GPU's own input of that
    link: the linear layers with oracle.linear, attention and residual + layer
    norm with the encoder oracle."""
    T, H, D = 197, 12, 768
    layers = wl.b_stack(M=n_seq * T, layers=blocks)
    chain = deit_chain(layers, lambda a: dev(a, "bf16"), n_seq, T, H)
    by_name = {w.name: w for w in layers}
    rows = np.concatenate([np.arange(s * T, (s + 1) * T) for s in seqs])
    rd = torch.from_numpy(rows).cuda()
    ones, zeros = np.ones(D), np.zeros(D)
    seen = []

    def dec(t):  # the GPU tensor's sampled rows, decoded exactly to float64
        return oracle.decode(host(t[rd].contiguous(), "bf16"), "bf16").reshape(len(rows), -1)

    def trace(name, ins, out):
        torch.cuda.synchronize()
        seen.append(name)
        if name in by_name:
            w = by_name[name]
            xin = host(ins["x"][rd].contiguous(), "bf16")
            r = oracle.linear(xin, w.W, "bf16", 32, 32, w.mask, w.bias, gelu=w.gelu)
            assert_close(f64(out[rd]), r, "bf16", name)
        elif name.endswith("attention"):
            r = enc.attention(dec(ins["qkv"]), len(seqs), T, H, 64)
            assert_close(f64(out[rd]), r, "bf16", name)
        else:
            y = dec(ins["y"]) if "y" in ins else None
            s_ref, o_ref = enc.add_layernorm(dec(ins["x"]), y, ones, zeros, 1e-6)
            if "s" in ins:
                assert_close(f64(ins["s"][rd]), s_ref, "bf16", name + " residual")
            assert_close(f64(out[rd]), o_ref, "bf16", name)

    say("encoder chain", n_seq, "sequences,", blocks, "blocks, checked on", list(seqs))
    x0 = dev(layers[0].X, "bf16")
    x, A = chain.run(x0, sparse=True, trace=trace)
    torch.cuda.synchronize()
    assert len(seen) == 1 + 7 * blocks
    assert torch.isfinite(A.float()).all()
    # the dense-linear chain computes the same function of the same weights
    # with every block of the masks kept: here only its finiteness and shape
    x2, A2 = chain.run(x0, sparse=False)
    torch.cuda.synchronize()
    assert torch.isfinite(A2.float()).all() and A2.shape == A.shape
    chain.close()


def test_encoder_chain_batch4_in_full():
    _check_chain(4, 2, range(4))


def test_encoder_chain_batch256_sampled():
    _check_chain(256, 1, (0, 77, 255))


@pytest.mark.parametrize("sparse", [True, False])
def test_encoder_chain_graph_replays(sparse):
    """The chain captured into a HIP graph: three replays, each after eager work
    that overwrites the outputs (and a synchronisation), give the eager pass's
    result bit for bit."""
    T, H = 197, 12
    layers = wl.b_stack(M=4 * T, layers=2)
    chain = deit_chain(layers, lambda a: dev(a, "bf16"), 4, T, H)
    x0 = dev(layers[0].X, "bf16")
    say("encoder graph", "block-sparse" if sparse else "dense", "4 sequences, 2 blocks")
    x, A = chain.run(x0, sparse=sparse)
    torch.cuda.synchronize()
    x_ref, A_ref = x.clone(), A.clone()
    graph, (xg, Ag) = chain.capture(x0, sparse=sparse)
    assert xg.data_ptr() == x.data_ptr() and Ag.data_ptr() == A.data_ptr()
    for i in range(3):
        # eager work between replays: the other path's forward, then the outputs cleared
        chain.run(x0, sparse=not sparse)
        xg.zero_()
        Ag.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(xg.view(torch.int16), x_ref.view(torch.int16)), "replay %d: x" % i
        assert torch.equal(Ag.view(torch.int16), A_ref.view(torch.int16)), "replay %d: A" % i
    chain.close()
