"""GPU pack (mask -> BSR) and tile schedule, against the oracle's pack
bit for bit, and the schedule against its definition."""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from gpu_util import bits, dev, host, say
from paper_2407_02068_amd import lpv

pytestmark = pytest.mark.gpu

SHAPES = ((16, 16), (16, 32), (32, 16), (32, 32), (64, 32), (32, 64), (64, 64), (16, 64), (64, 16))


def _case(seed, N, K, b_r, b_c, dtype, p_keep=0.5, nan_dropped=True):
    g = np.random.default_rng(seed)
    W = wl.quantize(g.normal(0, 1, (N, K)).astype(np.float32), dtype)
    mask = (g.random((N // b_r, K // b_c)) < p_keep).astype(np.uint8)
    if nan_dropped:
        exp = np.kron(mask, np.ones((b_r, b_c), np.uint8)) == 0
        W = W.copy()
        W[exp] = wl.quantize(np.array([np.nan], np.float32), dtype)[0]
    return W, mask


def _pack_and_compare(W, mask, dtype, b_r, b_c):
    N, K = W.shape
    h = lpv.bsr_pack(dev(W, dtype), dev(mask), b_r, b_c)
    rp, ci, vals = lpv.bsr_export(h)
    torch.cuda.synchronize()
    orp, oci, ovals = oracle.pack(W, dtype, b_r, b_c, mask)
    assert h.info["nnzb"] == int(mask.sum()) == len(oci)
    assert np.array_equal(rp.cpu().numpy(), orp)
    assert np.array_equal(ci.cpu().numpy(), oci)
    assert np.array_equal(bits(host(vals, dtype)), bits(ovals))
    Wu = lpv.bsr_unpack(h)
    torch.cuda.synchronize()
    assert np.array_equal(bits(host(Wu, dtype)), bits(oracle.unpack(orp, oci, ovals, dtype, N, K,
                                                                     b_r, b_c)))
    return h


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("b_r,b_c", SHAPES)
def test_pack_bit_exact(dtype, b_r, b_c):
    N, K = 192, 320 if b_c != 64 else 384
    say("pack", dtype, b_r, b_c, N, K)
    W, mask = _case(1000 + b_r + 7 * b_c, N, K, b_r, b_c, dtype)
    mask[0, :] = 0
    mask[-1, :] = 1
    h = _pack_and_compare(W, mask, dtype, b_r, b_c)
    if dtype != "f32":
        check_schedule(h, mask, b_r, b_c, N, K)


@pytest.mark.parametrize("kind", ["none", "all", "one", "ragged"])
def test_pack_edge_masks(kind):
    dtype, b_r, b_c = "bf16", 16, 16
    N, K = (48, 80) if kind == "ragged" else (128, 96)  # ragged: sides not multiples of 32
    W, mask = _case(77, N, K, b_r, b_c, dtype)
    if kind == "none":
        mask[:] = 0
    elif kind == "all":
        mask[:] = 1
    elif kind == "one":
        mask[:] = 0
        mask[-1, -1] = 1
    say("pack edge", kind, N, K, int(mask.sum()))
    h = _pack_and_compare(W, mask, dtype, b_r, b_c)
    check_schedule(h, mask, b_r, b_c, N, K)


@pytest.mark.parametrize("kind", ["zipf", "topk"])
def test_pack_deit_shapes(kind):
    if kind == "zipf":
        w = wl.b_stack(M=1, layers=1)[3]  # fc2: 768 x 3072, skewed rows
    else:
        w = wl.b_fc1(with_x=False)
    say("pack deit", w.name)
    h = _pack_and_compare(w.W, w.mask, w.dtype, w.b_r, w.b_c)
    check_schedule(h, w.mask, w.b_r, w.b_c, w.N, w.K)


def check_schedule(h, mask, b_r, b_c, N, K):
    """The exported schedule is the unique one its definition gives: for each
    group of tile rows, the tile columns holding a kept element (ascending),
    a bit per row, and the prefix sum of kept tiles; the launch order is a
    permutation sorted by cost (steps + kept tiles), ties by group index."""
    info = h.info
    T, G = info["tile_rows"], info["group_tiles"]
    assert T == info["tile_cols"] == 32
    NGR, NGC = math.ceil(N / T), math.ceil(K / T)
    ng = math.ceil(NGR / G)
    assert info["n_groups"] == ng
    em = np.zeros((NGR * T, NGC * T), bool)
    em[:N, :K] = np.kron(mask, np.ones((b_r, b_c), np.uint8)) != 0
    tile = em.reshape(NGR, T, NGC, T).any(axis=(1, 3))
    s = {k: v.cpu().numpy() for k, v in lpv.bsr_schedule_export(h).items()}
    torch.cuda.synchronize()
    steps_col, steps_bits, ptr, cost = [], [], [0], []
    for g in range(ng):
        rows = tile[g * G:(g + 1) * G]
        b = np.zeros(NGC, np.int64)
        for j in range(rows.shape[0]):
            b |= rows[j].astype(np.int64) << j
        cols = np.nonzero(b)[0]
        steps_col += cols.tolist()
        steps_bits += b[cols].tolist()
        ptr.append(ptr[-1] + len(cols))
        cost.append(len(cols) + int(sum(bin(int(x)).count("1") for x in b[cols])))
    assert info["n_steps"] == len(steps_col)
    assert np.array_equal(s["step_ptr"], ptr)
    assert np.array_equal(s["step_col"], steps_col)
    assert np.array_equal(s["step_bits"], steps_bits)
    pc = np.array([bin(int(x)).count("1") for x in steps_bits], np.int64)
    assert np.array_equal(s["step_tile"], np.concatenate([[0], np.cumsum(pc)[:-1]]) if len(pc) else [])
    assert info["n_tiles"] == int(pc.sum()) == int(tile.sum())
    order = s["group_order"]
    assert sorted(order.tolist()) == list(range(ng))
    want = sorted(range(ng), key=lambda g: (-cost[g], g))
    assert order.tolist() == want
