"""Seeded input generators: determinism, rounding, mask counts (CPU)."""
import math

import numpy as np
import pytest
import torch

import workloads as wl


def test_bf16_rounding_matches_torch():
    g = np.random.default_rng(0)
    a = np.concatenate([
        g.standard_normal(100000).astype(np.float32) * np.float32(10.0) ** g.integers(-30, 30, 100000).astype(np.float32),
        np.array([0.0, -0.0, np.inf, -np.inf, 3.3895314e38, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8,
                  1e-40, -1e-45], np.float32)])
    got = wl.bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, ref)
    nan = wl.bf16_bits(np.array([np.nan], np.float32))
    assert np.isnan(wl.bf16_to_f32(nan)[0])


def test_bf16_ties_to_even():
    # 1 + 2^-8 lies halfway between 1 and 1 + 2^-7: ties go to the even one (1.0)
    assert wl.bf16_to_f32(wl.bf16_bits(np.array([1.0 + 2 ** -8], np.float32)))[0] == 1.0
    assert wl.bf16_to_f32(wl.bf16_bits(np.array([1.0 + 3 * 2 ** -8], np.float32)))[0] == 1.0 + 2 ** -6


@pytest.mark.parametrize("R,C,p", [(96, 24, 50), (48, 12, 50), (72, 24, 40), (24, 96, 70),
                                   (192, 48, 90), (3, 7, 33), (1, 1, 99), (5, 5, 0), (5, 5, 100)])
def test_n_keep_is_ceiling(R, C, p):
    # the paper's kept-block count: ceil((1 - alpha) * number of blocks)
    from fractions import Fraction
    assert wl.n_keep(R, C, p) == math.ceil(Fraction(100 - p, 100) * R * C)


def test_topk_mask_counts_and_ties():
    s = np.array([[3.0, 1.0, 3.0], [2.0, 3.0, 0.0]])
    m = wl.mask_topk(s, 2)
    assert m.tolist() == [[1, 0, 1], [0, 0, 0]]  # three 3.0s: the two lowest indices win
    m = wl.mask_topk(s, 4)
    assert m.tolist() == [[1, 0, 1], [1, 1, 0]]
    w = wl.b_fc1(with_x=False)
    assert w.nnzb == wl.n_keep(96, 24, 50) == 1152


def test_configs_shapes_and_counts():
    t = wl.tiny_fc1()
    assert t.X.shape == (197, 192) and t.W.shape == (768, 192) and t.X.dtype == np.float32
    assert t.mask.shape == (48, 12) and 200 < t.nnzb < 380
    s = wl.s_fc1_gelu(M=197)
    assert s.W.shape == (1536, 384) and s.nnzb == 288 and s.gelu and s.X.dtype == np.uint16
    sc = wl.block_scores(wl.to_f32(s.W, "bf16"), 32, 32)
    assert sc[s.mask == 1].min() >= sc[s.mask == 0].max()
    layer = wl.b_layer(M=197, with_x=False)
    assert [l.nnzb for l in layer] == [1037, 288, 922, 692]
    assert [l.N for l in layer] == [2304, 768, 3072, 768]


def test_zipf_counts():
    g = wl.rng(3, 0, wl.T_ZIPF)
    cnt = wl.zipf_counts(g, 24, 96, wl.n_keep(24, 96, 40))
    assert cnt.sum() == wl.n_keep(24, 96, 40) and cnt.max() <= 96
    assert cnt.max() >= 3 * cnt.min()  # skewed
    # heavy demand: the cap binds and the overflow goes elsewhere
    cnt = wl.zipf_counts(wl.rng(3, 1, wl.T_ZIPF), 8, 10, 70)
    assert cnt.sum() == 70 and cnt.max() == 10


def test_seeded_determinism():
    a = wl.custom(9, 37, 64, 96, 16, 32, "bf16", "zipf", 40)
    b = wl.custom(9, 37, 64, 96, 16, 32, "bf16", "zipf", 40)
    for x, y in ((a.X, b.X), (a.W, b.W), (a.mask, b.mask), (a.bias, b.bias)):
        assert np.array_equal(x, y)
    c = wl.custom(10, 37, 64, 96, 16, 32, "bf16", "zipf", 40)
    assert not np.array_equal(a.W, c.W)
