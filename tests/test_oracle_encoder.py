"""The encoder-block oracle (oracle/encoder.py) against closed forms,
invariants and a brute-force loop (CPU)."""
import math

import numpy as np

from oracle import encoder as enc


def _qkv(rng, n, T, H, hd):
    return rng.normal(0, 1, (n * T, 3 * H * hd))


def test_attention_single_token_returns_v():
    # one key: its weight is 1, so the output is that token's v, head by head
    rng = np.random.default_rng(1)
    H, hd = 3, 4
    qkv = _qkv(rng, 5, 1, H, hd)
    out = enc.attention(qkv, 5, 1, H, hd)
    np.testing.assert_array_equal(out, qkv[:, 2 * H * hd:])


def test_attention_equal_keys_average_v():
    # equal scores: uniform weights, every query gets the mean of v
    rng = np.random.default_rng(2)
    T, H, hd = 7, 2, 4
    qkv = _qkv(rng, 1, T, H, hd)
    qkv[:, H * hd:2 * H * hd] = qkv[0, H * hd:2 * H * hd]
    out = enc.attention(qkv, 1, T, H, hd)
    mean_v = qkv[:, 2 * H * hd:].mean(axis=0)
    np.testing.assert_allclose(out, np.broadcast_to(mean_v, out.shape), rtol=0, atol=1e-14)


def test_attention_key_shift_invariance():
    # adding u to every key adds q.u to all scores of a query: no change;
    # a softmax over the wrong axis, or q and k swapped, breaks this
    rng = np.random.default_rng(3)
    T, H, hd = 6, 2, 8
    qkv = _qkv(rng, 2, T, H, hd)
    shifted = qkv.copy()
    shifted[:, H * hd:2 * H * hd] += rng.normal(0, 1, H * hd)
    np.testing.assert_allclose(enc.attention(shifted, 2, T, H, hd),
                               enc.attention(qkv, 2, T, H, hd), rtol=0, atol=1e-12)


def test_attention_two_keys_closed_form():
    # q = (a, 0, 0, 0) for both tokens, k0 = e0, k1 = 0, hd = 4: scores a / 2
    # and 0, so weight(k0) = 1 / (1 + exp(-a / 2)) for both queries
    a, hd = 3.0, 4
    v0, v1 = np.array([1.0, -2.0, 0.5, 4.0]), np.array([-3.0, 0.0, 2.0, 1.0])
    qkv = np.zeros((2, 3 * hd))
    qkv[:, 0] = a
    qkv[0, hd] = 1.0
    qkv[0, 2 * hd:], qkv[1, 2 * hd:] = v0, v1
    w0 = 1.0 / (1.0 + math.exp(-a / 2))
    want = w0 * v0 + (1 - w0) * v1
    out = enc.attention(qkv, 1, 2, 1, hd)
    np.testing.assert_allclose(out, np.stack([want, want]), rtol=0, atol=1e-15)


def test_attention_heads_are_separate():
    # head 0 gets equal keys (mean of its v); head 1 stays random
    rng = np.random.default_rng(4)
    T, H, hd = 5, 2, 3
    qkv = _qkv(rng, 1, T, H, hd)
    qkv[:, H * hd:H * hd + hd] = 0.7
    out = enc.attention(qkv, 1, T, H, hd)
    v = qkv[:, 2 * H * hd:]
    np.testing.assert_allclose(out[:, :hd], np.broadcast_to(v[:, :hd].mean(0), (T, hd)), atol=1e-14)
    assert np.abs(out[:, hd:] - v[:, hd:].mean(0)).max() > 1e-3


def test_attention_brute_force_loops():
    rng = np.random.default_rng(5)
    n, T, H, hd = 2, 3, 2, 2
    qkv = _qkv(rng, n, T, H, hd)
    out = enc.attention(qkv, n, T, H, hd)
    for s in range(n):
        for h in range(H):
            for t in range(T):
                row = qkv[s * T + t]
                q = row[h * hd:(h + 1) * hd]
                sc = []
                for u in range(T):
                    k = qkv[s * T + u][H * hd + h * hd:H * hd + (h + 1) * hd]
                    sc.append(sum(q[i] * k[i] for i in range(hd)) / math.sqrt(hd))
                m = max(sc)
                e = [math.exp(x - m) for x in sc]
                z = sum(e)
                for j in range(hd):
                    want = sum(e[u] / z * qkv[s * T + u][2 * H * hd + h * hd + j] for u in range(T))
                    assert abs(out[s * T + t, h * hd + j] - want) < 1e-13


def test_layernorm_two_columns_closed_form():
    # a row (a, b): mean (a + b) / 2, var ((a - b) / 2)^2
    x = np.array([[3.0, -1.0], [0.25, 0.75]])
    y = np.array([[1.0, 1.0], [0.0, 0.5]])
    g, b, eps = np.array([2.0, 0.5]), np.array([0.1, -0.2]), 1e-3
    s, out = enc.add_layernorm(x, y, g, b, eps)
    np.testing.assert_array_equal(s, x + y)
    for r in range(2):
        d = (s[r, 0] - s[r, 1]) / 2
        z = d / math.sqrt(d * d + eps)
        np.testing.assert_allclose(out[r], [z * g[0] + b[0], -z * g[1] + b[1]], rtol=0, atol=1e-15)


def test_layernorm_moments_and_affine_invariance():
    rng = np.random.default_rng(6)
    x = rng.normal(2.0, 3.0, (9, 64))
    one, zero = np.ones(64), np.zeros(64)
    _, out = enc.add_layernorm(x, None, one, zero, 0.0)
    np.testing.assert_allclose(out.mean(1), 0, atol=1e-14)
    np.testing.assert_allclose((out ** 2).mean(1), 1, atol=1e-13)
    _, out2 = enc.add_layernorm(5.0 * x - 7.0, None, one, zero, 0.0)
    np.testing.assert_allclose(out2, out, atol=1e-12)
    # with eps the mean square is var / (var + eps)
    eps = 0.5
    _, out3 = enc.add_layernorm(x, np.zeros_like(x), one, zero, eps)
    var = x.var(1)
    np.testing.assert_allclose((out3 ** 2).mean(1), var / (var + eps), rtol=1e-13)


# Plausible mistakes in the oracle; each must fail at least one pin above.
MUTANTS = [
    ("np.sqrt(hd)", "hd"),
    ("s.max(axis=1, keepdims=True)", "s.max(axis=0, keepdims=True)"),
    ("p /= p.sum(axis=1, keepdims=True)", "p /= p.sum(axis=0, keepdims=True)"),
    ("x[n, :, 0, h], x[n, :, 1, h]", "x[n, :, 1, h], x[n, :, 0, h]"),
    ("np.sqrt(var + eps)", "np.sqrt(var) + eps"),
    ("((s - mean) ** 2).mean(axis=1, keepdims=True)",
     "((s - mean) ** 2).sum(axis=1, keepdims=True) / (s.shape[1] - 1)"),
    ("* np.asarray(gamma, np.float64) + np.asarray(beta, np.float64)",
     "* np.asarray(gamma, np.float64)"),
    ("(s - mean) / np.sqrt", "(x - mean) / np.sqrt"),
]
PINS = [f for n, f in sorted(globals().items()) if n.startswith("test_") and callable(f)]


def test_pins_catch_oracle_mutants(monkeypatch):
    import types
    src = open(enc.__file__).read()
    for old, new in MUTANTS:
        assert src.count(old) == 1, old
        mod = types.ModuleType("encoder_mutant")
        exec(compile(src.replace(old, new), "encoder_mutant", "exec"), mod.__dict__)
        monkeypatch.setitem(globals(), "enc", mod)
        failed = 0
        for pin in PINS:
            try:
                pin()
            except AssertionError:
                failed += 1
        assert failed, "mutant not caught: %s -> %s" % (old, new)
    monkeypatch.setitem(globals(), "enc", enc)
