"""float64 CPU oracle for the rest of a ViT encoder block around the pruned
linear layers: the pre-norm residual step and multi-head self-attention.

TEST INFRASTRUCTURE ONLY, like the rest of this package: only ``tests/``,
``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline leg may use it.

The paper prunes the linear layers of DeiT and Swin encoders (Sec. 4) and
measures whole models (Tab. 2); the block between those layers is the standard
pre-norm ViT encoder block, which the paper takes as given:
    s   = x + y                                     (residual; y may be absent)
    out = (s - mean(s)) / sqrt(var(s) + eps) * gamma + beta   (per row; var biased)
    attention, per sequence and head:  softmax(Q K^T / sqrt(hd)) V,
where one row of the qkv projection's output holds q, k and v in that order,
each as H heads of hd contiguous elements.  Both are written here as their
definitions in float64 numpy, with no reordering beyond numpy's own sums.
"""
import numpy as np


def add_layernorm(x, y, gamma, beta, eps):
    """Residual sum and layer normalisation of each row (float64 arrays).
    Returns (s, out)."""
    x = np.asarray(x, dtype=np.float64)
    s = x if y is None else x + np.asarray(y, dtype=np.float64)
    mean = s.mean(axis=1, keepdims=True)
    var = ((s - mean) ** 2).mean(axis=1, keepdims=True)
    out = (s - mean) / np.sqrt(var + eps) * np.asarray(gamma, np.float64) + np.asarray(beta, np.float64)
    return s, out


def attention(qkv, n_seq, T, H, hd):
    """Multi-head self-attention over n_seq sequences of T tokens.  qkv is
    (n_seq T) x (3 H hd), row t = [q heads | k heads | v heads]; returns the
    (n_seq T) x (H hd) output, head h in columns h hd .. h hd + hd - 1."""
    x = np.asarray(qkv, dtype=np.float64).reshape(n_seq, T, 3, H, hd)
    out = np.empty((n_seq, T, H, hd))
    for n in range(n_seq):
        for h in range(H):
            q, k, v = x[n, :, 0, h], x[n, :, 1, h], x[n, :, 2, h]  # T x hd each
            s = (q @ k.T) / np.sqrt(hd)                             # queries x keys
            p = np.exp(s - s.max(axis=1, keepdims=True))
            p /= p.sum(axis=1, keepdims=True)
            out[n, :, h] = p @ v
    return out.reshape(n_seq * T, H * hd)
