"""float64 CPU oracle for the block-sparse linear layer (LPViT, arXiv 2407.02068).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  It shares no code
with the GPU library (``paper_2407_02068_amd``) and imports nothing from it.

It is a thin ctypes binding over ``liblpv_oracle.so`` (``lpv_oracle.c``), which
computes the paper's masked weight (Sec. 3.1) and the linear layer
``Y = g(X W~^T + b)`` in float64; see that file's header for the definitions.

Element types are given by name: ``"f32"`` (numpy float32 arrays), ``"f16"``
(numpy float16) and ``"bf16"`` (numpy uint16 arrays holding the bf16 bit
patterns).
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liblpv_oracle.so")
_CODES = {"f32": 0, "f16": 1, "bf16": 2}
_NP = {"f32": np.float32, "f16": np.float16, "bf16": np.uint16}


class Oracle:
    """Binding to one build of the oracle library (the default build, or a
    copy the tests compiled elsewhere)."""

    def __init__(self, path=_LIB_PATH):
        if path == _LIB_PATH and not os.path.exists(path):
            from . import build as _build  # plain C: build it on demand
            _build.build()
        lib = ctypes.CDLL(path)
        i64, i32, vp = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p
        lib.lpvo_elem_size.argtypes = [i32]
        lib.lpvo_elem_size.restype = i32
        lib.lpvo_decode.argtypes = [i32, vp, i64, vp]
        lib.lpvo_decode.restype = i32
        lib.lpvo_pack.argtypes = [i32, vp, i64, i64, i64, i32, i32, vp, vp, vp, vp]
        lib.lpvo_pack.restype = i64
        lib.lpvo_unpack.argtypes = [i32, i64, i64, i32, i32, vp, vp, vp, vp, i64]
        lib.lpvo_unpack.restype = i32
        lib.lpvo_gelu.argtypes = [ctypes.c_double]
        lib.lpvo_gelu.restype = ctypes.c_double
        lib.lpvo_linear.argtypes = [i32, vp, i64, i64, vp, i64, i64, i64, i32, i32, vp, vp,
                                    i32, vp, i64, i32]
        lib.lpvo_linear.restype = i32
        lib.lpvo_block_scores.argtypes = [i32, vp, i64, vp, i64, i64, i64, i32, i32, vp]
        lib.lpvo_block_scores.restype = i32
        lib.lpvo_keep_count.argtypes = [i64, i32]
        lib.lpvo_keep_count.restype = i64
        lib.lpvo_mask_topk.argtypes = [vp, i64, i64, vp]
        lib.lpvo_mask_topk.restype = i32
        lib.lpvo_grad_x.argtypes = [i32, vp, i64, i64, vp, i64, i64, i64, i32, i32, vp, vp,
                                    i64, i32]
        lib.lpvo_grad_x.restype = i32
        lib.lpvo_grad_w.argtypes = [i32, vp, i64, vp, i64, i64, i64, i64, i32, i32, vp, vp]
        lib.lpvo_grad_w.restype = i64
        lib.lpvo_grad_bias.argtypes = [i32, vp, i64, i64, i64, vp]
        lib.lpvo_grad_bias.restype = i32
        lib.lpvo_delta_curve.argtypes = [i32, vp, i64, i64, i64, i32, i32, vp, vp, i64,
                                         ctypes.c_double, vp, i32, vp]
        lib.lpvo_delta_curve.restype = i32
        self.lib = lib
        self.path = path

    def decode(self, arr, dtype):
        """Exact float64 value of every element of ``arr`` (same shape)."""
        arr = np.ascontiguousarray(arr)
        _check(arr, dtype, "arr")
        out = np.empty(arr.shape, np.float64)
        if self.lib.lpvo_decode(_CODES[dtype], _ptr(arr), arr.size, _ptr(out)):
            raise ValueError("lpvo_decode failed")
        return out

    def gelu(self, v):
        """Exact-erf GELU in float64 (scalar)."""
        return self.lib.lpvo_gelu(float(v))

    def pack(self, W, dtype, b_r, b_c, mask):
        """Plain BSR pack: ``(row_ptr int32[R+1], col_idx int32[nnzb],
        values[nnzb, b_r, b_c])``; ``values`` has W's numpy type and holds the
        raw element bits of each kept block, row-major."""
        W = np.ascontiguousarray(W)
        _check(W, dtype, "W")
        mask = np.ascontiguousarray(mask, dtype=np.uint8)
        N, K = W.shape
        if b_r <= 0 or b_c <= 0 or N % b_r or K % b_c:
            raise ValueError("block %dx%d does not divide weight %dx%d" % (b_r, b_c, N, K))
        R, C = N // b_r, K // b_c
        if mask.shape != (R, C):
            raise ValueError("mask shape %s, expected %s" % (mask.shape, (R, C)))
        code = _CODES[dtype]
        nnzb = self.lib.lpvo_pack(code, _ptr(W), K, N, K, b_r, b_c, _ptr(mask), None, None, None)
        if nnzb < 0:
            raise ValueError("lpvo_pack rejected its arguments")
        row_ptr = np.zeros(R + 1, np.int32)
        col_idx = np.zeros(nnzb, np.int32)
        values = np.zeros((nnzb, b_r, b_c), W.dtype)
        got = self.lib.lpvo_pack(code, _ptr(W), K, N, K, b_r, b_c, _ptr(mask), _ptr(row_ptr),
                                 _ptr(col_idx), _ptr(values))
        if got != nnzb:
            raise RuntimeError("lpvo_pack returned %d then %d blocks" % (nnzb, got))
        return row_ptr, col_idx, values

    def unpack(self, row_ptr, col_idx, values, dtype, N, K, b_r, b_c):
        """Inverse of :meth:`pack`: the pruned dense weight (N x K), +0.0 in
        dropped blocks."""
        row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int32)
        col_idx = np.ascontiguousarray(col_idx, dtype=np.int32)
        values = np.ascontiguousarray(values)
        _check(values, dtype, "values")
        out = np.empty((N, K), _NP[dtype])
        if self.lib.lpvo_unpack(_CODES[dtype], N, K, b_r, b_c, _ptr(row_ptr), _ptr(col_idx),
                                _ptr(values), _ptr(out), K):
            raise ValueError("lpvo_unpack rejected its arguments")
        return out

    def linear(self, X, W, dtype, b_r, b_c, mask, bias=None, gelu=False, nthreads=None):
        """``Y = g(X W~^T + b)`` in float64 (M x N), not rounded."""
        X = np.ascontiguousarray(X)
        W = np.ascontiguousarray(W)
        _check(X, dtype, "X")
        _check(W, dtype, "W")
        mask = np.ascontiguousarray(mask, dtype=np.uint8)
        M, K = X.shape
        N, K2 = W.shape
        if K2 != K:
            raise ValueError("X is %dx%d but W is %dx%d" % (M, K, N, K2))
        if b_r <= 0 or b_c <= 0 or N % b_r or K % b_c:
            raise ValueError("block %dx%d does not divide weight %dx%d" % (b_r, b_c, N, K))
        if mask.shape != (N // b_r, K // b_c):
            raise ValueError("mask shape %s, expected %s" % (mask.shape, (N // b_r, K // b_c)))
        if bias is not None:
            bias = np.ascontiguousarray(bias)
            _check(bias, dtype, "bias")
            if bias.shape != (N,):
                raise ValueError("bias shape %s, expected (%d,)" % (bias.shape, N))
        Y = np.empty((M, N), np.float64)
        nt = default_threads() if nthreads is None else int(nthreads)
        rc = self.lib.lpvo_linear(_CODES[dtype], _ptr(X), K, M, _ptr(W), K, N, K, b_r, b_c,
                                  _ptr(mask), _ptr(bias), 1 if gelu else 0, _ptr(Y), N, nt)
        if rc:
            raise RuntimeError("lpvo_linear failed (%d)" % rc)
        return Y


    def _grid(self, N, K, b_r, b_c, mask):
        if b_r <= 0 or b_c <= 0 or N % b_r or K % b_c:
            raise ValueError("block %dx%d does not divide weight %dx%d" % (b_r, b_c, N, K))
        mask = np.ascontiguousarray(mask, dtype=np.uint8)
        if mask.shape != (N // b_r, K // b_c):
            raise ValueError("mask shape %s, expected %s" % (mask.shape, (N // b_r, K // b_c)))
        return mask

    def grad_x(self, G, W, dtype, b_r, b_c, mask, nthreads=None):
        """``dX = G W~`` in float64 (M x K): the input gradient for the
        pre-activation gradient ``G`` (M x N)."""
        G = np.ascontiguousarray(G)
        W = np.ascontiguousarray(W)
        _check(G, dtype, "G")
        _check(W, dtype, "W")
        M, N = G.shape
        N2, K = W.shape
        if N2 != N:
            raise ValueError("G is %dx%d but W is %dx%d" % (M, N, N2, K))
        mask = self._grid(N, K, b_r, b_c, mask)
        dX = np.empty((M, K), np.float64)
        nt = default_threads() if nthreads is None else int(nthreads)
        rc = self.lib.lpvo_grad_x(_CODES[dtype], _ptr(G), N, M, _ptr(W), K, N, K, b_r, b_c,
                                  _ptr(mask), _ptr(dX), K, nt)
        if rc:
            raise RuntimeError("lpvo_grad_x failed (%d)" % rc)
        return dX

    def grad_w(self, G, X, dtype, b_r, b_c, mask):
        """``G^T X`` on the kept blocks only, float64 ``[nnzb, b_r, b_c]`` in BSR
        order (the order of :meth:`pack`'s values)."""
        G = np.ascontiguousarray(G)
        X = np.ascontiguousarray(X)
        _check(G, dtype, "G")
        _check(X, dtype, "X")
        M, N = G.shape
        M2, K = X.shape
        if M2 != M:
            raise ValueError("G is %dx%d but X is %dx%d" % (M, N, M2, K))
        mask = self._grid(N, K, b_r, b_c, mask)
        nnzb = int(mask.astype(bool).sum())
        out = np.empty((nnzb, b_r, b_c), np.float64)
        got = self.lib.lpvo_grad_w(_CODES[dtype], _ptr(G), N, _ptr(X), K, M, N, K, b_r, b_c,
                                   _ptr(mask), _ptr(out))
        if got != nnzb:
            raise RuntimeError("lpvo_grad_w returned %d, expected %d blocks" % (got, nnzb))
        return out

    def grad_bias(self, G, dtype):
        """``db[n] = sum_m G[m][n]`` in float64."""
        G = np.ascontiguousarray(G)
        _check(G, dtype, "G")
        M, N = G.shape
        db = np.empty(N, np.float64)
        if self.lib.lpvo_grad_bias(_CODES[dtype], _ptr(G), N, M, N, _ptr(db)):
            raise ValueError("lpvo_grad_bias rejected its arguments")
        return db

    def delta_curve(self, W, dtype, b_r, b_c, grad, samples, kappa, pcts):
        """The delta curve: float64 delta at each sparsity percentage in
        ``pcts`` (grad: N x K, samples: n x N x K per-sample gradients)."""
        W = np.ascontiguousarray(W)
        grad = np.ascontiguousarray(grad)
        samples = np.ascontiguousarray(samples)
        for a, nm in ((W, "W"), (grad, "grad"), (samples, "samples")):
            _check(a, dtype, nm)
        N, K = W.shape
        if grad.shape != (N, K) or samples.ndim != 3 or samples.shape[1:] != (N, K):
            raise ValueError("grad must be N x K and samples n x N x K")
        if b_r <= 0 or b_c <= 0 or N % b_r or K % b_c:
            raise ValueError("block %dx%d does not divide weight %dx%d" % (b_r, b_c, N, K))
        pcts = np.ascontiguousarray(pcts, dtype=np.int32)
        out = np.empty(len(pcts), np.float64)
        rc = self.lib.lpvo_delta_curve(_CODES[dtype], _ptr(W), K, N, K, b_r, b_c, _ptr(grad),
                                       _ptr(samples), samples.shape[0], float(kappa), _ptr(pcts),
                                       len(pcts), _ptr(out))
        if rc:
            raise ValueError("lpvo_delta_curve failed (%d)" % rc)
        return out

    def block_scores(self, W, dtype, b_r, b_c, G=None):
        """Block scores, float64 R x C: the mean of |W * G| per block (the
        paper's average-pooled Taylor score, Sec. 3.1), or without G the sum of
        squares per block."""
        W = np.ascontiguousarray(W)
        _check(W, dtype, "W")
        N, K = W.shape
        if G is not None:
            G = np.ascontiguousarray(G)
            _check(G, dtype, "G")
            if G.shape != W.shape:
                raise ValueError("G shape %s, expected %s" % (G.shape, W.shape))
        if b_r <= 0 or b_c <= 0 or N % b_r or K % b_c:
            raise ValueError("block %dx%d does not divide weight %dx%d" % (b_r, b_c, N, K))
        out = np.empty((N // b_r, K // b_c), np.float64)
        if self.lib.lpvo_block_scores(_CODES[dtype], _ptr(W), K, _ptr(G), K, N, K, b_r, b_c,
                                      _ptr(out)):
            raise ValueError("lpvo_block_scores rejected its arguments")
        return out

    def keep_count(self, n_blocks, sparsity_pct):
        """Kept blocks at an integer sparsity percentage (ceiling rule, Sec. 3.4)."""
        n = self.lib.lpvo_keep_count(int(n_blocks), int(sparsity_pct))
        if n < 0:
            raise ValueError("bad block count or sparsity")
        return int(n)

    def mask_topk(self, scores, n_keep):
        """uint8 mask (scores' shape) of the n_keep best-ranked blocks: higher
        score first, equal scores by lower row-major index."""
        scores = np.ascontiguousarray(scores, dtype=np.float64)
        mask = np.empty(scores.shape, np.uint8)
        rc = self.lib.lpvo_mask_topk(_ptr(scores), scores.size, int(n_keep), _ptr(mask))
        if rc:
            raise ValueError("lpvo_mask_topk failed (%d)" % rc)
        return mask

    def block_mask(self, W, dtype, b_r, b_c, sparsity_pct, G=None):
        """The pruning mask of Sec. 3.1: scores, then the top ceil((1 - alpha)
        R C) blocks."""
        s = self.block_scores(W, dtype, b_r, b_c, G)
        return self.mask_topk(s, self.keep_count(s.size, sparsity_pct)), s


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(arr, dtype, name):
    if dtype not in _CODES:
        raise ValueError("unknown element type %r" % (dtype,))
    if arr.dtype != _NP[dtype]:
        raise TypeError("%s: expected numpy %s for %s, got %s"
                        % (name, np.dtype(_NP[dtype]).name, dtype, arr.dtype))
    if not arr.flags.c_contiguous:
        raise ValueError("%s must be C-contiguous" % name)


def default_threads():
    """Host threads this process may run on."""
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


_default = None


def default():
    """The oracle built from ``lpv_oracle.c`` next to this file."""
    global _default
    if _default is None:
        _default = Oracle()
    return _default


def decode(arr, dtype):
    return default().decode(arr, dtype)


def gelu(v):
    return default().gelu(v)


def pack(W, dtype, b_r, b_c, mask):
    return default().pack(W, dtype, b_r, b_c, mask)


def unpack(row_ptr, col_idx, values, dtype, N, K, b_r, b_c):
    return default().unpack(row_ptr, col_idx, values, dtype, N, K, b_r, b_c)


def linear(X, W, dtype, b_r, b_c, mask, bias=None, gelu=False, nthreads=None):
    return default().linear(X, W, dtype, b_r, b_c, mask, bias, gelu, nthreads)


def grad_x(G, W, dtype, b_r, b_c, mask, nthreads=None):
    return default().grad_x(G, W, dtype, b_r, b_c, mask, nthreads)


def grad_w(G, X, dtype, b_r, b_c, mask):
    return default().grad_w(G, X, dtype, b_r, b_c, mask)


def grad_bias(G, dtype):
    return default().grad_bias(G, dtype)


def delta_curve(W, dtype, b_r, b_c, grad, samples, kappa, pcts):
    return default().delta_curve(W, dtype, b_r, b_c, grad, samples, kappa, pcts)


def block_scores(W, dtype, b_r, b_c, G=None):
    return default().block_scores(W, dtype, b_r, b_c, G)


def keep_count(n_blocks, sparsity_pct):
    return default().keep_count(n_blocks, sparsity_pct)


def mask_topk(scores, n_keep):
    return default().mask_topk(scores, n_keep)


def block_mask(W, dtype, b_r, b_c, sparsity_pct, G=None):
    return default().block_mask(W, dtype, b_r, b_c, sparsity_pct, G)


def rel_err(y, ref):
    """Infinity-norm relative error ``max|y - r| / max|r|`` (float64), the
    reading of "max relative error" used for every value check.  The scale is
    the reference's largest magnitude, never the result's.  When the reference
    is all zero (or empty), 0.0 if ``y`` is exactly zero there too, else inf.
    A non-finite ``y`` anywhere, or a shape mismatch, gives inf: the check
    ``rel_err(y, r) <= tol`` then fails."""
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    if y.shape != ref.shape or not np.all(np.isfinite(y)):
        return float("inf")
    if ref.size == 0:
        return 0.0
    scale = float(np.max(np.abs(ref)))
    diff = float(np.max(np.abs(y - ref)))
    if scale == 0.0:
        return 0.0 if diff == 0.0 else float("inf")
    return diff / scale


def rel_err_tiles(y, ref, tile_rows=32, tile_cols=32):
    """The same measure taken per output tile: the largest, over every
    ``tile_rows x tile_cols`` tile of the 2-D result (ragged tiles at the
    edges included), of ``max|y - r| / max|r|`` within the tile.  An error
    confined to small-magnitude rows or to one tile (a wrong bias, a dropped
    block) then shows even when the whole result's maximum is far larger.
    Same conventions as rel_err: a tile whose reference is all zero must be
    exactly zero; non-finite values or a shape mismatch give inf."""
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    if y.shape != ref.shape or not np.all(np.isfinite(y)):
        return float("inf")
    if ref.ndim == 1:
        y, ref = y[None, :], ref[None, :]
    if ref.ndim != 2:
        raise ValueError("rel_err_tiles takes 1-D or 2-D results")
    M, N = ref.shape
    if M == 0 or N == 0:
        return 0.0
    pm, pn = -M % tile_rows, -N % tile_cols
    # zero padding changes neither a tile's largest difference nor its scale
    d = np.pad(np.abs(y - ref), ((0, pm), (0, pn)))
    a = np.pad(np.abs(ref), ((0, pm), (0, pn)))
    shape = ((M + pm) // tile_rows, tile_rows, (N + pn) // tile_cols, tile_cols)
    diff = d.reshape(shape).max(axis=(1, 3))
    scale = a.reshape(shape).max(axis=(1, 3))
    if np.any((scale == 0.0) & (diff != 0.0)):
        return float("inf")
    nz = scale > 0.0
    return float(np.max(diff[nz] / scale[nz])) if np.any(nz) else 0.0
    return worst
