"""Python binding of liblpv (include/lpv.h): argument marshalling only.

Every computation runs in the HIP kernels of ``liblpv.so``.  PyTorch supplies
device memory and the current HIP stream; this module checks torch-level
properties (device, dtype, layout), passes raw pointers and sizes through
ctypes and turns status codes into exceptions.  There is no fallback: without
the built library every call raises.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblpv.so")

LPV_OK = 0
STATUS = {0: "LPV_OK", -1: "LPV_ERR_INVALID_ARG", -2: "LPV_ERR_SHAPE", -3: "LPV_ERR_DTYPE",
          -4: "LPV_ERR_BLOCK", -5: "LPV_ERR_ALIAS", -6: "LPV_ERR_ALLOC", -7: "LPV_ERR_HIP"}
DTYPES = {torch.float32: 0, torch.float16: 1, torch.bfloat16: 2}
EPI = {None: 0, "none": 0, "gelu": 1}
EXPORTED = ("lpv_bsr_pack", "lpv_bsr_info_get", "lpv_bsr_export", "lpv_bsr_schedule_export",
            "lpv_bsr_unpack", "lpv_bsr_linear", "lpv_dense_linear", "lpv_mask_topk",
            "lpv_bsr_transpose", "lpv_bsr_grad_w", "lpv_bias_grad", "lpv_bias_grad_noalloc",
            "lpv_delta_curve", "lpv_delta_curve_ws", "lpv_delta_curve_workspace_size",
            "lpv_add_layernorm", "lpv_attention", "lpv_bsr_destroy", "lpv_status_str",
            "lpv_last_error")


class LpvError(RuntimeError):
    def __init__(self, status, where, detail):
        self.status = status
        super().__init__("%s: %s (%s)" % (where, STATUS.get(status, status), detail))


class BsrInfo(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int64), ("K", ctypes.c_int64), ("b_r", ctypes.c_int32),
                ("b_c", ctypes.c_int32), ("R", ctypes.c_int32), ("C", ctypes.c_int32),
                ("nnzb", ctypes.c_int64), ("dtype", ctypes.c_int32), ("device", ctypes.c_int32),
                ("tile_rows", ctypes.c_int32), ("tile_cols", ctypes.c_int32),
                ("group_tiles", ctypes.c_int32), ("n_groups", ctypes.c_int32),
                ("n_steps", ctypes.c_int64), ("n_tiles", ctypes.c_int64)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


_lib = None


def lib():
    """The loaded liblpv.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("liblpv.so is not built (%s); run __graft_entry__.build() or "
                           "python paper_2407_02068_amd/build.py" % LIB_PATH)
    L = ctypes.CDLL(LIB_PATH)
    i64, i32, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
    L.lpv_bsr_pack.argtypes = [vp, i64, i64, i64, i32, i32, i32, vp, vp, ctypes.POINTER(vp)]
    L.lpv_bsr_info_get.argtypes = [vp, ctypes.POINTER(BsrInfo)]
    L.lpv_bsr_export.argtypes = [vp, vp, vp, vp, vp]
    L.lpv_bsr_schedule_export.argtypes = [vp, vp, vp, vp, vp, vp, vp]
    L.lpv_bsr_unpack.argtypes = [vp, vp, i64, vp]
    L.lpv_bsr_linear.argtypes = [vp, vp, i64, i64, vp, vp, i64, i32, vp]
    L.lpv_dense_linear.argtypes = [vp, i64, i64, i64, i32, vp, i64, i64, vp, vp, i64, i32, vp]
    L.lpv_mask_topk.argtypes = [vp, i64, i64, i64, i32, i32, i32, vp, i64, i32, vp, vp, vp]
    L.lpv_bsr_transpose.argtypes = [vp, vp, ctypes.POINTER(vp)]
    L.lpv_bsr_grad_w.argtypes = [vp, vp, i64, vp, i64, i64, vp, vp]
    L.lpv_bias_grad.argtypes = [vp, i64, i64, i64, i32, vp, vp]
    L.lpv_bias_grad_noalloc.argtypes = [vp, i64, i64, i64, i32, vp, vp]
    L.lpv_add_layernorm.argtypes = [vp, vp, i64, i64, i32, vp, vp, ctypes.c_double, vp, vp, vp]
    L.lpv_attention.argtypes = [vp, i64, i32, i32, i32, i32, vp, vp]
    L.lpv_delta_curve.argtypes = [vp, i64, i64, i64, i32, i32, i32, vp, i64, vp, i64, i64, i64,
                                  ctypes.c_double, vp, i32, vp, vp]
    L.lpv_delta_curve_ws.argtypes = [vp, i64, i64, i64, i32, i32, i32, vp, i64, vp, i64, i64,
                                     i64, ctypes.c_double, vp, i32, vp, vp, ctypes.c_size_t, vp]
    L.lpv_delta_curve_workspace_size.argtypes = [i64, i64, i32, i32, i64, i32,
                                                 ctypes.POINTER(ctypes.c_size_t)]
    for f in ("lpv_bsr_pack", "lpv_bsr_info_get", "lpv_bsr_export", "lpv_bsr_schedule_export",
              "lpv_bsr_unpack", "lpv_bsr_linear", "lpv_dense_linear", "lpv_mask_topk",
              "lpv_bsr_transpose", "lpv_bsr_grad_w", "lpv_bias_grad", "lpv_bias_grad_noalloc",
              "lpv_delta_curve", "lpv_delta_curve_ws", "lpv_delta_curve_workspace_size",
              "lpv_add_layernorm", "lpv_attention"):
        getattr(L, f).restype = i32
    L.lpv_bsr_destroy.argtypes = [vp]
    L.lpv_bsr_destroy.restype = None
    L.lpv_status_str.argtypes = [i32]
    L.lpv_status_str.restype = ctypes.c_char_p
    L.lpv_last_error.argtypes = []
    L.lpv_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def status_str(status):
    return lib().lpv_status_str(status).decode()


def last_error():
    return lib().lpv_last_error().decode()


def _check(status, where):
    if status != LPV_OK:
        raise LpvError(status, where, last_error())


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _mat(t, name):
    """(pointer, leading dimension) of a 2-D device tensor with unit column stride."""
    if not isinstance(t, torch.Tensor) or t.dim() != 2:
        raise TypeError("%s must be a 2-D torch tensor" % name)
    if not t.is_cuda:
        raise ValueError("%s must live on the GPU" % name)
    if t.dtype not in DTYPES:
        raise TypeError("%s: unsupported dtype %s" % (name, t.dtype))
    if t.shape[1] > 1 and t.stride(1) != 1:
        raise ValueError("%s must have unit stride along its columns" % name)
    ld = t.stride(0) if t.shape[0] > 1 else max(t.shape[1], t.stride(0))
    return ctypes.c_void_p(t.data_ptr()), ld


class BsrWeight:
    """A packed block-sparse weight (owns an lpv_bsr handle)."""

    def __init__(self, handle):
        self._h = ctypes.c_void_p(handle)
        info = BsrInfo()
        _check(lib().lpv_bsr_info_get(self._h, ctypes.byref(info)), "lpv_bsr_info_get")
        self.info = info.as_dict()
        self.dtype = {v: k for k, v in DTYPES.items()}[self.info["dtype"]]

    @property
    def handle(self):
        return self._h

    def __getattr__(self, k):
        info = self.__dict__.get("info")
        if info is not None and k in info:
            return info[k]
        raise AttributeError(k)

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            lib().lpv_bsr_destroy(self._h)
            self._h = ctypes.c_void_p(0)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def bsr_pack(W, mask, b_r, b_c, stream=None):
    """lpv_bsr_pack: W (N x K device tensor) and a uint8 block mask (device,
    N/b_r x K/b_c) -> BsrWeight.  Waits for the pack to finish."""
    wp, ldw = _mat(W, "W")
    if not isinstance(mask, torch.Tensor) or not mask.is_cuda or mask.dtype != torch.uint8:
        raise TypeError("mask must be a uint8 tensor on the GPU")
    if not mask.is_contiguous():
        raise ValueError("mask must be contiguous")
    N, K = W.shape
    if b_r > 0 and b_c > 0 and N % b_r == 0 and K % b_c == 0 \
            and mask.numel() != (N // b_r) * (K // b_c):
        raise ValueError("mask has %d entries, expected %d" % (mask.numel(), (N // b_r) * (K // b_c)))
    out = ctypes.c_void_p()
    _check(lib().lpv_bsr_pack(wp, ldw, N, K, DTYPES[W.dtype], b_r, b_c,
                              ctypes.c_void_p(mask.data_ptr()), _stream(stream), ctypes.byref(out)),
           "lpv_bsr_pack")
    return BsrWeight(out.value)


def bsr_info(h):
    return dict(h.info)


def bsr_export(h, stream=None):
    """lpv_bsr_export -> (row_ptr, col_idx, values) as new device tensors."""
    dev = torch.device("cuda", h.info["device"])
    row_ptr = torch.empty(h.info["R"] + 1, dtype=torch.int32, device=dev)
    col_idx = torch.empty(max(h.info["nnzb"], 1), dtype=torch.int32, device=dev)
    values = torch.empty((max(h.info["nnzb"], 1), h.info["b_r"], h.info["b_c"]), dtype=h.dtype,
                         device=dev)
    _check(lib().lpv_bsr_export(h.handle, ctypes.c_void_p(row_ptr.data_ptr()),
                                ctypes.c_void_p(col_idx.data_ptr()),
                                ctypes.c_void_p(values.data_ptr()), _stream(stream)),
           "lpv_bsr_export")
    n = h.info["nnzb"]
    return row_ptr, col_idx[:n], values[:n]


def bsr_schedule_export(h, stream=None):
    """lpv_bsr_schedule_export -> dict of int32 device tensors."""
    dev = torch.device("cuda", h.info["device"])
    ng, ns = h.info["n_groups"], h.info["n_steps"]
    t = {k: torch.empty(max(n, 1), dtype=torch.int32, device=dev)
         for k, n in (("group_order", ng), ("step_ptr", ng + 1), ("step_col", ns),
                      ("step_bits", ns), ("step_tile", ns))}
    _check(lib().lpv_bsr_schedule_export(
        h.handle, *[ctypes.c_void_p(t[k].data_ptr()) for k in
                    ("group_order", "step_ptr", "step_col", "step_bits", "step_tile")],
        _stream(stream)), "lpv_bsr_schedule_export")
    return {"group_order": t["group_order"][:ng], "step_ptr": t["step_ptr"][:ng + 1],
            "step_col": t["step_col"][:ns], "step_bits": t["step_bits"][:ns],
            "step_tile": t["step_tile"][:ns]}


def bsr_unpack(h, out=None, stream=None):
    """lpv_bsr_unpack -> the pruned dense weight (N x K)."""
    if out is None:
        out = torch.empty((h.info["N"], h.info["K"]), dtype=h.dtype,
                          device=torch.device("cuda", h.info["device"]))
    op, ld = _mat(out, "out")
    _check(lib().lpv_bsr_unpack(h.handle, op, ld, _stream(stream)), "lpv_bsr_unpack")
    return out


def _vec(b, name):
    if b is None:
        return None
    if not isinstance(b, torch.Tensor) or not b.is_cuda or b.dim() != 1:
        raise TypeError("%s must be a 1-D tensor on the GPU" % name)
    if b.stride(0) != 1 and b.numel() > 1:
        raise ValueError("%s must be contiguous" % name)
    return ctypes.c_void_p(b.data_ptr())


def bsr_linear(h, X, bias=None, Y=None, epi=None, stream=None):
    """lpv_bsr_linear: Y = g(X W~^T + b).  Allocates Y (M x N) if not given."""
    if X.dtype != h.dtype:
        raise TypeError("X is %s but the weight is %s" % (X.dtype, h.dtype))
    if bias is not None and (bias.dtype != h.dtype or bias.numel() != h.info["N"]):
        raise ValueError("bias must hold N = %d elements of %s" % (h.info["N"], h.dtype))
    M = X.shape[0]
    if X.dim() != 2 or X.shape[1] != h.info["K"]:
        raise ValueError("X must be M x K = ? x %d" % h.info["K"])
    if Y is None:
        Y = torch.empty((M, h.info["N"]), dtype=h.dtype, device=X.device)
    if Y.dtype != h.dtype or Y.dim() != 2 or Y.shape != (M, h.info["N"]):
        raise ValueError("Y must be M x N = %d x %d of %s" % (M, h.info["N"], h.dtype))
    xp, ldx = _mat(X, "X")
    yp, ldy = _mat(Y, "Y")
    _check(lib().lpv_bsr_linear(h.handle, xp, ldx, M, _vec(bias, "bias"), yp, ldy, EPI[epi],
                                _stream(stream)), "lpv_bsr_linear")
    return Y


def dense_linear(W, X, bias=None, Y=None, epi=None, stream=None):
    """lpv_dense_linear: Y = g(X W^T + b) with a dense W, on the library's own
    matrix-core kernel."""
    if X.dtype != W.dtype:
        raise TypeError("X is %s but W is %s" % (X.dtype, W.dtype))
    N, K = W.shape
    M = X.shape[0]
    if X.dim() != 2 or X.shape[1] != K:
        raise ValueError("X must be M x K = ? x %d" % K)
    if Y is None:
        Y = torch.empty((M, N), dtype=W.dtype, device=X.device)
    wp, ldw = _mat(W, "W")
    xp, ldx = _mat(X, "X")
    yp, ldy = _mat(Y, "Y")
    _check(lib().lpv_dense_linear(wp, ldw, N, K, DTYPES[W.dtype], xp, ldx, M, _vec(bias, "bias"),
                                  yp, ldy, EPI[epi], _stream(stream)), "lpv_dense_linear")
    return Y


def mask_topk(W, b_r, b_c, sparsity_pct, G=None, stream=None):
    """lpv_mask_topk: block scores of W (mean |W * G| per block, or the block
    sum of squares without G) and the uint8 mask that keeps the
    ceil((100 - sparsity_pct) R C / 100) best-ranked blocks.  Returns
    (mask [R, C] uint8, scores [R, C] float64), both on W's device."""
    wp, ldw = _mat(W, "W")
    N, K = W.shape
    gp, ldg = None, 0
    if G is not None:
        if G.dtype != W.dtype or G.shape != W.shape:
            raise ValueError("G must match W's shape and dtype")
        gp, ldg = _mat(G, "G")
    R, C = (N // b_r, K // b_c) if b_r > 0 and b_c > 0 else (0, 0)
    mask = torch.empty((max(R, 1), max(C, 1)), dtype=torch.uint8, device=W.device)
    scores = torch.empty((max(R, 1), max(C, 1)), dtype=torch.float64, device=W.device)
    _check(lib().lpv_mask_topk(wp, ldw, N, K, DTYPES[W.dtype], b_r, b_c, gp, ldg,
                               int(sparsity_pct), ctypes.c_void_p(mask.data_ptr()),
                               ctypes.c_void_p(scores.data_ptr()), _stream(stream)),
           "lpv_mask_topk")
    return mask, scores


def bsr_transpose(h, stream=None):
    """lpv_bsr_transpose: the handle of W~^T (K x N).  The input gradient of the
    layer is then ``bsr_linear(ht, G)`` = G W~.  Waits for the build."""
    out = ctypes.c_void_p()
    _check(lib().lpv_bsr_transpose(h.handle, _stream(stream), ctypes.byref(out)),
           "lpv_bsr_transpose")
    return BsrWeight(out.value)


def grad_w(h, G, X, out=None, stream=None):
    """lpv_bsr_grad_w: G^T X on the kept blocks, [nnzb, b_r, b_c] in BSR value
    order (G: M x N, X: M x K, the handle's dtype)."""
    if G.dtype != h.dtype or X.dtype != h.dtype:
        raise TypeError("G and X must be %s" % h.dtype)
    if G.dim() != 2 or X.dim() != 2 or G.shape[0] != X.shape[0] \
            or G.shape[1] != h.info["N"] or X.shape[1] != h.info["K"]:
        raise ValueError("G must be M x %d and X M x %d" % (h.info["N"], h.info["K"]))
    shape = (h.info["nnzb"], h.info["b_r"], h.info["b_c"])
    if out is None:
        out = torch.empty(shape, dtype=h.dtype, device=G.device)
    if out.dtype != h.dtype or tuple(out.shape) != shape or not out.is_contiguous():
        raise ValueError("out must be a contiguous %s tensor of shape %s" % (h.dtype, shape))
    gp, ldg = _mat(G, "G")
    xp, ldx = _mat(X, "X")
    _check(lib().lpv_bsr_grad_w(h.handle, gp, ldg, xp, ldx, G.shape[0],
                                ctypes.c_void_p(out.data_ptr()), _stream(stream)), "lpv_bsr_grad_w")
    return out


def bias_grad(G, out=None, stream=None):
    """lpv_bias_grad: the column sums of G (M x N) -> N elements of G's dtype."""
    gp, ldg = _mat(G, "G")
    M, N = G.shape
    if out is None:
        out = torch.empty(N, dtype=G.dtype, device=G.device)
    if out.dtype != G.dtype or out.numel() != N or not out.is_contiguous():
        raise ValueError("out must be a contiguous %s tensor of %d elements" % (G.dtype, N))
    _check(lib().lpv_bias_grad(gp, ldg, M, N, DTYPES[G.dtype], ctypes.c_void_p(out.data_ptr()),
                               _stream(stream)), "lpv_bias_grad")
    return out


def bias_grad_noalloc(G, out, stream=None):
    """lpv_bias_grad_noalloc: the column sums of G (M x N) into ``out`` (N
    elements of G's dtype, caller-allocated), with no allocation inside the
    library (a fixed per-device scratch; overlapping calls on one GPU race)."""
    gp, ldg = _mat(G, "G")
    M, N = G.shape
    if out is None or out.dtype != G.dtype or out.numel() != N or not out.is_contiguous():
        raise ValueError("out must be a contiguous %s tensor of %d elements" % (G.dtype, N))
    _check(lib().lpv_bias_grad_noalloc(gp, ldg, M, N, DTYPES[G.dtype],
                                       ctypes.c_void_p(out.data_ptr()), _stream(stream)),
           "lpv_bias_grad_noalloc")
    return out


def delta_curve_workspace_size(N, K, b_r, b_c, n_samples, n_points):
    """lpv_delta_curve_workspace_size: bytes of the caller workspace
    ``delta_curve(..., workspace=)`` needs for this shape."""
    nbytes = ctypes.c_size_t(0)
    _check(lib().lpv_delta_curve_workspace_size(N, K, b_r, b_c, n_samples, n_points,
                                                ctypes.byref(nbytes)),
           "lpv_delta_curve_workspace_size")
    return nbytes.value


def delta_curve(W, grad, samples, b_r, b_c, kappa, pcts, out=None, stream=None, workspace=None):
    """lpv_delta_curve: the layer's delta curve at the sparsity percentages
    ``pcts`` (non-decreasing).  W, grad: N x K; samples: n x N x K per-sample
    gradients (same dtype).  Returns a float64 device tensor of len(pcts).
    With ``workspace`` (a contiguous GPU tensor of at least
    ``delta_curve_workspace_size`` bytes) it calls lpv_delta_curve_ws, which
    allocates nothing."""
    if grad.dtype != W.dtype or samples.dtype != W.dtype:
        raise TypeError("W, grad and samples must share a dtype")
    if samples.dim() != 3 or tuple(samples.shape[1:]) != tuple(W.shape) or grad.shape != W.shape:
        raise ValueError("grad must be N x K and samples n x N x K")
    N, K = W.shape
    n = samples.shape[0]
    if n > 0 and (samples.stride(2) != 1 or (N > 1 and samples.stride(1) < K)):
        raise ValueError("samples must have unit stride along K")
    pc = (ctypes.c_int32 * len(pcts))(*[int(p) for p in pcts])
    if out is None:
        out = torch.empty(len(pcts), dtype=torch.float64, device=W.device)
    wp, ldw = _mat(W, "W")
    gp, ldg = _mat(grad, "grad")
    lds = samples.stride(1) if n > 0 else K
    stride = samples.stride(0) if n > 0 else N * K
    args = (wp, ldw, N, K, DTYPES[W.dtype], b_r, b_c, gp, ldg,
            ctypes.c_void_p(samples.data_ptr()), lds, stride, n, float(kappa), pc, len(pcts),
            ctypes.c_void_p(out.data_ptr()))
    if workspace is None:
        _check(lib().lpv_delta_curve(*args, _stream(stream)), "lpv_delta_curve")
    else:
        if not isinstance(workspace, torch.Tensor) or not workspace.is_cuda \
                or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous GPU tensor")
        nbytes = workspace.numel() * workspace.element_size()
        _check(lib().lpv_delta_curve_ws(*args, ctypes.c_void_p(workspace.data_ptr()), nbytes,
                                        _stream(stream)), "lpv_delta_curve_ws")
    return out


def _param(t, name, dtype, n):
    if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != dtype or t.numel() != n \
            or not t.is_contiguous():
        raise ValueError("%s must be a contiguous %s GPU tensor of %d elements" % (name, dtype, n))
    return ctypes.c_void_p(t.data_ptr())


def add_layernorm(x, y, gamma, beta, eps, S=None, out=None, stream=None):
    """lpv_add_layernorm: s = x + y (y may be None), out = LN(s) * gamma + beta
    per row; s is written to S when given.  x, y, S, out: contiguous M x D."""
    if x.dim() != 2 or not x.is_contiguous():
        raise ValueError("x must be a contiguous 2-D tensor")
    M, D = x.shape
    if out is None:
        out = torch.empty_like(x)
    for t, n in ((y, "y"), (S, "S"), (out, "out")):
        if t is not None and (t.shape != x.shape or t.dtype != x.dtype or not t.is_contiguous()):
            raise ValueError("%s must be a contiguous tensor shaped and typed like x" % n)
    ptr = lambda t: ctypes.c_void_p(t.data_ptr() if t is not None else 0)
    _check(lib().lpv_add_layernorm(ptr(x), ptr(y), M, D, DTYPES[x.dtype],
                                   _param(gamma, "gamma", x.dtype, D), _param(beta, "beta", x.dtype, D),
                                   float(eps), ptr(S), ptr(out), _stream(stream)),
           "lpv_add_layernorm")
    return out


def attention(qkv, n_seq, T, H, out=None, stream=None, hd=64):
    """lpv_attention: multi-head self-attention of n_seq sequences of T tokens
    from the qkv layer's output ((n_seq T) x (3 H hd), contiguous); returns
    (n_seq T) x (H hd)."""
    if qkv.dim() != 2 or not qkv.is_contiguous() or tuple(qkv.shape) != (n_seq * T, 3 * H * hd):
        raise ValueError("qkv must be a contiguous (n_seq T) x (3 H hd) tensor")
    if out is None:
        out = torch.empty((n_seq * T, H * hd), dtype=qkv.dtype, device=qkv.device)
    if tuple(out.shape) != (n_seq * T, H * hd) or out.dtype != qkv.dtype or not out.is_contiguous():
        raise ValueError("out must be a contiguous (n_seq T) x (H hd) tensor of qkv's dtype")
    _check(lib().lpv_attention(ctypes.c_void_p(qkv.data_ptr()), n_seq, T, H, hd, DTYPES[qkv.dtype],
                               ctypes.c_void_p(out.data_ptr()), _stream(stream)), "lpv_attention")
    return out

