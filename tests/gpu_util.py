"""Helpers of the GPU tests: moving generated inputs to the device, reading
results back, and the parity bar."""
import numpy as np
import torch

import oracle

TORCH = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
# infinity-norm relative error bound against the float64 oracle, fp32 accumulation
TOL = {"bf16": 2e-2, "f16": 5e-3, "f32": 1e-5}


def dev(a, dtype=None):
    """numpy array (element type ``dtype``) -> CUDA tensor; uint8 masks as is."""
    a = np.ascontiguousarray(a)
    if dtype == "bf16":
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).cuda()
    return torch.from_numpy(a.copy()).cuda()


def host(t, dtype):
    """CUDA tensor -> numpy array in the element type's representation."""
    t = t.detach().contiguous().cpu()
    if dtype == "bf16":
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def f64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def bits(a):
    a = np.ascontiguousarray(a)
    return a.view({2: np.uint16, 4: np.uint32}[a.dtype.itemsize])


def say(*args):
    print(*args, flush=True)


def assert_close(y, r, dtype, what="", tile=(32, 32)):
    """The parity bar on float values: the infinity-norm relative error of the
    whole result and, for 2-D results, of every output tile (so an error
    confined to one tile or to small-magnitude outputs cannot hide under the
    global maximum) must both be within the element type's bound."""
    err = oracle.rel_err(y, r)
    y2, r2 = np.asarray(y), np.asarray(r)
    if r2.ndim > 2:
        r2 = r2.reshape(-1, r2.shape[-1])
        y2 = y2.reshape(-1, y2.shape[-1]) if y2.size == r2.size else y2
    terr = oracle.rel_err_tiles(y2, r2, *tile) if r2.ndim <= 2 else err
    say("  %s rel err %.3e, per tile %.3e (bar %.0e)" % (what, err, terr, TOL[dtype]))
    assert err <= TOL[dtype], "%s: relative error %.3e above %.0e" % (what, err, TOL[dtype])
    assert terr <= TOL[dtype], "%s: per-tile relative error %.3e above %.0e" % (what, terr, TOL[dtype])
