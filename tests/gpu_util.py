"""Helpers of the GPU tests: moving generated inputs to the device, reading
results back, and the parity bar."""
import numpy as np
import torch

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
