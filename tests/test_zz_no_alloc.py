"""lpv_bias_grad_noalloc (no allocation inside the library: a fixed
per-device scratch) against lpv_bias_grad, the allocating entry point it
varies, and the float64 oracle, on two calls in a row (the second smaller),
called through the C ABI."""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from gpu_util import TOL, assert_close, dev, f64, say
from paper_2407_02068_amd import lpv

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
def test_bias_grad_noalloc_two_calls(dtype):
    for M, N, seed in ((50432, 3072, 1), (1000, 768, 2)):
        say("bias_grad_noalloc", dtype, "M=%d N=%d" % (M, N))
        G = wl.grad_output(110 + seed, 0, M, N, dtype)
        Gd = dev(G, dtype)
        ref_db = lpv.bias_grad(Gd)
        out = torch.full((N,), 7.0, dtype=Gd.dtype, device="cuda")
        db = lpv.bias_grad_noalloc(Gd, out)
        torch.cuda.synchronize()
        r = oracle.grad_bias(G, dtype)
        assert_close(f64(db), f64(ref_db), dtype, "noalloc vs allocating")
        assert_close(f64(db), r, dtype, "noalloc vs oracle")


def test_bias_grad_noalloc_empty_and_columns_past_scratch_share():
    # M = 0 gives zeros; N = 65536 (the largest N) caps the chunks at 16
    out = torch.full((64,), 3.0, dtype=torch.bfloat16, device="cuda")
    lpv.bias_grad_noalloc(torch.empty((0, 64), dtype=torch.bfloat16, device="cuda"), out)
    torch.cuda.synchronize()
    assert not out.float().abs().sum().item()
    M, N = 300, 65536
    G = wl.grad_output(113, 0, M, N, "bf16")
    Gd = dev(G, "bf16")
    db = lpv.bias_grad_noalloc(Gd, torch.empty(N, dtype=torch.bfloat16, device="cuda"))
    torch.cuda.synchronize()
    assert_close(f64(db), oracle.grad_bias(G, "bf16"), "bf16", "noalloc N=65536")
