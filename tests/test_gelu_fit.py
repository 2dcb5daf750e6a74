"""The GELU epilogue's error-function polynomial (csrc/lpv_device.h): its
coefficients are the ones paper_2407_02068_amd/gelu_fit.py produces, and the
kernel's formula, evaluated step by step in float32 here, meets the accuracy
the header states against scipy's float64 erfc (host logic; no GPU)."""
import os
import re

import numpy as np
from scipy.special import erfc

from paper_2407_02068_amd import gelu_fit

HERE = os.path.dirname(os.path.abspath(__file__))
DEVICE_H = os.path.join(HERE, "..", "paper_2407_02068_amd", "csrc", "lpv_device.h")


def device_coefficients():
    src = open(DEVICE_H).read()
    body = src[src.index("__device__ inline float gelu_erf(float v)"):]
    body = body[:body.index("__builtin_amdgcn_exp2f")]
    vals = [float(v) for v in re.findall(r"(-?\d\.\d+e[-+]\d+)f", body)]
    return np.array(vals[::-1], dtype=np.float32)  # Horner order -> constant term first


def gelu32(x, c):
    """The device formula, operation by operation, in float32."""
    x = np.asarray(x, np.float32)
    a = (np.abs(x) * np.float32(0.70710678118654752)).astype(np.float32)
    c = np.array(c, np.float32)
    c[0] = np.float32(c[0]) - np.float32(0.5)  # e = 2^(f(a) - 1/2) = erfc(a) / sqrt 2
    with np.errstate(over="ignore", invalid="ignore"):
        e = np.exp2(gelu_fit.horner32(c, a).astype(np.float64)).astype(np.float32)
        r = np.maximum(x, np.float32(0.0))
        # the fused multiply-add rounds once
        t = (r.astype(np.float64) - a.astype(np.float64) * e.astype(np.float64)).astype(np.float32)
    return np.where(a >= 4.0, r, t)


def test_device_coefficients_are_the_fit():
    c = gelu_fit.fit()
    d = device_coefficients()
    assert len(d) == gelu_fit.DEGREE + 1
    np.testing.assert_allclose(d, c, rtol=1e-8, atol=0)


def test_gelu_accuracy():
    c = device_coefficients()
    x = np.linspace(-40.0, 40.0, 800001).astype(np.float32)
    ref = x.astype(np.float64) * 0.5 * erfc(-x.astype(np.float64) / np.sqrt(2.0))
    err = np.abs(gelu32(x, c).astype(np.float64) - ref)
    big = np.abs(ref) > 1e-3
    assert (err[big] / np.abs(ref[big])).max() < 6e-6
    assert err.max() < 1e-6
    # the negative tail keeps its relative accuracy (no 1 + erf cancellation)
    tail = (x < -1.0) & (x > -5.5)
    assert (err[tail] / np.abs(ref[tail])).max() < 1e-5


def test_gelu_special_values():
    c = device_coefficients()
    g = gelu32(np.array([np.inf, -np.inf, 0.0, 6.0, -6.0], np.float32), c)
    assert g[0] == np.inf and g[1] == 0.0 and g[2] == 0.0
    assert g[3] == np.float32(6.0) and g[4] == 0.0
