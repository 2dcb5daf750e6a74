"""Coefficients of the GELU epilogue's error function (csrc/lpv_device.h).

The kernels evaluate Phi(x) = erfc(-x / sqrt 2) / 2 from e = erfc(a),
a = min(|x| / sqrt 2, 4), as e = 2^f(a) with f a polynomial fitted here to
log2 erfc on [0, 4]: least squares on 4000 Chebyshev-spaced points, the
weights raised where the error is largest (Lawson's iteration) to approach a
minimax fit.  Run to print the float32 coefficients (constant term first) and
the error of a float32 Horner evaluation against scipy's erfc.
"""
import numpy as np
from scipy.special import erfc

DEGREE = 7
A_MAX = 4.0


def fit(degree=DEGREE, a_max=A_MAX, iters=30):
    x = (np.cos(np.linspace(0.0, np.pi, 4000)) + 1.0) * (a_max / 2)
    y = np.log2(erfc(x))
    V = np.vander(x, degree + 1, increasing=True)
    w = np.ones_like(x)
    for _ in range(iters):
        c, *_ = np.linalg.lstsq(V * w[:, None], y * w, rcond=None)
        err = np.abs(V @ c - y)
        w = w * (1.0 + 2.0 * err / err.max())
    return c.astype(np.float32)


def horner32(c, a):
    r = np.full_like(a, c[-1], dtype=np.float32)
    for k in range(len(c) - 2, -1, -1):
        r = (r * a + c[k]).astype(np.float32)
    return r


if __name__ == "__main__":
    c = fit()
    for k, v in enumerate(c):
        print("c%-2d = %.9e" % (k, v))
    a = np.linspace(0.0, A_MAX, 400001).astype(np.float32)
    e = np.exp2(horner32(c, a).astype(np.float64))
    ref = erfc(a.astype(np.float64))
    print("erfc relative error %.2e, erf absolute error %.2e"
          % ((np.abs(e - ref) / ref).max(), np.abs(e - ref).max()))
