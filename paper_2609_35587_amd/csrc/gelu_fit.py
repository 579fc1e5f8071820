"""Fit of the GELU tail used by the matrix-core MLP kernel (mlp.hip).

GELU(a) = a Phi(a) = max(a, 0) - |a| Phi(-|a|), Phi the standard normal
distribution function.  For x >= 0, log2 Phi(-x) is smooth and concave, so
Phi(-x) ~ 2^P(x) with P a polynomial of low degree.  P (degree 3: the
kernel stores every activation in bf16, whose half-step is 2e-3 at 1, so an
error of 1e-4 costs nothing there and three FMAs are enough) is fitted on
[0, 5] by
iteratively reweighted least squares on the absolute GELU error
x |2^P(x) - Phi(-x)| (Lawson's iteration towards the minimax fit); the
coefficients are then rounded to fp32 and the error is checked in fp32
Horner arithmetic over [0, 12] and on a geometric grid up to 1e38.  Run
`python gelu_fit.py` to print the coefficients (highest degree first) and the
error bound.
"""
import numpy as np
from scipy.special import erfc


def phi_neg(x):
    return 0.5 * erfc(x / np.sqrt(2.0))


def fit(deg=3, xmax=5.0, iters=30):
    x = np.linspace(0.0, xmax, 120001)
    y = np.log2(phi_neg(x))
    w = np.maximum(x * phi_neg(x), 1e-6)      # d(abs GELU error) / d(error in P), up to ln 2
    A = np.vander(x, deg + 1)
    for _ in range(iters):
        c, *_ = np.linalg.lstsq(A * w[:, None], y * w, rcond=None)
        err = (np.polyval(c, x) - y) * w
        w = w * (1.0 + 3.0 * np.abs(err) / np.abs(err).max())
    return c.astype(np.float32)


def max_error(c32):
    xs = np.concatenate([np.linspace(0.0, 12.0, 400001), np.geomspace(12.0, 1e38, 10000)]).astype(np.float32)
    with np.errstate(over="ignore", under="ignore", invalid="ignore"):
        p = np.full_like(xs, c32[0])
        for ci in c32[1:]:
            p = (p * xs + ci).astype(np.float32)
        e = np.abs(xs.astype(np.float64) * (np.exp2(p.astype(np.float64)) - phi_neg(xs.astype(np.float64))))
    return float(e.max()), float(xs[e.argmax()])


if __name__ == "__main__":
    c = fit()
    err, at = max_error(c)
    print("coefficients (x^%d .. x^0):" % (len(c) - 1), ", ".join(repr(float(v)) for v in c))
    print("max |GELU error| = %.3g at |a| = %.3g" % (err, at))
