"""Coefficients of the bf16 path's GELU (``gelu_poly`` in common.h).

GELU(z) = z * Phi(z), Phi the standard normal CDF.  With s = clamp(z / Z, -1, 1),
Phi(z) - 1/2 = erf(z / sqrt 2) / 2 is approximated by s * q(s^2), q a
polynomial of degree NC - 1; the coefficients are a near-minimax fit on
[0, 1] (iteratively reweighted least squares on Chebyshev points, Lawson's
method), rounded to fp32.  Beyond |z| = Z the clamp holds Phi at
1/2 +- (erf(Z / sqrt 2) / 2), off by at most 3.4e-6.  The result is rounded to
bf16 (relative step 2^-8), so a fit error of order 1e-4 is below the output's
own rounding.

    python gelu_fit.py      # prints the C array
"""
import numpy as np
from scipy.special import erf

Z = 4.5
NC = 10


def fit(z_max=Z, nc=NC, iters=300):
    s = np.cos(np.linspace(0.0, np.pi, 40001))
    s = s[s > 0]
    h = 0.5 * erf(s * z_max / np.sqrt(2.0))
    A = np.stack([s ** (2 * k + 1) for k in range(nc)], 1)
    w = np.full_like(s, 1.0 / len(s))
    for _ in range(iters):
        sw = np.sqrt(w)
        c, *_ = np.linalg.lstsq(A * sw[:, None], h * sw, rcond=None)
        w = w * np.abs(A @ c - h)
        w /= w.sum()
    return c.astype(np.float32)


if __name__ == "__main__":
    c = fit()
    print(f"constexpr float kGeluZ = {Z}f;")
    print("constexpr float kGeluC[%d] = {" % NC + ", ".join(f"{float(v):.9e}f" for v in c) + "};")
