"""The bf16 GEMM epilogue's GELU (gelu_poly in common.h): its fp32 constants,
evaluated as the kernel evaluates them, stay within the stated error bound of
the exact erf GELU; and the committed fit script reproduces them."""
import importlib.util
import os
import re

import numpy as np
from scipy.special import erf

CSRC = os.path.join(os.path.dirname(__file__), "..", "paper_2609_10018_amd", "csrc")


def constants():
    src = open(os.path.join(CSRC, "common.h")).read()
    z = float(re.search(r"kGeluZ\s*=\s*([0-9.eE+-]+)f", src).group(1))
    body = re.search(r"kGeluC\[\d+\]\s*=\s*\{([^}]*)\}", src).group(1)
    c = np.array([float(t.strip().rstrip("f")) for t in body.split(",")], dtype=np.float32)
    return z, c


def fma32(a, b, c):
    return (a.astype(np.float64) * b.astype(np.float64) + np.float64(c)).astype(np.float32)


def gelu_poly(z, zmax, c):
    z = z.astype(np.float32)
    s = np.clip(z * np.float32(1.0 / zmax), np.float32(-1.0), np.float32(1.0))
    s2 = s * s
    q = np.full_like(z, c[-1])
    for k in range(len(c) - 2, -1, -1):
        q = fma32(q, s2, c[k])
    return z * fma32(s, q, np.float32(0.5))


def test_error_bound():
    zmax, c = constants()
    z = np.linspace(-12, 12, 2_400_001)
    exact = 0.5 * z * (1.0 + erf(z / np.sqrt(2.0)))
    got = gelu_poly(z, zmax, c).astype(np.float64)
    err = np.abs(got - exact)
    assert err.max() <= 1e-4
    big = np.abs(exact) > 0.1
    assert (err[big] / np.abs(exact[big])).max() <= 1e-4
    # far tails: identity above, zero below, within the clamp's 3.4e-6 relative
    far = np.array([20.0, 100.0, -20.0, -100.0], dtype=np.float32)
    g = gelu_poly(far, zmax, c).astype(np.float64)
    assert np.allclose(g[:2], far[:2], rtol=4e-6)
    assert np.all(np.abs(g[2:]) <= 4e-6 * np.abs(far[2:]))


def test_fit_script_reproduces_constants():
    spec = importlib.util.spec_from_file_location("gelu_fit", os.path.join(CSRC, "gelu_fit.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    zmax, c = constants()
    assert zmax == mod.Z
    np.testing.assert_allclose(mod.fit(), c, rtol=1e-6)
