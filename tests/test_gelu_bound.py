"""Error bound of the GPU's GELU (an erf polynomial on a clamped interval,
evaluated in fp32 with fused multiply-adds) against the exact erf GELU the
oracle uses.  The coefficients are read from the kernel source and the fp32
evaluation order is reproduced step by step (each fused multiply-add rounded
once); no GPU is needed."""
import os
import re

import numpy as np
from scipy.special import erf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
COMMON = os.path.join(ROOT, "paper_2609_35139_amd", "csrc", "common.h")


def _coefficients():
    src = open(COMMON).read()
    z0 = float(re.search(r"kGeluZ0\s*=\s*([0-9.eE+-]+)f", src).group(1))
    body = re.search(r"kGeluErfPoly\[\d+\]\s*=\s*\{([^}]*)\}", src).group(1)
    c = [float(v.strip().rstrip("f")) for v in body.split(",") if v.strip()]
    return np.float32(z0), [np.float32(v) for v in c]


def _fma(a, b, c):
    # one rounding to fp32 (the fp64 product of two fp32 values is exact)
    return (a.astype(np.float64) * b.astype(np.float64) + c.astype(np.float64)).astype(np.float32)


def _gelu_gpu(x, z0, c):
    x = np.asarray(x, np.float32)
    z = np.minimum(np.maximum((x * np.float32(0.70710678118654752)).astype(np.float32), -z0), z0)
    s = (z * z).astype(np.float32)
    p = np.full_like(s, c[-1])
    for k in range(len(c) - 2, -1, -1):
        p = _fma(p, s, np.full_like(s, c[k]))
    e = np.minimum(np.maximum((z * p).astype(np.float32), np.float32(-1)), np.float32(1))
    hx = (np.float32(0.5) * x).astype(np.float32)
    return _fma(hx, e, hx)


def _gelu_exact(x):
    x = np.asarray(x, np.float64)
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def test_gelu_polynomial_error_bound():
    z0, c = _coefficients()
    assert len(c) == 9 and z0 == np.float32(3.05)
    x = np.concatenate([np.linspace(-60, 60, 2_400_001), np.linspace(-6, 6, 1_200_001),
                        [0.0, -0.0, 1e-30, -1e-30, 4.3133, -4.3133]]).astype(np.float32)
    err = np.abs(_gelu_gpu(x, z0, c).astype(np.float64) - _gelu_exact(x))
    assert err.max() <= 5.6e-5, float(err.max())
    assert (err / np.maximum(1.0, np.abs(x))).max() <= 1.4e-5
    # far outside the fitted interval the result is x or -0 up to 1.4e-5 |x|
    big = np.array([-1e4, -100.0, 100.0, 1e4], np.float32)
    g = _gelu_gpu(big, z0, c).astype(np.float64)
    assert np.all(np.abs(g - _gelu_exact(big)) <= 1.4e-5 * np.abs(big))
    # GELU(0) = 0 exactly and the approximation is odd-symmetric in erf
    assert _gelu_gpu(np.zeros(1, np.float32), z0, c)[0] == 0.0


def test_gelu_error_is_far_below_a_bf16_rounding():
    """Over the range of FFN pre-activations (|x| <= 8), the approximation
    error is below an eighth of half a bf16 ulp of the exact value wherever
    that value exceeds 0.05 (GELU's minimum is -0.17)."""
    z0, c = _coefficients()
    x = np.linspace(-8, 8, 800_001).astype(np.float32)
    exact = _gelu_exact(x)
    err = np.abs(_gelu_gpu(x, z0, c).astype(np.float64) - exact)
    sel = np.abs(exact) > 0.05
    half_ulp = 2.0 ** (np.floor(np.log2(np.abs(exact[sel]))) - 8)
    assert np.all(err[sel] <= 0.125 * half_ulp)
