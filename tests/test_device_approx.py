"""Error bounds of the device-side function approximations, checked on the CPU.

The kernels compute GELU(x) = x Phi(x) as x sigmoid(g(x)) with an odd
quintic g (clamped at |x| = 6).  The coefficients are read from the device
header, so this checks the values the kernels are built with: the formula is
evaluated in float32 in the kernels' order and compared with x Phi(x) in
float64 (scipy's normal distribution function)."""
import os
import re

import numpy as np
from scipy.special import ndtr

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "paper_2609_23733_amd", "csrc", "vp_device.hpp")
LOG2E = np.float32(1.4426950408889634)


def _coeffs():
    src = open(HEADER).read()
    out = {}
    for name in ("kGeluA1", "kGeluA3", "kGeluA5"):
        m = re.search(name + r"\s*=\s*([-+0-9.eE]+)f", src)
        assert m, name
        out[name] = np.float32(float(m.group(1)))
    return out


def gelu_device_model(x):
    """The device formula in float32: x / (1 + 2^(-g log2 e))."""
    c = _coeffs()
    x = x.astype(np.float32)
    xc = np.clip(x, np.float32(-6), np.float32(6))
    x2 = xc * xc
    inner = x2 * np.float32(c["kGeluA5"] * LOG2E) + np.float32(c["kGeluA3"] * LOG2E)
    g = xc * (x2 * inner + np.float32(c["kGeluA1"] * LOG2E))
    e = np.exp2(-g).astype(np.float32)
    return x * (np.float32(1) / (np.float32(1) + e))


def test_gelu_error_bound():
    x = np.concatenate([np.linspace(-40, 40, 800001), np.array([0.0, -0.0, 1e-30, -1e-30])])
    exact = x * ndtr(x)
    got = gelu_device_model(x).astype(np.float64)
    err = np.abs(got - exact)
    assert err.max() <= 2.6e-5, (err.max(), x[err.argmax()])
    # far tails: x for large positive x, ~0 for large negative x
    assert np.allclose(gelu_device_model(np.array([7.0, 30.0, 1e6])), [7.0, 30.0, 1e6], rtol=1e-6)
    assert np.abs(gelu_device_model(np.array([-7.0, -30.0]))).max() < 1e-6


def test_gelu_below_bf16_rounding():
    """Where |GELU| >= 0.05 the error stays below half a bf16 ulp of the value."""
    x = np.linspace(-6, 6, 120001)
    exact = x * ndtr(x)
    got = gelu_device_model(x).astype(np.float64)
    m = np.abs(exact) >= 0.05
    half_ulp = 2.0 ** -9 * np.abs(exact[m])
    assert (np.abs(got[m] - exact[m]) <= half_ulp).all()


def test_gelu_nan_propagates():
    assert np.isnan(gelu_device_model(np.array([np.nan]))).all()
