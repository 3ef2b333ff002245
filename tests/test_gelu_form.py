"""CPU checks of the GELU form the bf16 translation kernels evaluate.

The fused kernel computes g * GELU(x) as g * x / (1 + 2^(x (K1 + K3 x^2))), the tanh
form of GELU written as a logistic (the two-GEMM path's epilogue x / (1 + 2^(...)),
the same form without the gate), with K1 and K3 defined in the device
header.  These tests read those two constants from the source and check, in
float64, that they are the tanh form's (K1 = -2 sqrt(2/pi) log2 e,
K3 = 0.044715 K1), that the form stays within 4.7e-4 of the exact erf GELU
(its rms deviation over normal pre-activations is an order below the rounding
to bf16 that the hidden value gets next), and that
GELU(x) - GELU(-x) = x still holds, which the E = 1 pass-through parity case
relies on.  Nothing here runs on a GPU."""
import math
import os
import re

import numpy as np
from scipy.special import erf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DEVICE_H = os.path.join(ROOT, "paper_2607_28979_amd", "csrc", "mot_device.h")


def _constants():
    txt = open(DEVICE_H).read()
    k = {}
    for name in ("MOT_GELU_K1", "MOT_GELU_K3"):
        m = re.search(r"#define\s+%s\s+\(?\s*([-+0-9.eE]+)f?\s*\)?" % name, txt)
        assert m, name + " not defined in the device header"
        k[name] = float(np.float32(float(m.group(1))))
    return k["MOT_GELU_K1"], k["MOT_GELU_K3"]


def _gelu_kernel_form(x, k1, k3):
    # exp2 overflows to inf for very negative x, as on the GPU; x / inf = 0
    with np.errstate(over="ignore"):
        return x / (1.0 + np.exp2(x * (k1 + k3 * x * x)))


def _gelu_erf(x):
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def test_constants_are_the_tanh_form():
    k1, k3 = _constants()
    want_k1 = -2.0 * math.sqrt(2.0 / math.pi) / math.log(2.0)
    assert abs(k1 - want_k1) <= 2 ** -22 * abs(want_k1)
    assert abs(k3 - 0.044715 * want_k1) <= 2 ** -22 * abs(0.044715 * want_k1)


def test_deviation_from_erf_gelu_within_documented_bound():
    k1, k3 = _constants()
    x = np.linspace(-12.0, 12.0, 1_200_001)
    d = np.abs(_gelu_kernel_form(x, k1, k3) - _gelu_erf(x))
    # largest absolute deviation 4.7e-4, at |x| ~ 2.7 (the deviation is even in x)
    assert d.max() <= 4.8e-4
    assert 2.5 < abs(x[int(d.argmax())]) < 2.9
    # below bf16's half step (2^-9 relative) wherever |GELU| >= 0.25
    big = np.abs(_gelu_erf(x)) >= 0.25
    assert (d[big] / np.abs(_gelu_erf(x[big]))).max() < 2 ** -9


def test_rms_deviation_an_order_below_bf16_rounding():
    # over normally distributed pre-activations the rms deviation is ~2e-4 of
    # the rms GELU value; rounding to bf16 alone gives ~1.7e-3
    k1, k3 = _constants()
    rng = np.random.default_rng(7)
    for sigma in (0.5, 1.0, 2.0, 3.0):
        x = rng.normal(0.0, sigma, 400_000)
        ge = _gelu_erf(x)
        dev = _gelu_kernel_form(x, k1, k3) - ge
        assert math.sqrt(np.mean(dev ** 2) / np.mean(ge ** 2)) < 2.5e-4


def test_odd_split_identity_and_limits():
    k1, k3 = _constants()
    x = np.linspace(-30.0, 30.0, 60_001)
    g = _gelu_kernel_form(x, k1, k3)
    gm = _gelu_kernel_form(-x, k1, k3)
    assert np.abs(g - gm - x).max() <= 1e-12 * (1.0 + np.abs(x)).max()
    # tails: GELU(x) -> x for large x, -> 0 for very negative x
    assert _gelu_kernel_form(np.array([40.0]), k1, k3)[0] == 40.0
    assert _gelu_kernel_form(np.array([-40.0]), k1, k3)[0] == 0.0
