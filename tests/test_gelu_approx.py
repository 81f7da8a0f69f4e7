"""Host checks of the kernels' branch-free GELU (ks_epilogue.h, gelu_f32).

The kernel evaluates GELU(x) = max(x, 0) - |x| Phi(-|x|) with the normal tail
Phi(-|x|) = u * 2^(-log2(e) x^2 / 2 + R(u)), u = 1 / (2 + |x| / sqrt 2), and R
a degree-9 polynomial whose coefficients are float literals in the header.
These tests read those literals, check that gelu_fit.py reproduces them, and
evaluate the same operation sequence in float32 on the CPU (each fused
multiply-add rounded once; the reciprocal and the power of two correctly
rounded, where the hardware's are within 1 ulp) against scipy's erfc in float64
and against the oracle's epilogue.  The GPU parity tests then compare the
kernels themselves with the oracle."""
import importlib.util
import os
import re

import numpy as np
from scipy.special import erfc

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2405_15013_amd", "csrc")


def header_coefficients(prefix="kGeluR"):
    text = open(os.path.join(CSRC, "ks_epilogue.h")).read()
    found = dict(re.findall(r"constexpr float %s(\d+) = ([-0-9.e+]+)f;" % prefix, text))
    return np.array([np.float32(found[str(k)]) for k in range(len(found))], dtype=np.float32)


def gelu_f32_emulated(x, prefix="kGeluR"):
    """prefix kGeluR: fp32 outputs (degree 9); kGeluS: 16-bit outputs (degree 5)."""
    f = np.float32
    x = np.asarray(x, dtype=np.float32)
    c = header_coefficients(prefix)

    def fma(a, b, d):
        return (a.astype(np.float64) * b.astype(np.float64) + np.float64(d) if np.ndim(d) == 0
                else a.astype(np.float64) * b.astype(np.float64) + d.astype(np.float64)).astype(np.float32)

    xc = np.clip(x, f(-16), f(16))
    ax = np.abs(xc)
    u = (1.0 / fma(ax, np.full_like(ax, f(0.70710678118654752)), f(2.0)).astype(np.float64)).astype(np.float32)
    r = np.full_like(u, c[-1])
    for ck in c[-2::-1]:
        r = fma(r, u, ck)
    t = fma((xc * f(-0.72134752044448170)).astype(np.float32), xc, r)
    tail = (u * np.exp2(t.astype(np.float64)).astype(np.float32)).astype(np.float32)
    with np.errstate(invalid="ignore"):
        return fma(-ax, tail, np.maximum(x, f(0)))


def test_coefficients_match_fit_script():
    spec = importlib.util.spec_from_file_location("gelu_fit", os.path.join(CSRC, "gelu_fit.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    fitted, err = mod.fit()
    assert err < 2e-7
    np.testing.assert_array_equal(fitted, header_coefficients())
    fitted, err = mod.fit(mod.DEGREE_16BIT)
    assert err < 2e-5 and len(fitted) == 6
    np.testing.assert_array_equal(fitted, header_coefficients("kGeluS"))


def test_gelu_16bit_form_accuracy():
    # the degree-5 tail for 16-bit outputs: errors far below the output's own
    # rounding (bf16: 2^-9 relative, fp16: 2^-12) and below 1e-5 of max(1, |x|)
    x = np.linspace(-17.0, 17.0, 1_000_001).astype(np.float32)
    y = gelu_f32_emulated(x, "kGeluS").astype(np.float64)
    x64 = x.astype(np.float64)
    ref = 0.5 * x64 * erfc(-x64 / np.sqrt(2.0))
    err = np.abs(y - ref)
    assert np.max(err / np.maximum(1.0, np.abs(x64))) < 2e-6
    mask = np.abs(ref) > 1e-30
    assert np.max(err[mask] / np.abs(ref[mask])) < 4e-5
    # rounded to fp16, every result is the correctly rounded value or its
    # neighbour (one ulp), and 999 in 1000 or more are the correctly rounded one
    y16 = y.astype(np.float16) + np.float16(0)  # -0 -> +0
    r16 = ref.astype(np.float16) + np.float16(0)
    ulps = np.abs(y16.view(np.int16).astype(np.int64) - r16.view(np.int16).astype(np.int64))
    same_sign = np.sign(y16) == np.sign(r16)
    assert np.all(ulps[same_sign] <= 1)
    assert np.mean(ulps != 0) < 2e-3


def test_gelu_accuracy_dense_grid():
    x = np.linspace(-17.0, 17.0, 1_000_001).astype(np.float32)
    y = gelu_f32_emulated(x).astype(np.float64)
    x64 = x.astype(np.float64)
    ref = 0.5 * x64 * erfc(-x64 / np.sqrt(2.0))  # x Phi(x) without the 1 + erf cancellation
    err = np.abs(y - ref)
    # absolute: a few float32 ulps of max(1, |x|)
    assert np.max(err / np.maximum(1.0, np.abs(x64))) < 2.5e-7
    # relative, also in the lower tail down to the float32 normal range
    mask = np.abs(ref) > 1e-30
    assert np.max(err[mask] / np.abs(ref[mask])) < 2e-5
    mid = np.abs(x64) < 5.0
    assert np.max(err[mid & mask] / np.abs(ref[mid & mask])) < 2e-6


def test_gelu_special_values():
    x = np.array([0.0, -0.0, np.inf, -np.inf, 1e-30, -1e-30, 16.0, -16.0, 40.0, -40.0], dtype=np.float32)
    y = gelu_f32_emulated(x)
    assert y[0] == 0.0 and y[1] == 0.0
    assert y[2] == np.inf and y[3] == 0.0
    np.testing.assert_allclose(y[4:6], 0.5 * x[4:6], rtol=1e-6)
    assert y[8] == np.float32(40.0) and y[9] == 0.0


def test_gelu_against_oracle_epilogue():
    rng = np.random.default_rng(7)
    y = rng.normal(scale=4.0, size=(64, 48))
    bias = rng.normal(size=48)
    ref = oracle.bias_act(y, bias, "bsf", "gelu")
    v = (y + bias).astype(np.float32)  # the kernel adds the bias in fp32
    got = gelu_f32_emulated(v).astype(np.float64)
    assert np.max(np.abs(got - ref)) / np.max(np.abs(ref)) < 1e-6
