"""Pins of the oracle's scalar number-format conversions.

The fp16 residual window (KIVI format, Sec. 3.1) stores binary16 values and
the projection emits bf16; the oracle implements both roundings itself.
They are pinned here against numpy's binary16 conversion (a library
routine) and against exact rational rounding.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle


def test_f32_to_f16_matches_numpy_on_random_and_edge_values():
    g = np.random.default_rng(0)
    vals = np.concatenate([
        g.standard_normal(4000).astype(np.float32) * s for s in (1e-6, 1e-3, 1.0, 100.0, 3e4)
    ] + [np.array([0.0, -0.0, 65504.0, 65519.996, 65520.0, 70000.0, -65520.0,
                   2.0 ** -24, 2.0 ** -25, 3 * 2.0 ** -25, 2.0 ** -14, 2.0 ** -14 - 2.0 ** -26,
                   1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11, np.inf, -np.inf], dtype=np.float32)])
    ours = oracle.f32_to_f16(vals)
    ref = vals.astype(np.float16).view(np.uint16)
    assert np.array_equal(ours, ref)


def test_f16_to_f32_exhaustive():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float32)
    finite = np.isfinite(ref) | np.isinf(ref)
    ours = oracle.f16_to_f32(bits[finite])
    assert np.array_equal(ours.view(np.uint32), ref[finite].view(np.uint32))


def _bf16_exact(x: float) -> int:
    """Round a double to bf16 by exact rational arithmetic (ties to even)."""
    if x == 0:
        return 0x8000 if np.signbit(x) else 0
    sign = 0x8000 if x < 0 else 0
    a = Fraction(abs(x))
    e = 0
    while a >= 2:
        a /= 2
        e += 1
    while a < 1:
        a *= 2
        e -= 1
    e = max(e, -126)
    q = Fraction(abs(x)) / Fraction(2) ** (e - 7)
    r = int(q)
    frac = q - r
    if frac > Fraction(1, 2) or (frac == Fraction(1, 2) and r % 2 == 1):
        r += 1
    if e >= -126 and r >= 128:
        value = r * Fraction(2) ** (e - 7)
        if value >= Fraction(2) ** 128:
            return sign | 0x7F80
        if r == 256:
            return sign | (((e + 1 + 127) << 7))
        return sign | (((e + 127) << 7) + (r - 128))
    return sign | r


def test_f64_to_bf16_matches_exact_rounding():
    g = np.random.default_rng(1)
    vals = list(g.standard_normal(3000) * 10.0 ** g.integers(-30, 30, 3000))
    # exact ties between bf16 neighbours (odd and even significands)
    vals += [1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(2.0 + 2.0 ** -7), 255.5, 256.5 * 2 ** 10]
    vals += [3.0e38, 3.4e38, 1e-40, 2.0 ** -133, 1.5 * 2.0 ** -133]
    ours = oracle.f64_to_bf16(np.array(vals))
    ref = np.array([_bf16_exact(float(v)) for v in vals], dtype=np.uint16)
    assert np.array_equal(ours, ref)


def test_f64_to_bf16_agrees_with_torch_on_float32_inputs():
    g = np.random.default_rng(2)
    x = (g.standard_normal(5000) * 7).astype(np.float32)
    ours = oracle.f64_to_bf16(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


@pytest.mark.parametrize("x", [np.nan])
def test_f16_nan_stays_nan(x):
    assert np.isnan(oracle.f16_to_f32(oracle.f32_to_f16([x]))[0])
