"""Pins of the oracle's grouped codes (Sec. 3.1, Eq. (3); symmetric control).

The paper prints no worked example of coding, so these pins come from the
closed form and from properties any correct coder must have: hand-worked
groups (including half-way ties), the range of codes, where the extremes
land, the s/2 reconstruction bound, a brute-force nearest-level search, and
exact recovery of values on the quantization grid.
"""
import numpy as np
import pytest

import oracle

F32_1E8 = np.float32(1e-8)


def recon_affine(codes, s, z):
    return codes.astype(np.float64) * np.float64(s) + np.float64(z)


def recon_sym(codes, s, bits):
    return (codes.astype(np.float64) - 2 ** (bits - 1)) * np.float64(s)


# ------------------------------------------------------------------ affine

def test_affine_tie_example_two_bit():
    # s = (3 - 0) / 3 = 1; (x - 0) / 1 = [0, .5, 1.5, 3] -> half-to-even [0, 0, 2, 3]
    codes, s, z = oracle.quant_affine([0.0, 0.5, 1.5, 3.0], 2)
    assert s == np.float32(1.0) and z == np.float32(0.0)
    assert codes.tolist() == [0, 0, 2, 3]


def test_affine_tie_example_four_bit_with_offset():
    # min = -2, s = 30 / 15 = 2; (x + 2) / 2 = [0, 2.5, 3.5, 6.5, 15] -> [0, 2, 4, 6, 15]
    codes, s, z = oracle.quant_affine([-2.0, 3.0, 5.0, 11.0, 28.0], 4)
    assert s == np.float32(2.0) and z == np.float32(-2.0)
    assert codes.tolist() == [0, 2, 4, 6, 15]


def test_affine_constant_group_uses_floor_and_reconstructs_exactly():
    for v in (0.0, 1.25, -3.5e4):
        x = np.full(32, v, dtype=np.float32)
        codes, s, z = oracle.quant_affine(x, 4)
        assert s == F32_1E8
        assert not codes.any()
        assert np.array_equal(recon_affine(codes, s, z), x.astype(np.float64))


def test_affine_floor_applies_to_tiny_ranges():
    x = np.array([1.0, 1.0 + 2 ** -23, 1.0], dtype=np.float32)  # range 1.19e-7 / 15 < 1e-8
    _, s, _ = oracle.quant_affine(x, 4)
    assert s == F32_1E8


def test_affine_signed_zero_offset_is_positive_zero():
    _, _, z = oracle.quant_affine(np.array([-0.0, 0.0, 1.0, 2.0], dtype=np.float32), 2)
    assert np.float32(z).view(np.uint32) == 0


@pytest.mark.parametrize("bits", [2, 4, 8])
@pytest.mark.parametrize("g", [32, 64, 128])
def test_affine_properties_on_random_groups(bits, g):
    rng = np.random.default_rng(bits * 1000 + g)
    top = 2 ** bits - 1
    for trial in range(200):
        scale = 10.0 ** rng.uniform(-3, 3)
        x = (rng.standard_normal(g) * scale + rng.uniform(-5, 5) * scale).astype(np.float32)
        codes, s, z = oracle.quant_affine(x, bits)
        assert codes.min() >= 0 and codes.max() <= top
        assert codes[np.argmin(x)] == 0
        assert codes[np.argmax(x)] == top
        assert z == x.min()
        # scale: the binary32 quotient of the range by 2^b - 1 (within 1 ulp of exact)
        exact = (np.float64(x.max()) - np.float64(x.min())) / top
        assert abs(np.float64(s) - exact) <= 2 * np.spacing(np.float32(exact))
        # reconstruction error bound: |x - xhat| <= s/2 + 4 ulp(max(|x|, |min|))
        xh = recon_affine(codes, s, z)
        ulp = np.spacing(np.maximum(np.abs(x), abs(x.min())).astype(np.float32)).astype(np.float64)
        assert np.all(np.abs(x - xh) <= np.float64(s) / 2 + 4 * ulp)
        # brute force: no other level reconstructs strictly closer (up to rounding slack)
        levels = np.arange(top + 1)[None, :] * np.float64(s) + np.float64(z)
        err = np.abs(x.astype(np.float64)[:, None] - levels)
        chosen = err[np.arange(g), codes]
        assert np.all(chosen <= err.min(axis=1) + 4 * ulp)


@pytest.mark.parametrize("bits", [2, 4])
def test_affine_exact_recovery_on_power_of_two_grid(bits):
    rng = np.random.default_rng(7 + bits)
    top = 2 ** bits - 1
    for e in (-6, 0, 3):
        step = 2.0 ** e
        k = rng.integers(0, top + 1, 64)
        k[0], k[1] = 0, top
        mn = np.float32(rng.integers(-50, 50) * step)
        x = (np.float64(mn) + k * step).astype(np.float32)
        codes, s, z = oracle.quant_affine(x, bits)
        assert s == np.float32(step)
        assert np.array_equal(codes, k.astype(np.uint8))
        assert np.array_equal(recon_affine(codes, s, z), x.astype(np.float64))


# --------------------------------------------------------------- symmetric

def test_symmetric_two_bit_is_ternary():
    # s = max|x| / 1 = 1; round(x / 1) = [-1, 0, 0, 1, 1] (0.5 ties to even 0); u = q + 2
    codes, s = oracle.quant_sym([-1.0, -0.4, 0.5, 0.6, 1.0], 2)
    assert s == np.float32(1.0)
    assert codes.tolist() == [1, 2, 2, 3, 3]


def test_symmetric_four_bit_example_with_ties():
    # qmax = 7, s = 14 / 7 = 2; x / 2 = [-7, -2.5, 0.25, 1.5, 3.5] -> [-7, -2, 0, 2, 4]; u = q + 8
    codes, s = oracle.quant_sym([-14.0, -5.0, 0.5, 3.0, 7.0], 4)
    assert s == np.float32(2.0)
    assert codes.tolist() == [1, 6, 8, 10, 12]


def test_symmetric_zero_group():
    codes, s = oracle.quant_sym(np.zeros(32, dtype=np.float32), 4)
    assert s == F32_1E8
    assert np.all(codes == 8)


@pytest.mark.parametrize("bits", [2, 4, 8])
@pytest.mark.parametrize("g", [32, 128])
def test_symmetric_properties_on_random_groups(bits, g):
    rng = np.random.default_rng(50 + bits + g)
    qmax = 2 ** (bits - 1) - 1
    for trial in range(200):
        x = (rng.standard_t(3, g) * 10.0 ** rng.uniform(-2, 2)).astype(np.float32)
        codes, s = oracle.quant_sym(x, bits)
        assert codes.min() >= 1 and codes.max() <= 2 ** bits - 1
        i = np.argmax(np.abs(x))
        assert codes[i] == (2 ** (bits - 1) + (qmax if x[i] > 0 else -qmax))
        exact = np.float64(np.abs(x).max()) / qmax
        assert abs(np.float64(s) - exact) <= 2 * np.spacing(np.float32(exact))
        xh = recon_sym(codes, s, bits)
        ulp = np.spacing(np.abs(x).max()).astype(np.float64)
        assert np.all(np.abs(x - xh) <= np.float64(s) / 2 + 4 * ulp)
        # mirror symmetry: coding -x reflects every code about 2^(b-1)
        codes_neg, s_neg = oracle.quant_sym(-x, bits)
        assert s_neg == s
        assert np.array_equal(codes_neg.astype(int), 2 ** bits - codes.astype(int))
        levels = np.arange(-qmax, qmax + 1)[None, :] * np.float64(s)
        err = np.abs(x.astype(np.float64)[:, None] - levels)
        chosen = np.abs(x - xh)
        assert np.all(chosen <= err.min(axis=1) + 4 * ulp)
