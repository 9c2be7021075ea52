"""The encoder's integer filter form, checked on the CPU against the oracle.

When every tap is a multiple of 2^-s with |tap| 2^s < 2^15, and KF^2 * 255 *
2^(e + s + 1) < 2^31 (e the largest binary exponent of a tap), every partial
sum of the filter's double accumulation over u8 pixels is a multiple of 2^-s
below 2^31 2^-s, so no sum rounds: the int32 sum of (tap 2^s) * pixel, times
2^-s and rounded once to float, is the definition's value (filter of the
"utils Module", the ky-then-kx double sum and one rounding).  The condition is
restated here as the kernel states it; these tests pin the claim to the
oracle bit for bit and check which banks take the form."""
import math

import numpy as np
import pytest
from scipy.signal import correlate2d

import oracle as orc
import synth

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def exact_form(bank: np.ndarray):
    """(s, True) when the bank takes the integer form, else (None, False)."""
    KF = bank.shape[-1]
    nz = bank[bank != 0].astype(np.float64)
    if nz.size == 0:
        return 0, True
    if not np.all(np.isfinite(nz)):
        return None, False
    frac, emax = 0, -10 ** 9
    for t in nz:
        m, e = math.frexp(abs(t))          # |t| = m 2^e, m in [0.5, 1)
        mant = int(m * (1 << 53))          # exact: float32 taps have 24 bits
        lsb = e - 53 + ((mant & -mant).bit_length() - 1)
        frac = max(frac, -lsb)
        emax = max(emax, e - 1)
    s = frac
    ok = s <= 126 and emax + s <= 14 and (emax + s + 1 < 0 or KF * KF * 255 * 2 ** (emax + s + 1) < 2 ** 31)
    return (s, True) if ok else (None, False)


def integer_filter(img: np.ndarray, bank: np.ndarray, s: int) -> np.ndarray:
    """Exact sums of (tap 2^s) * pixel, zero padding, same size; then 2^-s and
    one rounding to float32."""
    B, H, W = img.shape
    C = bank.shape[0]
    q = np.ldexp(bank.astype(np.float64), s)
    assert np.all(q == np.round(q)) and np.abs(q).max() < 2 ** 15
    q = q.astype(np.int64)
    out = np.empty((B, C, H, W), np.float32)
    for b in range(B):
        for c in range(C):
            acc = correlate2d(img[b].astype(np.int64), q[c], mode="same", boundary="fill", fillvalue=0)
            assert np.abs(acc).max() < 2 ** 31
            out[b, c] = np.ldexp(acc.astype(np.float64), -s).astype(np.float32)
    return out


def test_dog_bank_takes_the_integer_form_and_matches_the_oracle():
    bank = synth.dog_bank()
    s, ok = exact_form(bank)
    assert ok and s == 8
    g = synth.rng(31, 0)
    img = synth.stroke_images(g, 3, 28, 28)
    ref = orc.filter_images(img, bank, -np.inf)
    got = integer_filter(img, bank, s)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_dyadic_positive_bank_matches_with_saturated_pixels():
    g = synth.rng(32, 0)
    bank = (g.integers(1, 65, (4, 3, 3)) / 64.0).astype(np.float32)
    s, ok = exact_form(bank)
    assert ok and s <= 6
    img = np.full((2, 9, 11), 255, np.uint8)
    img[1] = g.integers(0, 256, (9, 11))
    ref = orc.filter_images(img, bank, -np.inf)
    assert np.array_equal(integer_filter(img, bank, s).view(np.uint32), ref.view(np.uint32))


def test_general_float_taps_and_large_sums_take_the_double_form():
    g = synth.rng(33, 0)
    base = (g.normal(0, 1, (3, 5, 5)) * np.exp2(g.integers(-20, 3, (3, 5, 5)))).astype(np.float32)
    assert not exact_form(base)[1]            # 24-bit mantissas over 22 octaves
    assert exact_form(np.full((1, 13, 13), 100.0, np.float32))[1]  # 169 * 255 * 2^7 < 2^31
    big = np.full((1, 31, 31), 16383.0, np.float32)  # each |tap| < 2^15, but 961 * 255 * 2^14 >= 2^31
    assert not exact_form(big)[1]
    wide = np.zeros((1, 3, 3), np.float32)
    wide[0, 1, 1], wide[0, 0, 0] = 1.0, 2.0 ** -20  # 2^20 * 1 >= 2^15
    assert not exact_form(wide)[1]
    assert exact_form(np.zeros((2, 5, 5), np.float32))[1]
