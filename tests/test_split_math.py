"""Host-side pins of the arithmetic the conv kernel relies on to carry fp32
weights through 16-bit matrix cores (checked with numpy's IEEE float16 and
a bf16 rounding written out here; no GPU):

* the spike operand's fp16 bits for 1.0 (0x3C00) read as bf16 are exactly 2^-7;
* two fp16 terms: with E the exponent of the layer's largest |w| and
  v = w * 2^(12 - E), every w with |w| >= 2^(E - 15) satisfies
  |v - hi - lo| <= 2^-22 |v| for hi = fp16(v), lo = fp16(v - hi);
* two bf16 terms: with v = w * 2^(60 - max(E, -60)), hi = bf16(v),
  lo = bf16(v - hi) satisfy |v - hi - lo| <= 2^-17 |v| for every float32 w
  of the layer with |w| >= 2^(E - 156) (every float32 when the largest |w|
  is below 2^8), v - hi is exact in float32, each term is zero or a normal
  bf16 even after the spike's 2^-7, and every v of at most 17 significant
  bits is carried exactly.
"""
import numpy as np
import pytest


def bf16_round(x):
    """float32 -> nearest bf16 (ties to even), returned as float32."""
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32)


def exponent(x):
    return np.frexp(np.float64(x))[1] - 1


def layer_samples(g, E, n=200000):
    """Weights of a layer whose largest |w| has exponent E: the maximum itself,
    values spread over the whole float32 range below it, subnormals and zeros."""
    mx = np.float32(np.ldexp(1.0 + g.random(), E))
    e = g.integers(-149, E + 1, n)
    w = np.ldexp(1.0 + g.random(n), e).astype(np.float32)
    w = np.minimum(w, mx)
    w[:8] = [mx, 0.0, np.float32(2.0 ** -149), np.float32(2.0 ** -126), np.float32(np.ldexp(1.0, E)),
             np.float32(np.nextafter(mx, 0, dtype=np.float32)), np.float32(1e-40), np.float32(3e-39)]
    return w, mx


def test_spike_bits_as_bf16():
    one = np.array([1.0], np.float16).view(np.uint16)[0]
    assert one == 0x3C00
    as_bf16 = np.array([np.uint32(one) << 16], np.uint32).view(np.float32)[0]
    assert as_bf16 == np.float32(2.0 ** -7)


@pytest.mark.parametrize("E", [-100, -30, -1, 0, 5, 40, 100])
def test_two_fp16_terms_within_2_pow_minus_22(E):
    g = np.random.default_rng(E + 1000)
    w, mx = layer_samples(g, E)
    assert exponent(mx) == E
    keep = np.abs(w) >= np.float32(np.ldexp(1.0, E - 15))
    v = (w[keep].astype(np.float64) * 2.0 ** (12 - E)).astype(np.float32)
    assert np.all(v == w[keep].astype(np.float64) * 2.0 ** (12 - E))  # the scaling is exact
    hi = v.astype(np.float16)
    rest = v - hi.astype(np.float32)
    assert np.all(rest.astype(np.float64) == v.astype(np.float64) - hi.astype(np.float64))  # exact in float32
    lo = rest.astype(np.float16)
    err = np.abs(v.astype(np.float64) - hi.astype(np.float64) - lo.astype(np.float64))
    assert np.all(err <= 2.0 ** -22 * np.abs(v.astype(np.float64)))
    assert np.all(np.isfinite(hi)) and np.abs(v).max() < 2.0 ** 13


def layer_or_subnormals(g, E):
    """A layer of subnormals only (E < -126), else layer_samples restricted to
    |w| >= 2^(E - 156); returns the weights and the largest one's exponent."""
    if E < -126:
        w = np.arange(1, 200001, dtype=np.uint32).view(np.float32) if E == -149 else \
            g.integers(1, 1 << 23, 200000).astype(np.uint32).view(np.float32)
        return w, exponent(np.abs(w).max())
    w, mx = layer_samples(g, E)
    w = w[np.abs(w) >= np.float32(np.ldexp(1.0, E - 156))] if E - 156 > -149 else w
    return w, E


def bf16_split(w, E):
    s = 60 - max(E, -60)
    v64 = w.astype(np.float64) * 2.0 ** s
    v = v64.astype(np.float32)
    assert np.all(v.astype(np.float64) == v64)  # exact scaling, no overflow
    assert np.abs(v).max() < 2.0 ** 61
    hi = bf16_round(v)
    r1 = v - hi
    assert np.all(r1.astype(np.float64) == v64 - hi.astype(np.float64))  # v - hi exact in float32
    return v64, hi, bf16_round(r1)


@pytest.mark.parametrize("E", [-149, -127, -100, -61, -60, -1, 0, 61, 127])
def test_two_bf16_terms_within_2_pow_minus_17(E):
    g = np.random.default_rng(E + 2000)
    w, E = layer_or_subnormals(g, E)
    v64, hi, lo = bf16_split(w, E)
    err = np.abs(v64 - hi.astype(np.float64) - lo.astype(np.float64))
    assert np.all(err <= 2.0 ** -17 * np.abs(v64))
    for t in (hi, lo):
        a = np.abs(t[t != 0]).astype(np.float64)
        # normal after the spike's 2^-7 as well, so that no flush to zero can touch a product
        assert np.all(a * 2.0 ** -7 >= 2.0 ** -126)


def test_two_bf16_terms_bound_is_attained_closely():
    # the bound is not loose: a significand 1.0000000 1 0000000 0 1 (bits 0, 8
    # and 17 below the leading one) loses its last bit, 2^-17 of the binade
    w = np.array([1.0 + 2.0 ** -8 + 2.0 ** -17], np.float32)
    v64, hi, lo = bf16_split(w, 0)
    err = abs(v64[0] - float(hi[0]) - float(lo[0]))
    assert err > 0 and err <= 2.0 ** -17 * abs(v64[0])


def test_two_bf16_terms_exact_up_to_17_bits():
    # every significand of at most 17 bits, at several binades: hi + lo == v
    g = np.random.default_rng(2100)
    m = np.concatenate([np.arange(1 << 16, 1 << 17), g.integers(1 << 16, 1 << 17, 50000)]).astype(np.float64)
    for e in (-120, -60, -17, 0, 20):  # normal floats: 17 bits need e >= -126
        w = np.ldexp(m, e - 16).astype(np.float32)
        assert np.all(w.astype(np.float64) == np.ldexp(m, e - 16))
        E = exponent(np.abs(w).max())
        v64, hi, lo = bf16_split(w, E)
        assert np.all(hi.astype(np.float64) + lo.astype(np.float64) == v64)
