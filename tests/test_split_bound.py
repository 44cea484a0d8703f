"""The packed column side's two-part binary16 representation of an fp32
entry: x = v / p (p a power of two at or above the row's bound, so
|x| <= 1) is taken as hi = binary16(x), lo = binary16(x - hi), both rounded
to nearest even.  The stated bound is |x - (hi + lo)| <= max(2^-22 |x|, 2^-25);
x - hi is exact in fp32.  Checked here on the rounding NumPy implements
(IEEE binary16, round to nearest even, the default of the GPU's conversion)
over every binade of fp32 in [-1, 1], subnormal binary16 range included, and
on the power-of-two scaling (exact both ways).
"""
import numpy as np


def split(x32):
    hi = x32.astype(np.float16)
    rest = x32 - hi.astype(np.float32)           # exact in fp32
    lo = rest.astype(np.float16)
    return hi, lo, rest


def test_split_bound_every_binade():
    rng = np.random.default_rng(7)
    e = rng.integers(-40, 1, size=400000)
    m = rng.uniform(0.5, 1.0, size=e.size)
    x = (np.ldexp(m, e) * rng.choice([-1.0, 1.0], size=e.size)).astype(np.float32)
    x = np.concatenate([x, np.float32([1.0, -1.0, 0.0, 2.0 ** -14, 2.0 ** -24, 2.0 ** -25, 0.999999])])
    hi, lo, rest = split(x)
    xd = x.astype(np.float64)
    # the rest is what hi missed, exactly
    assert np.array_equal(rest.astype(np.float64), xd - hi.astype(np.float64))
    err = np.abs(xd - hi.astype(np.float64) - lo.astype(np.float64))
    bound = np.maximum(2.0 ** -22 * np.abs(xd), 2.0 ** -25)
    assert np.all(err <= bound), float(np.max(err / bound))
    # the bound is not loose by more than a factor 2 in either regime
    big = np.abs(xd) >= 2.0 ** -2
    assert np.max(err[big] / np.abs(xd[big])) > 2.0 ** -24
    assert np.max(err[~big]) > 2.0 ** -27


def test_power_of_two_scale_is_exact():
    rng = np.random.default_rng(8)
    v = rng.standard_normal(100000).astype(np.float32) * np.float32(1e3)
    w = np.float32(np.abs(v).max() * 1.3)
    p = np.float32(2.0 ** np.ceil(np.log2(w)))    # the power of two at or above w
    assert p >= w and p < 2 * w
    x = v * (np.float32(1.0) / p)
    assert np.all(np.abs(x) <= 1.0)
    assert np.array_equal(x * p, v)               # back exactly
    hi, lo, _ = split(x)
    rec = (hi.astype(np.float64) + lo.astype(np.float64)) * float(p)
    err = np.abs(rec - v.astype(np.float64))
    assert np.all(err <= np.maximum(2.0 ** -22 * np.abs(v.astype(np.float64)), 2.0 ** -25 * float(p)))
