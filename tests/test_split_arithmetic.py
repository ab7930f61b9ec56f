"""The float32 path's product arithmetic (no GPU): every float32 value is split
into three bf16 terms hi + mid + lo (round to nearest even at each step) and
a product is taken from the six terms lo.hi + hi.lo + mid.mid + mid.hi +
hi.mid + hi.hi.  Pinned here against exact arithmetic:

* the split is exact (hi + mid + lo == x) over the float32 range the path
  meets, and each term fits bf16 (8 significant bits);
* the six-term product is within 2^-23 |x||y| of x y (the dropped terms
  mid.lo + lo.mid + lo.lo), i.e. at the size of one float32 rounding;
* a length-3072 dot product from six-term products summed in float32 is as
  close to the exact value as a plain float32 dot product.
"""
import numpy as np

from helpers import bf16_round


def split3(x):
    x = np.asarray(x, dtype=np.float32)
    hi = bf16_round(x)
    r = (x.astype(np.float64) - hi).astype(np.float32)
    assert np.array_equal(r.astype(np.float64), x.astype(np.float64) - hi)   # exact residual
    mid = bf16_round(r)
    r2 = (r.astype(np.float64) - mid).astype(np.float32)
    assert np.array_equal(r2.astype(np.float64), r.astype(np.float64) - mid)
    lo = bf16_round(r2)
    return hi, mid, lo


def significant_bits(v):
    m, _ = np.frexp(np.abs(v[v != 0]))
    scaled = m * 2.0 ** 8
    return np.all(scaled == np.round(scaled))


def test_split_is_exact():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(200000), rng.standard_normal(20000) * 1e-20,
                        rng.standard_normal(20000) * 1e20, [0.0, 1.0, -3.5]]).astype(np.float32)
    hi, mid, lo = split3(x)
    assert np.array_equal(hi + mid + lo, x.astype(np.float64))
    for t in (hi, mid, lo):
        assert significant_bits(t)
    nz = x != 0
    assert np.all(np.abs(lo[nz]) <= 2.0 ** -16 * np.abs(x[nz]))


def six_term(x, y):
    xh, xm, xl = split3(x)
    yh, ym, yl = split3(y)
    return xl * yh + xh * yl + xm * ym + xm * yh + xh * ym + xh * yh


def test_six_term_product_bound():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(500000).astype(np.float32)
    y = (rng.standard_normal(500000) * 3.0).astype(np.float32)
    exact = x.astype(np.float64) * y.astype(np.float64)
    err = np.abs(six_term(x, y) - exact)
    assert np.all(err <= 2.0 ** -23 * np.abs(exact) * (1 + 1e-6))
    # and the bound is attained to within a factor of a few: the dropped terms matter
    assert err.max() > 2.0 ** -27 * np.abs(exact).max()


def test_dot_product_as_accurate_as_float32():
    rng = np.random.default_rng(2)
    d = 3072
    worst_split, worst_f32 = 0.0, 0.0
    for _ in range(40):
        x = rng.standard_normal(d).astype(np.float32)
        mu = rng.standard_normal(d).astype(np.float32)
        exact = float(np.dot(x.astype(np.float64), mu.astype(np.float64)))
        scale = float(np.dot(np.abs(x).astype(np.float64), np.abs(mu).astype(np.float64)))
        # float32 accumulation of the six-term products, in a fixed order
        acc = np.float32(0.0)
        for t in six_term(x, mu).astype(np.float32):
            acc = np.float32(acc + t)
        f32 = np.float32(0.0)
        for a, b in zip(x, mu):
            f32 = np.float32(f32 + np.float32(a * b))
        worst_split = max(worst_split, abs(float(acc) - exact) / scale)
        worst_f32 = max(worst_f32, abs(float(f32) - exact) / scale)
    assert worst_split <= 2.0 * worst_f32 + 2.0 ** -22
