"""The three-part bf16 split behind AMS_F32_X3, checked on the CPU with an
independent bf16 rounding (round to nearest even on the float32 bit pattern):
every float32 x with |x| >= 2^-100 (all three parts then normal numbers)
equals h + m + l exactly, and the six part products the
kernel keeps (hh, hm, mh, hl, lh, mm) differ from x*y by less than 2^-22 |x y|
(the three left out, ml + lm + ll, are bounded by |m| <= 2^-8 |x| and
|l| <= 2^-16 |x|)."""
import numpy as np


def bf16_rne(x: np.ndarray) -> np.ndarray:
    u = x.astype(np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def split3(x):
    x = x.astype(np.float32)
    h = bf16_rne(x)
    r = (x - h).astype(np.float32)            # exact in float32
    m = bf16_rne(r)
    q = (r - m).astype(np.float32)
    l = bf16_rne(q)
    return h, m, l, q


def test_split_is_exact():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(200_000), rng.uniform(-1, 1, 200_000) * 10.0 ** rng.integers(-29, 30, 200_000),
                        [0.0, 1.0, -1.0, 3.0e38, 2.0 ** -100]]).astype(np.float32)
    h, m, l, q = split3(x)
    assert np.array_equal(l, q)                # the last residual needs no rounding
    s = h.astype(np.float64) + m.astype(np.float64) + l.astype(np.float64)
    assert np.array_equal(s, x.astype(np.float64))
    ax = np.abs(x.astype(np.float64))
    assert np.all(np.abs(m) <= 2.0 ** -8 * ax)
    assert np.all(np.abs(l) <= 2.0 ** -16 * ax)


def test_six_products_within_bound():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(500_000).astype(np.float32)
    y = (rng.standard_normal(500_000) * 0.05).astype(np.float32)
    hx, mx, lx, _ = split3(x)
    hy, my, ly, _ = split3(y)
    f = lambda a: a.astype(np.float64)
    six = (f(hx) * f(hy) + f(hx) * f(my) + f(mx) * f(hy) + f(hx) * f(ly) + f(lx) * f(hy) + f(mx) * f(my))
    exact = f(x) * f(y)
    assert np.all(np.abs(six - exact) <= 2.0 ** -22 * np.abs(exact))
    # and the bound is not loose by orders of magnitude: the left-out terms are real
    assert np.max(np.abs(six - exact) / np.maximum(np.abs(exact), 1e-300)) > 2.0 ** -30
