"""The exact three-part bf16 split behind the bf16 matrix-core path, checked
in numpy on the CPU (no GPU code is run here; the GPU path itself is checked
against the oracle by the -m gpu tests).

Claims checked, for float32 x: with RNE rounding to bf16 at each step,
h = bf16(x), m = bf16(x - h), l = bf16(x - h - m), the two subtractions are
exact in float32, l equals x - h - m exactly (so x = h + m + l), and
|m| <= 2^-8 |x|, |l| <= 2^-16 |x| (up to one rounding). For a product x y,
the six kept part products (hh, hm, mh, mm, hl, lh) miss the exact product
by less than 2^-23 |x y|.
"""

import numpy as np


def bf16_rne(x: np.ndarray) -> np.ndarray:
    """Round float32 to the nearest bfloat16 (ties to even), returned as float32."""
    b = x.astype(np.float32).view(np.uint32)
    lsb = (b >> 16) & 1
    r = (b + 0x7FFF + lsb) & 0xFFFF0000
    return r.astype(np.uint32).view(np.float32)


def split3(x: np.ndarray):
    x = x.astype(np.float32)
    h = bf16_rne(x)
    r = (x - h).astype(np.float32)
    m = bf16_rne(r)
    s = (r - m).astype(np.float32)
    l = bf16_rne(s)
    return h, m, l, r, s


def _samples(n, seed):
    g = np.random.default_rng(seed)
    mant = g.uniform(1.0, 2.0, n)
    expo = g.integers(-100, 100, n)
    sign = np.where(g.random(n) < 0.5, -1.0, 1.0)
    x = (sign * mant * np.exp2(expo)).astype(np.float32)
    # values whose low bits sit right at the rounding points
    b = g.integers(0, 2**31 - 2**24, n // 4, dtype=np.int64).astype(np.uint32)
    b = (b & 0xFFFF0000) | np.array([0x8000, 0x7FFF, 0x8001, 0x0001], np.uint32)[g.integers(0, 4, b.size)]
    return np.concatenate([x, b.view(np.float32)[np.isfinite(b.view(np.float32))]])


def test_split_is_exact():
    x = _samples(400_000, 1)
    x = x[np.abs(x) > 2.0**-100]            # keep the residuals normal in float32
    h, m, l, r, s = split3(x)
    x64, h64, m64, l64 = (v.astype(np.float64) for v in (x, h, m, l))
    assert np.array_equal(r.astype(np.float64), x64 - h64), "x - h is not exact"
    assert np.array_equal(s.astype(np.float64), x64 - h64 - m64), "x - h - m is not exact"
    assert np.array_equal(l, s), "the last part is not a bf16 value"
    assert np.array_equal(h64 + m64 + l64, x64), "h + m + l != x"
    for v in (h, m, l):                      # each part is a bf16 value
        assert np.all((v.view(np.uint32) & 0xFFFF) == 0)
    ax = np.abs(x64)
    assert np.all(np.abs(m64) <= ax * 2.0**-8 * (1 + 2.0**-7))
    assert np.all(np.abs(l64) <= ax * 2.0**-16 * (1 + 2.0**-6))


def test_six_products_bound():
    g = np.random.default_rng(2)
    x = _samples(200_000, 3)
    x = x[(np.abs(x) > 2.0**-60) & (np.abs(x) < 2.0**60)]
    y = x[g.permutation(x.size)]
    hx, mx, lx, _, _ = split3(x)
    hy, my, ly, _, _ = split3(y)
    f = lambda v: v.astype(np.float64)
    kept = (f(hx) * f(hy) + f(hx) * f(my) + f(mx) * f(hy) + f(mx) * f(my) + f(hx) * f(ly) + f(lx) * f(hy))
    exact = f(x) * f(y)
    assert np.all(np.abs(kept - exact) <= 2.0**-23 * np.abs(exact))
    # each kept product of two bf16 values is exact in float32
    for a, b in ((hx, hy), (hx, my), (mx, hy), (mx, my), (hx, ly), (lx, hy)):
        p32 = (a * b).astype(np.float32)
        small = np.abs(f(a) * f(b)) > 2.0**-120
        assert np.array_equal(f(p32)[small], (f(a) * f(b))[small])


def test_dot_product_matches_fp32_error_class():
    """A K = 1,600 dot product through the split (six products, float32
    accumulation) errs no more than a float32 dot product of the same
    values, up to a small factor, against float64."""
    g = np.random.default_rng(4)
    a = g.uniform(0, 2, (64, 1600)).astype(np.float32)        # ReLU outputs
    w = (g.standard_normal((64, 1600)) * 0.03).astype(np.float32)
    ha, ma, la, _, _ = split3(a)
    hw, mw, lw, _, _ = split3(w)
    acc = np.zeros(64, np.float32)
    for p, q in ((ha, hw), (ha, mw), (ma, hw), (ma, mw), (ha, lw), (la, hw)):
        for k in range(0, 1600, 32):         # one matrix-core step: 32 exact products summed
            acc = (acc + (p[:, k:k + 32].astype(np.float64) * q[:, k:k + 32]).sum(1).astype(np.float32)).astype(np.float32)
    ref = (a.astype(np.float64) * w).sum(1)
    f32 = np.zeros(64, np.float32)
    for k in range(1600):
        f32 = (f32 + a[:, k] * w[:, k]).astype(np.float32)
    scale = np.abs(a.astype(np.float64) * w).sum(1)
    err_split = np.abs(acc - ref) / scale
    err_f32 = np.abs(f32 - ref) / scale
    assert err_split.max() < 4 * max(err_f32.max(), 2.0**-24)
