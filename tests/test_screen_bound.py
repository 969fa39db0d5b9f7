"""The error bound the fp8 similarity screen of luffy_condense relies on.

The screen multiplies E4M3 copies of the unit rows scaled by 2^8 and
decides a pair from that product only when it lies farther from 2^16 h than
2^16 (rho_a + rho_b + rho_a rho_b), rho = |x_n - x^| / |x_n| the row's
quantisation error.  These tests check, with an E4M3 rounding written here
from the format's definition (1 sign, 4 exponent bits of bias 7, 3 mantissa
bits, largest finite 448, smallest normal 2^-6; values below 2^-6 stored as
0 as the kernel does), that every pair's fp8 estimate is within that bound
of its cosine, on rows shaped to stress it.  The GPU tests check that the
hardware conversion and the MFMA agree with it (screened and all-bf16
calls give the same graph)."""
import numpy as np
import pytest


def e4m3(v):
    """Round to E4M3 (ties to even); |v| < 2^-6 -> 0; |v| <= 448 assumed."""
    v = np.asarray(v, dtype=np.float64)
    a = np.abs(v)
    out = np.zeros_like(v)
    nz = a >= 2.0 ** -6
    e = np.floor(np.log2(a[nz]))
    step = 2.0 ** (e - 3)
    q = np.round(a[nz] / step) * step          # numpy rounds half to even
    out[nz] = np.sign(v[nz]) * q
    return out


def test_e4m3_model():
    assert e4m3(448.0) == 448.0
    assert e4m3(2.0 ** -6) == 2.0 ** -6
    assert e4m3(0.9 * 2.0 ** -6) == 0.0
    assert e4m3(1.0625) == 1.0          # tie between 1.0 and 1.125 -> even
    assert e4m3(1.1875) == 1.25         # tie between 1.125 and 1.25 -> even
    assert e4m3(-3.3) == -3.25
    assert e4m3(300.0) == 288.0         # spacing 32 in [256, 448]
    # relative error of a normal value is at most 2^-4
    v = np.random.default_rng(0).uniform(2.0 ** -6, 448.0, 100000)
    assert np.max(np.abs(e4m3(v) - v) / v) <= 2.0 ** -4


def quantise(x):
    """The screen's rows: x_n = x / |x| * 256 and its E4M3 copy, and rho."""
    xn = x / np.linalg.norm(x, axis=1, keepdims=True) * 256.0
    xh = e4m3(xn)
    rho = np.linalg.norm(xn - xh, axis=1) / np.linalg.norm(xn, axis=1)
    return xn, xh, rho


def _rows(kind, n, d, rng):
    if kind == "gaussian":
        return rng.standard_normal((n, d))
    if kind == "clustered":
        c = rng.standard_normal((4, d))
        return c[rng.integers(0, 4, n)] + 0.05 * rng.standard_normal((n, d))
    if kind == "heavy":
        return rng.standard_t(2.0, (n, d))
    if kind == "spiky":          # a few large entries, many tiny ones (flushed)
        x = 1e-4 * rng.standard_normal((n, d))
        idx = rng.integers(0, d, (n, 3))
        for i in range(n):
            x[i, idx[i]] = rng.standard_normal(3) * 10
        return x
    if kind == "antiparallel":   # pairs with cosines near -1, 0 and 1
        b = rng.standard_normal((n // 2, d))
        return np.concatenate([b, -b + 1e-3 * rng.standard_normal((n // 2, d))])
    raise ValueError(kind)


@pytest.mark.parametrize("kind", ["gaussian", "clustered", "heavy", "spiky", "antiparallel"])
def test_estimate_within_bound(kind):
    rng = np.random.default_rng(1)
    x = _rows(kind, 96, 2048, rng)
    xn, xh, rho = quantise(x)
    cos = (xn @ xn.T) / 65536.0
    est = (xh @ xh.T) / 65536.0
    bound = rho[:, None] + rho[None, :] + rho[:, None] * rho[None, :]
    err = np.abs(est - cos)
    assert np.all(err <= bound * (1 + 1e-12) + 1e-12), float((err - bound).max())
    # the bound is not loose by orders of magnitude (rho of a dense row is
    # about 2^-4 / sqrt(12) ~ 0.02)
    if kind in ("gaussian", "clustered"):
        assert 0.01 < rho.mean() < 0.04
        assert err.max() > 0.02 * bound.max()


def test_decided_pairs_match_exact_threshold():
    """Pairs outside the band take the exact comparison's side of h."""
    rng = np.random.default_rng(2)
    d = 2048
    u = rng.standard_normal(d)
    s = rng.uniform(0.15, 0.55, (128, 1))
    x = u + s * rng.standard_normal((128, d))
    xn, xh, rho = quantise(x)
    cos = (xn @ xn.T) / 65536.0
    est = (xh @ xh.T) / 65536.0
    h = 0.9
    band = 2 * rho.max() + rho.max() ** 2
    decided = np.abs(est - h) >= band
    assert decided.any() and (~decided).any()
    assert np.array_equal((est >= h)[decided], (cos >= h)[decided])
