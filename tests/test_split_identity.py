"""The three-way bf16 split behind the fp32-accurate preconditioning on the bf16
matrix cores (MKOR_GEMM_SPLIT), checked on the CPU with bf16 rounding written
from its definition (oracle/half.py): x = h + m + l exactly, and the three
partial products the kernel leaves out stay below 2^-23 |x x'|."""
import numpy as np

from oracle.half import round_bf16


def split3(x32):
    """h = bf16(x), m = bf16(x - h), l = bf16(x - h - m), each difference taken
    in fp32 (exact, which the asserts below confirm)."""
    x = np.asarray(x32, np.float32).astype(np.float64)
    h = round_bf16(x)
    r = x - h
    assert np.array_equal(r.astype(np.float32).astype(np.float64), r)   # exact in fp32
    m = round_bf16(r)
    s = r - m
    assert np.array_equal(s.astype(np.float32).astype(np.float64), s)
    l = round_bf16(s)
    return h, m, l, s


def _samples(rng, n, emin, emax):
    mant = rng.uniform(1.0, 2.0, n)
    e = rng.integers(emin, emax, n)
    sign = rng.choice([-1.0, 1.0], n)
    return (sign * np.ldexp(mant, e)).astype(np.float32)


def test_split_is_exact_over_the_stated_range():
    rng = np.random.default_rng(0)
    x = _samples(rng, 200_000, -110, 127)
    # plus values at the edges of each binade and exact bf16 values
    x = np.concatenate([x, np.float32([1.0, -1.0, 1.0 + 2.0 ** -23, 2.0 - 2.0 ** -23, 3.0e38, -3.39e38,
                                       2.0 ** -110, 1.5 * 2.0 ** -110, 0.0])])
    h, m, l, s = split3(x)
    assert np.array_equal(l, s)                       # the last piece needs no rounding
    assert np.array_equal(h + m + l, x.astype(np.float64))
    ax = np.abs(x.astype(np.float64))
    assert np.all(np.abs(m) <= 2.0 ** -8 * ax)
    assert np.all(np.abs(l) <= 2.0 ** -16 * ax)


def test_split_limits():
    # below 2^-110 the third piece can fall under bf16's subnormal spacing 2^-133
    x = np.float32(2.0 ** -120 * (1.0 + 2.0 ** -23))
    h, m, l, s = split3([x])
    assert not np.array_equal(l, s)
    # at the bf16 overflow midpoint (2 - 2^-8) 2^127 the first piece becomes infinite
    assert np.isinf(round_bf16([float(np.float32(3.397e38))])[0])
    assert np.isfinite(round_bf16([float(np.float32(3.395e38))])[0])


def test_dropped_products_are_below_one_fp32_rounding():
    rng = np.random.default_rng(1)
    x = _samples(rng, 100_000, -40, 40)
    y = _samples(rng, 100_000, -40, 40)
    hx, mx, lx, _ = split3(x)
    hy, my, ly, _ = split3(y)
    xy = x.astype(np.float64) * y.astype(np.float64)
    kept = hx * hy + hx * my + mx * hy + hx * ly + mx * my + lx * hy
    dropped = mx * ly + lx * my + lx * ly
    assert np.array_equal(kept + dropped, xy)
    assert np.all(np.abs(dropped) <= 2.0 ** -23 * np.abs(xy))
    # with a bf16 operand (G), three products are exact
    g = round_bf16(y)
    assert np.array_equal(hx * g + mx * g + lx * g, x.astype(np.float64) * g)
