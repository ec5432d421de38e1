"""The error analysis behind the three-piece bf16 products of the fp32 path
(CPU only): each fp32 value is the exact sum of its three round-to-nearest
bf16 pieces, and the six piece products the kernels take differ from the
exact product by at most 2^-23 of its magnitude.  Checked with an
independent numpy emulation of round-to-nearest-even to bf16 on random
values over a wide exponent range."""
import numpy as np


def bf16_rne(x):
    """Round float32 values to the nearest bf16 (ties to even), as float32."""
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return r.astype(np.uint32).view(np.float32)


def pieces(a):
    a = np.asarray(a, np.float32)
    p0 = bf16_rne(a)
    r1 = (a - p0).astype(np.float32)
    p1 = bf16_rne(r1)
    r2 = (r1 - p1).astype(np.float32)
    p2 = bf16_rne(r2)
    return p0, p1, p2


def _values(rng, n, emax=60):
    mant = rng.uniform(1.0, 2.0, n) * rng.choice([-1.0, 1.0], n)
    return (mant * 2.0 ** rng.integers(-emax, emax, n)).astype(np.float32)


def test_three_pieces_sum_exactly():
    rng = np.random.default_rng(11)
    a = _values(rng, 200000)
    p0, p1, p2 = pieces(a)
    s = p0.astype(np.float64) + p1.astype(np.float64) + p2.astype(np.float64)
    assert np.array_equal(s, a.astype(np.float64))
    # every piece is a bf16 value, and the pieces shrink by 2^-8 each
    for p in (p0, p1, p2):
        assert np.array_equal(bf16_rne(p), p)
    mag = np.abs(a.astype(np.float64))
    assert np.all(np.abs(p1) <= 2.0 ** -8 * mag)
    assert np.all(np.abs(p2) <= 2.0 ** -16 * mag)


def test_six_products_bound():
    rng = np.random.default_rng(12)
    # exponents kept where no piece product falls below the fp32 normal range
    a, b = _values(rng, 200000, 30), _values(rng, 200000, 30)
    (a0, a1, a2), (b0, b1, b2) = [[p.astype(np.float64) for p in pieces(v)] for v in (a, b)]
    six = a0 * b0 + a0 * b1 + a1 * b0 + a0 * b2 + a1 * b1 + a2 * b0
    exact = a.astype(np.float64) * b.astype(np.float64)
    rel = np.abs(six - exact) / np.abs(exact)
    assert rel.max() <= 2.0 ** -23
    # each piece product is exact in fp32 (8 x 8 significant bits)
    for x, y in ((a0, b0), (a0, b1), (a1, b0), (a0, b2), (a1, b1), (a2, b0)):
        p = x * y
        assert np.array_equal(p.astype(np.float32).astype(np.float64), p)
