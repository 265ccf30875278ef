"""Arithmetic identities the kernels rely on, checked exhaustively on the host.

- div6: the NV16 kernel forms fl32(amax / 6) -- the argument of the E4M3
  encode of a second-level P scale (Sec. 3.2) -- as q = x * fl32(1/6),
  r = fma(-q, 6, x), fl32(x / 6) = fma(r, fl32(1/6), q).  Scaling x by a power
  of two scales q, r and the result exactly, so checking every fp32 significand
  of one binade covers every exponent where the intermediates stay normal."""
import numpy as np


def fma32(a, b, c):
    """fl32(a * b + c) for float32 arrays: a * b is exact in float64; the float64
    sum may round, so also flag every result whose float64 value lies within that
    rounding error of a float32 midpoint (where a second rounding could differ)."""
    s = a.astype(np.float64) * b.astype(np.float64) + c.astype(np.float64)
    r = s.astype(np.float32)
    ulp = np.spacing(np.abs(r)).astype(np.float64)
    risky = np.abs(np.abs(s - r.astype(np.float64)) - ulp / 2) <= np.abs(s) * 2.0 ** -50
    return r, risky


def test_div6_is_the_correctly_rounded_quotient_on_every_significand():
    x = (np.arange(1 << 23, dtype=np.uint32) | np.uint32(0x3F800000)).view(np.float32)   # every fp32 in [1, 2)
    y = np.float32(1.0) / np.float32(6.0)
    assert y == np.float32(float.fromhex("0x1.555556p-3"))
    q = (x * y).astype(np.float32)
    r, k1 = fma32(-q, np.full_like(x, 6.0), x)
    q2, k2 = fma32(r, np.full_like(x, y), q)
    assert not (k1 | k2).any(), "a float64 sum fell near a float32 midpoint"
    ref = (x / np.float32(6.0)).astype(np.float32)        # IEEE division: correctly rounded
    bad = np.flatnonzero(q2 != ref)
    assert bad.size == 0, "x=%r: %r vs %r" % (float(x[bad[0]]), float(q2[bad[0]]), float(ref[bad[0]]))


def test_div6_planted_mistake_is_caught():
    """The same check with fl32(1/6) rounded the wrong way fails (the pin can fail)."""
    x = (np.arange(1 << 23, dtype=np.uint32) | np.uint32(0x3F800000)).view(np.float32)
    y = np.nextafter(np.float32(1.0) / np.float32(6.0), np.float32(0.0))
    q = (x * y).astype(np.float32)
    r, _ = fma32(-q, np.full_like(x, 6.0), x)
    q2 = (x * y).astype(np.float32)                      # and without the correction step
    assert (q2 != (x / np.float32(6.0))).any()
