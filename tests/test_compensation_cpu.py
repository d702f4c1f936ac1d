"""Why the decode needs compensated sums past 2^24 tokens, shown in float32 on
the CPU, and the float32 arithmetic the compensated decode uses for it.

The degree-0 row of the state sums [v_t, 1] over every token (App. A2), so its
normaliser entry is the token count; a decode step adds exactly 1.0 to it.  In
float32 that addition stops registering at 2^24: from there on the count (and
so every normaliser) falls behind by one per step.  The compensated decode
keeps such entries as a float pair (S, R) updated by exact two-sums (Knuth's
TwoSum), whose value S + R stays exact here.  numpy float32 follows IEEE
round-to-nearest-even, the rounding of the GPU's float32 adds.
"""
import numpy as np

F = np.float32


def two_sum(a, b):
    """s + e = a + b exactly, s = fl(a + b) (Knuth), in float32."""
    s = F(a + b)
    bp = F(s - a)
    e = F(F(a - F(s - bp)) + F(b - bp))
    return s, e


def comp_add(s, r, a):
    """(s, r) += a, then s becomes the rounded pair sum (two two-sums)."""
    t, e = two_sum(s, a)
    r1 = F(r + e)
    u, r2 = two_sum(t, r1)
    return u, r2


def test_float32_count_stops_at_2_pow_24():
    s = F(2 ** 24)
    for _ in range(4096):
        s = F(s + F(1.0))
    assert s == F(2 ** 24)                       # every increment absorbed
    # a normaliser short by 4096 of 2^24 puts y off by 2.4e-4, above the 1e-4 float32 tolerance
    assert 4096 / 2 ** 24 > 1e-4


def test_compensated_pair_keeps_every_increment():
    s, r = F(2 ** 24), F(0.0)
    for _ in range(4096):
        s, r = comp_add(s, r, F(1.0))
    assert float(s) + float(r) == 2 ** 24 + 4096
    assert s == F(2 ** 24 + 4096) and r == 0.0   # the pair sum is representable here


def test_compensated_pair_tracks_fractional_increments():
    """Increments far below the ulp of the sum (the degree-2 normaliser terms of
    a long context): the pair stays within float32 roundoff of the exact sum,
    the plain float32 sum does not."""
    rng = np.random.default_rng(0)
    inc = (rng.standard_normal(20000) ** 2 * 0.25).astype(F)   # ~ k~_i^2 / sqrt(2) at d = 8
    start = F(3.0e6)
    exact = float(start) + float(np.sum(inc.astype(np.float64)))
    s, r = start, F(0.0)
    plain = start
    for a in inc:
        s, r = comp_add(s, r, a)
        plain = F(plain + a)
    assert abs(float(s) + float(r) - exact) <= 1e-12 * exact + 1e-3
    assert abs(float(s) - exact) <= 2.0 ** -24 * exact
    assert abs(float(plain) - exact) > 100 * 2.0 ** -24 * exact
