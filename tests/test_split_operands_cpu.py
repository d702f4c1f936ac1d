"""The split-operand arithmetic of the float32 matrix-core prefill, on the CPU.

A float32 operand a is carried as two bfloat16 numbers, hi = bf16(a) and
lo = bf16(a - hi), and a product a*b as hi_a hi_b + hi_a lo_b + lo_a hi_b,
each partial product exact in float32 (8 x 8 significant bits) and summed in
float32.  The state bound for such a path (oracle.metrics.state_tol
"split") rests on two facts shown here on random operands: |a - hi - lo| is
at most u^2 |a| with u = 2^-8, and the three-term product is within 3 u^2
|a b| (+ float32 rounding) of a b.  bfloat16 rounding is written out here as
round-to-nearest-even on the upper 16 bits of the float32 pattern.
"""
import numpy as np

from oracle import metrics as me

U = 2.0 ** -8


def bf16(a):
    """float32 -> nearest bfloat16 (ties to even), as float32."""
    b = np.asarray(a, np.float32).view(np.uint32).astype(np.uint64)
    r = (b + 0x7FFF + ((b >> 16) & 1)) >> 16 << 16
    return r.astype(np.uint32).view(np.float32)


def split(a):
    a = np.asarray(a, np.float32)
    hi = bf16(a)
    return hi, bf16(np.float32(a - hi))


def test_bf16_rounding_hand_values():
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: to even (1); 1 + 3*2^-8 rounds up
    x = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, -2.5, 3.0e-3], np.float32)
    np.testing.assert_array_equal(bf16(x), np.array([1.0, 1.0, 1 + 2 ** -6, -2.5, bf16(3.0e-3)], np.float32))
    assert abs(bf16(np.float32(3.0e-3)) - 3.0e-3) <= U * 3.0e-3  # (relative rounding error at most u)


def test_split_holds_operand_to_u_squared():
    rng = np.random.default_rng(7)
    a = (rng.standard_normal(200000) * np.exp(rng.uniform(-20, 20, 200000))).astype(np.float32)
    hi, lo = split(a)
    rest = np.abs(a.astype(np.float64) - hi - lo)
    assert np.all(rest <= U * U * np.abs(a.astype(np.float64)))
    # a single bfloat16 rounding is far coarser: the split is needed
    assert np.max(np.abs(a.astype(np.float64) - hi) / np.abs(a)) > 100 * U * U


def test_three_products_within_bound():
    rng = np.random.default_rng(8)
    a = rng.standard_normal(200000).astype(np.float32)
    b = rng.standard_normal(200000).astype(np.float32)
    ah, al = split(a)
    bh, bl = split(b)
    f32 = np.float32
    prod = f32(f32(f32(ah * bh) + f32(ah * bl)) + f32(al * bh))
    exact = a.astype(np.float64) * b.astype(np.float64)
    err = np.abs(prod.astype(np.float64) - exact) / np.abs(exact)
    assert np.max(err) <= 3 * U * U + 3 * 2.0 ** -24
    # the per-term part of the state bound is twice this first-order term
    assert me.state_tol("split", 1, 64, 2) >= 2 * 3 * U * U
