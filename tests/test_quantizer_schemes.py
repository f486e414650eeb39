"""Exhaustive CPU checks of the two arithmetic shortcuts the matrix-core cache write takes in its
group quantizer, against the IEEE operations the quantizer is specified with (fp32, round to
nearest even; Sec. 5 implementation details, group-wise affine INT2):

* s32 = fp32(range / 3) is formed as a product with c = RN(1/3), then one remainder correction:
      q0 = RN(x c),  r = RN(x - 3 q0) (exact, one FMA),  q = RN(q0 + r c) (one FMA).
  This is Markstein's correction of a quotient estimate by the exact remainder times a correctly
  rounded reciprocal (P. Markstein, "Computation of elementary functions on the IBM RISC
  System/6000 processor", IBM J. Res. Dev. 34(1), 1990; J.-M. Muller et al., Handbook of
  Floating-Point Arithmetic, ch. on division with FMA). The theorem needs side conditions, so the
  scheme is checked here for every fp32 significand (2^23 of them, one binade; both products scale
  by powers of two, so every binade whose intermediates stay normal behaves alike) plus random
  exponents down to the 2^-100 bound below which the kernel divides instead.
* inv = fp32(1 / s) for an fp16 scale s is read from a table of the correctly rounded reciprocals
  of the 1024 normal fp16 significands and scaled by 2^(15 - e): checked for every normal fp16 s.

The FMA is emulated exactly with fp64 and an error-free transformation (no fp32 FMA in numpy).
"""
import numpy as np

C3 = np.float32(float.fromhex("0x1.555556p-2"))  # RN(1/3) in fp32


def _round_exact_to_f32(s: np.ndarray, e: np.ndarray) -> np.ndarray:
    """RN32(s + e) where s = RN64(s + e) and e is the exact fp64 rounding error (TwoSum).

    RN32(RN64(v)) equals RN32(v) unless RN64(v) is exactly an fp32 midpoint (rounding is monotone
    and fp32 midpoints are fp64 numbers); there the sign of e decides, e = 0 keeps the tie."""
    t = s.astype(np.float32)
    td = t.astype(np.float64)
    other = np.nextafter(t, np.where(td < s, np.float32(np.inf), np.float32(-np.inf)))
    od = other.astype(np.float64)
    mid = (td + od) * 0.5  # exact: two adjacent fp32 numbers
    is_mid = (s == mid) & (td != s)
    up = np.maximum(t, other)
    dn = np.minimum(t, other)
    res = np.where(is_mid & (e > 0), up, np.where(is_mid & (e < 0), dn, t))
    return res.astype(np.float32)


def _two_sum(a: np.ndarray, b: np.ndarray):
    s = a + b
    bb = s - a
    err = (a - (s - bb)) + (b - bb)
    return s, err


def div3_scheme(x: np.ndarray) -> np.ndarray:
    x = x.astype(np.float32)
    q0 = (x * C3).astype(np.float32)  # numpy fp32 product: RN
    # r = fma(-q0, 3, x): x - 3 q0 is exact in fp64 (3 q0 has 26 significant bits, the difference is
    # tiny relative to x), so one conversion gives the FMA's single rounding
    r = (x.astype(np.float64) - 3.0 * q0.astype(np.float64)).astype(np.float32)
    # q = fma(r, c, q0): r c is exact in fp64 (24 x 24 bits); the sum is rounded with TwoSum's error
    rc = r.astype(np.float64) * C3.astype(np.float64)
    s, err = _two_sum(q0.astype(np.float64), rc)
    return _round_exact_to_f32(s, err)


def test_emulated_fma_rounding_matches_exact_arithmetic():
    """The emulation itself against exact rational arithmetic on a few thousand values."""
    from fractions import Fraction
    rng = np.random.default_rng(7)
    x = (1.0 + rng.random(3000)).astype(np.float32)
    got = div3_scheme(x)
    for xi, gi in zip(x[:3000], got[:3000]):
        q0 = np.float32(xi * C3)
        r_exact = Fraction(float(xi)) - 3 * Fraction(float(q0))
        r = np.float32(float(r_exact))  # exact fraction -> nearest fp64 -> fp32 (r_exact fits fp64)
        assert Fraction(float(r_exact)) == r_exact
        v = Fraction(float(q0)) + Fraction(float(r)) * Fraction(float(C3))
        lo = np.float32(float(v))
        # nearest fp32 to v, ties to even, by exact comparison with both neighbours
        cands = {lo, np.nextafter(lo, np.float32(np.inf)), np.nextafter(lo, np.float32(-np.inf))}
        best = min(cands, key=lambda c: (abs(Fraction(float(c)) - v), int(np.float32(c).view(np.uint32)) & 1))
        assert gi == best


def test_div3_scheme_is_correctly_rounded_for_every_significand():
    sig = np.arange(1 << 23, dtype=np.uint32) | np.uint32(127 << 23)  # [1, 2)
    x = sig.view(np.float32)
    got = div3_scheme(x)
    ref = x / np.float32(3.0)  # IEEE fp32 division, RN
    bad = np.flatnonzero(got.view(np.uint32) != ref.view(np.uint32))
    assert bad.size == 0, f"{bad.size} significands misrounded, first x = {x[bad[:4]]}"


def test_div3_scheme_over_exponents():
    """Random significands at every exponent from 2^-100 up to the top of fp32, and zero."""
    rng = np.random.default_rng(11)
    exps = np.arange(-100, 127)
    m = rng.integers(0, 1 << 23, size=(exps.size, 2048), dtype=np.uint32)
    x = ((m | np.uint32(127 << 23)).view(np.float32) * np.ldexp(np.float32(1), exps)[:, None]).astype(np.float32)
    x = np.concatenate([x.ravel(), np.float32([0.0, 3.0, 1.5, float.fromhex("0x1.fffffep127")])])
    got = div3_scheme(x)
    ref = x / np.float32(3.0)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_reciprocal_table_scheme_for_every_normal_fp16_scale():
    m = np.arange(1024)
    tab = (np.float32(1.0) / (np.float32(1.0) + m.astype(np.float32) * np.float32(2.0 ** -10))).astype(np.float32)
    for e16 in range(1, 31):
        bits = ((e16 << 10) | m).astype(np.uint16)
        s = bits.view(np.float16).astype(np.float32)
        ref = (np.float32(1.0) / s).astype(np.float32)
        got = np.ldexp(tab, 15 - e16).astype(np.float32)
        assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), f"exponent field {e16}"
