"""Pins of the oracle's quantizers at scales whose reciprocal overflows (a
bucket whose max-norm is subnormal, below 2^-126), and of the bucket-level
quantization under a given scale that the parity harness uses for ties.

Example 1 and the stochastic quantizer divide by the bucket scale
(Section III: Q2(x / Q1(||x||_inf))).  Both are checked here against what the
definitions fix independently of the division's implementation: Example 1
against an exact rational argmin over its levels, the stochastic quantizer
for unbiasedness over a grid of draws and for its levels; zeros in such a
bucket must quantize like zeros anywhere else."""
from fractions import Fraction

import numpy as np
import pytest

import oracle as O

TINY = np.float32(2.0 ** -149)      # the smallest subnormal


def q_(kind, bits=0, scale=O.SCALE_MAX, bucket=256):
    return O.Quant(kind=kind, scale=scale, bits=bits, error_feedback=1, bucket=bucket)


def subnormal_bucket(seed, n=256, top=214):
    """Integer multiples of 2^-149 up to top * 2^-149 (3.0e-43 for 214),
    with zeros and both signs of zero."""
    rng = np.random.default_rng(seed)
    k = rng.integers(-top, top + 1, n)
    k[rng.random(n) < 0.4] = 0
    k[0] = top
    k[1] = 0
    p = (k.astype(np.float64) * 2.0 ** -149).astype(np.float32)
    p[1] = np.float32(-0.0)
    assert np.all(p[k != 0] != 0) and np.abs(p).max() == np.float32(top * 2.0 ** -149)
    return p, k


@pytest.mark.parametrize("k_ex1", [1, 2, 3, 7])
@pytest.mark.parametrize("top", [214, 1, 3, (1 << 23) - 1])
def test_example1_subnormal_scale_is_exact_argmin(k_ex1, top):
    p, kint = subnormal_bucket(k_ex1 * 7 + top, top=top)
    q = q_(O.Q_DET_UNIFORM, k_ex1 + 1, bucket=256)
    codes, deq, s = O.quantize(q, p)
    L = 2 ** k_ex1 - 1
    assert s[0] == np.abs(p).max()
    assert codes.max() <= 2 * L                    # every code is a level of M_2
    zero = kint == 0
    assert np.all(codes[zero] == L) and np.all(deq[zero] == 0)   # Q(0) = 0
    # x/s is the exact rational k/top; the chosen level is a nearest level of
    # i/L to it, ties toward zero, up to the binary32 rounding of x*L
    for j in range(p.size):
        x = Fraction(int(kint[j]), top)
        i = int(codes[j]) - L
        dist = abs(x - Fraction(i, L))
        best = min(abs(x - Fraction(m, L)) for m in range(-L, L + 1))
        assert dist <= best + Fraction(1, 1 << 22), (j, x, i)
        if dist == best:
            continue
        # off the exact nearest only at a half level, and then toward zero
        assert abs(abs(x * L) - (abs(i) + Fraction(1, 2))) <= Fraction(1, 1 << 20)
    # dequantized values are s times the level, exactly representable
    lev = (codes.astype(np.int64) - L).astype(np.float64) / L
    want = (np.float64(s[0]) * lev.astype(np.float32).astype(np.float64)).astype(np.float32)
    assert np.array_equal(deq, want)


@pytest.mark.parametrize("bits", [1, 2, 4, 8])
def test_stochastic_subnormal_scale_is_unbiased(bits):
    p, kint = subnormal_bucket(bits, top=214)
    q = q_(O.Q_STOCH_UNIFORM, bits, O.SCALE_MAX, 256)
    L = 2 ** bits - 1
    K = 2048
    acc = np.zeros(p.size)
    for k in range(K):
        u = np.full(p.size, (k + 0.5) / K, np.float32)
        codes, deq, s = O.quantize(q, p, u=u)
        assert codes.max() <= L
        # on the grid s * (2c - L) / L (as binary32 products)
        lev = ((2.0 * codes - L) / L).astype(np.float32)
        assert np.array_equal(deq, (np.float64(s[0]) * lev.astype(np.float64)).astype(np.float32))
        acc += deq.astype(np.float64)
    mean = acc / K
    sc = float(s[0])
    # E_u[Q(p)] = p up to the draw grid's resolution and the subnormal
    # rounding of each dequantized value (half of 2^-149)
    assert np.all(np.abs(mean - p.astype(np.float64)) <= 2 * sc / L / K + 2.0 ** -149)
    # zeros average to zero
    assert np.all(np.abs(mean[kint == 0]) <= 2 * sc / L / K + 2.0 ** -149)


def test_subnormal_scale_matches_scaled_bucket():
    """The reading for a scale below 2^-126: x and s are multiplied by 2^64
    first.  Codes then equal those of the same bucket scaled by 2^64 (a
    normal-scale bucket), so the subnormal case is no special rule of its
    own; the dequantized values scale back exactly."""
    for bits, kind, scale in ((2, O.Q_DET_UNIFORM, O.SCALE_MAX), (3, O.Q_DET_UNIFORM, O.SCALE_MAX),
                              (2, O.Q_STOCH_UNIFORM, O.SCALE_MAX), (4, O.Q_STOCH_UNIFORM, O.SCALE_MAX)):
        p, _ = subnormal_bucket(bits + 40, top=9999)
        big = (p.astype(np.float64) * 2.0 ** 64).astype(np.float32)
        assert np.array_equal(big.astype(np.float64), p.astype(np.float64) * 2.0 ** 64)   # exact
        q = q_(kind, bits, scale, 256)
        u = np.random.default_rng(bits).random(p.size, dtype=np.float32)
        c1, d1, s1 = O.quantize(q, p, u=u)
        c2, d2, s2 = O.quantize(q, big, u=u)
        assert np.array_equal(c1, c2)
        assert s2[0] == np.float32(float(s1[0]) * 2.0 ** 64)


def test_quantize_bucket_equals_quantize_under_its_own_scale():
    rng = np.random.default_rng(2)
    for qd in (dict(kind=O.Q_SCALED_SIGN, bits=1, scale=O.SCALE_L1), dict(kind=O.Q_STOCH_UNIFORM, bits=4,
               scale=O.SCALE_L2), dict(kind=O.Q_STOCH_UNIFORM, bits=2, scale=O.SCALE_MAX),
               dict(kind=O.Q_DET_UNIFORM, bits=3, scale=O.SCALE_MAX)):
        q = O.Quant(**qd, error_feedback=1, bucket=512)
        p = (rng.standard_t(3, 1500) * 1e-3).astype(np.float32)
        u = rng.random(1500, dtype=np.float32)
        codes, deq, s = O.quantize(q, p, u=u)
        for b in range(3):
            n = min(512, 1500 - 512 * b)
            c, dq = O.quantize_bucket(q, p[512 * b:512 * b + n], float(s[b]), u[512 * b:512 * b + n])
            assert np.array_equal(c, codes[512 * b:512 * b + n])
            assert np.array_equal(dq, deq[512 * b:512 * b + n])
        # under a scale one ulp larger: still a valid quantization of p on the
        # new grid (codes in range, deq = s' * level)
        s2 = np.nextafter(s[0], np.float32(1))
        c, dq = O.quantize_bucket(q, p[:512], float(s2), u[:512])
        assert c.max() < 2 ** O.code_bits(q)
        if qd["kind"] == O.Q_SCALED_SIGN:
            assert np.all(np.abs(dq) == s2)


@pytest.mark.parametrize("k_ex1", [1, 2, 3])
def test_example1_under_a_smaller_scale_takes_the_nearest_level(k_ex1):
    """Under a given scale below the bucket's max-norm (the tie check
    quantizes under another side's scale), x/s leaves [-1, 1]; Example 1's Q2
    still picks the nearest of its levels i/L, i = -L..L, which is +-1 beyond
    them, so every code stays a level of M_2 and |Q(x)| <= s."""
    rng = np.random.default_rng(k_ex1)
    L = 2 ** k_ex1 - 1
    kint = rng.integers(-64, 65, 256)
    kint[0] = 64
    p = kint.astype(np.float32)                     # max-norm 64
    q = q_(O.Q_DET_UNIFORM, k_ex1 + 1, bucket=256)
    s = 16.0                                        # x/s = k/16 exactly, up to 4
    codes, deq = O.quantize_bucket(q, p, s)
    assert codes.max() <= 2 * L and codes.min() >= 0
    assert np.all(np.abs(deq) <= s)
    for j in range(p.size):
        x = Fraction(int(kint[j]), 16)
        i = int(codes[j]) - L
        best = min(abs(x - Fraction(m, L)) for m in range(-L, L + 1))
        d = abs(x - Fraction(i, L))
        # the exact nearest level, or at a half level the one nearer zero
        assert d == best, (j, x, i)
        if abs(x) > 1:
            assert i == (L if x > 0 else -L)
