"""Pins of the oracle's Definition 3 compressors (top-k and random-k per
bucket) to what their definitions fix (CPU only).

Top-k is the best k-term approximation: a brute force over every k-subset in
exact rational arithmetic must find no subset with a smaller residual, and the
stated tie rule (lower index first) picks one minimiser.  Definition 3 asks for
||x - Q(x)|| <= (1 - delta) ||x||; top-k meets it with ||x - Q(x)||^2 <=
(1 - k/n) ||x||^2.  Random-k must keep a uniformly random k-subset, which a
chi-square test over counter-based draws checks, and meets the same bound in
expectation with equality.
"""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle as O


def sq(kind, keep, bucket, ef=1):
    return O.Quant(kind=kind, keep=keep, bucket=bucket, error_feedback=ef)


def _exact_residual(x, kept):
    return sum(Fraction(float(x[j])) ** 2 for j in range(len(x)) if j not in kept)


@pytest.mark.parametrize("seed", range(6))
def test_topk_is_best_k_term_approximation(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(3, 10))
    # magnitudes drawn from a small set, so that equal magnitudes (ties) occur
    x = (rng.choice([0.0, 0.25, 0.5, 1.0, 1.5, 3.0], size=n) * rng.choice([-1.0, 1.0], size=n)).astype(np.float32)
    x[rng.integers(0, n)] = float(rng.standard_normal())
    for keep in range(1, n + 2):
        codes, deq, vals = O.quantize(sq(O.Q_TOPK, keep, n), x)
        k = min(keep, n)
        kept = tuple(int(j) for j in np.nonzero(codes)[0])
        assert len(kept) == k
        best = min(_exact_residual(x, set(S)) for S in itertools.combinations(range(n), k))
        minimisers = [S for S in itertools.combinations(range(n), k) if _exact_residual(x, set(S)) == best]
        assert kept == min(minimisers), (x, keep, kept, minimisers)
        assert np.array_equal(deq, np.where(codes == 1, x, np.float32(0)))
        assert np.array_equal(vals[:k], x[list(kept)]) and np.all(vals[k:] == 0)


def test_topk_hand_examples():
    x = np.array([0.5, -3, 2, -2, 1, 0, 7, -7], np.float32)
    codes, deq, vals = O.quantize(sq(O.Q_TOPK, 3, 8), x)
    assert codes.tolist() == [0, 1, 0, 0, 0, 0, 1, 1]
    assert vals.tolist() == [-3.0, 7.0, -7.0]            # index order, not rank order
    assert deq.tolist() == [0, -3, 0, 0, 0, 0, 7, -7]
    # equal magnitudes: the lower indices win
    codes, _, vals = O.quantize(sq(O.Q_TOPK, 2, 4), np.array([1, -1, 1, 0.5], np.float32))
    assert codes.tolist() == [1, 1, 0, 0] and vals.tolist() == [1.0, -1.0]
    # +0 and -0 tie; their signs travel in the values
    codes, _, vals = O.quantize(sq(O.Q_TOPK, 3, 4), np.array([0.0, -0.0, 0.0, 1.0], np.float32))
    assert codes.tolist() == [1, 1, 0, 1]
    assert vals.tolist() == [0.0, 0.0, 1.0] and np.signbit(vals).tolist() == [False, True, False]
    # NaN ranks above infinity, infinity above every finite value
    codes, _, _ = O.quantize(sq(O.Q_TOPK, 1, 3), np.array([np.inf, np.nan, 1.0], np.float32))
    assert codes.tolist() == [0, 1, 0]
    codes, _, _ = O.quantize(sq(O.Q_TOPK, 1, 3), np.array([3e38, -np.inf, 1.0], np.float32))
    assert codes.tolist() == [0, 1, 0]


@pytest.mark.parametrize("n,bucket,keep", [(2048, 512, 16), (1000, 256, 1), (700, 512, 64), (300, 512, 400),
                                           (4096, 2048, 2048)])
def test_topk_definition3_bound(n, bucket, keep):
    rng = np.random.default_rng(n + keep)
    x = (rng.standard_normal(n) * np.exp(rng.standard_normal(n))).astype(np.float32)
    codes, deq, vals = O.quantize(sq(O.Q_TOPK, keep, bucket), x)
    for b0 in range(0, n, bucket):
        xb = x[b0:b0 + bucket].astype(np.float64)
        qb = deq[b0:b0 + bucket].astype(np.float64)
        nb = xb.size
        k = min(keep, nb)
        assert int(codes[b0:b0 + bucket].sum()) == k
        r2, x2 = float(np.sum((xb - qb) ** 2)), float(np.sum(xb ** 2))
        assert r2 <= (1.0 - k / nb) * x2 * (1 + 1e-12)
        # Definition 3 with delta = k / (2n): sqrt(1 - k/n) <= 1 - k/(2n)
        delta = k / (2.0 * nb)
        assert math.sqrt(r2) <= (1 - delta) * math.sqrt(x2) * (1 + 1e-12)
        assert math.sqrt(float(np.sum(qb ** 2))) <= (2 - delta) * math.sqrt(x2) * (1 + 1e-12)
    # the message holds keep values per bucket, zero-padded in a short last bucket
    nb_last = n - (n - 1) // bucket * bucket
    assert vals.size == -(-n // bucket) * keep
    assert np.all(vals[-keep:][min(keep, nb_last):] == 0)


def test_keep_at_least_bucket_is_identity():
    rng = np.random.default_rng(4)
    x = rng.standard_normal(777).astype(np.float32)
    for kind in (O.Q_TOPK, O.Q_RANDK):
        u = O.uniforms(9, 1, 0, 0, x.size)
        codes, deq, vals = O.quantize(sq(kind, 256, 256), x, u=u)
        assert np.all(codes == 1) and np.array_equal(deq, x)
        # buckets of 256, 256, 256, 9: the values are x itself, then zeros
        assert vals.size == 4 * 256
        assert np.array_equal(vals[:777], x) and np.all(vals[777:] == 0)


@pytest.mark.parametrize("kind", [O.Q_TOPK, O.Q_RANDK])
@pytest.mark.parametrize("n,bucket,keep", [(1300, 512, 16), (256, 256, 255), (5000, 1024, 3)])
def test_sparse_dequantize_inverts_the_message(kind, n, bucket, keep):
    rng = np.random.default_rng(keep)
    x = rng.standard_normal(n).astype(np.float32)
    q = sq(kind, keep, bucket)
    u = O.uniforms(3, 5, 2, 0, n)
    codes, deq, vals = O.quantize(q, x, u=u)
    words = O.pack(1, codes)
    assert np.array_equal(O.dequantize(q, O.unpack(1, words, n), vals), deq)


def test_randk_keeps_a_uniformly_random_subset():
    """n = 8, k = 3: each of the 56 subsets has probability 1/56; 11200 steps of
    counter-based draws give 200 expected per subset."""
    n, k, T = 8, 3, 11200
    x = np.arange(1, n + 1, dtype=np.float32)
    q = sq(O.Q_RANDK, k, n)
    counts = {}
    for t in range(1, T + 1):
        codes, deq, _ = O.quantize(q, x, u=O.uniforms(5, t, 0, 0, n))
        S = tuple(int(j) for j in np.nonzero(codes)[0])
        assert len(S) == k
        counts[S] = counts.get(S, 0) + 1
    assert len(counts) == 56
    exp = T / 56
    chi2 = sum((c - exp) ** 2 / exp for c in counts.values())
    assert chi2 < 100.0   # 55 degrees of freedom: P(chi2 > 100) < 2e-4


def test_randk_residual_in_expectation_and_independent_of_x():
    n, keep, T = 512, 32, 400
    rng = np.random.default_rng(7)
    x = rng.standard_normal(n).astype(np.float32)
    y = rng.standard_normal(n).astype(np.float32)
    q = sq(O.Q_RANDK, keep, n)
    r2 = []
    hits = np.zeros(n)
    for t in range(1, T + 1):
        u = O.uniforms(11, t, 4, 0, n)
        cx, dx, _ = O.quantize(q, x, u=u)
        cy, _, _ = O.quantize(q, y, u=u)
        assert np.array_equal(cx, cy)            # the kept set depends on the draws only
        assert u[cx == 1].min() >= u[cx == 0].max()   # and holds the largest draws
        r2.append(float(np.sum((x.astype(np.float64) - dx) ** 2)))
        hits += cx
    x2 = float(np.sum(x.astype(np.float64) ** 2))
    # E ||x - Q(x)||^2 = (1 - k/n) ||x||^2 for a uniform k-subset
    assert abs(np.mean(r2) / x2 - (1 - keep / n)) < 0.01
    # every position is kept with probability k/n: no drift along the bucket
    # (each half of the bucket holds half of the T*k kept elements, within 5 sigma)
    half = hits[: n // 2].sum()
    assert abs(half - T * keep / 2) < 5 * np.sqrt(T * keep / 4)
    quarters = hits.reshape(4, -1).sum(1)
    assert np.all(np.abs(quarters - T * keep / 4) < 5 * np.sqrt(T * keep * 3 / 16))


def test_sparse_segment_equals_slice_of_full_run():
    d, N = 5 * 512 + 100, 2
    qw, qs = sq(O.Q_TOPK, 20, 512), sq(O.Q_RANDK, 7, 256)
    cfg = O.Config(d=d, N=N, placement=O.ADAM_AT_SERVER, beta1=0.9, beta2=0.999, lr=1e-3, eps=1e-8,
                   seed=5, qw=qw, qs=qs)
    rng = np.random.default_rng(2)
    full = O.State.init(cfg, d)
    n0, ln = 1024, 1024 + 100 + 512
    part = O.State.init(cfg, ln)
    for t in range(1, 4):
        g = rng.standard_normal((N, d)).astype(np.float32)
        of = O.step(cfg, t, g, full)
        op = O.step(cfg, t, np.ascontiguousarray(g[:, n0:]), part, n0=n0)
        assert np.array_equal(part.x, full.x[n0:]) and np.array_equal(part.e_s, full.e_s[n0:])
        assert np.array_equal(op["wscales"], of["wscales"][:, n0 // 512 * 20:])
        assert np.array_equal(op["sscales"], of["sscales"][n0 // 256 * 7:])


def test_code_widths_and_rejections():
    assert O.code_bits(sq(O.Q_TOPK, 1, 512)) == 1
    assert O.code_bits(sq(O.Q_RANDK, 9, 256)) == 1
    assert O.code_bits(sq(O.Q_TOPK, 0, 512)) == -1
    assert O.num_scales(sq(O.Q_TOPK, 5, 512), 1300, 1300) == 3 * 5
    with pytest.raises(ValueError):
        O.quantize(sq(O.Q_RANDK, 4, 256), np.ones(300, np.float32))   # random-k needs draws
