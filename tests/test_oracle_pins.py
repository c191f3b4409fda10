"""Pins of the C oracle to what the paper and mathematics fix (CPU only).

Each test checks the oracle against something other than itself: a library
implementation, a closed form, a brute-force search over a definition, an
invariant of the paper, or a worked example derived by hand from a definition.
"""
import ctypes
import json
import math
import os
import subprocess

import numpy as np
import pytest

import oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = json.load(open(os.path.join(HERE, "golden", "paper_constants.json")))


def q_(kind, bits=0, scale=O.SCALE_L2, ef=1, bucket=0, kmin=0, kmax=0):
    return O.Quant(kind=kind, scale=scale, bits=bits, error_feedback=ef, bucket=bucket,
                   pow2_kmin=kmin, pow2_kmax=kmax)


# ---------------------------------------------------------------------------
# Philox4x32-10 against rocRAND's implementation of the same generator.
# ---------------------------------------------------------------------------
ROCRAND_HDR = "/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"


@pytest.fixture(scope="module")
def rocrand_philox(tmp_path_factory):
    if not os.path.exists(ROCRAND_HDR):
        pytest.skip("rocRAND headers not installed")
    so = str(tmp_path_factory.mktemp("pin") / "libphilox_pin.so")
    src = os.path.join(HERE, "pins", "philox_rocrand.cpp")
    subprocess.run(["g++", "-O1", "-fPIC", "-shared", "-D__HIP_PLATFORM_AMD__",
                    "-I/opt/rocm/include", src, "-o", so], check=True)
    lib = ctypes.CDLL(so)
    lib.pin_philox4x32_10.argtypes = [ctypes.c_void_p] * 3 + [ctypes.c_long]
    lib.pin_uniforms.argtypes = [ctypes.c_ulonglong, ctypes.c_uint, ctypes.c_uint, ctypes.c_longlong,
                                 ctypes.c_longlong, ctypes.c_void_p]
    return lib


def test_philox_matches_library(rocrand_philox):
    rng = np.random.default_rng(11)
    n = 3000
    ctr = rng.integers(0, 2**32, size=(n, 4), dtype=np.uint64).astype(np.uint32)
    key = rng.integers(0, 2**32, size=(n, 2), dtype=np.uint64).astype(np.uint32)
    ctr[0] = 0; key[0] = 0
    ctr[1] = 0xFFFFFFFF; key[1] = 0xFFFFFFFF
    ctr[2:40, 0] = np.arange(38)  # consecutive blocks, as the generator is used
    ctr[2:40, 1:] = 0
    ref = np.zeros((n, 4), np.uint32)
    rocrand_philox.pin_philox4x32_10(ctr.ctypes.data, key.ctypes.data, ref.ctypes.data, n)
    got = np.stack([O.philox(ctr[i], key[i]) for i in range(n)])
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("seed,t,stream,n0", [(7, 3, 2, 0), (0x123456789ABCDEF, 1, 0xFFFFFFFF, 5),
                                               (4, 4294967295, 15, (1 << 34) + 3), (1, 20, 1023, 109_999_999)])
def test_uniform_counter_layout_is_rocrand_subsequence(rocrand_philox, seed, t, stream, n0):
    """The draw layout (element n of stream s at step t: word n&3 of the block
    at counter {lo(n>>2), hi(n>>2), t, s}, key = seed) is rocRAND's Philox
    generator seeded with `seed` at subsequence s * 2^32 + t and offset n:
    a run of the oracle's draws equals that generator's successive outputs."""
    length = 4099
    ref = np.zeros(length, np.float32)
    rocrand_philox.pin_uniforms(seed, t, stream, n0, length, ref.ctypes.data)
    assert np.array_equal(O.uniforms(seed, t, stream, n0, length), ref)
    # a swapped t / stream, or a neighbouring word, gives other draws
    other = np.zeros(length, np.float32)
    rocrand_philox.pin_uniforms(seed, stream, t, n0, length, other.ctypes.data)
    assert (other != ref).mean() > 0.99 or t == stream
    rocrand_philox.pin_uniforms(seed, t, stream, n0 + 1, length, other.ctypes.data)
    assert np.array_equal(other[:-1], ref[1:])


def test_uniforms_are_uniform_and_counter_based():
    u = O.uniforms(seed=7, t=3, stream=2, n0=0, length=1 << 20)
    assert u.min() >= 0.0 and u.max() < 1.0
    # chi-square over 256 bins: mean 255, sd ~22.6; 6 sd bound
    hist = np.bincount((u * 256).astype(np.int64), minlength=256)
    exp = u.size / 256
    chi2 = float(((hist - exp) ** 2 / exp).sum())
    assert chi2 < 255 + 6 * math.sqrt(2 * 255)
    # every one of the 24 bits is balanced
    r = (u * 16777216.0).astype(np.uint32)
    for b in range(24):
        frac = ((r >> b) & 1).mean()
        assert abs(frac - 0.5) < 6 * 0.5 / math.sqrt(u.size)
    # any sub-range equals the same slice of the full range
    sub = O.uniforms(seed=7, t=3, stream=2, n0=123457, length=999)
    assert np.array_equal(sub, u[123457:123457 + 999])
    # different step / stream / seed give uncorrelated draws
    for kw in ({"seed": 7, "t": 4, "stream": 2}, {"seed": 7, "t": 3, "stream": 3},
               {"seed": 8, "t": 3, "stream": 2}):
        w = O.uniforms(n0=0, length=1 << 16, **kw)
        c = np.corrcoef(u[:1 << 16], w)[0, 1]
        assert abs(c) < 6 / math.sqrt(1 << 16)


# ---------------------------------------------------------------------------
# Scaled sign: closed form of its error (a Definition 3 compressor).
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("bucket", [256, 512, 2048, 0])
def test_scaled_sign_closed_form(bucket):
    rng = np.random.default_rng(bucket + 1)
    d = 5000
    p = (rng.standard_t(3, d) * 1e-3).astype(np.float32)
    p[17] = 0.0
    p[18] = -0.0
    q = q_(O.Q_SCALED_SIGN, 1, bucket=bucket)
    codes, deq, scales = O.quantize(q, p)
    B = d if bucket == 0 else bucket
    assert scales.size == -(-d // B)
    assert np.array_equal(codes, (p < 0).astype(np.uint32))
    assert deq[17] > 0 and deq[18] > 0  # zeros are sent as +s
    for b in range(scales.size):
        seg = p[b * B:(b + 1) * B].astype(np.float64)
        dq = deq[b * B:(b + 1) * B].astype(np.float64)
        n = seg.size
        l1, l2sq = np.abs(seg).sum(), (seg ** 2).sum()
        assert scales[b] == np.float32(l1 / n)
        err = ((seg - dq) ** 2).sum()
        # ||p - Q(p)||^2 = ||p||^2 - ||p||_1^2 / n  (since <p, Q> = ||Q||^2 = ||p||_1^2 / n)
        assert err == pytest.approx(l2sq - l1 ** 2 / n, rel=1e-5, abs=1e-7 * l2sq)
        # Definition 3 with (1-delta)^2 = 1 - ||p||_1^2 / (n ||p||^2) < 1
        assert err <= l2sq * (1 - l1 ** 2 / (n * l2sq)) * (1 + 1e-5)


# ---------------------------------------------------------------------------
# Stochastic uniform k-bit: bounded error, exact unbiasedness over the draw.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("bits", [1, 2, 4, 8])
@pytest.mark.parametrize("scale", [O.SCALE_MAX, O.SCALE_L2])
def test_stoch_uniform_bounded_error(bits, scale):
    rng = np.random.default_rng(bits * 10 + scale)
    d = 4096
    p = (rng.standard_normal(d) * np.exp(rng.uniform(-8, 2, d))).astype(np.float32)
    u = rng.random(d, dtype=np.float32)
    q = q_(O.Q_STOCH_UNIFORM, bits, scale=scale, bucket=512)
    codes, deq, scales = O.quantize(q, p, u=u)
    L = 2 ** bits - 1
    assert codes.max() <= L
    s = np.repeat(scales.astype(np.float64), 512)
    step = 2.0 / L
    err = np.abs(deq.astype(np.float64) - p)
    assert np.all(err <= s * step * (1 + 1e-6))
    # every output is s times a grid level (2c-L)/L
    lev = (2.0 * codes - L) / L
    assert np.allclose(deq, s * lev, rtol=2e-7, atol=0)
    seg = p.reshape(-1, 512).astype(np.float64)
    ref = np.abs(seg).max(1) if scale == O.SCALE_MAX else np.sqrt((seg ** 2).sum(1))
    assert np.allclose(scales, ref, rtol=1e-7)


@pytest.mark.parametrize("bits", [1, 2, 4])
def test_stoch_uniform_unbiased_over_draw_grid(bits):
    """E_u[Q(p)] = p: average over a uniform grid of draws u = (k+1/2)/K."""
    rng = np.random.default_rng(100 + bits)
    n = 300
    p = rng.standard_normal(n).astype(np.float32)
    q = q_(O.Q_STOCH_UNIFORM, bits, scale=O.SCALE_MAX, bucket=0)
    K = 2048
    acc = np.zeros(n)
    for k in range(K):
        u = np.full(n, (k + 0.5) / K, np.float32)
        _, deq, s = O.quantize(q, p, u=u)
        acc += deq
    mean = acc / K
    step = 2.0 / (2 ** bits - 1) * float(s[0])
    # grid resolution bound: |E - p| <= step / K (plus binary32 rounding)
    assert np.all(np.abs(mean - p) <= step / K + 4e-7 * np.abs(p).max())


def test_stoch_uniform_unbiased_with_philox():
    """Monte Carlo over the generator itself: mean of Q within 5 sigma of p."""
    rng = np.random.default_rng(5)
    n = 512
    p = rng.standard_normal(n).astype(np.float32)
    q = q_(O.Q_STOCH_UNIFORM, 2, scale=O.SCALE_MAX, bucket=0)
    S = 3000
    acc = np.zeros(n)
    for t in range(1, S + 1):
        u = O.uniforms(seed=99, t=t, stream=0, n0=0, length=n)
        _, deq, s = O.quantize(q, p, u=u)
        acc += deq
    mean = acc / S
    s = float(s[0])
    step = 2.0 / 3 * s
    y = (p / s + 1) * 1.5
    f = y - np.floor(y)
    sd = step * np.sqrt(f * (1 - f)) / math.sqrt(S)
    assert np.all(np.abs(mean - p) <= 5 * sd + 1e-6)


def test_stoch_uniform_zero_bucket():
    q = q_(O.Q_STOCH_UNIFORM, 4, scale=O.SCALE_L2, bucket=256)
    p = np.zeros(512, np.float32)
    p[300] = 1.5
    codes, deq, scales = O.quantize(q, p, u=np.full(512, 0.5, np.float32))
    assert scales[0] == 0 and np.all(deq[:256] == 0) and np.all(codes[:256] == 0)
    assert scales[1] == 1.5


# ---------------------------------------------------------------------------
# Example 1: brute-force argmin over M_2 and the paper's error bound.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("k", [1, 2, 3, 7])
def test_example1_is_argmin_over_grid(k):
    rng = np.random.default_rng(k)
    d = 1000
    p = (rng.standard_normal(d) * 3).astype(np.float32)
    p[5] = 0.0
    q = q_(O.Q_DET_UNIFORM, k + 1, bucket=0)
    codes, deq, s = O.quantize(q, p)
    L = 2 ** k - 1
    levels = np.arange(-L, L + 1) / L          # M_2
    s = float(s[0])
    assert s == np.abs(p).max()               # Q_1(max-norm) is the max-norm itself
    inv = np.float32(1.0) / np.float32(s)
    x = (p * inv).astype(np.float64)           # x / Q_1(|x|_inf), formed as x * (1/s)
    dist = np.abs(x[:, None] - levels[None, :])
    best = dist.min(1)
    chosen = (codes.astype(np.int64) - L) / L
    mine = np.abs(x - chosen)
    # the chosen level is a nearest one (up to one binary32 rounding of x*L)
    assert np.all(mine <= best + 2.0 ** -22)
    ties = np.isclose(dist, best[:, None], rtol=0, atol=2.0 ** -22).sum(1) > 1
    assert np.all(np.abs(chosen[ties]) <= np.abs(x[ties]) + 1e-12)  # tie goes toward zero
    assert deq[5] == 0.0 and codes[5] == L
    assert np.allclose(deq, s * chosen, rtol=2e-7)


def test_example1_zero_vector_and_hand_example():
    q = q_(O.Q_DET_UNIFORM, 2, bucket=0)     # k = 1: levels {-1, 0, 1} (ternary)
    codes, deq, s = O.quantize(q, np.zeros(10, np.float32))
    assert np.all(deq == 0) and np.all(codes == 1)
    # worked by hand: max-norm 2; x/s = [1, -0.25, 0.5, -0.75, 0.3]
    # nearest of {-1,0,1}: 1, 0, 0 (tie -> toward 0), -1, 0
    p = np.array([2.0, -0.5, 1.0, -1.5, 0.6], np.float32)
    codes, deq, s = O.quantize(q, p)
    assert s[0] == 2.0
    assert deq.tolist() == [2.0, 0.0, 0.0, -2.0, 0.0]
    assert codes.tolist() == [2, 1, 1, 0, 1]


def test_example1_bound_from_paper():
    bound = GOLDEN["example1_bound"]
    assert "sqrt" in bound["ratio"]
    rng = np.random.default_rng(3)
    for k in (1, 2, 3, 4):
        L = 2 ** k - 1
        q = q_(O.Q_DET_UNIFORM, k + 1, bucket=0)
        for trial in range(60):
            d = int(rng.integers(2, 400))
            if trial % 3 == 0:      # adversarial: coordinates just past a half level
                x = np.full(d, 0.5 / L * (1 + 1e-6), np.float32)
                x[0] = 1.0
            else:
                x = (rng.standard_normal(d) * 10.0 ** rng.uniform(-3, 3)).astype(np.float32)
            _, deq, _ = O.quantize(q, x)
            x64 = x.astype(np.float64)
            r = np.linalg.norm(deq - x64) / np.linalg.norm(x64)
            assert r <= math.sqrt((d - 1) / (d - 1 + 2 ** k)) * (1 + 1e-6)


# ---------------------------------------------------------------------------
# Example 2: brute-force argmin over M and Definition 1 with the paper's
# constants delta = 1/2, delta' = 2^k sqrt(d).
# ---------------------------------------------------------------------------
def test_example2_hand_example():
    q = q_(O.Q_POW2, kmin=-2, kmax=1)          # M = {1/4, 1/2, 1, 2}
    assert O.code_bits(q) == 1 + 3
    p = np.array([0.3, -0.75, 1.6, 3.1, 0.0, -0.1, 0.375, 1.5, 2.9, -0.0], np.float32)
    # by hand: 0.3->1/4; -0.75 ties 1/2,1 -> -1/2; 1.6->2; 3.1->2; 0->0;
    # -0.1->-1/4; 0.375 ties 1/4,1/2 -> 1/4; 1.5 ties 1,2 -> 1; 2.9->2; -0->0
    _, deq, _ = O.quantize(q, p)
    assert deq.tolist() == [0.25, -0.5, 2.0, 2.0, 0.0, -0.25, 0.25, 1.0, 2.0, 0.0]


@pytest.mark.parametrize("kmin,kmax", [(-17, -11), (-5, 3), (-126, 127), (0, 1)])
def test_example2_is_argmin_over_M(kmin, kmax):
    rng = np.random.default_rng(kmax - kmin)
    d = 4000
    mid = (kmin + kmax) / 2
    p = (rng.choice([-1, 1], d) * 2.0 ** rng.uniform(kmin - 3, min(kmax + 3, 127.9), d)).astype(np.float32)
    p[:4] = [0.0, 2.0 ** kmin * 1.5, -(2.0 ** kmax) * 1.5, 2.0 ** mid]
    q = q_(O.Q_POW2, kmin=kmin, kmax=kmax)
    codes, deq, _ = O.quantize(q, p)
    M = 2.0 ** np.arange(kmin, kmax + 1, dtype=np.float64)
    a = np.abs(p.astype(np.float64))
    dist = np.abs(a[:, None] - M[None, :])
    best = dist.min(1)
    got = np.abs(deq.astype(np.float64))
    nz = p != 0
    assert np.all(np.abs(a[nz] - got[nz]) <= best[nz] * (1 + 1e-12))
    ties = (np.isclose(dist, best[:, None], rtol=1e-12, atol=0).sum(1) > 1) & nz
    assert np.all(got[ties] <= a[ties])                      # ties go to the smaller power
    assert np.all(np.sign(deq[nz]) == np.sign(p[nz]))
    assert deq[0] == 0.0
    back = O.dequantize(q, codes, np.zeros(0, np.float32))
    assert np.array_equal(back, deq)


def test_example2_definition1_constants():
    c = GOLDEN["example2_definition1_constants"]
    k, K = GOLDEN["toy_problem"]["example2_k"], GOLDEN["toy_problem"]["example2_K"]
    q = q_(O.Q_POW2, kmin=k, kmax=K)
    rng = np.random.default_rng(17)
    for trial in range(40):
        d = int(rng.integers(1, 3000))
        hi = 2.0 ** K + 2.0 ** (K - 1)                      # validity range of the constants
        x = (rng.uniform(-1, 1, d) * hi * rng.random()).astype(np.float32)
        _, deq, _ = O.quantize(q, x)
        x64, q64 = x.astype(np.float64), deq.astype(np.float64)
        lhs = np.linalg.norm(x64 - q64)
        assert lhs <= (1 - c["delta"]) * np.linalg.norm(x64) + 2.0 ** k * math.sqrt(d) + 1e-12
        big = np.abs(x64) >= 2.0 ** k
        assert np.linalg.norm(q64[big]) <= c["q_norm_factor"] * np.linalg.norm(x64[big]) + 1e-12


def test_code_widths_match_paper_bit_ratio():
    toy = GOLDEN["toy_problem"]
    ex1 = q_(O.Q_DET_UNIFORM, toy["example1_k"] + 1)
    ex2 = q_(O.Q_POW2, kmin=toy["example2_k"], kmax=toy["example2_K"])
    assert O.code_bits(ex2) / O.code_bits(ex1) == GOLDEN["bits_ratio_example2_vs_example1"]["ratio"]
    mags = toy["example2_K"] - toy["example2_k"] + 1
    assert mags == GOLDEN["example2_bits"]["magnitude_codes"]
    assert O.code_bits(ex2) == 1 + math.ceil(math.log2(mags + 1))


# ---------------------------------------------------------------------------
# Full precision ("Ours_full"): identity messages, residual identically zero.
# ---------------------------------------------------------------------------
def test_none_quantizer_identity():
    rng = np.random.default_rng(4)
    p = rng.standard_normal(777).astype(np.float32)
    q = q_(O.Q_NONE)
    codes, deq, _ = O.quantize(q, p)
    assert np.array_equal(deq, p)
    assert np.array_equal(codes, p.view(np.uint32))
    words = O.pack(32, codes)
    assert np.array_equal(words.view(np.uint32)[:777], codes)


# ---------------------------------------------------------------------------
# Message layout: hand-worked positions and round trip.
# ---------------------------------------------------------------------------
def test_pack_layout_by_hand():
    n = 600
    codes = np.zeros(n, np.uint32)
    codes[5] = 0b10      # chunk 0, lane 1, slot 1, plane 1 -> word (0*4+1)*2+1 = 3, bit 1
    codes[300] = 0b01    # chunk 1, lane 11, slot 0, plane 0 -> word (1*4+0)*2+0 = 8, bit 11
    codes[599] = 0b11    # chunk 2, lane 21, slot 3 -> words (2*4+3)*2+{0,1} = 22, 23, bit 21
    w = O.pack(2, codes)
    assert w.size == 3 * 4 * 2
    expect = np.zeros(24, np.uint64)
    expect[3] = 1 << 1
    expect[8] = 1 << 11
    expect[22] = expect[23] = 1 << 21
    assert np.array_equal(w, expect)


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 8, 32])
def test_pack_round_trip(bits):
    rng = np.random.default_rng(bits)
    for n in (1, 63, 64, 255, 256, 257, 1000):
        hi = 2 ** 32 if bits == 32 else 2 ** bits
        codes = rng.integers(0, hi, n, dtype=np.uint64).astype(np.uint32)
        w = O.pack(bits, codes)
        assert np.array_equal(O.unpack(bits, w, n), codes)
        if bits < 32:   # no stray bits beyond the segment
            assert sum(bin(int(v)).count("1") for v in w) == sum(bin(int(c)).count("1") for c in codes)


# ---------------------------------------------------------------------------
# Adam (Algorithm 2): closed form under a constant gradient; Lemma 1.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("placement", [O.ADAM_AT_SERVER, O.ADAM_AT_WORKER])
def test_adam_closed_form_constant_gradient(placement):
    d, N, T = 512, 3, 60
    rng = np.random.default_rng(9)
    c = (rng.standard_normal(d) * 1e-2).astype(np.float32)
    q = q_(O.Q_NONE)
    cfg = O.Config(d=d, N=N, placement=placement, beta1=0.9, beta2=0.999, lr=1e-3, eps=1e-8,
                   seed=1, qw=q, qs=q)
    st = O.State.init(cfg, d)
    g = np.tile(c, (N, 1))
    for t in range(1, T + 1):
        O.step(cfg, t, g, st)
    b1, b2, eps = 0.9, 0.999, 1e-8
    m_exp = (1 - b1 ** T) * c.astype(np.float64)
    v_exp = b2 ** T * eps + (1 - b2 ** T) * c.astype(np.float64) ** 2
    m = st.m if placement == O.ADAM_AT_SERVER else st.m_w[0]
    v = st.v if placement == O.ADAM_AT_SERVER else st.v_w[0]
    assert np.allclose(m, m_exp, rtol=2e-5, atol=0)
    assert np.allclose(v, v_exp, rtol=2e-5, atol=0)
    assert np.all(st.e_w == 0) and np.all(st.e_s == 0)
    # x moved by the sum of the Adam steps lr*m_t/sqrt(v_t)
    steps = sum(1e-3 * (1 - b1 ** t) * c.astype(np.float64) /
                np.sqrt(b2 ** t * eps + (1 - b2 ** t) * c.astype(np.float64) ** 2) for t in range(1, T + 1))
    assert np.allclose(st.x, -steps, rtol=1e-4, atol=1e-9)


def test_lemma1_invariant():
    d, N, T = 1024, 4, 80
    b1, b2 = 0.9, 0.999
    gamma = b1 / b2
    bound = 1.0 / ((1 - gamma) * (1 - b2))
    q = q_(O.Q_STOCH_UNIFORM, 2, scale=O.SCALE_MAX, bucket=512)
    cfg = O.Config(d=d, N=N, placement=O.ADAM_AT_WORKER, beta1=b1, beta2=b2, lr=1e-3, eps=1e-8,
                   seed=3, qw=q, qs=q)
    st = O.State.init(cfg, d)
    rng = np.random.default_rng(12)
    for t in range(1, T + 1):
        g = (rng.standard_t(3, (N, d)) * 10.0 ** rng.uniform(-4, 1)).astype(np.float32)
        g[:, :10] = 0.0
        O.step(cfg, t, g, st)
        m, v = st.m_w.astype(np.float64), st.v_w.astype(np.float64)
        assert np.all(m ** 2 <= bound * v * (1 + 1e-5))


# ---------------------------------------------------------------------------
# Schedules: Assumption 2 (theta_t = 1 - theta/T, alpha_t = alpha/sqrt(T)) and
# the step decay of Section V-B, against their closed forms.
# ---------------------------------------------------------------------------
ULP = 2.0 ** -23


def sched_(kind, alpha=0.0, theta=0.0, factor=1.0, T=0, period=1):
    return O.Schedule(kind=kind, alpha=alpha, theta=theta, factor=factor, T=T, period=period)


def test_schedule_constant_returns_the_configured_values():
    s = sched_(O.SCHED_CONSTANT)
    for t in (1, 2, 10 ** 6):
        lr, b2 = O.schedule_at(s, 1e-3, 0.999, t)
        assert lr == np.float32(1e-3) and b2 == np.float32(0.999)


@pytest.mark.parametrize("alpha,theta,T", [(1e-3, 0.99, 1000), (0.05, 0.5, 19550), (1.0, 1.0, 1), (3e-4, 7.0, 12345)])
def test_schedule_assumption2_closed_form(alpha, theta, T):
    s = sched_(O.SCHED_ASSUMPTION2, alpha=alpha, theta=theta, T=T)
    a32, th32 = float(np.float32(alpha)), float(np.float32(theta))
    for t in (1, 2, T, T + 5):       # constant over t for a fixed horizon
        lr, b2 = O.schedule_at(s, 0.0, 0.0, t)
        assert abs(lr - a32 / math.sqrt(T)) <= 2 * ULP * (a32 / math.sqrt(T))
        assert abs(b2 - (1.0 - th32 / T)) <= 2 * ULP
        assert 0.0 <= b2 < 1.0


def test_schedule_step_decay_section_vb():
    cfg = GOLDEN["schedules"]
    factor, period = cfg["step_decay_factor"], cfg["step_decay_period"]
    alpha = 1e-3
    s = sched_(O.SCHED_STEP_DECAY, alpha=alpha, factor=factor, period=period)
    a32, f32 = float(np.float32(alpha)), float(np.float32(factor))
    # the first `period` iterations use alpha; the decay applies after them
    assert O.schedule_at(s, 0.0, 0.999, 1) == (np.float32(alpha), np.float32(0.999))
    assert O.schedule_at(s, 0.0, 0.999, period)[0] == np.float32(alpha)
    assert O.schedule_at(s, 0.0, 0.999, period + 1)[0] == np.float32(np.float32(alpha) * np.float32(factor))
    prev = math.inf
    for k in range(0, 40):
        for t in (k * period + 1, (k + 1) * period):
            lr, b2 = O.schedule_at(s, 0.0, 0.999, t)
            want = a32 * f32 ** k
            assert abs(lr - want) <= (2 * k.bit_length() + 2) * ULP * want + 1e-45
            assert b2 == np.float32(0.999)
            assert lr <= prev
            prev = lr


def test_schedule_step_decay_unit_factor_and_short_period():
    s = sched_(O.SCHED_STEP_DECAY, alpha=0.1, factor=1.0, period=1)
    assert all(O.schedule_at(s, 0.0, 0.9, t)[0] == np.float32(0.1) for t in (1, 2, 1000, 10 ** 9))
    s = sched_(O.SCHED_STEP_DECAY, alpha=1.0, factor=0.5, period=1)
    for t in (1, 2, 3, 30, 126, 127):
        assert O.schedule_at(s, 0.0, 0.9, t)[0] == np.float32(2.0 ** -(t - 1))


@pytest.mark.parametrize("s,t", [
    (sched_(O.SCHED_CONSTANT), 0),
    (sched_(O.SCHED_ASSUMPTION2, alpha=1e-3, theta=0.5, T=0), 1),
    (sched_(O.SCHED_ASSUMPTION2, alpha=1e-3, theta=2.0, T=1), 1),
    (sched_(O.SCHED_ASSUMPTION2, alpha=1e-3, theta=0.0, T=10), 1),
    (sched_(O.SCHED_ASSUMPTION2, alpha=1e-3, theta=0.5, T=1 << 24), 1),
    (sched_(O.SCHED_STEP_DECAY, alpha=1e-3, factor=1.5, period=10), 1),
    (sched_(O.SCHED_STEP_DECAY, alpha=1e-3, factor=0.0, period=10), 1),
    (sched_(O.SCHED_STEP_DECAY, alpha=1e-3, factor=0.2, period=0), 1),
    (sched_(7), 1),
])
def test_schedule_rejects_invalid(s, t):
    with pytest.raises(ValueError):
        O.schedule_at(s, 1e-3, 0.999, t)


# ---------------------------------------------------------------------------
# Error feedback: telescoping identities of Section IV (EF as delayed update)
# and the virtual-iterate identities of the appendix (Notation 1), with the
# sign of the second identity read as x_{t+1} - e_{t+1} = x_t - e_t - avg_t.
# ---------------------------------------------------------------------------
def _dequant_msgs(cfg, out, d):
    bw, bs = O.code_bits(cfg.qw), O.code_bits(cfg.qs)
    wq = [O.dequantize(cfg.qw, O.unpack(bw, out["wcodes"][i], d), out["wscales"][i], d)
          for i in range(cfg.N)]
    sq = O.dequantize(cfg.qs, O.unpack(bs, out["scodes"], d), out["sscales"], d)
    return np.stack(wq).astype(np.float64), sq.astype(np.float64)


CASES = [
    ("sign-server", O.ADAM_AT_SERVER, q_(O.Q_SCALED_SIGN, 1, bucket=512), q_(O.Q_SCALED_SIGN, 1, bucket=512)),
    ("stoch4-server", O.ADAM_AT_SERVER, q_(O.Q_STOCH_UNIFORM, 4, O.SCALE_L2, bucket=512),
     q_(O.Q_STOCH_UNIFORM, 4, O.SCALE_L2, bucket=512)),
    ("ex1-worker", O.ADAM_AT_WORKER, q_(O.Q_DET_UNIFORM, 2), q_(O.Q_DET_UNIFORM, 2)),
    ("ex2-worker", O.ADAM_AT_WORKER, q_(O.Q_POW2, kmin=-17, kmax=-11), q_(O.Q_POW2, kmin=-17, kmax=-11)),
    ("stoch2-worker", O.ADAM_AT_WORKER, q_(O.Q_STOCH_UNIFORM, 2, O.SCALE_MAX, bucket=256),
     q_(O.Q_SCALED_SIGN, 1, bucket=256)),
    ("topk-server", O.ADAM_AT_SERVER, O.Quant(kind=O.Q_TOPK, keep=16, bucket=512, error_feedback=1),
     O.Quant(kind=O.Q_TOPK, keep=8, bucket=256, error_feedback=1)),
    ("randk-worker", O.ADAM_AT_WORKER, O.Quant(kind=O.Q_RANDK, keep=32, bucket=256, error_feedback=1),
     O.Quant(kind=O.Q_TOPK, keep=64, bucket=1024, error_feedback=1)),
]


@pytest.mark.parametrize("name,placement,qw,qs", CASES, ids=[c[0] for c in CASES])
def test_error_feedback_telescoping_and_virtual_iterate(name, placement, qw, qs):
    d, N, T = 1500, 4, 30
    cfg = O.Config(d=d, N=N, placement=placement, beta1=0.9, beta2=0.999, lr=1e-3, eps=1e-8,
                   seed=21, qw=qw, qs=qs)
    rng = np.random.default_rng(31)
    x1 = (rng.standard_normal(d) * 0.02).astype(np.float32)
    st = O.State.init(cfg, d, x1)
    sum_a_w = np.zeros((N, d))      # inputs to Q_w (before adding e)
    sum_dw = np.zeros((N, d))       # dequantized worker messages
    sum_a_s = np.zeros(d)           # inputs to Q_s (before adding e_s)
    sum_ds = np.zeros(d)            # dequantized server messages
    scale = 0.0
    for t in range(1, T + 1):
        g = (rng.standard_normal((N, d)) * 1e-2).astype(np.float32)
        if placement == O.ADAM_AT_WORKER:
            m0, v0 = st.m_w.copy(), st.v_w.copy()
            a_w = np.empty((N, d), np.float32)
            for i in range(N):          # the worker's Adam step, recomputed in binary64
                m = 0.9 * m0[i].astype(np.float64) + 0.1 * g[i]
                v = 0.999 * v0[i].astype(np.float64) + 0.001 * g[i].astype(np.float64) ** 2
                a_w[i] = 1e-3 * m / np.sqrt(v)
        else:
            a_w = g
        out = O.step(cfg, t, g, st, want_srv_in=True)
        dw, ds = _dequant_msgs(cfg, out, d)
        sum_a_w += a_w
        sum_dw += dw
        sum_a_s += out["srv_in"]
        sum_ds += ds
        scale = max(scale, np.abs(a_w).max(), np.abs(out["srv_in"]).max())
        # x_{t+1} = x_t - server message: x equals x_1 minus the sum of broadcasts
        assert np.allclose(st.x, x1 - sum_ds, rtol=0, atol=(t + 2) * 2e-7 * (np.abs(x1).max() + 1))
    tol = T * 4 * 2.0 ** -24 * scale * 10 + 1e-12
    # sum of sent messages + final residual = sum of inputs (per worker, and server)
    tw = 3e-4 if placement == O.ADAM_AT_WORKER else 0.0  # worker Adam recomputed in binary64
    assert np.allclose(sum_dw + st.e_w, sum_a_w, rtol=tw, atol=tol)
    assert np.allclose(sum_ds + st.e_s, sum_a_s, rtol=0, atol=tol)
    # virtual iterate: x_{T+1} - e_s = x_1 - sum of server inputs
    assert np.allclose(st.x.astype(np.float64) - st.e_s, x1 - sum_a_s, rtol=0, atol=tol + T * 2e-7 * 0.1)
    # and the server input is the worker average: sum_t mean_i delta_i + mean_i e_i = sum_t mean_i a_i
    if placement == O.ADAM_AT_WORKER:
        lhs = sum_a_s + st.e_w.astype(np.float64).mean(0)
        assert np.allclose(lhs, sum_a_w.mean(0), rtol=tw, atol=tol)


def test_error_feedback_off_keeps_no_residual():
    d, N = 1024, 2
    q = q_(O.Q_SCALED_SIGN, 1, ef=0, bucket=256)
    cfg = O.Config(d=d, N=N, placement=O.ADAM_AT_SERVER, beta1=0.9, beta2=0.999, lr=1e-3, eps=1e-8,
                   seed=2, qw=q, qs=q)
    st = O.State.init(cfg, d)
    rng = np.random.default_rng(1)
    for t in range(1, 4):
        O.step(cfg, t, rng.standard_normal((N, d)).astype(np.float32), st)
        assert np.all(st.e_w == 0) and np.all(st.e_s == 0)


def test_workers_compress_independently():
    """Each worker compresses with randomness of its own, so the server's
    average of N stochastic messages of one input deviates from it by about
    1/N of one message's mean square error (identical draws on every worker
    would leave the ratio at 1), and worker i draws the documented stream i."""
    d, N = 4096, 8
    q = q_(O.Q_STOCH_UNIFORM, 2, O.SCALE_MAX, bucket=256)
    cfg = O.Config(d=d, N=N, placement=O.ADAM_AT_SERVER, beta1=0.9, beta2=0.999, lr=1e-3, eps=1e-8,
                   seed=5, qw=q, qs=q)
    st = O.State.init(cfg, d)
    g1 = np.random.default_rng(3).standard_normal(d).astype(np.float32)
    out = O.step(cfg, 1, np.tile(g1, (N, 1)), st)
    dw, _ = _dequant_msgs(cfg, out, d)
    err = dw - g1.astype(np.float64)
    one = np.mean(err ** 2)
    avg = np.mean(err.mean(0) ** 2)
    assert 0.6 / N < avg / one < 1.6 / N, avg / one
    for i in range(N):
        # at t = 1 with e_w = 0 the worker quantizes g itself
        codes, _, _ = O.quantize(q, g1, u=O.uniforms(cfg.seed, 1, i, 0, d))
        assert np.array_equal(O.unpack(2, out["wcodes"][i], d), codes), i


# ---------------------------------------------------------------------------
# Segments: the round is bucket-local, so a segment equals the same slice of
# the full run (this is what makes sampled full-size parity possible).
# ---------------------------------------------------------------------------
def test_segment_equals_slice_of_full_run():
    d, N = 6 * 512 + 300, 3
    qw = q_(O.Q_STOCH_UNIFORM, 4, O.SCALE_L2, bucket=512)
    qs = q_(O.Q_STOCH_UNIFORM, 2, O.SCALE_MAX, bucket=1024)
    cfg = O.Config(d=d, N=N, placement=O.ADAM_AT_SERVER, beta1=0.9, beta2=0.999, lr=1e-3, eps=1e-8,
                   seed=77, qw=qw, qs=qs)
    rng = np.random.default_rng(8)
    full = O.State.init(cfg, d)
    n0, ln = 1024, 2048
    part = O.State.init(cfg, ln)
    for t in range(1, 4):
        g = rng.standard_normal((N, d)).astype(np.float32)
        o_full = O.step(cfg, t, g, full)
        o_part = O.step(cfg, t, np.ascontiguousarray(g[:, n0:n0 + ln]), part, n0=n0)
        assert np.array_equal(part.x, full.x[n0:n0 + ln])
        assert np.array_equal(part.e_w, full.e_w[:, n0:n0 + ln])
        w0 = n0 // 256 * 16
        assert np.array_equal(o_part["wcodes"], o_full["wcodes"][:, w0:w0 + o_part["wcodes"].shape[1]])
        assert np.array_equal(o_part["sscales"], o_full["sscales"][1:3])


# ---------------------------------------------------------------------------
# Convergence: the toy quadratic of the benchmark, and the paper's toy problem
# (Section V-A) with the EF ablation claim of Figure 2.
# ---------------------------------------------------------------------------
def _toy_quadratic(kind, ef, T=100, d=65536, N=4, seed=1):
    rng = np.random.default_rng(seed)
    xs = rng.standard_normal(d).astype(np.float32)
    q = q_(kind, 1 if kind == O.Q_SCALED_SIGN else 0, ef=ef, bucket=0)
    cfg = O.Config(d=d, N=N, placement=O.ADAM_AT_SERVER, beta1=0.9, beta2=0.999, lr=1e-3, eps=1e-8,
                   seed=seed, qw=q, qs=q)
    st = O.State.init(cfg, d)
    F0 = 0.5 * np.sum((st.x.astype(np.float64) - xs) ** 2)
    for t in range(1, T + 1):
        g = (st.x - xs)[None, :] + (0.1 * rng.standard_normal((N, d))).astype(np.float32)
        O.step(cfg, t, g.astype(np.float32), st)
    return 0.5 * np.sum((st.x.astype(np.float64) - xs) ** 2) / F0


def test_toy_quadratic_converges():
    full = _toy_quadratic(O.Q_NONE, 1)
    sign_ef = _toy_quadratic(O.Q_SCALED_SIGN, 1)
    assert full < 0.6 and sign_ef < 0.6          # calibrated on the oracle: 0.47, 0.55
    assert sign_ef < 1.25 * full


def _paper_toy(kind, ef, lr, seed, T):
    toy = GOLDEN["toy_problem"]
    d, N = toy["A_shape"][0], toy["workers"]
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((d, d))
    xs = rng.standard_normal(d) * math.sqrt(toy["x_star_cov"])
    if kind == O.Q_DET_UNIFORM:
        q = q_(kind, toy["example1_k"] + 1, ef=ef)
    elif kind == O.Q_POW2:
        q = q_(kind, ef=ef, kmin=toy["example2_k"], kmax=toy["example2_K"])
    else:
        q = q_(O.Q_NONE, ef=ef)
    cfg = O.Config(d=d, N=N, placement=O.ADAM_AT_WORKER, beta1=toy["beta"], beta2=toy["theta"], lr=lr,
                   eps=1e-8, seed=seed, qw=q, qs=q)
    st = O.State.init(cfg, d)
    grad_sq = lambda x: float(np.sum((2 * A.T @ (A @ x - xs)) ** 2))  # noqa: E731
    first = grad_sq(st.x.astype(np.float64))
    for t in range(1, T + 1):
        x = st.x.astype(np.float64)
        xi = rng.standard_normal((N, d)) * math.sqrt(toy["xi_cov"])
        g = 2 * ((A @ x - xs)[None, :] - xi) @ A
        O.step(cfg, t, g.astype(np.float32), st)
    return first, grad_sq(st.x.astype(np.float64))


@pytest.mark.parametrize("seed", [0, 1])
def test_paper_toy_error_feedback_ablation(seed):
    lr, T = 1e-4, 1000
    g0, full = _paper_toy(O.Q_NONE, 1, lr, seed, T)
    _, com1 = _paper_toy(O.Q_DET_UNIFORM, 1, lr, seed, T)
    _, com1_err = _paper_toy(O.Q_DET_UNIFORM, 0, lr, seed, T)
    _, com2 = _paper_toy(O.Q_POW2, 1, lr, seed, T)
    assert full < g0 / 10 and com1 < g0 / 10 and com2 < g0 / 10   # ||grad F||^2 decreases
    assert com1 < 0.5 * com1_err       # Figure 2: with Example 1, error feedback helps
    assert com2 < 1.05 * full          # Example 2 is about as good as full precision


# ---------------------------------------------------------------------------
# Section V-A toy problem: the oracle's gradient against finite differences
# of the objective, special cases and the noise-free consistency.
# ---------------------------------------------------------------------------
def _toy_inputs(d, N, seed):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((d, d)).astype(np.float32)
    xs = (rng.standard_normal(d) * math.sqrt(0.1)).astype(np.float32)
    xi = (rng.standard_normal((N, d)) * math.sqrt(0.1)).astype(np.float32)
    x = rng.standard_normal(d).astype(np.float32)
    return A, xs, xi, x


def _objective(A, xs, xi_i, x):
    """||A x - (x* + xi)||^2 by plain loops in binary64."""
    d = len(x)
    tot = 0.0
    for k in range(d):
        r = sum(float(A[k, j]) * float(x[j]) for j in range(d)) - float(xs[k]) - float(xi_i[k])
        tot += r * r
    return tot


@pytest.mark.parametrize("d,N,seed", [(5, 2, 0), (9, 3, 1)])
def test_toy_grad_matches_finite_differences(d, N, seed):
    A, xs, xi, x = _toy_inputs(d, N, seed)
    g, _ = O.toy_grad(A, xs, xi, x)
    h = 1e-3
    for i in range(N):
        for j in range(d):
            xp, xm = x.astype(np.float64).copy(), x.astype(np.float64).copy()
            xp[j] += h
            xm[j] -= h
            # the objective is quadratic: central differences are exact up to rounding
            fd = (_objective(A, xs, xi[i], xp) - _objective(A, xs, xi[i], xm)) / (2 * h)
            assert abs(g[i, j] - fd) <= 1e-6 * (abs(fd) + 1.0), (i, j, g[i, j], fd)


def test_toy_grad_identity_matrix_and_noise_free_norm():
    d, N = 64, 4
    _, xs, xi, x = _toy_inputs(d, N, 3)
    A = np.eye(d, dtype=np.float32)
    g, gsq = O.toy_grad(A, xs, xi, x)
    want = (2.0 * (x.astype(np.float64) - xs - xi)).astype(np.float32)
    assert np.array_equal(g, want)
    assert gsq == pytest.approx(float(np.sum((2.0 * (x.astype(np.float64) - xs)) ** 2)), rel=1e-12)
    # a general matrix: the squared norm is that of the noise-free gradient,
    # and every worker's gradient differs from it by -2 A^T xi_i
    A, xs, xi, x = _toy_inputs(40, 3, 4)
    g, gsq = O.toy_grad(A, xs, xi, x)
    g0, gsq0 = O.toy_grad(A, xs, np.zeros((1, 40), np.float32), x)
    assert gsq == gsq0
    assert gsq == pytest.approx(float(np.sum(g0.astype(np.float64) ** 2)), rel=1e-6)
    lin = g0[0].astype(np.float64) - 2.0 * (xi.astype(np.float64) @ A.astype(np.float64))
    assert np.allclose(g, lin, rtol=1e-5, atol=1e-4)
