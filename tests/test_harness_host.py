"""The parity harness itself (tests/parity_util.py), on the CPU: it must be
able to fail.  "GPU" results here are made from the oracle's own output with a
planted mistake, and every planted mistake must be rejected; a one-ulp scale
tie whose codes are the oracle's quantization under the other scale must be
accepted, and only that."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from parity_util import RoundCheck, Stats, check_message, close, qfields

STOCH4 = qfields(O.Q_STOCH_UNIFORM, 4, O.SCALE_L2, 1, 512)


def test_close_rejects_nan_and_inf_garbage():
    want = np.array([1.0, -2.0, 3.0, 4.0], np.float32)
    close("ok", want.copy(), want, Stats())
    bad = want.copy()
    bad[2] = np.nan
    with pytest.raises(AssertionError, match="NaN"):
        close("nan", bad, want, Stats())
    with pytest.raises(AssertionError, match="NaN"):
        close("nan-want", want, bad, Stats())
    inf_want = want.copy()
    inf_want[1] = -np.inf
    garbage = inf_want.copy()
    garbage[1] = 1e30                  # finite garbage where the oracle has an infinity
    with pytest.raises(AssertionError, match="infinite"):
        close("inf", garbage, inf_want, Stats())
    flipped = inf_want.copy()
    flipped[1] = np.inf                # the wrong sign of infinity
    with pytest.raises(AssertionError, match="infinite"):
        close("inf-sign", flipped, inf_want, Stats())
    # the floor comes from the finite entries only: an infinity does not make
    # every finite error acceptable
    off = inf_want.copy()
    off[0] = 1.5
    with pytest.raises(AssertionError, match="beyond tolerance"):
        close("floor", off, inf_want, Stats())
    close("same-inf", inf_want.copy(), inf_want, Stats())
    nan_both = bad.copy()
    close("nan-both", nan_both, bad, Stats())


def _round(d=1300, N=3, t=2, seed=6):
    oc = O.Config(d=d, N=N, placement=O.ADAM_AT_SERVER, beta1=0.9, beta2=0.999, lr=1e-3, eps=1e-8, seed=seed,
                  qw=O.Quant(**STOCH4), qs=O.Quant(**STOCH4))
    w = W.Workload("h", "h", d, N, None, None, 1, seed, "student_t")
    st = O.State.init(oc, d)
    for s in range(1, t):
        O.step(oc, s, W.host_gradients(w, s, d=d), st)
    before = st.copy()
    out = O.step(oc, t, W.host_gradients(w, t, d=d), st, want_inputs=True)
    return oc, d, t, out, before, st


def _worker_msg(oc, d, t, out, i):
    return out["wcodes"][i].copy(), out["wscales"][i].copy()


def _tie_bucket(oc, d, t, out, i, b, bits_up=1):
    """Worker i's message with bucket b coded under its scale moved by one
    ulp, exactly as the oracle would code it under that scale."""
    words, scales = _worker_msg(oc, d, t, out, i)
    B = 512
    p = out["p_w"][i]
    s2 = np.nextafter(scales[b], np.float32(np.inf) if bits_up > 0 else np.float32(0), dtype=np.float32)
    n = min(B, d - b * B)
    u = O.uniforms(oc.seed, t, i, b * B, n)
    codes_t, deq_t = O.quantize_bucket(oc.qw, p[b * B:b * B + n], float(s2), u)
    codes = O.unpack(4, words, d)
    codes[b * B:b * B + n] = codes_t
    scales[b] = s2
    return O.pack(4, codes), scales, codes_t, (p[b * B:b * B + n] - deq_t).astype(np.float32)


def _check(oc, d, t, out, i, words, scales, stats=None):
    return check_message(oc.qw, d, 0, oc.seed, t, i, out["p_w"][i], words, scales, out["wcodes"][i],
                         out["wscales"][i], stats or Stats(), f"worker {i}")


def test_exact_message_passes_and_code_flip_fails():
    oc, d, t, out, _, _ = _round()
    words, scales = _worker_msg(oc, d, t, out, 1)
    assert _check(oc, d, t, out, 1, words, scales) == []
    codes = O.unpack(4, words, d)
    codes[700] ^= 1
    with pytest.raises(AssertionError, match="scales are equal"):
        _check(oc, d, t, out, 1, O.pack(4, codes), scales)


def test_validated_tie_is_accepted_and_reported():
    oc, d, t, out, _, _ = _round()
    words, scales, codes_t, res = _tie_bucket(oc, d, t, out, 0, 1)
    stats = Stats()
    tied = _check(oc, d, t, out, 0, words, scales, stats)
    assert len(tied) == 1 and tied[0][0] == 512 and np.array_equal(tied[0][2], res)
    assert stats.scale_ties == 1


def test_tie_with_a_wrong_code_fails():
    oc, d, t, out, _, _ = _round()
    words, scales, codes_t, _ = _tie_bucket(oc, d, t, out, 0, 1)
    codes = O.unpack(4, words, d)
    codes[512 + 37] = (codes[512 + 37] + 1) % 16      # not what the GPU's scale gives
    with pytest.raises(AssertionError, match="under the GPU's scale"):
        _check(oc, d, t, out, 0, O.pack(4, codes), scales)
    # a tie in one bucket does not excuse a flip in another
    codes = O.unpack(4, words, d)
    codes[5] ^= 2
    with pytest.raises(AssertionError, match="scales are equal"):
        _check(oc, d, t, out, 0, O.pack(4, codes), scales)


def test_two_ulp_scale_fails():
    oc, d, t, out, _, _ = _round()
    words, scales = _worker_msg(oc, d, t, out, 2)
    scales[0] = np.nextafter(np.nextafter(scales[0], np.float32(1)), np.float32(1))
    with pytest.raises(AssertionError, match="more than one ulp"):
        _check(oc, d, t, out, 2, words, scales)


def _gpu_state(st):
    return {k: (None if getattr(st, k) is None else getattr(st, k).copy())
            for k in ("e_w", "e_s", "x", "m", "v", "m_w", "v_w")}


def test_round_check_demands_bit_exact_state_without_a_tie():
    oc, d, t, out, _, st = _round()
    chk = RoundCheck(oc, d, 0, t, out, Stats())
    assert not chk.messages(out["wcodes"], out["wscales"], out["scodes"], out["sscales"])
    chk.state(_gpu_state(st), st)
    for name, idx in (("x", 100), ("e_s", 1299), ("m", 0), ("v", 640)):
        gpu = _gpu_state(st)
        gpu[name][idx] = np.nextafter(gpu[name][idx], np.float32(np.inf))   # one ulp: inside the tolerance
        with pytest.raises(AssertionError, match="not bit-identical"):
            chk.state(gpu, st)
    gpu = _gpu_state(st)
    gpu["e_w"][2, 3] = np.nan
    with pytest.raises(AssertionError, match="not bit-identical"):
        chk.state(gpu, st)


def test_round_check_with_a_tie_still_checks_what_the_tie_cannot_reach():
    oc, d, t, out, _, st = _round()
    words, scales, _, res = _tie_bucket(oc, d, t, out, 0, 1)
    wc, ws = out["wcodes"].copy(), out["wscales"].copy()
    wc[0], ws[0] = words, scales
    chk = RoundCheck(oc, d, 0, t, out, Stats())
    # the server's message over the tied span is not compared (its input changed)
    sc = out["scodes"].copy()
    scodes = O.unpack(4, sc, d)
    scodes[600] ^= 3
    assert chk.messages(wc, ws, O.pack(4, scodes), out["sscales"])
    gpu = _gpu_state(st)
    gpu["e_w"][0, 512:1024] = res
    gpu["x"][600] += 1.0                      # inside the reached span: not compared
    chk.state(gpu, st)
    gpu2 = _gpu_state(st)
    gpu2["e_w"][0, 512:1024] = res
    gpu2["x"][100] = np.nextafter(gpu2["x"][100], np.float32(1))   # outside it: must be exact
    with pytest.raises(AssertionError, match="not bit-identical"):
        chk.state(gpu2, st)
    gpu3 = _gpu_state(st)                     # the tied bucket's residual must be the GPU scale's
    with pytest.raises(AssertionError, match="tied bucket"):
        chk.state(gpu3, st)
    # a server code flip outside the reached span fails
    chk2 = RoundCheck(oc, d, 0, t, out, Stats())
    scodes = O.unpack(4, out["scodes"].copy(), d)
    scodes[100] ^= 1
    with pytest.raises(AssertionError, match="scales are equal"):
        chk2.messages(wc, ws, O.pack(4, scodes), out["sscales"])


def test_sparse_values_are_compared_bit_for_bit():
    q = qfields(O.Q_TOPK, bucket=512, keep=8)
    oc = O.Config(d=1100, N=2, placement=O.ADAM_AT_SERVER, beta1=0.9, beta2=0.999, lr=1e-3, eps=1e-8, seed=3,
                  qw=O.Quant(**q), qs=O.Quant(**q))
    w = W.Workload("h", "h", 1100, 2, None, None, 1, 3, "student_t")
    st = O.State.init(oc, 1100)
    out = O.step(oc, 1, W.host_gradients(w, 1, d=1100), st, want_inputs=True)
    vals = out["wscales"][1].copy()
    assert check_message(oc.qw, 1100, 0, 3, 1, 1, out["p_w"][1], out["wcodes"][1], vals, out["wcodes"][1],
                         out["wscales"][1], Stats(), "w") == []
    vals[9] = np.nextafter(vals[9], np.float32(np.inf))
    with pytest.raises(AssertionError, match="kept values"):
        check_message(oc.qw, 1100, 0, 3, 1, 1, out["p_w"][1], out["wcodes"][1], vals, out["wcodes"][1],
                      out["wscales"][1], Stats(), "w")
