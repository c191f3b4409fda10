"""Host-side checks of the C ABI (no GPU work): every symbol declared in
include/ea.h is exported, size queries agree with the oracle's independent
size rules, and invalid calls are rejected before any device work."""
import ctypes
import os
import re

import pytest

import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def E():
    from paper_2205_14473_amd import build as bld
    if bld.is_stale():
        bld.build()
    import paper_2205_14473_amd as E
    return E


def _declared():
    src = open(os.path.join(ROOT, "include", "ea.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ea_[a-z_0-9]+)\s*\(", src)))


def test_every_declared_symbol_is_exported(E):
    names = _declared()
    assert len(names) == 20, names
    for n in names:
        assert hasattr(E.lib, n), f"{n} declared in include/ea.h but not exported"


QUANTS = [
    dict(kind=0),
    dict(kind=1, scale=0, bucket=2048),
    dict(kind=1, bucket=0),
    dict(kind=2, scale=1, bits=4, bucket=512),
    dict(kind=2, scale=2, bits=2, bucket=1024),
    dict(kind=2, scale=2, bits=8, bucket=0),
    dict(kind=3, bits=2, bucket=0),
    dict(kind=3, bits=7, bucket=256),
    dict(kind=4, pow2_kmin=-17, pow2_kmax=-11),
    dict(kind=4, pow2_kmin=-126, pow2_kmax=127),
    dict(kind=5, bucket=512, keep=16),
    dict(kind=5, bucket=256, keep=1),
    dict(kind=6, bucket=2048, keep=2048),
    dict(kind=6, bucket=1024, keep=77),
]


@pytest.mark.parametrize("qd", QUANTS)
@pytest.mark.parametrize("d", [1, 255, 256, 257, 65536, 110_000_000, 355_000_001])
def test_sizes_agree_with_oracle(E, qd, d):
    qe, qo = E.Quant(**qd), O.Quant(**qd)
    assert E.ea_code_bits(qe) == O.code_bits(qo)
    assert E.ea_msg_words(qe, d) == O.msg_words(qo, d)
    assert E.ea_msg_scales(qe, d) == O.num_scales(qo, d, d)
    assert E.ea_msg_bits(qe, d) == d * O.code_bits(qo) + 32 * O.num_scales(qo, d, d)


def _cfg(E, **kw):
    q = E.Quant(kind=2, scale=1, bits=4, error_feedback=1, bucket=512)
    base = dict(d=110_000_000, N=16, placement=0, beta1=0.9, beta2=0.999, lr=1e-3, eps=1e-8, seed=4, qw=q, qs=q)
    base.update(kw)
    return E.Config(**base)


@pytest.mark.parametrize("field,value,code", [
    ("d", 0, -1), ("N", 0, -1), ("N", 1025, -1), ("placement", 2, -1), ("beta1", 1.0, -1),
    ("beta2", -0.1, -1), ("lr", float("inf"), -1), ("eps", -1.0, -1)])
def test_invalid_config_rejected(E, field, value, code):
    assert E.ea_validate(_cfg(E, **{field: value})) == code
    assert E.ea_last_error() != ""


@pytest.mark.parametrize("qd,code", [
    (dict(kind=9), -1), (dict(kind=2, scale=1, bits=3, bucket=512), -1), (dict(kind=2, scale=0, bits=2), -1),
    (dict(kind=3, bits=1), -1), (dict(kind=4, pow2_kmin=-3, pow2_kmax=-3), -1),
    (dict(kind=1, bucket=768), -4), (dict(kind=1, bucket=4096), -4), (dict(kind=1, bucket=-5), -1),
    (dict(kind=1, error_feedback=2, bucket=512), -1),
    (dict(kind=5, bucket=512, keep=0), -1), (dict(kind=6, bucket=512, keep=513), -1),
    (dict(kind=5, bucket=0, keep=4), -4), (dict(kind=6, bucket=768, keep=4), -4),
    (dict(kind=5, bucket=4096, keep=4), -4), (dict(kind=5, bucket=512, keep=4, reserved=1), -1)])
def test_invalid_quantizer_rejected(E, qd, code):
    assert E.ea_validate(_cfg(E, qw=E.Quant(**qd))) == code
    assert E.ea_validate(_cfg(E, qs=E.Quant(**qd))) == code


def test_valid_configs_and_workspace(E):
    assert E.ea_validate(_cfg(E)) == 0
    assert E.ea_workspace_bytes(_cfg(E)) == 0
    one = E.Quant(kind=1, bucket=0)
    ws = E.ea_workspace_bytes(_cfg(E, d=65536, N=4, qw=one, qs=one))
    # worker partials [N][tiles] + server partials [tiles] + server input [d], 256-byte aligned
    assert ws == 4 * 128 * 8 + 1024 + 65536 * 4


def test_calls_rejected_before_device_work(E):
    # Uses fake device addresses: only ever run where no GPU is visible, so a
    # validation bug can never turn into a kernel launch on real memory.
    torch = pytest.importorskip("torch")
    if torch.cuda.device_count() > 0:
        pytest.skip("bogus-pointer rejection test runs on GPU-less hosts only")
    c = _cfg(E, d=1024, N=2)
    P = ctypes.c_void_p
    good = [P(4096 * (k + 1)) for k in range(14)]
    # NULL pointer
    assert E.lib.ea_step(ctypes.byref(c), 1, None, *good[1:]) == E.EA_ERR_ARG
    assert "g is NULL" in E.ea_last_error()
    # misaligned float pointer
    args = list(good)
    args[0] = P(4098)
    assert E.lib.ea_step(ctypes.byref(c), 1, *args) == E.EA_ERR_ALIGN
    # step index out of range
    assert E.lib.ea_step(ctypes.byref(c), 0, *good) == E.EA_ERR_ARG
    assert E.lib.ea_step(ctypes.byref(c), 2 ** 32, *good) == E.EA_ERR_ARG
    # worker index out of range
    assert E.lib.ea_worker_compress(ctypes.byref(c), 2, 1, *good[:8]) == E.EA_ERR_ARG
    # misaligned code words (need 8 bytes)
    assert E.lib.ea_worker_apply(ctypes.byref(c), P(4100), P(4096), P(4096), None) == E.EA_ERR_ALIGN
    # missing workspace for a one-bucket quantizer
    one = E.Quant(kind=1, bucket=0)
    c1 = _cfg(E, d=1024, N=2, qw=one, qs=one)
    assert E.lib.ea_step(ctypes.byref(c1), 1, *good[:12], None, None) == E.EA_ERR_ARG
    assert "workspace" in E.ea_last_error()


SCHEDULES = [
    dict(kind=0),
    dict(kind=1, alpha=1e-3, theta=0.99, T=1000),
    dict(kind=1, alpha=0.05, theta=3.0, T=19550),
    dict(kind=2, alpha=1e-3, factor=0.2, period=19550),
    dict(kind=2, alpha=0.1, factor=0.5, period=3),
    dict(kind=2, alpha=1.0, factor=0.999, period=1),
]


@pytest.mark.parametrize("sd", SCHEDULES)
def test_schedule_values_agree_with_oracle(E, sd):
    """The library's host schedule and the oracle's are separate
    implementations of one definition: they agree to the bit."""
    c = _cfg(E)
    se, so = E.Schedule(**sd), O.Schedule(**sd)
    for t in [1, 2, 3, 4, 5, 17, 1000, 19550, 19551, 39101, 10 ** 6, 2 ** 32 - 1]:
        lr, b2 = E.ea_schedule_at(c, se, t)
        lo, bo = O.schedule_at(so, c.lr, c.beta2, t)
        assert lr == float(lo) and b2 == float(bo), (t, lr, lo, b2, bo)


@pytest.mark.parametrize("sd", [
    dict(kind=1, alpha=1e-3, theta=0.5, T=0),
    dict(kind=1, alpha=1e-3, theta=2.0, T=1),
    dict(kind=1, alpha=1e-3, theta=0.0, T=10),
    dict(kind=1, alpha=1e-3, theta=0.5, T=1 << 24),
    dict(kind=2, alpha=1e-3, factor=1.5, period=10),
    dict(kind=2, alpha=1e-3, factor=0.0, period=10),
    dict(kind=2, alpha=1e-3, factor=0.2, period=0),
    dict(kind=2, alpha=-1.0, factor=0.2, period=10),
    dict(kind=2, alpha=float("inf"), factor=0.2, period=10),
    dict(kind=7),
])
def test_invalid_schedule_rejected(E, sd):
    with pytest.raises(E.EAError):
        E.ea_schedule_at(_cfg(E), E.Schedule(**sd), 1)


def test_scheduled_calls_rejected_before_device_work(E):
    torch = pytest.importorskip("torch")
    if torch.cuda.device_count() > 0:
        pytest.skip("bogus-pointer rejection test runs on GPU-less hosts only")
    c = _cfg(E, d=1024, N=2)
    P = ctypes.c_void_p
    good = [P(4096 * (k + 1)) for k in range(14)]
    s = E.Schedule(kind=2, alpha=1e-3, factor=0.2, period=10)
    bad = E.Schedule(kind=2, alpha=1e-3, factor=0.0, period=10)
    sb = ctypes.byref
    # the step counter must be a 4-byte aligned device pointer
    assert E.lib.ea_step_scheduled(sb(c), sb(s), None, *good) == E.EA_ERR_ALIGN
    assert E.lib.ea_step_scheduled(sb(c), sb(s), P(4098), *good) == E.EA_ERR_ALIGN
    assert E.lib.ea_step_scheduled(sb(c), sb(bad), P(4096), *good) == E.EA_ERR_ARG
    assert E.lib.ea_step_scheduled(sb(c), sb(s), P(4096), None, *good[1:]) == E.EA_ERR_ARG
    # multi-step run: steps, first step, stride and schedule are checked up front
    g0, rest = good[0], good[1:]
    assert E.lib.ea_run(sb(c), sb(s), 1, -1, g0, 0, *rest) == E.EA_ERR_ARG
    assert E.lib.ea_run(sb(c), sb(s), 0, 3, g0, 0, *rest) == E.EA_ERR_ARG
    assert E.lib.ea_run(sb(c), sb(s), 2 ** 32 - 2, 3, g0, 0, *rest) == E.EA_ERR_ARG
    assert E.lib.ea_run(sb(c), sb(s), 1, 3, g0, -5, *rest) == E.EA_ERR_ARG
    assert E.lib.ea_run(sb(c), sb(bad), 1, 3, g0, 0, *rest) == E.EA_ERR_ARG
    assert E.lib.ea_run(sb(c), sb(s), 1, 3, None, 0, *rest) == E.EA_ERR_ARG
    assert E.lib.ea_run(sb(c), sb(s), 1, 0, g0, 0, *rest) == E.EA_OK   # nothing to do


def test_toy_grad_rejected_before_device_work(E):
    torch = pytest.importorskip("torch")
    if torch.cuda.device_count() > 0:
        pytest.skip("bogus-pointer rejection test runs on GPU-less hosts only")
    P = ctypes.c_void_p
    p = [P(4096 * (k + 1)) for k in range(5)]     # A, x_star, xi, x, g
    ws = P(1 << 20)
    assert E.lib.ea_toy_grad(0, 2, *p, None, ws, None) == E.EA_ERR_ARG
    assert E.lib.ea_toy_grad(65537, 2, *p, None, ws, None) == E.EA_ERR_ARG
    assert E.lib.ea_toy_grad(500, 0, *p, None, ws, None) == E.EA_ERR_ARG
    assert E.lib.ea_toy_grad(500, 1025, *p, None, ws, None) == E.EA_ERR_ARG
    assert E.lib.ea_toy_grad(500, 10, None, *p[1:], None, ws, None) == E.EA_ERR_ARG
    assert E.lib.ea_toy_grad(500, 10, *p[:4], P(4098), None, ws, None) == E.EA_ERR_ALIGN
    assert E.lib.ea_toy_grad(500, 10, *p, P(4100), ws, None) == E.EA_ERR_ALIGN
    assert E.lib.ea_toy_grad(500, 10, *p, None, None, None) == E.EA_ERR_ARG
    assert E.lib.ea_toy_grad(500, 10, *p, None, P(4100), None) == E.EA_ERR_ALIGN
    # r, per-block norms, 1 + 8 counters (five doubles), and at d = 500 the
    # fused round's row splits: 8 column groups x 8 splits of 64 rows, 16
    # column sums of 64 columns each
    assert E.ea_toy_workspace_bytes(500) == 8 * (500 + 8 + 5 + 8 * 8 * 16 * 64)
    # the column groups alone fill the GPU: no splits
    assert E.ea_toy_workspace_bytes(65536) == 8 * (65536 + 1024 + 513)
    with pytest.raises(E.EAError):
        E.ea_toy_workspace_bytes(0)


def test_noalloc_scratch_limit_matches_header_and_rejects_before_device_work(E):
    src = open(os.path.join(ROOT, "include", "ea.h")).read()
    m = re.search(r"#define EA_NOALLOC_SCRATCH_BYTES \((\d+) << (\d+)\)", src)
    assert m and int(m.group(1)) << int(m.group(2)) == E.EA_NOALLOC_SCRATCH_BYTES
    q = E.Quant(kind=1, scale=0, bits=1, error_feedback=1, bucket=0)
    c = E.Config(d=8_000_000, N=4, placement=0, beta1=0.9, beta2=0.999, lr=1e-3, eps=1e-8, seed=1, qw=q, qs=q)
    assert E.ea_workspace_bytes(c) > E.EA_NOALLOC_SCRATCH_BYTES
    # fake device pointers: the call must fail on the size before it touches any
    with pytest.raises(E.EAError) as ei:
        E.ea_step_noalloc(c, 1, *([1 << 20] * 12), stream=0)
    assert ei.value.code == E.EA_ERR_UNSUPPORTED and "scratch" in E.ea_last_error()


def test_toy_step_rejects_scaled_quantizers_before_device_work(E):
    q = E.Quant(kind=3, bits=2, error_feedback=1, bucket=0)      # Example 1: one max-norm scale
    c = E.Config(d=500, N=10, placement=1, beta1=0.9, beta2=0.99, lr=1e-4, eps=1e-8, seed=1, qw=q, qs=q)
    with pytest.raises(E.EAError) as ei:
        E.ea_toy_step(c, 1, *([1 << 20] * 15), stream=0)
    assert ei.value.code == E.EA_ERR_UNSUPPORTED
    q2 = E.Quant(kind=4, error_feedback=1, pow2_kmin=-17, pow2_kmax=-11)
    c2 = E.Config(d=70000, N=10, placement=1, beta1=0.9, beta2=0.99, lr=1e-4, eps=1e-8, seed=1, qw=q2, qs=q2)
    with pytest.raises(E.EAError) as ei:
        E.ea_toy_step(c2, 1, *([1 << 20] * 15), stream=0)
    assert ei.value.code == E.EA_ERR_ARG


def test_random_quantizer_fields(E):
    """2,000 seeded random quantizer records, valid and invalid: validation
    never fails without a message, accepts exactly the records the header's
    rules allow, and every accepted record's message sizes agree with the
    oracle's at random d."""
    import numpy as np
    rng = np.random.default_rng(99)
    ok_count = 0
    for _ in range(2000):
        qd = dict(kind=int(rng.integers(-1, 8)), scale=int(rng.integers(-1, 4)), bits=int(rng.integers(-1, 34)),
                  error_feedback=int(rng.integers(-1, 3)), bucket=int(rng.choice([-256, 0, 128, 256, 512, 768, 1024,
                                                                                  2048, 4096, 1 << 20])),
                  pow2_kmin=int(rng.integers(-130, 10)), pow2_kmax=int(rng.integers(-130, 130)),
                  keep=int(rng.integers(-1, 2100)))
        d = int(rng.integers(1, 1 << 21))
        cfg = _cfg(E, d=d, qw=E.Quant(**qd))
        rc = E.ea_validate(cfg)
        if rc != 0:
            assert rc in (-1, -4), (qd, rc)
            assert E.ea_last_error() != ""
            continue
        ok_count += 1
        k, b, B = qd["kind"], qd["bits"], qd["bucket"]
        # what the header allows (a bucket >= d is one bucket)
        assert k in (0, 1, 2, 3, 4, 5, 6), qd
        assert qd["error_feedback"] in (0, 1), qd
        if k == 2:
            assert b in (1, 2, 4, 8) and qd["scale"] in (1, 2), qd
        if k == 3:
            assert 2 <= b <= 8, qd
        if k == 4:
            assert -126 <= qd["pow2_kmin"] < qd["pow2_kmax"] <= 127, qd
        if k in (1, 2, 3):
            assert B in (0, 256, 512, 1024, 2048) or B >= d, qd
        if k in (5, 6):
            assert (B in (256, 512, 1024, 2048) or B >= d) and 1 <= qd["keep"] <= min(B, max(B, d)), qd
        qo = O.Quant(**qd)
        qe = E.Quant(**qd)
        assert E.ea_code_bits(qe) == O.code_bits(qo), qd
        assert E.ea_msg_words(qe, d) == O.msg_words(qo, d), (qd, d)
        assert E.ea_msg_scales(qe, d) == O.num_scales(qo, d, d), (qd, d)
    assert ok_count > 100
