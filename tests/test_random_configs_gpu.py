"""Seeded random configurations of the whole round against the oracle: the
quantizer kind, code width, norm, bucket (or one bucket) and error feedback
of each side drawn independently, 1 to 24 workers, tiny to mid-size d with
ragged tails, either Adam placement, fused or split calls.  Every message and
state array after every step must equal the oracle's bit for bit; the cases
reach the kernel tiers in combinations the targeted tests may not."""
import numpy as np
import pytest

import oracle as O
import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU-only host
    pytest.skip("needs a GPU", allow_module_level=True)

from parity_util import Pair, qfields  # noqa: E402

BUCKETS = [0, 256, 512, 1024, 2048]
SPARSE_BUCKETS = [256, 512, 1024, 2048]


def _quant(rng):
    kind = rng.choice(["sign", "stoch", "stoch", "det", "pow2", "none", "topk", "randk"])
    ef = 0 if rng.random() < 0.15 else 1
    if kind == "sign":
        return f"sign{int(b := rng.choice(BUCKETS))}", qfields(O.Q_SCALED_SIGN, 1, O.SCALE_L1, ef, int(b))
    if kind == "stoch":
        bits = int(rng.choice([1, 2, 4, 8]))
        sc = int(rng.choice([O.SCALE_L2, O.SCALE_MAX]))
        b = int(rng.choice(BUCKETS))
        return f"stoch{bits}{'l2' if sc == O.SCALE_L2 else 'max'}_{b}", qfields(O.Q_STOCH_UNIFORM, bits, sc, ef, b)
    if kind == "det":
        bits = int(rng.integers(2, 9))
        b = int(rng.choice(BUCKETS))
        return f"ex1b{bits}_{b}", qfields(O.Q_DET_UNIFORM, bits, ef=ef, bucket=b)
    if kind == "pow2":
        kmin = int(rng.integers(-40, -4))
        kmax = kmin + int(rng.integers(1, 30))
        return f"ex2[{kmin},{kmax}]", qfields(O.Q_POW2, ef=ef, kmin=kmin, kmax=kmax)
    if kind == "none":
        return "none", qfields(O.Q_NONE, ef=ef)
    b = int(rng.choice(SPARSE_BUCKETS))
    keep = int(rng.integers(1, b + 1)) if rng.random() < 0.3 else int(rng.integers(1, max(2, b // 16)))
    q = O.Q_TOPK if kind == "topk" else O.Q_RANDK
    return f"{kind}{keep}of{b}", qfields(q, ef=ef, bucket=b, keep=keep)


def _cases(n, seed=2024):
    rng = np.random.default_rng(seed)
    out = []
    for j in range(n):
        shape = rng.integers(0, 3)
        d = (int(rng.integers(1, 700)) if shape == 0 else
             256 * int(rng.integers(1, 40)) + int(rng.integers(0, 256)) if shape == 1 else
             2048 * int(rng.integers(1, 8)) + int(rng.integers(0, 2048)))
        N = int(rng.integers(1, 25))
        nw, qw = _quant(rng)
        ns, qs = _quant(rng)
        placement = int(rng.choice([O.ADAM_AT_SERVER, O.ADAM_AT_WORKER]))
        split = bool(rng.random() < 0.25)
        gen = str(rng.choice(["student_t", "outliers", "segscale"]))
        out.append(pytest.param(d, N, qw, qs, placement, split, gen, 100 + j,
                                id=f"{j}-d{d}-N{N}-{nw}-{ns}-{'srv' if placement == 0 else 'wrk'}"
                                   f"{'-split' if split else ''}"))
    return out


@pytest.mark.parametrize("d,N,qw,qs,placement,split,gen,seed", _cases(48))
def test_random_config(d, N, qw, qs, placement, split, gen, seed):
    pair = Pair(d, N, qw, qs, placement, seed=seed, split=split)
    for t in range(1, 3):
        w = W.Workload("r", "r", d, N, None, None, 1, seed, gen)
        pair.step(t, W.host_gradients(w, t, d=d))
    pair.check_tie_budget()
    assert pair.stats.resyncs == 0


# The quantizer pairs of the fully specialized kernels (the benchmark shapes).
SPECIAL_PAIRS = [
    ("stoch4l2_512", qfields(O.Q_STOCH_UNIFORM, 4, O.SCALE_L2, 1, 512), qfields(O.Q_STOCH_UNIFORM, 4, O.SCALE_L2, 1, 512)),
    ("stoch2max_512", qfields(O.Q_STOCH_UNIFORM, 2, O.SCALE_MAX, 1, 512),
     qfields(O.Q_STOCH_UNIFORM, 2, O.SCALE_MAX, 1, 512)),
    ("stoch2max_1024/sign1024", qfields(O.Q_STOCH_UNIFORM, 2, O.SCALE_MAX, 1, 1024),
     qfields(O.Q_SCALED_SIGN, 1, O.SCALE_L1, 1, 1024)),
    ("sign2048", qfields(O.Q_SCALED_SIGN, 1, O.SCALE_L1, 1, 2048), qfields(O.Q_SCALED_SIGN, 1, O.SCALE_L1, 1, 2048)),
    ("topk16_512", qfields(O.Q_TOPK, bucket=512, keep=16), qfields(O.Q_TOPK, bucket=512, keep=16)),
    ("randk16_512", qfields(O.Q_RANDK, bucket=512, keep=16), qfields(O.Q_RANDK, bucket=512, keep=16)),
    ("topk64_2048", qfields(O.Q_TOPK, bucket=2048, keep=64), qfields(O.Q_TOPK, bucket=2048, keep=64)),
    ("randk64_2048", qfields(O.Q_RANDK, bucket=2048, keep=64), qfields(O.Q_RANDK, bucket=2048, keep=64)),
]


def _special_cases(n, seed=2025):
    rng = np.random.default_rng(seed)
    out = []
    for j in range(n):
        name, qw, qs = SPECIAL_PAIRS[j % len(SPECIAL_PAIRS)]
        d = 2048 * int(rng.integers(1, 40)) + int(rng.integers(0, 2048)) // 4 * 4 + (0 if rng.random() < 0.8 else 1)
        N = int(rng.choice([1, 2, 3, int(rng.integers(4, 17)), int(rng.integers(17, 41))]))
        placement = int(rng.choice([O.ADAM_AT_SERVER, O.ADAM_AT_WORKER]))
        out.append(pytest.param(d, N, qw, qs, placement, 300 + j,
                                id=f"{j}-{name}-d{d}-N{N}-{'srv' if placement == 0 else 'wrk'}"))
    return out


@pytest.mark.parametrize("d,N,qw,qs,placement,seed", _special_cases(32))
def test_random_specialized_shapes(d, N, qw, qs, placement, seed):
    """The benchmark shapes' quantizer pairs (fully specialized kernels) with
    random worker counts (1 to 40: one wave per tile or per worker, several
    worker groups) and sizes (aligned or not, with ragged tails)."""
    pair = Pair(d, N, qw, qs, placement, seed=seed)
    for t in range(1, 3):
        w = W.Workload("r", "r", d, N, None, None, 1, seed, "student_t")
        pair.step(t, W.host_gradients(w, t, d=d))
    pair.check_tie_budget()
    assert pair.stats.resyncs == 0


SCHEDULES = [
    dict(kind=O.SCHED_CONSTANT),
    dict(kind=O.SCHED_ASSUMPTION2, alpha=2e-3, theta=0.99, T=400),
    dict(kind=O.SCHED_STEP_DECAY, alpha=1e-3, factor=0.5, period=1),
]


def _scheduled_cases(n, seed=2026, modes=("scheduled", "run")):
    rng = np.random.default_rng(seed)
    out = []
    for j in range(n):
        d = (int(rng.integers(1, 700)) if j % 3 == 0 else 512 * int(rng.integers(1, 30)) + int(rng.integers(0, 512)))
        N = int(rng.integers(1, 21))
        nw, qw = _quant(rng)
        ns, qs = _quant(rng)
        placement = int(rng.choice([O.ADAM_AT_SERVER, O.ADAM_AT_WORKER]))
        sched = int(rng.integers(0, len(SCHEDULES)))
        mode = modes[j % len(modes)]
        out.append(pytest.param(d, N, qw, qs, placement, sched, mode, 500 + j,
                                id=f"{j}-d{d}-N{N}-{nw}-{ns}-{'srv' if placement == 0 else 'wrk'}-s{sched}-{mode}"))
    return out


@pytest.mark.parametrize("d,N,qw,qs,placement,sched,mode,seed",
                         _scheduled_cases(16) + _scheduled_cases(8, seed=2027, modes=("graph",)))
def test_random_scheduled_rounds(d, N, qw, qs, placement, sched, mode, seed):
    """Random configurations through ea_step_scheduled (the step read on the
    device, lr_t and beta2_t from the schedule in the kernels), ea_run, and a
    HIP graph of ea_step_scheduled captured once and replayed every step
    (eager copies and synchronizations between the replays), three steps
    each, against the oracle's own schedule."""
    pair = Pair(d, N, qw, qs, placement, seed=seed, sched=SCHEDULES[sched], mode=mode)
    for t in range(1, 4):
        w = W.Workload("r", "r", d, N, None, None, 1, seed, "student_t")
        pair.step(t, W.host_gradients(w, t, d=d))
    pair.check_tie_budget()
    assert pair.stats.resyncs == 0
