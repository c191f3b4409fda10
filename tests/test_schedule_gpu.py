"""GPU parity of the scheduled and multi-step calls: ea_step_scheduled (step
index read on the device, lr_t and beta2_t from Assumption 2 or the Section
V-B step decay), ea_run, and a HIP-graph capture of ea_step_scheduled replayed
step after step.  The oracle takes the same steps with lr_t, beta2_t from its
own schedule code; comparison rules are those of tests/parity_util.py."""
import numpy as np
import pytest

import oracle as O
import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU-only host
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2205_14473_amd as E  # noqa: E402
from parity_util import Pair, Stats, close, configs, first_diff, qfields, same_values  # noqa: E402

SIGN = lambda b, ef=1: qfields(O.Q_SCALED_SIGN, 1, O.SCALE_L1, ef, b)  # noqa: E731
STOCH = lambda bits, sc, b, ef=1: qfields(O.Q_STOCH_UNIFORM, bits, sc, ef, b)  # noqa: E731

SCHEDS = {
    "constant": dict(kind=O.SCHED_CONSTANT),
    "assumption2": dict(kind=O.SCHED_ASSUMPTION2, alpha=2e-3, theta=0.99, T=400),
    "step_decay": dict(kind=O.SCHED_STEP_DECAY, alpha=1e-3, factor=0.2, period=2),
}
CASES = {
    # specialized whole-tile kernels (two tiles per block) plus the ragged tail
    "bert_like": (512 * 5 + 300, 16, STOCH(4, O.SCALE_L2, 512), STOCH(4, O.SCALE_L2, 512), O.ADAM_AT_SERVER),
    # generic kernels, Adam at the workers
    "generic_worker": (3000, 4, qfields(O.Q_DET_UNIFORM, 3, bucket=256), SIGN(512), O.ADAM_AT_WORKER),
    # one-bucket quantizers: norm kernels before and after the round
    "one_bucket": (4096, 3, SIGN(0), STOCH(2, O.SCALE_MAX, 0), O.ADAM_AT_SERVER),
}


def _grads(seed, t, N, d):
    w = W.Workload("t", "t", d, N, None, None, 1, seed, "student_t")
    return W.host_gradients(w, t, d=d)


def _run(case, sched, mode, T=6, first_mode=None):
    d, N, qw, qs, pl = CASES[case]
    pair = Pair(d, N, qw, qs, pl, seed=11, sched=SCHEDS[sched], mode=first_mode or mode)
    for t in range(1, T + 1):
        if t == 2:
            pair.mode = mode
        pair.step(t, _grads(11, t, N, d))
    pair.check_tie_budget()
    print(f"\n[sched] {case} {sched} {mode}: {pair.stats}", flush=True)
    return pair


@pytest.mark.parametrize("sched", list(SCHEDS))
@pytest.mark.parametrize("case", list(CASES))
def test_scheduled_step_reads_the_device_counter(case, sched):
    _run(case, sched, "scheduled")


@pytest.mark.parametrize("sched", ["assumption2", "step_decay"])
def test_run_one_step_per_call(sched):
    _run("bert_like", sched, "run")
    _run("generic_worker", sched, "run")


@pytest.mark.parametrize("sched", ["constant", "step_decay"])
@pytest.mark.parametrize("case", ["bert_like", "one_bucket"])
def test_graph_replay_takes_the_next_step(case, sched):
    """Step 1 runs eagerly (it also initializes the library's per-device
    caches); step 2 is captured into a HIP graph, and every later step is a
    replay, with eager copies, synchronizations and comparisons in between."""
    _run(case, sched, "graph", T=7, first_mode="scheduled")


def test_run_many_steps_in_one_call():
    """One ea_run call over T rounds with a [T][N][d] gradient array, against
    the oracle's T rounds: the state after the last round is bit-identical."""
    d, N, T = 2048 + 256, 4, 8
    sd = dict(kind=O.SCHED_STEP_DECAY, alpha=1e-3, factor=0.5, period=3)
    oc, ec = configs(d, N, SIGN(512), SIGN(512), O.ADAM_AT_SERVER, seed=5)
    so, se = O.Schedule(**sd), E.Schedule(**sd)
    from paper_2205_14473_amd.state import allocate, init_state
    rb = allocate(ec)
    init_state(ec, rb)
    st = O.State.init(oc, d)
    gs = np.stack([_grads(5, t, N, d) for t in range(1, T + 1)])
    for t in range(1, T + 1):
        c = O.Config.from_buffer_copy(oc)
        c.lr, c.beta2 = (float(v) for v in O.schedule_at(so, oc.lr, oc.beta2, t))
        out = O.step(c, t, gs[t - 1], st)
    g_dev = torch.from_numpy(gs).cuda()
    args = rb.step_args()
    args.pop("g")
    E.ea_run(ec, se, 1, T, g_dev, N * d, **args)
    torch.cuda.synchronize()
    stats = Stats()
    for name in ("x", "m", "v", "e_s", "e_w"):
        got, want = getattr(rb, name).cpu().numpy(), getattr(st, name)
        assert same_values(got, want), f"{name} after {T} steps: {first_diff(got, want)}"
        close(name, got, want, stats)
    # the messages left behind are the last round's
    words = E.ea_msg_words(ec.qs, d)
    assert np.array_equal(rb.scodes.cpu().numpy()[:words], out["scodes"])
    print(f"\n[sched] ea_run {T} steps: {stats}", flush=True)
