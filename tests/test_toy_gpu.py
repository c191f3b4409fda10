"""GPU parity of the Section V-A toy problem's gradient producer
(ea_toy_grad) against the oracle, and Figure 1's setting run on the device:
each step the workers' gradients come from ea_toy_grad at the current x and
feed the round, while the oracle runs the same steps."""
import math

import numpy as np
import pytest

import oracle as O

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU-only host
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2205_14473_amd as E  # noqa: E402
from parity_util import Pair, qfields  # noqa: E402


def _inputs(d, N, seed):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((d, d)).astype(np.float32)
    xs = (rng.standard_normal(d) * math.sqrt(0.1)).astype(np.float32)
    xi = (rng.standard_normal((N, d)) * math.sqrt(0.1)).astype(np.float32)
    x = rng.standard_normal(d).astype(np.float32)
    return A, xs, xi, x


def _gpu_grad(A, xs, xi, x):
    d, N = A.shape[0], xi.shape[0]
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    g = torch.empty((N, d), dtype=torch.float32, device="cuda")
    gs = torch.zeros(1, dtype=torch.float64, device="cuda")
    ws = torch.empty(E.ea_toy_workspace_bytes(d), dtype=torch.uint8, device="cuda")
    E.ea_toy_grad(d, N, dev(A), dev(xs), dev(xi), dev(x), g, gs, ws)
    torch.cuda.synchronize()
    return g.cpu().numpy(), float(gs.item())


def _check(got, want, gs_got, gs_want):
    # binary64 sums in another order: the binary32 results agree to the
    # rounding of the last place
    scale = np.max(np.abs(want))
    assert np.all(np.abs(got - want) <= 1e-6 * np.abs(want) + 1e-9 * scale)
    assert gs_got == pytest.approx(gs_want, rel=1e-12)


@pytest.mark.parametrize("d,N,seed", [(1, 1, 0), (7, 3, 1), (64, 8, 2), (65, 9, 8), (500, 10, 3), (1000, 17, 4),
                                      (4099, 2, 5), (8192, 1, 6)])
def test_toy_grad_matches_oracle(d, N, seed):
    A, xs, xi, x = _inputs(d, N, seed)
    g, gs = _gpu_grad(A, xs, xi, x)
    go, gso = O.toy_grad(A, xs, xi, x)
    _check(g, go, gs, gso)
    print(f"\n[toy] d={d} N={N}: exact entries {np.mean(g == go):.6f}", flush=True)


def test_toy_grad_without_norm():
    A, xs, xi, x = _inputs(300, 4, 7)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    g = torch.empty((4, 300), dtype=torch.float32, device="cuda")
    ws = torch.empty(E.ea_toy_workspace_bytes(300), dtype=torch.uint8, device="cuda")
    E.ea_toy_grad(300, 4, dev(A), dev(xs), dev(xi), dev(x), g, None, ws)
    torch.cuda.synchronize()
    go, _ = O.toy_grad(A, xs, xi, x, want_norm=False)
    _check(g.cpu().numpy(), go, 0.0, 0.0)


@pytest.mark.parametrize("example", ["ex1", "ex2"])
def test_figure1_setting_on_device(example):
    """Section V-A: d = 500, 10 workers, Adam at the workers, beta = 0.9,
    theta = 0.99, Example 1 (k = 1) or Example 2 (k = -17, K = -11); the
    gradients come from ea_toy_grad at the GPU's x each step."""
    d, N, T, lr = 500, 10, 40, 1e-4
    rng = np.random.default_rng(21)
    A = rng.standard_normal((d, d)).astype(np.float32)
    xs = (rng.standard_normal(d) * math.sqrt(0.1)).astype(np.float32)
    if example == "ex1":
        q = qfields(O.Q_DET_UNIFORM, 2, bucket=0)
    else:
        q = qfields(O.Q_POW2, kmin=-17, kmax=-11)
    pair = Pair(d, N, q, q, O.ADAM_AT_WORKER, seed=21, beta1=0.9, beta2=0.99, lr=lr)
    A_d, xs_d = torch.from_numpy(A).cuda(), torch.from_numpy(xs).cuda()
    g_d = torch.empty((N, d), dtype=torch.float32, device="cuda")
    gs_d = torch.zeros(1, dtype=torch.float64, device="cuda")
    ws = torch.empty(E.ea_toy_workspace_bytes(d), dtype=torch.uint8, device="cuda")
    norms = []
    for t in range(1, T + 1):
        xi = (rng.standard_normal((N, d)) * math.sqrt(0.1)).astype(np.float32)
        xi_d = torch.from_numpy(xi).cuda()
        E.ea_toy_grad(d, N, A_d, xs_d, xi_d, pair.rb.x, g_d, gs_d, ws)
        torch.cuda.synchronize()
        go, gso = O.toy_grad(A, xs, xi, pair.ost.x)
        _check(g_d.cpu().numpy(), go, float(gs_d.item()), gso)
        norms.append(gso)
        pair.step(t, go)        # the round on the same gradients, both sides
    pair.check_tie_budget()
    assert norms[-1] < norms[0]
    print(f"\n[toy] figure-1 setting {example}: |grad F|^2 {norms[0]:.4g} -> {norms[-1]:.4g}; {pair.stats}",
          flush=True)


# ---------------------------------------------------------------------------
# ea_toy_step: the gradient producer fused into the round.
# ---------------------------------------------------------------------------
from paper_2205_14473_amd.state import allocate, init_state  # noqa: E402
from parity_util import RoundCheck, Stats, configs  # noqa: E402

EX2 = qfields(O.Q_POW2, kmin=-17, kmax=-11)
NONE = qfields(O.Q_NONE)
FUSED = [(500, 10, EX2, O.ADAM_AT_WORKER), (500, 10, NONE, O.ADAM_AT_SERVER), (500, 10, EX2, O.ADAM_AT_SERVER),
         (64, 3, EX2, O.ADAM_AT_SERVER), (65, 1, EX2, O.ADAM_AT_WORKER), (1000, 17, EX2, O.ADAM_AT_WORKER),
         (777, 31, NONE, O.ADAM_AT_WORKER), (3000, 4, EX2, O.ADAM_AT_SERVER), (1, 2, EX2, O.ADAM_AT_WORKER),
         (300, 15, EX2, O.ADAM_AT_WORKER), (300, 16, NONE, O.ADAM_AT_SERVER), (520, 6, EX2, O.ADAM_AT_SERVER),
         (4096, 3, EX2, O.ADAM_AT_WORKER)]


def _ulps(a, b):
    ai = np.asarray(a, np.float32).view(np.int32).astype(np.int64)
    bi = np.asarray(b, np.float32).view(np.int32).astype(np.int64)
    ai = np.where(ai < 0, -(ai & 0x7FFFFFFF), ai)
    bi = np.where(bi < 0, -(bi & 0x7FFFFFFF), bi)
    return np.abs(ai - bi)


@pytest.mark.parametrize("d,N,q,placement", FUSED,
                         ids=[f"d{d}-N{N}-{'ex2' if q['kind'] == O.Q_POW2 else 'full'}-"
                              f"{'worker' if p == O.ADAM_AT_WORKER else 'server'}" for d, N, q, p in FUSED])
def test_toy_step_equals_gradient_then_round(d, N, q, placement):
    """Each step: the fused call's gradients (read back through g_out) equal
    the oracle's toy gradient at the same x to the last place (binary64 sums
    in another order), its squared norm to 1e-12, and the round on those
    gradients equals the oracle's round on them bit for bit."""
    rng = np.random.default_rng(d * 131 + N)
    A = rng.standard_normal((d, d)).astype(np.float32)
    xs = (rng.standard_normal(d) * math.sqrt(0.1)).astype(np.float32)
    x1 = (rng.standard_normal(d) * 0.01).astype(np.float32)
    lr = 1e-4 if q["kind"] == O.Q_POW2 else 1e-3
    oc, ec = configs(d, N, q, q, placement, seed=9, beta1=0.9, beta2=0.99, lr=lr)
    rb = allocate(ec)
    init_state(ec, rb)
    rb.x.copy_(torch.from_numpy(x1))
    st = O.State.init(oc, d, x1)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    A_d, xs_d = dev(A), dev(xs)
    g_d = torch.empty((N, d), dtype=torch.float32, device="cuda")
    gs_d = torch.zeros(1, dtype=torch.float64, device="cuda")
    ws = torch.empty(E.ea_toy_workspace_bytes(d), dtype=torch.uint8, device="cuda")
    stats = Stats()
    worst = 0
    for t in range(1, 7):
        xi = (rng.standard_normal((N, d)) * math.sqrt(0.1)).astype(np.float32)
        E.ea_toy_step(ec, t, A_d, xs_d, dev(xi), rb.e_w, rb.m_w, rb.v_w, rb.m, rb.v, rb.e_s, rb.x, rb.wcodes,
                      rb.scodes, gs_d, g_d, ws)
        torch.cuda.synchronize()
        g = g_d.cpu().numpy()
        go, gso = O.toy_grad(A, xs, xi, st.x)
        u = _ulps(g, go)
        worst = max(worst, int(u.max()))
        assert u.max() <= 1, f"step {t}: gradient differs from the oracle's by {u.max()} ulps"
        assert float(gs_d.item()) == pytest.approx(gso, rel=1e-12)
        out = O.step(oc, t, g, st, want_inputs=True)
        chk = RoundCheck(oc, d, 0, t, out, stats, what=f"step {t}: ")
        none = np.zeros((N, 0), np.float32)
        chk.messages(rb.wcodes.cpu().numpy(), none, rb.scodes.cpu().numpy(), none[0])
        host = lambda a: None if a is None else a.cpu().numpy()  # noqa: E731
        chk.state({k: host(getattr(rb, k)) for k in ("e_w", "e_s", "x", "m", "v", "m_w", "v_w")}, st)
        assert not chk.tied
        stats.steps += 1
    print(f"\n[toy step] d={d} N={N}: gradients within {worst} ulp; rounds bit-exact; {stats}", flush=True)


def test_toy_step_optional_outputs_change_nothing():
    """Without g_out and grad_sq the fused call leaves the same bits."""
    d, N = 500, 10
    rng = np.random.default_rng(5)
    A = torch.from_numpy(rng.standard_normal((d, d)).astype(np.float32)).cuda()
    xs = torch.from_numpy((rng.standard_normal(d) * 0.3).astype(np.float32)).cuda()
    _, ec = configs(d, N, EX2, EX2, O.ADAM_AT_WORKER, seed=9, beta1=0.9, beta2=0.99, lr=1e-4)
    a, b = allocate(ec), allocate(ec)
    for rb in (a, b):
        init_state(ec, rb)
        rb.x.zero_()
    ws_a = torch.empty(E.ea_toy_workspace_bytes(d), dtype=torch.uint8, device="cuda")
    ws_b = torch.empty_like(ws_a)
    g = torch.empty((N, d), dtype=torch.float32, device="cuda")
    gs = torch.zeros(1, dtype=torch.float64, device="cuda")
    for t in range(1, 5):
        xi = torch.from_numpy((rng.standard_normal((N, d)) * 0.3).astype(np.float32)).cuda()
        E.ea_toy_step(ec, t, A, xs, xi, a.e_w, a.m_w, a.v_w, a.m, a.v, a.e_s, a.x, a.wcodes, a.scodes, gs, g, ws_a)
        E.ea_toy_step(ec, t, A, xs, xi, b.e_w, b.m_w, b.v_w, b.m, b.v, b.e_s, b.x, b.wcodes, b.scodes, None, None,
                      ws_b)
    torch.cuda.synchronize()
    for k in ("e_w", "m_w", "v_w", "e_s", "x", "wcodes", "scodes"):
        assert torch.equal(getattr(a, k).view(torch.uint8), getattr(b, k).view(torch.uint8)), k


@pytest.mark.parametrize("d,N", [(500, 10), (300, 16)], ids=["split-rows", "one-split"])
def test_toy_steps_replayed_from_a_graph(d, N):
    """Five toy steps captured into a HIP graph (both launches of every step;
    the round's counters are cleared by a kernel, not a memset) and replayed
    three times from the same start, with eager resets and synchronizations
    between the replays: every replay leaves the bits that the same five
    steps leave when run eagerly."""
    rng = np.random.default_rng(d + N)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    A = dev(rng.standard_normal((d, d)).astype(np.float32))
    xs = dev((rng.standard_normal(d) * math.sqrt(0.1)).astype(np.float32))
    xi = dev((rng.standard_normal((5, N, d)) * math.sqrt(0.1)).astype(np.float32))
    _, ec = configs(d, N, EX2, EX2, O.ADAM_AT_WORKER, seed=9, beta1=0.9, beta2=0.99, lr=1e-4)
    rb = allocate(ec)
    init_state(ec, rb)
    rb.x.copy_(dev((rng.standard_normal(d) * 0.01).astype(np.float32)))
    keys = [k for k in ("e_w", "m_w", "v_w", "m", "v", "e_s", "x", "wcodes", "scodes") if getattr(rb, k) is not None]
    start = {k: getattr(rb, k).clone() for k in keys}
    gs = torch.zeros(5, dtype=torch.float64, device="cuda")
    ws = torch.empty(E.ea_toy_workspace_bytes(d), dtype=torch.uint8, device="cuda")

    def steps():
        for t in range(1, 6):
            E.ea_toy_step(ec, t, A, xs, xi[t - 1], rb.e_w, rb.m_w, rb.v_w, rb.m, rb.v, rb.e_s, rb.x, rb.wcodes,
                          rb.scodes, gs[t - 1:t], None, ws)

    def reset():
        for k in keys:
            getattr(rb, k).copy_(start[k])
        gs.zero_()
        torch.cuda.synchronize()

    steps()
    torch.cuda.synchronize()
    want = {k: getattr(rb, k).clone() for k in keys}
    want_gs = gs.clone()
    reset()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        steps()
    torch.cuda.synchronize()
    for rep in range(3):
        reset()
        graph.replay()
        torch.cuda.synchronize()
        for k in keys:
            assert torch.equal(getattr(rb, k).view(torch.uint8), want[k].view(torch.uint8)), (rep, k)
        assert torch.equal(gs, want_gs), rep


@pytest.mark.parametrize("d,N", [(500, 10), (777, 31), (65, 2)], ids=["split-rows", "two-passes", "ragged"])
def test_toy_grad_equals_fused_step_gradients(d, N):
    """ea_toy_grad and ea_toy_step (through g_out) sum in the same order: the
    same gradients bit for bit, and the same ||grad F||^2."""
    A, xs, xi, x = _inputs(d, N, 11)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    g, gs = _gpu_grad(A, xs, xi, x)
    _, ec = configs(d, N, EX2, EX2, O.ADAM_AT_WORKER, seed=9, beta1=0.9, beta2=0.99, lr=1e-4)
    rb = allocate(ec)
    init_state(ec, rb)
    rb.x.copy_(dev(x))
    g2 = torch.empty((N, d), dtype=torch.float32, device="cuda")
    gs2 = torch.zeros(1, dtype=torch.float64, device="cuda")
    ws = torch.empty(E.ea_toy_workspace_bytes(d), dtype=torch.uint8, device="cuda")
    E.ea_toy_step(ec, 1, dev(A), dev(xs), dev(xi), rb.e_w, rb.m_w, rb.v_w, rb.m, rb.v, rb.e_s, rb.x, rb.wcodes,
                  rb.scodes, gs2, g2, ws)
    torch.cuda.synchronize()
    assert np.array_equal(g.view(np.uint32), g2.cpu().numpy().view(np.uint32))
    assert gs == float(gs2.item())
