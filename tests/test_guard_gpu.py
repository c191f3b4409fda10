"""Writes stay inside the buffers the header sizes: every array an entry point
(the round, the no-allocation round, the scheduled round and the multi-step
run, the four split calls, the toy calls) writes (state, messages, scales,
workspace, the step counter) is placed at the front of a
larger allocation filled with a byte pattern, and after the calls every byte
past the array's end still holds the pattern.  The configurations cover a
ragged last tile, two-tile blocks, 8-chunk tiles, whole-vector scales (the
workspace's partial sums), sparse messages, raw messages, the no-allocation
round and the toy problem's split-row workspace."""
import math

import numpy as np
import pytest

import oracle as O

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU-only host
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2205_14473_amd as E  # noqa: E402
from paper_2205_14473_amd.state import allocate, init_state  # noqa: E402
from parity_util import configs, qfields  # noqa: E402

GUARD = 4096
PATTERN = 0xA5


class Guarded:
    """Tensors viewed from the front of larger pattern-filled allocations."""

    def __init__(self, pattern=PATTERN):
        self.bufs = {}
        self.pattern = pattern

    def wrap(self, name, t):
        if t is None:
            return None
        nbytes = t.numel() * t.element_size()
        big = torch.full((nbytes + GUARD,), self.pattern, dtype=torch.uint8, device="cuda")
        view = big[:nbytes].view(t.dtype).view(t.shape)
        view.copy_(t)
        self.bufs[name] = (big, nbytes)
        return view

    def check(self, what):
        torch.cuda.synchronize()
        for name, (big, nbytes) in self.bufs.items():
            tail = big[nbytes:]
            bad = int((tail != self.pattern).sum().item())
            assert bad == 0, f"{what}: {bad} bytes written past the end of {name} ({nbytes} bytes)"


def _step_args(ec, rb, gd):
    args = rb.step_args()
    nsw, nss = E.ea_msg_scales(ec.qw, ec.d), E.ea_msg_scales(ec.qs, ec.d)
    args["wscales"] = args["wscales"][:, :nsw] if nsw else None
    args["sscales"] = args["sscales"][:nss] if nss else None
    out = {}
    for k, t in args.items():
        out[k] = gd.wrap(k, t.contiguous() if t is not None else None)
    return out


ROUNDS = [
    ("stoch4-ragged", 5000, 3, qfields(O.Q_STOCH_UNIFORM, 4, O.SCALE_L2, bucket=512), O.ADAM_AT_SERVER),
    ("sign-global-worker", 3001, 5, qfields(O.Q_SCALED_SIGN, 1, bucket=0), O.ADAM_AT_WORKER),
    ("topk", 2500, 4, dict(kind=O.Q_TOPK, keep=16, bucket=512, error_feedback=1), O.ADAM_AT_SERVER),
    ("ex1-wide", 777, 17, qfields(O.Q_DET_UNIFORM, 3, bucket=2048), O.ADAM_AT_SERVER),
    ("stoch2-max-wide", 9000, 8, qfields(O.Q_STOCH_UNIFORM, 2, O.SCALE_MAX, bucket=2048), O.ADAM_AT_WORKER),
    ("raw", 1000, 2, qfields(O.Q_NONE), O.ADAM_AT_SERVER),
    ("randk-short-bucket", 1500, 3, dict(kind=O.Q_RANDK, keep=40, bucket=2048, error_feedback=1),
     O.ADAM_AT_WORKER),
]


@pytest.mark.parametrize("name,d,N,q,placement", ROUNDS, ids=[r[0] for r in ROUNDS])
@pytest.mark.parametrize("call", ["step", "noalloc", "scheduled", "run", "split"])
def test_round_writes_stay_in_bounds(name, d, N, q, placement, call):
    _, ec = configs(d, N, q, q, placement, seed=3)
    rb = allocate(ec, with_u=True)
    init_state(ec, rb)
    rng = np.random.default_rng(d + N)
    rb.g.copy_(torch.from_numpy((rng.standard_normal((N, d)) * 1e-2).astype(np.float32)))
    gd = Guarded()
    sched = E.Schedule(kind=E.EA_SCHED_STEP_DECAY, alpha=1e-3, factor=0.5, period=1)
    if call == "split":
        _split_rounds(ec, rb, gd)
        gd.check(f"split {name}")
        return
    args = _step_args(ec, rb, gd)
    if call == "run":
        a = dict(args)
        g = a.pop("g")
        E.ea_run(ec, sched, 1, 2, g, 0, **a)
    elif call == "scheduled":
        t_dev = gd.wrap("t_dev", torch.ones(1, dtype=torch.int32, device="cuda"))
        for _ in range(2):
            E.ea_step_scheduled(ec, sched, t_dev, **args)
    for t in (1, 2):
        if call == "step":
            E.ea_step(ec, t, **args)
        elif call == "noalloc":
            a = dict(args)
            a.pop("workspace")
            E.ea_step_noalloc(ec, t, **a)
    gd.check(f"{call} {name}")


def _split_rounds(ec, rb, gd):
    """Two rounds through the four split calls.  Each worker's rows and
    message sit in allocations of their own, so that a worker call writing
    past its row is caught (the next worker would overwrite it in a shared
    array); the server calls get the workers' messages side by side, as they
    take them."""
    d, N = ec.d, ec.N
    nsw, nss = E.ea_msg_scales(ec.qw, d), E.ea_msg_scales(ec.qs, d)
    ww = E.ea_msg_words(ec.qw, d)
    ws = gd.wrap("workspace", rb.workspace)
    rows = []
    for i in range(N):
        rows.append({k: gd.wrap(f"{k}[{i}]", None if getattr(rb, k) is None else getattr(rb, k)[i].contiguous())
                     for k in ("g", "e_w", "m_w", "v_w")})
        rows[i]["codes"] = gd.wrap(f"wcodes[{i}]", torch.zeros(ww, dtype=torch.uint64, device="cuda"))
        rows[i]["scales"] = gd.wrap(f"wscales[{i}]", torch.zeros(nsw, dtype=torch.float32, device="cuda")) \
            if nsw else None
    wcodes = gd.wrap("wcodes", torch.zeros((N, ww), dtype=torch.uint64, device="cuda"))
    wscales = gd.wrap("wscales", torch.zeros((N, nsw), dtype=torch.float32, device="cuda")) if nsw else None
    m, v, u = gd.wrap("m", rb.m), gd.wrap("v", rb.v), gd.wrap("u", rb.u)
    e_s, x = gd.wrap("e_s", rb.e_s), gd.wrap("x", rb.x)
    scodes = gd.wrap("scodes", rb.scodes)
    sscales = gd.wrap("sscales", rb.sscales[:nss].contiguous()) if nss else None
    for t in (1, 2):
        for i, r in enumerate(rows):
            E.ea_worker_compress(ec, i, t, r["g"], r["e_w"], r["m_w"], r["v_w"], r["codes"], r["scales"], ws)
            wcodes[i].copy_(r["codes"])
            if nsw:
                wscales[i].copy_(r["scales"])
        E.ea_server_aggregate_adam(ec, t, wcodes, wscales, m, v, u)
        E.ea_server_compress(ec, t, u, e_s, scodes, sscales, ws)
        E.ea_worker_apply(ec, scodes, sscales, x)


@pytest.mark.parametrize("d,N", [(500, 10), (65, 2), (777, 31), (4096, 3)])
def test_toy_writes_stay_in_bounds(d, N):
    rng = np.random.default_rng(d)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    A = dev(rng.standard_normal((d, d)).astype(np.float32))
    xs = dev((rng.standard_normal(d) * math.sqrt(0.1)).astype(np.float32))
    xi = dev((rng.standard_normal((N, d)) * math.sqrt(0.1)).astype(np.float32))
    ex2 = qfields(O.Q_POW2, kmin=-17, kmax=-11)
    _, ec = configs(d, N, ex2, ex2, O.ADAM_AT_WORKER, seed=9, beta1=0.9, beta2=0.99, lr=1e-4)
    rb = allocate(ec)
    init_state(ec, rb)
    gd = Guarded()
    st = {k: gd.wrap(k, getattr(rb, k)) for k in ("e_w", "m_w", "v_w", "e_s", "x", "wcodes", "scodes")}
    ws = gd.wrap("workspace", torch.zeros(E.ea_toy_workspace_bytes(d), dtype=torch.uint8, device="cuda"))
    g = gd.wrap("g", torch.zeros((N, d), dtype=torch.float32, device="cuda"))
    gs = gd.wrap("grad_sq", torch.zeros(1, dtype=torch.float64, device="cuda"))
    for t in (1, 2):
        E.ea_toy_step(ec, t, A, xs, xi, st["e_w"], st["m_w"], st["v_w"], None, None, st["e_s"], st["x"],
                      st["wcodes"], st["scodes"], gs, g, ws)
    E.ea_toy_grad(d, N, A, xs, xi, st["x"], g, gs, ws)
    gd.check(f"toy d={d} N={N}")


@pytest.mark.parametrize("name,d,N,q,placement", ROUNDS, ids=[r[0] for r in ROUNDS])
def test_round_reads_stay_in_bounds(name, d, N, q, placement):
    """The same two rounds from ordinary allocations and from allocations
    whose bytes past every array are 0xFF (a NaN in binary32): every output
    agrees bit for bit, so no read past an array's end reaches a result."""
    _, ec = configs(d, N, q, q, placement, seed=3)
    rng = np.random.default_rng(d * 3 + N)
    g0 = torch.from_numpy((rng.standard_normal((N, d)) * 1e-2).astype(np.float32)).cuda()
    outs = []
    for pattern in (None, 0xFF):
        rb = allocate(ec)
        init_state(ec, rb)
        rb.g.copy_(g0)
        if pattern is None:
            args = rb.step_args()
            nsw, nss = E.ea_msg_scales(ec.qw, d), E.ea_msg_scales(ec.qs, d)
            args["wscales"] = args["wscales"][:, :nsw].contiguous() if nsw else None
            args["sscales"] = args["sscales"][:nss].contiguous() if nss else None
        else:
            args = _step_args(ec, rb, Guarded(pattern))
        for t in (1, 2):
            E.ea_step(ec, t, **args)
        torch.cuda.synchronize()
        outs.append({k: v.clone() for k, v in args.items() if v is not None and k not in ("g", "workspace")})
    for k in outs[0]:
        assert torch.equal(outs[0][k].view(torch.uint8), outs[1][k].view(torch.uint8)), f"{name}: {k}"


@pytest.mark.parametrize("d,N", [(500, 10), (65, 2), (777, 31), (4096, 3)])
def test_toy_reads_stay_in_bounds(d, N):
    """Two toy steps and one ea_toy_grad from ordinary allocations and from
    allocations with NaN bytes past every array (A, x*, xi, the state, the
    workspace): the same bits everywhere, so no read past an array's end
    reaches a gradient, a norm or the round."""
    rng = np.random.default_rng(d + 7)
    A0 = torch.from_numpy(rng.standard_normal((d, d)).astype(np.float32)).cuda()
    xs0 = torch.from_numpy((rng.standard_normal(d) * math.sqrt(0.1)).astype(np.float32)).cuda()
    xi0 = torch.from_numpy((rng.standard_normal((N, d)) * math.sqrt(0.1)).astype(np.float32)).cuda()
    ex2 = qfields(O.Q_POW2, kmin=-17, kmax=-11)
    _, ec = configs(d, N, ex2, ex2, O.ADAM_AT_WORKER, seed=9, beta1=0.9, beta2=0.99, lr=1e-4)
    outs = []
    for pattern in (None, 0xFF):
        rb = allocate(ec)
        init_state(ec, rb)
        rb.x.copy_(xs0 * 0.5)
        gd = Guarded(pattern if pattern is not None else PATTERN)
        w = (lambda k, t: t) if pattern is None else gd.wrap
        A, xs, xi = w("A", A0.clone()), w("xs", xs0.clone()), w("xi", xi0.clone())
        st = {k: w(k, getattr(rb, k)) for k in ("e_w", "m_w", "v_w", "e_s", "x", "wcodes", "scodes")}
        ws = w("workspace", torch.zeros(E.ea_toy_workspace_bytes(d), dtype=torch.uint8, device="cuda"))
        g = w("g", torch.zeros((N, d), dtype=torch.float32, device="cuda"))
        gs = w("grad_sq", torch.zeros(1, dtype=torch.float64, device="cuda"))
        for t in (1, 2):
            E.ea_toy_step(ec, t, A, xs, xi, st["e_w"], st["m_w"], st["v_w"], None, None, st["e_s"], st["x"],
                          st["wcodes"], st["scodes"], gs, g, ws)
        g2 = w("g2", torch.zeros((N, d), dtype=torch.float32, device="cuda"))
        gs2 = w("grad_sq2", torch.zeros(1, dtype=torch.float64, device="cuda"))
        E.ea_toy_grad(d, N, A, xs, xi, st["x"], g2, gs2, ws)
        torch.cuda.synchronize()
        res = {k: v.clone() for k, v in st.items()}
        res.update(g=g.clone(), gs=gs.clone(), g2=g2.clone(), gs2=gs2.clone())
        outs.append(res)
    for k in outs[0]:
        assert torch.equal(outs[0][k].view(torch.uint8), outs[1][k].view(torch.uint8)), f"toy d={d} N={N}: {k}"
