"""ea_step_noalloc (the round for callers that cannot allocate) against ea_step
with a caller-allocated workspace: two rounds in a row through the C ABI, the
second on a smaller input, every message and state vector bit-identical.  The
first configuration has one-bucket quantizers on both sides, so the library's
own scratch array carries the per-tile partial norms and the server input;
the second reuses that array with other sizes, and a third has no scratch at
all."""
import numpy as np
import pytest

import oracle as O
import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU-only host
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2205_14473_amd as E  # noqa: E402
from paper_2205_14473_amd.state import allocate, init_state  # noqa: E402
from parity_util import configs, qfields  # noqa: E402

SIGN0 = qfields(O.Q_SCALED_SIGN, 1, O.SCALE_L1, 1, 0)
STOCH2MAX0 = qfields(O.Q_STOCH_UNIFORM, 2, O.SCALE_MAX, 1, 0)
EX1_0 = qfields(O.Q_DET_UNIFORM, 3, bucket=0)
STOCH4 = qfields(O.Q_STOCH_UNIFORM, 4, O.SCALE_L2, 1, 512)

KEYS = ("wcodes", "wscales", "scodes", "sscales", "e_w", "e_s", "x", "m", "v", "m_w", "v_w")


def _pair(d, N, qw, qs, placement, seed):
    _, ec = configs(d, N, qw, qs, placement, seed)
    a, b = allocate(ec), allocate(ec)
    init_state(ec, a)
    init_state(ec, b)
    w = W.Workload("n", "n", d, N, None, None, 1, seed, "student_t")
    return ec, a, b, w


def _round(ec, a, b, w, t, d):
    g = torch.from_numpy(W.host_gradients(w, t, d=d)).cuda()
    a.g.copy_(g)
    b.g.copy_(g)
    E.ea_step(ec, t, **a.step_args())
    args = b.step_args()
    args.pop("workspace")
    E.ea_step_noalloc(ec, t, **args)
    torch.cuda.synchronize()
    for k in KEYS:
        x, y = getattr(a, k), getattr(b, k)
        if x is None:
            continue
        assert torch.equal(x.view(torch.uint8), y.view(torch.uint8)), f"d={d} step {t}: {k} differs"


def test_noalloc_equals_step_with_workspace_two_calls_smaller_second():
    # one-bucket both sides: the scratch array holds partials and the server input
    d1, N1 = 200_000 + 77, 5
    ec, a, b, w = _pair(d1, N1, SIGN0, STOCH2MAX0, O.ADAM_AT_SERVER, 13)
    assert E.ea_workspace_bytes(ec) > 0
    _round(ec, a, b, w, 1, d1)
    _round(ec, a, b, w, 2, d1)
    del a, b
    # smaller input, other quantizers and placement: the same array, other sizes
    d2, N2 = 3000 + 5, 3
    ec2, a2, b2, w2 = _pair(d2, N2, EX1_0, SIGN0, O.ADAM_AT_WORKER, 14)
    assert 0 < E.ea_workspace_bytes(ec2) < E.ea_workspace_bytes(ec)
    _round(ec2, a2, b2, w2, 1, d2)
    _round(ec2, a2, b2, w2, 2, d2)
    # bucketed quantizers need no scratch
    d3, N3 = 512 * 9 + 100, 4
    ec3, a3, b3, w3 = _pair(d3, N3, STOCH4, STOCH4, O.ADAM_AT_SERVER, 15)
    assert E.ea_workspace_bytes(ec3) == 0
    _round(ec3, a3, b3, w3, 1, d3)


def test_noalloc_rejects_configurations_beyond_its_scratch():
    d, N = 8_000_000, 4
    _, ec = configs(d, N, SIGN0, SIGN0, O.ADAM_AT_SERVER, 3)
    assert E.ea_workspace_bytes(ec) > E.EA_NOALLOC_SCRATCH_BYTES
    with pytest.raises(E.EAError) as ei:
        E.ea_step_noalloc(ec, 1, *([1 << 20] * 12))
    assert ei.value.code == E.EA_ERR_UNSUPPORTED
    assert "scratch" in E.ea_last_error()


ONE_BUCKET_OR_NOT = [
    SIGN0, STOCH2MAX0, EX1_0, STOCH4,
    qfields(O.Q_STOCH_UNIFORM, 8, O.SCALE_L2, 1, 0),
    qfields(O.Q_SCALED_SIGN, 1, O.SCALE_L1, 0, 0),
    qfields(O.Q_TOPK, bucket=1024, keep=40),
    qfields(O.Q_POW2, kmin=-30, kmax=-2),
]


@pytest.mark.parametrize("j", range(10))
def test_noalloc_random_configurations(j):
    """Seeded random configurations (one-bucket and bucketed quantizers, 1 to
    12 workers, either placement), three rounds through ea_step_noalloc after
    the calls above left other contents in the scratch array: bit-identical to
    ea_step with a workspace of the caller's."""
    rng = np.random.default_rng(700 + j)
    d = int(rng.integers(1, 300_000))
    N = int(rng.integers(1, 13))
    qw = ONE_BUCKET_OR_NOT[int(rng.integers(0, len(ONE_BUCKET_OR_NOT)))]
    qs = ONE_BUCKET_OR_NOT[int(rng.integers(0, len(ONE_BUCKET_OR_NOT)))]
    placement = int(rng.choice([O.ADAM_AT_SERVER, O.ADAM_AT_WORKER]))
    ec, a, b, w = _pair(d, N, qw, qs, placement, 700 + j)
    assert E.ea_workspace_bytes(ec) <= E.EA_NOALLOC_SCRATCH_BYTES
    for t in range(1, 4):
        _round(ec, a, b, w, t, d)
