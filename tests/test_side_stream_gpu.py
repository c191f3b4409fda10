"""The ragged last tile of a fused round may run on the library's side stream,
forked from the caller's stream and joined back to it.  These tests issue such
rounds from two host threads at once, each on its own stream, and check that
every message and state array equals that of the same rounds issued one after
the other on one stream; and that work queued on the caller's stream right
after a round sees all of its results."""
import threading

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

SIGN = lambda b: qfields(O.Q_SCALED_SIGN, 1, O.SCALE_L1, 1, b)  # noqa: E731
STOCH4 = qfields(O.Q_STOCH_UNIFORM, 4, O.SCALE_L2, 1, 512)
# whole tiles plus a ragged one, few enough blocks that the side stream is taken
SHAPES = [
    (2048 * 37 + 1500, 8, SIGN(2048), SIGN(2048)),      # 8-chunk tiles, ResNet-18-like
    (512 * 301 + 77, 16, STOCH4, STOCH4),               # two-tile blocks, an odd tile count
]
STATE = ("e_w", "e_s", "x", "m", "v", "wcodes", "wscales", "scodes", "sscales")
T = 4


def _setup(k):
    d, N, qw, qs = SHAPES[k]
    _, ec = configs(d, N, qw, qs, O.ADAM_AT_SERVER, seed=20 + k)
    rb = allocate(ec)
    init_state(ec, rb)
    grads = [torch.from_numpy(W.host_gradients(W.Workload("s", "s", d, N, None, None, 1, 20 + k, "student_t"), t, d=d))
             .cuda() for t in range(1, T + 1)]
    torch.cuda.synchronize()
    return ec, rb, grads


def _rounds(ec, rb, grads, stream):
    with torch.cuda.stream(stream):
        for t in range(1, T + 1):
            rb.g.copy_(grads[t - 1])
            E.ea_step(ec, t, **rb.step_args())


def _snapshot(rb):
    return {k: getattr(rb, k).cpu().numpy().copy() for k in STATE}


def test_rounds_from_two_threads_equal_serial_rounds():
    ref = []
    for k in range(len(SHAPES)):
        ec, rb, grads = _setup(k)
        _rounds(ec, rb, grads, torch.cuda.current_stream())
        torch.cuda.synchronize()
        ref.append(_snapshot(rb))
    for rep in range(3):
        runs = [_setup(k) for k in range(len(SHAPES))]
        streams = [torch.cuda.Stream() for _ in SHAPES]
        errors = []

        def work(k):
            try:
                _rounds(*runs[k], streams[k])
            except Exception as exc:  # pragma: no cover - reported below
                errors.append(exc)

        threads = [threading.Thread(target=work, args=(k,)) for k in range(len(SHAPES))]
        for th in threads:
            th.start()
        for th in threads:
            th.join()
        torch.cuda.synchronize()
        assert not errors, errors
        for k in range(len(SHAPES)):
            got = _snapshot(runs[k][1])
            for name in STATE:
                assert np.array_equal(got[name].view(np.uint8), ref[k][name].view(np.uint8)), \
                    f"shape {k}, repetition {rep}: {name} differs"


def test_work_queued_after_a_round_sees_its_results():
    """A copy queued on the caller's stream right after each round, with no
    host synchronization in between, holds the round's final x and e_s
    (ragged tile included)."""
    ec, rb, grads = _setup(0)
    stream = torch.cuda.Stream()
    copies = []
    with torch.cuda.stream(stream):
        for t in range(1, T + 1):
            rb.g.copy_(grads[t - 1])
            E.ea_step(ec, t, **rb.step_args())
            copies.append((rb.x.clone(), rb.e_s.clone()))
    torch.cuda.synchronize()
    ec2, rb2, _ = _setup(0)
    for t in range(1, T + 1):
        rb2.g.copy_(grads[t - 1])
        E.ea_step(ec2, t, **rb2.step_args())
        torch.cuda.synchronize()
        x, es = copies[t - 1]
        assert torch.equal(x.view(torch.int32), rb2.x.view(torch.int32)), f"round {t}: x"
        assert torch.equal(es.view(torch.int32), rb2.e_s.view(torch.int32)), f"round {t}: e_s"
