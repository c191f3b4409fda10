"""GPU parity of the Definition 3 sparsifiers (top-k and random-k per bucket)
against the oracle: kept masks and kept values bit-exact, state within the
float tolerance, after every step of a trajectory.  Covers the specialized
whole-tile kernels (bucket 512, Adam at the server), the generic kernels, the
split calls (which decode the messages), ragged and tiny sizes, equal keys at
the threshold, and keep at its limits."""
import numpy as np
import pytest

import oracle as O
import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU-only host
    pytest.skip("needs a GPU", allow_module_level=True)

from parity_util import Pair, qfields  # noqa: E402

TOPK = lambda keep, b, ef=1: qfields(O.Q_TOPK, bucket=b, keep=keep, ef=ef)  # noqa: E731
RANDK = lambda keep, b, ef=1: qfields(O.Q_RANDK, bucket=b, keep=keep, ef=ef)  # noqa: E731
SPARSE = {"topk": TOPK, "randk": RANDK}


def _grads(gen, seed, t, N, d):
    w = W.Workload("t", "t", d, N, None, None, 1, seed, gen)
    return W.host_gradients(w, t, d=d)


def _tied_grads(seed, t, N, d):
    """Few distinct magnitudes and many zeros: most keys tie."""
    rng = np.random.default_rng(seed * 1000 + t)
    mag = rng.choice(np.array([0.0, 0.0, 1e-3, 2e-3, 4e-3], np.float32), size=(N, d))
    return (mag * rng.choice(np.array([-1.0, 1.0], np.float32), size=(N, d))).astype(np.float32)


def _run(d, N, qw, qs, placement, T, gen="student_t", seed=5, split=False, **hp):
    pair = Pair(d, N, qw, qs, placement, seed=seed, split=split, **hp)
    for t in range(1, T + 1):
        g = _tied_grads(seed, t, N, d) if gen == "tied" else _grads(gen, seed, t, N, d)
        pair.step(t, g)
    pair.check_tie_budget()
    print(f"\n[parity] sparse d={d} N={N} T={T} placement={placement} split={split}: {pair.stats}", flush=True)
    return pair


@pytest.mark.parametrize("kind", list(SPARSE))
@pytest.mark.parametrize("d", [512 * 41 + 384, 512 * 42, 512 * 41, 512 + 100, 300])
def test_lean_kernels(kind, d):
    """Bucket 512, Adam at the server, 16 workers: the specialized two-tile
    kernels plus the edge kernel of a ragged tail."""
    q = SPARSE[kind](16, 512)
    _run(d, 16, q, q, O.ADAM_AT_SERVER, T=4)


@pytest.mark.parametrize("gen", ["student_t", "tied"])
@pytest.mark.parametrize("keep", [64, 65, 150, 192, 193])
def test_lean_kernels_larger_keep(keep, gen):
    """Bucket 512 with keep past one key per lane: the threshold search starts
    below the bits shared by the lanes' largest and r-th largest keys for keep
    up to 3 keys per lane (192), and from the top above that."""
    q = TOPK(keep, 512)
    _run(512 * 9 + 200, 6, q, q, O.ADAM_AT_SERVER, T=3, gen=gen, seed=keep)


@pytest.mark.parametrize("placement", [O.ADAM_AT_SERVER, O.ADAM_AT_WORKER], ids=["server", "worker"])
@pytest.mark.parametrize("kind", list(SPARSE))
@pytest.mark.parametrize("bucket,keep", [(256, 1), (512, 37), (1024, 200), (2048, 64)])
def test_generic_kernels(kind, bucket, keep, placement):
    q = SPARSE[kind](keep, bucket)
    _run(4 * 1024 + 260, 3, q, q, placement, T=4, gen="outliers")


@pytest.mark.parametrize("kind", list(SPARSE))
@pytest.mark.parametrize("d,N,keep", [(2048 * 9 + 700, 16, 128), (2048 * 5, 11, 64), (2048 * 4 + 1030, 20, 300),
                                      (2048 * 3 + 2047, 8, 2048)])
def test_wide_tile_kernels(kind, d, N, keep):
    """Bucket 2048 on both sides with Adam at the server: the fully
    specialized 8-chunk kernels, whose server side runs Adam on eight waves,
    one chunk each, and selects on one of them.  Several worker groups (the
    last one partial with 11 and 20 workers), ragged tails, keep within and
    past the first search's range, and keep = bucket."""
    q = SPARSE[kind](keep, 2048)
    _run(d, N, q, q, O.ADAM_AT_SERVER, T=3, seed=keep)


def _random_wide_cases(n, seed=77):
    rng = np.random.default_rng(seed)
    out = []
    for j in range(n):
        kind = ("topk", "randk")[j % 2]
        placement = (O.ADAM_AT_SERVER, O.ADAM_AT_WORKER)[(j // 2) % 2]
        d = int(rng.integers(1, 12)) * 2048 + int(rng.integers(0, 2048))
        N = int(rng.integers(1, 41))
        keep = int(rng.choice([1, int(rng.integers(2, 129)), int(rng.integers(129, 2049))]))
        out.append((kind, placement, d, N, keep))
    return out


@pytest.mark.parametrize("kind,placement,d,N,keep", _random_wide_cases(12))
def test_wide_tile_random_shapes(kind, placement, d, N, keep):
    """Seeded random shapes on 2048-element buckets: d up to 12 tiles with a
    ragged tail, 1 to 40 workers (up to five worker groups of eight waves),
    keep from 1 to 2048, both placements (the fully specialized kernels with
    Adam at the server, the worker-specialized ones with Adam at the
    workers; random-k selects before reading the values on both)."""
    q = SPARSE[kind](keep, 2048)
    _run(d, N, q, q, placement, T=2, seed=N + keep)


@pytest.mark.parametrize("kind", list(SPARSE))
def test_split_calls(kind):
    q = SPARSE[kind](24, 512)
    _run(512 * 9 + 130, 5, q, q, O.ADAM_AT_SERVER, T=4, split=True)
    _run(256 * 7 + 3, 3, SPARSE[kind](5, 256), TOPK(100, 1024), O.ADAM_AT_WORKER, T=3, split=True)


@pytest.mark.parametrize("split", [False, True], ids=["fused", "split"])
def test_equal_keys_at_the_threshold(split):
    _run(512 * 9 + 200, 16, TOPK(16, 512), TOPK(16, 512), O.ADAM_AT_SERVER, T=4, gen="tied", split=split)
    _run(256 * 11 + 17, 3, TOPK(40, 256), TOPK(9, 512), O.ADAM_AT_WORKER, T=4, gen="tied", split=split)


def test_all_keys_equal():
    """Every key of a bucket equal (constant magnitudes; then half of them
    zero): the lane maxima all agree, the threshold is that key, and the kept
    elements are the lowest-indexed ones."""
    d, N = 512 * 6 + 300, 16
    pair = Pair(d, N, TOPK(16, 512), TOPK(16, 512), O.ADAM_AT_SERVER, seed=3)
    rng = np.random.default_rng(12)
    for t in range(1, 4):
        g = (np.float32(1e-3) * rng.choice(np.array([-1.0, 1.0], np.float32), size=(N, d))).astype(np.float32)
        if t == 2:
            g[:, ::2] = 0.0
        pair.step(t, g)
    pair.check_tie_budget()


@pytest.mark.parametrize("d", [1, 3, 100, 255, 256, 257, 1001])
def test_tiny_and_unaligned_sizes(d):
    """Sizes below a bucket and rows without 16-byte alignment; a bucket
    shorter than keep zero-fills its remaining value slots."""
    _run(d, 3, TOPK(4, 256), RANDK(300, 512), O.ADAM_AT_SERVER, T=3)
    _run(d, 2, RANDK(1, 256), TOPK(256, 256), O.ADAM_AT_WORKER, T=3)


@pytest.mark.parametrize("kind", list(SPARSE))
def test_keep_limits(kind):
    """keep = bucket sends everything (Q is the identity), keep = 1 one element."""
    _run(512 * 5 + 64, 4, SPARSE[kind](512, 512), SPARSE[kind](1, 512), O.ADAM_AT_SERVER, T=3)


def test_mixed_with_quantizers():
    """A sparsifier on one side, a scaled quantizer on the other."""
    _run(2048 * 3 + 500, 4, TOPK(64, 2048), qfields(O.Q_SCALED_SIGN, 1, O.SCALE_L1, 1, 256), O.ADAM_AT_SERVER,
         T=3)
    _run(1024 * 5 + 12, 3, qfields(O.Q_STOCH_UNIFORM, 4, O.SCALE_L2, 1, 512), RANDK(32, 1024), O.ADAM_AT_WORKER,
         T=3)


def test_error_feedback_off():
    _run(512 * 6 + 10, 4, TOPK(8, 512, ef=0), RANDK(8, 512, ef=0), O.ADAM_AT_SERVER, T=3)
