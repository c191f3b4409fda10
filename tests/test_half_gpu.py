"""GPU parity of the fused-round kernels specialized for the worker quantizer
only (the server quantizer and the Adam placement read at run time): every
worker quantizer of those tables (scaled sign; stochastic 1/2/4/8-bit with L2
or max-norm scale; top-k; random-k; Example 1 with 2 or 3 bits) at every
bucket size 256 to 2048, paired with a different server quantizer whose bucket
is no larger, in both placements; Example 2 and full precision (no bucket) at
the tile size of the server's bucket.  Sizes hold several whole tiles (the
specialized launch) and a ragged tail (the generic edge launch); one-chunk
tiles go two to a block, so odd and even tile counts both occur."""
import numpy as np
import pytest

import oracle as O
import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU-only host
    pytest.skip("needs a GPU", allow_module_level=True)

from parity_util import Pair, qfields  # noqa: E402

WORKER = {
    "sign": lambda b: qfields(O.Q_SCALED_SIGN, 1, O.SCALE_L1, 1, b),
    "stoch1_l2": lambda b: qfields(O.Q_STOCH_UNIFORM, 1, O.SCALE_L2, 1, b),
    "stoch1_max": lambda b: qfields(O.Q_STOCH_UNIFORM, 1, O.SCALE_MAX, 1, b),
    "stoch2_l2": lambda b: qfields(O.Q_STOCH_UNIFORM, 2, O.SCALE_L2, 1, b),
    "stoch2_max": lambda b: qfields(O.Q_STOCH_UNIFORM, 2, O.SCALE_MAX, 1, b),
    "stoch4_l2": lambda b: qfields(O.Q_STOCH_UNIFORM, 4, O.SCALE_L2, 1, b),
    "stoch4_max": lambda b: qfields(O.Q_STOCH_UNIFORM, 4, O.SCALE_MAX, 1, b),
    "stoch8_l2": lambda b: qfields(O.Q_STOCH_UNIFORM, 8, O.SCALE_L2, 1, b),
    "stoch8_max": lambda b: qfields(O.Q_STOCH_UNIFORM, 8, O.SCALE_MAX, 1, b),
    "topk": lambda b: qfields(O.Q_TOPK, bucket=b, keep=b // 32 + 1),
    "randk": lambda b: qfields(O.Q_RANDK, bucket=b, keep=b // 16),
    "ex1_2": lambda b: qfields(O.Q_DET_UNIFORM, 2, bucket=b),
    "ex1_3": lambda b: qfields(O.Q_DET_UNIFORM, 3, bucket=b),
    # no bucket: the tile size follows the server's bucket
    "ex2_4": lambda b: qfields(O.Q_POW2, kmin=-17, kmax=-11),
    "none": lambda b: qfields(O.Q_NONE),
}
# A server quantizer of another kind, bucket no larger than the worker's.
SERVER = [
    lambda b: qfields(O.Q_DET_UNIFORM, 3, bucket=b),
    lambda b: qfields(O.Q_STOCH_UNIFORM, 2, O.SCALE_MAX, 1, max(256, b // 2)),
    lambda b: qfields(O.Q_SCALED_SIGN, 1, O.SCALE_L1, 1, 256),
    lambda b: qfields(O.Q_TOPK, bucket=b, keep=7),
]


def _grads(seed, t, N, d):
    w = W.Workload("t", "t", d, N, None, None, 1, seed, "student_t")
    return W.host_gradients(w, t, d=d)


@pytest.mark.parametrize("bucket", [256, 512, 1024, 2048])
@pytest.mark.parametrize("kind", list(WORKER))
def test_worker_specialized_kernels(kind, bucket):
    qw = WORKER[kind](bucket)
    k = list(WORKER).index(kind)
    qs = SERVER[k % len(SERVER)](bucket)
    if kind in ("ex2_4", "none"):      # the server's bucket sets the tile size
        qs = qfields(O.Q_STOCH_UNIFORM, 2, O.SCALE_MAX, 1, bucket)
    placement = O.ADAM_AT_SERVER if k % 2 == 0 else O.ADAM_AT_WORKER
    tiles = 5 if bucket > 256 else 6          # one-chunk tiles: an even count, plus the tail
    d = bucket * tiles + 100
    pair = Pair(d, 5, qw, qs, placement, seed=11 + k)
    for t in range(1, 4):
        pair.step(t, _grads(11 + k, t, 5, d))
    pair.check_tie_budget()
    print(f"\n[parity] half {kind} bucket={bucket} placement={placement}: {pair.stats}", flush=True)


@pytest.mark.parametrize("placement", [O.ADAM_AT_SERVER, O.ADAM_AT_WORKER], ids=["server", "worker"])
def test_worker_specialized_with_one_bucket_server(placement):
    """The server's one-bucket quantizer makes the fused round stop after the
    server input (per-tile partial norms, then the finalize and server
    kernels)."""
    d = 512 * 7 + 32                    # rows 16-byte aligned: whole tiles take the specialized kernel
    pair = Pair(d, 6, WORKER["stoch4_max"](512), qfields(O.Q_SCALED_SIGN, 1, O.SCALE_L1, 1, 0), placement, seed=3)
    for t in range(1, 4):
        pair.step(t, _grads(3, t, 6, d))
    pair.check_tie_budget()


SYMMETRIC = ["sign", "stoch1_l2", "stoch2_max", "stoch4_l2", "stoch4_max", "stoch8_max", "topk", "randk"]


@pytest.mark.parametrize("bucket", [1024, 2048])
@pytest.mark.parametrize("kind", SYMMETRIC)
def test_symmetric_wide_tiles(kind, bucket):
    """The same quantizer on both sides with Adam at the server, 4- and 8-chunk
    tiles: the fully specialized wide-tile kernels."""
    q = WORKER[kind](bucket)
    d = bucket * 5 + 100
    pair = Pair(d, 6, q, q, O.ADAM_AT_SERVER, seed=21)
    for t in range(1, 4):
        pair.step(t, _grads(21, t, 6, d))
    pair.check_tie_budget()


@pytest.mark.parametrize("bucket,keep", [(1024, 80), (1024, 81), (1024, 300), (2048, 1), (2048, 80), (2048, 81),
                                         (2048, 700)])
@pytest.mark.parametrize("kind", ["topk", "randk"])
def test_symmetric_wide_sparse_keeps(kind, bucket, keep):
    """Wide-tile sparsifiers on both sides with keep on either side of the
    limit below which the threshold search first runs on each lane's largest
    keys, and far above it."""
    q = qfields(O.Q_TOPK if kind == "topk" else O.Q_RANDK, bucket=bucket, keep=keep)
    d = bucket * 4 + 300
    pair = Pair(d, 4, q, q, O.ADAM_AT_SERVER, seed=keep)
    for t in range(1, 4):
        pair.step(t, _grads(keep, t, 4, d))
    pair.check_tie_budget()


@pytest.mark.parametrize("bucket", [1024, 2048])
def test_symmetric_wide_topk_ties(bucket):
    """Few distinct magnitudes: most keys tie at the threshold on wide tiles."""
    d, N = bucket * 3 + 64, 3
    q = qfields(O.Q_TOPK, bucket=bucket, keep=bucket // 32)
    pair = Pair(d, N, q, q, O.ADAM_AT_SERVER, seed=8)
    rng = np.random.default_rng(bucket)
    for t in range(1, 4):
        mag = rng.choice(np.array([0.0, 1e-3, 2e-3, 4e-3], np.float32), size=(N, d))
        pair.step(t, (mag * rng.choice(np.array([-1.0, 1.0], np.float32), size=(N, d))).astype(np.float32))
    pair.check_tie_budget()
