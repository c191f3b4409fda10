"""GPU parity: the HIP path (through the C ABI) against the oracle, element by
element, after every step of a trajectory.  Sizes span several tiles and a
ragged tail; the comparison rule is in tests/parity_util.py."""
import numpy as np
import pytest

import oracle as O
import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU-only host
    pytest.skip("needs a GPU", allow_module_level=True)

from parity_util import Pair, qfields, same_values  # noqa: E402

SIGN = lambda b, ef=1: qfields(O.Q_SCALED_SIGN, 1, O.SCALE_L1, ef, b)  # noqa: E731
STOCH = lambda bits, sc, b, ef=1: qfields(O.Q_STOCH_UNIFORM, bits, sc, ef, b)  # noqa: E731


def _grads(gen, seed, t, N, d):
    w = W.Workload("t", "t", d, N, None, None, 1, seed, gen)
    return W.host_gradients(w, t, d=d)


def _run(d, N, qw, qs, placement, T, gen="student_t", seed=5, split=False, x1=None, **hp):
    pair = Pair(d, N, qw, qs, placement, seed=seed, x1=x1, split=split, **hp)
    for t in range(1, T + 1):
        pair.step(t, _grads(gen, seed, t, N, d))
    pair.check_tie_budget()
    print(f"\n[parity] d={d} N={N} T={T} placement={placement} split={split}: {pair.stats}", flush=True)
    return pair


# The five workload shapes at reduced d (same N, quantizers and buckets; the
# tails reproduce each workload's last partial bucket / 64-element group).
SHAPES = {
    "resnet18": (2048 * 9 + 1576, 8, SIGN(2048), SIGN(2048), "segscale"),
    "resnet50": (512 * 21 + 40, 32, STOCH(2, O.SCALE_MAX, 512), STOCH(2, O.SCALE_MAX, 512), "segscale"),
    "bert": (512 * 40 + 384, 16, STOCH(4, O.SCALE_L2, 512), STOCH(4, O.SCALE_L2, 512), "student_t"),
    "gpt2m": (1024 * 13 + 704, 8, STOCH(2, O.SCALE_MAX, 1024), SIGN(1024), "outliers"),
}


@pytest.mark.parametrize("placement", [O.ADAM_AT_SERVER, O.ADAM_AT_WORKER], ids=["server", "worker"])
@pytest.mark.parametrize("shape", list(SHAPES))
def test_workload_shapes_fused(shape, placement):
    d, N, qw, qs, gen = SHAPES[shape]
    _run(d, N, qw, qs, placement, T=12, gen=gen)


@pytest.mark.parametrize("shape", list(SHAPES))
def test_workload_shapes_split_calls(shape):
    d, N, qw, qs, gen = SHAPES[shape]
    _run(d, N, qw, qs, O.ADAM_AT_SERVER, T=6, gen=gen, split=True)


def test_toy_full_trajectory():
    """The toy quadratic at its full size, 100 steps, one-bucket scaled sign."""
    w = W.WORKLOADS["toy"]
    xs = W.toy_x_star(w)
    pair = Pair(w.d, w.N, SIGN(0), SIGN(0), O.ADAM_AT_SERVER, seed=w.seed, x1=W.initial_x(w))
    for t in range(1, w.steps + 1):
        g = W.host_gradients(w, t, x=pair.ost.x, x_star=xs)   # from the oracle's iterate
        pair.step(t, g)
    pair.check_tie_budget()
    print(f"\n[parity] toy: {pair.stats}", flush=True)


@pytest.mark.parametrize("placement", [O.ADAM_AT_SERVER, O.ADAM_AT_WORKER], ids=["server", "worker"])
def test_bert_shape_100_step_trajectory(placement):
    """The BERT workload's quantizers, N = 16 and ragged tail at reduced d,
    compared after every step of a 100-step trajectory."""
    d, N, qw, qs, gen = SHAPES["bert"]
    pair = _run(d, N, qw, qs, placement, T=100, gen=gen)
    assert pair.stats.steps == 100


@pytest.mark.parametrize("split", [False, True], ids=["fused", "split"])
@pytest.mark.parametrize("ex", ["ex1", "ex2"])
def test_paper_toy_examples(ex, split):
    """Examples 1 and 2 with Adam at the workers (Algorithms 1-2 as printed) on
    the paper's 500-dimensional toy problem shape, 10 workers."""
    t0 = W.PAPER_TOY
    d, N = t0["d"], t0["N"]
    q = qfields(O.Q_DET_UNIFORM, 2) if ex == "ex1" else qfields(O.Q_POW2, kmin=-17, kmax=-11)
    rng = np.random.default_rng(3)
    A = rng.standard_normal((d, d))
    xs = rng.standard_normal(d) * np.sqrt(0.1)
    pair = Pair(d, N, q, q, O.ADAM_AT_WORKER, seed=9, split=split, beta2=0.99, lr=1e-4)
    for t in range(1, 41):
        x = pair.ost.x.astype(np.float64)
        xi = rng.standard_normal((N, d)) * np.sqrt(0.1)
        pair.step(t, (2 * ((A @ x - xs)[None, :] - xi) @ A).astype(np.float32))
    pair.check_tie_budget()


KINDS = {
    "none": qfields(O.Q_NONE),
    "sign256": SIGN(256),
    "sign_one": SIGN(0),
    "stoch1_max": STOCH(1, O.SCALE_MAX, 256),
    "stoch8_l2": STOCH(8, O.SCALE_L2, 512),
    "stoch4_one": STOCH(4, O.SCALE_L2, 0),
    "det3_512": qfields(O.Q_DET_UNIFORM, 3, bucket=512),
    "det8_one": qfields(O.Q_DET_UNIFORM, 8),
    "pow2_wide": qfields(O.Q_POW2, kmin=-20, kmax=-3),
    "pow2_full": qfields(O.Q_POW2, kmin=-126, kmax=127),
}


@pytest.mark.parametrize("kind", list(KINDS))
def test_quantizer_kinds(kind):
    q = KINDS[kind]
    _run(4 * 1024 + 260, 3, q, q, O.ADAM_AT_WORKER, T=5, gen="outliers")
    _run(4 * 1024 + 260, 3, q, q, O.ADAM_AT_SERVER, T=5, gen="outliers")


@pytest.mark.parametrize("kind", list(KINDS))
def test_quantizer_kinds_split_calls(kind):
    """Every code width through the split calls, whose messages are decoded
    from HBM (9-bit codes span two registers of spread words)."""
    q = KINDS[kind]
    _run(4 * 1024 + 260, 3, q, q, O.ADAM_AT_WORKER, T=4, gen="outliers", split=True)
    _run(2 * 1024 + 700, 5, q, SIGN(512), O.ADAM_AT_SERVER, T=4, gen="outliers", split=True)


@pytest.mark.parametrize("ef", [(0, 0), (0, 1), (1, 0)], ids=["off-off", "off-on", "on-off"])
def test_error_feedback_switches(ef):
    _run(3000, 4, STOCH(2, O.SCALE_MAX, 512, ef[0]), SIGN(1024, ef[1]), O.ADAM_AT_SERVER, T=5)


@pytest.mark.parametrize("d", [1, 3, 100, 255, 256, 257, 1001, 2049])
def test_ragged_and_tiny_sizes(d):
    """Sizes below one chunk, odd sizes (no 16-byte row alignment: scalar path)."""
    _run(d, 3, STOCH(4, O.SCALE_L2, 256), SIGN(512), O.ADAM_AT_SERVER, T=4)
    _run(d, 2, SIGN(0), STOCH(2, O.SCALE_MAX, 0), O.ADAM_AT_WORKER, T=4)


def test_mixed_buckets_and_single_worker():
    _run(5000, 1, STOCH(4, O.SCALE_L2, 2048), STOCH(2, O.SCALE_MAX, 256), O.ADAM_AT_SERVER, T=4)
    _run(5000, 2, SIGN(256), SIGN(2048), O.ADAM_AT_WORKER, T=4)


def test_zero_gradients_give_zero_scales():
    d, N = 1300, 2
    pair = Pair(d, N, STOCH(4, O.SCALE_L2, 256), qfields(O.Q_DET_UNIFORM, 2, bucket=512), O.ADAM_AT_SERVER,
                eps=0.0)
    g = np.zeros((N, d), np.float32)
    g[:, 700:900] = 1e-3
    for t in range(1, 4):
        pair.step(t, g)


# Lean whole-tile kernels take two consecutive tiles per block: odd and even
# tile counts, with and without a ragged tail, a single tile, and more workers
# than waves per block (double-buffered handoff).
@pytest.mark.parametrize("d", [512 * 41 + 384, 512 * 41, 512 * 42, 512 + 100, 512, 1024 * 3])
def test_two_tile_blocks(d):
    _run(d, 16, STOCH(4, O.SCALE_L2, 512), STOCH(4, O.SCALE_L2, 512), O.ADAM_AT_SERVER, T=3)


def test_two_tile_blocks_many_workers():
    _run(512 * 7 + 200, 32, STOCH(2, O.SCALE_MAX, 512), STOCH(2, O.SCALE_MAX, 512), O.ADAM_AT_SERVER, T=3)
    _run(512 * 5, 20, SIGN(512), SIGN(512), O.ADAM_AT_SERVER, T=3)


@pytest.mark.parametrize("N", [100, 1024])
def test_many_workers(N):
    """Many groups of workers per block (double-buffered handoff), up to the
    largest N the library accepts: the specialized, worker-specialized and
    generic kernels, both placements."""
    d = 512 * 2 + 40 if N > 200 else 512 * 4 + 300
    _run(d, N, STOCH(4, O.SCALE_L2, 512), STOCH(4, O.SCALE_L2, 512), O.ADAM_AT_SERVER, T=2)
    _run(d, N, STOCH(4, O.SCALE_MAX, 512), SIGN(256), O.ADAM_AT_WORKER, T=2)
    _run(d, N, qfields(O.Q_DET_UNIFORM, 2, bucket=512), SIGN(1024), O.ADAM_AT_SERVER, T=2)


@pytest.mark.parametrize("N", [3, 4, 5, 8, 17, 100])
def test_one_chunk_tiles_worker_groups(N):
    """One-chunk tiles with Adam at the server run blocks of at most four
    waves, so each wave compresses several workers in turn: worker counts
    below, at and past a multiple of four."""
    d = 256 * 13 + 77
    _run(d, N, STOCH(4, O.SCALE_L2, 256), STOCH(4, O.SCALE_L2, 256), O.ADAM_AT_SERVER, T=3)
    _run(d, N, SIGN(256), qfields(O.Q_TOPK, bucket=256, keep=9), O.ADAM_AT_SERVER, T=2)


WIDE = {
    "sign": lambda b: SIGN(b),
    "stoch4_l2": lambda b: STOCH(4, O.SCALE_L2, b),
    "stoch2_max": lambda b: STOCH(2, O.SCALE_MAX, b),
    "stoch1_l2": lambda b: STOCH(1, O.SCALE_L2, b),
    "stoch8_max": lambda b: STOCH(8, O.SCALE_MAX, b),
}


@pytest.mark.parametrize("bucket", [1024, 2048])
@pytest.mark.parametrize("kind", list(WIDE))
def test_wide_tiles_same_quantizer(kind, bucket):
    """Buckets of 4 and 8 chunks with the same quantizer on both sides and
    Adam at the server: fully specialized kernels whose server side runs on
    one wave per chunk, with fewer workers than chunks (the block then has
    more waves than workers), as many, and more (two worker groups)."""
    q = WIDE[kind](bucket)
    for N in (3, bucket // 256, bucket // 256 + 5):
        _run(bucket * 5 + 700, N, q, q, O.ADAM_AT_SERVER, T=3)


@pytest.mark.parametrize("N", [1, 2, 8, 13])
def test_wide_specialized_workload_kernels(N):
    """The ResNet-18- and GPT-2-medium-sized rounds' kernels (sign 2048 both
    sides; stochastic 2-bit max-norm 1024 / sign 1024) with worker counts
    around the block's waves, both placements."""
    for pl in (O.ADAM_AT_SERVER, O.ADAM_AT_WORKER):
        _run(2048 * 6 + 1576, N, SIGN(2048), SIGN(2048), pl, T=3, gen="segscale")
        _run(1024 * 7 + 704, N, STOCH(2, O.SCALE_MAX, 1024), SIGN(1024), pl, T=3, gen="outliers")


EXTREME_KINDS = {
    "stoch4_l2": STOCH(4, O.SCALE_L2, 512),
    "stoch2_max": STOCH(2, O.SCALE_MAX, 512),
    "sign": SIGN(512),
    "ex1": qfields(O.Q_DET_UNIFORM, 3, bucket=512),
    "ex2": qfields(O.Q_POW2, kmin=-126, kmax=127),
    "topk": qfields(O.Q_TOPK, bucket=512, keep=16),
}


@pytest.mark.parametrize("placement", [O.ADAM_AT_SERVER, O.ADAM_AT_WORKER], ids=["server", "worker"])
@pytest.mark.parametrize("kind", list(EXTREME_KINDS))
def test_extreme_magnitudes(kind, placement):
    """Buckets of subnormal gradients (with and without zeros), of gradients
    near the binary32 maximum (their squares, L2 norms and Adam second moments
    overflow to infinity), of zeros, and mixed: both sides follow the same IEEE
    binary32 steps, so every output still matches."""
    import numpy as np
    d, N = 512 * 6 + 64, 4
    q = EXTREME_KINDS[kind]
    pair = Pair(d, N, q, q, placement, seed=8, eps=0.0)
    rng = np.random.default_rng(4)
    for t in range(1, 4):
        g = np.zeros((N, d), np.float32)
        sgn = rng.choice(np.array([-1.0, 1.0], np.float32), size=(N, d))
        g[:, 0:512] = sgn[:, 0:512] * rng.uniform(1, 100, (N, 512)).astype(np.float32) * np.float32(1e-43)
        g[:, 512:1024] = sgn[:, 512:1024] * rng.uniform(0.5, 3.0, (N, 512)).astype(np.float32) * np.float32(1e38)
        g[:, 1536:2048] = sgn[:, 1536:2048] * np.float32(1e30)
        # subnormal values with zeros: a max-norm below 2^-126, whose reciprocal
        # overflows, and zeros that must still quantize as zeros
        k = rng.integers(-214, 215, (N, 512))
        k[rng.random((N, 512)) < 0.4] = 0
        g[:, 2048:2560] = (k.astype(np.float64) * 2.0 ** -149).astype(np.float32)
        g[:, 2560:] = (sgn[:, 2560:] * rng.standard_normal((N, d - 2560)).astype(np.float32)
                       * np.exp(rng.uniform(-80, 80, (N, d - 2560))).astype(np.float32))
        pair.step(t, g)
        # the float comparison cannot see NaN or infinite entries: require the
        # state bit for bit, NaN in the same places
        for name in ("x", "e_w", "e_s") + (("m", "v") if placement == O.ADAM_AT_SERVER else ("m_w", "v_w")):
            got = getattr(pair.rb, name).cpu().numpy()
            assert same_values(got, getattr(pair.ost, name)), f"step {t}: {name} differs"
        assert pair.stats.resyncs == 0
    pair.check_tie_budget()


ONE_WORKER = [
    ("stoch4_512", STOCH(4, O.SCALE_L2, 512), O.ADAM_AT_SERVER, 512 * 9 + 300),
    ("topk16_512", qfields(O.Q_TOPK, bucket=512, keep=16), O.ADAM_AT_SERVER, 512 * 12 + 64),
    ("sign_256_server", SIGN(256), O.ADAM_AT_SERVER, 256 * 13 + 52),
    ("sign_256_worker", SIGN(256), O.ADAM_AT_WORKER, 256 * 13 + 52),
    ("stoch2_256", STOCH(2, O.SCALE_MAX, 256), O.ADAM_AT_SERVER, 256 * 6),
]


@pytest.mark.parametrize("name,q,placement,d", ONE_WORKER, ids=[c[0] for c in ONE_WORKER])
def test_one_worker_two_tile_blocks(name, q, placement, d):
    """One worker on kernels that take two tiles per block (the specialized
    512-element kernels, the worker-specialized 256-element ones): the block
    still has a wave for each tile's server side."""
    _run(d, 1, q, q, placement, T=3, seed=17)


@pytest.mark.parametrize("placement", [O.ADAM_AT_SERVER, O.ADAM_AT_WORKER], ids=["server", "worker"])
def test_xcd_runs_cover_every_tile(placement):
    """Rows whose byte length is not a multiple of 128 (d = 8 mod 32), one
    2048-element tile per block: the whole-tile launch deals each whole group
    of 128 blocks XCD-major.  300 whole tiles make two whole groups and a
    partial one, plus the ragged tile; every element is checked."""
    d, N = 2048 * 300 + 8, 8
    _run(d, N, SIGN(2048), SIGN(2048), placement, T=2, gen="segscale", seed=13)


@pytest.mark.parametrize("placement", [O.ADAM_AT_SERVER, O.ADAM_AT_WORKER], ids=["server", "worker"])
@pytest.mark.parametrize("eps", [0.0, 1.0], ids=["v0=0", "v0=1"])
def test_adam_magnitude_sweep(placement, eps):
    """Each 512-element tile takes gradients of one binary exponent, from
    2^-75 up to 2^45 (and 2^-149 .. 2^-140 subnormals in the first tiles): the
    Adam moments of successive tiles fall inside, outside and across the range
    in which the kernels form the square root and the division from the
    hardware estimates without operand scaling, so the results on either side
    of each bound are checked bit for bit against the oracle's sqrtf and '/'.
    With v0 = 1 the second moments stay near 1 while |m| crosses its lower
    bound."""
    d, N = 512 * 131, 4
    q = STOCH(4, O.SCALE_L2, 512)
    pair = Pair(d, N, q, q, placement, seed=9, eps=eps)
    rng = np.random.default_rng(21)
    expo = np.concatenate([np.arange(-149, -139), np.arange(-75, 46)]).astype(np.float64)
    assert expo.size * 512 == d
    scale = np.repeat(np.exp2(expo), 512)
    for t in range(1, 4):
        sgn = rng.choice(np.array([-1.0, 1.0]), size=(N, d))
        g = (sgn * rng.uniform(1.0, 2.0, (N, d)) * scale).astype(np.float32)
        g[:, 3 * 512 + 7] = 0.0     # a zero moment in a subnormal tile
        pair.step(t, g)
        for name in ("x", "e_w", "e_s") + (("m", "v") if placement == O.ADAM_AT_SERVER else ("m_w", "v_w")):
            got = getattr(pair.rb, name).cpu().numpy()
            assert same_values(got, getattr(pair.ost, name)), f"step {t}: {name} differs"
        assert pair.stats.resyncs == 0
    pair.check_tie_budget()


@pytest.mark.parametrize("kind", ["stoch2_max", "ex1"])
def test_subnormal_learning_rate(kind):
    """Adam at the workers with lr = 1e-40: every worker's update, hence the
    message scales on both sides (max-norms), is subnormal; x/s is then formed
    with the 2^64 pre-scale on both sides."""
    d, N = 512 * 4 + 300, 4
    q = EXTREME_KINDS[kind]
    pair = Pair(d, N, q, q, O.ADAM_AT_WORKER, seed=12, lr=1e-40)
    for t in range(1, 5):
        g = _grads("student_t", 12, t, N, d)
        g[:, 600:800] = 0.0
        pair.step(t, g)
    pair.check_tie_budget()
    assert np.abs(pair.ost.x).max() > 0


def test_full_precision_messages_unaligned():
    """Messages sent as raw values go out as float4 only when the message
    buffers are 16-byte aligned: an 8-byte aligned worker message array takes
    the checked kernels and gives the same results."""
    d, N = 512 * 6 + 64, 4
    q = qfields(O.Q_NONE)
    for shift in (0, 1):
        pair = Pair(d, N, q, STOCH(2, O.SCALE_MAX, 512), O.ADAM_AT_SERVER, seed=6)
        if shift:
            words = pair.rb.wcodes.shape[1]
            big = torch.zeros(N * words + 1, dtype=torch.uint64, device="cuda")
            pair.rb.wcodes = big[1:].view(N, words)
            assert pair.rb.wcodes.data_ptr() % 16 == 8
        for t in range(1, 4):
            pair.step(t, _grads("student_t", 6, t, N, d))
        pair.check_tie_budget()


def test_zero_buckets_in_lean_kernels():
    """Buckets whose scale is zero take the wave-uniform branch of the
    specialized kernels (bert quantizers, Adam at the server)."""
    d, N = 512 * 9, 16
    pair = Pair(d, N, STOCH(4, O.SCALE_L2, 512), STOCH(4, O.SCALE_L2, 512), O.ADAM_AT_SERVER, eps=0.0)
    g = np.zeros((N, d), np.float32)
    g[:, 1100:1700] = 1e-3
    g[3, 3000:3100] = -2e-3
    for t in range(1, 4):
        pair.step(t, g)
