"""Seeded synthetic workloads: shapes and gradient generators.

This module holds the workload table and the input generators only; it holds
none of the optimizer's arithmetic.  Both the HIP path's tests/benchmark and
the oracle's tests draw their inputs from here.

The paper's own workloads (CIFAR-100 / ResNet-18, IMDB / BiGRU on BERT
encodings; Section V-B and V-C) need datasets and trained encoders; these
generators stand in for their gradients with the parameter counts and value
distributions listed below.  The toy quadratic is fully synthetic.

Recipes (all float32):
  toy        g_i = (x - x_star) + 0.1 * z,  x_star ~ N(0, 1) drawn once, x_1 = 0
  segscale   g_i = sigma_seg * z, sigma_seg ~ LogUniform[1e-4, 1e-1] drawn once per
             run for each 4096-element segment (a stand-in for per-layer scale)
  student_t  g_i = 1e-3 * z / sqrt(chi2_3 / 3)  (Student-t with 3 degrees of freedom)
  outliers   g_i = 1e-3 * z, times 100 where a Bernoulli(0.01) draw is set
z ~ N(0, 1) is drawn fresh per (worker, step).
"""
from dataclasses import dataclass, field
from typing import Dict

import numpy as np

Q_NONE, Q_SCALED_SIGN, Q_STOCH_UNIFORM, Q_DET_UNIFORM, Q_POW2, Q_TOPK, Q_RANDK = 0, 1, 2, 3, 4, 5, 6
SCALE_L1, SCALE_L2, SCALE_MAX = 0, 1, 2
ADAM_AT_SERVER, ADAM_AT_WORKER = 0, 1


@dataclass(frozen=True)
class QSpec:
    kind: int
    bits: int = 0
    scale: int = SCALE_L2
    error_feedback: int = 1
    bucket: int = 0
    pow2_kmin: int = 0
    pow2_kmax: int = 0
    keep: int = 0

    def fields(self) -> Dict[str, int]:
        return dict(kind=self.kind, scale=self.scale, bits=self.bits,
                    error_feedback=self.error_feedback, bucket=self.bucket,
                    pow2_kmin=self.pow2_kmin, pow2_kmax=self.pow2_kmax, keep=self.keep)


@dataclass(frozen=True)
class Workload:
    key: str
    name: str
    d: int
    N: int
    qw: QSpec
    qs: QSpec
    steps: int
    seed: int
    gen: str
    beta1: float = 0.9
    beta2: float = 0.999
    lr: float = 1e-3
    eps: float = 1e-8
    placement: int = ADAM_AT_SERVER
    extra: Dict[str, float] = field(default_factory=dict)

    def config_fields(self, placement=None, d=None):
        return dict(d=self.d if d is None else d, N=self.N,
                    placement=self.placement if placement is None else placement,
                    beta1=self.beta1, beta2=self.beta2, lr=self.lr, eps=self.eps, seed=self.seed)


SIGN1 = lambda b: QSpec(Q_SCALED_SIGN, 1, SCALE_L1, 1, b)  # noqa: E731
SPARSE = lambda kind, keep, b: QSpec(kind, 0, SCALE_L2, 1, b, keep=keep)  # noqa: E731

WORKLOADS = {
    "toy": Workload("toy", "toy-convex d=65536 N=4", 65536, 4, SIGN1(0), SIGN1(0), 100, 1, "toy"),
    "resnet18": Workload("resnet18", "ResNet-18-sized d=11689512 N=8", 11_689_512, 8,
                         SIGN1(2048), SIGN1(2048), 50, 2, "segscale"),
    "resnet50": Workload("resnet50", "ResNet-50-sized d=25557032 N=32", 25_557_032, 32,
                         QSpec(Q_STOCH_UNIFORM, 2, SCALE_MAX, 1, 512),
                         QSpec(Q_STOCH_UNIFORM, 2, SCALE_MAX, 1, 512), 50, 3, "segscale"),
    "bert": Workload("bert", "BERT-base-sized d=110000000 N=16", 110_000_000, 16,
                     QSpec(Q_STOCH_UNIFORM, 4, SCALE_L2, 1, 512),
                     QSpec(Q_STOCH_UNIFORM, 4, SCALE_L2, 1, 512), 20, 4, "student_t"),
    "gpt2m": Workload("gpt2m", "GPT-2-medium-sized d=355000000 N=8", 355_000_000, 8,
                      QSpec(Q_STOCH_UNIFORM, 2, SCALE_MAX, 1, 1024), SIGN1(1024), 10, 5, "outliers"),
    # Definition 3 compressors on the BERT-sized round: 16 of every 512 kept
    # (a 1-bit kept mask plus 16 values per bucket: 2 bits per parameter).
    "bert_topk": Workload("bert_topk", "BERT-base-sized d=110000000 N=16, top-16 of 512", 110_000_000, 16,
                          SPARSE(Q_TOPK, 16, 512), SPARSE(Q_TOPK, 16, 512), 20, 4, "student_t"),
    "bert_randk": Workload("bert_randk", "BERT-base-sized d=110000000 N=16, random-16 of 512", 110_000_000, 16,
                           SPARSE(Q_RANDK, 16, 512), SPARSE(Q_RANDK, 16, 512), 20, 4, "student_t"),
    # the same density on 2048-element buckets (8-chunk tiles)
    "bert_topk2048": Workload("bert_topk2048", "BERT-base-sized d=110000000 N=16, top-64 of 2048", 110_000_000, 16,
                              SPARSE(Q_TOPK, 64, 2048), SPARSE(Q_TOPK, 64, 2048), 20, 4, "student_t"),
    "bert_randk2048": Workload("bert_randk2048", "BERT-base-sized d=110000000 N=16, random-64 of 2048", 110_000_000,
                               16, SPARSE(Q_RANDK, 64, 2048), SPARSE(Q_RANDK, 64, 2048), 20, 4, "student_t"),
}

# The paper's toy problem (Section V-A): 500x500, 10 workers, beta 0.9, theta 0.99.
PAPER_TOY = dict(d=500, N=10, beta1=0.9, beta2=0.99, x_star_var=0.1, xi_var=0.1)


def seg_sigma(seed: int, d: int, seg: int = 4096) -> np.ndarray:
    """Per-segment scales sigma ~ LogUniform[1e-4, 1e-1], one per 4096 elements."""
    rng = np.random.default_rng([seed, 0x5E6])
    nseg = -(-d // seg)
    return np.exp(rng.uniform(np.log(1e-4), np.log(1e-1), nseg)).astype(np.float32)


def host_gradients(w: Workload, t: int, d: int = None, x: np.ndarray = None,
                   x_star: np.ndarray = None) -> np.ndarray:
    """[N, d] float32 gradients for step t on the host (numpy)."""
    d = w.d if d is None else d
    rng = np.random.default_rng([w.seed, t, 0x6EAD])
    z = rng.standard_normal((w.N, d), dtype=np.float32)
    if w.gen == "toy":
        assert x is not None and x_star is not None
        return ((x - x_star)[None, :] + np.float32(0.1) * z).astype(np.float32)
    if w.gen == "segscale":
        sig = np.repeat(seg_sigma(w.seed, d), 4096)[:d]
        return (z * sig[None, :]).astype(np.float32)
    if w.gen == "student_t":
        chi = (rng.standard_normal((3, w.N, d), dtype=np.float32) ** 2).sum(0)
        return (np.float32(1e-3) * z / np.sqrt(chi / np.float32(3.0))).astype(np.float32)
    if w.gen == "outliers":
        hit = rng.random((w.N, d), dtype=np.float32) < 0.01
        return (np.float32(1e-3) * z * np.where(hit, np.float32(100.0), np.float32(1.0))).astype(np.float32)
    raise ValueError(w.gen)


def toy_x_star(w: Workload, d: int = None) -> np.ndarray:
    d = w.d if d is None else d
    return np.random.default_rng([w.seed, 0x57A2]).standard_normal(d, dtype=np.float32)


def initial_x(w: Workload, d: int = None) -> np.ndarray:
    """x_1: zero for the toy, N(0, 0.02^2) otherwise (Algorithm 1 leaves it free)."""
    d = w.d if d is None else d
    if w.gen == "toy":
        return np.zeros(d, np.float32)
    return (np.float32(0.02) * np.random.default_rng([w.seed, 0x1]).standard_normal(d, dtype=np.float32))


def device_gradients(w: Workload, t: int, out, d: int = None, x=None, x_star=None):
    """Fill a torch tensor out[N, d] on its device with step-t gradients (torch RNG).

    Used where host generation of N*d values would dominate (the benchmark and
    full-size checks); the recipe is the one in the module docstring.  The toy
    quadratic's gradient (x - x_star) + 0.1 z needs x and x_star (device
    tensors); without them only the noise term is drawn.
    """
    import torch
    d = w.d if d is None else d
    gen = torch.Generator(device=out.device)
    gen.manual_seed(w.seed * 1_000_003 + t)
    if w.gen == "segscale":
        sig = torch.from_numpy(np.repeat(seg_sigma(w.seed, d), 4096)[:d]).to(out.device)
    for i in range(w.N):
        row = out[i]
        torch.randn(d, generator=gen, device=out.device, out=row)
        if w.gen == "segscale":
            row.mul_(sig)
        elif w.gen == "student_t":
            chi = torch.zeros(d, device=out.device)
            for _ in range(3):
                zz = torch.randn(d, generator=gen, device=out.device)
                chi.addcmul_(zz, zz)
            row.mul_(1e-3).div_(torch.sqrt(chi / 3.0))
        elif w.gen == "outliers":
            hit = torch.rand(d, generator=gen, device=out.device) < 0.01
            row.mul_(1e-3)
            row[hit] *= 100.0
        elif w.gen == "toy":
            row.mul_(0.1)
            if x is not None:
                row.add_(x - x_star)
        else:
            raise ValueError(f"device generation not defined for {w.gen}")
    return out
