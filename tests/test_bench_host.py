"""The benchmark's byte accounting (CPU only): the algorithmic bytes that the
roofline divides by the round time, counted here from what each vector of the
round does (read, write, or both) and from message sizes derived from the
code width and bucket, for the workloads the benchmark reports."""
import math

import pytest

import bench
import workloads as W

E = pytest.importorskip("paper_2205_14473_amd")


def _cfg(key, placement=None):
    w = W.WORKLOADS[key]
    return E.Config(**w.config_fields(placement=placement), qw=E.Quant(**w.qw.fields()),
                    qs=E.Quant(**w.qs.fields())), w


def _message_bytes(q, d):
    """Codes: one bit plane per code bit over 256-element chunks (the last one
    padded); per bucket one 4-byte scale, or `keep` 4-byte values for a
    sparsifier; full precision sends the floats."""
    if q.kind == E.EA_Q_NONE:
        return 4 * d + (4 * d) % 8          # whole 8-byte words
    bits = 1 if q.kind in (E.EA_Q_TOPK, E.EA_Q_RANDK, E.EA_Q_SCALED_SIGN) else q.bits
    if q.kind == E.EA_Q_POW2:
        bits = 1 + math.ceil(math.log2(q.pow2_kmax - q.pow2_kmin + 2))
    codes = math.ceil(d / 256) * 256 * bits // 8
    nb = 1 if q.bucket == 0 else math.ceil(d / q.bucket)
    per = q.keep if q.kind in (E.EA_Q_TOPK, E.EA_Q_RANDK) else (0 if q.kind == E.EA_Q_POW2 else 1)
    return codes + 4 * nb * per


@pytest.mark.parametrize("key", ["bert", "gpt2m", "resnet50", "resnet18", "bert_topk", "bert_randk", "bert_topk2048",
                                 "bert_randk2048"])
@pytest.mark.parametrize("placement", [0, 1], ids=["server", "worker"])
def test_algorithmic_bytes(key, placement):
    cfg, w = _cfg(key, placement)
    d, N = w.d, w.N
    if placement == E.EA_ADAM_AT_SERVER:
        per_worker = 4 * d + 2 * 4 * d                  # g read; e_w read and written
        server = 4 * 2 * 4 * d                          # m, v, e_s, x read and written
    else:
        per_worker = 4 * d + 3 * 2 * 4 * d              # g read; e_w, m_w, v_w read and written
        server = 2 * 2 * 4 * d                          # e_s, x read and written
    want = N * (per_worker + _message_bytes(cfg.qw, d)) + server + _message_bytes(cfg.qs, d)
    assert bench.algorithmic_bytes(E, cfg) == want


def test_headline_bytes_per_parameter():
    """BERT-sized, 16 workers, 4-bit codes and 512-element buckets on both
    sides: 16 * (12 + 0.5 + 4/512) + 32 + 0.5 + 4/512 bytes per parameter, up
    to the padding of the last chunk and bucket."""
    cfg, w = _cfg("bert")
    per_param = bench.algorithmic_bytes(E, cfg) / w.d
    assert abs(per_param - (17 * (0.5 + 4 / 512) + 16 * 12 + 32)) < 1e-4
    assert round(per_param, 2) == 232.63


@pytest.mark.parametrize("key", ["bert", "resnet50", "bert_topk"])
def test_split_bytes(key):
    """The split calls add, to the fused round's bytes, every worker message
    read back, u written and read back, and the server message read back."""
    cfg, w = _cfg(key)
    d, N = w.d, w.N
    extra = N * _message_bytes(cfg.qw, d) + 2 * 4 * d + _message_bytes(cfg.qs, d)
    assert bench.split_bytes(E, cfg) == bench.algorithmic_bytes(E, cfg) + extra
