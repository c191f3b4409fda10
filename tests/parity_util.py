"""Run the HIP path (through the C ABI) and the oracle side by side on the same
seeded inputs and compare every output after every step.

Comparison rule
  * codes: bit-exact, except inside a bucket whose scale differs between the
    two sides; such a scale can differ by at most one binary32 ulp (its
    binary64 sum is formed in a different order) and the code flips it causes
    are counted as rounding-boundary ties (at most 1e-6 of the entries).
  * top-k / random-k messages: kept masks and kept values bit-exact (the
    selection is an integer decision on keys both sides compute exactly).
  * scales, e_w, e_s, x, m, v: |gpu - oracle| <= 1e-5 * |oracle| + floor, the
    floor being 1e-8 of the largest magnitude of that array.
After a step with any tie the GPU state is reset to the oracle's (counted).
"""
from dataclasses import dataclass, field

import numpy as np
import torch

import oracle as O
import paper_2205_14473_amd as E
from paper_2205_14473_amd.state import allocate, init_state

REL_TOL = 1e-5


def qfields(kind, bits=0, scale=O.SCALE_L2, ef=1, bucket=0, kmin=0, kmax=0, keep=0):
    return dict(kind=kind, scale=scale, bits=bits, error_feedback=ef, bucket=bucket, pow2_kmin=kmin,
                pow2_kmax=kmax, keep=keep)


SPARSE_KINDS = (O.Q_TOPK, O.Q_RANDK)


def same_values(got, want):
    """Bit-identical binary32 arrays (any NaN matches any NaN)."""
    got = np.ascontiguousarray(got, np.float32)
    want = np.ascontiguousarray(want, np.float32)
    same = got.view(np.uint32) == want.view(np.uint32)
    return bool(np.all(same | (np.isnan(got) & np.isnan(want))))


def configs(d, N, qw, qs, placement=O.ADAM_AT_SERVER, seed=1, beta1=0.9, beta2=0.999, lr=1e-3, eps=1e-8):
    common = dict(d=d, N=N, placement=placement, beta1=beta1, beta2=beta2, lr=lr, eps=eps, seed=seed)
    return (O.Config(**common, qw=O.Quant(**qw), qs=O.Quant(**qs)),
            E.Config(**common, qw=E.Quant(**qw), qs=E.Quant(**qs)))


@dataclass
class Stats:
    steps: int = 0
    code_entries: int = 0
    code_ties: int = 0
    scale_ties: int = 0
    resyncs: int = 0
    max_rel: dict = field(default_factory=dict)

    def note(self, name, rel):
        self.max_rel[name] = max(self.max_rel.get(name, 0.0), rel)


def _ulp_diff(a, b):
    ai = a.astype(np.float32).view(np.int32).astype(np.int64)
    bi = b.astype(np.float32).view(np.int32).astype(np.int64)
    return np.abs(ai - bi)


def close(name, got, want, stats):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, (name, got.shape, want.shape)
    if want.size == 0:
        return
    floor = 1e-8 * float(np.max(np.abs(want)))
    err = np.abs(got - want)
    bad = err > REL_TOL * np.abs(want) + floor
    rel = float(np.max(err / (np.abs(want) + floor + 1e-300)))
    stats.note(name, rel)
    if bad.any():
        idx = np.argwhere(bad)[:5]
        raise AssertionError(f"{name}: {int(bad.sum())} entries beyond tolerance; first {idx.tolist()} "
                             f"got {got[bad][:5]} want {want[bad][:5]}")


def _codes_match(q_o, bits, d, n0, got_words, want_words, got_scales, want_scales, stats, what):
    """Per-element code comparison with the bucket tie rule; returns ties."""
    if bits == 32:
        assert np.array_equal(got_words, want_words), f"{what}: raw message differs"
        return 0
    length = want_words.shape[-1] // (4 * bits) * 256
    gw = O.unpack(bits, np.ascontiguousarray(got_words), length)
    ow = O.unpack(bits, np.ascontiguousarray(want_words), length)
    diff = gw != ow
    if not diff.any():
        return 0
    if want_scales is None or want_scales.size == 0:
        raise AssertionError(f"{what}: {int(diff.sum())} code mismatches in a quantizer without scales")
    B = O.bucket_len(q_o, d)
    bad_buckets = np.nonzero(got_scales != want_scales)[0]
    where = np.nonzero(diff)[0]
    bucket_of = (n0 + where) // B - n0 // B
    untied = ~np.isin(bucket_of, bad_buckets)
    if untied.any():
        raise AssertionError(f"{what}: {int(untied.sum())} code mismatches in buckets with identical scales, "
                             f"first elements {where[untied][:8].tolist()}")
    return int(diff.sum())


class Pair:
    """The oracle and the HIP path stepping the same configuration."""

    def __init__(self, d, N, qw, qs, placement=O.ADAM_AT_SERVER, seed=1, x1=None, split=False, sched=None,
                 mode=None, **hp):
        """mode: "step" (ea_step), "split" (the four calls), "scheduled"
        (ea_step_scheduled, step index on the device), "run" (ea_run, one
        step per call) or "graph" (ea_step_scheduled captured once in a HIP
        graph and replayed); the last three take lr, beta2 from `sched`."""
        self.oc, self.ec = configs(d, N, qw, qs, placement, seed, **hp)
        self.mode = mode or ("split" if split else "step")
        self.sched = sched
        if sched is not None:
            self.so, self.se = O.Schedule(**sched), E.Schedule(**sched)
            self.t_dev = torch.zeros(1, dtype=torch.int32, device="cuda")
        self.graph = None
        self.d, self.N = d, N
        x1 = np.zeros(d, np.float32) if x1 is None else np.asarray(x1, np.float32)
        self.ost = O.State.init(self.oc, d, x1)
        self.rb = allocate(self.ec, with_u=True)
        init_state(self.ec, self.rb)
        self.rb.x.copy_(torch.from_numpy(x1))
        self.split = self.mode == "split"
        self.stats = Stats()
        self.bw, self.bs = O.code_bits(self.oc.qw), O.code_bits(self.oc.qs)
        self.nsw, self.nss = E.ea_msg_scales(self.ec.qw, d), E.ea_msg_scales(self.ec.qs, d)
        self.sparse_w, self.sparse_s = self.oc.qw.kind in SPARSE_KINDS, self.oc.qs.kind in SPARSE_KINDS
        torch.cuda.synchronize()

    def oracle_config(self, t):
        if self.sched is None:
            return self.oc
        c = O.Config.from_buffer_copy(self.oc)
        c.lr, c.beta2 = (float(v) for v in O.schedule_at(self.so, self.oc.lr, self.oc.beta2, t))
        return c

    def gpu_step(self, t):
        rb, c = self.rb, self.ec
        if self.mode == "step":
            E.ea_step(c, t, **rb.step_args())
            return
        args = rb.step_args()
        if self.mode == "scheduled":
            self.t_dev.fill_(t)
            E.ea_step_scheduled(c, self.se, self.t_dev, **args)
            return
        if self.mode == "run":
            g = args.pop("g")
            E.ea_run(c, self.se, t, 1, g, 0, **args)
            return
        if self.mode == "graph":
            if self.graph is None:
                self.t_dev.fill_(t)
                torch.cuda.synchronize()
                self.graph = torch.cuda.CUDAGraph()
                with torch.cuda.graph(self.graph):
                    E.ea_step_scheduled(c, self.se, self.t_dev, **args)
            assert int(self.t_dev.item()) == t, "graph replay out of step with the oracle"
            self.graph.replay()
            return
        for i in range(self.N):
            E.ea_worker_compress(c, i, t, rb.g[i], rb.e_w[i], None if rb.m_w is None else rb.m_w[i],
                                 None if rb.v_w is None else rb.v_w[i], rb.wcodes[i],
                                 rb.wscales[i] if self.nsw else None, rb.workspace)
        E.ea_server_aggregate_adam(c, t, rb.wcodes, rb.wscales if self.nsw else None, rb.m, rb.v, rb.u)
        E.ea_server_compress(c, t, rb.u, rb.e_s, rb.scodes, rb.sscales if self.nss else None, rb.workspace)
        E.ea_worker_apply(c, rb.scodes, rb.sscales if self.nss else None, rb.x)

    def step(self, t, g):
        g = np.ascontiguousarray(g, np.float32)
        out = O.step(self.oracle_config(t), t, g, self.ost, want_srv_in=self.split)
        self.rb.g.copy_(torch.from_numpy(g))
        self.gpu_step(t)
        torch.cuda.synchronize()
        if self.mode in ("scheduled", "graph"):
            assert int(self.t_dev.item()) == t + 1, "the round did not advance its step counter"
        self.compare(out)
        self.stats.steps += 1
        return out

    def compare(self, out):
        rb, st, s = self.rb, self.ost, self.stats
        ties = 0
        ws_g = rb.wscales.cpu().numpy()[:, :self.nsw]
        ss_g = rb.sscales.cpu().numpy()[:self.nss]
        if self.sparse_w:
            assert same_values(ws_g, out["wscales"]), "worker kept values differ"
        elif self.nsw:
            assert np.all(_ulp_diff(ws_g, out["wscales"]) <= 1), "worker scales differ by more than 1 ulp"
            s.scale_ties += int((ws_g != out["wscales"]).sum())
        if self.sparse_s:
            assert same_values(ss_g, out["sscales"]), "server kept values differ"
        elif self.nss:
            assert np.all(_ulp_diff(ss_g, out["sscales"]) <= 1), "server scales differ by more than 1 ulp"
            s.scale_ties += int((ss_g != out["sscales"]).sum())
        wsc = self.nsw and not self.sparse_w
        ssc = self.nss and not self.sparse_s
        wc = rb.wcodes.cpu().numpy()
        for i in range(self.N):
            ties += _codes_match(self.oc.qw, self.bw, self.d, 0, wc[i], out["wcodes"][i],
                                 ws_g[i] if wsc else None, out["wscales"][i] if wsc else None,
                                 s, f"worker {i} codes")
        ties += _codes_match(self.oc.qs, self.bs, self.d, 0, rb.scodes.cpu().numpy(), out["scodes"],
                             ss_g if ssc else None, out["sscales"] if ssc else None, s, "server codes")
        s.code_entries += (self.N + 1) * self.d
        s.code_ties += ties
        close("wscales", ws_g, out["wscales"], s)
        close("sscales", ss_g, out["sscales"], s)
        close("e_w", rb.e_w.cpu().numpy(), st.e_w, s)
        close("e_s", rb.e_s.cpu().numpy(), st.e_s, s)
        close("x", rb.x.cpu().numpy(), st.x, s)
        if st.m is not None:
            close("m", rb.m.cpu().numpy(), st.m, s)
            close("v", rb.v.cpu().numpy(), st.v, s)
        if st.m_w is not None:
            close("m_w", rb.m_w.cpu().numpy(), st.m_w, s)
            close("v_w", rb.v_w.cpu().numpy(), st.v_w, s)
        if self.split and out.get("srv_in") is not None:
            close("u", rb.u.cpu().numpy(), out["srv_in"], s)
        exact = (same_values(rb.x.cpu().numpy(), st.x) and same_values(rb.e_w.cpu().numpy(), st.e_w)
                 and same_values(rb.e_s.cpu().numpy(), st.e_s))
        if ties or not exact:
            self.resync()

    def resync(self):
        rb, st = self.rb, self.ost
        rb.e_w.copy_(torch.from_numpy(st.e_w))
        rb.e_s.copy_(torch.from_numpy(st.e_s))
        rb.x.copy_(torch.from_numpy(st.x))
        if st.m is not None:
            rb.m.copy_(torch.from_numpy(st.m))
            rb.v.copy_(torch.from_numpy(st.v))
        if st.m_w is not None:
            rb.m_w.copy_(torch.from_numpy(st.m_w))
            rb.v_w.copy_(torch.from_numpy(st.v_w))
        torch.cuda.synchronize()
        self.stats.resyncs += 1

    def check_tie_budget(self):
        s = self.stats
        assert s.code_ties <= max(1e-6 * s.code_entries, 0), (
            f"{s.code_ties} tie flips over {s.code_entries} entries exceed 1e-6")
