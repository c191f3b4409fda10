"""Run the HIP path (through the C ABI) and the oracle side by side on the same
seeded inputs and compare every output after every step.

Comparison rule
  * Every element step of the round is the same IEEE binary32 operation on
    both sides (no contraction, correctly rounded division and square root,
    workers added in ascending order), so with equal bucket scales the GPU's
    messages and state must equal the oracle's bit for bit.
  * A bucket sum (L1, L2) is formed in binary64 in another order on the GPU
    (lane partials, then a DPP/permlane tree) than in the oracle (serial).  The
    two can round to binary32 scales one ulp apart; simulated on 10^6
    Student-t buckets this never happened, and it is estimated at about 4e-8
    per bucket.  Such a "tied" bucket is checked exactly all the same: the
    oracle re-quantizes its own quantizer input for that bucket under the
    GPU's scale (same draws), and the GPU's codes and residuals must equal that
    result.  State that a tie cannot reach must still match bit for bit; the
    elements a tie reaches downstream are not compared that round, and the
    GPU state is then reset to the oracle's.  A round with a tie fails the
    test unless the test allows ties (max_tie_rounds), and a reset without a
    validated tie is impossible.
  * top-k / random-k messages: kept masks and kept values bit-exact (the
    selection is an integer decision on keys both sides compute exactly).
  * close() (the float tolerance |gpu - oracle| <= 1e-5 |oracle| + floor, the
    floor being 1e-8 of the largest finite magnitude of the array) is used for
    reporting and where a test compares against values the oracle did not
    produce by the same steps; it requires non-finite entries to match
    exactly (NaN where the oracle has NaN, the same signed infinities).
"""
from dataclasses import dataclass, field

import numpy as np

import oracle as O

REL_TOL = 1e-5
SPARSE_KINDS = (O.Q_TOPK, O.Q_RANDK)
SCALED_KINDS = (O.Q_SCALED_SIGN, O.Q_STOCH_UNIFORM, O.Q_DET_UNIFORM)
SERVER_STREAM = 0xFFFFFFFF


def qfields(kind, bits=0, scale=O.SCALE_L2, ef=1, bucket=0, kmin=0, kmax=0, keep=0):
    return dict(kind=kind, scale=scale, bits=bits, error_feedback=ef, bucket=bucket, pow2_kmin=kmin,
                pow2_kmax=kmax, keep=keep)


def same_values(got, want):
    """Bit-identical binary32 arrays (any NaN matches any NaN)."""
    got = np.ascontiguousarray(got, np.float32)
    want = np.ascontiguousarray(want, np.float32)
    if got.shape != want.shape:
        return False
    same = got.view(np.uint32) == want.view(np.uint32)
    return bool(np.all(same | (np.isnan(got) & np.isnan(want))))


def first_diff(got, want, k=5):
    got = np.ascontiguousarray(got, np.float32).ravel()
    want = np.ascontiguousarray(want, np.float32).ravel()
    bad = (got.view(np.uint32) != want.view(np.uint32)) & ~(np.isnan(got) & np.isnan(want))
    idx = np.nonzero(bad)[0][:k]
    return f"{int(bad.sum())} entries differ; first {idx.tolist()} got {got[idx].tolist()} want {want[idx].tolist()}"


def configs(d, N, qw, qs, placement=O.ADAM_AT_SERVER, seed=1, beta1=0.9, beta2=0.999, lr=1e-3, eps=1e-8):
    import paper_2205_14473_amd as E
    common = dict(d=d, N=N, placement=placement, beta1=beta1, beta2=beta2, lr=lr, eps=eps, seed=seed)
    return (O.Config(**common, qw=O.Quant(**qw), qs=O.Quant(**qs)),
            E.Config(**common, qw=E.Quant(**qw), qs=E.Quant(**qs)))


@dataclass
class Stats:
    steps: int = 0
    code_entries: int = 0
    code_ties: int = 0        # code flips inside tied buckets (validated under the GPU scale)
    scale_ties: int = 0       # buckets whose scales differ by one ulp
    tie_rounds: int = 0       # rounds with at least one tied bucket
    resyncs: int = 0          # GPU state resets to the oracle's (one per tie round)
    max_rel: dict = field(default_factory=dict)

    def note(self, name, rel):
        self.max_rel[name] = max(self.max_rel.get(name, 0.0), rel)


def _ulp_diff(a, b):
    ai = np.asarray(a, np.float32).view(np.int32).astype(np.int64)
    bi = np.asarray(b, np.float32).view(np.int32).astype(np.int64)
    return np.abs(ai - bi)


def close(name, got, want, stats):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, (name, got.shape, want.shape)
    if want.size == 0:
        return
    gnan, wnan = np.isnan(got), np.isnan(want)
    if (gnan != wnan).any():
        idx = np.argwhere(gnan != wnan)[:5]
        raise AssertionError(f"{name}: {int((gnan != wnan).sum())} entries NaN on one side only; first "
                             f"{idx.tolist()} got {got[gnan != wnan][:5]} want {want[gnan != wnan][:5]}")
    ginf, winf = np.isinf(got), np.isinf(want)
    if (ginf != winf).any() or (got[winf] != want[winf]).any():
        bad = (ginf != winf) | (winf & (got != want))
        idx = np.argwhere(bad)[:5]
        raise AssertionError(f"{name}: {int(bad.sum())} infinite entries differ; first {idx.tolist()} "
                             f"got {got[bad][:5]} want {want[bad][:5]}")
    fin = np.isfinite(want)
    if not fin.any():
        return
    gf, wf = got[fin], want[fin]
    floor = 1e-8 * float(np.max(np.abs(wf)))
    err = np.abs(gf - wf)
    bad = err > REL_TOL * np.abs(wf) + floor
    rel = float(np.max(err / (np.abs(wf) + floor + 1e-300)))
    stats.note(name, rel)
    if bad.any():
        pos = np.argwhere(fin)[bad][:5]
        raise AssertionError(f"{name}: {int(bad.sum())} entries beyond tolerance; first {pos.tolist()} "
                             f"got {gf[bad][:5]} want {wf[bad][:5]}")


def needs_draws(q):
    return q.kind in (O.Q_STOCH_UNIFORM, O.Q_RANDK)


def check_message(q, d, n0, seed, t, stream, p, got_words, got_scales, want_words, want_scales, stats, what,
                  skip=None):
    """One message on the segment [n0, n0 + len(p)) against the oracle's.

    `skip` (a bool mask over the segment, or None) marks elements whose input
    an earlier tie in the round has changed; buckets that contain one are not
    compared.  Returns the tied buckets as (start, length, residual), the
    residual being what the GPU must hold there: p - Q(p) under the GPU's
    scale (0 without error feedback)."""
    length = p.size
    bits = O.code_bits(q)
    keep = np.ones(length, bool) if skip is None else ~np.asarray(skip, bool)
    gc = O.unpack(bits, np.ascontiguousarray(got_words), length)
    oc = O.unpack(bits, np.ascontiguousarray(want_words), length)
    if q.kind not in SCALED_KINDS:
        if not np.array_equal(gc[keep], oc[keep]):
            where = np.nonzero((gc != oc) & keep)[0][:8]
            raise AssertionError(f"{what}: codes differ at {where.tolist()} (no scale, so no tie is possible)")
        if q.kind in SPARSE_KINDS:
            B, k = O.bucket_len(q, d), q.keep
            for b in range(-(-length // B)):
                if keep[b * B] and not same_values(got_scales[b * k:(b + 1) * k], want_scales[b * k:(b + 1) * k]):
                    raise AssertionError(f"{what}: kept values of bucket {b} differ: "
                                         f"{first_diff(got_scales[b * k:(b + 1) * k], want_scales[b * k:(b + 1) * k])}")
        return []
    B = O.bucket_len(q, d)
    gs = np.ascontiguousarray(got_scales, np.float32)
    ws = np.ascontiguousarray(want_scales, np.float32)
    assert gs.shape == ws.shape, (what, gs.shape, ws.shape)
    live = keep[::B][:gs.size]
    equal = (gs.view(np.uint32) == ws.view(np.uint32)) | (np.isnan(gs) & np.isnan(ws))
    ulps = _ulp_diff(gs, ws)
    wrong = live & ~equal & ((ulps > 1) | np.isnan(gs) | np.isnan(ws) | (np.signbit(gs) != np.signbit(ws)))
    if wrong.any():
        bad = np.nonzero(wrong)[0][:5]
        raise AssertionError(f"{what}: scales differ by more than one ulp in buckets {bad.tolist()}: "
                             f"got {gs[bad].tolist()} want {ws[bad].tolist()}")
    tied = []
    for b in np.nonzero(live & ~equal)[0].tolist():
        b0 = b * B
        n = min(B, length - b0)
        u = O.uniforms(seed, t, stream, n0 + b0, n) if needs_draws(q) else None
        codes_t, deq_t = O.quantize_bucket(q, p[b0:b0 + n], float(gs[b]), u)
        if not np.array_equal(gc[b0:b0 + n], codes_t):
            bad = np.nonzero(gc[b0:b0 + n] != codes_t)[0][:8]
            raise AssertionError(f"{what}: bucket {b} (scale {gs[b]!r} vs {ws[b]!r}): codes differ from the "
                                 f"oracle's quantization under the GPU's scale at {bad.tolist()}")
        stats.scale_ties += 1
        stats.code_ties += int((codes_t != oc[b0:b0 + n]).sum())
        res = (p[b0:b0 + n] - deq_t).astype(np.float32) if q.error_feedback else np.zeros(n, np.float32)
        tied.append((b0, n, res))
    untied = keep.copy()
    for b0, n, _ in tied:
        untied[b0:b0 + n] = False
    if not np.array_equal(gc[untied], oc[untied]):
        where = np.nonzero((gc != oc) & untied)[0][:8]
        raise AssertionError(f"{what}: codes differ in buckets whose scales are equal, first elements "
                             f"{where.tolist()}")
    return tied


class RoundCheck:
    """Compares one round of the GPU on the segment [n0, n0+len) of the
    d-vector (the whole vector, or a bucket-aligned piece) with the oracle's
    O.step(..., want_inputs=True) output `out` for the same segment."""

    def __init__(self, oc, d, n0, t, out, stats, what=""):
        self.oc, self.d, self.n0, self.t, self.out, self.stats, self.what = oc, d, n0, t, out, stats, what
        self.length = out["p_w"].shape[1]
        self.worker_ties = {}       # worker -> [(b0, n, residual)]
        self.server_ties = []
        self.reach = np.zeros(self.length, bool)   # elements a tie reaches downstream

    def _widen(self, ties):
        # A worker's tie changes the server's input over its bucket, hence the
        # server's scale over every server bucket that overlaps it; a server
        # tie changes its bucket.  Buckets nest, so widen to the larger one.
        oc = self.oc
        span = max(O.bucket_len(oc.qw, self.d), O.bucket_len(oc.qs, self.d))
        for b0, n, _ in ties:
            lo = (self.n0 + b0) // span * span - self.n0
            hi = -(-(self.n0 + b0 + n) // span) * span - self.n0
            self.reach[max(lo, 0):min(hi, self.length)] = True

    def messages(self, wcodes, wscales, scodes, sscales):
        oc, out = self.oc, self.out
        N = oc.N
        none = np.zeros(0, np.float32)
        for i in range(N):
            tw = check_message(oc.qw, self.d, self.n0, oc.seed, self.t, i, out["p_w"][i], wcodes[i],
                               wscales[i] if out["wscales"].size else none, out["wcodes"][i],
                               out["wscales"][i] if out["wscales"].size else none,
                               self.stats, f"{self.what}worker {i} message")
            if tw:
                self.worker_ties[i] = tw
                self._widen(tw)
        self.server_ties = check_message(oc.qs, self.d, self.n0, oc.seed, self.t, SERVER_STREAM, out["q_s"],
                                         scodes, sscales, out["scodes"], out["sscales"], self.stats,
                                         f"{self.what}server message", skip=self.reach)
        self._widen(self.server_ties)
        self.stats.code_entries += (N + 1) * self.length
        return self.tied

    @property
    def tied(self):
        return bool(self.worker_ties) or bool(self.server_ties)

    def _exact(self, name, got, want, mask=None):
        got = np.ascontiguousarray(got, np.float32)
        want = np.ascontiguousarray(want, np.float32)
        assert got.shape == want.shape, (name, got.shape, want.shape)
        if mask is not None:
            got, want = got[..., mask], want[..., mask]
        if not same_values(got, want):
            rep = Stats()
            try:
                close(name, got, want, rep)
                verdict = f"within the float tolerance (max rel {rep.max_rel.get(name, 0.0):.3g})"
            except AssertionError as e:
                verdict = f"beyond the float tolerance: {e}"
            raise AssertionError(f"{self.what}{name}: not bit-identical to the oracle ({first_diff(got, want)}); "
                                 f"{verdict}")

    def state(self, gpu, st, srv_in=None, gpu_u=None):
        """gpu: dict of numpy arrays (e_w [N][len], e_s, x, m, v, m_w, v_w) for
        the segment; st: the oracle's State after the round."""
        keep = ~self.reach
        e_w = np.array(gpu["e_w"], np.float32, copy=True)
        want_e_w = np.array(st.e_w, np.float32, copy=True)
        for i, ties in self.worker_ties.items():
            for b0, n, res in ties:
                self._exact(f"e_w[{i}] of tied bucket at {self.n0 + b0}", e_w[i, b0:b0 + n], res)
                want_e_w[i, b0:b0 + n] = e_w[i, b0:b0 + n]
        self._exact("e_w", e_w, want_e_w)
        for name in ("m_w", "v_w"):
            if getattr(st, name) is not None:
                self._exact(name, gpu[name], getattr(st, name))     # before any quantization
        for name in ("e_s", "x", "m", "v"):
            if getattr(st, name) is not None:
                self._exact(name, gpu[name], getattr(st, name), keep)
        if srv_in is not None and gpu_u is not None:
            self._exact("u", gpu_u, srv_in, keep)
        if not self.tied:       # all exact: record the (zero) errors
            for name in ("e_w", "e_s", "x", "m", "v", "m_w", "v_w"):
                if getattr(st, name) is not None:
                    close(name, gpu[name], getattr(st, name), self.stats)


class Pair:
    """The oracle and the HIP path stepping the same configuration."""

    def __init__(self, d, N, qw, qs, placement=O.ADAM_AT_SERVER, seed=1, x1=None, split=False, sched=None,
                 mode=None, max_tie_rounds=0, **hp):
        """mode: "step" (ea_step), "split" (the four calls), "scheduled"
        (ea_step_scheduled, step index on the device), "run" (ea_run, one
        step per call) or "graph" (ea_step_scheduled captured once in a HIP
        graph and replayed); the last three take lr, beta2 from `sched`.
        max_tie_rounds: rounds with a validated one-ulp scale tie the test
        accepts (0: every round must be bit-exact)."""
        import torch
        import paper_2205_14473_amd as E
        from paper_2205_14473_amd.state import allocate, init_state
        self.torch, self.E = torch, E
        self.oc, self.ec = configs(d, N, qw, qs, placement, seed, **hp)
        self.mode = mode or ("split" if split else "step")
        self.sched = sched
        self.max_tie_rounds = max_tie_rounds
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
        self.nsw, self.nss = E.ea_msg_scales(self.ec.qw, d), E.ea_msg_scales(self.ec.qs, d)
        torch.cuda.synchronize()

    def oracle_config(self, t):
        if self.sched is None:
            return self.oc
        c = O.Config.from_buffer_copy(self.oc)
        c.lr, c.beta2 = (float(v) for v in O.schedule_at(self.so, self.oc.lr, self.oc.beta2, t))
        return c

    def gpu_step(self, t):
        rb, c, E, torch = self.rb, self.ec, self.E, self.torch
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
        torch = self.torch
        g = np.ascontiguousarray(g, np.float32)
        out = O.step(self.oracle_config(t), t, g, self.ost, want_srv_in=self.split, want_inputs=True)
        self.rb.g.copy_(torch.from_numpy(g))
        self.gpu_step(t)
        torch.cuda.synchronize()
        if self.mode in ("scheduled", "graph"):
            assert int(self.t_dev.item()) == t + 1, "the round did not advance its step counter"
        self.compare(t, out)
        self.stats.steps += 1
        return out

    def compare(self, t, out):
        rb, st, s = self.rb, self.ost, self.stats
        chk = RoundCheck(self.oracle_config(t), self.d, 0, t, out, s, what=f"step {t}: ")
        chk.messages(rb.wcodes.cpu().numpy(), rb.wscales.cpu().numpy()[:, :self.nsw], rb.scodes.cpu().numpy(),
                     rb.sscales.cpu().numpy()[:self.nss])
        host = lambda a: None if a is None else a.cpu().numpy()  # noqa: E731
        gpu = {k: host(getattr(rb, k)) for k in ("e_w", "e_s", "x", "m", "v", "m_w", "v_w")}
        chk.state(gpu, st, out.get("srv_in") if self.split else None, host(rb.u) if self.split else None)
        if chk.tied:
            s.tie_rounds += 1
            assert s.tie_rounds <= self.max_tie_rounds, (
                f"step {t}: a validated one-ulp scale tie ({s.scale_ties} buckets so far); this test allows "
                f"{self.max_tie_rounds} such rounds")
            self.resync()

    def resync(self):
        rb, st, torch = self.rb, self.ost, self.torch
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
        assert s.resyncs == s.tie_rounds, f"{s.resyncs} resets for {s.tie_rounds} rounds with a validated tie"
        assert s.tie_rounds <= self.max_tie_rounds
        assert s.code_ties <= 1e-6 * s.code_entries, (
            f"{s.code_ties} tie flips over {s.code_entries} entries exceed 1e-6")
