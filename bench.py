#!/usr/bin/env python3
"""Benchmark: Efficient-Adam rounds per second on one MI355X.

One "step" is one full round (ea_step): N worker compressions, the server's
dequantize-average + Adam, the server compression and the update of x, on the
BERT-base-sized workload (d = 110,000,000, N = 16, stochastic 4-bit with L2
bucket scale, bucket 512, two-way error feedback) unless --workload says
otherwise.  Inputs are synthetic (workloads.py) and already in HBM when the
timed region starts; the N gradient buffers are generated once and reused.

Prints ONE JSON line.  `roofline` covers step_kernel, the only kernel of a
bucketed round (one launch over the tiles that lie wholly inside d, plus a
one-block launch for the ragged last tile when d is not a multiple of the
tile): achieved = algorithmic HBM bytes per round / mean round time from HIP
events on the launch stream, i.e. over both launches.
`cpu_baseline` times the oracle (single-threaded C) on a bounded sample.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402

PEAK_HBM_GBS = 8000.0
METRIC = "Efficient-Adam step throughput (Gparam/s, N workers) + % of HBM peak GB/s"
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2205_14473_amd", "csrc", f)
                  for f in ("ea_round.hpp", "ea_kernels.hip", "ea_half_c1.hip", "ea_half_c2.hip", "ea_half_c4.hip",
                            "ea_half_c8.hip", "ea_sym_c4.hip", "ea_sym_c8.hip", "ea_device.hpp", "ea_launch.hpp",
                            "ea_api.cpp")]


def source_digest() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def algorithmic_bytes(E, cfg) -> int:
    """Minimum HBM bytes of one fused round: every vector crosses HBM once
    in each direction it must, messages are written once."""
    d, N = cfg.d, cfg.N
    ww, sw = E.ea_msg_words(cfg.qw, d), E.ea_msg_words(cfg.qs, d)
    nw, ns = E.ea_msg_scales(cfg.qw, d), E.ea_msg_scales(cfg.qs, d)
    if cfg.placement == E.EA_ADAM_AT_SERVER:
        worker = 12 * d          # read g, read e_w, write e_w
        server = 32 * d          # m, v, e_s, x: read + write
    else:
        worker = 28 * d          # g; e_w, m_w, v_w read + write
        server = 16 * d          # e_s, x: read + write
    return N * (worker + 8 * ww + 4 * nw) + server + 8 * sw + 4 * ns


def split_bytes(E, cfg) -> int:
    """Minimum HBM bytes of the round made of the four split calls: the fused
    round's, plus what the calls hand over through HBM: the worker messages
    read back by ea_server_aggregate_adam, its output u written and read back
    by ea_server_compress, and the server message read back by
    ea_worker_apply."""
    d, N = cfg.d, cfg.N
    ww, sw = E.ea_msg_words(cfg.qw, d), E.ea_msg_words(cfg.qs, d)
    nw, ns = E.ea_msg_scales(cfg.qw, d), E.ea_msg_scales(cfg.qs, d)
    return algorithmic_bytes(E, cfg) + N * (8 * ww + 4 * nw) + 8 * d + 8 * sw + 4 * ns


def traffic_from_profile(workload: str, placement: str, call: str = "step"):
    """HBM bytes per round measured by rocprofv3 counters (FETCH_SIZE and
    WRITE_SIZE summed over the round's launches of the library's kernels,
    each scaled by what it reads for a plain copy of known size), if the
    committed counter summary was taken on the current kernel sources."""
    kind = "split_calls" if call == "split" else "step_kernel"
    path = os.path.join(ROOT, "profiles", f"{kind}_{workload}_{placement}_pmc.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as f:
        for line in f:
            if line.startswith("#") or ":" not in line:
                continue
            k, v = line.split(":", 1)
            rec[k.strip()] = v.strip()
    if rec.get("source_digest") != source_digest():
        return None
    return int(rec["hbm_bytes_per_round"])


def stream_reference(rb, stream, reps=5):
    """A plain in-place streaming op on the same buffers, timed the same way:
    torch's e_w += g over N*d floats (two reads and one write per element),
    the access mix closest to the round's.  Context for the roofline fraction;
    it leaves e_w changed, so it runs after the timed rounds."""
    import torch
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    rb.e_w.add_(rb.g)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(reps):
        rb.e_w.add_(rb.g)
    stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / reps
    nbytes = 12 * rb.g.numel()
    return {"op": "torch e_w.add_(g), in place", "bytes": nbytes, "ms": round(ms, 4),
            "GB/s": round(nbytes / (ms * 1e-3) / 1e9, 1)}


def host_cpu():
    """Model name of the host CPU and the logical CPUs this process may use."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return model, len(os.sched_getaffinity(0)), os.cpu_count()


def cpu_baseline(E, w, cfg, rb, sample):
    """The oracle, as it stands, on the first `sample` parameters (one round)."""
    import numpy as np
    import oracle as O
    n = min(sample, cfg.d)
    B = max(O.bucket_len(O.Quant(**w.qw.fields()), cfg.d), O.bucket_len(O.Quant(**w.qs.fields()), cfg.d))
    if B < cfg.d:
        n = max(B, n // B * B)
    else:
        n = cfg.d
    oc = O.Config(d=cfg.d, N=cfg.N, placement=cfg.placement, beta1=cfg.beta1, beta2=cfg.beta2, lr=cfg.lr,
                  eps=cfg.eps, seed=cfg.seed, qw=O.Quant(**w.qw.fields()), qs=O.Quant(**w.qs.fields()))
    g = np.ascontiguousarray(rb.g[:, :n].cpu().numpy())
    st = O.State.init(oc, n, rb.x[:n].cpu().numpy())
    t0 = time.perf_counter()
    O.step(oc, 1, g, st, n0=0)
    dt = time.perf_counter() - t0
    model, usable, total = host_cpu()
    return {"value": round(n / dt / 1e9, 6), "unit": "Gparam/s", "cores": 1, "kind": "oracle",
            "sample": f"one round over the first {n} of {cfg.d} parameters, N={cfg.N}, single thread, "
                      f"{dt:.2f} s",
            "host_cpu": model, "nproc": usable, "cpu_count": total}


def paper_toy(args, E, allocate, init_state):
    """Section V-A on the device: per step, the N workers' gradients
    2 A^T (A x - x* - xi_i) at the current x and one round (Example 2 with
    k = -17, K = -11, Adam at the workers, beta = 0.9, theta = 0.99,
    lr = 1e-4), plus ||grad F||^2 at x.  By default one ea_toy_step call (the
    gradient producer fused into the round: two launches, the gradients never
    leave the chip); --call split times ea_toy_grad followed by ea_step.  The
    noise draws of all steps are generated before the timed region.  The
    problem lives in cache and is bound by the latency of its dependent
    memory trips, so the roofline fraction is reported for completeness."""
    import torch
    toy = W.PAPER_TOY
    d, N = toy["d"], toy["N"]
    q = E.Quant(kind=E.EA_Q_POW2, pow2_kmin=-17, pow2_kmax=-11, error_feedback=1)
    cfg = E.Config(d=d, N=N, placement=E.EA_ADAM_AT_WORKER, beta1=toy["beta1"], beta2=toy["beta2"], lr=1e-4,
                   eps=1e-8, seed=7, qw=q, qs=q)
    rb = allocate(cfg)
    init_state(cfg, rb)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(7)
    A = torch.randn((d, d), generator=gen, device="cuda")
    xs = torch.randn(d, generator=gen, device="cuda") * toy["x_star_var"] ** 0.5
    total = args.warmup + args.steps
    xi = torch.randn((total, N, d), generator=gen, device="cuda") * toy["xi_var"] ** 0.5
    gsq = torch.zeros(total, dtype=torch.float64, device="cuda")
    ws = torch.empty(E.ea_toy_workspace_bytes(d), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    step_args = rb.step_args()
    fused = args.call != "split"

    def one(k, s):
        if fused:
            E.ea_toy_step(cfg, k + 1, A, xs, xi[k], rb.e_w, rb.m_w, rb.v_w, rb.m, rb.v, rb.e_s, rb.x, rb.wcodes,
                          rb.scodes, gsq[k:k + 1], None, ws, stream=s)
        else:
            E.ea_toy_grad(d, N, A, xs, xi[k], rb.x, rb.g, gsq[k:k + 1], ws, stream=s)
            E.ea_step(cfg, k + 1, **step_args, stream=s)

    for k in range(args.warmup):
        one(k, stream)
    torch.cuda.synchronize()
    # A step is about 20 us of GPU work, close to what the host takes to
    # issue it from Python, so by default the timed steps are captured into
    # one HIP graph (capture records the launches without running them) and
    # replayed: the time is then the GPU's alone.
    graph = None
    if not args.eager:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            cs = torch.cuda.current_stream()
            for k in range(args.warmup, total):
                one(k, cs)
        torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    if graph is not None:
        graph.replay()
    else:
        for k in range(args.warmup, total):
            one(k, stream)
    stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    alg = algorithmic_bytes(E, cfg) + 4 * d * d      # the round + A read once by the gradient producer
    if not fused:
        alg += 4 * d * d + 2 * 4 * N * d             # A read again, g written and read back
    g = gsq.cpu().numpy()
    line = {
        "metric": "Section V-A toy problem, steps per second (gradient producer + round)",
        "value": round(1e3 / ms, 1), "unit": "steps/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": "paper_toy d=500 N=10 Example 2, Adam at the workers", "d": d, "N": N,
                   "call": "ea_toy_step" if fused else "ea_toy_grad + ea_step",
                   "launch": "eager" if args.eager else f"one HIP graph of the {args.steps} timed steps"},
        "roofline": {"bound": "hbm", "achieved": round(alg / (ms * 1e-3) / 1e9, 1), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(alg / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 5), "traffic": None,
                     "kernel": ("toy residual + toy_round_kernel" if fused
                                else "toy residual + toy_round_kernel (gradients only) + step_kernel")
                     + " (cache-resident; bound by dependent memory latency)"},
        "grad_sq_first_last": [float(g[0]), float(g[-1])],
    }
    print(json.dumps(line), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="bert", choices=list(W.WORKLOADS) + ["paper_toy"],
                    help="paper_toy: Section V-A's problem (d = 500, N = 10, Example 2, Adam at the "
                         "workers), each step = ea_toy_grad at the current x + one round")
    ap.add_argument("--call", default="step", choices=["step", "scheduled", "graph", "split"],
                    help="time ea_step (default), ea_step_scheduled with the step on the device and a "
                         "Section V-B step-decay schedule, that call captured once in a HIP graph and "
                         "replayed, or the four split calls (ea_worker_compress for each worker, "
                         "ea_server_aggregate_adam, ea_server_compress, ea_worker_apply)")
    ap.add_argument("--placement", default="server", choices=["server", "worker"])
    ap.add_argument("--eager", action="store_true",
                    help="paper_toy: issue every timed step from the host instead of replaying them "
                         "from one HIP graph")
    ap.add_argument("--cpu-sample", type=int, default=1 << 24, help="parameters in the oracle's timed sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calib-gib", type=float, default=0.0,
                    help="only run a plain torch copy of this many GiB (HBM counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)

    if args.copy_calib_gib > 0:
        n = int(args.copy_calib_gib * (1 << 30)) // 4
        a = torch.ones(n, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n * 4, "bytes_written": n * 4}), flush=True)
        return

    import paper_2205_14473_amd as E
    from paper_2205_14473_amd.state import allocate, init_state

    if args.workload == "paper_toy":
        return paper_toy(args, E, allocate, init_state)

    w = W.WORKLOADS[args.workload]
    placement = E.EA_ADAM_AT_SERVER if args.placement == "server" else E.EA_ADAM_AT_WORKER
    cfg = E.Config(**w.config_fields(placement=placement), qw=E.Quant(**w.qw.fields()), qs=E.Quant(**w.qs.fields()))
    rb = allocate(cfg, with_u=args.call == "split")
    init_state(cfg, rb)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(w.seed)
    torch.randn(cfg.d, generator=gen, device="cuda", out=rb.x)
    rb.x.mul_(0.02)
    W.device_gradients(w, 1, rb.g)
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    sched = E.Schedule(kind=E.EA_SCHED_STEP_DECAY, alpha=cfg.lr, factor=0.2, period=19550)
    t_dev = torch.ones(1, dtype=torch.int32, device="cuda")
    graph = None
    if args.call == "graph":
        E.ea_step_scheduled(cfg, sched, t_dev, **rb.step_args(), stream=stream)   # per-device setup, step 1
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            E.ea_step_scheduled(cfg, sched, t_dev, **rb.step_args())
        stream = torch.cuda.current_stream()
    t = 1

    nsw, nss = E.ea_msg_scales(cfg.qw, cfg.d), E.ea_msg_scales(cfg.qs, cfg.d)

    def one_round():
        nonlocal t
        if args.call == "step":
            E.ea_step(cfg, t, **rb.step_args(), stream=stream)
        elif args.call == "split":
            for i in range(cfg.N):
                E.ea_worker_compress(cfg, i, t, rb.g[i], rb.e_w[i], None if rb.m_w is None else rb.m_w[i],
                                     None if rb.v_w is None else rb.v_w[i], rb.wcodes[i],
                                     rb.wscales[i] if nsw else None, rb.workspace, stream=stream)
            E.ea_server_aggregate_adam(cfg, t, rb.wcodes, rb.wscales if nsw else None, rb.m, rb.v, rb.u,
                                       stream=stream)
            E.ea_server_compress(cfg, t, rb.u, rb.e_s, rb.scodes, rb.sscales if nss else None, rb.workspace,
                                 stream=stream)
            E.ea_worker_apply(cfg, rb.scodes, rb.sscales if nss else None, rb.x, stream=stream)
        elif args.call == "scheduled":
            E.ea_step_scheduled(cfg, sched, t_dev, **rb.step_args(), stream=stream)
        else:
            graph.replay()
        t += 1

    for _ in range(args.warmup):
        one_round()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(args.steps):
        one_round()
    stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps

    alg = split_bytes(E, cfg) if args.call == "split" else algorithmic_bytes(E, cfg)
    achieved = alg / (ms * 1e-3) / 1e9
    value = cfg.d / (ms * 1e-3) / 1e9
    roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4),
            "traffic": (traffic_from_profile(args.workload, args.placement, args.call)
                        if args.call in ("step", "split") else None),
            "kernel": ("worker_kernel x N, aggregate_kernel, server_kernel, apply_kernel" if args.call == "split"
                       else "step_kernel (whole tiles + ragged tail)"),
            "algorithmic_bytes_per_round": alg,
            "bytes_per_param": round(alg / cfg.d, 2)}
    line = {
        "metric": METRIC, "value": round(value, 4), "unit": "Gparam/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": w.name, "d": cfg.d, "N": cfg.N, "call": args.call,
                   "placement": "adam_at_server" if placement == 0 else "adam_at_worker",
                   "qw": w.qw.fields(), "qs": w.qs.fields()},
        "param_workers_per_s": round(cfg.N * value, 3),
        "hbm_frac": round(achieved / PEAK_HBM_GBS, 4),
        "roofline": roof,
    }
    line["stream_reference"] = stream_reference(rb, stream)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(E, w, cfg, rb, args.cpu_sample)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
