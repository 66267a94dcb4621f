"""Throughput of the fused speculative-sampling verification step on one GPU.

One step is one complete ``spec_verify_*`` call over one batch of synthetic
logits already resident in device memory.  Prints one JSON line with
verify-steps/s, the roofline position of the step (algorithmic HBM bytes per
step / measured step time, against MI355X's 8 TB/s), and the CPU oracle timed
on a bounded sample of the same workload.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--gpus 1]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "verify-steps/sec and achieved HBM GB/s (fraction of peak) at 1 MI355X"


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def algorithmic_bytes(w, accepted_len=None) -> int:
    """Bytes a step must move at least: exact mode reads every logit once
    (B (2 gamma + 1) V s); sigmoid mode reads the drafted-token logits and the
    row(s) the next token is drawn from -- one row for an element that
    accepts every draft, two otherwise (all elements counted as two when
    ``accepted_len`` is not given).  Plus tokens, uniforms and the two
    outputs."""
    from paper_2406_11016_amd.workloads import BYTES_PER_LOGIT
    s = BYTES_PER_LOGIT[w.dtype]
    small = w.batch * (w.gamma * 4 + (w.gamma + 1) * 4 + 2 * 4)
    if w.mode == "exact":
        return w.batch * (2 * w.gamma + 1) * w.vocab * s + small
    if accepted_len is None:
        rows = 2 * w.batch
    else:
        rows = sum(1 if int(L) == w.gamma else 2 for L in accepted_len)
    return w.batch * 2 * w.gamma * s + rows * w.vocab * s + small


KERNEL_SOURCES = ("spec_verify.hip", "sv_device.hpp", "plan.hpp")


def source_hash() -> str:
    """sha256 prefix of the kernel's sources (to match recorded counter data)."""
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2406_11016_amd", "csrc", name), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def recorded_traffic(workload: str):
    """HBM bytes per launch from the recorded rocprofv3 counter runs, or None
    if none were recorded for this workload or the kernel changed since."""
    path = os.path.join(ROOT, "profiles", "verify_kernel_traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != source_hash():
        return None
    w = rec.get("workloads", {}).get(workload)
    return None if w is None else int(w["traffic_bytes"])


_POOL_INPUTS = None


def _single_thread_blas() -> None:
    from threadpoolctl import threadpool_limits
    threadpool_limits(1)


def _oracle_on(x, lo: int, hi: int) -> int:
    import numpy as np

    import oracle
    with np.errstate(all="ignore"):
        oracle.verify(x.draft[lo:hi], x.target[lo:hi], x.tokens[lo:hi], x.uniforms[lo:hi], dtype=x.dtype,
                      mode=x.mode, temperature=x.temperature, alpha=x.alpha, beta=x.beta)
    return hi - lo


def _oracle_element(b: int) -> int:
    return _oracle_on(_POOL_INPUTS, b, b + 1)


def host_description() -> dict:
    import numpy as np
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpu_count": os.cpu_count(), "usable_cores": len(os.sched_getaffinity(0)), "cpu_model": model,
            "numpy": np.__version__}


def cpu_baseline(w, x, min_seconds: float, max_workers: int = 16):
    """The oracle as it stands, timed on the host: (i) one thread on a bounded
    sample of batch elements, scaled to whole steps; (ii) a process pool over
    the batch elements of whole steps, one worker per usable core (at most
    ``max_workers``), each worker single-threaded.

    Must run before the process touches the GPU: the pool forks."""
    import multiprocessing as mp

    from threadpoolctl import threadpool_limits
    global _POOL_INPUTS

    nb = min(w.batch, 16)
    with threadpool_limits(1):
        _oracle_on(x, 0, 1)
        reps, t0 = 0, time.perf_counter()
        while True:
            for b in range(nb):
                _oracle_on(x, b, b + 1)
            reps += 1
            el = time.perf_counter() - t0
            if el >= min_seconds:
                break
    single = {"value": reps * nb / w.batch / el, "unit": "verify-steps/s", "cores": 1, "kind": "oracle",
              "sample": f"float64 NumPy oracle on batch elements 0..{nb - 1} of {w.batch} "
                        f"one element per call ({reps} repetitions, {el:.1f} s, one thread), scaled to whole steps"}

    workers = max(1, min(len(os.sched_getaffinity(0)), max_workers, w.batch))
    _POOL_INPUTS = x
    try:
        with mp.get_context("fork").Pool(workers, initializer=_single_thread_blas) as pool:
            pool.map(_oracle_element, range(min(w.batch, workers)), chunksize=1)   # start-up, imports
            steps, t0 = 0, time.perf_counter()
            while True:
                pool.map(_oracle_element, range(w.batch), chunksize=1)
                steps += 1
                el = time.perf_counter() - t0
                if el >= min_seconds:
                    break
    finally:
        _POOL_INPUTS = None
    out = {"value": steps / el, "unit": "verify-steps/s", "cores": workers, "kind": "oracle",
           "sample": f"float64 NumPy oracle over all {w.batch} batch elements of {steps} whole steps "
                     f"({el:.1f} s), a process pool of {workers} single-threaded workers, one batch "
                     f"element per task"}
    out["single_thread"] = single
    out["host"] = host_description()
    return out


def latency_percentiles(step, calls: int, stream) -> dict:
    """Per-call device time of ``calls`` consecutive steps, each bracketed by
    its own pair of HIP events on the launch stream."""
    import torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(calls)]
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(evs):
        a.record(stream)
        step(i)
        b.record(stream)
    torch.cuda.synchronize()
    us = sorted(a.elapsed_time(b) * 1000.0 for a, b in evs)

    def pct(q):
        return round(us[min(len(us) - 1, int(q * len(us)))], 2)

    return {"p50_us": pct(0.50), "p99_us": pct(0.99), "min_us": round(us[0], 2), "max_us": round(us[-1], 2),
            "calls": calls}


def graph_timing(step, nrot: int, steps: int, warmup: int, dev) -> dict:
    """The same steps captured into one HIP graph (one captured call per input
    copy, replayed until ``steps`` calls have run), timed with HIP events."""
    import torch
    per = max(nrot, 32)
    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        for i in range(per):        # eager warm-up on the capture stream
            step(i)
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize(dev)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        for i in range(per):
            step(i)
    torch.cuda.synchronize(dev)
    reps = max(1, steps // per)
    for _ in range(max(1, warmup // per)):
        g.replay()
    stream = torch.cuda.current_stream(dev)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize(dev)
    ev0.record(stream)
    for _ in range(reps):
        g.replay()
    ev1.record(stream)
    torch.cuda.synchronize(dev)
    ms = ev0.elapsed_time(ev1) / (reps * per)
    return {"value": round(1000.0 / ms, 1), "unit": "verify-steps/s", "ms_per_step": round(ms, 6),
            "steps": reps * per, "what": f"{per} calls captured into one HIP graph, replayed {reps} times"}


def unfused_baseline(w, sets, tok, uni, steps: int, warmup: int):
    """The same step with stock PyTorch operators (one eager kernel per
    operator, fp32 probabilities), timed with HIP events on the current stream
    over the same rotating inputs."""
    import torch

    from paper_2406_11016_amd import unfused_torch
    nrot = len(sets)

    def step(i):
        d, t = sets[i % nrot]
        return unfused_torch.verify(d, t, tok, uni, mode=w.mode, temperature=w.temperature, alpha=w.alpha,
                                    beta=w.beta)

    for i in range(warmup):
        step(i)
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for i in range(steps):
        step(i)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    return {"value": round(1000.0 / ms, 1), "unit": "verify-steps/s", "ms_per_step": round(ms, 6),
            "steps": steps, "what": "stock PyTorch operators on the same GPU and inputs: softmax/sigmoid, gather, "
                                    "eq. (1), cumprod scan, residual, cumsum + searchsorted (fp32)"}


def divergence_from_exact(w, dev, input_sets: int = 4) -> dict:
    """How far the sigmoid approximation's decisions are from the exact mode's
    on the same inputs (Sec. 3.2.2; the workload's own comparison): both modes
    run through the GPU path with their probe outputs on ``input_sets`` seeded
    input sets of the workload's shape.  Acceptance rate = mean accepted
    length / gamma; TV = half the L1 distance between the two modes' final
    distributions (the weights divided by their mass) of each element; token
    disagreement = fraction of elements whose next tokens differ."""
    import numpy as np
    import torch

    from paper_2406_11016_amd import binding
    from paper_2406_11016_amd import workloads as W
    acc_s, acc_e, tv, dis = [], [], [], []
    for k in range(input_sets):
        x = W.generate(w, seed=w.seed * 100 + k)
        d, t, tok, u = binding.to_device(x, dev)
        res = {}
        for mode in ("sigmoid", "exact"):
            a, n, pr = binding.verify(d, t, tok, u, mode=mode, temperature=w.temperature, alpha=w.alpha,
                                      beta=w.beta, probe=True)
            res[mode] = (a, n, pr.weights.double() / pr.mass[:, None])
        (a_s, n_s, f_s), (a_e, n_e, f_e) = res["sigmoid"], res["exact"]
        ok = (a_s >= 0) & (a_e >= 0)
        acc_s.append(a_s[ok].double().cpu().numpy() / w.gamma)
        acc_e.append(a_e[ok].double().cpu().numpy() / w.gamma)
        tv.append((0.5 * (f_s[ok] - f_e[ok]).abs().sum(-1)).cpu().numpy())
        dis.append((n_s[ok] != n_e[ok]).double().cpu().numpy())
    torch.cuda.synchronize()
    acc_s, acc_e, tv, dis = (np.concatenate(v) for v in (acc_s, acc_e, tv, dis))
    return {"elements": int(acc_s.size), "accept_rate_sigmoid": round(float(acc_s.mean()), 4),
            "accept_rate_exact": round(float(acc_e.mean()), 4),
            "accept_rate_delta": round(float(acc_s.mean() - acc_e.mean()), 4),
            "mean_tv_final": round(float(tv.mean()), 4), "token_disagreement": round(float(dis.mean()), 4),
            "what": f"GPU path, both modes with probes on {input_sets} seeded input sets of this shape; "
                    "acceptance = mean accepted length / gamma, TV between the two modes' final distributions"}


def copy_calibration(nbytes: int, reps: int) -> None:
    """A plain device-to-device copy of known size, for scaling HBM counters."""
    import torch
    a = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    b = torch.empty_like(a)
    for _ in range(reps):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "reps": reps}), flush=True)


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--rotate-mb", type=float, default=768.0,
                    help="device copies of the inputs are rotated so that at least this many MB are cycled "
                         "(defeats the 256 MB last-level cache)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-unfused", action="store_true", help="skip timing the unfused PyTorch comparison")
    ap.add_argument("--graph", choices=("auto", "on", "off"), default="auto",
                    help="also time the calls replayed from a HIP graph (auto: for workloads under 8 MB)")
    ap.add_argument("--sweep", choices=("gamma", "alpha_beta", "top_k", "ragged", "early_exit", "decode_loop",
                                        "loop_early_exit"),
                    default=None,
                    help="instead of the benchmark line: one JSON line with a sweep over gamma (1..20), over "
                         "the sigmoid constants alpha = -beta, over a top-k mask of the logits, over ragged "
                         "per-element gamma, the exact mode's early exit against its single pass, or the decoding "
                         "loop with the gamma rule (--steps iterations), or that loop at the headline shape choosing "
                         "the early exit per step (--steps iterations)")
    ap.add_argument("--noise", type=float, default=None,
                    help="normal logits (scale 2) with this draft-target noise instead of the workload's own law "
                         "(e.g. 2.0: most elements reject an early draft, so the residual path runs for nearly "
                         "every element)")
    ap.add_argument("--copy-calibration-mb", type=float, default=0.0,
                    help="only run a plain copy of this size (for counter calibration) and exit")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(batch elements are independent, so N GPUs would each run this step on B/N)", file=sys.stderr)
        return 2
    if args.copy_calibration_mb > 0:
        copy_calibration(int(args.copy_calibration_mb * 1e6), 20)
        return 0
    if args.sweep is not None:
        import bench_sweeps
        return bench_sweeps.run(args.sweep, args.steps, args.warmup)

    from paper_2406_11016_amd import workloads as W

    w = W.WORKLOADS[args.workload or W.HEADLINE]
    if args.noise is not None:
        w = w.with_(name=f"{w.name}_normal_noise{args.noise:g}", base="normal", base_scale=2.0,
                    noise_scale=args.noise)
    log(f"generating {w.name} ({w.logit_bytes / 1e6:.1f} MB of logits)")
    t0 = time.perf_counter()
    x = W.generate(w)
    log(f"generated in {time.perf_counter() - t0:.1f} s")

    # the CPU leg runs first: its process pool forks, which must happen
    # before this process initialises the GPU
    cpu = None
    if not args.no_cpu_baseline:
        log(f"timing the CPU oracle: one thread, then a process pool, ~{args.cpu_seconds:.0f} s each")
        cpu = cpu_baseline(w, x, args.cpu_seconds)
        log(f"CPU oracle: {cpu['single_thread']['value']:.4f} steps/s on one thread, "
            f"{cpu['value']:.4f} steps/s on {cpu['cores']} processes")

    import torch

    from paper_2406_11016_amd import binding

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        return 1
    dev = torch.device("cuda:0")
    binding.load_library()
    log("uploading")
    d0, t0_, tok, uni = binding.to_device(x, dev)
    nrot = max(1, int((args.rotate_mb * 1e6 + w.logit_bytes - 1) // w.logit_bytes))
    sets = [(d0, t0_)] + [(d0.clone(), t0_.clone()) for _ in range(nrot - 1)]
    acc = torch.empty(w.batch, dtype=torch.int32, device=dev)
    nxt = torch.empty(w.batch, dtype=torch.int32, device=dev)
    ws = binding.new_workspace(w.batch, w.gamma, w.vocab, d0.dtype, dev)
    torch.cuda.synchronize(dev)

    def step(i):
        d, t = sets[i % nrot]
        binding.verify(d, t, tok, uni, mode=w.mode, temperature=w.temperature, alpha=w.alpha, beta=w.beta,
                       accepted_len=acc, next_token=nxt, workspace=ws)

    log(f"warmup {args.warmup} steps over {nrot} rotating input copies")
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize(dev)

    stream = torch.cuda.current_stream(dev)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    log(f"timing {args.steps} steps")
    torch.cuda.synchronize(dev)
    wall0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        step(i)
    ev1.record(stream)
    torch.cuda.synchronize(dev)
    wall = time.perf_counter() - wall0
    ms = ev0.elapsed_time(ev1)
    ms_per_step = ms / args.steps
    steps_per_s = 1000.0 / ms_per_step
    log(f"{ms_per_step * 1000:.2f} us/step (events), wall {wall:.3f} s")

    ncalls = min(max(args.steps, 50), 1000)
    log(f"per-call latency over {ncalls} calls")
    latency = latency_percentiles(step, ncalls, stream)

    graph = None
    if args.graph == "on" or (args.graph == "auto" and w.logit_bytes < 8e6):
        log("timing the same calls replayed from a HIP graph")
        graph = graph_timing(step, nrot, args.steps, args.warmup, dev)

    # the decisions of the timed steps are real: check one against the oracle
    # later in the tests; here just make sure they are in range
    a, n = acc.cpu(), nxt.cpu()
    if bool(((a < 0) | (a > w.gamma)).any()) or bool(((n < 0) | (n >= w.vocab)).any()):
        log("warning: sentinel outputs in the timed workload")

    alg = algorithmic_bytes(w, a.numpy())
    achieved = alg / (ms_per_step * 1e-3) / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": recorded_traffic(w.name),
                "kernel": "verify_kernel<exact> (the whole step is one launch)" if w.mode == "exact"
                else "verify_kernel<sigmoid> (the whole step is one launch)", "algorithmic_bytes_per_step": alg}

    divergence = None
    if w.mode == "sigmoid":
        log("divergence from the exact mode on the same inputs")
        divergence = divergence_from_exact(w, dev)

    unfused = None
    if not args.no_unfused:
        log("timing the unfused PyTorch comparison")
        unfused = unfused_baseline(w, sets, tok, uni, steps=max(20, min(200, args.steps // 10)), warmup=5)
        unfused["speedup_of_fused"] = round(steps_per_s / unfused["value"], 2)

    out = {
        "metric": METRIC, "value": round(steps_per_s, 1), "unit": "verify-steps/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "mode": w.mode, "batch": w.batch, "gamma": w.gamma, "vocab": w.vocab,
                   "logits": w.dtype, "temperature": w.temperature, "rotating_copies": nrot},
        "roofline": roofline,
        "latency": latency,
        "graph": graph,
        "cpu_baseline": cpu,
        "unfused_torch": unfused,
    }
    if divergence is not None:
        out["divergence_from_exact"] = divergence
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
