"""Parameter sweeps of the fused verification step on one GPU (``bench.py --sweep``).

* ``gamma``: the number of drafted tokens, 1 .. 20 (the paper sweeps gamma in
  Sec. 4.3 and Fig. 3), on B = 1 workloads shaped like the paper's ASR
  (V = 51,865, fp32 logits) and summarisation (V = 32,000, fp16 logits) runs,
  and on the batched bf16 workload (B = 64, V = 128,256) at a few gamma.  Per
  point: time per step, verify-steps/s, the fraction of 8 TB/s on the
  algorithmic bytes, and, from a batch of 32 independent elements of the same
  value law, the acceptance rate (mean accepted length / gamma), the chance
  that every draft is accepted and the tokens emitted per step (L + 1).
* ``alpha_beta``: the sigmoid approximation's constants alpha = -beta in
  {10, 1e3, 1e4, 1e5} (Sec. 3.2, eq. (5); Tables 2, 7, 8) on the fp16 sigmoid
  workload (B = 32, gamma = 10, V = 50,272, T = 0.7).  The exact mode runs on
  the same inputs and uniforms.  Per point: time per step; acceptance rate of
  both modes and its change; token disagreement rate; mean total-variation
  distance between the two final-token distributions where both modes select
  the same row; and the number of sentinel or non-finite outputs (fp16
  logits scaled by 1/(beta - alpha) stay finite in the fp32 arithmetic).

Every statistic comes from the GPU path's own outputs (its probe buffers for
the distributions).  Inputs are the seeded synthetic workloads.
"""
from __future__ import annotations

import json
import sys
import time

HBM_PEAK_GBPS = 8000.0


def log(msg: str) -> None:
    print(f"[sweep] {msg}", file=sys.stderr, flush=True)


def _time_steps(w, x, steps: int, warmup: int, rotate_mb: float = 768.0, gammas=None,
                early_exit: bool = False) -> float:
    """Microseconds per call, HIP events on the launch stream, rotating input copies."""
    import torch

    from paper_2406_11016_amd import binding
    dev = torch.device("cuda:0")
    d0, t0, tok, uni = binding.to_device(x, dev)
    nrot = max(1, int((rotate_mb * 1e6 + w.logit_bytes - 1) // w.logit_bytes))
    sets = [(d0, t0)] + [(d0.clone(), t0.clone()) for _ in range(nrot - 1)]
    acc = torch.empty(w.batch, dtype=torch.int32, device=dev)
    nxt = torch.empty(w.batch, dtype=torch.int32, device=dev)
    ws = binding.new_workspace(w.batch, w.gamma, w.vocab, d0.dtype, dev)
    gd = None if gammas is None else torch.as_tensor(gammas, dtype=torch.int32).to(dev)

    def step(i):
        d, t = sets[i % nrot]
        binding.verify(d, t, tok, uni, mode=w.mode, temperature=w.temperature, alpha=w.alpha, beta=w.beta,
                       accepted_len=acc, next_token=nxt, workspace=ws, gammas=gd, early_exit=early_exit)

    for i in range(warmup):
        step(i)
    stream = torch.cuda.current_stream(dev)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize(dev)
    ev0.record(stream)
    for i in range(steps):
        step(i)
    ev1.record(stream)
    torch.cuda.synchronize(dev)
    us = ev0.elapsed_time(ev1) / steps * 1000.0
    del sets, d0, t0, ws
    torch.cuda.empty_cache()
    return us


def _acceptance(w, batch: int, seed: int):
    """Accepted lengths of `batch` independent elements of the workload's law."""
    import torch

    from paper_2406_11016_amd import binding
    from paper_2406_11016_amd import workloads as W
    x = W.generate(w.with_(batch=batch), seed=seed)
    d, t, tok, uni = binding.to_device(x, "cuda")
    acc, nxt = binding.verify(d, t, tok, uni, mode=w.mode, temperature=w.temperature, alpha=w.alpha,
                              beta=w.beta)
    torch.cuda.synchronize()
    return acc.cpu().numpy(), nxt.cpu().numpy()


def sweep_gamma(steps: int, warmup: int) -> dict:
    import numpy as np

    from bench import algorithmic_bytes
    from paper_2406_11016_amd import workloads as W
    plan = [("exact_b1_g5_v51865_f32", list(range(1, 21))),
            ("exact_b1_g10_v32000_f16", list(range(1, 21))),
            ("exact_b64_g8_v128256_bf16", [1, 2, 4, 8, 12, 16, 20])]
    points = []
    for base, gammas in plan:
        for g in gammas:
            w = W.WORKLOADS[base].with_(gamma=g)
            x = W.generate(w)
            n = steps if w.batch == 1 else max(50, steps // 5)
            us = _time_steps(w, x, n, warmup)
            del x
            L, _ = _acceptance(w, 32 if w.batch == 1 else 16, seed=w.seed * 1000 + g)
            valid = L >= 0
            Lv = L[valid].astype(np.float64)
            alg = algorithmic_bytes(w)
            p = {"workload": base, "gamma": g, "batch": w.batch, "vocab": w.vocab, "logits": w.dtype,
                 "us_per_step": round(us, 3), "steps_per_s": round(1e6 / us, 1),
                 "frac_of_8TBs": round(alg / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                 "accept_rate": round(float(Lv.mean() / g), 4),
                 "p_all_accepted": round(float((Lv == g).mean()), 4),
                 "tokens_per_step": round(float(Lv.mean() + 1.0), 3),
                 "us_per_token_per_element": round(us / float(Lv.mean() + 1.0) / w.batch, 3),
                 "sentinels": int((~valid).sum()), "acceptance_sample": int(L.size)}
            log(json.dumps(p))
            points.append(p)
    return {"sweep": "gamma", "points": points}


def sweep_alpha_beta(steps: int, warmup: int) -> dict:
    import numpy as np
    import torch

    from paper_2406_11016_amd import binding
    from paper_2406_11016_amd import workloads as W
    base = W.WORKLOADS["sigmoid_b32_g10_v50272_f16_t0.7"]
    sets = [W.generate(base, seed=base.seed * 100 + k) for k in range(4)]
    points = []

    def run(x, mode, a, b):
        d, t, tok, uni = binding.to_device(x, "cuda")
        acc, nxt, pr = binding.verify(d, t, tok, uni, mode=mode, temperature=x.temperature, alpha=a, beta=b,
                                      probe=True)
        torch.cuda.synchronize()
        return acc.cpu().numpy(), nxt.cpu().numpy(), pr.weights, pr.mass

    exact = [run(x, "exact", -1.0, 1.0) for x in sets]
    for ab in (10.0, 1e3, 1e4, 1e5):
        w = base.with_(alpha=-ab, beta=ab)
        us = _time_steps(w, sets[0], steps, warmup)
        Ls, Le, dis, tvs, bad = [], [], [], [], 0
        for x, (le, ne, we, me) in zip(sets, exact):
            ls, ns, wsg, ms = run(x, "sigmoid", -ab, ab)
            bad += int((ls < 0).sum() + (ns < 0).sum())
            bad += int((~torch.isfinite(ms)).sum().item())
            Ls.append(ls)
            Le.append(le)
            dis.append((ls != le) | (ns != ne))
            same = torch.from_numpy((ls == le) & (ls >= 0)).to(wsg.device)
            if bool(same.any()):
                ps = wsg[same].double() / ms[same][:, None]
                pe = we[same].double() / me[same][:, None]
                tvs.append((0.5 * (ps - pe).abs().sum(dim=1)).cpu().numpy())
        Ls, Le = np.concatenate(Ls), np.concatenate(Le)
        g = base.gamma
        p = {"alpha": -ab, "beta": ab, "us_per_step": round(us, 3), "steps_per_s": round(1e6 / us, 1),
             "accept_rate_sigmoid": round(float(Ls[Ls >= 0].mean() / g), 5),
             "accept_rate_exact": round(float(Le[Le >= 0].mean() / g), 5),
             "token_disagreement": round(float(np.concatenate(dis).mean()), 4),
             "mean_tv_same_row": round(float(np.concatenate(tvs).mean()), 4) if tvs else None,
             "sentinel_or_nonfinite": bad, "elements": int(Ls.size)}
        p["accept_delta"] = round(p["accept_rate_sigmoid"] - p["accept_rate_exact"], 5)
        log(json.dumps(p))
        points.append(p)
    return {"sweep": "alpha_beta", "workload": base.name, "points": points}


def sweep_top_k(steps: int, warmup: int) -> dict:
    """Exact and sigmoid acceptance when both models' logits pass a top-k
    processor (the rest -inf), on the fp16 sigmoid workload's shape, T = 0.7,
    alpha = -beta = 1e4; time per step of both modes."""
    import numpy as np
    import torch

    from paper_2406_11016_amd import binding
    from paper_2406_11016_amd import workloads as W
    base = W.WORKLOADS["sigmoid_b32_g10_v50272_f16_t0.7"]
    points = []
    for k in (1, 2, 5, 10, 20, 50, 200, 1000, 0):
        w = base.with_(top_k=k)
        x = W.generate(w, seed=base.seed * 10 + 1)
        d, t, tok, uni = binding.to_device(x, "cuda")
        out = {}
        for mode in ("exact", "sigmoid"):
            acc, nxt = binding.verify(d, t, tok, uni, mode=mode, temperature=w.temperature, alpha=w.alpha,
                                      beta=w.beta)
            torch.cuda.synchronize()
            out[mode] = (acc.cpu().numpy(), nxt.cpu().numpy())
        us = {m: _time_steps(w.with_(mode=m), x, steps, warmup) for m in ("exact", "sigmoid")}
        le, ls = out["exact"][0], out["sigmoid"][0]
        g = w.gamma
        p = {"top_k": k if k else w.vocab, "accept_rate_exact": round(float(le[le >= 0].mean() / g), 4),
             "accept_rate_sigmoid": round(float(ls[ls >= 0].mean() / g), 4),
             "token_disagreement": round(float(((le != ls) | (out["exact"][1] != out["sigmoid"][1])).mean()), 4),
             "us_per_step_exact": round(us["exact"], 3), "us_per_step_sigmoid": round(us["sigmoid"], 3),
             "sentinels": int((le < 0).sum() + (ls < 0).sum()), "elements": int(le.size)}
        log(json.dumps(p))
        points.append(p)
    return {"sweep": "top_k", "workload": base.name, "alpha": base.alpha, "beta": base.beta, "points": points}


def sweep_ragged(steps: int, warmup: int) -> dict:
    """The ragged variant on the batched bf16 workload (B = 64, gamma_max = 8,
    V = 128,256): time per step and the fraction of 8 TB/s on the bytes the
    elements' own rows hold, sum_b (2 gammas[b] + 1) V s, for several
    distributions of gammas[b]."""
    import numpy as np

    from paper_2406_11016_amd import workloads as W
    w = W.WORKLOADS["exact_b64_g8_v128256_bf16"]
    x = W.generate(w)
    rng = np.random.default_rng(5)
    dists = {"all 8 (plain shape)": np.full(w.batch, 8), "uniform 1..8": rng.integers(1, 9, size=w.batch),
             "all 4": np.full(w.batch, 4), "all 1": np.full(w.batch, 1)}
    us_plain = _time_steps(w, x, steps, warmup)
    points = [{"gammas": "plain call (no gammas array)", "us_per_step": round(us_plain, 3),
               "frac_of_8TBs": round(w.logit_bytes / (us_plain * 1e-6) / 8e12, 4)}]
    for name, gam in dists.items():
        us = _time_steps(w, x, steps, warmup, gammas=gam.astype(np.int32))
        own = int(np.sum(2 * gam + 1)) * w.vocab * 2
        p = {"gammas": name, "mean_gamma": round(float(gam.mean()), 3), "us_per_step": round(us, 3),
             "own_row_bytes": own, "frac_of_8TBs": round(own / (us * 1e-6) / 8e12, 4)}
        log(json.dumps(p))
        points.append(p)
    return {"sweep": "ragged", "workload": w.name, "points": points}


def sweep_early_exit(steps: int, warmup: int) -> dict:
    """spec_verify_exact_early_exit against spec_verify_exact on the bf16 shape
    with the largest vocabulary (gamma = 8, V = 128,256) at B = 64 and 128, over
    target-minus-draft noise levels that take the acceptance from ~0.97 down.
    needed_bytes = sum_b of the rows the method uses: 2 (L_b + 1) V s when b
    rejects at L_b, (2 gamma + 1) V s when it accepts every draft."""
    import numpy as np

    from paper_2406_11016_amd import binding
    from paper_2406_11016_amd import workloads as W
    head = W.WORKLOADS["exact_b64_g8_v128256_bf16"]
    plan = [(64, "student_t3", 0.7), (64, "normal", 1.0), (64, "normal", 2.0), (64, "normal", 4.0),
            (128, "student_t3", 0.7), (128, "normal", 2.0)]
    points = []
    for batch, base, noise in plan:
        w = head.with_(batch=batch, base=base, noise_scale=noise)
        x = W.generate(w)
        d, t, tok, uni = binding.to_device(x, "cuda")
        L = binding.verify(d, t, tok, uni, mode="exact")[0].cpu().numpy()
        del d, t
        full = w.logit_bytes
        row = w.vocab * 2
        needed = int(np.sum(np.where(L >= w.gamma, 2 * w.gamma + 1, 2 * (np.maximum(L, 0) + 1)))) * row
        us_single = _time_steps(w, x, steps, warmup)
        us_early = _time_steps(w, x, steps, warmup, early_exit=True)
        p = {"batch": batch, "base": base, "noise": noise, "mean_accepted": round(float(L.mean()), 3),
             "p_all_accepted": round(float((L == w.gamma).mean()), 3),
             "us_single_pass": round(us_single, 3), "us_early_exit": round(us_early, 3),
             "speedup": round(us_single / us_early, 4), "full_bytes": full, "needed_bytes": needed,
             "single_frac_of_8TBs": round(full / (us_single * 1e-6) / 8e12, 4),
             "early_needed_frac_of_8TBs": round(needed / (us_early * 1e-6) / 8e12, 4)}
        log(json.dumps(p))
        points.append(p)
        del x
    return {"sweep": "early_exit", "points": points}


def decode_loop(iterations: int, gamma_max: int = 20, pool: int = 32) -> dict:
    """The decoding loop (gamma rule, one captured graph per gamma) on the B = 1
    workloads, against the same loop with eager calls."""
    import numpy as np

    from paper_2406_11016_amd import workloads as W
    from paper_2406_11016_amd.decode_loop import DecodeLoop, SyntheticSteps
    import torch
    runs = []
    for name in ("exact_b1_g5_v51865_f32", "exact_b1_g10_v32000_f16"):
        w = W.WORKLOADS[name]
        src = SyntheticSteps(w, gamma_max=gamma_max, pool=pool)
        # the synthetic producer alone (four device copies per iteration from
        # torch), at the loop's mean gamma, to separate it from the loop
        probe = DecodeLoop(w.batch, w.vocab, w.dtype, mode=w.mode, gamma_max=gamma_max, use_graphs=False)
        for i in range(20):
            src(probe, i, 5)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(iterations):
            src(probe, i, 5)
        probe.stream.synchronize()
        producer_us = (time.perf_counter() - t0) / iterations * 1e6
        log(f"{name}: producer alone {producer_us:.1f} us per iteration")
        for native, graphs in ((False, True), (False, False), (True, True), (True, False)):
            loop = DecodeLoop(w.batch, w.vocab, w.dtype, mode=w.mode, temperature=w.temperature, alpha=w.alpha,
                              beta=w.beta, gamma0=5, gamma_max=gamma_max, use_graphs=graphs, native=native)
            if graphs:
                loop.capture_all()
            loop.run(src, 20)                                   # warm-up (captures the native graphs)
            t0 = time.perf_counter()
            st = loop.run(src, iterations)
            wall = time.perf_counter() - t0
            dev = loop.run(src, min(iterations, 500), time_device=True).device_us or [float("nan")]
            loop.close()
            gam = np.array(st.gammas)
            p = {"workload": name, "loop": "native" if native else "python", "graphs": graphs,
                 "iterations": iterations, "producer_us_per_iteration": round(producer_us, 2),
                 "us_per_iteration": round(wall / iterations * 1e6, 2),
                 "tokens_per_iteration": round(st.tokens / iterations / w.batch, 3),
                 "tokens_per_s": round(st.tokens / wall, 1),
                 "mean_gamma": round(float(gam.mean()), 2),
                 "gamma_histogram": {int(k): int(v) for k, v in zip(*np.unique(gam, return_counts=True))},
                 "step_device_us_p50": round(float(np.percentile(dev, 50)), 2),
                 "step_device_us_p99": round(float(np.percentile(dev, 99)), 2)}
            log(json.dumps(p))
            runs.append(p)
    return {"sweep": "decode_loop", "gamma0": 5, "gamma_max": gamma_max, "runs": runs,
            "what": "iterations of: copy the next synthetic step's logits into the loop's static buffers, "
                    "verify, copy L and the next token to pinned host memory, synchronise, apply the gamma rule; "
                    "python = torch calls per iteration, native = one library call per iteration "
                    "(spec_verify_loop_step); step_device_us only for the python loop"}


def loop_early_exit(iterations: int, block: int = 8) -> dict:
    """The decoding loop at the headline shape (B = 64, V = 128,256 bf16, gamma
    held at 8: with 64 elements the gamma rule, which grows gamma only when
    every element accepts every draft, soon keeps gamma at 1-2, where the
    early exit has nothing to skip) over iterations alternating in blocks of `block` between the
    headline law (most drafts accepted) and rejection-heavy logits (normal,
    noise 2.0), with the early exit never, always, or chosen per step from the
    previous step's acceptance ("auto"): the step's device time per iteration
    (HIP events around the launch) in each regime."""
    import numpy as np

    from paper_2406_11016_amd import workloads as W
    from paper_2406_11016_amd.decode_loop import DecodeLoop, SyntheticSteps
    head = W.WORKLOADS[W.HEADLINE]
    hi = SyntheticSteps(head, gamma_max=8, pool=2)
    lo = SyntheticSteps(head.with_(base="normal", noise_scale=2.0), gamma_max=8, pool=2)
    plan = [(i // block) % 2 == 0 for i in range(iterations)]      # True: the headline law

    def producer(loop, i, gamma):
        (hi if plan[i] else lo)(loop, i, gamma)

    runs = []
    for mode in ("never", "always", "auto"):
        loop = DecodeLoop(head.batch, head.vocab, head.dtype, gamma0=8, gamma_max=8, early_exit=mode,
                          adapt_gamma=False)
        loop.run(producer, 2 * block)                              # warm-up
        st = loop.run(producer, iterations, time_device=True)
        loop.close()
        dev = np.array(st.device_us)
        ee = np.array(st.early_exit)
        acc = np.array([float(np.mean(np.maximum(a, 0))) for a in st.accepted])
        pl = np.array(plan)
        p = {"early_exit": mode, "iterations": iterations,
             "step_us_mean": round(float(dev.mean()), 2),
             "step_us_headline_law": round(float(dev[pl].mean()), 2),
             "step_us_rejection_heavy": round(float(dev[~pl].mean()), 2),
             "early_exit_share_headline_law": round(float(ee[pl].mean()), 3),
             "early_exit_share_rejection_heavy": round(float(ee[~pl].mean()), 3),
             "mean_accepted_headline_law": round(float(acc[pl].mean()), 2),
             "mean_accepted_rejection_heavy": round(float(acc[~pl].mean()), 2),
             "mean_gamma": round(float(np.mean(st.gammas)), 2)}
        log(json.dumps(p))
        runs.append(p)
    return {"sweep": "loop_early_exit", "block": block, "runs": runs,
            "what": "decoding loop at B=64, gamma=8, V=128256 bf16; blocks of iterations alternate between the "
                    "headline law and normal logits with noise 2.0; step_us = device time of the verification "
                    "step per iteration"}


def run(kind: str, steps: int, warmup: int) -> int:
    import torch
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        return 1
    from paper_2406_11016_amd import binding
    binding.load_library()
    t0 = time.perf_counter()
    if kind == "gamma":
        out = sweep_gamma(steps, warmup)
    elif kind == "alpha_beta":
        out = sweep_alpha_beta(steps, warmup)
    elif kind == "top_k":
        out = sweep_top_k(steps, warmup)
    elif kind == "ragged":
        out = sweep_ragged(steps, warmup)
    elif kind == "early_exit":
        out = sweep_early_exit(steps, warmup)
    elif kind == "loop_early_exit":
        out = loop_early_exit(steps)
    else:
        out = decode_loop(steps)
    out["seconds"] = round(time.perf_counter() - t0, 1)
    print(json.dumps(out), flush=True)
    return 0
