"""Helpers of the GPU parity tests: run the HIP path and the oracle on the same
inputs and compare them element by element."""
from dataclasses import dataclass

import numpy as np
import scipy.special
import torch

import oracle
from paper_2406_11016_amd import binding

FLAG_EPS = 1e-6                       # decisions within this of a threshold are flagged
PROB_RTOL = {"f32": 1e-5, "f16": 2e-3, "bf16": 2e-3, "f64": 1e-5}


@dataclass
class GpuResult:
    accepted_len: np.ndarray
    next_token: np.ndarray
    tau: np.ndarray
    weights: np.ndarray
    mass: np.ndarray
    lognorm: np.ndarray = None


def run_gpu(x, probe=True, workspace=None, device="cuda"):
    d, t, tok, u = binding.to_device(x, device)
    out = binding.verify(d, t, tok, u, mode=x.mode, temperature=x.temperature, alpha=x.alpha, beta=x.beta,
                         probe=probe, workspace=workspace)
    torch.cuda.synchronize()
    if not probe:
        return out[0].cpu().numpy(), out[1].cpu().numpy()
    acc, nxt, pr = out
    return GpuResult(acc.cpu().numpy(), nxt.cpu().numpy(), pr.tau.cpu().numpy(), pr.weights.cpu().numpy(),
                     pr.mass.cpu().numpy(), None if pr.lognorm is None else pr.lognorm.cpu().numpy())


def run_oracle(x):
    with np.errstate(all="ignore"):
        return oracle.verify(x.draft, x.target, x.tokens, x.uniforms, dtype=x.dtype, mode=x.mode,
                             temperature=x.temperature, alpha=x.alpha, beta=x.beta)


def compare(x, g: GpuResult, o, *, check_probs=True, label=""):
    """Bit-exact decisions outside the flagged cases; probabilities within the
    tolerance of the storage dtype.  Returns the number of flagged elements."""
    flagged = o.flagged(FLAG_EPS)
    ok = ~flagged
    bad_len = np.nonzero(ok & (g.accepted_len != o.accepted_len))[0]
    assert bad_len.size == 0, (label, "accepted_len", bad_len[:8], g.accepted_len[bad_len[:8]],
                               o.accepted_len[bad_len[:8]], o.accept_margin[bad_len[:8]])
    bad_tok = np.nonzero(ok & (g.next_token != o.next_token))[0]
    assert bad_tok.size == 0, (label, "next_token", bad_tok[:8], g.next_token[bad_tok[:8]],
                               o.next_token[bad_tok[:8]], o.cdf_margin[bad_tok[:8]])
    # outputs are in range
    valid = o.accepted_len >= 0
    assert np.all((g.accepted_len[valid] >= 0) & (g.accepted_len[valid] <= x.gamma)), label
    assert np.all((g.next_token[valid] >= 0) & (g.next_token[valid] < x.vocab)), label
    if not check_probs:
        return int(flagged.sum())
    rtol = PROB_RTOL[x.dtype]
    # eq. (1): tau where the oracle's is finite
    fin = np.isfinite(o.tau)
    assert np.all(np.abs(g.tau[fin] - o.tau[fin]) <= rtol * np.abs(o.tau[fin]) + 1e-300), (
        label, "tau", np.max(np.abs(g.tau[fin] - o.tau[fin]) / np.maximum(o.tau[fin], 1e-300)))
    # the final distribution a/b, on elements where decisions agree on the row
    same = valid & (g.accepted_len == o.accepted_len) & ~o.fallback
    if same.any():
        gw = g.weights[same] / g.mass[same][:, None]
        ow = o.final_weights[same]
        scale = np.abs(ow)
        if x.mode == "exact":
            # residual rows: the error of p - q is bounded by the operands (p + q)/(2b)
            L = o.accepted_len[same]
            zt = oracle.logits_as_float64(x.target, x.dtype)[same]
            zd = oracle.logits_as_float64(x.draft, x.dtype)[same]
            res = L < x.gamma
            if res.any():
                idx = np.nonzero(res)[0]
                P = scipy.special.softmax(zt[idx, L[idx]] / x.temperature, axis=-1)
                Q = scipy.special.softmax(zd[idx, L[idx]] / x.temperature, axis=-1)
                scale[idx] = np.maximum(scale[idx], (P + Q) / (2.0 * o.mass[same][idx, None]))
        err = np.abs(gw - ow)
        lim = rtol * scale + 1e-12 * np.max(ow, axis=-1, keepdims=True)
        worst = np.unravel_index(np.argmax(err - lim), err.shape)
        assert np.all(err <= lim), (label, "final weights", worst, gw[worst], ow[worst], scale[worst])
        assert np.allclose(g.mass[same], o.mass[same], rtol=rtol, atol=0), (label, "mass")
    if g.lognorm is not None:
        zt = oracle.logits_as_float64(x.target, x.dtype) / x.temperature
        zd = oracle.logits_as_float64(x.draft, x.dtype) / x.temperature
        with np.errstate(all="ignore"):
            ref = np.concatenate([scipy.special.logsumexp(zt, axis=-1), scipy.special.logsumexp(zd, axis=-1)], 1)
        fin = np.isfinite(ref)
        assert np.all(np.abs(g.lognorm[fin] - ref[fin]) <= 1e-6 * np.maximum(1.0, np.abs(ref[fin]))), (
            label, "lognorm", np.max(np.abs(g.lognorm[fin] - ref[fin])))
    return int(flagged.sum())
