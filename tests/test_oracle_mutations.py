"""Plausible mistakes planted in the oracle (on the CPU) must fail its pins.

Each mutation replaces one step of ``oracle.spec_oracle`` with a subtly wrong
version; the hand-worked examples must then disagree with the oracle.
"""
import numpy as np
import pytest

import oracle.spec_oracle as so
from tests.golden_util import example_arrays, frac


def _wrong_residual_sign(f):
    a = np.maximum(0.0, -f)
    return a, np.sum(a, axis=-1)


def _no_clamp_ratio(p_x, q_x):
    with np.errstate(divide="ignore", invalid="ignore"):
        return np.where(q_x > 0.0, p_x / np.where(q_x > 0.0, q_x, 1.0), 1.0)


def _cdf_left_closed(weights, u):
    S = np.cumsum(weights, axis=-1)
    t = u * S[..., -1]
    j = np.sum(S < t[..., None], axis=-1)
    return j.astype(np.int64), np.ones_like(t)


def _sigmoid_unscaled(w, alpha, beta):
    return so.sigmoid(w - alpha)


def _softmax_no_temperature_guard(w):
    e = np.exp(w)
    return e / np.sum(e, axis=-1, keepdims=True) ** 2


def _margin_over_all_drafts(r, tau, L):
    with np.errstate(invalid="ignore"):
        return np.nanmin(np.abs(r - tau), axis=-1)


def _margin_without_reject(r, tau, L):
    gamma = tau.shape[-1]
    examined = np.arange(gamma)[None, :] < L[:, None]     # drops the rejected draft itself
    with np.errstate(invalid="ignore"):
        return np.where(examined, np.abs(r - tau), np.inf).min(axis=-1)


MUTATIONS = {
    "residual_sign": ("max_norm", _wrong_residual_sign),
    "ratio_unclamped": ("acceptance_ratio", _no_clamp_ratio),
    "cdf_left_closed": ("inverse_cdf", _cdf_left_closed),
    "sigmoid_unscaled": ("sigmoid_approximation", _sigmoid_unscaled),
    "softmax_wrong_norm": ("softmax", _softmax_no_temperature_guard),
    "margin_over_unexamined_drafts": ("acceptance_margin", _margin_over_all_drafts),
    "margin_without_the_rejected_draft": ("acceptance_margin", _margin_without_reject),
}


def _golden_failures(examples):
    failures = 0
    for ex in examples:
        draft, target, tokens, uniforms = example_arrays(ex)
        try:
            with np.errstate(all="ignore"):
                res = so.verify(draft, target, tokens, uniforms, dtype="f64", mode=ex["mode"],
                                temperature=ex["temperature"], alpha=ex["alpha"], beta=ex["beta"])
        except Exception:
            failures += 1
            continue
        e = ex["expect"]
        ok = (int(res.accepted_len[0]) == e["accepted_len"]
              and int(res.next_token[0]) == e["next_token"]
              and all(t is None or abs(res.tau[0, c] - frac(t)) < 1e-9 for c, t in enumerate(e["tau"]))
              and np.allclose(res.final_weights[0], [frac(v) for v in e["final"]], atol=1e-9)
              and abs(res.accept_margin[0] - frac(e["accept_margin"])) < 1e-9)
        failures += 0 if ok else 1
    return failures


def _unit_failures():
    """Boundary checks of the inverse CDF: left-closed intervals, zero-mass tokens."""
    w = np.array([0.0, 0.5, 0.0, 0.0, 0.5, 0.0])
    got = [int(so.inverse_cdf(w, np.array(u))[0]) for u in (0.0, 0.25, 0.5, 0.75)]
    return int(got != [1, 1, 4, 4])


def test_unmutated_oracle_passes_golden(golden_examples):
    assert _golden_failures(golden_examples) == 0
    assert _unit_failures() == 0


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(golden_examples, monkeypatch, name):
    attr, fn = MUTATIONS[name]
    monkeypatch.setattr(so, attr, fn)
    assert _golden_failures(golden_examples) + _unit_failures() > 0, name


def test_off_by_one_scan_is_caught(golden_examples, monkeypatch):
    real = so.first_rejection

    def wrong(stop):
        return np.minimum(real(stop) + 1, stop.shape[-1])

    monkeypatch.setattr(so, "first_rejection", wrong)
    assert _golden_failures(golden_examples) > 0
