"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than its own formulas:
closed forms, textbook/library routines, invariants the paper states, and the
hand-worked examples in ``tests/golden``.
"""
import math

import numpy as np
import pytest
import scipy.special

from oracle import (acceptance_ratio, first_rejection, inverse_cdf, max_norm,
                    sigmoid, sigmoid_approximation, softmax, verify)
from tests.golden_util import example_arrays, frac

RNG = np.random.default_rng(20240616)


# --- eq. (4): softmax -------------------------------------------------------

def test_softmax_constant_row_is_uniform():
    for V in (1, 2, 7, 64, 1000):
        p = softmax(np.full((3, V), 4.25))
        assert np.allclose(p, 1.0 / V, rtol=0, atol=1e-15)


def test_softmax_two_classes_is_logistic():
    for a, b in [(0.0, 0.0), (1.5, -2.0), (-30.0, 12.0), (700.0, 699.0)]:
        p = softmax(np.array([a, b]))
        assert p[0] == pytest.approx(1.0 / (1.0 + math.exp(b - a)), rel=1e-14)


def test_softmax_matches_library_and_is_shift_invariant():
    w = RNG.normal(0, 3, size=(5, 333))
    assert np.allclose(softmax(w), scipy.special.softmax(w, axis=-1), rtol=1e-13, atol=0)
    assert np.allclose(softmax(w + 1234.5), softmax(w), rtol=1e-10, atol=0)
    assert np.allclose(softmax(w).sum(-1), 1.0, rtol=0, atol=1e-14)


def test_softmax_masked_entries_are_zero():
    p = softmax(np.array([0.0, -np.inf, math.log(3.0), -np.inf]))
    assert np.allclose(p, [0.25, 0.0, 0.75, 0.0], rtol=1e-15, atol=0)


# --- eq. (5): sigmoid approximation ----------------------------------------

def test_sigmoid_closed_forms():
    assert sigmoid(np.array(0.0)) == 0.5
    x = RNG.normal(0, 5, size=1000)
    assert np.allclose(sigmoid(x) + sigmoid(-x), 1.0, rtol=0, atol=1e-15)
    assert np.allclose(sigmoid(x), scipy.special.expit(x), rtol=1e-14, atol=0)
    for k in (0.5, 2.0, 3.0, 9.0):
        assert sigmoid(np.array(math.log(k))) == pytest.approx(k / (1.0 + k), rel=1e-15)


def test_sigmoid_approximation_symmetric_scaling():
    # with alpha = -beta the scaled logit is 1/2 + w / (2 beta)
    beta = 1.0e3
    w = RNG.normal(0, 4, size=257)
    expect = scipy.special.expit(0.5 + w / (2.0 * beta))
    assert np.allclose(sigmoid_approximation(w, -beta, beta), expect, rtol=1e-14, atol=0)
    # unnormalised: positive, below one, and not a distribution
    v = sigmoid_approximation(w, -beta, beta)
    assert np.all(v > 0) and np.all(v < 1) and abs(v.sum() - 1.0) > 1.0


# --- eq. (1): acceptance ratio and first rejection ---------------------------

def test_acceptance_ratio_cases():
    p = np.array([0.2, 0.5, 0.3, 0.0, 0.4])
    q = np.array([0.4, 0.25, 0.3, 0.1, 0.0])
    assert np.allclose(acceptance_ratio(p, q), [0.5, 1.0, 1.0, 0.0, 1.0], rtol=0, atol=0)


def test_first_rejection_index():
    stop = np.array([[False, False, True, True],
                     [True, False, False, False],
                     [False, False, False, False]])
    assert first_rejection(stop).tolist() == [2, 0, 4]


def test_tie_accepts():
    # r == tau accepts: p(x) = 3/4 exactly representable, q(x) = 1 -> tau = 0.75
    z_p = np.log(np.array([[[0.75, 0.25], [0.5, 0.5]]]))
    z_q = np.array([[[0.0, -np.inf]]])
    res = verify(z_q, z_p, np.array([[0]]), np.array([[0.75, 0.3]]), dtype="f64")
    assert res.tau[0, 0] == pytest.approx(0.75, rel=1e-15)
    if res.tau[0, 0] == 0.75:
        assert res.accepted_len[0] == 1


# --- eqs. (2)-(3): residual ------------------------------------------------

def test_max_norm_sums_to_one():
    for V in (2, 9, 500):
        p = softmax(RNG.normal(0, 2, size=(4, V)))
        q = softmax(RNG.normal(0, 2, size=(4, V)))
        a, b = max_norm(p - q)
        assert np.all(a >= 0)
        assert np.allclose((a / b[:, None]).sum(-1), 1.0, rtol=0, atol=1e-12)
        # b is the total-variation distance: sum max(0, p-q) = 1/2 sum |p-q|
        assert np.allclose(b, 0.5 * np.abs(p - q).sum(-1), rtol=1e-12, atol=0)


def test_residual_disjoint_support_is_p():
    p = np.array([0.3, 0.7, 0.0, 0.0])
    q = np.array([0.0, 0.0, 0.6, 0.4])
    a, b = max_norm(p - q)
    assert b == pytest.approx(1.0) and np.allclose(a / b, p)


def test_residual_one_hot_draft_removes_token():
    p = softmax(RNG.normal(0, 1, size=6))
    x0 = 4
    q = np.zeros(6)
    q[x0] = 1.0
    a, b = max_norm(p - q)
    expect = p.copy()
    expect[x0] = 0.0
    assert np.allclose(a / b, expect / expect.sum(), rtol=1e-13, atol=1e-16)
    assert acceptance_ratio(p[x0:x0 + 1], q[x0:x0 + 1])[0] == pytest.approx(p[x0])


# --- inverse CDF -------------------------------------------------------------

def test_inverse_cdf_interval_midpoints():
    w = np.array([0.1, 0.0, 0.25, 0.05, 0.0, 0.6])
    S = np.concatenate([[0.0], np.cumsum(w)])
    for j in range(len(w)):
        if w[j] == 0:
            continue
        u = 0.5 * (S[j] + S[j + 1]) / S[-1]
        got, margin = inverse_cdf(w, np.array(u))
        assert int(got) == j
        assert float(margin) == pytest.approx(0.5 * w[j] / S[-1], rel=1e-12)


def test_inverse_cdf_never_picks_zero_mass():
    w = np.array([0.0, 0.5, 0.0, 0.0, 0.5, 0.0])
    us = np.linspace(0.0, 1.0 - 2.0 ** -24, 2001)
    js, _ = inverse_cdf(np.broadcast_to(w, (us.size, w.size)), us)
    assert set(js.tolist()) == {1, 4}
    assert int(inverse_cdf(w, np.array(0.0))[0]) == 1
    assert int(inverse_cdf(w, np.array(0.5))[0]) == 4   # left-closed intervals


# --- whole steps -------------------------------------------------------------

@pytest.mark.parametrize("idx", range(9))
def test_golden_worked_examples(golden_examples, idx):
    ex = golden_examples[idx]
    draft, target, tokens, uniforms = example_arrays(ex)
    with np.errstate(invalid="ignore"):
        res = verify(draft, target, tokens, uniforms, dtype="f64", mode=ex["mode"],
                     temperature=ex["temperature"], alpha=ex["alpha"], beta=ex["beta"])
    e = ex["expect"]
    assert int(res.accepted_len[0]) == e["accepted_len"], ex["name"]
    assert int(res.next_token[0]) == e["next_token"], ex["name"]
    for c, t in enumerate(e["tau"]):
        if t is not None:
            assert res.tau[0, c] == pytest.approx(frac(t), rel=1e-12, abs=1e-15)
    assert np.allclose(res.final_weights[0], [frac(v) for v in e["final"]], rtol=1e-12, atol=1e-15)
    assert res.mass[0] == pytest.approx(frac(e["mass"]), rel=1e-12)
    assert res.cdf_margin[0] == pytest.approx(frac(e["cdf_margin"]), rel=1e-9)
    assert res.accept_margin[0] == pytest.approx(frac(e["accept_margin"]), rel=1e-9)


def test_golden_examples_are_all_pinned(golden_examples):
    assert len(golden_examples) == 9


@pytest.mark.parametrize("mode", ["exact", "sigmoid"])
def test_identical_draft_and_target_accept_everything(mode):
    B, g, V = 6, 7, 300
    z = RNG.normal(0, 2, size=(B, g + 1, V))
    u = RNG.random((B, g + 1))
    u[0, :g] = 1.0 - 2.0 ** -24
    tokens = RNG.integers(0, V, size=(B, g))
    res = verify(z[:, :g], z, tokens, u, dtype="f64", mode=mode, temperature=0.9,
                 alpha=-1e3, beta=1e3)
    assert np.all(res.tau == 1.0)
    assert np.all(res.accepted_len == g)


def test_disjoint_support_rejects_first_and_samples_target():
    B, g, V = 3, 4, 10
    z_p = np.full((B, g + 1, V), -np.inf)
    z_q = np.full((B, g, V), -np.inf)
    z_p[..., :5] = RNG.normal(0, 1, size=(B, g + 1, 5))
    z_q[..., 5:] = RNG.normal(0, 1, size=(B, g, 5))
    tokens = RNG.integers(5, V, size=(B, g))
    u = RNG.random((B, g + 1)) * 0.999 + 1e-4
    res = verify(z_q, z_p, tokens, u, dtype="f64")
    assert np.all(res.accepted_len == 0)
    assert np.all(res.next_token < 5)
    assert np.allclose(res.final_weights[:, :5], softmax(z_p[:, 0, :5]), rtol=1e-13)


def test_sentinels_and_unread_rows():
    g, V = 3, 16
    z = RNG.normal(0, 1, size=(5, g + 1, V))
    zq = z[:, :g].copy()
    zp = z.copy()
    tokens = RNG.integers(0, V, size=(5, g))
    u = np.full((5, g + 1), 0.5)
    tokens[0, 2] = V                      # invalid token -> sentinel
    zp[1, 0, 3] = np.nan                  # NaN in a read row -> sentinel
    zq[2, 1, 0] = np.inf                  # +inf in a read row (exact) -> sentinel
    zp[3, 0, :] = -np.inf                 # all -inf read row -> sentinel
    # batch 4: reject at c = 0 (p(x) = 0), NaN only in unread rows
    zp[4, 0, tokens[4, 0]] = -np.inf
    zp[4, 1:, 5] = np.nan
    zq[4, 1:, 6] = np.nan
    with np.errstate(invalid="ignore"):
        res = verify(zq, zp, tokens, u, dtype="f64")
    assert res.accepted_len.tolist()[:4] == [-1, -1, -1, -1]
    assert res.next_token.tolist()[:4] == [-1, -1, -1, -1]
    assert res.accepted_len[4] == 0 and 0 <= res.next_token[4] < V


def test_temperature_divides_logits():
    B, g, V = 4, 3, 50
    z = RNG.normal(0, 2, size=(B, g + 1, V))
    zq = z[:, :g] + RNG.normal(0, 1, size=(B, g, V))
    tokens = RNG.integers(0, V, size=(B, g))
    u = RNG.random((B, g + 1))
    a = verify(zq, z, tokens, u, dtype="f64", temperature=0.5)
    b = verify(2 * zq, 2 * z, tokens, u, dtype="f64", temperature=1.0)
    assert np.allclose(a.tau, b.tau, rtol=1e-13)
    assert a.accepted_len.tolist() == b.accepted_len.tolist()


def test_sigmoid_mode_equals_exact_mode_when_masses_agree():
    """When sum(p_hat_c) == sum(q_hat_c) for every row, p_hat/q_hat is the ratio of
    the normalised distributions, so the approximate step (Sec. 3.2.2) must give
    the exact step (Sec. 3.1) run on logits log(p_hat).  Draft rows are
    permutations of the target rows, which makes the sums equal."""
    B, g, V = 40, 3, 24
    alpha, beta = -10.0, 10.0
    z_p = RNG.normal(0, 4, size=(B, g + 1, V))
    z_q = np.stack([np.stack([RNG.permutation(z_p[b, c]) for c in range(g)]) for b in range(B)])
    tokens = RNG.integers(0, V, size=(B, g))
    u = RNG.random((B, g + 1))
    s = verify(z_q, z_p, tokens, u, dtype="f64", mode="sigmoid", alpha=alpha, beta=beta)
    lp = np.log(scipy.special.expit((z_p - alpha) / (beta - alpha)))
    lq = np.log(scipy.special.expit((z_q - alpha) / (beta - alpha)))
    e = verify(lq, lp, tokens, u, dtype="f64", mode="exact")
    assert np.allclose(s.tau, e.tau, rtol=1e-12)
    ok = ~(s.flagged(1e-9) | e.flagged(1e-9))
    assert ok.sum() > 30
    assert s.accepted_len[ok].tolist() == e.accepted_len[ok].tolist()
    assert s.next_token[ok].tolist() == e.next_token[ok].tolist()
    assert np.allclose(s.final_weights, e.final_weights, rtol=1e-10, atol=1e-14)


def test_storage_dtype_decoding():
    from oracle import logits_as_float64
    bits = np.array([0x3F80, 0xC000, 0x7F80, 0xFF80, 0x0000, 0x3E80], dtype=np.uint16)
    assert logits_as_float64(bits, "bf16").tolist() == [1.0, -2.0, np.inf, -np.inf, 0.0, 0.25]
    h = np.array([65504.0, -0.5, 1.0 / 1024], dtype=np.float16)
    assert logits_as_float64(h, "f16").tolist() == [65504.0, -0.5, 1.0 / 1024]
