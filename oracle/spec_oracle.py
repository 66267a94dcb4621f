"""Plain float64 CPU oracle of the speculative-sampling verification step.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the CPU
baseline leg of the benchmark may import this module; the library path never
does, and this module imports nothing from the library.

It follows "Optimized Speculative Sampling for GPU Hardware Accelerators"
(Wagner et al., arXiv 2406.11016):

* Sec. 3.1 (Speculative sampling): acceptance of drafted token ``x_c`` iff
  ``r_c <= tau_c(x_c)`` with ``tau_c = min(1, p/q)`` -- eq. (1); stop at the
  first rejection; on rejection resample from ``max_norm(p - q)`` -- eq. (2),
  where ``max_norm(f) = max(0, f) / sum max(0, f) = a(x) / b`` -- eq. (3).
* Sec. 3.2.2 (Approximated optimization): the numerically stable softmax of
  eq. (4) parameterises ``p`` and ``q`` in the exact mode; the sigmoid of the
  rescaled logits, eq. (5), replaces it in the approximate mode, with the same
  acceptance test and residual applied to ``p_hat``, ``q_hat``.

Every array is computed in float64, batch element by batch element
vectorised over the batch axis only; there is no blocking, fusion or
reordering of the sums beyond what the equations state (``numpy.sum`` /
``numpy.cumsum`` over the vocabulary).

Readings where the paper is silent (each is also listed in the design notes):

1. all ``gamma`` drafts accepted: the next token is drawn from the target's
   distribution at position ``gamma`` (the standard rule of the speculative
   sampling papers the method builds on); in sigmoid mode that distribution is
   ``p_hat_gamma / sum p_hat_gamma`` -- *parity unpinned* by the paper;
2. sampling is by inverse CDF with a caller-supplied uniform ``u``: the first
   index ``j`` with ``cumsum(a)[j] > u * b``;
3. ``uniforms[b, c]`` is ``r_c`` for ``c < gamma``; ``uniforms[b, gamma]`` drives
   the final sample;
4. a tie ``r_c == tau_c`` accepts (eq. (1) uses ``<=``);
5. ``q(x_c) == 0`` gives ``tau_c = 1`` (the limit of ``min(1, p/q)``);
6. ``b == 0`` after a rejection (possible in sigmoid mode, where ``p_hat`` and
   ``q_hat`` are unnormalised) falls back to sampling ``p_L / sum p_L``;
7. temperature ``T`` divides the logits before the softmax and before the
   sigmoid rescaling;
8. a drafted token outside ``[0, V)``, a read row whose probabilities are not
   finite (NaN logit, +inf logit in exact mode, an all ``-inf`` row in exact
   mode), or a non-finite / zero final mass yields the sentinel
   ``accepted_len = next_token = -1`` for that batch element.  Rows after the
   first rejection are not read.  In the exact mode a row is read whole (its
   softmax needs every logit); the sigmoid mode is element-wise, so for the
   drafts it examines it reads only the values at the drafted tokens, and it
   reads whole only the row(s) the next token is drawn from.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

SENTINEL = -1


# ---------------------------------------------------------------------------
# input decoding
# ---------------------------------------------------------------------------

def logits_as_float64(stored: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of stored logits.  ``dtype`` is "f64", "f32",
    "f16" or "bf16" (the latter given as raw uint16 bit patterns)."""
    if dtype == "bf16":
        bits = np.asarray(stored, dtype=np.uint16).astype(np.uint32) << 16
        return bits.view(np.float32).astype(np.float64)
    if dtype in ("f64", "f32", "f16"):
        return np.asarray(stored).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


# ---------------------------------------------------------------------------
# the distributions
# ---------------------------------------------------------------------------

def softmax(w: np.ndarray) -> np.ndarray:
    """Numerically stable softmax over the last axis, eq. (4):
    ``exp(w_j - w_max) / sum_l exp(w_l - w_max)``."""
    w_max = np.max(w, axis=-1, keepdims=True)
    e = np.exp(w - w_max)
    return e / np.sum(e, axis=-1, keepdims=True)


def sigmoid(x: np.ndarray) -> np.ndarray:
    """``sigma(x) = 1 / (1 + exp(-x))`` (definition under eq. (5))."""
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-x))


def sigmoid_approximation(w: np.ndarray, alpha: float, beta: float) -> np.ndarray:
    """Eq. (5): ``sigma((w - alpha) / (beta - alpha))`` element-wise; the values
    are positive but do not sum to one."""
    return sigmoid((w - alpha) / (beta - alpha))


# ---------------------------------------------------------------------------
# the steps of the verification
# ---------------------------------------------------------------------------

def acceptance_ratio(p_x: np.ndarray, q_x: np.ndarray) -> np.ndarray:
    """Eq. (1): ``tau = min(1, p(x) / q(x))``; ``tau = 1`` where ``q(x) == 0``."""
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(q_x > 0.0, p_x / np.where(q_x > 0.0, q_x, 1.0), 1.0)
    return np.minimum(1.0, ratio)


def first_rejection(stop: np.ndarray) -> np.ndarray:
    """Index of the first ``True`` along the last axis (the first drafted
    token that is rejected), or the axis length when there is none."""
    gamma = stop.shape[-1]
    any_stop = np.any(stop, axis=-1)
    return np.where(any_stop, np.argmax(stop, axis=-1), gamma)


def max_norm(f: np.ndarray):
    """Eq. (3): returns the numerator ``a(x) = max(0, f(x))`` and the
    denominator ``b = sum_x a(x)`` (over the last axis)."""
    a = np.maximum(0.0, f)
    return a, np.sum(a, axis=-1)


def inverse_cdf(weights: np.ndarray, u: np.ndarray):
    """Sample index ``j`` from unnormalised non-negative ``weights`` ([..., V])
    with uniform ``u`` ([...]): the first ``j`` with ``cumsum(w)[j] > u * sum(w)``.

    Returns ``(j, margin)``, where ``margin`` is the distance of ``u * sum(w)``
    to the nearer edge of the chosen interval, relative to ``sum(w)``."""
    S = np.cumsum(weights, axis=-1)
    total = S[..., -1]
    t = u * total
    j = np.sum(S <= t[..., None], axis=-1)
    V = weights.shape[-1]
    # t < total whenever u < 1 and total > 0; guard the degenerate case by
    # the last index carrying positive weight.
    last_pos = V - 1 - np.argmax((weights > 0)[..., ::-1], axis=-1)
    j = np.where(j >= V, last_pos, j)
    upper = np.take_along_axis(S, j[..., None], axis=-1)[..., 0]
    lower = np.where(j > 0, np.take_along_axis(S, np.maximum(j - 1, 0)[..., None], axis=-1)[..., 0], 0.0)
    with np.errstate(divide="ignore", invalid="ignore"):
        margin = np.minimum(upper - t, t - lower) / total
    return j.astype(np.int64), margin


def acceptance_margin(r: np.ndarray, tau: np.ndarray, L: np.ndarray) -> np.ndarray:
    """How close the examined acceptance decisions came to flipping: the
    minimum of ``|r_c - tau_c|`` over the drafts the scan of Sec. 3.1 looks
    at, ``c = 0 .. min(L, gamma - 1)`` (it stops at the first rejection, so
    later drafts play no part).  ``r``, ``tau`` are [B, gamma], ``L`` is [B];
    returns [B] (the parity bar's near-threshold flag, reading 12)."""
    gamma = tau.shape[-1]
    examined = np.arange(gamma)[None, :] <= L[:, None]
    with np.errstate(invalid="ignore"):
        return np.where(examined, np.abs(r - tau), np.inf).min(axis=-1)


# ---------------------------------------------------------------------------
# the whole step
# ---------------------------------------------------------------------------

@dataclass
class OracleResult:
    accepted_len: np.ndarray     # [B] int64, in [0, gamma] or -1
    next_token: np.ndarray       # [B] int64, in [0, V) or -1
    tau: np.ndarray              # [B, gamma] acceptance ratios, eq. (1) / its approximation
    final_weights: np.ndarray    # [B, V] a(x)/b of the distribution the next token is drawn from
    mass: np.ndarray             # [B] its denominator b (1 for a softmax bonus row)
    accept_margin: np.ndarray    # [B] min |r_c - tau_c| over the drafts examined
    cdf_margin: np.ndarray       # [B] margin of the final inverse-CDF draw
    fallback: np.ndarray         # [B] bool: b == 0 after a rejection (reading 6)

    def flagged(self, eps: float = 1e-6) -> np.ndarray:
        """Batch elements whose decisions lie within ``eps`` of a threshold."""
        return (self.accept_margin < eps) | (self.cdf_margin < eps)


def verify(draft_logits: np.ndarray, target_logits: np.ndarray,
           draft_tokens: np.ndarray, uniforms: np.ndarray, *, dtype: str,
           mode: str = "exact", temperature: float = 1.0,
           alpha: float = -1.0e4, beta: float = 1.0e4) -> OracleResult:
    """One verification step for every batch element.

    ``draft_logits`` [B, gamma, V] and ``target_logits`` [B, gamma+1, V] are
    the stored logits (decoded exactly to float64), ``draft_tokens`` [B, gamma]
    the drafted tokens, ``uniforms`` [B, gamma+1] the uniforms (reading 3).
    """
    if mode not in ("exact", "sigmoid"):
        raise ValueError(mode)
    z_q = logits_as_float64(draft_logits, dtype)
    z_p = logits_as_float64(target_logits, dtype)
    B, gamma, V = z_q.shape
    assert z_p.shape == (B, gamma + 1, V)
    r = np.asarray(uniforms, dtype=np.float64)
    x = np.asarray(draft_tokens, dtype=np.int64)

    # temperature (reading 7), then the two distributions
    w_q = z_q / temperature
    w_p = z_p / temperature
    with np.errstate(invalid="ignore", over="ignore"):
        if mode == "exact":
            P = softmax(w_p)                                   # eq. (4)
            Q = softmax(w_q)
        else:
            P = sigmoid_approximation(w_p, alpha, beta)        # eq. (5)
            Q = sigmoid_approximation(w_q, alpha, beta)
    row_ok_p = np.all(np.isfinite(P), axis=-1)                 # [B, gamma+1]
    row_ok_q = np.all(np.isfinite(Q), axis=-1)                 # [B, gamma]
    token_ok = np.all((x >= 0) & (x < V), axis=-1)             # [B]
    xs = np.clip(x, 0, V - 1)

    # eq. (1) at the drafted tokens
    p_x = np.take_along_axis(P[:, :gamma, :], xs[..., None], axis=-1)[..., 0]
    q_x = np.take_along_axis(Q, xs[..., None], axis=-1)[..., 0]
    with np.errstate(invalid="ignore"):
        tau = acceptance_ratio(p_x, q_x)
    accepted = r[:, :gamma] <= tau
    if mode == "exact":
        row_ok = row_ok_p[:, :gamma] & row_ok_q & np.isfinite(tau)
    else:
        row_ok = np.isfinite(tau)

    # first rejection; an unreadable row also ends the scan (as a sentinel)
    stop = (~accepted) | (~row_ok)
    L = first_rejection(stop)                                  # [B]
    bad = ~token_ok.copy()
    Lc = np.minimum(L, gamma - 1)
    bad |= (L < gamma) & ~row_ok[np.arange(B), Lc]
    bad |= (L == gamma) & ~row_ok_p[:, gamma]

    # margins of the examined acceptance decisions
    acc_margin = acceptance_margin(r[:, :gamma], tau, L)

    # the distribution of the next token, eqs. (2)-(3) or the bonus row
    bi = np.arange(B)
    rows_p = P[bi, np.minimum(L, gamma)]                       # [B, V]
    rows_q = Q[bi, Lc]                                         # [B, V]
    with np.errstate(invalid="ignore"):
        a_res, b_res = max_norm(rows_p - rows_q)
    rejected = L < gamma
    bad |= rejected & ~np.isfinite(b_res)
    fallback = rejected & (b_res == 0.0)
    use_p = (~rejected) | fallback
    weights = np.where(use_p[:, None], rows_p, a_res)
    mass = np.where(use_p, np.sum(rows_p, axis=-1), b_res)
    bad |= ~(np.isfinite(mass) & (mass > 0.0))

    safe_w = np.where(bad[:, None], 1.0, weights)
    j, cdf_margin = inverse_cdf(safe_w, r[:, gamma])
    with np.errstate(invalid="ignore", divide="ignore"):
        final = safe_w / np.sum(safe_w, axis=-1, keepdims=True)

    accepted_len = np.where(bad, SENTINEL, L).astype(np.int64)
    next_token = np.where(bad, SENTINEL, j).astype(np.int64)
    return OracleResult(accepted_len, next_token, tau, final, mass,
                        np.where(bad, np.inf, acc_margin),
                        np.where(bad, np.inf, cdf_margin), fallback & ~bad)


def verify_ragged(draft_logits: np.ndarray, target_logits: np.ndarray,
                  draft_tokens: np.ndarray, uniforms: np.ndarray, gammas: np.ndarray, *, dtype: str,
                  mode: str = "exact", temperature: float = 1.0,
                  alpha: float = -1.0e4, beta: float = 1.0e4) -> OracleResult:
    """Batch elements with their own number of drafts, in padded tensors.

    Sec. 3.1 verifies each sequence's drafts on their own, so element ``b``
    with ``g = gammas[b]`` drafts is exactly the step of :func:`verify` on its
    draft rows ``0..g-1``, target rows ``0..g``, tokens ``0..g-1`` and
    uniforms ``0..g`` (the last one driving the final draw); whatever the
    padded tensors hold beyond that is not read.  An element with ``g``
    outside ``1 .. gamma_max`` gets the sentinel.  ``tau`` is padded with NaN.
    """
    B, gmax, V = np.shape(draft_logits)
    acc = np.full(B, SENTINEL, dtype=np.int64)
    nxt = np.full(B, SENTINEL, dtype=np.int64)
    tau = np.full((B, gmax), np.nan)
    final = np.zeros((B, V))
    mass = np.full(B, np.nan)
    am = np.full(B, np.inf)
    cm = np.full(B, np.inf)
    fb = np.zeros(B, dtype=bool)
    for b in range(B):
        g = int(gammas[b])
        if not 1 <= g <= gmax:
            continue
        o = verify(draft_logits[b:b + 1, :g], target_logits[b:b + 1, :g + 1], draft_tokens[b:b + 1, :g],
                   uniforms[b:b + 1, :g + 1], dtype=dtype, mode=mode, temperature=temperature,
                   alpha=alpha, beta=beta)
        acc[b], nxt[b] = o.accepted_len[0], o.next_token[0]
        tau[b, :g] = o.tau[0]
        final[b], mass[b] = o.final_weights[0], o.mass[0]
        am[b], cm[b], fb[b] = o.accept_margin[0], o.cdf_margin[0], o.fallback[0]
    return OracleResult(acc, nxt, tau, final, mass, am, cm, fb)
