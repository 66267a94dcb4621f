"""Pins of the oracle's ragged variant (each batch element with its own
number of drafts in padded tensors).  Sec. 3.1 verifies each sequence's
drafts independently; what is pinned here is what that fixes without
re-deriving the step: padding is never read, an element drafting gamma_max
tokens is the plain step, acceptance of identical rows runs to the element's
own gamma, and the bonus token of a one-hot target row is that row's token."""
import numpy as np
import pytest

from oracle import SENTINEL, verify, verify_ragged

RNG = np.random.default_rng(77)


def _case(B, gmax, V):
    zq = RNG.normal(0, 2, size=(B, gmax, V))
    zp = np.concatenate([zq, RNG.normal(0, 2, size=(B, 1, V))], axis=1) + RNG.normal(0, 0.3, size=(B, gmax + 1, V))
    tok = RNG.integers(0, V, size=(B, gmax)).astype(np.int32)
    u = RNG.random((B, gmax + 1)) * 0.999
    return zq, zp, tok, u


@pytest.mark.parametrize("mode", ["exact", "sigmoid"])
def test_full_gamma_is_the_plain_step(mode):
    zq, zp, tok, u = _case(5, 6, 40)
    a = verify(zq, zp, tok, u, dtype="f64", mode=mode, alpha=-10.0, beta=10.0)
    r = verify_ragged(zq, zp, tok, u, np.full(5, 6), dtype="f64", mode=mode, alpha=-10.0, beta=10.0)
    assert np.array_equal(a.accepted_len, r.accepted_len)
    assert np.array_equal(a.next_token, r.next_token)
    assert np.allclose(a.final_weights, r.final_weights, rtol=0, atol=0)


@pytest.mark.parametrize("mode", ["exact", "sigmoid"])
def test_padding_is_not_read(mode):
    B, gmax, V = 6, 7, 30
    zq, zp, tok, u = _case(B, gmax, V)
    gam = np.array([1, 3, 7, 2, 5, 4])
    ref = verify_ragged(zq, zp, tok, u, gam, dtype="f64", mode=mode, alpha=-10.0, beta=10.0)
    zq2, zp2, tok2, u2 = zq.copy(), zp.copy(), tok.copy(), u.copy()
    for b, g in enumerate(gam):
        zq2[b, g:] = np.nan
        zp2[b, g + 1:] = np.nan
        tok2[b, g:] = -5                # invalid tokens beyond the element's drafts
        u2[b, g + 1:] = np.nan
    got = verify_ragged(zq2, zp2, tok2, u2, gam, dtype="f64", mode=mode, alpha=-10.0, beta=10.0)
    assert np.array_equal(ref.accepted_len, got.accepted_len)
    assert np.array_equal(ref.next_token, got.next_token)
    assert np.all(ref.accepted_len >= 0) and np.all(ref.accepted_len <= gam)


def test_identical_rows_accept_to_own_gamma_and_draw_the_bonus_token():
    B, gmax, V = 4, 6, 12
    zq = RNG.normal(0, 1, size=(B, gmax, V))
    zp = np.concatenate([zq, np.full((B, 1, V), -np.inf)], axis=1)
    gam = np.array([1, 2, 4, 6])
    tok = RNG.integers(0, V, size=(B, gmax)).astype(np.int32)
    u = RNG.random((B, gmax + 1)) * 0.999
    # target row g (the bonus row) of element b is one-hot at token 3 + b
    for b, g in enumerate(gam):
        zp[b, g] = -np.inf
        zp[b, g, 3 + b] = 0.0
    r = verify_ragged(zq, zp, tok, u, gam, dtype="f64")
    assert r.accepted_len.tolist() == gam.tolist()          # p == q: eq. (1) gives tau = 1
    assert r.next_token.tolist() == [3, 4, 5, 6]


def test_out_of_range_gamma_is_a_sentinel():
    zq, zp, tok, u = _case(3, 4, 10)
    r = verify_ragged(zq, zp, tok, u, np.array([0, 5, 2]), dtype="f64")
    assert r.accepted_len[0] == SENTINEL and r.next_token[0] == SENTINEL
    assert r.accepted_len[1] == SENTINEL and r.next_token[1] == SENTINEL
    assert 0 <= r.accepted_len[2] <= 2
