"""The exact mode's early-exit variant (spec_verify_exact_early_exit) through
the C ABI: the same outputs as spec_verify_exact on the same inputs (its row
chunks are twice as long, so its normalisers can differ in the last bits; no
uniform of these seeds lies that close to a threshold), and the oracle's
decisions outside the flagged cases.

Its tiles of a draft position c skip their rows when an element has already
rejected a draft `gate` stages earlier, gate = max(2, ceil(56e6 / (2 B V s)))
(a stage is 2 B V s bytes of stream); when gate >= gamma nothing could be
skipped and the entry point runs the single pass.  The gated shapes below
assert gate < gamma, so that they run the staged kernel; the small shapes check
the fall-back."""
import math

import numpy as np
import pytest
import torch

from paper_2406_11016_amd import binding
from paper_2406_11016_amd import workloads as W
from tests.gpu_util import compare, run_oracle

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    binding.load_library()
    torch.cuda.init()


class _Decisions:
    def __init__(self, acc, nxt):
        self.accepted_len, self.next_token = acc, nxt


def _run(x, early_exit, workspace=None):
    d, t, tok, u = binding.to_device(x)
    acc, nxt = binding.verify(d, t, tok, u, mode="exact", temperature=x.temperature, workspace=workspace,
                              early_exit=early_exit)
    torch.cuda.synchronize()
    return _Decisions(acc.cpu().numpy(), nxt.cpu().numpy())


def _subset(x, idx):
    return W.Inputs(x.draft[idx], x.target[idx], x.tokens[idx], x.uniforms[idx], x.dtype, x.mode,
                    x.temperature, x.alpha, x.beta)


def _check(x, label, oracle_sample=None, seed=0):
    print(f"[early-exit] {label}: B={x.batch} gamma={x.gamma} V={x.vocab} {x.dtype}", flush=True)
    e = _run(x, True)
    s = _run(x, False)
    assert np.array_equal(e.accepted_len, s.accepted_len), (label, e.accepted_len, s.accepted_len)
    assert np.array_equal(e.next_token, s.next_token), (label, e.next_token, s.next_token)
    if oracle_sample is None or oracle_sample >= x.batch:
        idx = np.arange(x.batch)
    else:
        idx = np.sort(np.random.default_rng(seed).choice(x.batch, oracle_sample, replace=False))
    xs = _subset(x, idx)
    compare(xs, _Decisions(e.accepted_len[idx], e.next_token[idx]), run_oracle(xs), check_probs=False,
            label=label)
    return e


EXACT = [n for n, w in W.WORKLOADS.items() if w.mode == "exact"]


@pytest.mark.parametrize("name", EXACT)
def test_named_workloads(name):
    _check(W.generate(W.WORKLOADS[name]), name)


@pytest.mark.parametrize("batch,noise", [(64, 0.7), (64, 3.0), (128, 0.7), (128, 3.0)])
def test_gated_stages_at_the_largest_vocabulary(batch, noise):
    # noise 3.0 rejects early in most elements, so most later rows are skipped
    w = W.WORKLOADS["exact_b64_g8_v128256_bf16"].with_(batch=batch, noise_scale=noise, seed=2100 + batch)
    assert _gate(w.batch, w.vocab, w.dtype) < w.gamma
    x = W.generate(w)
    e = _check(x, f"B={batch} noise={noise}", oracle_sample=24, seed=batch)
    print(f"[early-exit]   mean accepted {e.accepted_len.mean():.2f} of {x.gamma}", flush=True)


def _gate(batch, vocab, dtype):
    s = {"f32": 4, "f16": 2, "bf16": 2}[dtype]
    return max(2, math.ceil(56e6 / (2 * batch * vocab * s)))


# (gamma, B, V, dtype): each with gate < gamma; the row-normaliser merge groups
# 16, 8, 4, 2 or 1 lanes per row by the number of rows (2 gamma)
GATED = [(3, 56, 128256, "bf16"), (5, 28, 128256, "bf16"), (16, 10, 51865, "f32"), (17, 10, 51865, "f32"),
         (33, 10, 50000, "f16"), (64, 40, 3001, "f32"), (128, 24, 5003, "f32")]


@pytest.mark.parametrize("gamma,batch,vocab,dtype", GATED, ids=[f"g{g[0]}" for g in GATED])
@pytest.mark.parametrize("noise", [0.05, 1.0])
def test_gamma_range(gamma, batch, vocab, dtype, noise):
    assert _gate(batch, vocab, dtype) < gamma
    x = W.small_case(batch, gamma, vocab, dtype, seed=300 + gamma, noise_scale=noise)
    _check(x, f"gamma={gamma} noise={noise} {dtype} gate={_gate(batch, vocab, dtype)}", oracle_sample=6,
           seed=gamma)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("V", [1, 2, 7, 65, 300007])
def test_fall_back_to_the_single_pass(dtype, V):
    # too short a stream to gate any decision row (gate >= gamma): the single
    # pass runs; the result is the same
    x = W.small_case(3, 3, V, dtype, seed=400 + V)
    assert _gate(3, V, dtype) >= 3
    _check(x, f"V={V} {dtype}")


@pytest.mark.parametrize("name", ["exact_b1_g5_v51865_f32", "exact_b16_g5_v51865_f32"])
def test_fall_back_on_the_small_batch_workloads(name):
    """The named small-batch workloads gate nothing, so the early exit runs the
    single pass (the host's choice is checked on the CPU by
    tests/native/plan_check.cpp; the two entry points' times are compared in
    bench_sweeps.py): the outputs are the single pass's and the oracle's."""
    w = W.WORKLOADS[name]
    assert _gate(w.batch, w.vocab, w.dtype) >= w.gamma
    _check(W.generate(w), name)


def test_sentinels():
    """Sentinel elements inside a gated shape (bf16 bits: NaN 0x7fc0, -inf 0xff80)."""
    x = W.small_case(56, 3, 128256, "bf16", seed=41)
    assert _gate(56, 128256, "bf16") < 3
    nan, ninf = np.uint16(0x7fc0), np.uint16(0xff80)
    x.tokens[0, 1] = 128256                   # invalid token
    x.tokens[1, 0] = -3
    x.target[2, 0, :] = nan                   # NaN in the first row pair
    x.uniforms[3, :] = 0.0                    # accept everything -> bonus row read
    x.target[3, 3, :] = nan
    x.draft[4, 2, 7] = nan                    # NaN in a row the scan reaches
    x.tokens[4, 2] = 8
    x.uniforms[4, :3] = 0.0
    x.target[5, :2, :] = ninf                 # all -inf rows
    x.target[6, 0, x.tokens[6, 0]] = ninf     # rejected at the first draft ...
    x.draft[6, 2, :] = nan                    # ... so a NaN row after it is never needed
    e = _run(x, True)
    s = _run(x, False)
    assert e.accepted_len.tolist() == s.accepted_len.tolist()
    assert e.next_token.tolist() == s.next_token.tolist()
    idx = np.arange(8)
    o = run_oracle(_subset(x, idx))
    assert e.accepted_len[idx].tolist() == o.accepted_len.tolist(), (e.accepted_len[idx], o.accepted_len)
    assert e.next_token[idx].tolist() == o.next_token.tolist(), (e.next_token[idx], o.next_token)
    assert e.accepted_len[:6].tolist() == [-1] * 6
    assert e.accepted_len[6] == 0 and e.next_token[6] >= 0


def test_rows_past_the_first_rejection_do_not_matter():
    """NaN fills every row after an element's first rejection (and its bonus
    row); the method never needs them (Sec. 3.1), so the element's outputs
    are those of the oracle.  At this shape the tiles of a position gate on
    the decision two stages earlier, so most of those rows are skipped."""
    w = W.WORKLOADS["exact_b64_g8_v128256_bf16"].with_(batch=128, gamma=4, seed=2200)
    assert _gate(w.batch, w.vocab, w.dtype) < w.gamma
    x = W.generate(w)
    nan = np.uint16(0x7fc0)                   # bf16 NaN bits
    for b in range(0, 128, 3):
        L = b % 4
        x.uniforms[b, :L] = 0.0
        x.target[b, L, x.tokens[b, L]] = np.uint16(0xff80)   # -inf: tau = 0, rejected at L
        x.target[b, L + 1:, :] = nan
        x.draft[b, L + 1:, :] = nan
    idx = np.arange(0, 128, 3)
    e = _run(x, True)
    assert np.all(e.accepted_len[idx] == idx % 4), e.accepted_len[idx]
    xs = _subset(x, idx)
    compare(xs, _Decisions(e.accepted_len[idx], e.next_token[idx]), run_oracle(xs), check_probs=False,
            label="rows past the first rejection")
    # the other elements still match the single pass
    s = _run(x, False)
    rest = np.setdiff1d(np.arange(128), idx)
    assert np.array_equal(e.accepted_len[rest], s.accepted_len[rest])
    assert np.array_equal(e.next_token[rest], s.next_token[rest])


def test_workspace_shared_with_the_single_pass_returns_to_zero():
    big = W.generate(W.WORKLOADS["exact_b64_g8_v128256_bf16"].with_(batch=96, noise_scale=2.0, seed=2300))
    small = W.small_case(5, 4, 7001, "f16", seed=81)
    small.tokens[1, 0] = -1                    # a sentinel element must clean up too
    ws = binding.new_workspace(96, 8, 128256, torch.bfloat16, "cuda")
    first = None
    for i in range(4):
        for x in (big, small):
            for ee in (True, False):
                r = _run(x, ee, workspace=ws)
                assert int(torch.count_nonzero(ws)) == 0, (i, x.batch, ee)
                if x is big:
                    if first is None:
                        first = r
                    assert np.array_equal(r.accepted_len, first.accepted_len)
                    assert np.array_equal(r.next_token, first.next_token)


def test_binding_rejects_other_modes():
    x = W.small_case(2, 2, 100, "f32", mode="sigmoid", seed=5)
    d, t, tok, u = binding.to_device(x)
    with pytest.raises(binding.SpecVerifyError):
        binding.verify(d, t, tok, u, mode="sigmoid", early_exit=True)
    with pytest.raises(binding.SpecVerifyError):
        binding.verify(d, t, tok, u, mode="exact", early_exit=True, probe=True)
