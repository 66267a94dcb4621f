"""The multi-step decoding loop: every iteration's decisions are the
oracle's on the inputs that iteration verified, gamma follows the draft-length
rule, and replayed graphs give exactly what eager calls give."""
import numpy as np
import pytest
import torch

from paper_2406_11016_amd import binding
from paper_2406_11016_amd import workloads as W
from paper_2406_11016_amd.decode_loop import DecodeLoop, SyntheticSteps, next_gamma
from tests.gpu_util import run_oracle

pytestmark = pytest.mark.gpu

# B = 1 as in the paper's experiments; noise low enough that gamma grows as well as shrinks
CASES = [
    dict(batch=1, vocab=5003, dtype="f32", mode="exact", noise=0.15),
    dict(batch=1, vocab=32000, dtype="f16", mode="exact", noise=0.3),
    dict(batch=4, vocab=2001, dtype="bf16", mode="exact", noise=0.05),
    dict(batch=2, vocab=3001, dtype="f16", mode="sigmoid", noise=0.5),
]


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    binding.load_library()
    torch.cuda.init()


def _workload(c):
    return W.Workload(f"loop_{c['mode']}_{c['dtype']}", c["mode"], c["batch"], 5, c["vocab"], c["dtype"], "normal",
                      2.0, c["noise"], seed=4242, temperature=1.0, alpha=-1e3, beta=1e3)


@pytest.mark.parametrize("case", CASES, ids=[f"{c['mode']}-B{c['batch']}-{c['dtype']}" for c in CASES])
def test_decode_loop_matches_oracle_and_rule(case):
    w = _workload(case)
    gmax, iters = 12, 40
    src = SyntheticSteps(w, gamma_max=gmax, pool=8)
    runs = {}
    for graphs in (True, False):
        loop = DecodeLoop(w.batch, w.vocab, w.dtype, mode=w.mode, temperature=w.temperature, alpha=w.alpha,
                          beta=w.beta, gamma0=5, gamma_max=gmax, use_graphs=graphs)
        runs[graphs] = loop.run(src, iters)
    for graphs in (True, False):
        loop = DecodeLoop(w.batch, w.vocab, w.dtype, mode=w.mode, temperature=w.temperature, alpha=w.alpha,
                          beta=w.beta, gamma0=5, gamma_max=gmax, use_graphs=graphs, native=True)
        runs[("native", graphs)] = loop.run(src, iters)
        loop.close()
    st = runs[True]
    # replayed graphs, eager calls and the native loop (with and without its
    # own graphs): identical trajectories and outputs
    for key in (False, ("native", True), ("native", False)):
        other = runs[key]
        assert st.gammas == other.gammas, key
        for a, b in zip(st.accepted, other.accepted):
            assert np.array_equal(a, b), key
        for a, b in zip(st.next_tokens, other.next_tokens):
            assert np.array_equal(a, b), key
    # the rule, and the oracle on each iteration's inputs
    assert st.gammas[0] == 5
    grew = shrank = 0
    for i in range(iters):
        g = st.gammas[i]
        if i + 1 < iters:
            assert st.gammas[i + 1] == next_gamma(g, st.accepted[i], gmax)
            grew += st.gammas[i + 1] > g
            shrank += st.gammas[i + 1] < g
        x = src.host_inputs(i, g)
        o = run_oracle(x)
        ok = ~o.flagged(1e-6)
        assert np.array_equal(st.accepted[i][ok], o.accepted_len[ok]), (i, g, st.accepted[i], o.accepted_len)
        assert np.array_equal(st.next_tokens[i][ok], o.next_token[ok]), (i, g, st.next_tokens[i], o.next_token)
    print(f"[loop] {case}: gammas {st.gammas[:20]}... grew {grew} shrank {shrank} tokens {st.tokens}", flush=True)
    assert grew >= 1
