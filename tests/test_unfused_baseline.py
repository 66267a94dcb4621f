"""The unfused PyTorch comparison baseline computes the same step.

It works in fp32 (softmax, cumsum), so it is compared with the oracle only
where the oracle's acceptance and CDF margins exceed 1e-5 (an fp32 softmax
carries ~1e-7 relative error, and an fp32 parallel running sum over V entries
about log2(V) 2^-24 of the total); there its decisions must match exactly.
The sigmoid mode's final distribution is nearly uniform, so its CDF margins
are naturally of order 1 / (2 V)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2406_11016_amd import binding, unfused_torch
from paper_2406_11016_amd import workloads as W

pytestmark = pytest.mark.gpu

CASES = [
    ("exact_b16_g5_v51865_f32", dict(vocab=5003)),
    ("exact_b1_g10_v32000_f16", dict(batch=8, vocab=6007)),
    ("exact_b64_g8_v128256_bf16", dict(batch=8, vocab=20011)),
    ("sigmoid_b32_g10_v50272_f16_t0.7", dict(batch=8, vocab=10007)),
]


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")


@pytest.mark.parametrize("name,over", CASES, ids=[c[0] for c in CASES])
def test_unfused_matches_oracle(name, over):
    w = W.WORKLOADS[name].with_(**over)
    x = W.generate(w)
    d, t, tok, u = binding.to_device(x, "cuda")
    L, nxt = unfused_torch.verify(d, t, tok, u, mode=x.mode, temperature=x.temperature, alpha=x.alpha,
                                  beta=x.beta)
    o = oracle.verify(x.draft, x.target, x.tokens, x.uniforms, dtype=x.dtype, mode=x.mode,
                      temperature=x.temperature, alpha=x.alpha, beta=x.beta)
    L, nxt = L.cpu().numpy(), nxt.cpu().numpy()
    sure = (o.accept_margin > 1e-5) & (o.cdf_margin > 1e-5) & (o.accepted_len >= 0) & ~o.fallback
    assert sure.sum() >= len(sure) // 2, (name, int(sure.sum()))
    assert np.array_equal(L[sure], o.accepted_len[sure]), (name, L[sure], o.accepted_len[sure])
    assert np.array_equal(nxt[sure], o.next_token[sure]), (name, nxt[sure], o.next_token[sure])
