"""Verification calls captured into a HIP graph and replayed.

A captured call must give, on every replay, exactly what the same call gives
eagerly (the step is deterministic: every reduction has a fixed order).  The
replays are interleaved with eager work of the program, including eager calls
that share the workspace, and with synchronisations."""
import numpy as np
import pytest
import torch

from paper_2406_11016_amd import binding
from paper_2406_11016_amd import workloads as W
from tests.gpu_util import run_oracle

pytestmark = pytest.mark.gpu

CASES = [
    ("exact_b1_g5_v51865_f32", {}),
    ("exact_b1_g10_v32000_f16", {}),
    ("exact_b64_g8_v128256_bf16", dict(batch=8, vocab=20011)),
    ("sigmoid_b32_g10_v50272_f16_t0.7", dict(batch=8, vocab=10007)),
]


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    binding.load_library()
    torch.cuda.init()


@pytest.mark.parametrize("name,over", CASES, ids=[c[0] for c in CASES])
def test_graph_replays_match_eager(name, over):
    w = W.WORKLOADS[name].with_(**over)
    dev = torch.device("cuda:0")
    xs = [W.generate(w, seed=w.seed * 10 + k) for k in range(3)]
    ins = [binding.to_device(x, dev) for x in xs]
    ws = binding.new_workspace(w.batch, w.gamma, w.vocab, ins[0][0].dtype, dev)
    kw = dict(mode=w.mode, temperature=w.temperature, alpha=w.alpha, beta=w.beta)

    eager = []
    for d, t, tok, u in ins:
        a, n = binding.verify(d, t, tok, u, workspace=ws, **kw)
        eager.append((a.clone(), n.clone()))
    torch.cuda.synchronize()
    # the eager results are the oracle's (decisions away from thresholds)
    for x, (a, n) in zip(xs, eager):
        o = run_oracle(x)
        ok = ~o.flagged(1e-6)
        assert np.array_equal(a.cpu().numpy()[ok], o.accepted_len[ok]), name
        assert np.array_equal(n.cpu().numpy()[ok], o.next_token[ok]), name

    outs = [(torch.empty(w.batch, dtype=torch.int32, device=dev),
             torch.empty(w.batch, dtype=torch.int32, device=dev)) for _ in ins]
    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        for (d, t, tok, u), (a, n) in zip(ins, outs):
            binding.verify(d, t, tok, u, accepted_len=a, next_token=n, workspace=ws, **kw)
    torch.cuda.synchronize()

    for rep in range(4):
        for a, n in outs:
            a.fill_(-7)
            n.fill_(-7)
        g.replay()
        torch.cuda.synchronize()
        for k, ((a, n), (ea, en)) in enumerate(zip(outs, eager)):
            assert torch.equal(a, ea), (name, rep, k, a.cpu(), ea.cpu())
            assert torch.equal(n, en), (name, rep, k, n.cpu(), en.cpu())
        # eager work between the replays, on the same workspace
        d, t, tok, u = ins[rep % len(ins)]
        a2, n2 = binding.verify(d, t, tok, u, workspace=ws, **kw)
        junk = torch.randn(1 << 20, device=dev).sum()
        torch.cuda.synchronize()
        assert torch.equal(a2, eager[rep % len(ins)][0]) and torch.equal(n2, eager[rep % len(ins)][1]), name
        assert torch.isfinite(junk)
    print(f"[graph] {name}: B={w.batch} gamma={w.gamma} V={w.vocab}: 4 replays of 3 captured calls match",
          flush=True)
