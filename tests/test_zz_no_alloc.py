"""The allocation-free entry point spec_verify_exact_static (the library's
static per-GPU workspace) gives spec_verify_exact's outputs, bit for bit, on
two calls in a row (the second with smaller inputs), and rejects sizes past
its workspace before launching anything."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2406_11016_amd import binding
from paper_2406_11016_amd import workloads as W
from tests.gpu_util import run_oracle

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    binding.load_library()
    torch.cuda.init()


def _both(x, dev):
    d, t, tok, u = binding.to_device(x, dev)
    acc, nxt = binding.verify(d, t, tok, u, mode="exact", temperature=x.temperature)
    sacc = torch.full((x.batch,), 0x5eed, dtype=torch.int32, device=dev)
    snxt = torch.full((x.batch,), 0x5eed, dtype=torch.int32, device=dev)
    binding.verify_static(d, t, tok, u, sacc, snxt, temperature=x.temperature)
    torch.cuda.synchronize()
    return (acc.cpu().numpy(), nxt.cpu().numpy()), (sacc.cpu().numpy(), snxt.cpu().numpy())


def test_static_workspace_matches_the_allocating_entry_point():
    dev = torch.device("cuda:0")
    big = W.small_case(16, 8, 40000, "bf16", seed=91, noise_scale=1.0)
    small = W.small_case(3, 2, 999, "f32", seed=92, noise_scale=1.0)
    for label, x in (("first, larger", big), ("second, smaller", small), ("third, larger again", big)):
        print(f"[no-alloc] {label}: B={x.batch} gamma={x.gamma} V={x.vocab} {x.dtype}", flush=True)
        ref, got = _both(x, dev)
        assert np.array_equal(ref[0], got[0]) and np.array_equal(ref[1], got[1]), (label, ref, got)
        o = run_oracle(x)
        ok = ~o.flagged(1e-6)
        assert np.array_equal(got[0][ok], o.accepted_len[ok]) and np.array_equal(got[1][ok], o.next_token[ok])


def test_static_workspace_reset_and_size_limit():
    dev = torch.device("cuda:0")
    x = W.small_case(4, 5, 3001, "f16", seed=93)
    d, t, tok, u = binding.to_device(x, dev)
    acc = torch.empty(4, dtype=torch.int32, device=dev)
    nxt = torch.empty(4, dtype=torch.int32, device=dev)
    binding.verify_static(d, t, tok, u, acc, nxt, reset=True)
    a1, n1 = acc.cpu().numpy(), nxt.cpu().numpy()
    binding.verify_static(d, t, tok, u, acc, nxt)
    assert np.array_equal(a1, acc.cpu().numpy()) and np.array_equal(n1, nxt.cpu().numpy())
    # a size whose workspace exceeds the static array: rejected before any launch
    lib = binding.load_library()
    B, g, V = 4096, 5, 50000
    assert lib.spec_verify_workspace_bytes(B, g, V, binding.SV_F16) > binding.STATIC_WORKSPACE_BYTES
    st = lib.spec_verify_exact_static(0x1000, 0x2000, binding.SV_F16, 0x3000, 0x4000, B, g, V, ctypes.c_float(1.0),
                                      0x5000, 0x6000, 0, None)
    assert st == -5, st   # SV_ERR_WORKSPACE
