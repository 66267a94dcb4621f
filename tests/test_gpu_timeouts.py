"""Timed-out waits between workgroups are visible and safe (the "Timed-out
waits" contract of include/spec_verify.h), and the step stays correct while
other work runs on the GPU.

The timeout path is forced from the host, never by a fault: either the
workspace's sticky error flag is set before a call (as a timed-out wait of an
earlier call would leave it), or the workspace header's spin-limit word makes
every wait give up after one poll, so that every kernel still exits
normally."""
import numpy as np
import pytest
import torch

from paper_2406_11016_amd import binding
from paper_2406_11016_amd import workloads as W
from paper_2406_11016_amd.decode_loop import DecodeLoop, SyntheticSteps
from tests.gpu_util import run_oracle

pytestmark = pytest.mark.gpu

FLAG = binding.ERROR_FLAG_OFFSET
SPIN = binding.SPIN_LIMIT_OFFSET


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    binding.load_library()
    torch.cuda.init()


def _set_word(ws, offset, value):
    ws[offset:offset + 4].view(torch.int32).fill_(value)
    torch.cuda.synchronize()


def _word(ws, offset):
    torch.cuda.synchronize()
    return int(ws[offset:offset + 4].view(torch.int32).item())


CASES = [
    # (batch, gamma, vocab, dtype, mode, early_exit)
    (8, 8, 20011, "bf16", "exact", False),
    (3, 5, 9001, "f32", "exact", False),
    (4, 6, 3001, "f16", "sigmoid", False),
    (56, 3, 128256, "bf16", "exact", True),  # gated (gate 2 < gamma): the row-staged kernel
]
IDS = [f"{c[4]}-B{c[0]}-{c[3]}" + ("-early" if c[5] else "") for c in CASES]


def _inputs(c, seed):
    B, g, V, dt, mode, _ = c
    return W.small_case(B, g, V, dt, mode=mode, seed=seed, noise_scale=0.5, temperature=0.8, alpha=-1e3, beta=1e3)


def _call(x, dev, ws, early, **kw):
    d, t, tok, u = binding.to_device(x, dev)
    acc, nxt = binding.verify(d, t, tok, u, mode=x.mode, temperature=x.temperature, alpha=x.alpha, beta=x.beta,
                              workspace=ws, early_exit=early, **kw)
    torch.cuda.synchronize()
    return acc.cpu().numpy(), nxt.cpu().numpy()


def _reference(x, dev):
    """The expected outputs and the elements they bind: the oracle's, or for
    the large gated shape the single pass's on a fresh workspace (the single
    pass itself is checked against the oracle by the parity tests)."""
    if x.batch * (2 * x.gamma + 1) * x.vocab > 5e6:
        ws = binding.new_workspace(x.batch, x.gamma, x.vocab, binding.STORAGE_TORCH_DTYPES[x.dtype], dev)
        acc, nxt = _call(x, dev, ws, False, check=True)
        return acc, nxt, np.ones(x.batch, dtype=bool)
    o = run_oracle(x)
    return o.accepted_len, o.next_token, ~o.flagged(1e-6)


def _assert_ref(ref, acc, nxt, label):
    ra, rn, ok = ref
    assert np.array_equal(acc[ok], ra[ok]), (label, acc, ra)
    assert np.array_equal(nxt[ok], rn[ok]), (label, nxt, rn)


@pytest.mark.parametrize("case", CASES, ids=IDS)
def test_sticky_flag_makes_every_output_a_sentinel_until_reinitialised(case):
    dev = torch.device("cuda:0")
    x = _inputs(case, seed=11)
    ws = binding.new_workspace(x.batch, x.gamma, x.vocab, binding.STORAGE_TORCH_DTYPES[x.dtype], dev)
    _set_word(ws, FLAG, 1)
    print(f"[timeouts] sticky flag {IDS[CASES.index(case)]}", flush=True)
    with pytest.raises(binding.WorkspaceTimeoutError):
        _call(x, dev, ws, case[5], check=True)
    acc, nxt = _call(x, dev, ws, case[5])
    assert np.all(acc == -1) and np.all(nxt == -1), (acc, nxt)
    with pytest.raises(binding.WorkspaceTimeoutError):
        binding.check_workspace(ws)
    # the workspace stays usable after it is zero-filled again
    binding.init_workspace(ws)
    acc, nxt = _call(x, dev, ws, case[5], check=True)
    _assert_ref(_reference(x, dev), acc, nxt, "after re-initialisation")
    assert torch.count_nonzero(ws).item() == 0


@pytest.mark.parametrize("case", CASES, ids=IDS)
def test_waits_that_give_up_set_the_flag_and_every_wave_exits(case):
    """Every wait gives up after one poll: the kernel exits, the flag is set,
    every output is written (-1 or a value in its range), and a call without
    a timed-out wait is the oracle's."""
    dev = torch.device("cuda:0")
    x = _inputs(case, seed=12)
    d, t, tok, u = binding.to_device(x, dev)
    ws = binding.new_workspace(x.batch, x.gamma, x.vocab, d.dtype, dev)
    acc = torch.empty(x.batch, dtype=torch.int32, device=dev)
    nxt = torch.empty(x.batch, dtype=torch.int32, device=dev)
    ref = _reference(x, dev)
    gave_up = 0
    for rep in range(3):
        binding.init_workspace(ws)
        _set_word(ws, SPIN, 1)
        acc.fill_(0x5eed)
        nxt.fill_(0x5eed)
        print(f"[timeouts] spin limit 1 {IDS[CASES.index(case)]} rep {rep}", flush=True)
        binding.verify(d, t, tok, u, mode=x.mode, temperature=x.temperature, alpha=x.alpha, beta=x.beta,
                       accepted_len=acc, next_token=nxt, workspace=ws, early_exit=case[5])
        torch.cuda.synchronize()
        a, n = acc.cpu().numpy(), nxt.cpu().numpy()
        flag = _word(ws, FLAG)
        assert np.all((a == -1) | ((a >= 0) & (a <= x.gamma))), a
        assert np.all((n == -1) | ((n >= 0) & (n < x.vocab))), n
        if flag == 0:
            _assert_ref(ref, a, n, "no wait gave up")
        else:
            gave_up += 1
    # with every wait limited to one poll, some wait gives up
    assert gave_up >= 1
    # the workspace is dirty after such a call; zero-filled, it works again
    binding.init_workspace(ws)
    a2, n2 = _call(x, dev, ws, case[5], check=True)
    _assert_ref(ref, a2, n2, "after re-initialisation")


@pytest.mark.parametrize("native", [False, True], ids=["python-loop", "native-loop"])
def test_decoding_loop_reports_the_flag(native):
    w = W.Workload("loop_flag", "exact", 2, 5, 3001, "f32", "normal", 2.0, 0.3, seed=77)
    src = SyntheticSteps(w, gamma_max=8, pool=2)
    loop = DecodeLoop(w.batch, w.vocab, w.dtype, gamma0=5, gamma_max=8, native=native)
    try:
        loop.run(src, 2)
        _set_word(loop.ws, FLAG, 1)
        with pytest.raises(binding.WorkspaceTimeoutError if native else binding.SpecVerifyError):
            loop.run(src, 1)
        loop.reset_workspace()
        st = loop.run(src, 2)
        assert st.iterations == 2 and all(np.all(a >= 0) for a in st.accepted)
    finally:
        loop.close()


def test_correct_while_a_copy_runs_on_another_stream():
    """The step's workgroups wait only on workgroups dispatched before them;
    a bandwidth-heavy copy on a second stream (default priority) shares the
    GPU with the calls: every call matches the oracle and no wait times out."""
    dev = torch.device("cuda:0")
    w = W.WORKLOADS[W.HEADLINE]
    x = W.generate(w.with_(batch=16))
    d, t, tok, u = binding.to_device(x, dev)
    ws = binding.new_workspace(x.batch, x.gamma, x.vocab, d.dtype, dev)
    acc = torch.empty(x.batch, dtype=torch.int32, device=dev)
    nxt = torch.empty(x.batch, dtype=torch.int32, device=dev)
    src = torch.ones(256 << 20, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    side = torch.cuda.Stream(dev)
    o = run_oracle(x)
    ok = ~o.flagged(1e-6)
    torch.cuda.synchronize()
    for rep in range(10):
        with torch.cuda.stream(side):
            for _ in range(4):
                dst.copy_(src)
        outs = []
        for _ in range(20):
            binding.verify(d, t, tok, u, accepted_len=acc, next_token=nxt, workspace=ws)
            outs.append((acc.clone(), nxt.clone()))
        torch.cuda.synchronize()
        binding.check_workspace(ws)
        for a, n in outs:
            a, n = a.cpu().numpy(), n.cpu().numpy()
            assert np.array_equal(a[ok], o.accepted_len[ok]) and np.array_equal(n[ok], o.next_token[ok]), rep
    assert torch.equal(dst[:16], src[:16])
