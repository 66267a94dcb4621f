"""The C ABI on the host: the library loads, exports every function the header
declares, sizes its workspace, and rejects invalid arguments before launching
anything (none of these calls reaches the GPU)."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2406_11016_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "spec_verify.h")

SV_OK, SV_ERR_NULL, SV_ERR_SHAPE, SV_ERR_DTYPE, SV_ERR_PARAM, SV_ERR_WORKSPACE = 0, -1, -2, -3, -4, -5
SV_ERR_TIMEOUT = -8


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(spec_verify_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(binding.LIB_PATH):
        pytest.fail("libspec_verify.so not built; run __graft_entry__.build()")
    return binding.load_library()


def test_header_declares_the_boundary():
    fns = declared_functions()
    assert fns == sorted(binding.SYMBOLS), fns


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", binding.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT (spec_verify_\w+)", out))
    for fn in declared_functions():
        assert fn in exported, fn
        assert getattr(lib, fn) is not None


def test_status_strings(lib):
    for st in (0, -1, -2, -3, -4, -5, -6, -7, -8):
        assert binding.status_string(st) and binding.status_string(st) != "unknown status"
    assert binding.status_string(0) == "ok"
    assert "timed out" in binding.status_string(SV_ERR_TIMEOUT)
    assert "unknown" in binding.status_string(7)


def test_workspace_check_validates_before_touching_the_gpu(lib):
    f = lib.spec_verify_workspace_check
    assert f(None, 4096, None) == SV_ERR_NULL
    assert f(0x7008, 4096, None) == SV_ERR_WORKSPACE    # not 16-byte aligned
    assert f(0x7000, 255, None) == SV_ERR_WORKSPACE     # smaller than the header


def test_out_of_range_dtype_codes_are_rejected(lib):
    for code in (3, 7, -1, 1 << 30):
        assert lib.spec_verify_workspace_bytes(2, 3, 100, code) == 0
        assert _exact(lib, _args(dtype=code)) == SV_ERR_DTYPE
        assert _sigmoid(lib, _args(dtype=code)) == SV_ERR_DTYPE


def test_workspace_bytes(lib):
    f = lib.spec_verify_workspace_bytes
    for args in [(1, 5, 51865, 0), (64, 8, 128256, 2), (32, 10, 50272, 1), (1, 1, 1, 0), (3, 128, 7, 1)]:
        n = f(*args)
        assert n > 0 and n % 256 == 0
    assert f(64, 8, 128256, 2) >= 64 * 17 * 16       # at least one normaliser partial per row
    for bad in [(0, 5, 100, 0), (1, 0, 100, 0), (1, 129, 100, 0), (1, 5, 0, 0), (1, 5, 100, 3), (-1, 5, 100, 0)]:
        assert f(*bad) == 0


def test_workspace_bytes_small_batches_large_vocabularies(lib):
    """Every batch size plans the largest vocabularies the header allows
    (2^20 fp32, 2^21 fp16/bf16) and rejects the next size up."""
    f = lib.spec_verify_workspace_bytes
    for B in (1, 2, 3, 5, 17, 64):
        for gamma in (1, 8, 128):
            for V, dt in ((300007, 0), (1 << 20, 0), (600011, 2), (1 << 21, 1), (1 << 21, 2)):
                assert f(B, gamma, V, dt) > 0, (B, gamma, V, dt)
            assert f(B, gamma, (1 << 20) + 1, 0) == 0
            assert f(B, gamma, (1 << 21) + 1, 2) == 0


def _args(**kw):
    base = dict(draft=0x1000, target=0x2000, dtype=0, tokens=0x3000, uniforms=0x4000, B=2, gamma=3, V=100,
                T=1.0, acc=0x5000, nxt=0x6000, ws=0x7000, ws_bytes=1 << 20, stream=None)
    base.update(kw)
    return base


def _exact(lib, a):
    return lib.spec_verify_exact(a["draft"], a["target"], a["dtype"], a["tokens"], a["uniforms"], a["B"],
                                 a["gamma"], a["V"], a["T"], a["acc"], a["nxt"], a["ws"], a["ws_bytes"], a["stream"])


def _sigmoid(lib, a, alpha=-1e4, beta=1e4):
    return lib.spec_verify_sigmoid(a["draft"], a["target"], a["dtype"], a["tokens"], a["uniforms"], a["B"],
                                   a["gamma"], a["V"], a["T"], alpha, beta, a["acc"], a["nxt"], a["ws"],
                                   a["ws_bytes"], a["stream"])


def _ragged(lib, a, gammas=0x8000, sigmoid=False, alpha=-1e4, beta=1e4):
    head = [a["draft"], a["target"], a["dtype"], a["tokens"], a["uniforms"], gammas, a["B"], a["gamma"], a["V"],
            a["T"]]
    tail = [a["acc"], a["nxt"], a["ws"], a["ws_bytes"], a["stream"]]
    if sigmoid:
        return lib.spec_verify_sigmoid_ragged(*head, alpha, beta, *tail)
    return lib.spec_verify_exact_ragged(*head, *tail)


@pytest.mark.parametrize("field", ["draft", "target", "tokens", "uniforms", "acc", "nxt", "ws"])
def test_null_pointers_rejected(lib, field):
    assert _exact(lib, _args(**{field: None})) == SV_ERR_NULL
    assert _sigmoid(lib, _args(**{field: None})) == SV_ERR_NULL
    assert _ragged(lib, _args(**{field: None})) == SV_ERR_NULL
    assert _ragged(lib, _args(**{field: None}), sigmoid=True) == SV_ERR_NULL


def test_ragged_checks(lib):
    assert _ragged(lib, _args(), gammas=None) == SV_ERR_NULL
    assert _ragged(lib, _args(), gammas=None, sigmoid=True) == SV_ERR_NULL
    assert _ragged(lib, _args(gamma=129)) == SV_ERR_SHAPE
    assert _ragged(lib, _args(T=0.0)) == SV_ERR_PARAM
    assert _ragged(lib, _args(), sigmoid=True, alpha=1.0, beta=1.0) == SV_ERR_PARAM
    need = lib.spec_verify_workspace_bytes(2, 3, 100, 0)
    assert _ragged(lib, _args(ws_bytes=need - 1)) == SV_ERR_WORKSPACE


def test_invalid_shapes_dtype_params_workspace(lib):
    assert _exact(lib, _args(B=0)) == SV_ERR_SHAPE
    assert _exact(lib, _args(gamma=0)) == SV_ERR_SHAPE
    assert _exact(lib, _args(gamma=129)) == SV_ERR_SHAPE
    assert _exact(lib, _args(V=0)) == SV_ERR_SHAPE
    assert _exact(lib, _args(dtype=5)) == SV_ERR_DTYPE
    for T in (0.0, -1.0, float("inf"), float("nan"), 1e-45):
        assert _exact(lib, _args(T=T)) == SV_ERR_PARAM, T
    for alpha, beta in [(1.0, 1.0), (2.0, -2.0), (float("nan"), 1.0), (-1.0, float("inf"))]:
        assert _sigmoid(lib, _args(), alpha, beta) == SV_ERR_PARAM
    need = lib.spec_verify_workspace_bytes(2, 3, 100, 0)
    assert _exact(lib, _args(ws_bytes=need - 1)) == SV_ERR_WORKSPACE
    assert _exact(lib, _args(ws=0x7004)) == SV_ERR_WORKSPACE
    assert lib.spec_verify_workspace_init(None, 256, None) == SV_ERR_NULL
    assert lib.spec_verify_workspace_init(0x7004, 256, None) == SV_ERR_WORKSPACE


def _early_exit(lib, a):
    return lib.spec_verify_exact_early_exit(a["draft"], a["target"], a["dtype"], a["tokens"], a["uniforms"],
                                            a["B"], a["gamma"], a["V"], a["T"], a["acc"], a["nxt"], a["ws"],
                                            a["ws_bytes"], a["stream"])


def test_early_exit_validates_like_the_single_pass(lib):
    need = lib.spec_verify_workspace_bytes(2, 3, 100, 0)
    cases = [dict(B=0), dict(gamma=0), dict(gamma=129), dict(V=0), dict(dtype=5), dict(T=0.0),
             dict(T=float("nan")), dict(ws_bytes=need - 1), dict(ws=0x7004)]
    cases += [{f: None} for f in ("draft", "target", "tokens", "uniforms", "acc", "nxt", "ws")]
    for kw in cases:
        st = _early_exit(lib, _args(**kw))
        assert st != SV_OK and st == _exact(lib, _args(**kw)), (kw, st)


def test_probe_entry_points_validate_too(lib):
    a = _args(B=0)
    st = lib.spec_verify_exact_probe(a["draft"], a["target"], a["dtype"], a["tokens"], a["uniforms"], a["B"],
                                     a["gamma"], a["V"], a["T"], a["acc"], a["nxt"], a["ws"], a["ws_bytes"],
                                     a["stream"], None, None, None, None)
    assert st == SV_ERR_SHAPE
    a = _args(T=-1.0)
    st = lib.spec_verify_sigmoid_probe(a["draft"], a["target"], a["dtype"], a["tokens"], a["uniforms"], a["B"],
                                       a["gamma"], a["V"], a["T"], -10.0, 10.0, a["acc"], a["nxt"], a["ws"],
                                       a["ws_bytes"], a["stream"], None, None, None)
    assert st == SV_ERR_PARAM


def test_no_cpu_fallback_in_binding():
    src = open(os.path.join(ROOT, "paper_2406_11016_amd", "binding.py")).read()
    assert "oracle" not in src
    # the unfused PyTorch comparison is never a fallback of the library
    assert "unfused" not in src
    for f in os.listdir(os.path.join(ROOT, "paper_2406_11016_amd")):
        if f.endswith(".py"):
            assert "import oracle" not in open(os.path.join(ROOT, "paper_2406_11016_amd", f)).read()
            assert "from oracle" not in open(os.path.join(ROOT, "paper_2406_11016_amd", f)).read()


def _loop_desc(**kw):
    d = dict(mode=0, dtype=0, batch=2, gamma_max=6, vocab=100, temperature=1.0, alpha=-1.0, beta=1.0,
             draft=0x1000, target=0x2000, tokens=0x3000, uniforms=0x4000, accepted_len=0x5000, next_token=0x6000,
             host_out=0x7000, workspace=0x8000, workspace_bytes=1 << 22, stream=None, use_graphs=1)
    d.update(kw)
    return binding.LoopDesc(**d)


def test_loop_create_checks(lib):
    """The native decoding loop validates its descriptor before touching the GPU."""
    import ctypes
    h = ctypes.c_void_p()
    assert lib.spec_verify_loop_create(None, ctypes.byref(h)) == SV_ERR_NULL
    for field in ("draft", "target", "tokens", "uniforms", "accepted_len", "next_token", "host_out", "workspace"):
        assert lib.spec_verify_loop_create(ctypes.byref(_loop_desc(**{field: None})), ctypes.byref(h)) == SV_ERR_NULL
    assert lib.spec_verify_loop_create(ctypes.byref(_loop_desc(mode=2)), ctypes.byref(h)) == SV_ERR_PARAM
    for bad in (-1, 3):
        assert lib.spec_verify_loop_create(ctypes.byref(_loop_desc(early_exit=bad)), ctypes.byref(h)) == SV_ERR_PARAM
    assert lib.spec_verify_loop_create(ctypes.byref(_loop_desc(gamma_max=0)), ctypes.byref(h)) == SV_ERR_SHAPE
    assert lib.spec_verify_loop_create(ctypes.byref(_loop_desc(gamma_max=129)), ctypes.byref(h)) == SV_ERR_SHAPE
    need = max(lib.spec_verify_workspace_bytes(2, g, 100, 0) for g in range(1, 7))
    assert lib.spec_verify_loop_create(ctypes.byref(_loop_desc(workspace_bytes=need - 1)),
                                       ctypes.byref(h)) == SV_ERR_WORKSPACE
    # a valid descriptor: the host object only (graphs come with the first step)
    assert lib.spec_verify_loop_create(ctypes.byref(_loop_desc(workspace_bytes=need)), ctypes.byref(h)) == 0
    assert lib.spec_verify_loop_last_early_exit(h) == -1      # no step yet
    assert lib.spec_verify_loop_last_early_exit(None) == -1
    nxt = ctypes.c_int32()
    assert lib.spec_verify_loop_step(h, 0, ctypes.byref(nxt)) == SV_ERR_PARAM
    assert lib.spec_verify_loop_step(h, 7, ctypes.byref(nxt)) == SV_ERR_PARAM
    assert lib.spec_verify_loop_step(None, 3, ctypes.byref(nxt)) == SV_ERR_NULL
    assert lib.spec_verify_loop_destroy(h) == 0
    assert lib.spec_verify_loop_destroy(None) == 0
