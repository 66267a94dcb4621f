"""Python binding of ``libspec_verify.so`` (ctypes; argument marshalling only).

Every step of the verification runs in the library's HIP kernels.  PyTorch is
used for device memory and streams: tensors are passed as raw device pointers
together with the current HIP stream.  There is no fallback: if the library
is missing or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "libspec_verify.so")

SV_F32, SV_F16, SV_BF16 = 0, 1, 2
DTYPE_CODES = {torch.float32: SV_F32, torch.float16: SV_F16, torch.bfloat16: SV_BF16}
STORAGE_TORCH_DTYPES = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
MAX_GAMMA = 128
SV_ERR_TIMEOUT = -8
ERROR_FLAG_OFFSET = 4     # workspace header: the sticky error flag (int32)
SPIN_LIMIT_OFFSET = 8     # workspace header: bound on each wait in polls, 0 = default (a test hook)

SYMBOLS = (
    "spec_verify_workspace_bytes",
    "spec_verify_workspace_init",
    "spec_verify_workspace_check",
    "spec_verify_exact",
    "spec_verify_exact_early_exit",
    "spec_verify_exact_static",
    "spec_verify_sigmoid",
    "spec_verify_exact_probe",
    "spec_verify_sigmoid_probe",
    "spec_verify_exact_ragged",
    "spec_verify_sigmoid_ragged",
    "spec_verify_loop_create",
    "spec_verify_loop_step",
    "spec_verify_loop_destroy",
    "spec_verify_loop_last_early_exit",
    "spec_verify_status_string",
)


class SpecVerifyError(RuntimeError):
    pass


class WorkspaceTimeoutError(SpecVerifyError):
    """The workspace's error flag is set: a wait between workgroups timed out."""


_lib = None


class LoopDesc(ctypes.Structure):
    """``sv_loop_desc_t`` of the decoding loop (see spec_verify.h)."""
    _fields_ = [("mode", ctypes.c_int32), ("dtype", ctypes.c_int), ("batch", ctypes.c_int32),
                ("gamma_max", ctypes.c_int32), ("vocab", ctypes.c_int32), ("temperature", ctypes.c_float),
                ("alpha", ctypes.c_float), ("beta", ctypes.c_float), ("draft", ctypes.c_void_p),
                ("target", ctypes.c_void_p), ("tokens", ctypes.c_void_p), ("uniforms", ctypes.c_void_p),
                ("accepted_len", ctypes.c_void_p), ("next_token", ctypes.c_void_p), ("host_out", ctypes.c_void_p),
                ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t), ("stream", ctypes.c_void_p),
                ("use_graphs", ctypes.c_int32), ("early_exit", ctypes.c_int32)]

_vp = ctypes.c_void_p
_i32 = ctypes.c_int32
_f32 = ctypes.c_float
_sz = ctypes.c_size_t


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise SpecVerifyError(
            f"{path} is missing: build it with `python -c 'import __graft_entry__ as g; g.build()'` "
            "or `python paper_2406_11016_amd/build.py`")
    lib = ctypes.CDLL(path)
    lib.spec_verify_workspace_bytes.argtypes = [_i32, _i32, _i32, ctypes.c_int]
    lib.spec_verify_workspace_bytes.restype = _sz
    lib.spec_verify_workspace_init.argtypes = [_vp, _sz, _vp]
    lib.spec_verify_workspace_init.restype = ctypes.c_int
    lib.spec_verify_workspace_check.argtypes = [_vp, _sz, _vp]
    lib.spec_verify_workspace_check.restype = ctypes.c_int
    common = [_vp, _vp, ctypes.c_int, _vp, _vp, _i32, _i32, _i32, _f32]
    outs = [_vp, _vp, _vp, _sz, _vp]
    lib.spec_verify_exact.argtypes = common + outs
    lib.spec_verify_exact.restype = ctypes.c_int
    lib.spec_verify_exact_early_exit.argtypes = common + outs
    lib.spec_verify_exact_early_exit.restype = ctypes.c_int
    lib.spec_verify_exact_static.argtypes = common + [_vp, _vp, _i32, _vp]
    lib.spec_verify_exact_static.restype = ctypes.c_int
    lib.spec_verify_sigmoid.argtypes = common + [_f32, _f32] + outs
    lib.spec_verify_sigmoid.restype = ctypes.c_int
    lib.spec_verify_exact_probe.argtypes = common + outs + [_vp, _vp, _vp, _vp]
    lib.spec_verify_exact_probe.restype = ctypes.c_int
    lib.spec_verify_sigmoid_probe.argtypes = common + [_f32, _f32] + outs + [_vp, _vp, _vp]
    lib.spec_verify_sigmoid_probe.restype = ctypes.c_int
    ragged = [_vp, _vp, ctypes.c_int, _vp, _vp, _vp, _i32, _i32, _i32, _f32]
    lib.spec_verify_exact_ragged.argtypes = ragged + outs
    lib.spec_verify_exact_ragged.restype = ctypes.c_int
    lib.spec_verify_sigmoid_ragged.argtypes = ragged + [_f32, _f32] + outs
    lib.spec_verify_sigmoid_ragged.restype = ctypes.c_int
    lib.spec_verify_loop_create.argtypes = [ctypes.POINTER(LoopDesc), ctypes.POINTER(ctypes.c_void_p)]
    lib.spec_verify_loop_create.restype = ctypes.c_int
    lib.spec_verify_loop_step.argtypes = [_vp, _i32, ctypes.POINTER(ctypes.c_int32)]
    lib.spec_verify_loop_step.restype = ctypes.c_int
    lib.spec_verify_loop_destroy.argtypes = [_vp]
    lib.spec_verify_loop_destroy.restype = ctypes.c_int
    lib.spec_verify_loop_last_early_exit.argtypes = [_vp]
    lib.spec_verify_loop_last_early_exit.restype = ctypes.c_int32
    lib.spec_verify_status_string.argtypes = [ctypes.c_int]
    lib.spec_verify_status_string.restype = ctypes.c_char_p
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().spec_verify_status_string(status).decode()


def _check(status: int, what: str) -> None:
    if status != 0:
        cls = WorkspaceTimeoutError if status == SV_ERR_TIMEOUT else SpecVerifyError
        raise cls(f"{what}: {status_string(status)} (status {status})")


def workspace_bytes(batch: int, gamma: int, vocab: int, dtype) -> int:
    code = DTYPE_CODES[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    n = load_library().spec_verify_workspace_bytes(batch, gamma, vocab, code)
    if n == 0:
        raise SpecVerifyError(f"invalid sizes: batch={batch} gamma={gamma} vocab={vocab}")
    return int(n)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


# the current stream's raw handle; torch's private accessor skips building a
# Stream object (about 2 us per call), with the public path as the fallback
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream(device) -> int:
    index = device.index if device.index is not None else torch.cuda.current_device()
    if _raw_stream is not None:
        return _raw_stream(index)
    return torch.cuda.current_stream(device).cuda_stream


def new_workspace(batch: int, gamma: int, vocab: int, dtype, device) -> torch.Tensor:
    """A zero-filled workspace for these sizes (reusable across ordered calls;
    each call leaves it zero-filled)."""
    n = workspace_bytes(batch, gamma, vocab, dtype)
    return torch.zeros((n + 15) // 16 * 16, dtype=torch.uint8, device=device)


def init_workspace(ws: torch.Tensor) -> None:
    """Zero-fill a workspace on the current stream (e.g. after a timed-out wait)."""
    lib = load_library()
    nbytes = ws.numel() * ws.element_size()
    _check(lib.spec_verify_workspace_init(_ptr(ws), nbytes // 16 * 16, _stream(ws.device)),
           "spec_verify_workspace_init")


def check_workspace(ws: torch.Tensor) -> None:
    """Wait for the current stream and raise WorkspaceTimeoutError if the
    workspace's error flag is set (spec_verify_workspace_check)."""
    lib = load_library()
    _check(lib.spec_verify_workspace_check(_ptr(ws), ws.numel() * ws.element_size(), _stream(ws.device)),
           "spec_verify_workspace_check")


@dataclass
class Probe:
    tau: torch.Tensor          # [B, gamma] fp64
    weights: torch.Tensor      # [B, V] fp32 (unnormalised a(x))
    mass: torch.Tensor         # [B] fp64
    lognorm: Optional[torch.Tensor] = None  # [B, 2 gamma + 1] fp64 (exact mode)


def _validate(draft, target, tokens, uniforms):
    dev = draft.get_device()  # -1 for host tensors
    for name, t in (("draft", draft), ("target", target), ("tokens", tokens), ("uniforms", uniforms)):
        if not t.is_cuda:
            raise SpecVerifyError(f"{name} must be a device tensor")
        if not t.is_contiguous():
            raise SpecVerifyError(f"{name} must be contiguous")
        if t.get_device() != dev:
            raise SpecVerifyError(f"{name} is on {t.device}, draft on {draft.device}")
    if draft.dtype not in DTYPE_CODES or target.dtype != draft.dtype:
        raise SpecVerifyError(f"logits must share one of {list(DTYPE_CODES)}; got {draft.dtype}/{target.dtype}")
    if draft.dim() != 3 or target.dim() != 3:
        raise SpecVerifyError("logits must be [B, gamma, V] and [B, gamma+1, V]")
    B, g, V = draft.shape
    if tuple(target.shape) != (B, g + 1, V):
        raise SpecVerifyError(f"target shape {tuple(target.shape)} != {(B, g + 1, V)}")
    if tokens.dtype != torch.int32 or tuple(tokens.shape) != (B, g):
        raise SpecVerifyError("tokens must be int32 [B, gamma]")
    if uniforms.dtype != torch.float32 or tuple(uniforms.shape) != (B, g + 1):
        raise SpecVerifyError("uniforms must be float32 [B, gamma+1]")
    return B, g, V


def verify(draft: torch.Tensor, target: torch.Tensor, tokens: torch.Tensor, uniforms: torch.Tensor, *,
           mode: str = "exact", temperature: float = 1.0, alpha: float = -1.0e4, beta: float = 1.0e4,
           accepted_len: Optional[torch.Tensor] = None, next_token: Optional[torch.Tensor] = None,
           workspace: Optional[torch.Tensor] = None, probe: bool = False, gammas: Optional[torch.Tensor] = None,
           early_exit: bool = False, check: bool = False):
    """One verification step on the current stream.

    Returns ``(accepted_len, next_token)`` (int32 [B] device tensors), plus a
    :class:`Probe` when ``probe`` is true.  ``workspace`` (zero-filled before
    its first use) may be passed to avoid an allocation per call.  ``gammas``
    (int32 [B] device tensor) selects the ragged variant: element b uses its
    first ``gammas[b]`` drafts of the padded tensors (no probes).
    ``early_exit`` (exact mode, no probes, not ragged) selects
    ``spec_verify_exact_early_exit``: the same outputs, skipping most rows
    after each element's first rejection.  ``check`` waits for the stream
    after the call and raises :class:`WorkspaceTimeoutError` if the
    workspace's error flag is set (see :func:`check_workspace`).
    """
    if mode not in ("exact", "sigmoid"):
        raise ValueError(mode)
    if early_exit and (mode != "exact" or probe or gammas is not None):
        raise SpecVerifyError("the early exit is an exact-mode variant without probes or ragged gammas")
    lib = _lib if _lib is not None else load_library()
    B, g, V = _validate(draft, target, tokens, uniforms)
    dev = draft.device
    di = draft.get_device()
    if gammas is not None:
        if probe:
            raise SpecVerifyError("the ragged variant has no probes")
        if gammas.get_device() != di or gammas.dtype != torch.int32 or tuple(gammas.shape) != (B,) or \
                not gammas.is_contiguous():
            raise SpecVerifyError(f"gammas must be a contiguous int32 [{B}] tensor on {dev}")
    if accepted_len is None:
        accepted_len = torch.empty(B, dtype=torch.int32, device=dev)
    if next_token is None:
        next_token = torch.empty(B, dtype=torch.int32, device=dev)
    for name, t in (("accepted_len", accepted_len), ("next_token", next_token)):
        # the kernel writes B entries: anything else would be written out of bounds
        if t.dtype != torch.int32 or tuple(t.shape) != (B,) or not t.is_contiguous() or t.get_device() != di:
            raise SpecVerifyError(f"{name} must be a contiguous int32 [{B}] tensor on {dev}")
    if workspace is None:
        workspace = new_workspace(B, g, V, draft.dtype, dev)
    elif not workspace.is_contiguous() or workspace.get_device() != di:
        raise SpecVerifyError(f"workspace must be a contiguous tensor on {dev}")
    code = DTYPE_CODES[draft.dtype]
    head = [_ptr(draft), _ptr(target), code, _ptr(tokens), _ptr(uniforms), B, g, V, float(temperature)]
    tail = [_ptr(accepted_len), _ptr(next_token), _ptr(workspace), workspace.numel() * workspace.element_size(),
            _stream(dev)]
    if gammas is not None:
        rhead = [_ptr(draft), _ptr(target), code, _ptr(tokens), _ptr(uniforms), _ptr(gammas), B, g, V,
                 float(temperature)]
        if mode == "exact":
            st = lib.spec_verify_exact_ragged(*rhead, *tail)
        else:
            st = lib.spec_verify_sigmoid_ragged(*rhead, float(alpha), float(beta), *tail)
        _check(st, f"spec_verify_{mode}_ragged")
        if check:
            check_workspace(workspace)
        return accepted_len, next_token
    pr = None
    if probe:
        pr = Probe(tau=torch.full((B, g), float("nan"), dtype=torch.float64, device=dev),
                   weights=torch.zeros((B, V), dtype=torch.float32, device=dev),
                   mass=torch.full((B,), float("nan"), dtype=torch.float64, device=dev),
                   lognorm=(torch.full((B, 2 * g + 1), float("nan"), dtype=torch.float64, device=dev)
                            if mode == "exact" else None))
    if mode == "exact":
        if probe:
            st = lib.spec_verify_exact_probe(*head, *tail, _ptr(pr.tau), _ptr(pr.weights), _ptr(pr.mass),
                                             _ptr(pr.lognorm))
        elif early_exit:
            st = lib.spec_verify_exact_early_exit(*head, *tail)
        else:
            st = lib.spec_verify_exact(*head, *tail)
    else:
        ab = [float(alpha), float(beta)]
        if probe:
            st = lib.spec_verify_sigmoid_probe(*head, *ab, *tail, _ptr(pr.tau), _ptr(pr.weights), _ptr(pr.mass))
        else:
            st = lib.spec_verify_sigmoid(*head, *ab, *tail)
    _check(st, "spec_verify_exact_early_exit" if early_exit else f"spec_verify_{mode}")
    if check:
        check_workspace(workspace)
    return (accepted_len, next_token, pr) if probe else (accepted_len, next_token)


STATIC_WORKSPACE_BYTES = 8 << 20


def verify_static(draft: torch.Tensor, target: torch.Tensor, tokens: torch.Tensor, uniforms: torch.Tensor,
                  accepted_len: torch.Tensor, next_token: torch.Tensor, *, temperature: float = 1.0,
                  reset: bool = False) -> None:
    """spec_verify_exact_static on the current stream: the exact-mode step
    with the library's static per-GPU workspace (no allocation anywhere; the
    caller provides the outputs)."""
    lib = _lib if _lib is not None else load_library()
    B, g, V = _validate(draft, target, tokens, uniforms)
    di = draft.get_device()
    for name, t in (("accepted_len", accepted_len), ("next_token", next_token)):
        if t.dtype != torch.int32 or tuple(t.shape) != (B,) or not t.is_contiguous() or t.get_device() != di:
            raise SpecVerifyError(f"{name} must be a contiguous int32 [{B}] tensor on {draft.device}")
    st = lib.spec_verify_exact_static(_ptr(draft), _ptr(target), DTYPE_CODES[draft.dtype], _ptr(tokens),
                                      _ptr(uniforms), B, g, V, float(temperature), _ptr(accepted_len),
                                      _ptr(next_token), 1 if reset else 0, _stream(draft.device))
    _check(st, "spec_verify_exact_static")


def to_device(inputs, device="cuda"):
    """Upload generator output (host NumPy arrays in storage form) to device tensors."""
    import numpy as np
    tdt = STORAGE_TORCH_DTYPES[inputs.dtype]
    if inputs.dtype == "bf16":
        d = torch.from_numpy(np.ascontiguousarray(inputs.draft).view(np.int16)).view(torch.bfloat16)
        t = torch.from_numpy(np.ascontiguousarray(inputs.target).view(np.int16)).view(torch.bfloat16)
    else:
        d = torch.from_numpy(np.ascontiguousarray(inputs.draft))
        t = torch.from_numpy(np.ascontiguousarray(inputs.target))
    assert d.dtype == tdt
    return (d.to(device), t.to(device),
            torch.from_numpy(np.ascontiguousarray(inputs.tokens)).to(device),
            torch.from_numpy(np.ascontiguousarray(inputs.uniforms)).to(device))


def loop_create(desc: LoopDesc) -> ctypes.c_void_p:
    """A native decoding loop over the caller's buffers (spec_verify_loop_create)."""
    h = ctypes.c_void_p()
    _check(load_library().spec_verify_loop_create(ctypes.byref(desc), ctypes.byref(h)), "spec_verify_loop_create")
    return h


def loop_step(handle: ctypes.c_void_p, gamma: int) -> int:
    """One iteration of the native loop (waits for it); returns the next gamma."""
    nxt = ctypes.c_int32()
    _check(load_library().spec_verify_loop_step(handle, int(gamma), ctypes.byref(nxt)), "spec_verify_loop_step")
    return int(nxt.value)


def loop_last_early_exit(handle: ctypes.c_void_p) -> int:
    """Whether the native loop's last step ran the early exit (1), the single pass (0), or no step yet (-1)."""
    return int(load_library().spec_verify_loop_last_early_exit(handle))


def loop_destroy(handle: ctypes.c_void_p) -> None:
    _check(load_library().spec_verify_loop_destroy(handle), "spec_verify_loop_destroy")
