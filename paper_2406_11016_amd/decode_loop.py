"""A multi-step decoding loop around the fused verification step.

Each iteration verifies gamma drafted tokens per batch element with one call
of the step and then sets gamma for the next iteration with the draft-length
rule the paper's experiments use (Sec. 4, hyperparameters; the rule of the
assisted-generation baseline it compares with): gamma starts at 5, grows by 2
after an iteration in which every drafted token was accepted and otherwise
shrinks by 1.  Readings where the paper is silent: gamma never drops below 1
nor exceeds ``gamma_max``, and with several batch elements "every drafted
token accepted" must hold for all of them.

The loop owns static device buffers sized for ``gamma_max``.  Whatever
produces the logits (the draft and target models of a decoder; a synthetic
source here) writes an iteration's ``[B, gamma, V]`` / ``[B, gamma + 1, V]``
logits, drafted tokens and uniforms into the leading part of those buffers;
an iteration then costs one launch of the step, three small device-to-host
copies into pinned memory (the accepted lengths, the next tokens and the
workspace's error flag) and one stream synchronisation -- the host needs the
accepted length to decide the next gamma and which tokens to append.  With
``use_graphs`` the call for each gamma is captured once into a HIP graph
(lazily, on first use) and replayed instead; on ROCm 7 that measured slower
than launching this one-kernel step directly, so it is off by default.

In the exact mode ``early_exit`` picks the entry point of each step:
``"never"`` (the single pass), ``"always"`` (the early exit, which stops
streaming an element's rows at its first rejection, Sec. 3.1) or ``"auto"``:
the early exit when the previous step's mean accepted length was below half
of its gamma, the single pass otherwise and at the first step.  Both give
the same outputs.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np
import torch

from . import binding
from .binding import STORAGE_TORCH_DTYPES


def next_gamma(gamma: int, accepted: np.ndarray, gamma_max: int, grow: int = 2, shrink: int = 1) -> int:
    """The draft-length rule: ``gamma + grow`` (at most ``gamma_max``) if every
    element accepted all ``gamma`` drafts, else ``gamma - shrink`` (at least 1).
    Elements with the sentinel (-1) count as not accepted."""
    if accepted.size > 0 and bool(np.all(accepted == gamma)):
        return min(gamma + grow, gamma_max)
    return max(gamma - shrink, 1)


EARLY_EXIT_CODES = {"never": 0, "always": 1, "auto": 2}


def early_exit_pays(accepted: np.ndarray, gamma: int) -> bool:
    """The automatic choice for the next step: the early exit when the mean
    accepted length of the last step (sentinels counting 0) was below half
    of its gamma (the native loop's rule, early_exit_pays in plan.hpp)."""
    return accepted.size > 0 and 2 * int(np.sum(np.maximum(accepted, 0))) < gamma * accepted.size


@dataclass
class LoopStats:
    iterations: int = 0
    tokens: int = 0                                   # accepted drafts + 1 per element and iteration
    gammas: List[int] = field(default_factory=list)
    accepted: List[np.ndarray] = field(default_factory=list)
    next_tokens: List[np.ndarray] = field(default_factory=list)
    device_us: List[float] = field(default_factory=list)   # per iteration, when timed
    early_exit: List[bool] = field(default_factory=list)   # per iteration: the early exit ran


class DecodeLoop:
    """Static buffers, one captured graph per gamma, and the gamma rule."""

    def __init__(self, batch: int, vocab: int, dtype: str, *, mode: str = "exact", temperature: float = 1.0,
                 alpha: float = -1.0e4, beta: float = 1.0e4, gamma0: int = 5, gamma_max: int = 20,
                 use_graphs: bool = False, native: bool = False, early_exit: str = "never",
                 adapt_gamma: bool = True, device="cuda"):
        if not (1 <= gamma0 <= gamma_max):
            raise ValueError("need 1 <= gamma0 <= gamma_max")
        if early_exit not in EARLY_EXIT_CODES:
            raise ValueError(f"early_exit must be one of {sorted(EARLY_EXIT_CODES)}")
        if native and not adapt_gamma:
            raise ValueError("the native loop always applies the gamma rule")
        self.early_exit = early_exit
        self.adapt_gamma = adapt_gamma   # False: every iteration verifies gamma0 drafts (measurements)
        self._early_next = mode == "exact" and early_exit == "always"
        self.B, self.V, self.dtype, self.mode = batch, vocab, dtype, mode
        self.temperature, self.alpha, self.beta = temperature, alpha, beta
        self.gamma0, self.gamma_max, self.use_graphs = gamma0, gamma_max, use_graphs
        self.device = torch.device(device)
        tdt = STORAGE_TORCH_DTYPES[dtype]
        B, G, V = batch, gamma_max, vocab
        self.draft = torch.empty(B * G * V, dtype=tdt, device=self.device)
        self.target = torch.empty(B * (G + 1) * V, dtype=tdt, device=self.device)
        self.tokens = torch.zeros(B * G, dtype=torch.int32, device=self.device)
        self.uniforms = torch.zeros(B * (G + 1), dtype=torch.float32, device=self.device)
        self.acc = torch.empty(B, dtype=torch.int32, device=self.device)
        self.nxt = torch.empty(B, dtype=torch.int32, device=self.device)
        self.host = torch.empty(2 * B, dtype=torch.int32, pin_memory=True)
        self.flag_host = torch.zeros(1, dtype=torch.int32, pin_memory=True)
        ws = max(binding.workspace_bytes(B, g, V, tdt) for g in range(1, G + 1))
        self.ws = torch.zeros((ws + 15) // 16 * 16, dtype=torch.uint8, device=self.device)
        self.stream = torch.cuda.Stream(self.device)
        self.graphs: Dict[Tuple[int, bool], torch.cuda.CUDAGraph] = {}
        # the native loop: one library call per iteration (graph replay or
        # launch, the copies to pinned memory, the wait and the gamma rule)
        self.native = None
        if native:
            desc = binding.LoopDesc(
                mode=0 if mode == "exact" else 1, dtype=binding.DTYPE_CODES[tdt], batch=B, gamma_max=G, vocab=V,
                temperature=temperature, alpha=alpha, beta=beta, draft=self.draft.data_ptr(),
                target=self.target.data_ptr(), tokens=self.tokens.data_ptr(), uniforms=self.uniforms.data_ptr(),
                accepted_len=self.acc.data_ptr(), next_token=self.nxt.data_ptr(), host_out=self.host.data_ptr(),
                workspace=self.ws.data_ptr(), workspace_bytes=self.ws.numel(), stream=self.stream.cuda_stream,
                use_graphs=1 if use_graphs else 0, early_exit=EARLY_EXIT_CODES[early_exit])
            self.native = binding.loop_create(desc)

    def close(self) -> None:
        if self.native is not None:
            binding.loop_destroy(self.native)
            self.native = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- the buffers an iteration's producer writes ---------------------------
    def views(self, gamma: int) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor, torch.Tensor]:
        """Contiguous ``draft [B, gamma, V]``, ``target [B, gamma + 1, V]``,
        ``tokens [B, gamma]``, ``uniforms [B, gamma + 1]`` on the static buffers."""
        if not (1 <= gamma <= self.gamma_max):
            raise ValueError(f"gamma {gamma} outside 1 .. {self.gamma_max}")
        B, V = self.B, self.V
        return (self.draft[:B * gamma * V].view(B, gamma, V), self.target[:B * (gamma + 1) * V].view(B, gamma + 1, V),
                self.tokens[:B * gamma].view(B, gamma), self.uniforms[:B * (gamma + 1)].view(B, gamma + 1))

    def _call(self, gamma: int, early: bool = False) -> None:
        d, t, tok, u = self.views(gamma)
        binding.verify(d, t, tok, u, mode=self.mode, temperature=self.temperature, alpha=self.alpha,
                       beta=self.beta, accepted_len=self.acc, next_token=self.nxt, workspace=self.ws,
                       early_exit=early)

    def _graph(self, gamma: int, early: bool = False) -> torch.cuda.CUDAGraph:
        g = self.graphs.get((gamma, early))
        if g is None:
            with torch.cuda.stream(self.stream):
                self._call(gamma, early)   # eager once on the capture stream (checks the arguments)
            self.stream.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=self.stream):
                self._call(gamma, early)
            self.stream.synchronize()
            self.graphs[(gamma, early)] = g
        return g

    def capture_all(self) -> None:
        """Capture every gamma up front (keeps capture out of a timed loop)."""
        if self.native is not None:
            return
        for g in range(1, self.gamma_max + 1):
            for early in ((False, True) if self.mode == "exact" and self.early_exit != "never" else (False,)):
                self._graph(g, early)

    # -- one iteration ---------------------------------------------------------
    def launch(self, gamma: int, early: bool = False) -> None:
        """Enqueue the verification of the buffers' current contents on the loop's stream."""
        if self.use_graphs:
            graph = self._graph(gamma, early)
            with torch.cuda.stream(self.stream):
                graph.replay()
        else:
            with torch.cuda.stream(self.stream):
                self._call(gamma, early)

    def collect(self) -> Tuple[np.ndarray, np.ndarray]:
        """Wait for the launched call; its accepted lengths and next tokens."""
        B = self.B
        with torch.cuda.stream(self.stream):
            self.host[:B].copy_(self.acc, non_blocking=True)
            self.host[B:].copy_(self.nxt, non_blocking=True)
            self.flag_host.copy_(self.ws[binding.ERROR_FLAG_OFFSET:binding.ERROR_FLAG_OFFSET + 4].view(torch.int32),
                                 non_blocking=True)
        self.stream.synchronize()
        if int(self.flag_host[0]) != 0:
            raise binding.SpecVerifyError("a wait between workgroups timed out: the outputs are not valid; "
                                          "re-initialise the workspace (reset_workspace)")
        h = self.host.numpy()
        return h[:B].copy(), h[B:].copy()

    def reset_workspace(self) -> None:
        """Zero-fill the workspace (after a timed-out wait)."""
        with torch.cuda.stream(self.stream):
            binding.init_workspace(self.ws)
        self.stream.synchronize()

    def run(self, producer, iterations: int, stats: Optional[LoopStats] = None,
            time_device: bool = False) -> LoopStats:
        """``iterations`` rounds of: producer(self, i, gamma) fills the buffers
        (on ``self.stream``), the step runs, gamma is updated.  With
        ``time_device`` each step is bracketed by HIP events on the stream."""
        stats = stats or LoopStats()
        gamma = self.gamma0
        ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) if time_device else None
        for i in range(iterations):
            producer(self, i, gamma)
            if self.native is not None:
                nxt_gamma = binding.loop_step(self.native, gamma)
                h = self.host.numpy()
                L, nx = h[:self.B].copy(), h[self.B:].copy()
                stats.early_exit.append(binding.loop_last_early_exit(self.native) == 1)
                stats.iterations += 1
                stats.gammas.append(gamma)
                stats.accepted.append(L)
                stats.next_tokens.append(nx)
                stats.tokens += int(np.sum(np.where(L >= 0, L + 1, 0)))
                gamma = nxt_gamma
                continue
            early = self._early_next
            if ev is not None:
                ev[0].record(self.stream)
            self.launch(gamma, early)
            if ev is not None:
                ev[1].record(self.stream)
            L, nx = self.collect()
            stats.early_exit.append(early)
            if self.mode == "exact" and self.early_exit == "auto":
                self._early_next = early_exit_pays(L, gamma)
            if ev is not None:
                stats.device_us.append(ev[0].elapsed_time(ev[1]) * 1000.0)
            stats.iterations += 1
            stats.gammas.append(gamma)
            stats.accepted.append(L)
            stats.next_tokens.append(nx)
            stats.tokens += int(np.sum(np.where(L >= 0, L + 1, 0)))
            if self.adapt_gamma:
                gamma = next_gamma(gamma, L, self.gamma_max)
        return stats


class SyntheticSteps:
    """A device-resident pool of synthetic verification inputs at ``gamma_max``
    drafts; iteration i uses entry ``i % len(pool)``, cut to the iteration's
    gamma (rows are drawn independently, so the first gamma drafts of an
    entry are a valid gamma-draft)."""

    def __init__(self, workload, gamma_max: int, pool: int, device="cuda", seed0: Optional[int] = None):
        from . import workloads as W
        self.inputs = []
        self.dev = []
        base = workload.with_(gamma=gamma_max)
        for k in range(pool):
            x = W.generate(base, seed=(seed0 if seed0 is not None else base.seed * 1000) + k)
            self.inputs.append(x)
            self.dev.append(binding.to_device(x, device))
        torch.cuda.synchronize(device)

    def __len__(self) -> int:
        return len(self.dev)

    def __call__(self, loop: DecodeLoop, i: int, gamma: int) -> None:
        d, t, tok, u = self.dev[i % len(self.dev)]
        vd, vt, vtok, vu = loop.views(gamma)
        with torch.cuda.stream(loop.stream):
            vd.copy_(d[:, :gamma], non_blocking=True)
            vt.copy_(t[:, :gamma + 1], non_blocking=True)
            vtok.copy_(tok[:, :gamma], non_blocking=True)
            vu.copy_(u[:, :gamma + 1], non_blocking=True)

    def host_inputs(self, i: int, gamma: int):
        """The host (storage-form) inputs iteration i verified at this gamma."""
        from dataclasses import replace
        x = self.inputs[i % len(self.inputs)]
        return replace(x, draft=np.ascontiguousarray(x.draft[:, :gamma]),
                       target=np.ascontiguousarray(x.target[:, :gamma + 1]),
                       tokens=np.ascontiguousarray(x.tokens[:, :gamma]),
                       uniforms=np.ascontiguousarray(x.uniforms[:, :gamma + 1]))
