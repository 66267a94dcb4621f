"""Seeded synthetic inputs for the speculative-sampling verification step.

This module produces the *inputs* of one verification step -- draft logits
``[B, gamma, V]``, target logits ``[B, gamma+1, V]``, the drafted tokens
``[B, gamma]`` and the uniforms ``[B, gamma+1]`` -- for the named workloads
below.  It holds none of the verification arithmetic (no softmax, no
acceptance ratio, no residual, no inverse CDF): the drafted tokens are drawn
with the Gumbel-max trick, ``x = argmax_v (z_q[v]/T + G[v])`` with
``G ~ Gumbel(0, 1)``, which samples from the draft model's categorical
distribution without normalising it.

Both the CPU oracle (through the tests) and the GPU library consume exactly
the arrays returned here, already rounded to the storage dtype.  bf16 values
are returned as their raw 16-bit patterns (``uint16``), because NumPy has no
bfloat16 type.

Recipe (paper: Sec. 4.1 describes the ASR / summarisation workloads; the
datasets and trained models are not available, so these synthetic logits
stand in for them):

* batch element ``b`` of a workload with seed ``s`` draws from its own
  ``PCG64(SeedSequence([s, b]))`` stream, so any ``b`` can be regenerated on
  its own;
* draw order per ``b``: ``base [gamma+1, V]`` (normal or scaled Student-t),
  ``noise [gamma+1, V]`` (normal), the Gumbel noise ``[gamma, V]`` for the
  drafted tokens, then the uniforms ``[gamma+1]``;
* ``draft = base[:gamma]``, ``target = base + noise``; both are rounded to the
  storage dtype (fp32 / fp16 round-to-nearest-even, bf16 round-to-nearest-even
  from the fp32 bits);
* the drafted tokens are sampled from the *rounded* draft logits at
  temperature ``T``;
* uniforms are U(0,1) rounded to fp32 and clamped to ``<= 1 - 2**-24``;
  columns ``0..gamma-1`` are the acceptance uniforms ``r_c`` of eq. (1) and
  column ``gamma`` drives the final inverse-CDF sample.
"""
from __future__ import annotations

from dataclasses import dataclass, replace
from typing import Dict, Optional

import numpy as np

STORAGE_DTYPES = ("f32", "f16", "bf16")
BYTES_PER_LOGIT = {"f32": 4, "f16": 2, "bf16": 2}
UNIFORM_MAX = np.float32(1.0 - 2.0 ** -24)


@dataclass(frozen=True)
class Workload:
    """One synthetic verification workload (shape, storage dtype, value law)."""

    name: str
    mode: str            # "exact" or "sigmoid"
    batch: int           # B
    gamma: int           # number of drafted tokens
    vocab: int           # V
    dtype: str           # storage dtype of the logits: "f32" | "f16" | "bf16"
    base: str            # law of the shared base logits: "normal" | "student_t3"
    base_scale: float    # std of the normal base, or the multiplier of t(3)
    noise_scale: float   # std of the target-minus-draft noise
    seed: int
    temperature: float = 1.0
    alpha: float = -1.0e4   # sigmoid scaling constants (eq. (5)); unused in exact mode
    beta: float = 1.0e4
    top_k: int = 0          # > 0: every row keeps its k largest logits, the rest are -inf

    @property
    def logit_bytes(self) -> int:
        """Bytes of both logit tensors: B * (2*gamma + 1) * V * s."""
        return self.batch * (2 * self.gamma + 1) * self.vocab * BYTES_PER_LOGIT[self.dtype]

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# Named by what they are.  ASR-shaped workloads use a Whisper-sized vocabulary
# (51,865) with fp32 or fp16 logits; summarisation-shaped ones use LLM
# vocabularies (32,000 / 50,272 / 128,256).
WORKLOADS: Dict[str, Workload] = {
    w.name: w
    for w in (
        Workload("exact_b1_g5_v51865_f32", "exact", 1, 5, 51865, "f32",
                 "normal", 2.0, 0.5, seed=1000),
        Workload("exact_b1_g10_v32000_f16", "exact", 1, 10, 32000, "f16",
                 "normal", 3.0, 1.0, seed=1001),
        Workload("exact_b16_g5_v51865_f32", "exact", 16, 5, 51865, "f32",
                 "normal", 2.0, 0.5, seed=1002),
        Workload("exact_b64_g8_v128256_bf16", "exact", 64, 8, 128256, "bf16",
                 "student_t3", 2.0, 0.7, seed=1003),
        Workload("sigmoid_b32_g10_v50272_f16_t0.7", "sigmoid", 32, 10, 50272, "f16",
                 "normal", 2.0, 0.5, seed=1004, temperature=0.7,
                 alpha=-1.0e4, beta=1.0e4),
    )
}

#: the largest workload; the benchmark's default
HEADLINE = "exact_b64_g8_v128256_bf16"


@dataclass
class Inputs:
    """Inputs of one verification step, in storage form (host NumPy arrays)."""

    draft: np.ndarray      # [B, gamma, V]    float32 | float16 | uint16 (bf16 bits)
    target: np.ndarray     # [B, gamma+1, V]  same dtype as draft
    tokens: np.ndarray     # [B, gamma]       int32
    uniforms: np.ndarray   # [B, gamma+1]     float32
    dtype: str
    mode: str
    temperature: float
    alpha: float
    beta: float

    @property
    def batch(self) -> int:
        return int(self.draft.shape[0])

    @property
    def gamma(self) -> int:
        return int(self.draft.shape[1])

    @property
    def vocab(self) -> int:
        return int(self.draft.shape[2])


# ---------------------------------------------------------------------------
# storage encodings (rounding only)
# ---------------------------------------------------------------------------

def encode_bf16(values: np.ndarray) -> np.ndarray:
    """Round to bf16 (round-to-nearest-even on the fp32 bits); returns uint16 bits."""
    f = np.ascontiguousarray(values, dtype=np.float32)
    bits = f.view(np.uint32).astype(np.uint64)
    rounded = (bits + 0x7FFF + ((bits >> 16) & 1)) >> 16
    out = rounded.astype(np.uint16)
    nan = np.isnan(f)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float32 values (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def encode(values: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.asarray(values, dtype=np.float32)
    if dtype == "f16":
        return np.asarray(values, dtype=np.float16)
    if dtype == "bf16":
        return encode_bf16(values)
    raise ValueError(f"unknown storage dtype {dtype!r}")


def stored_as_float64(stored: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of stored logits (generator-internal use)."""
    if dtype == "bf16":
        return decode_bf16(stored).astype(np.float64)
    return np.asarray(stored).astype(np.float64)


# ---------------------------------------------------------------------------
# generation
# ---------------------------------------------------------------------------

def _draw_base(g: np.random.Generator, law: str, scale: float, shape) -> np.ndarray:
    if law == "normal":
        return g.normal(0.0, scale, size=shape)
    if law == "student_t3":
        return scale * g.standard_t(3.0, size=shape)
    raise ValueError(f"unknown base law {law!r}")


def make_uniforms(g: np.random.Generator, n: int) -> np.ndarray:
    u = g.random(n).astype(np.float32)
    return np.minimum(u, UNIFORM_MAX)


def gumbel_max_tokens(g: np.random.Generator, draft_f64: np.ndarray,
                      temperature: float) -> np.ndarray:
    """Draw one token per row of ``draft_f64`` ([rows, V]) from its softmax(z/T)
    law by the Gumbel-max trick."""
    gum = g.gumbel(size=draft_f64.shape)
    return np.argmax(draft_f64 / temperature + gum, axis=-1).astype(np.int32)


def mask_top_k(stored: np.ndarray, dtype: str, k: int) -> np.ndarray:
    """A top-k logit processor: each row (last axis) keeps its k largest
    stored logits (ties broken towards the lower index) and every other logit
    becomes -inf.  k <= 0 or k >= V leaves the rows unchanged."""
    V = stored.shape[-1]
    if k <= 0 or k >= V:
        return stored
    vals = stored_as_float64(stored, dtype)
    drop = np.argsort(-vals, axis=-1, kind="stable")[..., k:]
    out = stored.copy()
    np.put_along_axis(out, drop, encode(np.array([-np.inf]), dtype)[0], axis=-1)
    return out


def generate(w: Workload, seed: Optional[int] = None,
             batch_indices: Optional[range] = None) -> Inputs:
    """Generate the inputs of ``w``.  ``batch_indices`` selects a subset of the
    batch elements (each element has its own seeded stream, so a subset equals
    the corresponding slice of the full batch)."""
    seed = w.seed if seed is None else seed
    idx = range(w.batch) if batch_indices is None else batch_indices
    G, V = w.gamma, w.vocab
    store_np = {"f32": np.float32, "f16": np.float16, "bf16": np.uint16}[w.dtype]
    n = len(idx)
    draft = np.empty((n, G, V), dtype=store_np)
    target = np.empty((n, G + 1, V), dtype=store_np)
    tokens = np.empty((n, G), dtype=np.int32)
    uniforms = np.empty((n, G + 1), dtype=np.float32)
    for i, b in enumerate(idx):
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, b])))
        base = _draw_base(g, w.base, w.base_scale, (G + 1, V))
        noise = g.normal(0.0, w.noise_scale, size=(G + 1, V))
        draft[i] = mask_top_k(encode(base[:G], w.dtype), w.dtype, w.top_k)
        target[i] = mask_top_k(encode(base + noise, w.dtype), w.dtype, w.top_k)
        del base, noise
        tokens[i] = gumbel_max_tokens(g, stored_as_float64(draft[i], w.dtype), w.temperature)
        uniforms[i] = make_uniforms(g, G + 1)
    return Inputs(draft, target, tokens, uniforms, w.dtype, w.mode,
                  float(w.temperature), float(w.alpha), float(w.beta))


def small_case(batch: int, gamma: int, vocab: int, dtype: str, mode: str = "exact",
               seed: int = 7, base_scale: float = 2.0, noise_scale: float = 0.5,
               temperature: float = 1.0, alpha: float = -1.0e4, beta: float = 1.0e4,
               base: str = "normal", top_k: int = 0) -> Inputs:
    """A small workload of arbitrary shape with the same value law (tests)."""
    w = Workload(f"{mode}_b{batch}_g{gamma}_v{vocab}_{dtype}", mode, batch, gamma, vocab,
                 dtype, base, base_scale, noise_scale, seed=seed,
                 temperature=temperature, alpha=alpha, beta=beta, top_k=top_k)
    return generate(w)
