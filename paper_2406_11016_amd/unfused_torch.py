"""The verification step written with stock PyTorch operators: a comparison
baseline, not part of the library.

The paper's headline measurement is the reduction of sampling time against an
unfused implementation of the same step (Sec. 4, Tables 1 and 6).  This module
is that unfused implementation for the same GPU: full-size softmax (or
sigmoid) tensors, a gather at the drafted tokens, eq. (1), the first-rejection
scan, the residual of eqs. (2)-(3) or target row gamma, and an inverse-CDF draw
with ``cumsum`` / ``searchsorted`` -- one eager PyTorch kernel per operator,
fp32 throughout, as a typical framework implementation computes it.
``binding.verify`` never calls it.

Same conventions as the fused path: ``uniforms[b, c]`` is r_c for c < gamma and
``uniforms[b, gamma]`` drives the final draw; ties r_c == tau_c accept; the
draw takes the first index whose running sum exceeds ``u * sum``; a zero
residual mass falls back to the target row L (sigmoid mode).  It does not
reproduce the fused path's sentinels for invalid tokens or non-finite rows.
"""
from __future__ import annotations

import torch


def _first_rejection(accept: torch.Tensor) -> torch.Tensor:
    """Number of leading True values per row: the accepted length L."""
    return accept.to(torch.int32).cumprod(dim=-1).sum(dim=-1)


def verify(draft: torch.Tensor, target: torch.Tensor, tokens: torch.Tensor, uniforms: torch.Tensor, *,
           mode: str = "exact", temperature: float = 1.0, alpha: float = -1e4, beta: float = 1e4):
    """draft [B, gamma, V], target [B, gamma+1, V] (float32/float16/bfloat16),
    tokens [B, gamma] int32/int64, uniforms [B, gamma+1] float32; all on one
    device.  Returns (accepted_len [B] int32, next_token [B] int64)."""
    B, gamma, V = draft.shape
    zq = draft.float() / temperature
    zp = target.float() / temperature
    if mode == "exact":
        p = torch.softmax(zp, dim=-1)                       # eq. (4), target rows 0..gamma
        q = torch.softmax(zq, dim=-1)                       # draft rows 0..gamma-1
    elif mode == "sigmoid":
        span = beta - alpha
        p = torch.sigmoid((zp - alpha) / span)              # eq. (5), unnormalised
        q = torch.sigmoid((zq - alpha) / span)
    else:
        raise ValueError(mode)
    idx = tokens.long().unsqueeze(-1)
    px = p[:, :gamma].gather(-1, idx).squeeze(-1)
    qx = q.gather(-1, idx).squeeze(-1)
    tau = torch.where(qx > 0, torch.clamp(px / qx, max=1.0), torch.ones_like(px))   # eq. (1)
    L = _first_rejection(uniforms[:, :gamma] <= tau)

    rows = torch.arange(B, device=draft.device)
    pL = p[rows, L.long()]                                   # target row L (row gamma if all accepted)
    qL = q[rows, torch.clamp(L, max=gamma - 1).long()]
    rejected = (L < gamma).unsqueeze(-1)
    a = torch.where(rejected, torch.clamp(pL - qL, min=0.0), pL)   # eqs. (2)-(3) or the bonus row
    total = a.sum(dim=-1, keepdim=True)
    a = torch.where(total > 0, a, pL)                        # zero residual mass: draw from row L
    cdf = torch.cumsum(a, dim=-1)
    t = uniforms[:, gamma:gamma + 1] * cdf[:, -1:]
    nxt = torch.searchsorted(cdf, t, right=True).squeeze(-1)
    return L, torch.clamp(nxt, max=V - 1)
