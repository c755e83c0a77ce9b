"""One rank's attention share over all outer-ring steps, through the C ABI.

Forward: one partial per ring step, merged exactly into (O, LSE) with a bf16 copy of O
(Sec. 5.2.2, "as in standard ring CP").  Backward: every step differentiates with the
final merged O and LSE; dQ accumulates over steps, dK/dV are per KV chunk.  The
exchange that would move K/V between ranks is not here (one GPU); each step's chunk is
simply another buffer with its global offsets.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import torch

from . import hydra

D_QK, D_V = 192, 128


@dataclass
class Share:
    """Problems and device buffers for one rank's share."""
    problems: List[hydra.Problem]
    workspace: torch.Tensor
    o_acc: torch.Tensor
    lse_acc: torch.Tensor
    o_tmp: Optional[torch.Tensor]
    lse_tmp: Optional[torch.Tensor]
    o_bf16: torch.Tensor

    @property
    def nq(self) -> int:
        return self.problems[0].nq

    @property
    def n_heads(self) -> int:
        return self.problems[0].n_heads


def make_share(cu_seqlens, n_heads: int, q_segs, kv_steps: Sequence, device="cuda",
               softmax_scale: float = 0.0, n_kv_heads: int = 0) -> Share:
    """Plans every ring step of one rank; n_kv_heads (0: n_heads) < n_heads for grouped K/V."""
    probs = [hydra.Problem(cu_seqlens, n_heads, q_segs, s, softmax_scale, n_kv_heads=n_kv_heads) for s in kv_steps]
    ws = max(hydra.workspace_size(p) for p in probs)
    if ws == 0:
        raise hydra.HydraError(-1, "hydra_workspace_size")
    nq = probs[0].nq
    f32 = dict(dtype=torch.float32, device=device)
    multi = len(probs) > 1
    return Share(
        problems=probs,
        workspace=torch.empty(ws, dtype=torch.uint8, device=device),
        o_acc=torch.empty((nq, n_heads, D_V), **f32),
        lse_acc=torch.empty((n_heads, nq), **f32),
        o_tmp=torch.empty((nq, n_heads, D_V), **f32) if multi else None,
        lse_tmp=torch.empty((n_heads, nq), **f32) if multi else None,
        o_bf16=torch.empty((nq, n_heads, D_V), dtype=torch.bfloat16, device=device),
    )


def forward(sh: Share, q: torch.Tensor, kv: Sequence[Tuple[torch.Tensor, torch.Tensor]]):
    """Runs every ring step and the merges; returns (O fp32, LSE, O bf16)."""
    n = len(sh.problems)
    for i, (p, (k, v)) in enumerate(zip(sh.problems, kv)):
        if i == 0:
            hydra.attn_fwd(p, q, k, v, sh.o_acc, sh.lse_acc, sh.workspace, o_bf16=sh.o_bf16 if n == 1 else None)
        else:
            hydra.attn_fwd(p, q, k, v, sh.o_tmp, sh.lse_tmp, sh.workspace)
            hydra.lse_merge(sh.o_acc, sh.lse_acc, sh.o_tmp, sh.lse_tmp, o_bf16=sh.o_bf16 if i == n - 1 else None)
    return sh.o_acc, sh.lse_acc, sh.o_bf16


def backward(sh: Share, q, kv, d_o, dq: torch.Tensor, dkv: Sequence[Tuple[torch.Tensor, torch.Tensor]]):
    """Accumulates dQ (over steps) and each step's dK/dV; buffers are += targets."""
    for p, (k, v), (dk, dv) in zip(sh.problems, kv, dkv):
        hydra.attn_bwd(p, q, k, v, sh.o_bf16, sh.lse_acc, d_o, dq, dk, dv, sh.workspace)
