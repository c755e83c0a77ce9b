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
    workspace: torch.Tensor          # shared by the steps when each call uploads its plan
    step_workspaces: Optional[List[torch.Tensor]]  # one per step, for planned (graph) calls
    o_acc: torch.Tensor
    lse_acc: torch.Tensor
    o_tmp: Optional[torch.Tensor]
    lse_tmp: Optional[torch.Tensor]
    o_bf16: torch.Tensor
    ds_buf: Optional[torch.Tensor] = None   # dS scratch of the stored-dS backward

    @property
    def nq(self) -> int:
        return self.problems[0].nq

    @property
    def n_heads(self) -> int:
        return self.problems[0].n_heads


# Device memory for the stored dS of one backward pass: on the 128K zigzag share one K/V
# head per pass (16 GiB) measured faster than four (64 GiB).
DEFAULT_DS_BUDGET_BYTES = 18 << 30


def ds_kv_heads_within(probs: Sequence[hydra.Problem], budget_bytes: int) -> int:
    """The most K/V heads per pass whose stored dS fits budget_bytes in every step (0: none,
    or the stored-dS path does not apply)."""
    hkv = probs[0].n_kv_heads
    best = 0
    for g in range(1, hkv + 1):
        need = [hydra.bwd_ds_bytes(p, g) for p in probs]
        if max(need) == 0 or max(need) > budget_bytes:
            break
        best = g
    return best


def make_share(cu_seqlens, n_heads: int, q_segs, kv_steps: Sequence, device="cuda",
               softmax_scale: float = 0.0, n_kv_heads: int = 0, graph_ready: bool = False,
               ds_kv_heads: int = 0, ds_budget_bytes: int = 0) -> Share:
    """Plans every ring step of one rank; n_kv_heads (0: n_heads) < n_heads for grouped K/V.
    graph_ready: one workspace per step, for plan() and the planned calls that a graph can
    record.  ds_kv_heads > 0: the backward stores dS instead of recomputing it for dQ, in
    passes of that many K/V heads (a dS scratch sized for the largest step), wherever the
    stored-dS path applies; or ds_budget_bytes > 0: as many K/V heads per pass as fit it."""
    probs = [hydra.Problem(cu_seqlens, n_heads, q_segs, s, softmax_scale, n_kv_heads=n_kv_heads) for s in kv_steps]
    ws = max(hydra.workspace_size(p) for p in probs)
    if ws == 0:
        raise hydra.HydraError(-1, "hydra_workspace_size")
    nq = probs[0].nq
    if ds_kv_heads <= 0 and ds_budget_bytes > 0:
        ds_kv_heads = ds_kv_heads_within(probs, ds_budget_bytes)
    ds = max(hydra.bwd_ds_bytes(p, ds_kv_heads) for p in probs) if ds_kv_heads > 0 else 0
    f32 = dict(dtype=torch.float32, device=device)
    multi = len(probs) > 1
    return Share(
        problems=probs,
        workspace=torch.empty(ws, dtype=torch.uint8, device=device),
        step_workspaces=[torch.empty(hydra.workspace_size(p), dtype=torch.uint8, device=device) for p in probs]
        if graph_ready else None,
        o_acc=torch.empty((nq, n_heads, D_V), **f32),
        lse_acc=torch.empty((n_heads, nq), **f32),
        o_tmp=torch.empty((nq, n_heads, D_V), **f32) if multi else None,
        lse_tmp=torch.empty((n_heads, nq), **f32) if multi else None,
        o_bf16=torch.empty((nq, n_heads, D_V), dtype=torch.bfloat16, device=device),
        ds_buf=torch.empty(ds, dtype=torch.uint8, device=device) if ds > 0 else None,
    )


def plan(sh: Share, stream=None):
    """Uploads every step's plan into its own workspace (a graph_ready share), outside any
    capture; afterwards forward/backward(planned=True) only launch kernels."""
    if sh.step_workspaces is None:
        raise ValueError("plan() needs a share made with graph_ready=True")
    for p, ws in zip(sh.problems, sh.step_workspaces):
        hydra.attn_plan(p, ws, stream)


def _ws(sh: Share, i: int, planned: bool):
    return sh.step_workspaces[i] if planned else sh.workspace


def forward(sh: Share, q: torch.Tensor, kv: Sequence[Tuple[torch.Tensor, torch.Tensor]], planned: bool = False):
    """Runs every ring step and the merges; returns (O fp32, LSE, O bf16)."""
    n = len(sh.problems)
    for i, (p, (k, v)) in enumerate(zip(sh.problems, kv)):
        ws = _ws(sh, i, planned)
        if i == 0:
            hydra.attn_fwd(p, q, k, v, sh.o_acc, sh.lse_acc, ws, o_bf16=sh.o_bf16 if n == 1 else None,
                           planned=planned)
        else:
            hydra.attn_fwd(p, q, k, v, sh.o_tmp, sh.lse_tmp, ws, planned=planned)
            hydra.lse_merge(sh.o_acc, sh.lse_acc, sh.o_tmp, sh.lse_tmp, o_bf16=sh.o_bf16 if i == n - 1 else None)
    return sh.o_acc, sh.lse_acc, sh.o_bf16


def backward(sh: Share, q, kv, d_o, dq: torch.Tensor, dkv: Sequence[Tuple[torch.Tensor, torch.Tensor]],
             planned: bool = False):
    """Accumulates dQ (over steps) and each step's dK/dV; buffers are += targets."""
    for i, (p, (k, v), (dk, dv)) in enumerate(zip(sh.problems, kv, dkv)):
        if sh.ds_buf is not None and not planned:
            hydra.attn_bwd_ds(p, q, k, v, sh.o_bf16, sh.lse_acc, d_o, dq, dk, dv, sh.ds_buf, sh.workspace)
        else:
            hydra.attn_bwd(p, q, k, v, sh.o_bf16, sh.lse_acc, d_o, dq, dk, dv, _ws(sh, i, planned),
                           planned=planned)
