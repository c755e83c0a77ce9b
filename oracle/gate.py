"""fp64 CPU oracle for the gated attention output around the output exchange.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call this
module; only the tests do.  It shares no code with the HIP path: numpy
elementwise arithmetic and the layout oracle's indexing.

What is computed (the paper's setting, restated):

* The paper's model uses gated MLA (Sec. 5.2.2 and the figure of its asynchronous
  all-to-all schedule, citing Qiu et al. 2025).  Beside Q, K and V a gate
  projection of the layer input is computed, and it needs no context-parallel
  communication.  The paper prints no gate formula; the reading used here is the
  cited work's gate: the attention output Y of every head is multiplied
  elementwise by the logistic sigmoid of the gate logits G,

      Y'[t, h, d] = Y[t, h, d] * sigmoid(G[t, h, e]),   sigmoid(x) = 1 / (1 + e^-x)

  with either one logit per (token, head, channel) ("elementwise", e = d) or one
  per (token, head) ("headwise", G of last dimension 1, e = 0 for every d).
* Because the gate projection runs on the rank's own tokens with every head, the
  product is taken where the output is back in that layout: after the reverse
  (head -> sequence) exchange, i.e. fused with its unpack.  Its backward is fused
  with the pack that starts the backward exchange.
* Gradients of a loss with output gradient dY' (chain rule; sigmoid' = s (1 - s),
  where 1 - s is evaluated as sigmoid(-G), the same number without the cancellation that
  rounds it to 0 once s rounds to 1):

      dY[t, h, d] = dY'[t, h, d] * s[t, h, e]
      dG[t, h, d] = dY'[t, h, d] * Y[t, h, d] * s (1 - s)          (elementwise)
      dG[t, h]    = sum_d dY'[t, h, d] * Y[t, h, d] * s (1 - s)    (headwise)
"""
from __future__ import annotations

import numpy as np

from . import layout as L


def sigmoid(x) -> np.ndarray:
    """The logistic function in fp64, written so neither branch overflows."""
    x = np.asarray(x, np.float64)
    out = np.empty_like(x)
    pos = x >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-x[pos]))
    e = np.exp(x[~pos])
    out[~pos] = e / (1.0 + e)
    return out


def _gate_shape(y, g):
    if g.shape[:2] != y.shape[:2] or g.shape[2] not in (1, y.shape[2]):
        raise ValueError(f"gate {g.shape} does not fit output {y.shape}: last dim must be 1 or {y.shape[2]}")


def gate_fwd(y, g) -> np.ndarray:
    """Y' = Y * sigmoid(G), G of shape [T][H][1] (headwise) or [T][H][d] (elementwise)."""
    y, g = np.asarray(y, np.float64), np.asarray(g, np.float64)
    _gate_shape(y, g)
    return y * sigmoid(g)


def gate_bwd(y, g, dy_gated):
    """(dY, dG) for Y' = Y * sigmoid(G), given dY'.  Y is the output before the gate."""
    y, g, dyg = (np.asarray(a, np.float64) for a in (y, g, dy_gated))
    _gate_shape(y, g)
    s = sigmoid(g)
    dy = dyg * s
    dg = dyg * y * s * sigmoid(-g)        # 1 - s = sigmoid(-g)
    if g.shape[2] == 1:
        dg = dg.sum(axis=2, keepdims=True)
    return dy, dg


def unpack_gated(recv, g) -> np.ndarray:
    """The reverse exchange's receive side with the gate: recv[j] holds this rank's tokens
    for head group j; the result is [T][H][d] with every head, gated."""
    return gate_fwd(L.unpack_heads(np.asarray(recv, np.float64)), g)


def pack_gated_bwd(y, g, dy_gated, cp_u: int):
    """Backward of unpack_gated: the send buffers [cp_u][T][H/cp_u][d] of dY (the gradient
    that travels back through the exchange to the attention) and dG in the token layout."""
    dy, dg = gate_bwd(y, g, dy_gated)
    return L.pack_heads(dy, cp_u), dg
