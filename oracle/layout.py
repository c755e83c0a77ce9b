"""CPU oracle for the Ulysses x ring data layout of one context-parallel group.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call this
module; only the tests (and the smoke check) do.  It shares no code with the HIP
path: every function below is plain numpy indexing.

What is computed (the paper's setting, restated):

* A sequence split over P ranks is factored into an inner Ulysses degree cp_u over
  heads and an outer ring degree cp_r over the sequence, cp_u = min(P, h) and
  cp_r = P / cp_u (Sec. 5.2.1, Eq. (usp)).
* Ulysses partitions the attention heads across the ranks of a group with
  all-to-all transposes (Sec. 3.5, "Ulysses scales down ..."): before the exchange
  a rank holds a slice of the tokens with every head, after it all the tokens of
  the group with a slice of the heads.  The reverse exchange returns the output.
* The ring circulates K/V chunks between the cp_r groups (Sec. 3.5, "Ring reaches
  any degree"; Sec. 5.2.2, last paragraph).  Which tokens a ring rank holds is not
  printed; the reading used here is the usual causal load balancing: the sequence
  is cut into 2*cp_r equal chunks and ring rank r holds chunks r and 2*cp_r-1-r,
  in that order ("zigzag").

Layouts are token-major: X[token][head][dim].  A ring shard's token list is the
concatenation of its two chunks; Ulysses rank u of ring group r starts with the
u-th of cp_u equal slices of that list.
"""
from __future__ import annotations

import numpy as np


def usp_degrees(P: int, h: int):
    """(cp_u, cp_r) for a CP degree P and h heads (Eq. (usp))."""
    if P < 1 or h < 1:
        raise ValueError("P and h must be positive")
    cp_u = min(P, h)
    if P % cp_u:
        raise ValueError("P must be a multiple of min(P, h)")
    return cp_u, P // cp_u


def zigzag_rows(s: int, cp_r: int, r: int) -> np.ndarray:
    """Global token indices held by ring rank r, in local order."""
    if s % (2 * cp_r):
        raise ValueError("sequence length must split into 2*cp_r equal chunks")
    c = s // (2 * cp_r)
    return np.concatenate([np.arange(r * c, (r + 1) * c), np.arange((2 * cp_r - 1 - r) * c, (2 * cp_r - r) * c)])


def seq_shard(X: np.ndarray, cp_u: int, cp_r: int, u: int, r: int) -> np.ndarray:
    """Rank (u, r)'s tokens before the Ulysses exchange: all heads, s/P tokens."""
    rows = zigzag_rows(X.shape[0], cp_r, r)
    n = rows.size // cp_u
    return X[rows[u * n:(u + 1) * n]]


def head_shard(X: np.ndarray, cp_u: int, cp_r: int, u: int, r: int) -> np.ndarray:
    """Rank (u, r)'s tensor after the exchange: every token of ring shard r, head group u."""
    rows = zigzag_rows(X.shape[0], cp_r, r)
    g = X.shape[1] // cp_u
    return X[rows][:, u * g:(u + 1) * g]


def pack_heads(x_seq: np.ndarray, cp_u: int) -> np.ndarray:
    """Send buffers of the forward exchange: send[j] = this rank's tokens, head group j."""
    t, h, d = x_seq.shape
    g = h // cp_u
    return np.stack([x_seq[:, j * g:(j + 1) * g] for j in range(cp_u)])


def unpack_heads(recv: np.ndarray) -> np.ndarray:
    """Inverse of pack_heads: recv[j] (tokens, head group j) -> tokens with every head."""
    return np.concatenate(list(recv), axis=1)


def alltoall(sends):
    """The exchange inside one Ulysses group as a permutation: recv[u][j] = sends[j][u]."""
    n = len(sends)
    return [np.stack([sends[j][u] for j in range(n)]) for u in range(n)]


def gather_tokens(recv: np.ndarray) -> np.ndarray:
    """After the forward exchange: the group's token slices in rank order."""
    return np.concatenate(list(recv), axis=0)


def split_tokens(x_head: np.ndarray, cp_u: int) -> np.ndarray:
    """Send buffers of the reverse exchange: cp_u equal token slices."""
    n = x_head.shape[0] // cp_u
    return np.stack([x_head[j * n:(j + 1) * n] for j in range(cp_u)])
