"""From the scheduler's placement to one rank's attention share (host only).

hydra.schedule gives every sequence of a batch its micro-batch m and its group of ranks
[start, start + k) (Sec. 5.1, Alg. 1): the group's ranks share that sequence with context-
parallel degree k, and every sequence piggybacked on the group shares its ranks and its
degree.  This module turns (m, rank) into the attention problems that rank solves:

* the documents it holds, 𝒢[m][r]: the sequences of its group, in batch order, packed
  into one window (their cu_seqlens), since packed documents are masked across their
  boundaries (Sec. 2.2);
* the factorisation of the degree, k = cp_u * cp_r with cp_u = min(k, h) (Sec. 5.2.1,
  Eq. (usp)); group member g = rank - start is Ulysses rank u = g % cp_u of ring rank
  rho = g // cp_u, so the Ulysses group is the consecutive ranks;
* its head shard, query heads [u h / cp_u, (u + 1) h / cp_u) (Sec. 3.5: Ulysses splits
  the heads), and the K/V heads they use: split the same way, or, with fewer K/V heads
  than Ulysses ranks (grouped heads), the one K/V head of the shard's group;
* its query rows: in every sequence, the ring rank's zigzag chunks rho and 2 cp_r - 1 - rho
  of 2 cp_r chunks (chunk j covers [floor(j s / (2 cp_r)), floor((j + 1) s / (2 cp_r)))) --
  the reading of which rows a ring rank holds, as in the layout calls;
* per ring step i, the K/V chunks that reach it: those of ring rank (rho - i) mod cp_r.

A problem holds at most HYDRA_MAX_SEGS segments per chunk, so the documents are split into
sub-shares of 2 documents when cp_r > 1 (2 segments each); attention never crosses a
document, so solving the sub-shares one after another is the same computation.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import numpy as np

from . import hydra

Segs = List[Tuple[int, int]]


@dataclass
class SubShare:
    """One problem family of a rank: documents, their window, its rows per ring step."""
    seqs: List[int]              # batch indices of the documents, in window order
    cu: List[int]                # document boundaries in the sub-share's packed window
    q_segs: Segs                 # the rank's query rows
    kv_steps: List[Segs]         # K/V rows arriving at each ring step


@dataclass
class RankShare:
    m: int
    rank: int
    group_start: int
    k: int                       # the group's context-parallel degree
    cp_u: int
    cp_r: int
    u: int                       # Ulysses rank within the ring rank's group
    rho: int                     # ring rank
    head0: int                   # first query head of the shard
    n_heads: int                 # query heads held
    kv_head0: int
    n_kv_heads: int
    parts: List[SubShare]


def usp_degrees(k: int, h: int) -> Tuple[int, int]:
    """(cp_u, cp_r) = (min(k, h), k / min(k, h)) (Sec. 5.2.1, Eq. (usp))."""
    cp_u = min(k, h)
    if k % cp_u:
        raise ValueError(f"degree {k} is not a multiple of min({k}, {h})")
    return cp_u, k // cp_u


def zigzag_chunks(s: int, cp_r: int, r: int) -> Segs:
    """Local (start, length) of ring rank r's two chunks of a sequence of s tokens."""
    n = 2 * cp_r
    edge = lambda j: (j * s) // n
    return [(edge(r), edge(r + 1) - edge(r)), (edge(n - 1 - r), edge(n - r) - edge(n - 1 - r))]


def rank_share(lengths: Sequence[int], mb: Sequence[int], gstart: Sequence[int], gsize: Sequence[int], m: int,
               rank: int, n_heads: int, n_kv_heads: int = 0) -> Optional[RankShare]:
    """Rank `rank`'s share of micro-batch m, or None if it holds nothing there."""
    lengths = [int(x) for x in lengths]
    mine = [i for i in range(len(lengths)) if mb[i] == m and gstart[i] <= rank < gstart[i] + gsize[i]]
    if not mine:
        return None
    start, k = int(gstart[mine[0]]), int(gsize[mine[0]])
    if any(int(gstart[i]) != start or int(gsize[i]) != k for i in mine):
        raise ValueError("a rank belongs to one group per micro-batch")
    hkv = n_kv_heads or n_heads
    cp_u, cp_r = usp_degrees(k, n_heads)
    if n_heads % cp_u:
        raise ValueError("the Ulysses degree must divide the head count")
    g = rank - start
    u, rho = g % cp_u, g // cp_u
    h_rank = n_heads // cp_u
    if hkv % cp_u == 0:                  # K/V heads split like the query heads
        kv0, n_kv = u * (hkv // cp_u), hkv // cp_u
    elif cp_u % hkv == 0:                # fewer K/V heads than Ulysses ranks: each rank holds
        kv0, n_kv = (u * h_rank) // (n_heads // hkv), 1   # the one its query heads use
    else:
        raise ValueError("the Ulysses degree and the K/V head count must divide one another")
    per = 1 if cp_r == 1 else 2          # documents per sub-share (2 segments each when split)
    parts = []
    groups = [mine] if cp_r == 1 else [mine[i:i + per] for i in range(0, len(mine), per)]
    for docs in groups:
        cu = [0] + list(np.cumsum([lengths[d] for d in docs]))
        if cp_r == 1:
            q = [(0, int(cu[-1]))]
            steps = [list(q)]
        else:
            def rows_of(r):
                out = []
                for d, base in zip(docs, cu[:-1]):
                    out += [(int(base) + a, n) for a, n in zigzag_chunks(lengths[d], cp_r, r)]
                return out
            q = rows_of(rho)
            steps = [rows_of((rho - i) % cp_r) for i in range(cp_r)]
        parts.append(SubShare(list(docs), [int(x) for x in cu], q, steps))
    return RankShare(m, rank, start, k, cp_u, cp_r, u, rho, u * h_rank, h_rank, kv0, n_kv, parts)


def problems(share: RankShare, softmax_scale: float = 0.0) -> List[List[hydra.Problem]]:
    """The hydra problems of every sub-share: one per ring step."""
    nkv = share.n_kv_heads if share.n_kv_heads != share.n_heads else 0
    return [[hydra.Problem(p.cu, share.n_heads, p.q_segs, st, softmax_scale, n_kv_heads=nkv) for st in p.kv_steps]
            for p in share.parts]
