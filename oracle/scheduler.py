"""CPU oracle for the load-driven dynamic-CP scheduler (linear scans, exact arithmetic).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call this module;
only the tests and the benchmark's CPU-baseline leg do.  It shares no code with the C++
scheduler: it follows the paper's steps with plain Python lists and linear scans.

The method (Sec. 5.1), restated:

* A length-s sequence split over cp ranks puts s/cp tokens and s^2/cp quadratic load on
  each of them (Sec. 5.1.1, Eq. (packing-density)); the heaviest micro-batch paces the
  iteration.
* Targets (Sec. 5.1.1): W = sum s_i^2; the CP-degree cap
      C_mem = ceil2(s_max / B),  C_hat = s_max^2 sqrt((pp-1) (theta/c) G / W),
      C* = min(G, ceil2(max(C_mem, C_hat)))                          (Eq. (cstar-cont), (cstar))
  the per-rank load target Lambda* = s_max^2 / C* (Eq. (load-target)), the micro-batch
  count target M* = ceil(C* W / (s_max^2 G)) (Eq. (mstar)), and each sequence's degree
      cp(s) = min(C*, ceil2(max(s^2 / Lambda*, s / B)))              (Eq. (cp))
  where ceil2(x) is the smallest power of two >= x.
* Placement (Alg. 1): sequences longest first; one micro-batch at a time over all G ranks.
  A sequence of degree k opens a new k-aligned group on free ranks if it can, otherwise it
  piggybacks on the smallest open group of size >= k that stays feasible (load(g) +
  s^2/|g| <= Lambda* and tokens(g) + s/|g| <= B), ties broken by load; if neither works
  the micro-batch is closed.  After closing, idle ranks are backfilled by doubling the
  smallest group.  The realized micro-batch count is returned.

Readings where the paper is silent (each one is also stated in the C++ header):

1. Opening a group needs a free k-aligned block of ranks (a "prebuilt power-of-two rank
   chunk"), not just k free ranks; the lowest such block is taken.  G must be a multiple
   of C*.
2. Ties: sequences of equal length keep their input order; among equally small and equally
   loaded feasible groups the one starting at the lowest rank wins.
3. The early stop "k has shrunk and MB balanced": k is smaller than the degree of the
   sequence that opened the micro-batch, and the micro-batch is balanced: no rank is free
   and the least loaded group carries at least balance_ratio (default 0.9) of the most
   loaded one.
4. Backfill: repeatedly take the smallest group (size, then start rank) whose aligned
   buddy block of the same size is entirely free and whose doubled size stays <= C*, and
   double it (its per-rank load and tokens halve); stop when no group can double.
5. theta/c (the cost ratio the paper says is measured on the cluster) is an input; with
   pp = 1 the bubble term vanishes and C* = min(G, C_mem).  An explicit cap may be given
   instead (then Eq. (cstar) is skipped).
6. Exact arithmetic: loads and tokens are kept multiplied by C* (integers), so the budget
   tests never depend on rounding.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence


def ceil2(x: float) -> int:
    """Smallest power of two >= x (>= 1)."""
    p = 1
    while p < x:
        p *= 2
    return p


@dataclass
class Targets:
    W: int
    s_max: int
    C_mem: int
    C_hat: float
    C: int          # C*
    M_target: int   # M*


def targets(lengths: Sequence[int], G: int, B: int, pp: int = 1, theta_over_c: float = 0.0,
            cap: Optional[int] = None) -> Targets:
    """Phase 1: W, the cap C* (Eq. (cstar)) and M* (Eq. (mstar))."""
    if not lengths or min(lengths) < 1 or G < 1 or B < 1:
        raise ValueError("need positive lengths, ranks and budget")
    s_max = max(lengths)
    W = sum(s * s for s in lengths)
    C_mem = ceil2(s_max / B)
    C_hat = s_max * s_max * math.sqrt((pp - 1) * theta_over_c * G / W) if pp > 1 else 0.0
    C = cap if cap is not None else min(G, ceil2(max(C_mem, C_hat)))
    if C < 1 or C & (C - 1) or C > G or G % C:
        raise ValueError("the cap must be a power of two dividing G")
    if C < C_mem:
        raise ValueError("the longest sequence does not fit the token budget under this cap")
    M = -(-C * W // (s_max * s_max * G))
    return Targets(W, s_max, C_mem, C_hat, C, M)


def cp_degree(s: int, s_max: int, C: int, B: int) -> int:
    """Eq. (cp): smallest power of two k with s^2/k <= Lambda* = s_max^2/C and s/k <= B, capped at C."""
    k = 1
    while k < C and (k * s_max * s_max < s * s * C or k * B < s):
        k *= 2
    return k


@dataclass
class Group:
    start: int
    size: int
    load: int = 0      # per-rank quadratic load, times C
    tokens: int = 0    # per-rank tokens, times C
    docs: List[int] = field(default_factory=list)


@dataclass
class Schedule:
    targets: Targets
    mbs: List[List[Group]]           # per micro-batch, its groups (in opening order)

    def placement(self):
        """(micro-batch, group start, group size) per input sequence."""
        out = {}
        for m, groups in enumerate(self.mbs):
            for g in groups:
                for d in g.docs:
                    out[d] = (m, g.start, g.size)
        return [out[i] for i in range(len(out))]


def schedule(lengths: Sequence[int], G: int, B: int, pp: int = 1, theta_over_c: float = 0.0,
             cap: Optional[int] = None, balance_ratio: float = 0.9) -> Schedule:
    t = targets(lengths, G, B, pp, theta_over_c, cap)
    C, s_max = t.C, t.s_max
    lam = s_max * s_max            # Lambda* times C
    budget = B * C                 # B times C
    order = sorted(range(len(lengths)), key=lambda i: (-lengths[i], i))
    mbs: List[List[Group]] = []
    pos = 0
    while pos < len(order):
        free = [True] * G
        groups: List[Group] = []
        k_open = None
        while pos < len(order):
            d = order[pos]
            s = lengths[d]
            k = cp_degree(s, s_max, C, B)
            g = None
            for a in range(0, G, k):                       # lowest free aligned block
                if all(free[a:a + k]):
                    g = Group(a, k)
                    for r in range(a, a + k):
                        free[r] = False
                    groups.append(g)
                    break
            if g is None:                                  # piggyback
                best = None
                for h in groups:
                    if h.size < k:
                        continue
                    f = C // h.size
                    if h.load + s * s * f > lam or h.tokens + s * f > budget:
                        continue
                    key = (h.size, h.load, h.start)
                    if best is None or key < best[0]:
                        best = (key, h)
                if best is None:
                    break
                g = best[1]
            f = C // g.size
            g.load += s * s * f
            g.tokens += s * f
            g.docs.append(d)
            pos += 1
            if k_open is None:
                k_open = k
            if k < k_open and not any(free):
                loads = [h.load for h in groups]
                if min(loads) >= balance_ratio * max(loads):
                    break
        if not groups:
            raise ValueError("a sequence fits no empty micro-batch")
        # backfill: double the smallest group whose buddy block is free
        while True:
            cand = None
            for h in groups:
                if 2 * h.size > C:
                    continue
                b = h.start ^ h.size
                if all(free[b:b + h.size]):
                    key = (h.size, h.start)
                    if cand is None or key < cand[0]:
                        cand = (key, h)
            if cand is None:
                break
            h = cand[1]
            b = h.start ^ h.size
            for r in range(b, b + h.size):
                free[r] = False
            h.start = min(h.start, b)
            h.size *= 2
            h.load //= 2
            h.tokens //= 2
        mbs.append(groups)
    return Schedule(t, mbs)
