"""fp64 CPU oracle for one context-parallel rank's attention share.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call this
module; only the tests, the smoke check and the benchmark's CPU-baseline leg do.
It shares no code with the HIP path: it takes plain arrays and recomputes every
step from the definition, with numpy matrix products as the only library help.

What is computed (the paper's setting, restated):

* Documents are packed into one window and attention is masked across their
  boundaries (Sec. 2.2).  A query at global position p sees the keys of its own
  document up to and including p (causal, diagonal included).
* Under context parallelism a rank holds a chunk of the queries and, at each
  outer-ring step, one chunk of the keys/values that circulate around the ring
  (Sec. 2.1; Sec. 3.5 "Ring reaches any degree"; Sec. 5.2.1 Eq. (usp)).  Chunks are
  lists of segments of global positions; masking always uses global positions.
* Each step yields a partial output and its log-sum-exp; partials combine
  exactly, as in standard ring CP (Sec. 5.2.2, last paragraph).
* Under MLA every head has its own K and V (Sec. 1), here d_qk=192, d_v=128.
  With grouped-query attention a rank holds fewer K/V heads than query heads,
  h_kv <= h (Sec. 3.5, ring traffic "only the h_kv key/value heads").  How query
  heads share K/V heads is not printed; the reading used here is the usual one:
  h_kv contiguous groups of h / h_kv query heads, query head i using K/V head
  i // (h / h_kv).  h_kv = h is the MLA case.

The attention itself is the textbook masked softmax (the paper names
FlashAttention, Sec. 1 and Sec. 3.5, and computes the same function):

    s_ij  = tau * <q_i, k_j>                    over visible (i, j)
    LSE_i = log sum_j exp(s_ij)                 (-inf when nothing is visible)
    O_i   = sum_j exp(s_ij - LSE_i) v_j         (0 when nothing is visible)

and its gradient for a loss with output gradient dO, using the *final* merged
O and LSE of the row (so every ring step differentiates the same function):

    D_i   = <dO_i, O_i>
    P_ij  = exp(s_ij - LSE_i)
    dV_j  = sum_i P_ij dO_i
    dS_ij = P_ij (<dO_i, v_j> - D_i)
    dQ_i  = tau sum_j dS_ij k_j
    dK_j  = tau sum_i dS_ij q_i

Inputs may be any float dtype (the tests pass bf16-rounded values as float32,
which is exact); everything is promoted to float64.
"""
from __future__ import annotations

import math
from typing import Iterable, Optional, Sequence, Tuple

import numpy as np

NEG_INF = -np.inf
_SCORE_BLOCK = 1 << 24  # max fp64 score elements held at once (128 MiB)


def default_scale(d_qk: int) -> float:
    return 1.0 / math.sqrt(d_qk)


def row_positions(segments: Sequence[Tuple[int, int]]) -> np.ndarray:
    """Global position of every local row: the segments' ranges, concatenated."""
    parts = [np.arange(s, s + n, dtype=np.int64) for s, n in segments]
    return np.concatenate(parts) if parts else np.zeros(0, dtype=np.int64)


def doc_of(cu_seqlens: Sequence[int], pos: np.ndarray) -> np.ndarray:
    """Index d of the document with cu[d] <= pos < cu[d+1]."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    return np.searchsorted(cu, pos, side="right") - 1


def _group(H: int, Hkv: int) -> int:
    """Query heads per K/V head."""
    if Hkv < 1 or H % Hkv:
        raise ValueError("the K/V head count must divide the query head count")
    return H // Hkv


def _f64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


def _groups(cu, qpos, kpos):
    """Per document: (query rows, key rows) of that document present in the chunks."""
    qd = doc_of(cu, qpos)
    kd = doc_of(cu, kpos)
    for d in np.unique(qd):
        yield np.nonzero(qd == d)[0], np.nonzero(kd == d)[0]


def attn_fwd(q, k, v, cu_seqlens, q_segs, kv_segs, scale: Optional[float] = None,
             heads: Optional[Iterable[int]] = None, q_rows: Optional[np.ndarray] = None):
    """Partial output and LSE of one ring step.

    q [Nq,H,dqk], k [Nk,Hkv,dqk], v [Nk,Hkv,dv] (Hkv divides H; query head h uses
    K/V head h // (H/Hkv)).  Returns O [Nq,H,dv] float64 and
    LSE [H,Nq] float64 (natural log).  ``heads`` / ``q_rows`` restrict the work
    to a subset (other entries stay O=0, LSE=-inf); the full-size tests use them.
    """
    Q, K, V = np.asarray(q), np.asarray(k), np.asarray(v)   # promoted to fp64 slice by slice
    nq, H, dqk = Q.shape
    grp = _group(H, K.shape[1])
    tau = default_scale(dqk) if scale is None else float(scale)
    qpos, kpos = row_positions(q_segs), row_positions(kv_segs)
    assert len(qpos) == nq and len(kpos) == K.shape[0]
    O = np.zeros((nq, H, V.shape[2]))
    L = np.full((H, nq), NEG_INF)
    sel = np.ones(nq, bool) if q_rows is None else np.isin(np.arange(nq), q_rows)
    for h in (range(H) if heads is None else heads):
        for qi, ki in _groups(cu_seqlens, qpos, kpos):
            qi = qi[sel[qi]]
            if len(qi) == 0 or len(ki) == 0:
                continue
            Kd, Vd = _f64(K[ki, h // grp, :]), _f64(V[ki, h // grp, :])
            step = max(1, _SCORE_BLOCK // len(ki))
            for b in range(0, len(qi), step):
                rows = qi[b:b + step]
                s = tau * (_f64(Q[rows, h, :]) @ Kd.T)
                vis = kpos[ki][None, :] <= qpos[rows][:, None]
                s = np.where(vis, s, NEG_INF)
                m = s.max(axis=1)
                empty = ~np.isfinite(m)
                m_safe = np.where(empty, 0.0, m)
                e = np.exp(s - m_safe[:, None])          # exp(-inf) = 0 on masked entries
                l = e.sum(axis=1)
                with np.errstate(divide="ignore"):
                    L[h, rows] = np.where(empty, NEG_INF, m_safe + np.log(l))
                num = e @ Vd
                O[rows, h, :] = np.where(empty[:, None], 0.0, num / np.where(empty, 1.0, l)[:, None])
    return O, L


def lse_merge(o_a, lse_a, o_b, lse_b):
    """Exact combination of two partials of the same rows (ring CP merge).

    L = log(e^La + e^Lb);  O = e^(La-L) O_a + e^(Lb-L) O_b.  (0, -inf) is the
    identity; two empty partials stay empty.  O [N,H,dv], LSE [H,N].
    """
    Oa, Ob = _f64(o_a), _f64(o_b)
    La, Lb = _f64(lse_a), _f64(lse_b)
    M = np.maximum(La, Lb)
    empty = ~np.isfinite(M)
    Ms = np.where(empty, 0.0, M)
    wa = np.exp(La - Ms)
    wb = np.exp(Lb - Ms)
    tot = wa + wb
    with np.errstate(divide="ignore"):
        L = np.where(empty, NEG_INF, Ms + np.log(np.where(empty, 1.0, tot)))
    fa = np.where(empty, 0.0, wa / np.where(empty, 1.0, tot))
    fb = np.where(empty, 0.0, wb / np.where(empty, 1.0, tot))
    O = fa.T[:, :, None] * Oa + fb.T[:, :, None] * Ob
    return O, L


def attn_bwd(q, k, v, o, lse, do, cu_seqlens, q_segs, kv_segs, scale: Optional[float] = None,
             heads: Optional[Iterable[int]] = None, q_rows: Optional[np.ndarray] = None):
    """Gradients of one ring step, given the final merged O and LSE of the rows.

    Returns dQ [Nq,H,dqk] (this step's contribution), dK [Nk,Hkv,dqk], dV [Nk,Hkv,dv]
    (with grouped K/V heads, a K/V head's gradient sums over the query heads of its group).
    ``q_rows`` restricts the queries taken into account: dQ is then computed for
    those rows only, and dK/dV hold only their contributions (complete for a key
    when every query that sees it is selected).
    """
    Q, K, V, O, dO = (np.asarray(x) for x in (q, k, v, o, do))   # fp64 slice by slice
    L = _f64(lse)
    nq, H, dqk = Q.shape
    grp = _group(H, K.shape[1])
    tau = default_scale(dqk) if scale is None else float(scale)
    qpos, kpos = row_positions(q_segs), row_positions(kv_segs)
    dQ = np.zeros(Q.shape)
    dK = np.zeros(K.shape)
    dV = np.zeros(V.shape)
    sel = np.ones(nq, bool) if q_rows is None else np.isin(np.arange(nq), q_rows)
    for h in (range(H) if heads is None else heads):
        D = np.einsum("nc,nc->n", _f64(dO[:, h, :]), _f64(O[:, h, :]))
        for qi, ki in _groups(cu_seqlens, qpos, kpos):
            qi = qi[sel[qi]]
            if len(qi) == 0 or len(ki) == 0:
                continue
            kh = h // grp
            Kd, Vd = _f64(K[ki, kh, :]), _f64(V[ki, kh, :])
            step = max(1, _SCORE_BLOCK // len(ki))
            for b in range(0, len(qi), step):
                rows = qi[b:b + step]
                Qr, dOr = _f64(Q[rows, h, :]), _f64(dO[rows, h, :])
                s = tau * (Qr @ Kd.T)
                vis = kpos[ki][None, :] <= qpos[rows][:, None]
                s = np.where(vis, s, NEG_INF)
                lse_r = L[h, rows]
                shift = np.where(np.isfinite(lse_r), lse_r, 0.0)
                p = np.exp(s - shift[:, None])             # 0 on masked entries
                p[~np.isfinite(lse_r)] = 0.0
                dV[ki, kh, :] += p.T @ dOr
                dp = dOr @ Vd.T
                ds = p * (dp - D[rows][:, None])
                dQ[rows, h, :] += tau * (ds @ Kd)
                dK[ki, kh, :] += tau * (ds.T @ Qr)
    return dQ, dK, dV


# ------------------------------------------------------------------ closed forms
# With every logit equal (Q = 0 or K = 0) the softmax is uniform over the visible
# keys, so the whole computation has a closed form needing only prefix sums.
# These give exact references at any size.

def _visible_ranges(cu_seqlens, qpos, kv_segs):
    """For each query, per KV segment, the local key-row range [a, b) it sees."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    lo = cu[doc_of(cu, qpos)]  # start of the query's document
    out = []
    base = 0
    for s, n in kv_segs:
        a = np.clip(lo, s, s + n) - s
        b = np.clip(qpos + 1, s, s + n) - s
        b = np.maximum(a, b)
        out.append((base + a, base + b))
        base += n
    return out


def uniform_fwd(v, cu_seqlens, q_segs, kv_segs, heads=None, n_q_heads=None):
    """O and LSE when all logits are equal: O_i = mean of visible v, LSE_i = ln n_i.
    ``n_q_heads`` (default: as many as V has) gives grouped K/V heads: query head h
    averages V head h // (n_q_heads / Hkv)."""
    V = _f64(v)
    qpos = row_positions(q_segs)
    nk, Hkv, dv = V.shape
    H = Hkv if n_q_heads is None else int(n_q_heads)
    grp = _group(H, Hkv)
    rng = _visible_ranges(cu_seqlens, qpos, kv_segs)
    n = sum(b - a for a, b in rng).astype(np.float64)
    O = np.zeros((len(qpos), H, dv))
    for h in (range(H) if heads is None else heads):
        pre = np.zeros((nk + 1, dv))
        np.cumsum(V[:, h // grp, :], axis=0, out=pre[1:])
        acc = np.zeros((len(qpos), dv))
        for a, b in rng:
            acc += pre[b] - pre[a]
        O[:, h, :] = np.where(n[:, None] > 0, acc / np.maximum(n, 1.0)[:, None], 0.0)
    with np.errstate(divide="ignore"):
        L = np.where(n > 0, np.log(np.maximum(n, 1.0)), NEG_INF)
    return O, np.broadcast_to(L, (H, len(qpos))).copy(), n


def uniform_bwd_k0(q, v, o, do, n_total, cu_seqlens, q_segs, kv_segs, key_rows,
                   scale=None, heads=None):
    """dK and dV rows of one ring step when K = 0, so P_ij = 1/n_i on visible pairs.

    ``o`` is the final merged output and ``n_total`` [Nq] the number of keys each
    row sees over the whole ring.  For a key j of this step's chunk, with the sums
    over the queries i that see it:
        dV_j = sum_i dO_i / n_i,   dK_j = tau * sum_i (<dO_i, v_j> - D_i) q_i / n_i.
    (dQ is exactly zero since K = 0.)  With grouped K/V heads (v has Hkv < H heads) the
    gradient of K/V head g sums these over its query heads g*grp .. g*grp + grp-1,
    grp = H / Hkv (Sec. 3.5: one K/V head serves a group of query heads).  ``heads``
    selects K/V heads.  Returns arrays [len(key_rows), len(heads), d].
    """
    Q, V, O, dO = _f64(q), _f64(v), _f64(o), _f64(do)
    nq, H, dqk = Q.shape
    Hkv = V.shape[1]
    grp = _group(H, Hkv)
    tau = default_scale(dqk) if scale is None else float(scale)
    qpos, kpos = row_positions(q_segs), row_positions(kv_segs)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    qdoc = doc_of(cu, qpos)
    kdoc = doc_of(cu, kpos)
    key_rows = np.asarray(key_rows)
    hs = list(range(Hkv) if heads is None else heads)
    dK = np.zeros((len(key_rows), len(hs), dqk))
    dV = np.zeros((len(key_rows), len(hs), V.shape[2]))
    inv_n = np.where(n_total > 0, 1.0 / np.maximum(n_total, 1), 0.0)
    for hi, g in enumerate(hs):
        for h in range(g * grp, (g + 1) * grp):
            D = np.einsum("nc,nc->n", dO[:, h, :], O[:, h, :])
            for r, j in enumerate(key_rows):
                sees = (qdoc == kdoc[j]) & (qpos >= kpos[j])
                w = inv_n[sees]
                dV[r, hi] += (w[:, None] * dO[sees, h, :]).sum(axis=0)
                coef = w * (dO[sees, h, :] @ V[j, g, :] - D[sees])
                dK[r, hi] += tau * (coef[:, None] * Q[sees, h, :]).sum(axis=0)
    return dK, dV


def visible_pairs_bruteforce(cu_seqlens, q_segs, kv_segs) -> int:
    """Number of visible (query, key) pairs per head, by enumeration (small inputs)."""
    qpos, kpos = row_positions(q_segs), row_positions(kv_segs)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    qd, kd = doc_of(cu, qpos), doc_of(cu, kpos)
    vis = (qd[:, None] == kd[None, :]) & (kpos[None, :] <= qpos[:, None])
    return int(vis.sum())
