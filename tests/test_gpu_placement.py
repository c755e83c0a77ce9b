"""One rank of a scheduled batch, end to end on the GPU: the scheduler places the batch
(Alg. 1), placement.rank_share turns one rank's group into its attention problems, the
library runs them ring step by ring step through the C ABI, and every output of the
rank's rows and head shard matches the fp64 oracle's unsplit attention of its documents."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_34318_amd import hydra, inputs, placement, ring

from gpu_util import assert_grad_close, assert_lse_close, assert_o_close, dev_bf16, f32
from test_placement import _batch

pytestmark = pytest.mark.gpu
D_QK, D_V = 192, 128


def _run_part(part, sh, H):
    """Inputs drawn for the part's whole window and every model head, sliced to the rank's
    rows and heads; returns (GPU results, oracle results)."""
    total = part.cu[-1]
    win = [(0, total)]
    full = {t: inputs.rows(t, win, H, d, seed=5, dist="sharp") for t, d in (("q", D_QK), ("k", D_QK), ("v", D_V),
                                                                           ("do", D_V))}
    hs = slice(sh.head0, sh.head0 + sh.n_heads)
    ks = slice(sh.kv_head0, sh.kv_head0 + sh.n_kv_heads)
    rows = lambda segs: np.concatenate([np.arange(a, a + n) for a, n in segs]) if segs else np.zeros(0, int)
    qr = rows(part.q_segs)
    q, do = full["q"][qr][:, hs], full["do"][qr][:, hs]
    kv = [(full["k"][rows(st)][:, ks], full["v"][rows(st)][:, ks]) for st in part.kv_steps]
    nkv = sh.n_kv_heads if sh.n_kv_heads != sh.n_heads else 0
    share = ring.make_share(part.cu, sh.n_heads, part.q_segs, part.kv_steps, n_kv_heads=nkv)
    qd, dod = dev_bf16(q), dev_bf16(do)
    kvd = [(dev_bf16(k), dev_bf16(v)) for k, v in kv]
    o, lse, _ = ring.forward(share, qd, kvd)
    dq = torch.zeros((share.nq, sh.n_heads, D_QK), device="cuda")
    dkv = [(torch.zeros((k.shape[0], sh.n_kv_heads, D_QK), device="cuda"),
            torch.zeros((k.shape[0], sh.n_kv_heads, D_V), device="cuda")) for k, _ in kv]
    ring.backward(share, qd, kvd, dod, dq, dkv)
    torch.cuda.synchronize()
    # the oracle: the rank's rows against every key of its documents, unsplit
    union = [s for st in part.kv_steps for s in st]
    k_all = np.concatenate([f32(k) for k, _ in kv])
    v_all = np.concatenate([f32(v) for _, v in kv])
    O, L = oracle.attn_fwd(f32(q), k_all, v_all, part.cu, part.q_segs, union)
    ref_dq = np.zeros(q.shape)
    ref_dkv = []
    for st, (k, v) in zip(part.kv_steps, kv):
        a, b, c = oracle.attn_bwd(f32(q), f32(k), f32(v), O, L, f32(do), part.cu, part.q_segs, st)
        ref_dq += a
        ref_dkv.append((b, c))
    got = {"o": o.cpu().numpy(), "lse": lse.cpu().numpy(), "dq": dq.cpu().numpy(),
           "dkv": [(a.cpu().numpy(), b.cpu().numpy()) for a, b in dkv]}
    return got, {"o": O, "lse": L, "dq": ref_dq, "dkv": ref_dkv}


def _check(got, ref, rank):
    assert_o_close(got["o"], ref["o"], what=f"O rank {rank}")
    assert_lse_close(got["lse"], ref["lse"], what=f"LSE rank {rank}")
    assert_grad_close(got["dq"], ref["dq"], what=f"dQ rank {rank}")
    for i, ((a, b), (c, d)) in enumerate(zip(got["dkv"], ref["dkv"])):
        if np.linalg.norm(c) > 0:
            assert_grad_close(a, c, what=f"dK step {i}")
            assert_grad_close(b, d, what=f"dV step {i}")


def test_scheduled_rank_shares_match_the_oracle():
    """8 ranks, 2 heads: micro-batch 0 is one 64K-token sequence over all 8 ranks (cp_u = 2,
    cp_r = 4: four ring steps over zigzag chunks); in micro-batch 2, the ring group of 4
    ranks holding 62 piggybacked documents (2-document sub-shares) and the non-ring group
    holding the most documents."""
    lens = _batch()
    G, B, H = 8, 32768, 2
    mb, st, sz, _ = hydra.schedule(lens, G, B, pp=4, theta_over_c=1.0)
    first = placement.rank_share(lens, mb, st, sz, 0, 3, H)
    assert (first.k, first.cp_u, first.cp_r, first.rho, len(first.parts)) == (8, 2, 4, 1, 1)
    got, ref = _run_part(first.parts[0], first, H)
    _check(got, ref, first.rank)
    cands = [placement.rank_share(lens, mb, st, sz, 2, r, H) for r in range(G)]
    ringed = max((c for c in cands if c is not None and c.cp_r > 1),
                 key=lambda c: (sum(len(p.seqs) for p in c.parts), -c.rank))
    plain = max((c for c in cands if c is not None and c.cp_r == 1), key=lambda c: (len(c.parts[0].seqs), -c.rank))
    assert ringed.cp_r == 2 and len(ringed.parts) > 2 and len(plain.parts[0].seqs) > 2
    for sh, parts in ((ringed, ringed.parts[:3]), (plain, plain.parts[:1])):
        for part in parts:
            got, ref = _run_part(part, sh, H)
            _check(got, ref, sh.rank)
