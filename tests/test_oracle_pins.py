"""Pins for the fp64 oracle: facts fixed by the definition, by a library routine or
by brute force, chosen so that a plausible slip in the oracle (dropped scale, wrong
diagonal, transposed operand, wrong LSE base, missing D term, wrong merge weight)
fails at least one of them.  CPU only."""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import attention as A
from paper_2609_34318_amd import inputs

D_QK, D_V = 192, 128


def _f32(bits):
    return inputs.bf16_bits_to_f32(bits)


def _tensors(cu, q_segs, kv_segs, H, seed=0, dist="paper", do=False):
    q = _f32(inputs.rows("q", q_segs, H, D_QK, seed, dist))
    k = _f32(inputs.rows("k", kv_segs, H, D_QK, seed, dist))
    v = _f32(inputs.rows("v", kv_segs, H, D_V, seed, dist))
    g = _f32(inputs.rows("do", q_segs, H, D_V, seed, dist)) if do else None
    return q, k, v, g


def _block_causal_mask(cu, qpos, kpos):
    cu = np.asarray(cu)
    qd = np.searchsorted(cu, qpos, side="right") - 1
    kd = np.searchsorted(cu, kpos, side="right") - 1
    return (qd[:, None] == kd[None, :]) & (kpos[None, :] <= qpos[:, None])


def _sdpa(q, k, v, mask=None, causal=False, grad=None, scale=None):
    """torch fp64 CPU scaled_dot_product_attention, heads first."""
    tq = torch.tensor(q, dtype=torch.float64).permute(1, 0, 2).contiguous().requires_grad_(grad is not None)
    tk = torch.tensor(k, dtype=torch.float64).permute(1, 0, 2).contiguous().requires_grad_(grad is not None)
    tv = torch.tensor(v, dtype=torch.float64).permute(1, 0, 2).contiguous().requires_grad_(grad is not None)
    m = None if mask is None else torch.tensor(mask)
    o = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=m, is_causal=causal, scale=scale)
    if grad is None:
        return o.detach().permute(1, 0, 2).numpy(), None
    o.backward(torch.tensor(grad, dtype=torch.float64).permute(1, 0, 2))
    gr = [t.grad.permute(1, 0, 2).numpy() for t in (tq, tk, tv)]
    return o.detach().permute(1, 0, 2).numpy(), gr


# ------------------------------------------------------------ library special cases

def test_fwd_single_doc_equals_torch_causal_sdpa():
    cu = [0, 300]
    segs = [(0, 300)]
    q, k, v, _ = _tensors(cu, segs, segs, 3, dist="sharp")
    O, L = oracle.attn_fwd(q, k, v, cu, segs, segs)
    ref, _ = _sdpa(q, k, v, causal=True)
    np.testing.assert_allclose(O, ref, rtol=0, atol=1e-12)


def test_fwd_packed_docs_equal_sdpa_with_block_causal_mask():
    cu = [0, 37, 38, 150, 211, 400]
    segs = [(0, 400)]
    q, k, v, _ = _tensors(cu, segs, segs, 2, dist="spiky")
    O, L = oracle.attn_fwd(q, k, v, cu, segs, segs)
    pos = np.arange(400)
    ref, _ = _sdpa(q, k, v, mask=_block_causal_mask(cu, pos, pos))
    np.testing.assert_allclose(O, ref, rtol=0, atol=1e-12)


def test_bwd_equals_torch_autograd_through_sdpa():
    cu = [0, 50, 51, 170]
    segs = [(0, 170)]
    q, k, v, g = _tensors(cu, segs, segs, 2, dist="sharp", do=True)
    O, L = oracle.attn_fwd(q, k, v, cu, segs, segs)
    pos = np.arange(170)
    ref_o, (rq, rk, rv) = _sdpa(q, k, v, mask=_block_causal_mask(cu, pos, pos), grad=g)
    dq, dk, dv = oracle.attn_bwd(q, k, v, O, L, g, cu, segs, segs)
    for a, b in ((dq, rq), (dk, rk), (dv, rv)):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-11 * max(1.0, np.abs(b).max()))


def test_nondefault_scale_equals_sdpa_with_scaled_query():
    cu = [0, 90]
    segs = [(0, 90)]
    q, k, v, _ = _tensors(cu, segs, segs, 1, dist="sharp")
    O, _ = oracle.attn_fwd(q, k, v, cu, segs, segs, scale=0.3)
    ref, _ = _sdpa(q, k, v, causal=True, scale=0.3)
    np.testing.assert_allclose(O, ref, rtol=0, atol=1e-12)


# ------------------------------------------------------------ brute force

def _brute(q, k, v, cu, qpos, kpos, tau):
    nq, H, _ = q.shape
    O = np.zeros((nq, H, v.shape[2]))
    L = np.full((H, nq), -np.inf)
    docs = lambda p: max(d for d in range(len(cu) - 1) if cu[d] <= p)
    for h in range(H):
        for i in range(nq):
            s = []
            for j in range(k.shape[0]):
                if docs(int(kpos[j])) == docs(int(qpos[i])) and kpos[j] <= qpos[i]:
                    s.append((j, tau * sum(float(q[i, h, c]) * float(k[j, h, c]) for c in range(q.shape[2]))))
            if not s:
                continue
            z = sum(math.exp(x) for _, x in s)
            L[h, i] = math.log(z)
            for j, x in s:
                O[i, h] += math.exp(x) / z * v[j, h].astype(np.float64)
    return O, L


def test_fwd_bruteforce_tiny_split_chunks():
    cu = [0, 5, 12]
    q_segs = [(0, 12)]
    kv_segs = [(4, 3), (9, 3)]          # positions 4,5,6, 9,10,11: crosses a doc boundary
    q, k, v, _ = _tensors(cu, q_segs, kv_segs, 2, dist="spiky")
    O, L = oracle.attn_fwd(q, k, v, cu, q_segs, kv_segs)
    bO, bL = _brute(q, k, v, cu, A.row_positions(q_segs), A.row_positions(kv_segs), 1 / math.sqrt(D_QK))
    np.testing.assert_array_equal(np.isinf(L), np.isinf(bL))
    fin = np.isfinite(bL)
    np.testing.assert_allclose(L[fin], bL[fin], rtol=0, atol=1e-12)
    np.testing.assert_allclose(O, bO, rtol=0, atol=1e-12)
    assert np.isinf(L[:, :4]).all() and (O[:4] == 0).all()      # rows 0-3 see nothing


def test_visible_pairs_bruteforce_matches_closed_count():
    # causal within docs, unsplit: sum s(s+1)/2
    lens = [64, 128, 320]
    cu = inputs.cu_from_lengths(lens)
    assert A.visible_pairs_bruteforce(cu, [(0, 512)], [(0, 512)]) == sum(s * (s + 1) // 2 for s in lens)


# ------------------------------------------------------------ invariants of the definition

def test_rows_sum_to_one():
    cu = [0, 33, 160, 161, 300]
    segs = [(0, 300)]
    q, k, v, _ = _tensors(cu, segs, segs, 2, dist="spiky")
    O, L = oracle.attn_fwd(q, k, v, cu, segs, segs)
    # with V = 1 the output is exactly the row sum of the softmax weights
    O1, L1 = oracle.attn_fwd(q, k, np.ones_like(v), cu, segs, segs)
    np.testing.assert_allclose(O1, 1.0, rtol=0, atol=1e-13)
    np.testing.assert_array_equal(L1, L)


def test_constant_v_gives_constant():
    cu = inputs.cu_from_lengths([64, 128, 320])
    q, k, v, _ = _tensors(cu, [(0, 512)], [(0, 512)], 4)
    O, _ = oracle.attn_fwd(q, k, np.full_like(v, 0.5), cu, [(0, 512)], [(0, 512)])
    np.testing.assert_allclose(O, 0.5, rtol=0, atol=1e-14)


def test_single_key_rows_return_their_value():
    cu = inputs.cu_from_lengths([64, 128, 320])
    q, k, v, _ = _tensors(cu, [(0, 512)], [(0, 512)], 4, dist="sharp")
    O, L = oracle.attn_fwd(q, k, v, cu, [(0, 512)], [(0, 512)])
    tau = 1 / math.sqrt(D_QK)
    for r in (0, 64, 192):                       # first token of each document
        np.testing.assert_allclose(O[r], v[r], rtol=0, atol=1e-15)
        s_rr = tau * np.einsum("hc,hc->h", q[r].astype(np.float64), k[r].astype(np.float64))
        np.testing.assert_allclose(L[:, r], s_rr, rtol=0, atol=1e-14)


def test_uniform_logits_closed_form_lse_is_log_count():
    cu = inputs.cu_from_lengths([64, 128, 320])
    segs = [(0, 512)]
    _, k, v, _ = _tensors(cu, segs, segs, 2)
    O, L = oracle.attn_fwd(np.zeros((512, 2, D_QK)), k, v, cu, segs, segs)
    pos = np.arange(512)
    n = pos - np.asarray(cu)[np.searchsorted(cu, pos, side="right") - 1] + 1
    np.testing.assert_allclose(L, np.log(n)[None, :].repeat(2, 0), rtol=0, atol=1e-13)
    Uo, UL, un = oracle.uniform_fwd(v, cu, segs, segs)
    np.testing.assert_array_equal(un, n)
    np.testing.assert_allclose(Uo, O, rtol=0, atol=1e-13)
    np.testing.assert_allclose(UL, L, rtol=0, atol=1e-13)


def test_uniform_closed_form_on_split_chunks_merges_to_unsplit():
    cu = [0, 1000, 1400]
    q_segs = [(200, 300), (1100, 300)]
    steps = [[(0, 350)], [(350, 650)], [(1000, 400)]]
    v_all = _f32(inputs.rows("v", [(0, 1400)], 2, D_V))
    parts = []
    for s in steps:
        v = _f32(inputs.rows("v", s, 2, D_V))
        Uo, UL, _ = oracle.uniform_fwd(v, cu, q_segs, s)
        parts.append((Uo, UL))
    Om, Lm = parts[0]
    for Oi, Li in parts[1:]:
        Om, Lm = oracle.lse_merge(Om, Lm, Oi, Li)
    Uo, UL, _ = oracle.uniform_fwd(v_all, cu, q_segs, [(0, 1400)])
    np.testing.assert_allclose(Om, Uo, rtol=0, atol=1e-12)
    np.testing.assert_allclose(Lm, UL, rtol=0, atol=1e-12)


def test_bwd_finite_differences():
    cu = [0, 5, 12]
    segs = [(0, 12)]
    q, k, v, g = _tensors(cu, segs, segs, 2, dist="sharp", do=True)
    q, k, v, g = (x.astype(np.float64) for x in (q, k, v, g))
    O, L = oracle.attn_fwd(q, k, v, cu, segs, segs)
    dq, dk, dv = oracle.attn_bwd(q, k, v, O, L, g, cu, segs, segs)

    def loss(q_, k_, v_):
        o, _ = oracle.attn_fwd(q_, k_, v_, cu, segs, segs)
        return float((o * g).sum())

    rng = np.random.default_rng(1)
    eps = 1e-6
    for name, x, grad in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        for _ in range(6):
            idx = tuple(int(rng.integers(0, s)) for s in x.shape)
            xp, xm = x.copy(), x.copy()
            xp[idx] += eps
            xm[idx] -= eps
            args = {"q": (q, k, v), "k": (q, k, v), "v": (q, k, v)}[name]
            sel = "qkv".index(name)
            ap, am = list(args), list(args)
            ap[sel], am[sel] = xp, xm
            fd = (loss(*ap) - loss(*am)) / (2 * eps)
            assert abs(fd - grad[idx]) <= 1e-6 * max(1.0, abs(fd)), (name, idx, fd, grad[idx])


def test_bwd_column_sums():
    # sum_j dK_j = 0 (rows of dS sum to zero) and sum_j dV_j = sum_i dO_i, per doc and head
    cu = [0, 40, 41, 200]
    segs = [(0, 200)]
    q, k, v, g = _tensors(cu, segs, segs, 2, dist="spiky", do=True)
    O, L = oracle.attn_fwd(q, k, v, cu, segs, segs)
    dq, dk, dv = oracle.attn_bwd(q, k, v, O, L, g, cu, segs, segs)
    for a, b in zip(cu[:-1], cu[1:]):
        np.testing.assert_allclose(dk[a:b].sum(0), 0.0, atol=1e-12)
        np.testing.assert_allclose(dv[a:b].sum(0), g[a:b].astype(np.float64).sum(0), atol=1e-12)


# ------------------------------------------------------------ ring split + exact merge

def _split_and_merge(q, kv_all, cu, q_segs, steps, all_segs):
    k_all, v_all = kv_all
    pos_all = A.row_positions(all_segs)
    O = np.zeros((q.shape[0], q.shape[1], D_V))
    L = np.full((q.shape[1], q.shape[0]), -np.inf)
    for s in steps:
        idx = np.concatenate([np.nonzero((pos_all >= a) & (pos_all < a + n))[0] for a, n in s]) if s else np.zeros(0, int)
        Oi, Li = oracle.attn_fwd(q, k_all[idx], v_all[idx], cu, q_segs, s)
        O, L = oracle.lse_merge(O, L, Oi, Li)
    return O, L


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_random_ring_split_merges_to_unsplit(seed):
    rng = np.random.default_rng(seed)
    cu = [0, 77, 300, 301, 480]
    all_segs = [(0, 480)]
    q, k, v, _ = _tensors(cu, all_segs, all_segs, 2, seed=seed, dist="spiky")
    cuts = np.sort(rng.choice(np.arange(0, 481), size=4, replace=True))
    bounds = [0, *cuts.tolist(), 480]
    steps = [[(a, b - a)] for a, b in zip(bounds[:-1], bounds[1:])]   # may contain empty pieces
    rng.shuffle(steps)
    O, L = _split_and_merge(q, (k, v), cu, all_segs, steps, all_segs)
    Oref, Lref = oracle.attn_fwd(q, k, v, cu, all_segs, all_segs)
    np.testing.assert_allclose(O, Oref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(L, Lref, rtol=0, atol=1e-12)


def test_zigzag_share_merges_to_unsplit_rows():
    # 1 doc of 256 tokens, cp_r = 2: rank 0 holds quarters 0 and 3
    cu = [0, 256]
    q_segs = list(inputs.zigzag_segments(256, 2, 0))
    steps = [list(inputs.zigzag_segments(256, 2, r)) for r in (0, 1)]
    full = [(0, 256)]
    qf, kf, vf, _ = _tensors(cu, full, full, 2, dist="sharp")
    q = _f32(inputs.rows("q", q_segs, 2, D_QK, 0, "sharp"))
    O, L = _split_and_merge(q, (kf, vf), cu, q_segs, steps, full)
    Oref, Lref = oracle.attn_fwd(qf, kf, vf, cu, full, full)
    rows = A.row_positions(q_segs)
    np.testing.assert_allclose(O, Oref[rows], rtol=0, atol=1e-12)
    np.testing.assert_allclose(L, Lref[:, rows], rtol=0, atol=1e-12)


def test_merge_identity_and_commutativity():
    rng = np.random.default_rng(3)
    Oa, La = rng.standard_normal((7, 2, 4)), rng.standard_normal((2, 7))
    Ob, Lb = rng.standard_normal((7, 2, 4)), rng.standard_normal((2, 7))
    La[0, 2] = -np.inf
    Oa[2, 0] = 0.0
    O, L = oracle.lse_merge(Oa, La, np.zeros_like(Oa), np.full_like(La, -np.inf))
    np.testing.assert_array_equal(O, Oa)
    np.testing.assert_array_equal(L, La)
    O1, L1 = oracle.lse_merge(Oa, La, Ob, Lb)
    O2, L2 = oracle.lse_merge(Ob, Lb, Oa, La)
    np.testing.assert_allclose(O1, O2, atol=1e-15)
    np.testing.assert_allclose(L1, L2, atol=1e-15)
    # both empty stays empty, without NaN
    E, EL = oracle.lse_merge(np.zeros((1, 1, 4)), np.full((1, 1), -np.inf), np.zeros((1, 1, 4)), np.full((1, 1), -np.inf))
    assert np.isneginf(EL).all() and (E == 0).all()


def test_bwd_ring_split_sums_to_unsplit():
    cu = [0, 120, 260]
    full = [(0, 260)]
    q, k, v, g = _tensors(cu, full, full, 2, dist="spiky", do=True)
    O, L = oracle.attn_fwd(q, k, v, cu, full, full)
    dq, dk, dv = oracle.attn_bwd(q, k, v, O, L, g, cu, full, full)
    steps = [[(0, 90)], [(90, 100), (230, 30)], [(190, 40)]]
    dq_acc = np.zeros_like(dq)
    for s in steps:
        idx = A.row_positions(s)
        sq, sk, sv = oracle.attn_bwd(q, k[idx], v[idx], O, L, g, cu, full, s)
        dq_acc += sq
        np.testing.assert_allclose(sk, dk[idx], atol=1e-13)
        np.testing.assert_allclose(sv, dv[idx], atol=1e-13)
    np.testing.assert_allclose(dq_acc, dq, atol=1e-13)


def test_row_subset_and_head_subset_match_full():
    cu = [0, 100, 333]
    segs = [(0, 333)]
    q, k, v, _ = _tensors(cu, segs, segs, 3, dist="sharp")
    O, L = oracle.attn_fwd(q, k, v, cu, segs, segs)
    rows = np.array([0, 99, 100, 101, 332])
    Os, Ls = oracle.attn_fwd(q, k, v, cu, segs, segs, heads=[1], q_rows=rows)
    np.testing.assert_array_equal(Os[rows, 1], O[rows, 1])
    np.testing.assert_array_equal(Ls[1, rows], L[1, rows])
    assert np.isneginf(Ls[0]).all()


def test_heads_and_documents_are_independent():
    lens = [40, 70, 25]
    cu = inputs.cu_from_lengths(lens)
    segs = [(0, 135)]
    q, k, v, _ = _tensors(cu, segs, segs, 3, dist="sharp")
    O, L = oracle.attn_fwd(q, k, v, cu, segs, segs)
    hp = [2, 0, 1]
    Oh, Lh = oracle.attn_fwd(q[:, hp], k[:, hp], v[:, hp], cu, segs, segs)
    np.testing.assert_array_equal(Oh, O[:, hp])
    # reorder documents: 25, 40, 70
    order = [2, 0, 1]
    starts = np.asarray(cu)[:-1]
    perm = np.concatenate([np.arange(starts[d], starts[d] + lens[d]) for d in order])
    cu2 = inputs.cu_from_lengths([lens[d] for d in order])
    O2, L2 = oracle.attn_fwd(q[perm], k[perm], v[perm], cu2, segs, segs)
    np.testing.assert_allclose(O2, O[perm], atol=1e-15)
    np.testing.assert_allclose(L2, L[:, perm], atol=1e-14)


def test_uniform_bwd_k0_matches_general_oracle():
    cu = [0, 100, 230]
    full = [(0, 230)]
    q, _, v, g = _tensors(cu, full, full, 2, dist="sharp", do=True)
    k = np.zeros((230, 2, D_QK))
    O, L = oracle.attn_fwd(q, k, v, cu, full, full)
    dq, dk, dv = oracle.attn_bwd(q, k, v, O, L, g, cu, full, full)
    np.testing.assert_array_equal(dq, 0.0)
    Uo, UL, n = oracle.uniform_fwd(v, cu, full, full)
    keys = np.array([0, 5, 99, 100, 150, 229])
    # as a split: keys of the step chunk [(90, 60)] are local rows 0..59
    s = [(90, 60)]
    idx = A.row_positions(s)
    uk, uv = oracle.uniform_bwd_k0(q, v[idx], Uo, g, n, cu, full, s, key_rows=np.arange(60))
    np.testing.assert_allclose(uk, dk[idx], atol=1e-12)
    np.testing.assert_allclose(uv, dv[idx], atol=1e-12)
    uk, uv = oracle.uniform_bwd_k0(q, v, Uo, g, n, cu, full, full, key_rows=keys)
    np.testing.assert_allclose(uk, dk[keys], atol=1e-12)
    np.testing.assert_allclose(uv, dv[keys], atol=1e-12)


def test_uniform_bwd_k0_grouped_heads_matches_general_oracle():
    """Grouped K/V heads (8 query heads, 2 K/V heads): the closed form sums each K/V
    head's gradient over its four query heads and indexes V by the group, as the general
    oracle (pinned against SDPA on repeated heads) does."""
    cu = [0, 70, 190]
    full = [(0, 190)]
    H, Hkv = 8, 2
    q, _, _, g = _tensors(cu, full, full, H, dist="sharp", do=True)
    _, _, v, _ = _tensors(cu, full, full, Hkv, dist="sharp")
    k = np.zeros((190, Hkv, D_QK))
    O, L = oracle.attn_fwd(q, k, v, cu, full, full)
    dq, dk, dv = oracle.attn_bwd(q, k, v, O, L, g, cu, full, full)
    np.testing.assert_array_equal(dq, 0.0)
    Uo, UL, n = oracle.uniform_fwd(v, cu, full, full, n_q_heads=H)
    np.testing.assert_allclose(Uo, O, atol=1e-12)
    keys = np.array([0, 1, 69, 70, 71, 150, 189])
    uk, uv = oracle.uniform_bwd_k0(q, v, Uo, g, n, cu, full, full, key_rows=keys)
    assert uk.shape == (len(keys), Hkv, D_QK) and uv.shape == (len(keys), Hkv, D_V)
    np.testing.assert_allclose(uk, dk[keys], atol=1e-12)
    np.testing.assert_allclose(uv, dv[keys], atol=1e-12)
    uk1, uv1 = oracle.uniform_bwd_k0(q, v, Uo, g, n, cu, full, full, key_rows=keys, heads=[1])
    np.testing.assert_allclose(uk1[:, 0], dk[keys, 1], atol=1e-12)
    np.testing.assert_allclose(uv1[:, 0], dv[keys, 1], atol=1e-12)
    # a grouping that does not divide is refused rather than indexed past the end
    with pytest.raises(ValueError, match="divide"):
        oracle.uniform_bwd_k0(q[:, :7], v, Uo[:, :7], g[:, :7], n, cu, full, full, key_rows=keys)
    with pytest.raises(ValueError, match="divide"):
        oracle.uniform_bwd_k0(q, np.concatenate([v, v[:, :1]], axis=1), Uo, g, n, cu, full, full, key_rows=keys)


# ------------------------------------------------------------ input recipe

def test_packed_doc_list_reproduces_from_sampler():
    assert inputs.sample_packed_docs() == inputs.PACKED32K_DOCS
    assert sum(inputs.PACKED32K_DOCS) == 32768


def test_position_keyed_inputs_are_split_invariant():
    a = inputs.rows("k", [(4000, 300)], 2, D_QK)
    b = np.concatenate([inputs.rows("k", [(4000, 96)], 2, D_QK), inputs.rows("k", [(4096, 204)], 2, D_QK)])
    np.testing.assert_array_equal(a, b)


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.00390625, 1.01171875, -2.5e-3, 3.0e38], dtype=np.float32)
    t = torch.tensor(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(inputs.bf16_round_bits(x), t)


# ------------------------------------------------------------ grouped K/V heads (GQA)

@pytest.mark.parametrize("H,Hkv", [(4, 1), (4, 2), (6, 3)])
def test_gqa_fwd_bwd_equal_mha_on_repeated_heads(H, Hkv):
    """Grouped K/V heads are the same function as one K/V head per query head with every
    K/V head repeated over its group; the gradient of a shared head is the sum over its
    group (chain rule through the repeat).  The reference is torch SDPA on the repeated
    tensors, so the grouping, the head index map and the reduction are checked against an
    independent formulation."""
    cu = [0, 9, 20]
    segs = [(0, 20)]
    rng = np.random.default_rng(H * 10 + Hkv)
    q = rng.standard_normal((20, H, D_QK)) * 0.3
    k = rng.standard_normal((20, Hkv, D_QK)) * 0.3
    v = rng.standard_normal((20, Hkv, D_V))
    g = rng.standard_normal((20, H, D_V))
    grp = H // Hkv
    kr, vr = np.repeat(k, grp, axis=1), np.repeat(v, grp, axis=1)   # head i -> K/V head i // grp
    mask = _block_causal_mask(cu, np.arange(20), np.arange(20))
    o_ref, (dq_r, dk_r, dv_r) = _sdpa(q, kr, vr, mask=mask, grad=g)
    O, L = oracle.attn_fwd(q, k, v, cu, segs, segs)
    assert np.abs(O - o_ref).max() < 1e-12
    dq, dk, dv = oracle.attn_bwd(q, k, v, O, L, g, cu, segs, segs)
    assert dk.shape == k.shape and dv.shape == v.shape
    assert np.abs(dq - dq_r).max() < 1e-11
    assert np.abs(dk - dk_r.reshape(20, Hkv, grp, D_QK).sum(axis=2)).max() < 1e-11
    assert np.abs(dv - dv_r.reshape(20, Hkv, grp, D_V).sum(axis=2)).max() < 1e-11


def test_gqa_bwd_finite_differences_on_a_shared_head():
    cu = [0, 6, 11]
    segs = [(0, 11)]
    rng = np.random.default_rng(5)
    q = rng.standard_normal((11, 4, D_QK)) * 0.2
    k = rng.standard_normal((11, 2, D_QK)) * 0.2
    v = rng.standard_normal((11, 2, D_V))
    g = rng.standard_normal((11, 4, D_V))
    O, L = oracle.attn_fwd(q, k, v, cu, segs, segs)
    _, dk, dv = oracle.attn_bwd(q, k, v, O, L, g, cu, segs, segs)

    def loss(k_, v_):
        o, _ = oracle.attn_fwd(q, k_, v_, cu, segs, segs)
        return float((o * g).sum())

    eps = 1e-6
    for x, grad, is_k in ((k, dk, True), (v, dv, False)):
        for idx in ((3, 1, 7), (10, 0, 2), (6, 1, 100)):
            xp, xm = x.copy(), x.copy()
            xp[idx] += eps
            xm[idx] -= eps
            fd = (loss(xp, v) - loss(xm, v)) / (2 * eps) if is_k else (loss(k, xp) - loss(k, xm)) / (2 * eps)
            assert abs(fd - grad[idx]) <= 1e-6 * max(1.0, abs(fd)), (idx, fd, grad[idx])


def test_gqa_rejects_non_divisor_head_counts():
    q = np.zeros((4, 6, D_QK))
    k = np.zeros((4, 4, D_QK))
    v = np.zeros((4, 4, D_V))
    with pytest.raises(ValueError):
        oracle.attn_fwd(q, k, v, [0, 4], [(0, 4)], [(0, 4)])


def test_gqa_uniform_closed_form_matches_general_oracle():
    cu = [0, 7, 19]
    segs = [(0, 19)]
    rng = np.random.default_rng(9)
    v = rng.standard_normal((19, 2, D_V))
    q = np.zeros((19, 6, D_QK))
    k = rng.standard_normal((19, 2, D_QK))
    O, L = oracle.attn_fwd(q, k, v, cu, segs, segs)
    Ou, Lu, _ = oracle.uniform_fwd(v, cu, segs, segs, n_q_heads=6)
    assert np.abs(O - Ou).max() < 1e-12 and np.abs(L - Lu).max() < 1e-12
