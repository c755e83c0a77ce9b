"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Small and medium problems are compared element by element; the full-size workloads
(32K packed microbatch, 256K ring steps, 128K zigzag share) on sampled rows the oracle
computes one by one, on uniform-logit closed forms over every element, and on
identities that hold at any size."""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import attention as A
from paper_2609_34318_amd import hydra, inputs, ring

from gpu_util import (TOL_GRAD, TOL_LSE, TOL_O, assert_grad_close, assert_lse_close, assert_o_close,
                      dev_bf16, f32, rel_l2)

pytestmark = pytest.mark.gpu

D_QK, D_V = 192, 128
BENCH_DS = -1  # bench.py's default: stored-dS backward, passes sized to ring.DEFAULT_DS_BUDGET_BYTES


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hydra.lib()
    yield
    torch.cuda.synchronize()


def _run_share(cu, H, q_segs, steps, q_bits, kv_bits, do_bits=None, scale=0.0, Hkv=0, ds_kv_heads=0):
    """Forward (and backward if dO given) of a share; returns numpy results.  ds_kv_heads > 0:
    the backward stores dS for dQ (passes of that many K/V heads) where that path applies;
    BENCH_DS: passes as bench.py sizes them by default."""
    budget = ring.DEFAULT_DS_BUDGET_BYTES if ds_kv_heads == BENCH_DS else 0
    sh = ring.make_share(cu, H, q_segs, steps, softmax_scale=scale, n_kv_heads=Hkv, ds_kv_heads=ds_kv_heads,
                         ds_budget_bytes=budget)
    Hk = Hkv or H
    q = dev_bf16(q_bits)
    kv = [(dev_bf16(k), dev_bf16(v)) for k, v in kv_bits]
    o, lse, o16 = ring.forward(sh, q, kv)
    res = {"o": o.cpu().numpy(), "lse": lse.cpu().numpy(), "o16": o16.float().cpu().numpy()}
    if do_bits is not None:
        d_o = dev_bf16(do_bits)
        dq = torch.zeros((sh.nq, H, D_QK), dtype=torch.float32, device="cuda")
        dkv = [(torch.zeros((k.shape[0], Hk, D_QK), dtype=torch.float32, device="cuda"),
                torch.zeros((k.shape[0], Hk, D_V), dtype=torch.float32, device="cuda")) for k, _ in kv]
        ring.backward(sh, q, kv, d_o, dq, dkv)
        res["dq"] = dq.cpu().numpy()
        res["dkv"] = [(a.cpu().numpy(), b.cpu().numpy()) for a, b in dkv]
    torch.cuda.synchronize()
    return res


def _gen(cu, H, q_segs, steps, dist="paper", seed=0, bwd=False, Hkv=0):
    Hk = Hkv or H
    q = inputs.rows("q", q_segs, H, D_QK, seed, dist)
    kv = [(inputs.rows("k", s, Hk, D_QK, seed, dist), inputs.rows("v", s, Hk, D_V, seed, dist)) for s in steps]
    do = inputs.rows("do", q_segs, H, D_V, seed, dist) if bwd else None
    return q, kv, do


def _union(steps):
    return [seg for s in steps for seg in s]


def _oracle_share(cu, q_segs, steps, q, kv, do=None, scale=None):
    """Unsplit forward over the union of the steps' chunks, then per-step backward."""
    union = _union(steps)
    k_all = np.concatenate([f32(k) for k, _ in kv]) if kv else np.zeros((0, q.shape[1], D_QK), np.float32)
    v_all = np.concatenate([f32(v) for _, v in kv]) if kv else np.zeros((0, q.shape[1], D_V), np.float32)
    O, L = oracle.attn_fwd(f32(q), k_all, v_all, cu, q_segs, union, scale=scale)
    out = {"o": O, "lse": L}
    if do is not None:
        out["dq"] = np.zeros(q.shape)
        out["dkv"] = []
        for s, (k, v) in zip(steps, kv):
            dq, dk, dv = oracle.attn_bwd(f32(q), f32(k), f32(v), O, L, f32(do), cu, q_segs, s, scale=scale)
            out["dq"] += dq
            out["dkv"].append((dk, dv))
    return out


def _check_fwd(res, ref):
    assert_lse_close(res["lse"], ref["lse"])
    assert_o_close(res["o"], ref["o"])
    assert_o_close(res["o16"], ref["o"], what="O bf16")


def _check_bwd(res, ref):
    assert_grad_close(res["dq"], ref["dq"], what="dQ")
    for i, ((dk, dv), (rk, rv)) in enumerate(zip(res["dkv"], ref["dkv"])):
        if np.linalg.norm(rk) > 0:
            assert_grad_close(dk, rk, what=f"dK step {i}")
            assert_grad_close(dv, rv, what=f"dV step {i}")
        else:
            assert np.abs(dk).max() == 0 and np.abs(dv).max() == 0


# ----------------------------------------------------------------- small: element by element

def test_tiny_two_step_forward_partials_and_merge():
    w = inputs.WORKLOADS["tiny_2step"]
    cu, H = list(w.cu_seqlens), w.n_heads
    steps = [list(s) for s in w.kv_steps]
    q, kv, _ = _gen(cu, H, list(w.q_segs), steps)
    # each partial on its own
    for s, (k, v) in zip(steps, kv):
        res = _run_share(cu, H, list(w.q_segs), [s], q, [(k, v)])
        O, L = oracle.attn_fwd(f32(q), f32(k), f32(v), cu, list(w.q_segs), s)
        _check_fwd(res, {"o": O, "lse": L})
    # step B (keys 256..511) leaves rows 0..255 empty: the -inf path
    res = _run_share(cu, H, list(w.q_segs), steps, q, kv)
    _check_fwd(res, _oracle_share(cu, list(w.q_segs), steps, q, kv))


MEDIUM = {
    # documents with an empty one and single-token ones; lengths not multiples of any tile
    "contiguous_1step": ([0, 300, 300, 301, 1000, 1050, 1333], [(0, 1333)], [[(0, 1333)]]),
    "ragged_3step": ([0, 300, 300, 301, 1000, 1050, 1333], [(0, 1333)],
                     [[(0, 77)], [(77, 500), (1300, 33)], [(577, 723)]]),
    "zigzag_2step": ([0, 1024], list(inputs.zigzag_segments(1024, 2, 0)),
                     [list(inputs.zigzag_segments(1024, 2, 0)), list(inputs.zigzag_segments(1024, 2, 1))]),
    "q_subset_4seg": ([0, 200, 900, 1400], [(50, 100), (850, 200), (1300, 37), (0, 1)],
                      [[(0, 450)], [(450, 950)]]),
}


@pytest.mark.parametrize("dist", ["paper", "sharp", "spiky"])
@pytest.mark.parametrize("layout", list(MEDIUM))
def test_medium_forward_backward(layout, dist):
    cu, q_segs, steps = MEDIUM[layout]
    H = 3
    q, kv, do = _gen(cu, H, q_segs, steps, dist=dist, seed=1, bwd=True)
    res = _run_share(cu, H, q_segs, steps, q, kv, do)
    ref = _oracle_share(cu, q_segs, steps, q, kv, do)
    _check_fwd(res, ref)
    _check_bwd(res, ref)


@pytest.mark.parametrize("layout", ["ragged_3step", "zigzag_2step"])
@pytest.mark.parametrize("H,Hkv", [(8, 1), (8, 2), (6, 3)])
def test_gqa_medium_forward_backward(layout, H, Hkv):
    """Grouped K/V heads: query head i uses K/V head i // (H/Hkv); dK/dV of a K/V head sum
    over its group (the dK/dV kernel walks the group's query heads one after another)."""
    cu, q_segs, steps = MEDIUM[layout]
    q, kv, do = _gen(cu, H, q_segs, steps, dist="sharp", seed=2, bwd=True, Hkv=Hkv)
    res = _run_share(cu, H, q_segs, steps, q, kv, do, Hkv=Hkv)
    ref = _oracle_share(cu, q_segs, steps, q, kv, do)
    _check_fwd(res, ref)
    _check_bwd(res, ref)


# 32-aligned segments: the stored-dS backward applies (documents stay ragged)
ALIGNED = {
    "contiguous_1step": ([0, 300, 300, 301, 1000, 1050, 1344], [(0, 1344)], [[(0, 1344)]]),
    "ragged_docs_3step": ([0, 300, 300, 301, 1000, 1050, 1344], [(0, 1344)],
                          [[(0, 96)], [(96, 480), (1312, 32)], [(576, 736)]]),
    "zigzag_2step": ([0, 1024], list(inputs.zigzag_segments(1024, 2, 0)),
                     [list(inputs.zigzag_segments(1024, 2, 0)), list(inputs.zigzag_segments(1024, 2, 1))]),
    "q_subset_4seg": ([0, 200, 900, 1408], [(32, 128), (832, 224), (1280, 64), (0, 32)],
                      [[(0, 448)], [(448, 960)]]),
}


@pytest.mark.parametrize("dist", ["paper", "sharp", "spiky"])
@pytest.mark.parametrize("layout", list(ALIGNED))
def test_stored_ds_backward(layout, dist):
    """The backward that stores dS in the dK/dV kernel and reads it back for dQ: every
    element against the oracle, dK/dV bit-identical to the recomputing path, and dQ within
    bf16 rounding of it; one K/V head per pass (the scratch reused across passes)."""
    cu, q_segs, steps = ALIGNED[layout]
    H = 3
    q, kv, do = _gen(cu, H, q_segs, steps, dist=dist, seed=11, bwd=True)
    for st in steps:
        assert hydra.bwd_ds_bytes(hydra.Problem(cu, H, q_segs, st), 1) > 0
    res = _run_share(cu, H, q_segs, steps, q, kv, do, ds_kv_heads=1)
    ref = _oracle_share(cu, q_segs, steps, q, kv, do)
    _check_fwd(res, ref)
    _check_bwd(res, ref)
    base = _run_share(cu, H, q_segs, steps, q, kv, do)
    for (a, b), (c, d) in zip(res["dkv"], base["dkv"]):
        assert np.array_equal(a, c) and np.array_equal(b, d)
    assert rel_l2(res["dq"], base["dq"]) < 1e-2


@pytest.mark.parametrize("H,Hkv,per_pass", [(8, 2, 1), (8, 2, 2), (6, 3, 2), (4, 1, 1)])
def test_stored_ds_backward_grouped_heads(H, Hkv, per_pass):
    """Grouped K/V heads on the stored-dS path, with passes that split the K/V heads
    unevenly (6/3 heads in passes of 2 K/V heads leaves a last pass of 1)."""
    cu, q_segs, steps = ALIGNED["ragged_docs_3step"]
    q, kv, do = _gen(cu, H, q_segs, steps, dist="sharp", seed=12, bwd=True, Hkv=Hkv)
    res = _run_share(cu, H, q_segs, steps, q, kv, do, Hkv=Hkv, ds_kv_heads=per_pass)
    ref = _oracle_share(cu, q_segs, steps, q, kv, do)
    _check_fwd(res, ref)
    _check_bwd(res, ref)


def test_stored_ds_falls_back_where_it_does_not_apply():
    """Unaligned segments (or no scratch): hydra_attn_bwd_ds computes exactly what
    hydra_attn_bwd computes."""
    cu, q_segs, steps = MEDIUM["ragged_3step"]
    H = 2
    p = hydra.Problem(cu, H, q_segs, steps[1])
    assert hydra.bwd_ds_bytes(p, 1) == 0
    q, kv, do = _gen(cu, H, q_segs, steps, dist="sharp", seed=13, bwd=True)
    sh = ring.make_share(cu, H, q_segs, steps)
    qd, dod = dev_bf16(q), dev_bf16(do)
    kvd = [(dev_bf16(k), dev_bf16(v)) for k, v in kv]
    ring.forward(sh, qd, kvd)
    outs = []
    for use_ds in (False, True):
        dq = torch.zeros((sh.nq, H, D_QK), device="cuda")
        dk = torch.zeros((kv[1][0].shape[0], H, D_QK), device="cuda")
        dv = torch.zeros((kv[1][0].shape[0], H, D_V), device="cuda")
        k, v = kvd[1]
        if use_ds:
            scratch = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
            hydra.attn_bwd_ds(p, qd, k, v, sh.o_bf16, sh.lse_acc, dod, dq, dk, dv, scratch, sh.workspace)
        else:
            hydra.attn_bwd(p, qd, k, v, sh.o_bf16, sh.lse_acc, dod, dq, dk, dv, sh.workspace)
        torch.cuda.synchronize()
        outs.append([t.cpu().numpy() for t in (dq, dk, dv)])
    for a, b in zip(*outs):
        assert np.array_equal(a, b)


def test_gqa_rejected_when_groups_do_not_divide():
    p = hydra.Problem([0, 64], 6, [(0, 64)], [(0, 64)], n_kv_heads=4)
    assert hydra.lib().hydra_workspace_size(p.ref) == 0


def test_nondefault_scale():
    cu, q_segs, steps = MEDIUM["ragged_3step"]
    q, kv, do = _gen(cu, 2, q_segs, steps, dist="sharp", seed=2, bwd=True)
    res = _run_share(cu, 2, q_segs, steps, q, kv, do, scale=0.11)
    ref = _oracle_share(cu, q_segs, steps, q, kv, do, scale=0.11)
    _check_fwd(res, ref)
    _check_bwd(res, ref)


def test_constant_v_gives_constant_and_single_key_rows():
    cu = [0, 64, 192, 512]
    segs = [(0, 512)]
    q, kv, _ = _gen(cu, 4, segs, [segs], dist="sharp")
    k, v = kv[0]
    half = np.full(v.shape, inputs.bf16_round_bits(np.float32([0.5]))[0], dtype=np.uint16)
    res = _run_share(cu, 4, segs, [segs], q, [(k, half)])
    assert np.abs(res["o"] - 0.5).max() <= 2e-3
    res = _run_share(cu, 4, segs, [segs], q, [(k, v)])
    tau = 1 / math.sqrt(D_QK)
    for r in (0, 64, 192):
        np.testing.assert_allclose(res["o"][r], f32(v)[r], atol=1e-6)
        s_rr = tau * np.einsum("hc,hc->h", f32(q)[r].astype(np.float64), f32(k)[r].astype(np.float64))
        np.testing.assert_allclose(res["lse"][:, r], s_rr, atol=TOL_LSE)


def test_thousands_of_tiny_documents():
    """2500 documents of 1-4 tokens, one zero-length, in one segment: every tile straddles
    many document starts.  Single-token documents see only themselves: O = V, dV = dO, and
    dQ = dK = 0 up to rounding (dS = P (dP - D) with dP and D two fp32 evaluations of the
    same 128-term dot product); everything against the oracle, forward and backward."""
    rng = np.random.default_rng(8)
    lens = rng.integers(1, 5, size=2500)
    lens[7] = 0
    cu = [0] + list(np.cumsum(lens))
    segs = [(0, int(cu[-1]))]
    H = 2
    q, kv, do = _gen(cu, H, segs, [segs], dist="sharp", seed=8, bwd=True)
    res = _run_share(cu, H, segs, [segs], q, kv, do)
    ref = _oracle_share(cu, segs, [segs], q, kv, do)
    _check_fwd(res, ref)
    _check_bwd(res, ref)
    ones = [int(cu[d]) for d in range(len(lens)) if lens[d] == 1]
    np.testing.assert_allclose(res["o"][ones], f32(kv[0][1])[ones], atol=1e-6)
    assert np.abs(res["dq"][ones]).max() <= 1e-5 * np.abs(res["dq"]).max()
    assert np.abs(res["dkv"][0][0][ones]).max() <= 1e-5 * np.abs(res["dkv"][0][0]).max()
    np.testing.assert_allclose(res["dkv"][0][1][ones], f32(do)[ones], atol=1e-6)


def test_largest_head_count():
    """4096 heads (the largest accepted): token rows of 786432 elements; two short documents,
    a handful of heads checked against the oracle, forward and backward."""
    cu, segs, H = [0, 40, 72], [(0, 72)], 4096
    rng = np.random.default_rng(9)
    draw = lambda d, sc: inputs.bf16_round_bits(rng.standard_normal((72, H, d), dtype=np.float32) * np.float32(sc))
    q, kv, do = draw(D_QK, D_QK ** -0.5), [(draw(D_QK, D_QK ** -0.5), draw(D_V, D_V ** -0.5))], draw(D_V, 1.0)
    res = _run_share(cu, H, segs, [segs], q, kv, do)
    heads = [0, 1, 2047, 4095]
    sub = lambda x: f32(x)[:, heads]
    O, L = oracle.attn_fwd(sub(q), sub(kv[0][0]), sub(kv[0][1]), cu, segs, segs)
    dq, dk, dv = oracle.attn_bwd(sub(q), sub(kv[0][0]), sub(kv[0][1]), O, L, sub(do), cu, segs, segs)
    assert_o_close(res["o"][:, heads], O)
    assert_lse_close(res["lse"][heads], L)
    assert_grad_close(res["dq"][:, heads], dq, what="dQ")
    assert_grad_close(res["dkv"][0][0][:, heads], dk, what="dK")
    assert_grad_close(res["dkv"][0][1][:, heads], dv, what="dV")


def test_empty_kv_chunk_and_fully_masked_step():
    cu = [0, 700]
    q_segs = [(300, 200)]
    q, _, _ = _gen(cu, 2, q_segs, [])
    for steps in ([[]], [[(600, 100)]], [[(0, 0), (650, 0)]]):
        kv = [(inputs.rows("k", s, 2, D_QK), inputs.rows("v", s, 2, D_V)) for s in steps]
        res = _run_share(cu, 2, q_segs, steps, q, kv)
        assert np.isneginf(res["lse"]).all()
        assert (res["o"] == 0).all()


def test_every_output_written_and_deterministic():
    cu, q_segs, steps = MEDIUM["ragged_3step"]
    H = 2
    q, kv, do = _gen(cu, H, q_segs, steps, dist="spiky", seed=3, bwd=True)
    p = hydra.Problem(cu, H, q_segs, steps[1])
    ws = torch.empty(hydra.workspace_size(p), dtype=torch.uint8, device="cuda")
    qd = dev_bf16(q)
    kd, vd = dev_bf16(kv[1][0]), dev_bf16(kv[1][1])
    outs = []
    for _ in range(2):
        o = torch.full((p.nq, H, D_V), float("nan"), device="cuda")
        lse = torch.full((H, p.nq), float("nan"), device="cuda")
        hydra.attn_fwd(p, qd, kd, vd, o, lse, ws)
        torch.cuda.synchronize()
        assert not torch.isnan(o).any() and not torch.isnan(lse).any()
        outs.append((o.clone(), lse.clone()))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
    grads = []
    for _ in range(2):
        res = _run_share(cu, H, q_segs, steps, q, kv, do)
        grads.append(res)
    assert np.array_equal(grads[0]["dq"], grads[1]["dq"])
    for (a, b), (c, d) in zip(grads[0]["dkv"], grads[1]["dkv"]):
        assert np.array_equal(a, c) and np.array_equal(b, d)


def test_binding_refuses_strided_mistyped_and_missized_tensors():
    """Checked in the binding before the library is called (nothing is launched)."""
    cu, segs, H = [0, 64], [(0, 64)], 2
    p = hydra.Problem(cu, H, segs, segs)
    ws = torch.empty(hydra.workspace_size(p), dtype=torch.uint8, device="cuda")
    q = torch.zeros((64, H, D_QK), dtype=torch.bfloat16, device="cuda")
    v = torch.zeros((64, H, D_V), dtype=torch.bfloat16, device="cuda")
    o = torch.zeros((64, H, D_V), device="cuda")
    lse = torch.zeros((H, 64), device="cuda")
    with pytest.raises(ValueError, match="contiguous"):
        hydra.attn_fwd(p, torch.zeros((64, D_QK, H), dtype=torch.bfloat16, device="cuda").transpose(1, 2), q, v,
                       o, lse, ws)
    with pytest.raises(ValueError, match="shape"):
        hydra.attn_fwd(p, q.transpose(0, 1), q, v, o, lse, ws)
    with pytest.raises(ValueError, match="dtype"):
        hydra.attn_fwd(p, q.float(), q, v, o, lse, ws)
    with pytest.raises(ValueError, match="elements"):
        hydra.attn_fwd(p, q, q, v, o[:32], lse, ws)
    # broadcast rows (token stride 0) and overlapping rows never reach the library
    q_row = torch.zeros((1, H, D_QK), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ValueError, match="overlap"):
        hydra.attn_fwd(p, q_row.expand(64, H, D_QK), q, v, o, lse, ws)
    with pytest.raises(ValueError, match="overlap"):
        hydra.attn_fwd(p, q, q, torch.zeros((1, H, D_V), dtype=torch.bfloat16, device="cuda").expand(64, H, D_V),
                       o, lse, ws)
    flat = torch.zeros(64 * H * D_QK, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ValueError, match="overlap"):
        hydra.attn_fwd(p, q, flat.as_strided((64, H, D_QK), (D_QK, D_QK, 1)), v, o, lse, ws)
    with pytest.raises(ValueError, match="dtype"):
        hydra.pack_heads(q, torch.empty((2, 64, 1, D_QK), device="cuda"), 2)
    torch.cuda.synchronize()


@pytest.mark.parametrize("layout,H,Hkv", [("ragged_3step", 3, 0), ("zigzag_2step", 8, 2)])
def test_strided_qkv_views_match_dense(layout, H, Hkv):
    """Q, K, V as views into fused per-token buffers (token rows further apart than dense,
    heads contiguous): every output equals the dense run bit for bit."""
    cu, q_segs, steps = MEDIUM[layout]
    Hk = Hkv or H
    q, kv, do = _gen(cu, H, q_segs, steps, dist="sharp", seed=4, bwd=True, Hkv=Hkv)
    dense = _run_share(cu, H, q_segs, steps, q, kv, do, Hkv=Hkv)

    def fused(parts):
        """One buffer [rows, sum(widths) + 8] holding the parts side by side; the views."""
        rows = parts[0].shape[0]
        widths = [p.shape[1] * p.shape[2] for p in parts]
        buf = torch.zeros((rows, sum(widths) + 8), dtype=torch.bfloat16, device="cuda")
        views, c = [], 0
        for p, w in zip(parts, widths):
            buf[:, c:c + w] = dev_bf16(p).reshape(rows, w)
            views.append(buf[:, c:c + w].view(rows, p.shape[1], p.shape[2]))
            c += w
        return buf, views

    qbuf, (qv,) = fused([q])
    kvbufs = [fused([k, v]) for k, v in kv]
    kvv = [tuple(views) for _, views in kvbufs]
    assert qv.stride(0) > H * D_QK and kvv[0][0].stride(0) > Hk * D_QK
    sh = ring.make_share(cu, H, q_segs, steps, n_kv_heads=Hkv)
    o, lse, o16 = ring.forward(sh, qv, kvv)
    d_o = dev_bf16(do)
    dq = torch.zeros((sh.nq, H, D_QK), device="cuda")
    dkv = [(torch.zeros((k.shape[0], Hk, D_QK), device="cuda"), torch.zeros((k.shape[0], Hk, D_V), device="cuda"))
           for k, _ in kv]
    ring.backward(sh, qv, kvv, d_o, dq, dkv)
    torch.cuda.synchronize()
    assert np.array_equal(o.cpu().numpy(), dense["o"]) and np.array_equal(lse.cpu().numpy(), dense["lse"])
    assert np.array_equal(dq.cpu().numpy(), dense["dq"])
    for (a, b), (c, d) in zip(dkv, dense["dkv"]):
        assert np.array_equal(a.cpu().numpy(), c) and np.array_equal(b.cpu().numpy(), d)


def test_graph_capture_replays_match_eager():
    """The planned calls (plan uploaded once, outside the capture) recorded into a graph:
    forward, merges and backward of a 3-step share with GQA; three replays with eager work
    and synchronisation between them, each equal to the eager run bit for bit."""
    cu, q_segs, steps = MEDIUM["ragged_3step"]
    H, Hkv = 4, 2
    q, kv, do = _gen(cu, H, q_segs, steps, dist="sharp", seed=6, bwd=True, Hkv=Hkv)
    eager = _run_share(cu, H, q_segs, steps, q, kv, do, Hkv=Hkv)
    qd, dod = dev_bf16(q), dev_bf16(do)
    kvd = [(dev_bf16(k), dev_bf16(v)) for k, v in kv]
    sh = ring.make_share(cu, H, q_segs, steps, n_kv_heads=Hkv, graph_ready=True)
    ring.plan(sh)
    dq = torch.empty((sh.nq, H, D_QK), device="cuda")
    dkv = [(torch.empty((k.shape[0], Hkv, D_QK), device="cuda"), torch.empty((k.shape[0], Hkv, D_V), device="cuda"))
           for k, _ in kv]
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        dq.fill_(0.0)
        for a, b in dkv:
            a.fill_(0.0)
            b.fill_(0.0)
        ring.forward(sh, qd, kvd, planned=True)
        ring.backward(sh, qd, kvd, dod, dq, dkv, planned=True)
    for rep in range(3):
        sh.o_acc.fill_(float(rep + 7))          # eager work on the graph's buffers
        dq.fill_(-1.0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(sh.o_acc.cpu().numpy(), eager["o"]), rep
        assert np.array_equal(sh.lse_acc.cpu().numpy(), eager["lse"]), rep
        assert np.array_equal(dq.cpu().numpy(), eager["dq"]), rep
        for (a, b), (c, d) in zip(dkv, eager["dkv"]):
            assert np.array_equal(a.cpu().numpy(), c) and np.array_equal(b.cpu().numpy(), d), rep


def test_planned_calls_check_which_plan_the_workspace_holds():
    """A planned call launches on the plan in the workspace, so it is refused
    (HYDRA_ERR_WORKSPACE, nothing launched) when the workspace's last upload was for
    another problem, or, for the backward, was the forward's query-side items only."""
    cu, H = [0, 300, 700], 2
    pa = hydra.Problem(cu, H, [(0, 700)], [(0, 350)])
    pb = hydra.Problem(cu, H, [(0, 700)], [(350, 350)])   # same sizes, other KV offsets
    q, kv, do = _gen(cu, H, [(0, 700)], [[(0, 350)]], seed=8, bwd=True)
    qd, kd, vd, dod = dev_bf16(q), dev_bf16(kv[0][0]), dev_bf16(kv[0][1]), dev_bf16(do)
    ws = torch.empty(max(hydra.workspace_size(pa), hydra.workspace_size(pb)), dtype=torch.uint8, device="cuda")
    o = torch.full((700, H, D_V), float("nan"), device="cuda")
    lse = torch.full((H, 700), float("nan"), device="cuda")
    hydra.attn_plan(pa, ws)
    with pytest.raises(hydra.HydraError) as e:
        hydra.attn_fwd(pb, qd, kd, vd, o, lse, ws, planned=True)
    assert e.value.status == -4
    torch.cuda.synchronize()
    assert torch.isnan(o).all() and torch.isnan(lse).all()          # nothing was launched
    hydra.attn_fwd(pa, qd, kd, vd, o, lse, ws, planned=True)
    o16 = o.to(torch.bfloat16)
    dq = torch.zeros((700, H, D_QK), device="cuda")
    dk = torch.zeros((350, H, D_QK), device="cuda")
    dv = torch.zeros((350, H, D_V), device="cuda")
    hydra.attn_fwd(pb, qd, kd, vd, torch.empty_like(o), torch.empty_like(lse), ws)   # query-side plan only
    with pytest.raises(hydra.HydraError) as e:
        hydra.attn_bwd(pb, qd, kd, vd, o16, lse, dod, dq, dk, dv, ws, planned=True)
    assert e.value.status == -4
    hydra.attn_plan(pb, ws)
    hydra.attn_plan(pa, ws)                                            # the latest upload counts
    with pytest.raises(hydra.HydraError):
        hydra.attn_bwd(pb, qd, kd, vd, o16, lse, dod, dq, dk, dv, ws, planned=True)
    torch.cuda.synchronize()
    assert dq.abs().max().item() == 0 and dk.abs().max().item() == 0 and dv.abs().max().item() == 0
    hydra.attn_bwd(pa, qd, kd, vd, o16, lse, dod, dq, dk, dv, ws, planned=True)
    torch.cuda.synchronize()
    ref = oracle.attn_fwd(f32(q), f32(kv[0][0]), f32(kv[0][1]), cu, [(0, 700)], [(0, 350)])
    assert_o_close(o.cpu().numpy(), ref[0])
    rq, rk, rv = oracle.attn_bwd(f32(q), f32(kv[0][0]), f32(kv[0][1]), o16.float().cpu().numpy(),
                                 lse.cpu().numpy(), f32(do), cu, [(0, 700)], [(0, 350)])
    assert_grad_close(dq.cpu().numpy(), rq, what="dQ")
    assert_grad_close(dk.cpu().numpy(), rk, what="dK")
    assert_grad_close(dv.cpu().numpy(), rv, what="dV")


def test_gradient_canaries_untouched():
    """dK/dV rows outside the KV chunk's rows are never written (guard bands)."""
    cu = [0, 500]
    segs = [(0, 500)]
    H = 2
    q, kv, do = _gen(cu, H, segs, [segs], bwd=True)
    p = hydra.Problem(cu, H, segs, segs)
    sh = ring.make_share(cu, H, segs, [segs])
    qd, kd, vd, dod = dev_bf16(q), dev_bf16(kv[0][0]), dev_bf16(kv[0][1]), dev_bf16(do)
    ring.forward(sh, qd, [(kd, vd)])
    guard = 64
    dq = torch.full((500 + 2 * guard, H, D_QK), 7.0, device="cuda")
    dk = torch.full((500 + 2 * guard, H, D_QK), 7.0, device="cuda")
    dv = torch.full((500 + 2 * guard, H, D_V), 7.0, device="cuda")
    hydra.attn_bwd(p, qd, kd, vd, sh.o_bf16, sh.lse_acc, dod, dq[guard:-guard], dk[guard:-guard],
                   dv[guard:-guard], sh.workspace)
    torch.cuda.synchronize()
    for t in (dq, dk, dv):
        assert (t[:guard] == 7.0).all() and (t[-guard:] == 7.0).all()


# ----------------------------------------------------------------- full-size workloads

def _sample_rows(n, extra, count, seed):
    rng = np.random.default_rng(seed)
    r = set(int(x) for x in rng.choice(n, size=min(count, n), replace=False))
    r.update(int(x) for x in extra if 0 <= x < n)
    return np.array(sorted(r))


def test_packed32k_forward_sampled_rows():
    w = inputs.WORKLOADS["packed32k_fwd"]
    cu, H, q_segs, steps = list(w.cu_seqlens), w.n_heads, list(w.q_segs), [list(s) for s in w.kv_steps]
    q, kv, _ = _gen(cu, H, q_segs, steps)
    res = _run_share(cu, H, q_segs, steps, q, kv)
    assert np.isfinite(res["o"]).all() and np.isfinite(res["lse"]).all()
    edges = [c + d for c in cu for d in (-1, 0, 1)] + [127, 128, 129, 16383]
    rows = _sample_rows(32768, edges, 160, 0)
    heads = [0, 5, 15]
    O, L = oracle.attn_fwd(f32(q)[:, heads], f32(kv[0][0])[:, heads], f32(kv[0][1])[:, heads], cu, q_segs,
                           steps[0], q_rows=rows)
    assert_o_close(res["o"][rows][:, heads], O[rows])
    assert_o_close(res["o16"][rows][:, heads], O[rows], what="O bf16")
    assert_lse_close(res["lse"][heads][:, rows], L[:, rows])


def test_ring256k_three_steps_uniform_closed_form_and_sampled_rows():
    w = inputs.WORKLOADS["ring256k_3step"]
    cu, H, q_segs, steps = list(w.cu_seqlens), w.n_heads, list(w.q_segs), [list(s) for s in w.kv_steps]
    q, kv, _ = _gen(cu, H, q_segs, steps)
    # (1) Q = 0: every logit is 0, so O is the mean of the visible V and LSE = ln(count), all rows
    zq = np.zeros_like(q)
    res = _run_share(cu, H, q_segs, steps, zq, kv)
    v_all = np.concatenate([f32(v) for _, v in kv])
    Uo, UL, n = oracle.uniform_fwd(v_all, cu, q_segs, _union(steps))
    assert_lse_close(res["lse"], UL)
    assert_o_close(res["o"], Uo)
    # (2) real inputs, sampled rows of all steps merged; step (c) alone is fully masked
    res = _run_share(cu, H, q_segs, steps, q, kv)
    rows = _sample_rows(32768, [0, 1, 127, 128, 32767], 48, 1)
    heads = [3, 12]
    k_all = np.concatenate([f32(k)[:, heads] for k, _ in kv])
    O, L = oracle.attn_fwd(f32(q)[:, heads], k_all, v_all[:, heads], cu, q_segs, _union(steps), q_rows=rows)
    assert_o_close(res["o"][rows][:, heads], O[rows])
    assert_lse_close(res["lse"][heads][:, rows], L[:, rows])
    res_c = _run_share(cu, H, q_segs, [steps[2]], q, [kv[2]])
    assert np.isneginf(res_c["lse"]).all() and (res_c["o"] == 0).all()


def test_gqa_zigzag256k_share_uniform_forward_and_sampled_rows():
    """The benchmark share with 16 query heads over 2 K/V heads: Q = 0 closed form on every
    element, then real inputs on sampled rows of two heads of different groups."""
    w = inputs.WORKLOADS["zigzag256k_share"]
    cu, H, q_segs, steps = list(w.cu_seqlens), w.n_heads, list(w.q_segs), [list(s) for s in w.kv_steps]
    Hkv = 2
    q, kv, _ = _gen(cu, H, q_segs, steps, Hkv=Hkv)
    res = _run_share(cu, H, q_segs, steps, np.zeros_like(q), kv, Hkv=Hkv)
    v_all = np.concatenate([f32(v) for _, v in kv])
    Uo, UL, _ = oracle.uniform_fwd(v_all, cu, q_segs, _union(steps), n_q_heads=H)
    assert_lse_close(res["lse"], UL)
    assert_o_close(res["o"], Uo)
    res = _run_share(cu, H, q_segs, steps, q, kv, Hkv=Hkv)
    rows = _sample_rows(131072, [0, 65535, 65536, 131071], 12, 4)
    heads = [5, 9]                      # groups 0 and 1
    k_all = np.concatenate([f32(k) for k, _ in kv])
    O, L = oracle.attn_fwd(f32(q)[:, heads], k_all[:, [0, 1]], v_all[:, [0, 1]], cu, q_segs, _union(steps),
                           q_rows=rows)
    assert_o_close(res["o"][rows][:, heads], O[rows])
    assert_lse_close(res["lse"][heads][:, rows], L[:, rows])


def test_packed32k_backward_full_heads():
    w = inputs.WORKLOADS["packed32k_fwdbwd"]
    cu, H, q_segs, steps = list(w.cu_seqlens), w.n_heads, list(w.q_segs), [list(s) for s in w.kv_steps]
    q, kv, do = _gen(cu, H, q_segs, steps, bwd=True)
    res = _run_share(cu, H, q_segs, steps, q, kv, do, ds_kv_heads=BENCH_DS)
    heads = [1, 9]
    sub = lambda x: f32(x)[:, heads]
    O, L = oracle.attn_fwd(sub(q), sub(kv[0][0]), sub(kv[0][1]), cu, q_segs, steps[0])
    dq, dk, dv = oracle.attn_bwd(sub(q), sub(kv[0][0]), sub(kv[0][1]), O, L, sub(do), cu, q_segs, steps[0])
    assert_o_close(res["o"][:, heads], O)
    assert_lse_close(res["lse"][heads], L)
    assert_grad_close(res["dq"][:, heads], dq, what="dQ")
    assert_grad_close(res["dkv"][0][0][:, heads], dk, what="dK")
    assert_grad_close(res["dkv"][0][1][:, heads], dv, what="dV")
    # identities over every head: per document, sum_j dK_j = 0 and sum_j dV_j = sum_i dO_i
    # (exact in the oracle; here the per-row errors, within tolerance, add up randomly)
    gdk, gdv = (x.astype(np.float64) for x in res["dkv"][0])
    dof = f32(do).astype(np.float64)
    for a, b in zip(cu[:-1], cu[1:]):
        for h in range(H):
            assert np.linalg.norm(gdk[a:b, h].sum(0)) <= 0.05 * np.linalg.norm(gdk[a:b, h]) + 1e-6
            err = np.linalg.norm(gdv[a:b, h].sum(0) - dof[a:b, h].sum(0))
            assert err <= 0.05 * np.linalg.norm(gdv[a:b, h]) + 1e-6


def test_zigzag256k_share_sampled_rows_and_tail_keys():
    w = inputs.WORKLOADS["zigzag256k_share"]
    cu, H, q_segs, steps = list(w.cu_seqlens), w.n_heads, list(w.q_segs), [list(s) for s in w.kv_steps]
    q, kv, do = _gen(cu, H, q_segs, steps, bwd=True)
    res = _run_share(cu, H, q_segs, steps, q, kv, do, ds_kv_heads=BENCH_DS)
    heads = [2, 13]
    nq = 131072
    # query rows: head quarter, tail quarter, its last rows (which see the tail keys below)
    tail_q = np.arange(nq - 64, nq)
    rows = np.unique(np.concatenate([_sample_rows(nq, [0, 65535, 65536], 24, 2), tail_q]))
    union = [(0, 262144)]
    k_all = f32(inputs.rows("k", union, H, D_QK))[:, heads]
    v_all = f32(inputs.rows("v", union, H, D_V))[:, heads]
    qh, doh = f32(q)[:, heads], f32(do)[:, heads]
    O, L = oracle.attn_fwd(qh, k_all, v_all, cu, q_segs, union, q_rows=rows)
    assert_o_close(res["o"][rows][:, heads], O[rows])
    assert_lse_close(res["lse"][heads][:, rows], L[:, rows])
    # dQ of the sampled rows, summed over both steps, and dK/dV of the last 64 keys of step 0
    # (positions 262080..262143, seen only by the 64 tail queries)
    dq_ref = np.zeros((nq, 2, D_QK))
    for si, s in enumerate(steps):
        kk = f32(kv[si][0])[:, heads]
        vv = f32(kv[si][1])[:, heads]
        dq, dk, dv = oracle.attn_bwd(qh, kk, vv, O, L, doh, cu, q_segs, s, q_rows=rows)
        dq_ref += dq
        if si == 0:
            tail_k = np.arange(nq - 64, nq)
            assert_grad_close(res["dkv"][0][0][tail_k][:, heads], dk[tail_k], what="dK tail")
            assert_grad_close(res["dkv"][0][1][tail_k][:, heads], dv[tail_k], what="dV tail")
    assert_grad_close(res["dq"][rows][:, heads], dq_ref[rows], what="dQ rows")


def test_zigzag256k_uniform_closed_form_backward():
    """K = 0: softmax is uniform; O, LSE over every row and dK/dV of sampled keys of the
    peer chunk (each seen by 64K queries) have closed forms."""
    w = inputs.WORKLOADS["zigzag256k_share"]
    cu, H, q_segs, steps = list(w.cu_seqlens), 2, list(w.q_segs), [list(s) for s in w.kv_steps]
    q, kv, do = _gen(cu, H, q_segs, steps, bwd=True)
    kv0 = [(np.zeros_like(k), v) for k, v in kv]
    res = _run_share(cu, H, q_segs, steps, q, kv0, do, ds_kv_heads=1)
    v_all = np.concatenate([f32(v) for _, v in kv])
    Uo, UL, n = oracle.uniform_fwd(v_all, cu, q_segs, _union(steps))
    assert_lse_close(res["lse"], UL)
    assert_o_close(res["o"], Uo)
    assert np.abs(res["dq"]).max() == 0.0
    keys = np.array([0, 1, 4095, 65535, 65536, 100000, 131071])
    dk, dv = oracle.uniform_bwd_k0(f32(q), f32(kv[1][1]), Uo, f32(do), n, cu, q_segs, steps[1], keys)
    assert_grad_close(res["dkv"][1][0][keys], dk, what="dK uniform")
    assert_grad_close(res["dkv"][1][1][keys], dv, what="dV uniform")


def test_zigzag256k_share_dkdv_at_several_depths_and_column_sums():
    """The benchmark share as bench.py runs it (stored-dS backward): dK/dV of the last 4096
    keys of step 0 (positions 258048..262143, each seen by 1 to 4096 queries, all tail
    rows) element by element at several depths, on two heads; then over all 16 heads the
    identities that hold at any size (Sec. 2.2: rows sum over their document's keys):
    summed over both steps' keys, sum_j dK_j = 0 and sum_j dV_j = sum_i dO_i."""
    w = inputs.WORKLOADS["zigzag256k_share"]
    cu, H, q_segs, steps = list(w.cu_seqlens), w.n_heads, list(w.q_segs), [list(s) for s in w.kv_steps]
    q, kv, do = _gen(cu, H, q_segs, steps, bwd=True)
    res = _run_share(cu, H, q_segs, steps, q, kv, do, ds_kv_heads=BENCH_DS)
    nq = 131072
    heads = [0, 11]
    tail = np.arange(nq - 4096, nq)                     # positions 258048 .. 262143
    union = [(0, 262144)]
    k_all = f32(inputs.rows("k", union, H, D_QK))[:, heads]
    v_all = f32(inputs.rows("v", union, H, D_V))[:, heads]
    qh, doh = f32(q)[:, heads], f32(do)[:, heads]
    O, L = oracle.attn_fwd(qh, k_all, v_all, cu, q_segs, union, q_rows=tail)
    _, dk, dv = oracle.attn_bwd(qh, f32(kv[0][0])[:, heads], f32(kv[0][1])[:, heads], O, L, doh, cu, q_segs,
                                steps[0], q_rows=tail)
    for depth, keys in (("last 64", tail[-64:]), ("1K deep", tail[2048 - 64:2048]), ("4K deep", tail[:64]),
                        ("sampled", tail[::97])):
        assert_grad_close(res["dkv"][0][0][keys][:, heads], dk[keys], what=f"dK {depth}")
        assert_grad_close(res["dkv"][0][1][keys][:, heads], dv[keys], what=f"dV {depth}")
    dk_sum = sum(res["dkv"][i][0].astype(np.float64).sum(0) for i in range(2))    # [H, 192]
    dv_sum = sum(res["dkv"][i][1].astype(np.float64).sum(0) for i in range(2))
    do_sum = f32(do).astype(np.float64).sum(0)
    for h in range(H):
        dk_norm = np.sqrt(sum(np.linalg.norm(res["dkv"][i][0][:, h].astype(np.float64)) ** 2 for i in range(2)))
        dv_norm = np.sqrt(sum(np.linalg.norm(res["dkv"][i][1][:, h].astype(np.float64)) ** 2 for i in range(2)))
        assert np.linalg.norm(dk_sum[h]) <= 0.05 * dk_norm, h
        assert np.linalg.norm(dv_sum[h] - do_sum[h]) <= 0.05 * dv_norm, h


def test_gqa_zigzag256k_share_uniform_backward():
    """16 query heads over 2 K/V heads at the benchmark share's size, stored-dS backward:
    with K = 0 the softmax is uniform, dQ is exactly 0 and each K/V head's dK/dV (summed over
    its 8 query heads, Sec. 3.5) has a closed form, checked on keys of both chunks."""
    w = inputs.WORKLOADS["zigzag256k_share"]
    cu, H, q_segs, steps = list(w.cu_seqlens), w.n_heads, list(w.q_segs), [list(s) for s in w.kv_steps]
    Hkv = 2
    q, kv, do = _gen(cu, H, q_segs, steps, bwd=True, Hkv=Hkv)
    kv0 = [(np.zeros_like(k), v) for k, v in kv]
    res = _run_share(cu, H, q_segs, steps, q, kv0, do, Hkv=Hkv, ds_kv_heads=1)
    v_all = np.concatenate([f32(v) for _, v in kv])
    Uo, UL, n = oracle.uniform_fwd(v_all, cu, q_segs, _union(steps), n_q_heads=H)
    assert_lse_close(res["lse"], UL)
    assert_o_close(res["o"], Uo)
    assert np.abs(res["dq"]).max() == 0.0
    for si, keys in ((0, np.array([0, 4095, 65535, 65536, 131071])), (1, np.array([0, 65535, 65536, 131071]))):
        dk, dv = oracle.uniform_bwd_k0(f32(q), f32(kv[si][1]), Uo, f32(do), n, cu, q_segs, steps[si], keys)
        assert_grad_close(res["dkv"][si][0][keys], dk, what=f"dK uniform step {si}")
        assert_grad_close(res["dkv"][si][1][keys], dv, what=f"dV uniform step {si}")


def test_ring256k_3step_uniform_backward_as_benchmarked():
    """The 256K ring configuration (32K query chunk against three 32K KV chunks: the own
    chunk, a fully visible one, a fully masked one) with the backward bench.py times on it
    (stored dS, passes sized by the default budget): with K = 0 the softmax is uniform, so
    O, LSE, dQ (exactly 0) and the dK/dV of sampled keys of every step have closed forms;
    the masked step's dK/dV stay exactly zero."""
    w = inputs.WORKLOADS["ring256k_3step"]
    cu, H, q_segs, steps = list(w.cu_seqlens), w.n_heads, list(w.q_segs), [list(s) for s in w.kv_steps]
    q, kv, do = _gen(cu, H, q_segs, steps, bwd=True)
    kv0 = [(np.zeros_like(k), v) for k, v in kv]
    res = _run_share(cu, H, q_segs, steps, q, kv0, do, ds_kv_heads=BENCH_DS)
    v_all = np.concatenate([f32(v) for _, v in kv])
    Uo, UL, n = oracle.uniform_fwd(v_all, cu, q_segs, _union(steps))
    assert_lse_close(res["lse"], UL)
    assert_o_close(res["o"], Uo)
    assert np.abs(res["dq"]).max() == 0.0
    for si, keys in ((0, np.array([0, 1, 8191, 16384, 32767])), (1, np.array([0, 4095, 20000, 32767]))):
        dk, dv = oracle.uniform_bwd_k0(f32(q), f32(kv[si][1]), Uo, f32(do), n, cu, q_segs, steps[si], keys)
        assert_grad_close(res["dkv"][si][0][keys], dk, what=f"dK uniform step {si}")
        assert_grad_close(res["dkv"][si][1][keys], dv, what=f"dV uniform step {si}")
    assert np.abs(res["dkv"][2][0]).max() == 0.0 and np.abs(res["dkv"][2][1]).max() == 0.0


@pytest.mark.parametrize("ds", [0, 1])
def test_head_and_document_permutations_permute_the_outputs(ds):
    """Heads are independent and documents only see themselves: permuting the heads permutes
    every output bit for bit (each (tile, head) runs the same code); reordering the packed
    documents moves their rows, whose values change only by rounding (the tiles fall
    differently), compared within the parity tolerances."""
    cu, q_segs, steps = ALIGNED["contiguous_1step"]
    H = 4
    q, kv, do = _gen(cu, H, q_segs, steps, dist="sharp", seed=21, bwd=True)
    base = _run_share(cu, H, q_segs, steps, q, kv, do, ds_kv_heads=ds)
    perm = [2, 0, 3, 1]
    ph = _run_share(cu, H, q_segs, steps, q[:, perm], [(k[:, perm], v[:, perm]) for k, v in kv], do[:, perm],
                    ds_kv_heads=ds)
    assert np.array_equal(ph["o"], base["o"][:, perm]) and np.array_equal(ph["lse"], base["lse"][perm])
    assert np.array_equal(ph["dq"], base["dq"][:, perm])
    assert np.array_equal(ph["dkv"][0][0], base["dkv"][0][0][:, perm])
    assert np.array_equal(ph["dkv"][0][1], base["dkv"][0][1][:, perm])
    lens = np.diff(cu)
    order = [4, 1, 5, 0, 3, 2]
    starts = np.asarray(cu)[:-1]
    rows = np.concatenate([np.arange(starts[d], starts[d] + lens[d]) for d in order])
    cu2 = [0] + list(np.cumsum(lens[order]))
    pd = _run_share(cu2, H, q_segs, steps, q[rows], [(k[rows], v[rows]) for k, v in kv], do[rows], ds_kv_heads=ds)
    assert_o_close(pd["o"], base["o"][rows])
    assert_lse_close(pd["lse"], base["lse"][:, rows])
    assert_grad_close(pd["dq"], base["dq"][rows], what="dQ")
    assert_grad_close(pd["dkv"][0][0], base["dkv"][0][0][rows], what="dK")
    assert_grad_close(pd["dkv"][0][1], base["dkv"][0][1][rows], what="dV")


def test_offsets_past_two_to_the_31_elements():
    """1,048,876 rows x 16 heads in 2048 documents of 512 tokens and a ragged one of 300:
    Q and dQ hold 3.2e9 elements and O 2.1e9, so late rows sit past every 32-bit element
    offset.  Inputs are drawn on the device (seeded); the first document, the one holding
    element 2^31 of Q, and the last two are checked against the oracle (two heads)."""
    H, L, n_full = 16, 512, 2048
    lens = [L] * n_full + [300]
    cu = [0] + list(np.cumsum(lens))
    nq = cu[-1]
    segs = [(0, nq)]
    gen = torch.Generator(device="cuda").manual_seed(17)
    draw = lambda d, s: (torch.randn((nq, H, d), generator=gen, device="cuda") * s).to(torch.bfloat16)
    q, k, v, d_o = draw(D_QK, 1.0), draw(D_QK, 1.0), draw(D_V, 1.0), draw(D_V, 1.0)
    sh = ring.make_share(cu, H, segs, [segs])
    o, lse, _ = ring.forward(sh, q, [(k, v)])
    dq = torch.zeros((nq, H, D_QK), dtype=torch.float32, device="cuda")
    dk = torch.zeros((nq, H, D_QK), dtype=torch.float32, device="cuda")
    dv = torch.zeros((nq, H, D_V), dtype=torch.float32, device="cuda")
    ring.backward(sh, q, [(k, v)], d_o, dq, [(dk, dv)])
    torch.cuda.synchronize()
    assert nq * H * D_QK > 3 * 2 ** 30 and nq * H * D_V > 2 ** 31
    heads = [3, 15]
    docs = [0, (2 ** 31 // (H * D_QK)) // L, n_full - 1, n_full]
    for d in docs:
        a, b = cu[d], cu[d + 1]
        host = lambda t: t[a:b][:, heads].float().cpu().numpy().astype(np.float64)
        qq, kk, vv, dd = host(q), host(k), host(v), host(d_o)
        dcu, dseg = [0, b - a], [(0, b - a)]
        O, Lse = oracle.attn_fwd(qq, kk, vv, dcu, dseg, dseg)
        rq, rk, rv = oracle.attn_bwd(qq, kk, vv, O, Lse, dd, dcu, dseg, dseg)
        assert_o_close(o[a:b][:, heads].cpu().numpy(), O, what=f"O doc {d}")
        assert_lse_close(lse[heads][:, a:b].cpu().numpy(), Lse, what=f"LSE doc {d}")
        assert_grad_close(dq[a:b][:, heads].cpu().numpy(), rq, what=f"dQ doc {d}")
        assert_grad_close(dk[a:b][:, heads].cpu().numpy(), rk, what=f"dK doc {d}")
        assert_grad_close(dv[a:b][:, heads].cpu().numpy(), rv, what=f"dV doc {d}")
