"""CPU tests of the C library: it loads, exports every declared symbol, validates its
arguments, and its work plan covers exactly the visible (query, key) pairs."""
import os
import re

import numpy as np
import pytest

from oracle import attention as A
from paper_2609_34318_amd import hydra, inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not os.path.exists(hydra.LIB_PATH):
        from paper_2609_34318_amd import build_lib
        build_lib.build()
    return hydra.lib()


def test_library_exports_every_declared_function():
    names = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        text = open(os.path.join(ROOT, "include", h)).read()
        names |= set(re.findall(r"\b(hydra_[a-z0-9_]+)\s*\(", text))
    assert {"hydra_attn_fwd", "hydra_attn_bwd", "hydra_lse_merge", "hydra_workspace_size", "hydra_attn_plan",
            "hydra_attn_fwd_planned", "hydra_attn_bwd_planned",
            "hydra_pack_heads", "hydra_unpack_heads", "hydra_zigzag_gather", "hydra_zigzag_scatter",
            "hydra_unpack_heads_gated", "hydra_pack_heads_gated_bwd", "hydra_schedule"} <= names
    L = hydra.lib()
    for n in sorted(names):
        assert hasattr(L, n), f"{n} not exported"


def test_layout_arguments_checked_on_host():
    L = hydra.lib()
    # heads not divisible by the Ulysses degree, sizes not multiples of 16 bytes, NULL
    assert L.hydra_pack_heads(8, 6, 256, 4, 16, 1 << 20, None) == -1
    assert L.hydra_pack_heads(8, 8, 24, 4, 16, 1 << 20, None) == -1
    assert L.hydra_pack_heads(8, 8, 256, 4, None, 1 << 20, None) == -1
    assert L.hydra_unpack_heads(-1, 8, 256, 4, 16, 1 << 20, None) == -1
    # misaligned, overlapping
    assert L.hydra_pack_heads(8, 8, 256, 4, 24, 1 << 20, None) == -3
    assert L.hydra_pack_heads(8, 8, 256, 4, 16, 16 + 256, None) == -1
    assert L.hydra_pack_heads(0, 8, 256, 4, 16, 1 << 20, None) == 0
    # zigzag: rows must split into 2*cp_r chunks, rank in range, no overlap
    assert L.hydra_zigzag_gather(30, 64, 4, 0, 16, 1 << 20, None) == -1
    assert L.hydra_zigzag_gather(32, 64, 4, 4, 16, 1 << 20, None) == -1
    assert L.hydra_zigzag_gather(32, 64, 4, -1, 16, 1 << 20, None) == -1
    assert L.hydra_zigzag_gather(32, 40, 4, 0, 16, 1 << 20, None) == -1
    assert L.hydra_zigzag_scatter(32, 64, 4, 1, 16, 16 + 256, None) == -1
    assert L.hydra_zigzag_scatter(32, 64, 4, 1, 16, 8, None) == -3
    assert L.hydra_zigzag_gather(0, 64, 4, 1, 16, 1 << 20, None) == 0


def test_gate_arguments_checked_on_host():
    L = hydra.lib()
    a, b, c, d, e = 16, 1 << 24, 2 << 24, 3 << 24, 4 << 24     # disjoint, aligned, never dereferenced
    f = L.hydra_unpack_heads_gated
    assert f(8, 8, 128, 1, 3, a, b, c, None) == -1          # heads not a multiple of cp_u
    assert f(8, 8, 96, 1, 4, a, b, c, None) == -1           # d_v not a power of two
    assert f(8, 8, 1024, 1, 4, a, b, c, None) == -1         # d_v above 512
    assert f(8, 8, 128, 8, 4, a, b, c, None) == -1          # gate_dim neither 1 nor d_v
    assert f(8, 70000, 128, 1, 1, a, b, c, None) == -1      # too many heads
    assert f(-1, 8, 128, 1, 4, a, b, c, None) == -1
    assert f(8, 8, 128, 1, 4, None, b, c, None) == -1
    assert f(8, 8, 128, 1, 4, a + 8, b, c, None) == -3      # misaligned
    assert f(8, 8, 128, 128, 4, a, b, b + 16, None) == -1   # output overlaps the gate
    assert f(8, 8, 128, 1, 4, a, b, a + 8 * 8 * 128 * 2 - 16, None) == -1   # ... the input
    assert f(0, 8, 128, 1, 4, None, None, None, None) == 0  # no rows: no-op
    g = L.hydra_pack_heads_gated_bwd
    assert g(8, 8, 128, 1, 4, a, b, c, d, None, None) == -1     # d_gate missing
    assert g(8, 8, 128, 1, 4, a, b, c, d, e + 4, None) == -3
    assert g(8, 8, 128, 128, 4, a, b, c, d, d + 16, None) == -1  # the two outputs overlap
    assert g(8, 8, 128, 1, 4, a, b, c, d, c, None) == -1         # d_gate aliases d_y
    assert g(0, 8, 128, 1, 4, None, None, None, None, None, None) == 0


def test_status_strings():
    for code in (0, -1, -2, -3, -4, -5, 7):
        assert isinstance(hydra.lib().hydra_strerror(code), bytes)


def _problem(cu, H, q, kv, **kw):
    return hydra.Problem(cu, H, q, kv, **kw)


@pytest.mark.parametrize("case", [
    dict(cu=[0, 100], H=0, q=[(0, 10)], kv=[(0, 10)]),            # no heads
    dict(cu=[1, 100], H=2, q=[(0, 10)], kv=[(0, 10)]),            # cu[0] != 0
    dict(cu=[0, 100, 50], H=2, q=[(0, 10)], kv=[(0, 10)]),        # not monotone
    dict(cu=[0, 100], H=2, q=[(95, 10)], kv=[(0, 10)]),           # segment past the window
    dict(cu=[0, 100], H=2, q=[(0, 10)], kv=[(-1, 5)]),            # negative start
    dict(cu=[0, 100], H=2, q=[(0, 10)], kv=[(0, -5)]),            # negative length
])
def test_invalid_problems_rejected_on_host(case):
    p = _problem(case["cu"], case["H"], case["q"], case["kv"])
    assert hydra.workspace_size(p) == 0
    assert hydra.lib().hydra_visible_pairs(p.ref) == -1
    # the compute calls reject before touching the GPU (null pointers would fault otherwise)
    L = hydra.lib()
    assert L.hydra_attn_fwd(p.ref, None, None, None, None, None, None, None, 0, None) == -1
    assert L.hydra_attn_bwd(p.ref, *([None] * 10), 0, None) == -1
    assert L.hydra_attn_plan(p.ref, None, 0, None) == -1
    assert L.hydra_attn_fwd_planned(p.ref, None, None, None, None, None, None, None, 0, None) == -1
    assert L.hydra_attn_bwd_planned(p.ref, *([None] * 10), 0, None) == -1


def test_unsupported_dims_and_bad_pointers():
    L = hydra.lib()
    p = _problem([0, 64], 2, [(0, 64)], [(0, 64)], d_qk=128)
    assert L.hydra_attn_fwd(p.ref, None, None, None, None, None, None, None, 0, None) == -2
    p = _problem([0, 64], 2, [(0, 64)], [(0, 64)])
    ws = hydra.workspace_size(p)
    assert ws > 0
    # misaligned device pointers: rejected with HYDRA_ERR_ALIGN before any HIP call
    assert L.hydra_attn_fwd(p.ref, 8, 16, 16, 16, 16, None, 16, ws, None) == -3
    # workspace too small / missing
    assert L.hydra_attn_fwd(p.ref, 16, 16, 16, 16, 16, None, 16, ws - 1, None) == -4
    assert L.hydra_attn_fwd(p.ref, 16, 16, 16, 16, 16, None, None, ws, None) == -4
    assert L.hydra_attn_plan(p.ref, 16, ws - 1, None) == -4
    assert L.hydra_attn_plan(p.ref, 8, ws, None) == -3
    assert L.hydra_attn_fwd_planned(p.ref, 8, 16, 16, 16, 16, None, 16, ws, None) == -3
    # merge argument checks
    assert L.hydra_lse_merge(10, 2, 64, 16, 16, 16, 16, None, None) == -2
    assert L.hydra_lse_merge(-1, 2, 128, 16, 16, 16, 16, None, None) == -1
    assert L.hydra_lse_merge(10, 2, 128, 16, 16, 8, 16, None, None) == -3
    assert L.hydra_lse_merge(0, 2, 128, None, None, None, None, None, None) == 0


def test_overlapping_buffers_rejected_on_host():
    """Outputs that overlap each other or an input are rejected before any HIP call."""
    L = hydra.lib()
    p = _problem([0, 64], 2, [(0, 64)], [(0, 32)], n_kv_heads=1)
    ws = hydra.workspace_size(p)
    M = 1 << 24                       # disjoint, aligned, never dereferenced
    q, k, v, o, lse, obf, w = (M * i for i in range(1, 8))
    fwd = L.hydra_attn_fwd
    assert fwd(p.ref, q, k, v, q + 64 * 2 * 192 * 2 - 16, lse, None, w, ws, None) == -1   # O over Q's tail
    assert fwd(p.ref, q, k, v, o, o + 64 * 2 * 128 * 4 - 16, None, w, ws, None) == -1     # LSE over O's tail
    assert fwd(p.ref, q, k, v, o, lse, obf, k + 32 * 192 * 2 - 16, ws, None) == -1        # workspace over K
    assert fwd(p.ref, q, k, v, o, lse, lse, w, ws, None) == -1                            # O bf16 aliases LSE
    dq, dk, dv, of, lf, do = (M * i for i in range(8, 14))
    bwd = L.hydra_attn_bwd
    args = dict(q=q, k=k, v=v, of=of, lf=lf, do=do, dq=dq, dk=dk, dv=dv)
    call = lambda **kw: bwd(p.ref, *[{**args, **kw}[n] for n in ("q", "k", "v", "of", "lf", "do", "dq", "dk", "dv")],
                            w, ws, None)
    assert call(dk=dq + 64 * 2 * 192 * 4 - 16) == -1      # dK over dQ's tail
    assert call(dv=dk + 32 * 192 * 4 - 16) == -1          # dV over dK's tail (one K/V head)
    assert call(dq=do) == -1                              # dQ aliases dO
    assert call(dv=v + 32 * 128 * 2 - 16) == -1           # dV over V's tail
    assert call(dk=w) == -1                               # dK aliases the workspace
    # inputs may share memory with each other (still rejected here only for alignment)
    assert call(k=q + 8) == -3
    mg = L.hydra_lse_merge
    assert mg(10, 2, 128, o, lse, o + 10 * 2 * 128 * 4 - 16, lf, None, None) == -1   # partial over acc
    assert mg(10, 2, 128, o, lse, of, lf, lse, None) == -1                           # bf16 aliases LSE


def test_planned_calls_refuse_an_unplanned_workspace():
    """The planned calls launch on the plan the workspace holds; a workspace no plan was
    uploaded into through the library is refused with HYDRA_ERR_WORKSPACE before any HIP
    call (the addresses below are never dereferenced)."""
    L = hydra.lib()
    p = _problem([0, 64], 2, [(0, 64)], [(0, 64)])
    ws = hydra.workspace_size(p)
    M = 1 << 24
    q, k, v, o, lse, w = (M * i for i in range(1, 7))
    assert L.hydra_attn_fwd_planned(p.ref, q, k, v, o, lse, None, w, ws, None) == -4
    dq, dk, dv, of, lf, do = (M * i for i in range(8, 14))
    assert L.hydra_attn_bwd_planned(p.ref, q, k, v, of, lf, do, dq, dk, dv, w, ws, None) == -4


def test_noalloc_backward_checks_before_any_hip_call():
    """The no-allocation backward rejects malformed problems (-1) and problems whose
    workspace exceeds its 32 MiB scratch (-6) on the host; nothing is dereferenced."""
    L = hydra.lib()
    assert L.hydra_noalloc_scratch_bytes() == 32 << 20
    bad = _problem([0, 100], 0, [(0, 10)], [(0, 10)])
    assert L.hydra_attn_bwd_noalloc(bad.ref, *([None] * 10)) == -1
    big = _problem([0, 1 << 22], 16, [(0, 1 << 22)], [(0, 256)])
    assert hydra.workspace_size(big) > 32 << 20
    assert L.hydra_attn_bwd_noalloc(big.ref, *([16] * 9), None) == -6
    assert L.hydra_strerror(-6).decode().startswith("problem needs more workspace")


def test_binding_refuses_host_tensors():
    """The library takes plain device pointers; the binding refuses a host tensor before
    any call (its address would reach a kernel)."""
    import torch
    p = _problem([0, 64], 2, [(0, 64)], [(0, 64)])
    q = torch.zeros((64, 2, 192), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="device tensor"):
        hydra.attn_fwd(p, q, q, q, None, None, torch.zeros(16, dtype=torch.uint8))
    with pytest.raises(ValueError, match="device tensor"):
        hydra.pack_heads(q, q, 2)


def test_token_strides_checked_on_host():
    """q/k/v token strides: 0 or at least dense, a multiple of 8, below 2^22."""
    def ws(**strides):
        p = _problem([0, 64], 2, [(0, 64)], [(0, 64)], n_kv_heads=1)
        for name, val in strides.items():
            setattr(p.c, name, val)
        return hydra.workspace_size(p)
    assert ws() > 0
    assert ws(q_tok_stride=2 * 192 + 8, k_tok_stride=192 + 128, v_tok_stride=192 + 128 + 8) > 0
    assert ws(q_tok_stride=2 * 192 - 8) == 0          # below dense
    assert ws(k_tok_stride=191) == 0                  # below dense for one K/V head
    assert ws(v_tok_stride=128 + 4) == 0              # rows not 16-byte aligned
    assert ws(q_tok_stride=1 << 22) == 0              # too far apart
    assert ws(v_tok_stride=-8) == 0


def test_launch_size_limit_checked_on_host():
    """One 512-lane workgroup per (tile, head) and fewer than 2^32 lanes per dispatch:
    2^23 (query tile, head) pairs are refused, one fewer is planned."""
    ok = _problem([0, 2 ** 20], 4096, [(0, 2 ** 19 - 256)], [(0, 256)])
    big = _problem([0, 2 ** 20], 4096, [(0, 2 ** 19)], [(0, 256)])
    assert hydra.workspace_size(ok) > 0
    assert hydra.workspace_size(big) == 0
    L = hydra.lib()
    assert L.hydra_attn_fwd(big.ref, 16, 32, 48, 64, 80, None, 96, 1 << 20, None) == -1
    kv_big = _problem([0, 2 ** 21], 8192 // 8, [(0, 256)], [(0, 2 ** 20)], n_kv_heads=1024)
    assert hydra.workspace_size(kv_big) == 0


def test_ring_plan_needs_per_step_workspaces():
    """Planned (graph-recordable) calls need one workspace per ring step."""
    from paper_2609_34318_amd import ring
    cu, q, steps = [0, 512], [(0, 256)], [[(0, 128)], [(128, 128)]]
    sh = ring.make_share(cu, 2, q, steps, device="cpu")
    with pytest.raises(ValueError, match="graph_ready"):
        ring.plan(sh)
    sh = ring.make_share(cu, 2, q, steps, device="cpu", graph_ready=True)
    assert [w.numel() for w in sh.step_workspaces] == [hydra.workspace_size(p) for p in sh.problems]


def test_zero_rows_is_noop():
    L = hydra.lib()
    p = _problem([0, 64], 2, [], [(0, 64)])
    assert L.hydra_attn_fwd(p.ref, None, None, None, None, None, None, None, 0, None) == 0
    p = _problem([0, 64], 2, [(0, 64)], [])
    assert L.hydra_attn_bwd(p.ref, *([None] * 10), 0, None) == 0


def _random_problem(rng):
    n_docs = int(rng.integers(1, 8))
    lens = rng.integers(0, 400, size=n_docs)
    lens[int(rng.integers(0, n_docs))] += 1
    cu = inputs.cu_from_lengths(lens)
    total = int(cu[-1])

    def chunk():
        segs = []
        for _ in range(int(rng.integers(0, 5))):
            a = int(rng.integers(0, total + 1))
            b = int(rng.integers(a, total + 1))
            segs.append((a, b - a))
        return segs

    return cu, chunk(), chunk()


def _covered(items, nq, nk, which):
    """Count how often each (query row, key row) pair is visited by the plan."""
    cov = np.zeros((nq, nk), dtype=np.int32)
    for it in items:
        r0, n, nr = it[0], it[2], it[3]
        for r in range(nr):
            o0, on = it[4 + 3 * r], it[6 + 3 * r]
            if which == 0:
                cov[r0:r0 + n, o0:o0 + on] += 1
            else:
                cov[o0:o0 + on, r0:r0 + n] += 1
    return cov


@pytest.mark.parametrize("seed", range(25))
def test_plan_covers_exactly_the_visible_pairs(seed):
    rng = np.random.default_rng(seed)
    cu, q_segs, kv_segs = _random_problem(rng)
    p = _problem(cu, 3, q_segs, kv_segs)
    qpos, kpos = A.row_positions(q_segs), A.row_positions(kv_segs)
    qd, kd = A.doc_of(cu, qpos), A.doc_of(cu, kpos)
    vis = (qd[:, None] == kd[None, :]) & (kpos[None, :] <= qpos[:, None])
    assert hydra.visible_pairs(p) == int(vis.sum()) == A.visible_pairs_bruteforce(cu, q_segs, kv_segs)
    bq, bk = hydra.tile_rows()
    for which, rows_per_tile in ((0, bq), (1, bk)):
        items = hydra.plan_items(p, which)
        cov = _covered(items, len(qpos), len(kpos), which)
        assert (cov <= 1).all(), "a pair is visited twice"
        assert (cov[vis] == 1).all(), "a visible pair is never visited"
        own = qpos if which == 0 else kpos
        own_rows = sorted(r for it in items for r in range(it[0], it[0] + it[2]))
        assert own_rows == list(range(len(own))), "tiles must cover every own row once"
        for it in items:
            assert 1 <= it[2] <= rows_per_tile
            seg_pos = own[it[0]:it[0] + it[2]]
            assert seg_pos[0] == it[1] and (np.diff(seg_pos) == 1).all(), "tile rows must be consecutive"
        cost = [sum(it[6 + 3 * r] for r in range(it[3])) for it in items]
        assert cost == sorted(cost, reverse=True), "heaviest tiles first"


def test_visible_pairs_of_the_workloads():
    expect = {"tiny_2step": [28800, 32896],
              "packed32k_fwd": [144931409],
              "ring256k_3step": [536887296, 1073741824, 0],
              "zigzag256k_share": [8590000128, 8589934592]}
    for name, counts in expect.items():
        w = inputs.WORKLOADS[name]
        got = [hydra.visible_pairs(hydra.Problem(w.cu_seqlens, w.n_heads, w.q_segs, s)) for s in w.kv_steps]
        assert got == counts, name
    # the packed microbatch: sum of s(s+1)/2 over its documents
    assert 144931409 == sum(s * (s + 1) // 2 for s in inputs.PACKED32K_DOCS)


def test_stored_ds_bytes_and_the_budget_choice():
    """The dS buffer of the stored-dS backward: per query head it holds every visible pair
    (2 bytes each) in 24 KB slots, so at least 2 bytes per pair and at most the slots that
    the pairs touch; the pass size bench.py picks is the most K/V heads that fit a budget;
    a problem with a segment off the 32-row grid gets no dS buffer (recompute path)."""
    from paper_2609_34318_amd import ring
    w = inputs.WORKLOADS["zigzag256k_share"]
    probs = [hydra.Problem(w.cu_seqlens, w.n_heads, w.q_segs, s) for s in w.kv_steps]
    for p in probs:
        one = hydra.bwd_ds_bytes(p, 1)
        assert one % (24 * 1024) == 0
        assert 2 * hydra.visible_pairs(p) <= one <= 2 * hydra.visible_pairs(p) * 1.01
        assert hydra.bwd_ds_bytes(p, 4) == 4 * one
    need4 = max(hydra.bwd_ds_bytes(p, 4) for p in probs)
    assert ring.ds_kv_heads_within(probs, 72 << 30) == 4
    assert ring.ds_kv_heads_within(probs, need4) == 4
    assert ring.ds_kv_heads_within(probs, need4 - 1) == 3
    assert ring.ds_kv_heads_within(probs, 0) == 0
    packed = inputs.WORKLOADS["packed32k_fwdbwd"]
    pp = [hydra.Problem(packed.cu_seqlens, packed.n_heads, packed.q_segs, s) for s in packed.kv_steps]
    assert ring.ds_kv_heads_within(pp, 72 << 30) == 16
    # the default budget: one K/V head per pass on the share, one pass on the packed batch
    assert ring.ds_kv_heads_within(probs, ring.DEFAULT_DS_BUDGET_BYTES) == 1
    assert ring.ds_kv_heads_within(pp, ring.DEFAULT_DS_BUDGET_BYTES) == 16
    ragged = hydra.Problem([0, 100, 300], 4, [(0, 300)], [(0, 300)])
    assert hydra.bwd_ds_bytes(ragged, 1) == 0
    assert ring.ds_kv_heads_within([ragged], 72 << 30) == 0


def test_oracle_timings_run_on_the_host():
    """bench.py --oracle-timings times the oracle on every workload without a GPU: one JSON
    line each, the small share whole, every line with a one-thread figure."""
    import json
    import subprocess
    import sys
    env = dict(os.environ, HIP_VISIBLE_DEVICES="", CUDA_VISIBLE_DEVICES="")
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--oracle-timings", "--cpu-rows", "64"],
                         capture_output=True, text=True, timeout=600, env=env, check=True).stdout
    recs = [json.loads(line) for line in out.splitlines() if line.startswith("{")]
    assert [r["workload"] for r in recs] == list(inputs.WORKLOADS)
    for r in recs:
        assert r["value"] > 0 and r["one_core"]["value"] > 0 and r["one_core"]["cores"] == 1
        assert r["whole"] == (r["workload"] == "tiny_2step")
        assert r["host"]["nproc"] >= 1
