"""The no-allocation backward (hydra_attn_bwd_noalloc) against hydra_attn_bwd: the same
kernels on the library's own per-GPU scratch instead of a caller workspace, so the results
must be equal bit for bit; two calls in a row, the second on a smaller problem (the scratch
keeps the first call's contents)."""
import numpy as np
import pytest
import torch

from paper_2609_34318_amd import hydra, inputs, ring

from gpu_util import dev_bf16

pytestmark = pytest.mark.gpu
D_QK, D_V = 192, 128


def _case(cu, H, q_segs, kv_segs, Hkv, seed):
    Hk = Hkv or H
    q = dev_bf16(inputs.rows("q", q_segs, H, D_QK, seed, "sharp"))
    k = dev_bf16(inputs.rows("k", kv_segs, Hk, D_QK, seed, "sharp"))
    v = dev_bf16(inputs.rows("v", kv_segs, Hk, D_V, seed, "sharp"))
    do = dev_bf16(inputs.rows("do", q_segs, H, D_V, seed, "sharp"))
    sh = ring.make_share(cu, H, q_segs, [kv_segs], n_kv_heads=Hkv)
    ring.forward(sh, q, [(k, v)])
    p = sh.problems[0]
    outs = []
    for noalloc in (False, True):
        dq = torch.full((sh.nq, H, D_QK), 0.25, device="cuda")       # += targets
        dk = torch.full((k.shape[0], Hk, D_QK), -0.5, device="cuda")
        dv = torch.full((k.shape[0], Hk, D_V), 1.0, device="cuda")
        if noalloc:
            hydra.attn_bwd_noalloc(p, q, k, v, sh.o_bf16, sh.lse_acc, do, dq, dk, dv)
        else:
            hydra.attn_bwd(p, q, k, v, sh.o_bf16, sh.lse_acc, do, dq, dk, dv, sh.workspace)
        torch.cuda.synchronize()
        outs.append([t.cpu().numpy() for t in (dq, dk, dv)])
    return outs


def test_noalloc_backward_equals_the_workspace_backward_twice():
    assert hydra.lib().hydra_noalloc_scratch_bytes() == 32 << 20
    big = ([0, 300, 300, 301, 1000, 1050, 1333], 6, [(0, 1333)], [(77, 500), (1300, 33)], 2, 31)
    small = ([0, 100, 260], 4, [(0, 260)], [(0, 200)], 0, 32)
    for cu, H, qs, ks, Hkv, seed in (big, small):
        (a_dq, a_dk, a_dv), (b_dq, b_dk, b_dv) = _case(cu, H, qs, ks, Hkv, seed)
        assert np.array_equal(a_dq, b_dq) and np.array_equal(a_dk, b_dk) and np.array_equal(a_dv, b_dv)
        assert np.abs(a_dq - 0.25).max() > 0      # the gradients did accumulate


def test_noalloc_refuses_what_its_scratch_cannot_hold():
    # 16 heads x 2^22 rows: D and LSE alone need 512 MiB
    p = hydra.Problem([0, 1 << 22], 16, [(0, 1 << 22)], [(0, 256)])
    assert hydra.workspace_size(p) > hydra.lib().hydra_noalloc_scratch_bytes()
    with pytest.raises(hydra.HydraError) as e:
        hydra.attn_bwd_noalloc(p, *([None] * 9))
    assert e.value.status == -6
