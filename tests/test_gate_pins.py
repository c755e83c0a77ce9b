"""Pins of the gated-output oracle (CPU only): special values of the logistic gate,
finite differences, torch autograd in fp64, and the exchange it is fused with."""
import numpy as np
import pytest
import torch

from oracle import gate as Gt
from oracle import layout as L


def _inputs(rng, T=5, H=4, d=8, e=None):
    e = d if e is None else e
    return rng.normal(size=(T, H, d)), rng.normal(scale=2.0, size=(T, H, e)), rng.normal(size=(T, H, d))


def test_sigmoid_special_values_and_symmetry():
    x = np.array([0.0, 1.0, -1.0, 40.0, -40.0, 800.0, -800.0])
    s = Gt.sigmoid(x)
    assert s[0] == 0.5
    assert abs(s[1] - 1 / (1 + np.exp(-1))) < 1e-16 and abs(s[1] + s[2] - 1) < 1e-16
    assert s[5] == 1.0 and s[6] == 0.0 and np.all(np.isfinite(s))     # no overflow either side
    assert abs(s[3] - 1) < 1e-17 and 0 < s[4] < 1e-17


@pytest.mark.parametrize("e", [1, 8])
def test_gate_special_cases(e):
    rng = np.random.default_rng(1)
    y, g, _ = _inputs(rng, e=e)
    assert np.array_equal(Gt.gate_fwd(y, np.zeros_like(g)), y / 2)
    assert np.allclose(Gt.gate_fwd(y, np.full_like(g, 50.0)), y, rtol=1e-15, atol=0)
    assert np.abs(Gt.gate_fwd(y, np.full_like(g, -50.0))).max() < 1e-20
    # sigmoid(g) + sigmoid(-g) = 1: the two gated outputs add back to Y
    assert np.allclose(Gt.gate_fwd(y, g) + Gt.gate_fwd(y, -g), y, rtol=0, atol=1e-15)


def test_headwise_gate_is_the_broadcast_elementwise_gate():
    rng = np.random.default_rng(2)
    y, g, dyg = _inputs(rng, e=1)
    gb = np.repeat(g, y.shape[2], axis=2)
    assert np.array_equal(Gt.gate_fwd(y, g), Gt.gate_fwd(y, gb))
    dy1, dg1 = Gt.gate_bwd(y, g, dyg)
    dyb, dgb = Gt.gate_bwd(y, gb, dyg)
    assert np.allclose(dy1, dyb, rtol=1e-15, atol=0)
    assert np.allclose(dg1[..., 0], dgb.sum(axis=2), rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("e", [1, 8])
def test_gradients_match_finite_differences(e):
    rng = np.random.default_rng(3 + e)
    y, g, dyg = _inputs(rng, T=3, H=2, d=8, e=e)
    dy, dg = Gt.gate_bwd(y, g, dyg)

    def loss(yy, gg):
        return float((Gt.gate_fwd(yy, gg) * dyg).sum())

    h = 1e-6
    for idx in [(0, 0, 0), (1, 1, 3), (2, 0, 7)]:
        yp, ym = y.copy(), y.copy()
        yp[idx] += h
        ym[idx] -= h
        assert abs((loss(yp, g) - loss(ym, g)) / (2 * h) - dy[idx]) < 1e-8
        gi = idx if e > 1 else idx[:2] + (0,)
        gp, gm = g.copy(), g.copy()
        gp[gi] += h
        gm[gi] -= h
        assert abs((loss(y, gp) - loss(y, gm)) / (2 * h) - dg[gi]) < 1e-8


@pytest.mark.parametrize("e", [1, 8])
def test_gate_gradient_at_saturated_logits(e):
    # sigmoid'(g) = e^-|g| / (1 + e^-|g|)^2 for either sign: tiny but not zero (fp64 holds
    # e^-100); the relative accuracy must survive s rounding to 1
    rng = np.random.default_rng(11)
    y, _, dyg = _inputs(rng, T=2, H=2, d=8, e=e)
    for gv in (37.0, 60.0, 100.0, -60.0, -100.0):
        g = np.full((2, 2, e), gv)
        _, dg = Gt.gate_bwd(y, g, dyg)
        t = np.exp(-abs(gv))
        want = dyg * y * (t / (1 + t) ** 2)
        if e == 1:
            want = want.sum(axis=2, keepdims=True)
        assert np.all(dg != 0)
        assert np.allclose(dg, want, rtol=1e-13, atol=0)


@pytest.mark.parametrize("e", [1, 16])
def test_gradients_match_torch_autograd(e):
    rng = np.random.default_rng(7)
    y, g, dyg = _inputs(rng, T=6, H=3, d=16, e=e)
    ty = torch.tensor(y, requires_grad=True)
    tg = torch.tensor(g, requires_grad=True)
    out = ty * torch.sigmoid(tg)
    out.backward(torch.tensor(dyg))
    assert np.allclose(Gt.gate_fwd(y, g), out.detach().numpy(), rtol=1e-15, atol=1e-16)
    dy, dg = Gt.gate_bwd(y, g, dyg)
    assert np.allclose(dy, ty.grad.numpy(), rtol=1e-14, atol=1e-16)
    assert np.allclose(dg, tg.grad.numpy(), rtol=1e-13, atol=1e-15)


def test_bad_gate_shapes_rejected():
    y = np.zeros((2, 3, 8))
    for shape in [(2, 3, 4), (2, 2, 8), (3, 3, 1)]:
        with pytest.raises(ValueError):
            Gt.gate_fwd(y, np.zeros(shape))


@pytest.mark.parametrize("cp_u,e", [(1, 1), (2, 8), (4, 1), (4, 8)])
def test_fused_exchange_steps_equal_exchange_then_gate(cp_u, e):
    """The gate in the token layout after the reverse exchange: every rank of a Ulysses
    group gets its own tokens' output of every head, gated by its own logits; the backward
    send buffers, exchanged, give each rank dY of its head group for every group token."""
    rng = np.random.default_rng(10 + cp_u)
    T, H, d = 3, 8, 8
    # the attention output of the whole group in head-shard layout: rank j holds all
    # cp_u * T tokens of head group j
    y_all = rng.normal(size=(cp_u * T, H, d))
    g_all = rng.normal(size=(cp_u * T, H, e))
    dyg_all = rng.normal(size=(cp_u * T, H, d))
    hg = H // cp_u
    head_side = [y_all[:, j * hg:(j + 1) * hg] for j in range(cp_u)]
    recv = L.alltoall([L.split_tokens(x, cp_u) for x in head_side])
    for u in range(cp_u):
        tok = slice(u * T, (u + 1) * T)
        out = Gt.unpack_gated(recv[u], g_all[tok])
        assert np.array_equal(out, y_all[tok] * Gt.sigmoid(g_all[tok]))
    sends, dgs = zip(*[Gt.pack_gated_bwd(y_all[u * T:(u + 1) * T], g_all[u * T:(u + 1) * T],
                                         dyg_all[u * T:(u + 1) * T], cp_u) for u in range(cp_u)])
    back = L.alltoall(list(sends))
    dy_all, dg_all = Gt.gate_bwd(y_all, g_all, dyg_all)
    for j in range(cp_u):
        assert np.array_equal(L.gather_tokens(back[j]), dy_all[:, j * hg:(j + 1) * hg])
    assert np.array_equal(np.concatenate(dgs), dg_all)
