"""GPU parity of the gated output fused with the reverse exchange against the gate oracle.

Tolerances (derived from the arithmetic): the kernels form products of exact bf16 inputs
in fp32 with the logistic computed from v_exp_f32 / v_rcp_f32 (relative error of s below
(|g| + 5) 2^-24, under 1e-5 for the logits used here) and round once to bf16, which is
within half an ulp, at most 2^-8 relative; an fp32 error at a rounding tie can move the
result one ulp, so elementwise outputs are within 2^-7 relative of the fp64 oracle, and
nearly all are its exact bf16 rounding.  The gate gradient is formed from the bf16 gated
output (Y * s = Y', itself within 2^-8), so it gets 2^-6; the per-head gradient is a sum
over d_v channels whose cancellation the bound scales by the sum of magnitudes.
"""
import numpy as np
import pytest

from oracle import gate as Gt
from oracle import layout as L

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _hydra():
    from paper_2609_34318_amd import hydra
    hydra.lib()
    return hydra


def _bf16(a):
    """fp64 -> bf16 bit patterns (round to nearest even) and the values they hold."""
    t = torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16), t.to(torch.float64).numpy()


def _to_f64(bits):
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()


def _inputs(T, H, d, e, seed):
    rng = np.random.default_rng(seed)
    y = rng.normal(scale=0.5, size=(T, H, d))
    g = rng.normal(scale=3.0, size=(T, H, e))
    # saturated logits and exact zeros: s = 1, s = 0, s = 1/2
    flat = g.reshape(-1)
    k = max(1, flat.size // 50)
    idx = rng.choice(flat.size, 3 * k if flat.size >= 3 * k else flat.size, replace=False)
    flat[idx[:k]] = 60.0
    flat[idx[k:2 * k]] = -100.0
    flat[idx[2 * k:]] = 0.0
    dy = rng.normal(size=(T, H, d))
    return _bf16(y), _bf16(g), _bf16(dy)


def _close(got_bits, want, rtol, what, exact_frac=0.99):
    got = _to_f64(got_bits)
    err = np.abs(got - want)
    bad = err > rtol * np.abs(want) + 1e-30
    assert not bad.any(), f"{what}: {bad.sum()} elements off, worst at {np.argwhere(bad)[0]}"
    if exact_frac and got_bits.size >= 256:
        want_bits, _ = _bf16(want)
        assert (got_bits == want_bits).mean() >= exact_frac, f"{what}: too few exact roundings"


CASES = [  # T, H, d_v, gate_dim, cp_u
    (1, 1, 8, 1, 1), (1, 1, 8, 8, 1), (7, 4, 8, 1, 4), (37, 16, 128, 128, 8), (37, 16, 128, 1, 8),
    (300, 8, 128, 1, 2), (300, 8, 128, 128, 1), (5, 12, 16, 16, 3), (33, 6, 512, 1, 3), (65, 128, 128, 128, 16),
    (65, 128, 128, 1, 16),
]


@pytest.mark.parametrize("T,H,d,e,cp_u", CASES)
def test_unpack_gated_matches_oracle(T, H, d, e, cp_u):
    hydra = _hydra()
    (yb, y), (gb, g), _ = _inputs(T, H, d, e, seed=T * 7 + H + e)
    recv = _dev(L.pack_heads(yb, cp_u))               # what the reverse exchange delivers
    out = torch.full((T, H, d), 0x7fc0, dtype=torch.int16, device="cuda")   # NaN poison
    hydra.unpack_heads_gated(recv, _dev(gb), out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint16)
    _close(got, Gt.unpack_gated(L.pack_heads(y, cp_u), g), 2.0 ** -7, "y")


@pytest.mark.parametrize("T,H,d,e,cp_u", CASES)
def test_pack_gated_bwd_matches_oracle(T, H, d, e, cp_u):
    hydra = _hydra()
    (yb, y), (gb, g), (dyb, dy) = _inputs(T, H, d, e, seed=T * 11 + H + e)
    # the forward's gated output, as bf16 (the oracle's value rounded once)
    ygb, _ = _bf16(Gt.gate_fwd(y, g))
    d_send = torch.full((cp_u, T, H // cp_u, d), 0x7fc0, dtype=torch.int16, device="cuda")
    d_gate = torch.full((T, H, e), 0x7fc0, dtype=torch.int16, device="cuda")
    hydra.pack_heads_gated_bwd(_dev(ygb), _dev(gb), _dev(dyb), d_send, d_gate)
    torch.cuda.synchronize()
    want_send, want_dg = Gt.pack_gated_bwd(y, g, dy, cp_u)
    _close(d_send.cpu().numpy().view(np.uint16), want_send, 2.0 ** -7, "d_send")
    got_dg = _to_f64(d_gate.cpu().numpy().view(np.uint16))
    if e == d:
        # formed from the rounded Y': within the bound, not expected to be the exact rounding
        _close(d_gate.cpu().numpy().view(np.uint16), want_dg, 2.0 ** -6, "d_gate", exact_frac=0)
    else:
        s = Gt.sigmoid(g)
        scale = (np.abs(dy * y * s) * Gt.sigmoid(-g)).sum(axis=2, keepdims=True)
        err = np.abs(got_dg - want_dg)
        assert np.all(err <= 2.0 ** -8 * np.abs(want_dg) + 2.0 ** -7 * scale + 1e-30)


def test_empty_and_rejected():
    hydra = _hydra()
    x = torch.zeros((0, 4, 8), dtype=torch.int16, device="cuda")
    hydra.unpack_heads_gated(x.view(1, 0, 4, 8), torch.zeros((0, 4, 1), dtype=torch.int16, device="cuda"), x)
    y = torch.zeros((4, 4, 96), dtype=torch.int16, device="cuda")
    with pytest.raises(hydra.HydraError):       # d_v not a power of two
        hydra.unpack_heads_gated(torch.zeros((1, 4, 4, 96), dtype=torch.int16, device="cuda"),
                                 torch.zeros((4, 4, 1), dtype=torch.int16, device="cuda"), y)
    y = torch.zeros((4, 4, 64), dtype=torch.int16, device="cuda")
    with pytest.raises(hydra.HydraError):       # gate_dim neither 1 nor d_v
        hydra.unpack_heads_gated(torch.zeros((2, 4, 2, 64), dtype=torch.int16, device="cuda"),
                                 torch.zeros((4, 4, 8), dtype=torch.int16, device="cuda"), y)
    with pytest.raises(hydra.HydraError):       # output aliases the input
        hydra.unpack_heads_gated(y.view(1, 4, 4, 64), torch.zeros((4, 4, 1), dtype=torch.int16, device="cuda"), y)


def test_gated_path_round_trip_through_the_group():
    """A Ulysses group of 4 ranks: head-shard outputs -> token slices -> exchange (tensor
    copies) -> gated unpack on every rank; backward: gated pack -> exchange -> each rank's dY
    of its head group for every group token, against the oracle's gradient of the whole."""
    hydra = _hydra()
    cp_u, T, H, d = 4, 24, 8, 128
    (yb, y), (gb, g), (dyb, dy) = _inputs(cp_u * T, H, d, d, seed=5)
    hg = H // cp_u
    heads = [_dev(np.ascontiguousarray(yb[:, j * hg:(j + 1) * hg])) for j in range(cp_u)]
    out = []
    for u in range(cp_u):
        recv = torch.stack([heads[j][u * T:(u + 1) * T] for j in range(cp_u)])   # the exchange
        o = torch.empty((T, H, d), dtype=torch.int16, device="cuda")
        hydra.unpack_heads_gated(recv, _dev(gb[u * T:(u + 1) * T]), o)
        out.append(o)
    torch.cuda.synchronize()
    got = np.concatenate([o.cpu().numpy().view(np.uint16) for o in out])
    _close(got, Gt.gate_fwd(y, g), 2.0 ** -7, "y")
    sends = []
    for u in range(cp_u):
        ds = torch.empty((cp_u, T, hg, d), dtype=torch.int16, device="cuda")
        dg = torch.empty((T, H, d), dtype=torch.int16, device="cuda")
        hydra.pack_heads_gated_bwd(out[u], _dev(gb[u * T:(u + 1) * T]), _dev(dyb[u * T:(u + 1) * T]), ds, dg)
        sends.append(ds)
    dy_all, _ = Gt.gate_bwd(y, g, dy)
    for j in range(cp_u):
        back = torch.cat([sends[u][j] for u in range(cp_u)])                      # the exchange
        torch.cuda.synchronize()
        _close(back.cpu().numpy().view(np.uint16), dy_all[:, j * hg:(j + 1) * hg], 2.0 ** -7, "dY")


def test_full_size_gate_sampled_and_timed():
    """The output of one rank of the 256K-token, 128-head benchmark share split over 16
    ranks (16K tokens x 128 heads x 128), per-channel gate: sampled tokens against the
    oracle, and GB/s of both kernels printed beside a plain device copy."""
    hydra = _hydra()
    T, H, d, cp_u = 16384, 128, 128, 16
    gen = torch.Generator(device="cuda").manual_seed(9)
    recv = (torch.randn((cp_u, T, H // cp_u, d), device="cuda", generator=gen) * 0.5).to(torch.bfloat16)
    gate = (torch.randn((T, H, d), device="cuda", generator=gen) * 3).to(torch.bfloat16)
    dy = torch.randn((T, H, d), device="cuda", generator=gen).to(torch.bfloat16)
    y = torch.empty((T, H, d), dtype=torch.bfloat16, device="cuda")
    d_send = torch.empty_like(recv)
    d_gate = torch.empty_like(gate)
    hydra.unpack_heads_gated(recv, gate, y)
    hydra.pack_heads_gated_bwd(y, gate, dy, d_send, d_gate)
    torch.cuda.synchronize()
    rows = torch.from_numpy(np.sort(np.random.default_rng(1).choice(T, 48, replace=False))).cuda()
    f64 = lambda t: t.to(torch.float64).cpu().numpy()
    bits = lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)
    y_s, g_s, dy_s = L.unpack_heads(f64(recv[:, rows])), f64(gate[rows]), f64(dy[rows])
    _close(bits(y[rows]), Gt.gate_fwd(y_s, g_s), 2.0 ** -7, "y")
    want_send, want_dg = Gt.pack_gated_bwd(y_s, g_s, dy_s, cp_u)
    _close(bits(d_send[:, rows]), want_send, 2.0 ** -7, "d_send")
    _close(bits(d_gate[rows]), want_dg, 2.0 ** -6, "d_gate", exact_frac=0)

    def timed(fn, n=10):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        fn()
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    n = y.numel()
    t_f = timed(lambda: hydra.unpack_heads_gated(recv, gate, y))
    t_b = timed(lambda: hydra.pack_heads_gated_bwd(y, gate, dy, d_send, d_gate))
    t_c = timed(lambda: d_send.view(-1).copy_(y.view(-1)))
    gbs_f, gbs_b, gbs_c = 6 * n / t_f / 1e6, 10 * n / t_b / 1e6, 4 * n / t_c / 1e6
    print(f"gated unpack {T}x{H}x{d}: {t_f:.3f} ms, {gbs_f:.0f} GB/s; gated pack bwd: {t_b:.3f} ms, "
          f"{gbs_b:.0f} GB/s; plain device copy: {gbs_c:.0f} GB/s")
    assert gbs_f > 500 and gbs_b > 500

