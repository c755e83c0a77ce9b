"""GPU parity of the Ulysses x ring layout calls against the layout oracle (bit-exact)."""
import numpy as np
import pytest

from oracle import layout as L

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _hydra():
    from paper_2609_34318_amd import hydra
    hydra.lib()
    return hydra


def _bits(shape, seed, dtype=np.uint16):
    rng = np.random.default_rng(seed)
    return rng.integers(0, np.iinfo(dtype).max, size=shape, dtype=dtype)


def _dev(a):
    return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a.view(np.int32)).cuda()


def _host(t, dtype):
    return t.cpu().numpy().view(dtype)


@pytest.mark.parametrize("T,H,d,cp_u,dtype", [(1, 1, 8, 1, np.uint16), (37, 16, 192, 8, np.uint16),
                                              (64, 16, 128, 16, np.uint16), (5, 12, 4, 3, np.uint32),
                                              (300, 8, 192, 2, np.uint16)])
def test_pack_unpack_heads_bit_exact(T, H, d, cp_u, dtype):
    hydra = _hydra()
    x = _bits((T, H, d), T * 131 + H, dtype)
    src = _dev(x)
    packed = torch.empty((cp_u, T, H // cp_u, d), dtype=src.dtype, device="cuda")
    hydra.pack_heads(src, packed, cp_u)
    torch.cuda.synchronize()
    assert np.array_equal(_host(packed, dtype), L.pack_heads(x, cp_u))
    back = torch.full_like(src, -1)
    hydra.unpack_heads(packed, back, cp_u)
    torch.cuda.synchronize()
    assert np.array_equal(_host(back, dtype), x)


@pytest.mark.parametrize("S,row,cp_r", [(2, 16, 1), (64, 384, 2), (96, 128, 3), (4096, 48, 4)])
def test_zigzag_gather_scatter_bit_exact(S, row, cp_r):
    hydra = _hydra()
    x = _bits((S, row // 2), S + cp_r)
    src = _dev(x)
    for r in range(cp_r):
        shard = torch.empty((S // cp_r, row // 2), dtype=src.dtype, device="cuda")
        hydra.zigzag_gather(src, shard, cp_r, r)
        torch.cuda.synchronize()
        assert np.array_equal(_host(shard, np.uint16), x[L.zigzag_rows(S, cp_r, r)])
        # scatter writes exactly rank r's rows and leaves every other row alone
        dst = torch.full_like(src, 0x1234)
        hydra.zigzag_scatter(shard, dst, cp_r, r)
        torch.cuda.synchronize()
        want = np.full_like(x, 0x1234)
        want[L.zigzag_rows(S, cp_r, r)] = x[L.zigzag_rows(S, cp_r, r)]
        assert np.array_equal(_host(dst, np.uint16), want)


def test_group_exchange_reaches_head_shards():
    """Natural order -> zigzag ring shard -> token slice per Ulysses rank -> pack -> (the
    all-to-all, done here by tensor copies) -> the head shard each rank attends with."""
    hydra = _hydra()
    P, h, s, d = 8, 8, 256, 192
    cp_u, cp_r = L.usp_degrees(P, h)
    assert (cp_u, cp_r) == (8, 1)
    P, h = 16, 8
    cp_u, cp_r = L.usp_degrees(P, h)
    x = _bits((s, h, d), 7)
    X = _dev(x)
    for r in range(cp_r):
        shard = torch.empty((s // cp_r, h, d), dtype=X.dtype, device="cuda")
        hydra.zigzag_gather(X, shard, cp_r, r)
        n = s // P
        sends = []
        for u in range(cp_u):
            buf = torch.empty((cp_u, n, h // cp_u, d), dtype=X.dtype, device="cuda")
            hydra.pack_heads(shard[u * n:(u + 1) * n].contiguous(), buf, cp_u)
            sends.append(buf)
        for u in range(cp_u):
            recv = torch.stack([sends[j][u] for j in range(cp_u)])  # the exchange
            got = recv.reshape(cp_u * n, h // cp_u, d)
            torch.cuda.synchronize()
            assert np.array_equal(_host(got, np.uint16), L.head_shard(x, cp_u, cp_r, u, r))


def test_full_size_pack_sampled_and_timed():
    """Q of one rank before the exchange at the benchmark's scale (256K tokens, 128 heads,
    P = 16 ranks: 16K tokens x 128 heads x 192), checked on sampled tokens; prints GB/s."""
    hydra = _hydra()
    T, H, d, cp_u = 16384, 128, 192, 8
    g = torch.Generator(device="cuda").manual_seed(3)
    src = torch.randint(-32768, 32767, (T, H, d), dtype=torch.int16, device="cuda", generator=g)
    dst = torch.empty((cp_u, T, H // cp_u, d), dtype=torch.int16, device="cuda")
    hydra.pack_heads(src, dst, cp_u)
    torch.cuda.synchronize()
    rows = np.random.default_rng(0).choice(T, 64, replace=False)
    want = L.pack_heads(src[torch.from_numpy(rows).cuda()].cpu().numpy(), cp_u)
    assert np.array_equal(dst[:, torch.from_numpy(rows).cuda()].cpu().numpy(), want)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        hydra.pack_heads(src, dst, cp_u)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / 10
    gbs = 2 * src.numel() * 2 / (ms / 1e3) / 1e9
    e0.record()
    for _ in range(10):
        dst.view(-1).copy_(src.view(-1))
    e1.record()
    torch.cuda.synchronize()
    ref = 2 * src.numel() * 2 / (e0.elapsed_time(e1) / 10 / 1e3) / 1e9
    print(f"pack_heads {T}x{H}x{d} bf16: {ms:.3f} ms, {gbs:.0f} GB/s (read + write); "
          f"a plain device copy of the same bytes: {ref:.0f} GB/s")
    assert gbs > 500
