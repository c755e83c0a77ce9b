"""Pins of the Ulysses x ring layout oracle (CPU only)."""
import numpy as np
import pytest

from oracle import layout as L


def test_usp_degrees_closed_form():
    # Sec. 5.2.1, Eq. (usp): pure Ulysses up to the head count, the ring takes the rest;
    # the paper's example: P = 256 with h = 64 leaves an outer ring of four ranks.
    assert L.usp_degrees(256, 64) == (64, 4)
    for P in (1, 2, 4, 8, 16):
        assert L.usp_degrees(P, 16) == (P, 1)
    assert L.usp_degrees(32, 16) == (16, 2)
    with pytest.raises(ValueError):
        L.usp_degrees(24, 16)


@pytest.mark.parametrize("s,cp_r", [(16, 1), (16, 2), (48, 3), (64, 4)])
def test_zigzag_partitions_the_sequence(s, cp_r):
    rows = [L.zigzag_rows(s, cp_r, r) for r in range(cp_r)]
    allr = np.sort(np.concatenate(rows))
    assert np.array_equal(allr, np.arange(s))
    assert all(x.size == s // cp_r for x in rows)


@pytest.mark.parametrize("s,cp_r", [(32, 2), (96, 3), (256, 4), (262144, 2)])
def test_zigzag_balances_causal_work(s, cp_r):
    # one causal document: the query at position p sees p + 1 keys; every ring rank
    # must carry the same number of visible pairs (closed form: s(s+1) / (2 cp_r))
    loads = [int((L.zigzag_rows(s, cp_r, r) + 1).sum()) for r in range(cp_r)]
    assert len(set(loads)) == 1
    assert loads[0] * cp_r == s * (s + 1) // 2


def _brute_head_shard(X, cp_u, cp_r, u, r):
    s, h, d = X.shape
    c = s // (2 * cp_r)
    g = h // cp_u
    out = np.empty((s // cp_r, g, d), X.dtype)
    for i in range(s // cp_r):
        tok = r * c + i if i < c else (2 * cp_r - 1 - r) * c + (i - c)
        for k in range(g):
            out[i, k] = X[tok, u * g + k]
    return out


@pytest.mark.parametrize("P,h,s", [(4, 4, 32), (8, 4, 64), (2, 8, 16), (6, 3, 24)])
def test_exchange_reaches_the_head_shards(P, h, s):
    cp_u, cp_r = L.usp_degrees(P, h)
    rng = np.random.default_rng(1)
    X = rng.standard_normal((s, h, 5)).astype(np.float32)
    for r in range(cp_r):
        sends = [L.pack_heads(L.seq_shard(X, cp_u, cp_r, u, r), cp_u) for u in range(cp_u)]
        recvs = L.alltoall(sends)
        for u in range(cp_u):
            got = L.gather_tokens(recvs[u])
            assert np.array_equal(got, _brute_head_shard(X, cp_u, cp_r, u, r))
        # reverse exchange (the attention output going home) restores the token shards
        back = L.alltoall([L.split_tokens(L.gather_tokens(recvs[u]), cp_u) for u in range(cp_u)])
        for u in range(cp_u):
            assert np.array_equal(L.unpack_heads(back[u]), L.seq_shard(X, cp_u, cp_r, u, r))


def test_shards_partition_tokens_and_heads():
    P, h, s = 8, 4, 64
    cp_u, cp_r = L.usp_degrees(P, h)
    X = np.arange(s * h, dtype=np.int64).reshape(s, h, 1)
    seen = np.concatenate([L.head_shard(X, cp_u, cp_r, u, r).ravel() for u in range(cp_u) for r in range(cp_r)])
    assert np.array_equal(np.sort(seen), np.arange(s * h))
    seen = np.concatenate([L.seq_shard(X, cp_u, cp_r, u, r).ravel() for u in range(cp_u) for r in range(cp_r)])
    assert np.array_equal(np.sort(seen), np.arange(s * h))
