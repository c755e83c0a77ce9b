"""The scheduler's placement turned into each rank's attention share (host logic).

For every micro-batch of a scheduled batch and every rank of the pool, the rank's share
(documents of its group, head shard, zigzag rows, ring steps) is checked against what the
placement and Eq. (usp) fix: a group's ranks cover every (token, head) of each of its
sequences exactly once, every rank's ring steps bring every K/V row of its documents once,
and every problem is one the library plans."""
import numpy as np
import pytest

from paper_2609_34318_amd import hydra, inputs, placement


def _batch(seed=3, n=90):
    rng = np.random.default_rng(seed)
    lens = np.clip(np.rint(rng.lognormal(np.log(1024), 1.3, n)), 16, 65536).astype(int)
    lens[:3] = [65536, 40000, 24576]
    return [int(x) for x in lens]


@pytest.mark.parametrize("G,B,H,Hkv,multi", [(16, 16384, 16, 0, False), (16, 8192, 8, 2, False),
                                              (8, 32768, 4, 0, False), (8, 32768, 2, 0, True)])
def test_group_ranks_partition_tokens_and_heads(G, B, H, Hkv, multi):
    """multi: a configuration whose ring groups (cp_r > 1) hold several piggybacked
    documents, split into 2-document sub-shares."""
    lens = _batch()
    mb, st, sz, info = hydra.schedule(lens, G, B, pp=4, theta_over_c=1.0)
    seen_multi = False
    for m in range(int(mb.max()) + 1):
        cover = {i: np.zeros((lens[i], H), np.int32) for i in range(len(lens)) if mb[i] == m}
        for r in range(G):
            sh = placement.rank_share(lens, mb, st, sz, m, r, H, Hkv)
            if sh is None:
                continue
            assert sh.cp_u * sh.cp_r == sh.k and sh.cp_u == min(sh.k, H)
            hkv = Hkv or H
            assert sh.n_heads == H // sh.cp_u
            assert sh.n_kv_heads == max(1, hkv // sh.cp_u)
            # the shard's query heads use exactly its K/V heads
            grp = H // hkv
            used = {h // grp for h in range(sh.head0, sh.head0 + sh.n_heads)}
            assert used == set(range(sh.kv_head0, sh.kv_head0 + sh.n_kv_heads))
            seen_multi |= sh.cp_r > 1 and len(sh.parts) > 1
            for part, probs in zip(sh.parts, placement.problems(sh)):
                assert len(part.kv_steps) == sh.cp_r
                for p in probs:
                    assert hydra.workspace_size(p) > 0
                # the rank's query rows, document by document
                for d, a, b in zip(part.seqs, part.cu[:-1], part.cu[1:]):
                    for s0, n in part.q_segs:
                        lo, hi = max(s0, a), min(s0 + n, b)
                        if hi > lo:
                            cover[d][lo - a:hi - a, sh.head0:sh.head0 + sh.n_heads] += 1
                # every K/V row of the documents arrives at exactly one ring step
                kv = np.zeros(part.cu[-1], np.int32)
                for step in part.kv_steps:
                    for s0, n in step:
                        kv[s0:s0 + n] += 1
                assert (kv == 1).all()
        for i, c in cover.items():
            assert (c == 1).all(), (m, i)
    assert info["n_mbs"] == int(mb.max()) + 1
    assert seen_multi == multi


def test_zigzag_chunks_balance_causal_work():
    """Chunks rho and 2 cp_r - 1 - rho give every ring rank the same number of causal pairs
    when the length splits evenly (Sec. 3.5's ring with the zigzag reading)."""
    for s, cp_r in ((4096, 2), (4096, 4), (262144, 2)):
        pairs = []
        for r in range(cp_r):
            rows = np.concatenate([np.arange(a, a + n) for a, n in placement.zigzag_chunks(s, cp_r, r)])
            pairs.append(int((rows + 1).sum()))
        assert len(set(pairs)) == 1
        rows = np.sort(np.concatenate([np.arange(a, a + n) for r in range(cp_r)
                                       for a, n in placement.zigzag_chunks(s, cp_r, r)]))
        assert np.array_equal(rows, np.arange(s))


def test_usp_degrees_follow_the_equation():
    assert placement.usp_degrees(256, 64) == (64, 4)      # the paper's example
    assert placement.usp_degrees(8, 16) == (8, 1)
    assert placement.usp_degrees(1, 16) == (1, 1)
    with pytest.raises(ValueError):
        placement.usp_degrees(24, 16)
