"""Pins of the scheduler oracle (CPU only): closed forms of the targets, hand-worked
placements, and invariants every schedule must satisfy."""
import math

import numpy as np
import pytest

from oracle import scheduler as S


def test_ceil2_and_cp_degree_closed_forms():
    assert [S.ceil2(x) for x in (0.2, 1, 1.01, 2, 3, 4, 4.5, 1000)] == [1, 1, 2, 2, 4, 4, 8, 1024]
    # Lambda* = s_max^2 / C: with s_max = 8192 and C = 8 a sequence needs k >= s^2 * 8 / 8192^2
    s_max, C, B = 8192, 8, 1 << 30
    assert S.cp_degree(8192, s_max, C, B) == 8
    assert S.cp_degree(4096, s_max, C, B) == 2        # s^2/Lambda* = 2 exactly
    assert S.cp_degree(2897, s_max, C, B) == 2        # 2897^2 * 8 > 8192^2
    assert S.cp_degree(2896, s_max, C, B) == 1        # 2896^2 * 8 < 8192^2
    # the token budget: s / k <= B
    assert S.cp_degree(4096, s_max, C, 1024) == 4
    assert S.cp_degree(100000, 100000, 4, 1024) == 4  # capped at C


def test_cap_is_the_minimiser_of_the_cost_model():
    """Eq. (capcost)-(bgamma): T(C) = T0 + beta/C + gamma*C with beta = (pp-1) theta s_max^2,
    gamma = c W / (s_max^2 G); its continuous minimiser sqrt(beta/gamma) is C_hat."""
    rng = np.random.default_rng(0)
    lengths = [int(x) for x in rng.integers(100, 60000, 300)]
    G, B, pp, theta, c = 1024, 16384, 8, 3.0, 0.5
    t = S.targets(lengths, G, B, pp, theta / c)
    s_max, W = max(lengths), sum(s * s for s in lengths)
    beta, gamma = (pp - 1) * theta * s_max ** 2, c * W / (s_max ** 2 * G)
    grid = np.exp(np.linspace(math.log(1e-3), math.log(1e12), 400001))
    best = grid[np.argmin(beta / grid + gamma * grid)]
    assert abs(best / t.C_hat - 1) < 1e-3
    assert t.C == min(G, S.ceil2(max(t.C_mem, t.C_hat)))
    assert t.C_mem == S.ceil2(s_max / B)
    assert t.M_target == math.ceil(t.C * W / (s_max ** 2 * G))


def _check_invariants(lengths, G, B, sch, balance_ratio=0.9):
    t = sch.targets
    C, s_max = t.C, t.s_max
    seen = []
    for groups in sch.mbs:
        used = np.zeros(G, int)
        for g in groups:
            assert g.size & (g.size - 1) == 0 and g.start % g.size == 0 and g.start + g.size <= G
            assert g.size <= C
            used[g.start:g.start + g.size] += 1
            # per-rank load and tokens recomputed from the documents (exact, times C)
            load = sum(lengths[d] ** 2 * C // g.size for d in g.docs)
            tok = sum(lengths[d] * C // g.size for d in g.docs)
            assert load == g.load and tok == g.tokens
            assert load <= s_max * s_max and tok <= B * C
            for d in g.docs:
                assert g.size >= S.cp_degree(lengths[d], s_max, C, B)
            seen += g.docs
        assert used.max() <= 1                      # groups of one micro-batch are disjoint
    assert sorted(seen) == list(range(len(lengths)))
    # work conservation: a micro-batch holds at most G * Lambda* of quadratic work
    assert len(sch.mbs) >= t.M_target


@pytest.mark.parametrize("seed", range(8))
def test_invariants_on_random_batches(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(20, 400))
    lengths = [int(x) for x in np.clip(rng.lognormal(math.log(1024), 1.2, n), 16, 65536)]
    B = int(2 ** rng.integers(11, 15))
    G = max(int(2 ** rng.integers(3, 8)), S.ceil2(max(lengths) / B))   # the longest must fit
    pp = int(rng.integers(1, 9))
    sch = S.schedule(lengths, G, B, pp, theta_over_c=float(rng.uniform(0.5, 8)))
    _check_invariants(lengths, G, B, sch)


def test_longest_sequence_must_fit_the_pool():
    with pytest.raises(ValueError):
        S.targets([100000], G=8, B=1024)        # needs 128 ranks


def test_hand_worked_piggyback_without_cp():
    # pp = 1: C* = C_mem = 1, Lambda* = 64; the 2s and the 1 piggyback on the least loaded rank
    sch = S.schedule([8, 4, 4, 2, 2, 1], G=4, B=100)
    assert sch.targets.C == 1 and len(sch.mbs) == 1
    assert sch.placement() == [(0, 0, 1), (0, 1, 1), (0, 2, 1), (0, 3, 1), (0, 3, 1), (0, 3, 1)]


def test_hand_worked_capped_groups_and_ties():
    # cap 4: Lambda* = 16^2/4 = 64.  16 opens ranks 0-3 at the target, the 8s take ranks 4
    # and 5 at the target, the first 4s ranks 6 and 7; the later 4s and the 2 piggyback on
    # the least loaded of the two, the lower rank on ties.
    sch = S.schedule([16, 8, 8, 4, 4, 4, 4, 2], G=8, B=1 << 20, cap=4)
    assert sch.placement() == [(0, 0, 4), (0, 4, 1), (0, 5, 1), (0, 6, 1), (0, 7, 1), (0, 6, 1), (0, 7, 1),
                               (0, 6, 1)]
    g6 = [g for g in sch.mbs[0] if g.start == 6][0]
    assert g6.load == (16 + 16 + 4) * 4      # per-rank load times C


def test_hand_worked_full_groups_close_the_micro_batch():
    # cap 2: Lambda* = 32; each 8 needs 2 ranks and fills them to the target, so two per
    # micro-batch; the 2s fit nowhere beside them and end up in a third micro-batch
    sch = S.schedule([8, 8, 8, 8, 2, 2], G=4, B=1 << 20, cap=2)
    assert [len(m) for m in sch.mbs] == [2, 2, 2]
    assert sch.placement() == [(0, 0, 2), (0, 2, 2), (1, 0, 2), (1, 2, 2), (2, 0, 1), (2, 1, 1)]


def test_hand_worked_backfill_doubles_into_idle_ranks():
    # the 1 cannot join the full group of the 4, opens a second micro-batch on rank 0 and is
    # then spread by doubling over ranks 0-1 and 0-3 (its per-rank load drops to 1/4)
    sch = S.schedule([4, 1], G=4, B=1 << 20, cap=4)
    assert sch.placement() == [(0, 0, 4), (1, 0, 4)]
    assert sch.mbs[1][0].load == 1 and sch.mbs[1][0].tokens == 1


def test_balance_rule_stops_a_balanced_micro_batch():
    # cap 2, Lambda* times C = 64.  The 8 takes ranks 0-1 at the target, the 5s ranks 2 and 3
    # at 50 each (degree 1).  The micro-batch is then full (no free rank) and its loads are
    # within 50/64 = 0.78 of each other: with balance_ratio 0.75 it is balanced and the
    # shorter 1 opens the next micro-batch (and is backfilled over ranks 0-1); with 0.9 it is
    # not, and the 1 piggybacks on rank 2.
    sch = S.schedule([8, 5, 5, 1], G=4, B=1 << 20, cap=2, balance_ratio=0.75)
    assert sch.placement() == [(0, 0, 2), (0, 2, 1), (0, 3, 1), (1, 0, 2)]
    sch = S.schedule([8, 5, 5, 1], G=4, B=1 << 20, cap=2, balance_ratio=0.9)
    assert sch.placement() == [(0, 0, 2), (0, 2, 1), (0, 3, 1), (0, 2, 1)]
