"""The heap-accelerated C++ scheduler against the linear-scan oracle: identical placements
(integers, so bit-exact) on random and adversarial batches.  CPU only."""
import math

import numpy as np
import pytest

from oracle import scheduler as S
from paper_2609_34318_amd import hydra


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import os
    if not os.path.exists(hydra.LIB_PATH):
        from paper_2609_34318_amd import build_lib
        build_lib.build()
    return hydra.lib()


def _both(lengths, G, B, pp=1, toc=0.0, cap=None, ratio=0.9):
    try:
        ref = S.schedule(lengths, G, B, pp, toc, cap, ratio)
    except ValueError:   # e.g. a pool that is not a multiple of the derived cap: both refuse
        with pytest.raises(hydra.HydraError):
            hydra.schedule(lengths, G, B, pp, toc, cap or 0, ratio)
        return None
    mb, st, sz, info = hydra.schedule(lengths, G, B, pp, toc, cap or 0, ratio)
    got = list(zip(mb.tolist(), st.tolist(), sz.tolist()))
    assert got == ref.placement()
    t = ref.targets
    assert (info["cap"], info["c_mem"], info["m_target"], info["s_max"], info["W"]) == (t.C, t.C_mem, t.M_target,
                                                                                       t.s_max, t.W)
    assert info["c_hat"] == t.C_hat
    assert info["n_mbs"] == len(ref.mbs)
    return ref


def _paper_like(rng, n, s_hi=262144):
    # lengths spanning orders of magnitude, most under 2K, a few very long (Sec. 2.3)
    x = np.exp(rng.normal(math.log(1024), 0.67, n))
    long = rng.random(n) < 0.01
    x[long] = rng.uniform(16384, s_hi, long.sum())
    return [int(v) for v in np.clip(np.rint(x), 1, s_hi)]


@pytest.mark.parametrize("seed", range(40))
def test_random_batches_match_the_oracle(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 600))
    lengths = _paper_like(rng, n) if seed % 2 else [int(v) for v in rng.integers(1, 5000, n)]
    B = int(rng.choice([512, 2048, 4096, 16384, 65536]))
    G_pow = S.ceil2(max(lengths) / B)
    G = max(G_pow, int(2 ** rng.integers(0, 8))) * int(rng.choice([1, 1, 3]))   # some pools not a power of 2
    pp = int(rng.integers(1, 17))
    toc = float(rng.choice([0.0, 0.25, 1.0, 7.5, 100.0]))
    ratio = float(rng.choice([0.5, 0.75, 0.9, 1.0]))
    _both(lengths, G, B, pp, toc, None, ratio)


@pytest.mark.parametrize("seed", range(12))
def test_fixed_caps_and_tight_budgets(seed):
    """Small budgets make the token test bind (groups demoted to and re-admitted from the
    capacity heap); fixed caps exercise wide groups, pruning and backfill."""
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(50, 500))
    lengths = [int(v) for v in rng.integers(1, 3000, n)]
    B = int(rng.integers(200, 1500))
    c_mem = S.ceil2(max(lengths) / B)
    cap = c_mem * int(2 ** rng.integers(0, 4))
    G = cap * int(rng.integers(1, 5))
    _both(lengths, G, B, pp=1, cap=cap, ratio=float(rng.choice([0.6, 0.9])))


def test_ties_equal_lengths_and_single_sequences():
    _both([1000] * 97, 8, 1000)
    _both([3] * 50 + [2] * 50, 4, 10, cap=4)
    _both([1], 1, 1)
    _both([262144], 16, 16384)
    _both([5, 5, 5, 5, 5, 5, 5, 5, 5], 2, 5, cap=2)


def test_hand_worked_cases_through_the_library():
    for args in (([8, 4, 4, 2, 2, 1], 4, 100, 1, 0.0, None, 0.9),
                 ([16, 8, 8, 4, 4, 4, 4, 2], 8, 1 << 20, 1, 0.0, 4, 0.9),
                 ([8, 8, 8, 8, 2, 2], 4, 1 << 20, 1, 0.0, 2, 0.9),
                 ([4, 1], 4, 1 << 20, 1, 0.0, 4, 0.9),
                 ([8, 5, 5, 1], 4, 1 << 20, 1, 0.0, 2, 0.75)):
        _both(*args)


def test_invalid_arguments_rejected():
    L = hydra.lib()
    with pytest.raises(hydra.HydraError):
        hydra.schedule([100000], 8, 1024)              # the longest needs 128 ranks
    with pytest.raises(hydra.HydraError):
        hydra.schedule([10, 0], 8, 1024)               # empty sequence
    with pytest.raises(hydra.HydraError):
        hydra.schedule([10], 8, 1024, cap=3)           # cap not a power of two
    with pytest.raises(hydra.HydraError):
        hydra.schedule([10], 12, 1024, cap=8)          # cap does not divide the pool
    with pytest.raises(hydra.HydraError):
        hydra.schedule([10], 8, 1024, balance_ratio=1.5)
    mb, st, sz, info = hydra.schedule([], 8, 1024)
    assert mb.size == 0 and info["n_mbs"] == 0


def test_paper_like_batch_at_256_ranks_timed_beside_the_oracle():
    """A batch with the paper's length profile for a 256-rank pool (4 micro-batches' worth of
    16K-token ranks): identical placement; both times printed."""
    import time
    from paper_2609_34318_amd import sched_bench
    G, B = 256, 16384
    lengths = sched_bench.batch(4 * G * B, seed=G)
    t0 = time.perf_counter()
    ref = S.schedule(lengths, G, B, 8, 1.0)
    t_or = time.perf_counter() - t0
    t0 = time.perf_counter()
    mb, st, sz, info = hydra.schedule(lengths, G, B, 8, 1.0)
    t_cc = time.perf_counter() - t0
    assert list(zip(mb.tolist(), st.tolist(), sz.tolist())) == ref.placement()
    print(f"256 ranks, {len(lengths)} sequences, {len(ref.mbs)} micro-batches: oracle {t_or:.3f} s, "
          f"C++ {t_cc * 1e3:.2f} ms")
