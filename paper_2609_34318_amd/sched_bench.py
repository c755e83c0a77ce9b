"""Scheduling time of the DCP scheduler at pool sizes of 2K-16K ranks (host CPU only).

    python -m paper_2609_34318_amd.sched_bench [--ranks 2048 4096 8192 16384]

Batches are synthetic, with the length profile the paper reports for its training data:
lengths spanning orders of magnitude, most under 2K, under 0.6% above 32K, and a 256K
context.  A batch holds about four micro-batches' worth of tokens for the pool (4 * G * B).
Prints one JSON line per pool size with the scheduler's median time.  (The linear-scan
reference is timed beside it, on a 256-rank batch, by the scheduler parity tests.)
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def batch(n_tokens: int, seed: int = 0):
    """Sequence lengths summing to about n_tokens: log-normal with median 1K and
    sigma = ln 2 / Phi^-1(0.85) = 0.66878 (85% under 2K), clipped to [128, 16K], with 0.6%
    of the sequences drawn from 32K-256K."""
    rng = np.random.default_rng(seed)
    out, tot = [], 0
    while tot < n_tokens:
        if rng.random() < 0.006:
            s = int(rng.integers(32768, 262145))
        else:
            s = int(np.clip(np.rint(rng.lognormal(math.log(1024), 0.66878)), 128, 16384))
        out.append(s)
        tot += s
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--ranks", type=int, nargs="+", default=[2048, 4096, 8192, 16384])
    ap.add_argument("--budget", type=int, default=16384, help="tokens per rank (B)")
    ap.add_argument("--pp", type=int, default=8)
    ap.add_argument("--theta-over-c", type=float, default=1.0)
    ap.add_argument("--repeats", type=int, default=5)
    args = ap.parse_args()

    from paper_2609_34318_amd import hydra
    hydra.lib()
    for G in args.ranks:
        lengths = batch(4 * G * args.budget, seed=G)
        times = []
        for _ in range(args.repeats):
            t0 = time.perf_counter()
            mb, st, sz, info = hydra.schedule(lengths, G, args.budget, args.pp, args.theta_over_c)
            times.append(time.perf_counter() - t0)
        print(json.dumps({"scheduler": "hydra_schedule (C++, heaps)", "ranks": G, "sequences": len(lengths),
                          "tokens": int(sum(lengths)), "cap": info["cap"], "m_target": info["m_target"],
                          "micro_batches": info["n_mbs"], "median_s": round(float(np.median(times)), 4),
                          "min_s": round(min(times), 4)}), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
