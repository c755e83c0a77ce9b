#!/usr/bin/env python3
"""Throughput of one context-parallel rank's attention share on one MI355X.

A step is one pass of the whole hot path over the rank's share: zero the gradient
accumulators, the forward partial of every outer-ring step, the exact LSE merges (with the
bf16 cast of the final O), and the backward of every ring step (D preprocess, dQ, dK/dV).
Inputs are resident in HBM before timing starts.  Work is counted as exact visible
(query, key) pairs per head times 640 FLOP forward and 1664 FLOP backward (S recompute
included), i.e. causal FLOPs, never the masked dense work.

Prints one JSON line.  Default workload: a 256K-token document under outer ring degree 2
x inner Ulysses degree 8, rank 0's 128K zigzag share, 16 heads, d_qk = 192, d_v = 128.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

D_QK, D_V = 192, 128
FWD_FLOP_PER_PAIR = 2 * (D_QK + D_V)            # S = QK^T, O = PV
BWD_FLOP_PER_PAIR = 2 * (3 * D_QK + 2 * D_V)    # S recompute, dP, dV, dQ, dK
# contraction FLOPs each kernel performs per visible pair
KERNEL_FLOP_PER_PAIR = {"attn_fwd": FWD_FLOP_PER_PAIR,
                        "bwd_dkdv": 2 * (2 * D_QK + 2 * D_V),   # S, dP, dV, dK
                        "bwd_dq": 2 * (2 * D_QK + D_V)}         # S, dP (recomputed), dQ
PEAK_BF16_TFLOPS = 2516.6                        # 256 CU x 4096 FLOP/clk x 2.4 GHz, dense
KERNEL_SOURCES = {"attn_fwd": "attn_fwd.hip", "bwd_dkdv": "attn_bwd.hip", "bwd_dq": "attn_bwd.hip"}


def _code(path: str) -> bytes:
    """A source file without comments and with whitespace collapsed: what the compiler sees."""
    with open(path) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split()).encode()


def _source_sha(kernel: str) -> str:
    """Hash of the code a kernel is built from (its source and the shared header)."""
    csrc = os.path.join(ROOT, "paper_2609_34318_amd", "csrc")
    h = hashlib.sha256()
    for name in (KERNEL_SOURCES[kernel], "kernels.h"):
        h.update(_code(os.path.join(csrc, name)))
    return h.hexdigest()[:16]


def _traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if still current."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f)[f"{kernel}@{workload}"]
    except (OSError, KeyError, ValueError):
        return None
    if rec.get("source_sha") != _source_sha(kernel):
        return None
    return rec.get("bytes_per_launch")


def cpu_baseline(w, q, kv, do, budget_rows: int):
    """The fp64 oracle on a bounded sample of the same workload: one head, the last
    `budget_rows` query rows (the longest rows of the share), forward over all ring steps
    and the backward of every step.  Returns counted TFLOP/s and what was sampled."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import oracle
    from paper_2609_34318_amd import inputs

    f = inputs.bf16_bits_to_f32
    head = [0]
    nq = q.shape[0]
    rows = np.arange(nq - budget_rows, nq)
    union = [seg for s in w.kv_steps for seg in s]
    qh, doh = f(q[:, head]), f(do[:, head])
    k_all = np.concatenate([f(k[:, head]) for k, _ in kv])
    v_all = np.concatenate([f(v[:, head]) for _, v in kv])
    qpos = oracle.row_positions(w.q_segs)[rows]
    pairs = sum(oracle.visible_pairs_bruteforce(list(w.cu_seqlens), [(int(p), 1) for p in qpos], list(s))
                for s in w.kv_steps)
    t0 = time.perf_counter()
    O, L = oracle.attn_fwd(qh, k_all, v_all, list(w.cu_seqlens), list(w.q_segs), union, q_rows=rows)
    for s, (k, v) in zip(w.kv_steps, kv):
        oracle.attn_bwd(qh, f(k[:, head]), f(v[:, head]), O, L, doh, list(w.cu_seqlens), list(w.q_segs),
                        list(s), q_rows=rows)
    dt = time.perf_counter() - t0
    threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("internal_api") in
                   ("openblas", "mkl", "blis")] or [1])
    flops = pairs * (FWD_FLOP_PER_PAIR + BWD_FLOP_PER_PAIR)
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"1 of {w.n_heads} heads, last {budget_rows} of {nq} query rows, forward over "
                      f"both ring steps + backward of each step ({pairs} visible pairs, {dt:.1f} s)"}


# What share of a context-parallel group each workload is (its heads are h / cp_u).
PARALLELISM = {
    "zigzag256k_share": "one rank of cp_r=2 x cp_u=8",
    "ring256k_3step": "one rank of an 8-chunk ring (3 of its steps) x cp_u=8",
    "packed32k_fwd": "one rank of cp_u=8, no ring",
    "packed32k_fwdbwd": "one rank of cp_u=8, no ring",
    "tiny_2step": "one rank, 2 ring steps",
}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="zigzag256k_share")
    ap.add_argument("--cpu-rows", type=int, default=2048, help="query rows in the oracle timing sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--kv-heads", type=int, default=0,
                    help="K/V heads (grouped-query attention); 0: one per query head (MLA)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="run one plain device copy of this size first (counter calibration)")
    ap.add_argument("--graph", action="store_true",
                    help="plan once, record one step into a HIP graph and time its replays "
                         "(per-kernel times then come from one eager step of the same calls)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build measures one GPU only (asked for --gpus {args.gpus}); "
              "run with --gpus 1", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2609_34318_amd import hydra, inputs, ring

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    hydra.lib()
    w = inputs.WORKLOADS[args.workload]
    H = w.n_heads
    t_gen = time.perf_counter()
    Hkv = args.kv_heads or H
    if Hkv == H:
        q_b, kv_b, do_b = inputs.make_tensors(w)
    else:  # grouped K/V heads: the same query side, Hkv heads of K and V
        q_b, _, do_b = inputs.make_tensors(w)
        kv_b = [(inputs.rows("k", list(st), Hkv, D_QK), inputs.rows("v", list(st), Hkv, D_V)) for st in w.kv_steps]
    if do_b is None:
        do_b = inputs.rows("do", list(w.q_segs), H, D_V)
    dev = lambda b: torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).cuda()
    q, d_o = dev(q_b), dev(do_b)
    kv = [(dev(k), dev(v)) for k, v in kv_b]
    t_gen = time.perf_counter() - t_gen

    if args.copy_probe_mib > 0:
        src = torch.ones(args.copy_probe_mib << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    sh = ring.make_share(w.cu_seqlens, H, w.q_segs, w.kv_steps, n_kv_heads=Hkv, graph_ready=args.graph)
    if args.graph:
        ring.plan(sh)
    pairs_step = [hydra.visible_pairs(p) for p in sh.problems]
    dq = torch.empty((sh.nq, H, D_QK), dtype=torch.float32, device="cuda")
    dkv = [(torch.empty((k.shape[0], Hkv, D_QK), dtype=torch.float32, device="cuda"),
            torch.empty((k.shape[0], Hkv, D_V), dtype=torch.float32, device="cuda")) for k, _ in kv]

    def step():
        dq.fill_(0.0)
        for a, b in dkv:
            a.fill_(0.0)
            b.fill_(0.0)
        ring.forward(sh, q, kv, planned=args.graph)
        ring.backward(sh, q, kv, d_o, dq, dkv, planned=args.graph)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    run = step
    if args.graph:
        hydra.profile_start()  # per-kernel times from one eager step of the same calls
        step()
        prof = hydra.profile_stop()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        run = graph.replay
        run()
    else:
        hydra.profile_start()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record()
    for _ in range(args.steps):
        run()
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    if not args.graph:
        prof = hydra.profile_stop()
    ms_per_step = ev0.elapsed_time(ev1) / args.steps

    pairs = sum(pairs_step) * H
    flop_step = pairs * (FWD_FLOP_PER_PAIR + BWD_FLOP_PER_PAIR)
    value = flop_step / (ms_per_step / 1e3) / 1e12

    kernels = {}
    for name, st in prof.items():
        rec = {"launches": st["launches"], "avg_ms": round(st["avg_ms"], 4)}
        if name in KERNEL_FLOP_PER_PAIR:
            per_launch = pairs * KERNEL_FLOP_PER_PAIR[name] / len(pairs_step)
            rec["tflops"] = round(per_launch / (st["avg_ms"] / 1e3) / 1e12, 1)
        kernels[name] = rec
    dom = max((k for k in prof if k in KERNEL_FLOP_PER_PAIR), key=lambda k: prof[k]["total_ms"])
    achieved = pairs * KERNEL_FLOP_PER_PAIR[dom] / len(pairs_step) / (prof[dom]["avg_ms"] / 1e3) / 1e12
    roofline = {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": _traffic(dom, w.name)}

    out = {
        "metric": "causal attention TFLOP/s fwd+bwd per rank; % of MI355X bf16 MFMA peak",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "seq_len": int(w.cu_seqlens[-1]), "rank_tokens": sh.nq,
                   "n_heads": H, "n_kv_heads": Hkv, "d_qk": D_QK, "d_v": D_V, "ring_steps": len(w.kv_steps),
                   "q_segments": [list(s) for s in w.q_segs],
                   "visible_pairs_per_head": pairs_step, "counted_tflop_per_step": round(flop_step / 1e12, 3),
                   "parallelism": PARALLELISM.get(w.name, "one rank"),
                   "launch": "hip graph replay" if args.graph else "eager"},
        "pct_of_peak": round(100 * value / PEAK_BF16_TFLOPS, 2),
        "kernels": kernels,
        "roofline": roofline,
        "wall_s_timed": round(wall, 3),
        "input_gen_s": round(t_gen, 1),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, q_b, kv_b, do_b, args.cpu_rows)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
