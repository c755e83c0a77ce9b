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
                        "bwd_dkdv_ds": 2 * (2 * D_QK + 2 * D_V),  # the same, and stores dS
                        "bwd_dq": 2 * (2 * D_QK + D_V),         # S, dP (recomputed), dQ
                        "bwd_dq_ds": 2 * D_QK}                  # dQ from the stored dS
PEAK_BF16_TFLOPS = 2516.6                        # 256 CU x 4096 FLOP/clk x 2.4 GHz, dense
KERNEL_SOURCES = {"attn_fwd": "attn_fwd.hip", "bwd_dkdv": "attn_bwd.hip", "bwd_dq": "attn_bwd.hip",
                  "bwd_dkdv_ds": "attn_bwd.hip", "bwd_dq_ds": "attn_bwd.hip"}


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
    for name in (KERNEL_SOURCES[kernel], "kernels.h", "tiles.h"):
        h.update(_code(os.path.join(csrc, name)))
    return h.hexdigest()[:16]


def _traffic(kernel: str, workload: str, ds_heads: int = 0):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if still current
    (same kernel code; for the stored-dS kernels also the same K/V heads per pass, since a
    launch covers one pass)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f)[f"{kernel}@{workload}"]
    except (OSError, KeyError, ValueError):
        return None
    if rec.get("source_sha") != _source_sha(kernel):
        return None
    if kernel.endswith("_ds") and rec.get("kv_heads_per_pass") != ds_heads:
        return None
    return rec.get("bytes_per_launch")


class ClockSampler:
    """Samples the GPU engine clock (and socket power when available) from a background
    thread while a timed region runs: amdsmi when the driver answers it, else rocm-smi."""

    def __init__(self, period_s: float = 0.05):
        import threading
        self.period = period_s
        self.mhz, self.watts, self.source = [], [], None
        self._stop = threading.Event()
        self._thread = threading.Thread(target=self._run, daemon=True)
        self._read = self._open()

    def _open(self):
        try:
            import amdsmi
            amdsmi.amdsmi_init()
            h = amdsmi.amdsmi_get_processor_handles()[0]
            amdsmi.amdsmi_get_clock_info(h, amdsmi.AmdSmiClkType.GFX)
            self.source = "amdsmi"

            def read():
                mhz = amdsmi.amdsmi_get_clock_info(h, amdsmi.AmdSmiClkType.GFX)["clk"]
                w = None
                try:
                    pw = amdsmi.amdsmi_get_power_info(h)
                    w = pw.get("current_socket_power") or pw.get("average_socket_power")
                    w = float(w) if isinstance(w, (int, float)) else None
                except Exception:
                    pass
                return float(mhz), w
            return read
        except Exception:
            pass
        import subprocess

        def read_smi():
            out = subprocess.run(["rocm-smi", "--showclocks"], capture_output=True, text=True, timeout=10).stdout
            m = re.search(r"sclk clock level: \d+: \((\d+)Mhz\)", out)
            return (float(m.group(1)), None) if m else (None, None)
        self.source = "rocm-smi"
        return read_smi

    def _run(self):
        while not self._stop.is_set():
            try:
                mhz, w = self._read()
                if mhz:
                    self.mhz.append(mhz)
                if w:
                    self.watts.append(w)
            except Exception:
                pass
            self._stop.wait(self.period)

    def __enter__(self):
        self._thread.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        self._thread.join(timeout=15)

    MIN_SAMPLES = 5

    def summary(self):
        """Mean, median and range of the samples; `held_mhz` (the median) is what the
        "% of peak at the measured clock" uses, and is None when the timed region was too
        short for MIN_SAMPLES readings (a reading can then be the idle clock before the
        work ramps up)."""
        if not self.mhz:
            return None
        import statistics
        med = statistics.median(self.mhz)
        out = {"source": self.source, "samples": len(self.mhz), "mean_mhz": round(statistics.fmean(self.mhz), 1),
               "median_mhz": med, "min_mhz": min(self.mhz), "max_mhz": max(self.mhz),
               "held_mhz": med if len(self.mhz) >= self.MIN_SAMPLES else None}
        if self.watts:
            out["mean_w"] = round(statistics.fmean(self.watts), 1)
        return out


def host_info() -> dict:
    """CPU model, core counts and BLAS thread settings of the host the oracle runs on."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count()
    return {"cpu_model": model, "nproc": usable, "cpu_count": os.cpu_count(),
            "OPENBLAS_NUM_THREADS": os.environ.get("OPENBLAS_NUM_THREADS"),
            "OMP_NUM_THREADS": os.environ.get("OMP_NUM_THREADS")}


def _oracle_pass(w, q, kv, do, heads, rows):
    """The oracle's forward over all ring steps (and, for a training workload, the backward
    of every step) for the given heads and query rows; returns (visible pairs x heads,
    counted FLOP, seconds)."""
    import numpy as np

    import oracle
    from paper_2609_34318_amd import inputs

    f = inputs.bf16_bits_to_f32
    union = [seg for s in w.kv_steps for seg in s]
    qh = f(q[:, heads])
    k_all = np.concatenate([f(k[:, heads]) for k, _ in kv])
    v_all = np.concatenate([f(v[:, heads]) for _, v in kv])
    qpos = oracle.row_positions(w.q_segs)[rows]
    pairs = len(heads) * sum(oracle.visible_pairs_bruteforce(list(w.cu_seqlens), [(int(p), 1) for p in qpos],
                                                             list(s)) for s in w.kv_steps)
    t0 = time.perf_counter()
    O, L = oracle.attn_fwd(qh, k_all, v_all, list(w.cu_seqlens), list(w.q_segs), union, q_rows=rows)
    if do is not None:
        doh = f(do[:, heads])
        for s, (k, v) in zip(w.kv_steps, kv):
            oracle.attn_bwd(qh, f(k[:, heads]), f(v[:, heads]), O, L, doh, list(w.cu_seqlens), list(w.q_segs),
                            list(s), q_rows=rows)
    dt = time.perf_counter() - t0
    flops = pairs * (FWD_FLOP_PER_PAIR + (BWD_FLOP_PER_PAIR if do is not None else 0))
    return pairs, flops, dt


def cpu_baseline(w, q, kv, do, budget_rows: int, heads=(0,), one_core_rows: int = -1):
    """The fp64 oracle on a bounded sample of the same workload: the given heads, the last
    `budget_rows` query rows (the longest rows of the share), forward over all ring steps
    and the backward of every step, with the host's BLAS threads; then the last
    `one_core_rows` rows (default budget_rows / 8) with one thread.  Returns counted
    TFLOP/s and what was sampled."""
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits

    nq = q.shape[0]
    heads = list(heads)
    budget_rows = min(budget_rows, nq)
    pairs, flops, dt = _oracle_pass(w, q, kv, do, heads, np.arange(nq - budget_rows, nq))
    threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("internal_api") in
                   ("openblas", "mkl", "blis")] or [1])
    what = "forward over all ring steps" + (" + backward of each step" if do is not None else "")
    out = {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
           "sample": f"{len(heads)} of {w.n_heads} heads, last {budget_rows} of {nq} query rows, {what} "
                     f"({pairs} visible pairs, {dt:.1f} s)",
           "host": host_info()}
    one = budget_rows // 8 if one_core_rows < 0 else min(one_core_rows, nq)
    if one > 0:
        with threadpool_limits(limits=1):
            p1, f1, d1 = _oracle_pass(w, q, kv, do, heads, np.arange(nq - one, nq))
        out["one_core"] = {"value": f1 / d1 / 1e12, "cores": 1,
                           "sample": f"last {one} query rows, same heads ({p1} visible pairs, {d1:.1f} s)"}
    return out


def oracle_timings(cpu_rows: int) -> int:
    """Oracle timings on every workload (host only, no GPU): the small two-step share whole
    (all heads and rows), the others on the bounded sample the bench line uses."""
    from paper_2609_34318_amd import inputs

    for name, w in inputs.WORKLOADS.items():
        q, kv, do = inputs.make_tensors(w)
        whole = q.shape[0] * w.n_heads <= 4096
        heads = range(w.n_heads) if whole else (0,)
        rows = q.shape[0] if whole else cpu_rows
        rec = cpu_baseline(w, q, kv, do, rows, heads=heads, one_core_rows=rows if whole else -1)
        print(json.dumps({"workload": name, "whole": whole, **rec}), flush=True)
    return 0


# What share of a context-parallel group each workload is (its heads are h / cp_u).
PARALLELISM = {
    "zigzag256k_share": "one rank of cp_r=2 x cp_u=8",
    "ring256k_3step": "one rank of an 8-chunk ring (3 of its steps) x cp_u=8",
    "packed32k_fwd": "one rank of cp_u=8, no ring",
    "packed32k_fwdbwd": "one rank of cp_u=8, no ring",
    "tiny_2step": "one rank, 2 ring steps",
}


def _stats(ms):
    import statistics
    return {"median_ms": round(statistics.median(ms), 3), "min_ms": round(min(ms), 3), "max_ms": round(max(ms), 3)}


def measure(w, steps: int, warmup: int, kv_heads: int = 0, graph: bool = False, fwd_only: bool = False,
            prof_steps: int = 3, copy_probe_mib: int = 0, ds_kv_heads: int = 0, ds_budget_gib: float = 0.0):
    """Runs one workload: warmup, a timed region of `steps` uninstrumented steps (per-step
    HIP events on the launch stream, engine clock sampled meanwhile), then `prof_steps`
    steps with the library's per-kernel timing on.  Returns the raw figures."""
    import numpy as np
    import torch

    from paper_2609_34318_amd import hydra, inputs, ring

    H = w.n_heads
    t_gen = time.perf_counter()
    Hkv = kv_heads or H
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

    if copy_probe_mib > 0:
        src = torch.ones(copy_probe_mib << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    sh = ring.make_share(w.cu_seqlens, H, w.q_segs, w.kv_steps, n_kv_heads=Hkv, graph_ready=graph,
                         ds_kv_heads=0 if (graph or fwd_only) else ds_kv_heads,
                         ds_budget_bytes=0 if (graph or fwd_only or ds_kv_heads == 0) else int(ds_budget_gib * 2**30))
    if graph:
        ring.plan(sh)
    pairs_step = [hydra.visible_pairs(p) for p in sh.problems]
    dq = torch.empty((sh.nq, H, D_QK), dtype=torch.float32, device="cuda")
    dkv = [(torch.empty((k.shape[0], Hkv, D_QK), dtype=torch.float32, device="cuda"),
            torch.empty((k.shape[0], Hkv, D_V), dtype=torch.float32, device="cuda")) for k, _ in kv]

    def step():
        if not fwd_only:
            dq.fill_(0.0)
            for a, b in dkv:
                a.fill_(0.0)
                b.fill_(0.0)
        ring.forward(sh, q, kv, planned=graph)
        if not fwd_only:
            ring.backward(sh, q, kv, d_o, dq, dkv, planned=graph)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    run = step
    if graph:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        run = g.replay
        run()
    # timed region: no per-kernel instrumentation, one event pair per step
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    with ClockSampler() as clk:
        t0 = time.perf_counter()
        evs[0].record()
        for i in range(steps):
            run()
            evs[i + 1].record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    step_ms = [evs[i].elapsed_time(evs[i + 1]) for i in range(steps)]
    total_ms = evs[0].elapsed_time(evs[steps])
    # per-kernel times: the same steps (eager) with the library's launch events on
    hydra.profile_start()
    for _ in range(prof_steps):
        step()
    torch.cuda.synchronize()
    prof = hydra.profile_stop()
    ds_bytes = 0 if sh.ds_buf is None else sh.ds_buf.numel()
    ds_heads = ring.ds_kv_heads_within(sh.problems, ds_bytes) if ds_bytes else 0
    return dict(H=H, Hkv=Hkv, nq=sh.nq, pairs_step=pairs_step, step_ms=step_ms, total_ms=total_ms, wall=wall,
                clock=clk.summary(), prof=prof, t_gen=t_gen, tensors=(q_b, kv_b, do_b), ds_bytes=ds_bytes,
                ds_heads=ds_heads)


def _kernel_tflops(st, pairs, name, prof_steps):
    """A kernel's own contraction FLOP/s over the profiled steps: every launch of it in a
    step (one per ring step, times the head passes of the stored-dS path) together covers
    the step's visible pairs once."""
    return pairs * KERNEL_FLOP_PER_PAIR[name] * prof_steps / (st["total_ms"] / 1e3) / 1e12


def _kernels(prof, pairs, prof_steps):
    kernels = {}
    for name, st in prof.items():
        rec = {"launches": st["launches"], "avg_ms": round(st["avg_ms"], 4), "min_ms": round(st["min_ms"], 4),
               "max_ms": round(st["max_ms"], 4), "ms_per_step": round(st["total_ms"] / prof_steps, 3)}
        if name in KERNEL_FLOP_PER_PAIR:
            rec["tflops_executed"] = round(_kernel_tflops(st, pairs, name, prof_steps), 1)
        kernels[name] = rec
    return kernels


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="zigzag256k_share")
    ap.add_argument("--cpu-rows", type=int, default=2048, help="query rows in the oracle timing sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--oracle-timings", action="store_true",
                    help="host only: time the oracle on every workload (the small share whole, the others "
                         "on the --cpu-rows sample), with the host's threads and with one; no GPU is used")
    ap.add_argument("--no-ring-config", action="store_true",
                    help="skip the 256K ring-step configuration (three KV chunks of 32K) timed after the headline")
    ap.add_argument("--ring-steps", type=int, default=20)
    ap.add_argument("--prof-steps", type=int, default=3, help="steps timed with per-kernel launch events")
    ap.add_argument("--ds-kv-heads", type=int, default=-1,
                    help="backward: K/V heads per pass of the stored-dS path (dQ from the dS the dK/dV "
                         "kernel stores, no recompute); -1: as many as fit --ds-budget-gib; 0: recompute "
                         "S and dP for dQ")
    ap.add_argument("--ds-budget-gib", type=float, default=None,
                    help="device memory for the stored dS of one pass (of 288 GB); default: the library's "
                         "(18 GiB: one K/V head per pass on the 128K share, measured faster than four)")
    ap.add_argument("--kv-heads", type=int, default=0,
                    help="K/V heads (grouped-query attention); 0: one per query head (MLA)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="run one plain device copy of this size first (counter calibration)")
    ap.add_argument("--graph", action="store_true",
                    help="plan once, record one step into a HIP graph and time its replays "
                         "(per-kernel times then come from eager steps of the same calls)")
    args = ap.parse_args()
    if args.oracle_timings:
        return oracle_timings(args.cpu_rows)
    if args.gpus != 1:
        print(f"bench.py: this build measures one GPU only (asked for --gpus {args.gpus}); "
              "run with --gpus 1", file=sys.stderr)
        return 2

    import torch

    from paper_2609_34318_amd import hydra, inputs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    hydra.lib()
    if args.ds_budget_gib is None:
        from paper_2609_34318_amd import ring
        args.ds_budget_gib = ring.DEFAULT_DS_BUDGET_BYTES / 2**30
    w = inputs.WORKLOADS[args.workload]
    r = measure(w, args.steps, args.warmup, args.kv_heads, args.graph, prof_steps=args.prof_steps,
                copy_probe_mib=args.copy_probe_mib, ds_kv_heads=args.ds_kv_heads,
                ds_budget_gib=args.ds_budget_gib)
    H, Hkv, pairs_step = r["H"], r["Hkv"], r["pairs_step"]
    ms_per_step = r["total_ms"] / args.steps
    pairs = sum(pairs_step) * H
    flop_step = pairs * (FWD_FLOP_PER_PAIR + BWD_FLOP_PER_PAIR)
    value = flop_step / (ms_per_step / 1e3) / 1e12
    prof = r["prof"]
    kernels = _kernels(prof, pairs, args.prof_steps)
    dom = max((k for k in prof if k in KERNEL_FLOP_PER_PAIR), key=lambda k: prof[k]["total_ms"])
    # per launch: the launch's share of the step's pairs x FLOP/pair over its average duration
    achieved = _kernel_tflops(prof[dom], pairs, dom, args.prof_steps)
    roofline = {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": _traffic(dom, w.name, r["ds_heads"])}
    clock = r["clock"]
    if clock:
        # the same rate against the dense peak at the engine clock held during the timed region
        clock["pct_of_peak_at_measured_clock"] = (
            round(100 * value / (PEAK_BF16_TFLOPS * clock["held_mhz"] / 2400), 2) if clock["held_mhz"] else None)
        if clock.get("mean_w") and clock["held_mhz"]:
            # the device runs at its power limit: energy per step is what a step costs
            clock["joules_per_step"] = round(clock["mean_w"] * ms_per_step / 1e3, 1)
            clock["counted_tflop_per_joule"] = round(flop_step / 1e12 / (clock["mean_w"] * ms_per_step / 1e3), 4)

    out = {
        "metric": "causal attention TFLOP/s fwd+bwd per rank; % of MI355X bf16 MFMA peak",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "step_ms": _stats(r["step_ms"]),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "seq_len": int(w.cu_seqlens[-1]), "rank_tokens": r["nq"],
                   "n_heads": H, "n_kv_heads": Hkv, "d_qk": D_QK, "d_v": D_V, "ring_steps": len(w.kv_steps),
                   "q_segments": [list(x) for x in w.q_segs],
                   "visible_pairs_per_head": pairs_step, "counted_tflop_per_step": round(flop_step / 1e12, 3),
                   "parallelism": PARALLELISM.get(w.name, "one rank"),
                   "launch": "hip graph replay" if args.graph else "eager",
                   "backward": (f"stored dS, {r['ds_heads']} K/V heads per pass ({r['ds_bytes'] / 2**30:.1f} GiB "
                                "scratch)") if r["ds_bytes"] else "dS recomputed for dQ"},
        "pct_of_peak": round(100 * value / PEAK_BF16_TFLOPS, 2),
        "flop_note": {"counted_per_pair": {"fwd": FWD_FLOP_PER_PAIR, "bwd": BWD_FLOP_PER_PAIR},
                      "bwd_without_s_recompute": BWD_FLOP_PER_PAIR - 2 * D_QK,
                      "value_without_s_recompute": round(value * (FWD_FLOP_PER_PAIR + BWD_FLOP_PER_PAIR - 2 * D_QK)
                                                         / (FWD_FLOP_PER_PAIR + BWD_FLOP_PER_PAIR), 2)},
        "clock": clock,
        "kernels": kernels,
        "kernel_timing": f"library launch events over {args.prof_steps} further eager steps; tflops_executed "
                         "counts each kernel's own contractions (bwd_dq's include its S and dP recompute, "
                         "640 of its 1024 FLOP per pair, which are not part of the counted work)",
        "roofline": roofline,
        "wall_s_timed": round(r["wall"], 3),
        "input_gen_s": round(r["t_gen"], 1),
    }
    if not args.no_ring_config and w.name != "ring256k_3step":
        # the other 256K per-rank configuration: a 32K query chunk against three 32K KV chunks
        # (diagonal, fully visible, masked), merged; forward as configured, and fwd+bwd
        wr = inputs.WORKLOADS["ring256k_3step"]
        ring_out = {}
        for label, fwd_only in (("fwd", True), ("fwd_bwd", False)):
            rr = measure(wr, args.ring_steps, 3, fwd_only=fwd_only, prof_steps=2,
                         ds_kv_heads=args.ds_kv_heads, ds_budget_gib=args.ds_budget_gib)
            pr = sum(rr["pairs_step"]) * rr["H"]
            fl = pr * (FWD_FLOP_PER_PAIR + (0 if fwd_only else BWD_FLOP_PER_PAIR))
            ms = rr["total_ms"] / args.ring_steps
            v = fl / (ms / 1e3) / 1e12
            rec = {"ms_per_step": round(ms, 3), **_stats(rr["step_ms"]), "tflops": round(v, 1),
                   "pct_of_peak": round(100 * v / PEAK_BF16_TFLOPS, 2), "counted_tflop_per_step": round(fl / 1e12, 3),
                   "kernels": {k: round(x["avg_ms"], 4) for k, x in rr["prof"].items()}}
            if rr["clock"]:
                held = rr["clock"]["held_mhz"]
                rec["clock_mean_mhz"] = rr["clock"]["mean_mhz"]
                rec["clock_held_mhz"] = held
                rec["clock_samples"] = rr["clock"]["samples"]
                rec["pct_of_peak_at_measured_clock"] = (
                    round(100 * v / (PEAK_BF16_TFLOPS * held / 2400), 2) if held else None)
            ring_out[label] = rec
        out["ring256k_3step"] = {"steps": args.ring_steps, "visible_pairs_per_head": rr["pairs_step"],
                                 **ring_out}
    if not args.no_cpu_baseline:
        q_b, kv_b, do_b = r["tensors"]
        out["cpu_baseline"] = cpu_baseline(w, q_b, kv_b, do_b, args.cpu_rows)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
