"""Seeded synthetic inputs for one context-parallel rank's attention share.

This module only *draws* inputs: it holds no attention arithmetic.  Both the HIP
path (through the tests and the benchmark) and the fp64 oracle receive arrays
made here, so the two sides see bit-identical bf16 values.

Values are keyed by *global token position*: tensor ``t`` (Q=0, K=1, V=2, dO=3)
at positions ``[4096 b, 4096 (b+1))`` comes from
``numpy.random.default_rng([seed, t, b])``.  A ring chunk is the concatenation
of its segments' global rows, so any way of cutting a sequence into chunks sees
the same tokens, which is what makes "split + merge == unsplit" testable.

Workload shapes follow the paper's setting: a rank holds ``h / cp_u`` heads after
the Ulysses all-to-all and a chunk of the sequence per outer-ring step (Sec. 5.2.1,
Eq. (usp)); documents are packed into one window with attention masked across
their boundaries (Sec. 2.2); MLA materialises one K/V per head with
``d_qk = 192`` and ``d_v = 128`` (Sec. 1; Sec. 5.2.1, discussion after Eq. (comm)).
The paper's long-context datasets are internal; the document-length mix here
imitates their stated profile (Sec. 2.2: most sequences short, a few very long).
"""
from __future__ import annotations

import concurrent.futures as cf
import dataclasses
import math
import os
from typing import List, Sequence, Tuple

import numpy as np

BLOCK_ROWS = 4096
TENSOR_ID = {"q": 0, "k": 1, "v": 2, "do": 3}
D_QK = 192
D_V = 128

Segments = List[Tuple[int, int]]  # (global start, length) per segment, in local row order


def bf16_round_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round-to-nearest-even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (r >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _dist_scale(name: str, dist: str, d: int) -> float:
    if dist == "paper":      # N(0,1)/sqrt(d) for every tensor, dO unscaled
        return 1.0 if name == "do" else 1.0 / math.sqrt(d)
    if dist == "sharp":      # logits with std ~1: Q, K ~ N(0,1)
        return 1.0 if name in ("q", "k", "do") else 1.0 / math.sqrt(d)
    if dist == "spiky":      # logits with std ~4: exercises running-max rescales
        return {"q": 4.0, "k": 1.0, "do": 1.0}.get(name, 1.0 / math.sqrt(d))
    raise ValueError(f"unknown distribution {dist!r}")


def _block(t: int, b: int, seed: int, n_heads: int, d: int, scale: np.float32) -> np.ndarray:
    g = np.random.default_rng([seed, t, b])
    blk = g.standard_normal((BLOCK_ROWS, n_heads, d), dtype=np.float32)
    if scale != 1:
        blk *= scale
    return bf16_round_bits(blk)


def rows(name: str, segments: Segments, n_heads: int, d: int, seed: int = 0,
         dist: str = "paper") -> np.ndarray:
    """bf16 bit patterns, shape [sum(len), n_heads, d], rows in segment order."""
    t = TENSOR_ID[name]
    scale = np.float32(_dist_scale(name, dist, d))
    total = sum(n for _, n in segments)
    out = np.empty((total, n_heads, d), dtype=np.uint16)
    pieces = []   # (out offset, block, lo, hi)
    o = 0
    for start, n in segments:
        p, end = start, start + n
        while p < end:
            b = p // BLOCK_ROWS
            lo = p - b * BLOCK_ROWS
            hi = min(end, (b + 1) * BLOCK_ROWS) - b * BLOCK_ROWS
            pieces.append((o, b, lo, hi))
            o += hi - lo
            p += hi - lo
    blocks = sorted({b for _, b, _, _ in pieces})

    def fill(b):
        blk = _block(t, b, seed, n_heads, d, scale)
        for off, bb, lo, hi in pieces:
            if bb == b:
                out[off:off + hi - lo] = blk[lo:hi]

    if len(blocks) <= 1:
        for b in blocks:
            fill(b)
    else:
        with cf.ThreadPoolExecutor(max_workers=min(len(blocks), _threads())) as ex:
            list(ex.map(fill, blocks))
    return out


def _threads() -> int:
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:
        return max(1, min(16, os.cpu_count() or 1))


# ---------------------------------------------------------------- document mixes

#: 32K packed microbatch: one forced 16K document plus log-normal lengths with
#: median 1024 and sigma chosen so that 85% of draws fall below 2048, clipped to
#: [128, 16384], filled to 32768 tokens, order shuffled (numpy default_rng(0)).
PACKED32K_DOCS = [2449, 1304, 1098, 439, 937, 1571, 716, 675, 445, 640, 285, 628,
                  1929, 216, 1053, 1114, 16384, 885]


def sample_packed_docs(total: int = 32768, forced: int = 16384, seed: int = 0) -> List[int]:
    """The sampler that produced ``PACKED32K_DOCS`` (kept to document the recipe)."""
    from statistics import NormalDist
    sigma = math.log(2.0) / NormalDist().inv_cdf(0.85)
    rng = np.random.default_rng(seed)
    docs = [forced]
    acc = forced
    while acc < total:
        x = int(np.clip(np.rint(rng.lognormal(math.log(1024.0), sigma)), 128, 16384))
        x = min(x, total - acc)
        docs.append(x)
        acc += x
    perm = rng.permutation(len(docs))
    return [docs[i] for i in perm]


def cu_from_lengths(lengths: Sequence[int]) -> np.ndarray:
    return np.concatenate([[0], np.cumsum(np.asarray(lengths, dtype=np.int64))]).astype(np.int32)


# ---------------------------------------------------------------- workloads

@dataclasses.dataclass(frozen=True)
class Workload:
    """One rank's share: its Q chunk, the KV chunk of every ring step, the packing."""
    name: str
    cu_seqlens: Tuple[int, ...]
    n_heads: int
    q_segs: Tuple[Tuple[int, int], ...]
    kv_steps: Tuple[Tuple[Tuple[int, int], ...], ...]
    backward: bool
    d_qk: int = D_QK
    d_v: int = D_V

    @property
    def n_q(self) -> int:
        return sum(n for _, n in self.q_segs)


def zigzag_segments(seq_len: int, cp_r: int, rank: int) -> Tuple[Tuple[int, int], ...]:
    """Zigzag layout: 2*cp_r equal pieces, rank r holds pieces r and 2*cp_r-1-r."""
    q = seq_len // (2 * cp_r)
    return ((rank * q, q), ((2 * cp_r - 1 - rank) * q, q))


def _w(name, cu, h, q, steps, bwd):
    return Workload(name, tuple(int(x) for x in cu), h, tuple(q), tuple(tuple(s) for s in steps), bwd)


WORKLOADS = {
    # 3 packed docs (64, 128, 320 tokens), 4 heads, two 256-token KV chunks.
    "tiny_2step": _w("tiny_2step", [0, 64, 192, 512], 4, [(0, 512)],
                     [[(0, 256)], [(256, 256)]], False),
    # 32K packed microbatch, 16 heads (a 128-head model at Ulysses degree 8).
    "packed32k_fwd": _w("packed32k_fwd", cu_from_lengths(PACKED32K_DOCS), 16, [(0, 32768)],
                        [[(0, 32768)]], False),
    # one 256K document cut in 8 chunks of 32K; the rank's Q chunk is chunk 4.
    # steps: (a) its own chunk (diagonal), (b) chunk 0 (fully visible), (c) chunk 7 (masked).
    "ring256k_3step": _w("ring256k_3step", [0, 262144], 16, [(131072, 32768)],
                         [[(131072, 32768)], [(0, 32768)], [(229376, 32768)]], False),
    "packed32k_fwdbwd": _w("packed32k_fwdbwd", cu_from_lengths(PACKED32K_DOCS), 16, [(0, 32768)],
                           [[(0, 32768)]], True),
    # 256K document, outer ring degree 2 x inner Ulysses degree 8: rank 0 holds
    # 128K tokens in zigzag layout (quarters 0 and 3); step 1 brings rank 1's quarters 1 and 2.
    "zigzag256k_share": _w("zigzag256k_share", [0, 262144], 16, zigzag_segments(262144, 2, 0),
                           [zigzag_segments(262144, 2, 0), zigzag_segments(262144, 2, 1)], True),
}


def make_tensors(w: Workload, seed: int = 0, dist: str = "paper"):
    """bf16 bit arrays: q, dO for the Q chunk; (k, v) per ring step."""
    q = rows("q", list(w.q_segs), w.n_heads, w.d_qk, seed, dist)
    kv = [(rows("k", list(s), w.n_heads, w.d_qk, seed, dist),
           rows("v", list(s), w.n_heads, w.d_v, seed, dist)) for s in w.kv_steps]
    do = rows("do", list(w.q_segs), w.n_heads, w.d_v, seed, dist) if w.backward else None
    return q, kv, do
