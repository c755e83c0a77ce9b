"""ctypes binding of libhydra_attn.so: argument marshalling only.

Every compute step runs in the library's HIP kernels; torch supplies device memory and
the current stream.  If the library is missing this module raises on first use: there
is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libhydra_attn.so")

HYDRA_OK = 0
MAX_SEGS = 4
STATUS = {0: "ok", -1: "invalid", -2: "unsupported", -3: "align", -4: "workspace", -5: "hip", -6: "too large"}


class Chunk(ctypes.Structure):
    _fields_ = [("n_segs", ctypes.c_int32),
                ("start", ctypes.c_int32 * MAX_SEGS),
                ("len", ctypes.c_int32 * MAX_SEGS)]


class ProblemC(ctypes.Structure):
    _fields_ = [("n_heads", ctypes.c_int32),
                ("d_qk", ctypes.c_int32),
                ("d_v", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float),
                ("cu_seqlens", ctypes.POINTER(ctypes.c_int32)),
                ("n_docs", ctypes.c_int32),
                ("q", Chunk),
                ("kv", Chunk),
                ("n_kv_heads", ctypes.c_int32),
                ("q_tok_stride", ctypes.c_int32),
                ("k_tok_stride", ctypes.c_int32),
                ("v_tok_stride", ctypes.c_int32)]


class SchedConfig(ctypes.Structure):
    _fields_ = [("n_ranks", ctypes.c_int32),
                ("token_budget", ctypes.c_int64),
                ("pp", ctypes.c_int32),
                ("theta_over_c", ctypes.c_double),
                ("cap", ctypes.c_int32),
                ("balance_ratio", ctypes.c_double)]


class SchedSummary(ctypes.Structure):
    _fields_ = [("w_hi", ctypes.c_int64),
                ("w_lo", ctypes.c_int64),
                ("s_max", ctypes.c_int64),
                ("c_mem", ctypes.c_int32),
                ("c_hat", ctypes.c_double),
                ("cap", ctypes.c_int32),
                ("m_target", ctypes.c_int64),
                ("n_mbs", ctypes.c_int32),
                ("max_load_x_cap", ctypes.c_int64)]


class KernelStat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32),
                ("launches", ctypes.c_int64),
                ("total_ms", ctypes.c_double),
                ("min_ms", ctypes.c_double),
                ("max_ms", ctypes.c_double)]


class HydraError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what} failed: status {status} ({lib().hydra_strerror(status).decode()})")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_34318_amd.build_lib`")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER(ProblemC)
        vp, f = ctypes.c_void_p, ctypes.POINTER(ctypes.c_float)
        L.hydra_workspace_size.argtypes = [P]
        L.hydra_workspace_size.restype = ctypes.c_size_t
        L.hydra_attn_fwd.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
        L.hydra_attn_fwd.restype = ctypes.c_int
        L.hydra_attn_bwd.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
        L.hydra_attn_bwd.restype = ctypes.c_int
        L.hydra_attn_bwd_ds.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp,
                                        ctypes.c_size_t, vp]
        L.hydra_attn_bwd_ds.restype = ctypes.c_int
        L.hydra_bwd_ds_bytes.argtypes = [P, ctypes.c_int32]
        L.hydra_bwd_ds_bytes.restype = ctypes.c_size_t
        L.hydra_attn_bwd_noalloc.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.hydra_attn_bwd_noalloc.restype = ctypes.c_int
        L.hydra_noalloc_scratch_bytes.argtypes = []
        L.hydra_noalloc_scratch_bytes.restype = ctypes.c_size_t
        L.hydra_attn_plan.argtypes = [P, vp, ctypes.c_size_t, vp]
        L.hydra_attn_plan.restype = ctypes.c_int
        L.hydra_attn_fwd_planned.argtypes = L.hydra_attn_fwd.argtypes
        L.hydra_attn_fwd_planned.restype = ctypes.c_int
        L.hydra_attn_bwd_planned.argtypes = L.hydra_attn_bwd.argtypes
        L.hydra_attn_bwd_planned.restype = ctypes.c_int
        L.hydra_lse_merge.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, vp, vp, vp, vp, vp, vp]
        L.hydra_lse_merge.restype = ctypes.c_int
        L.hydra_strerror.argtypes = [ctypes.c_int]
        L.hydra_strerror.restype = ctypes.c_char_p
        L.hydra_visible_pairs.argtypes = [P]
        L.hydra_visible_pairs.restype = ctypes.c_int64
        L.hydra_plan_items.argtypes = [P, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32), ctypes.c_int64]
        L.hydra_plan_items.restype = ctypes.c_int64
        L.hydra_tile_rows.argtypes = [ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32)]
        L.hydra_tile_rows.restype = None
        L.hydra_profile_start.argtypes = []
        L.hydra_profile_start.restype = ctypes.c_int
        L.hydra_profile_stop.argtypes = [ctypes.POINTER(KernelStat), ctypes.c_int32]
        L.hydra_profile_stop.restype = ctypes.c_int
        i32, i64 = ctypes.c_int32, ctypes.c_int64
        for name in ("hydra_pack_heads", "hydra_unpack_heads"):
            getattr(L, name).argtypes = [i64, i32, i32, i32, vp, vp, vp]
            getattr(L, name).restype = ctypes.c_int
        L.hydra_schedule.argtypes = [ctypes.POINTER(ctypes.c_int64), i64, ctypes.POINTER(SchedConfig),
                                     ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32),
                                     ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(SchedSummary)]
        L.hydra_schedule.restype = ctypes.c_int
        for name in ("hydra_zigzag_gather", "hydra_zigzag_scatter"):
            getattr(L, name).argtypes = [i64, i64, i32, i32, vp, vp, vp]
            getattr(L, name).restype = ctypes.c_int
        L.hydra_unpack_heads_gated.argtypes = [i64, i32, i32, i32, i32, vp, vp, vp, vp]
        L.hydra_unpack_heads_gated.restype = ctypes.c_int
        L.hydra_pack_heads_gated_bwd.argtypes = [i64, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp]
        L.hydra_pack_heads_gated_bwd.restype = ctypes.c_int
        _lib = L
    return _lib


def _chunk(segs: Sequence[Tuple[int, int]]) -> Chunk:
    segs = list(segs)
    if len(segs) > MAX_SEGS:
        raise ValueError(f"at most {MAX_SEGS} segments per chunk")
    c = Chunk()
    c.n_segs = len(segs)
    for i, (s, n) in enumerate(segs):
        c.start[i] = int(s)
        c.len[i] = int(n)
    return c


class Problem:
    """One ring step of one rank: head shard, documents, Q chunk and KV chunk."""

    def __init__(self, cu_seqlens, n_heads: int, q_segs, kv_segs, softmax_scale: float = 0.0,
                 d_qk: int = 192, d_v: int = 128, n_kv_heads: int = 0):
        self.cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
        self.q_segs = [tuple(map(int, s)) for s in q_segs]
        self.kv_segs = [tuple(map(int, s)) for s in kv_segs]
        self.c = ProblemC()
        self.c.n_heads = n_heads
        self.c.d_qk = d_qk
        self.c.d_v = d_v
        self.c.softmax_scale = softmax_scale
        self.c.cu_seqlens = self.cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        self.c.n_docs = len(self.cu) - 1
        self.c.q = _chunk(self.q_segs)
        self.c.kv = _chunk(self.kv_segs)
        self.c.n_kv_heads = n_kv_heads
        self.n_heads = n_heads
        self.n_kv_heads = n_kv_heads or n_heads
        self.nq = sum(n for _, n in self.q_segs)
        self.nk = sum(n for _, n in self.kv_segs)

    @property
    def ref(self):
        return ctypes.byref(self.c)


def workspace_size(p: Problem) -> int:
    return int(lib().hydra_workspace_size(p.ref))


def visible_pairs(p: Problem) -> int:
    n = int(lib().hydra_visible_pairs(p.ref))
    if n < 0:
        raise HydraError(-1, "hydra_visible_pairs")
    return n


def plan_items(p: Problem, which: int) -> np.ndarray:
    n = int(lib().hydra_plan_items(p.ref, which, None, 0))
    if n < 0:
        raise HydraError(n, "hydra_plan_items")
    out = np.zeros((max(n, 1), 16), dtype=np.int32)
    lib().hydra_plan_items(p.ref, which, out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), n)
    return out[:n]


def tile_rows() -> Tuple[int, int]:
    a, b = ctypes.c_int32(), ctypes.c_int32()
    lib().hydra_tile_rows(ctypes.byref(a), ctypes.byref(b))
    return a.value, b.value


# ------------------------------------------------------------------ device calls (torch tensors)

def _ptr(t, what: str = "tensor", dtypes=None, numel: Optional[int] = None) -> Optional[int]:
    """Device address of a dense device tensor (None passes through).  The library only sees
    plain pointers, so a host, strided, wrongly typed or wrongly sized tensor is refused here
    instead of reaching a kernel."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{what}: a device tensor is required")
    if not t.is_contiguous():
        raise ValueError(f"{what}: a contiguous tensor is required")
    if dtypes is not None and _dt(t) not in dtypes:
        raise ValueError(f"{what}: dtype {t.dtype} is not one of {dtypes}")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{what}: {t.numel()} elements, expected {numel}")
    return t.data_ptr()


def _dt(t) -> str:
    return str(t.dtype).replace("torch.", "")


_BF16 = ("bfloat16", "int16")  # bf16 values, or their raw 16-bit patterns


def _rows(t, what: str, rows: int, heads: int, d: int) -> Tuple[Optional[int], int]:
    """Address and token-row stride (elements) of a token-major [rows, heads, d] bf16 device
    tensor whose heads are contiguous within a row; its rows may be further apart (a view
    into a fused buffer).  None passes through with stride 0 (dense)."""
    if t is None:
        return None, 0
    if not t.is_cuda:
        raise ValueError(f"{what}: a device tensor is required")
    if _dt(t) not in _BF16:
        raise ValueError(f"{what}: dtype {t.dtype} is not one of {_BF16}")
    if tuple(t.shape) != (rows, heads, d):
        raise ValueError(f"{what}: shape {tuple(t.shape)}, expected {(rows, heads, d)}")
    if rows and (t.stride(2) != 1 or (heads > 1 and t.stride(1) != d)):
        raise ValueError(f"{what}: heads and channels must be contiguous within a token row")
    if rows > 1 and t.stride(0) < heads * d:
        # an expanded (broadcast) or overlapping view: the library would read rows that the
        # allocation does not hold (a stride of 0 even means "dense" to it)
        raise ValueError(f"{what}: token rows {t.stride(0)} elements apart overlap; at least {heads * d} needed")
    return t.data_ptr(), (t.stride(0) if rows > 1 else heads * d)
_F32 = ("float32",)


def _stream(stream) -> int:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _check(rc: int, what: str):
    if rc != HYDRA_OK:
        raise HydraError(rc, what)


def _set_rows(p: Problem, q, k, v):
    """Checks q, k, v against the problem and records their token-row strides in it."""
    qp, p.c.q_tok_stride = _rows(q, "q", p.nq, p.n_heads, 192)
    kp, p.c.k_tok_stride = _rows(k, "k", p.nk, p.n_kv_heads, 192)
    vp, p.c.v_tok_stride = _rows(v, "v", p.nk, p.n_kv_heads, 128)
    return qp, kp, vp


def attn_plan(p: Problem, workspace, stream=None):
    """Uploads the complete work plan of p into workspace (outside any graph capture), for
    the planned calls below."""
    _check(lib().hydra_attn_plan(p.ref, _ptr(workspace, "workspace"), workspace.numel() * workspace.element_size(),
                                 _stream(stream)), "hydra_attn_plan")


def attn_fwd(p: Problem, q, k, v, o_part, lse_part, workspace, o_bf16=None, stream=None, planned=False):
    """Partial O (fp32) and LSE of one ring step; optional bf16 copy of O.  q, k, v may be
    views whose token rows are further apart than dense (e.g. slices of a fused buffer).
    planned: the workspace already holds p's plan (attn_plan); only kernels are launched,
    so the call can be recorded into a graph."""
    nqh = p.nq * p.n_heads
    qp, kp, vp = _set_rows(p, q, k, v)
    fn = lib().hydra_attn_fwd_planned if planned else lib().hydra_attn_fwd
    _check(fn(p.ref, qp, kp, vp, _ptr(o_part, "o_part", _F32, nqh * 128),
                                _ptr(lse_part, "lse_part", _F32, nqh), _ptr(o_bf16, "o_bf16", _BF16, nqh * 128),
                                _ptr(workspace, "workspace"), workspace.numel() * workspace.element_size(),
                                _stream(stream)), "hydra_attn_fwd")


def attn_bwd(p: Problem, q, k, v, o_final_bf16, lse_final, d_o, dq_acc, dk_acc, dv_acc, workspace,
             stream=None, planned=False):
    """dQ/dK/dV of one ring step, accumulated (+=) into fp32 buffers (q, k, v and planned as
    in attn_fwd)."""
    nqh, nkh = p.nq * p.n_heads, p.nk * p.n_kv_heads
    qp, kp, vp = _set_rows(p, q, k, v)
    fn = lib().hydra_attn_bwd_planned if planned else lib().hydra_attn_bwd
    _check(fn(p.ref, qp, kp, vp, _ptr(o_final_bf16, "o_final", _BF16, nqh * 128),
                                _ptr(lse_final, "lse_final", _F32, nqh), _ptr(d_o, "d_o", _BF16, nqh * 128),
                                _ptr(dq_acc, "dq_acc", _F32, nqh * 192), _ptr(dk_acc, "dk_acc", _F32, nkh * 192),
                                _ptr(dv_acc, "dv_acc", _F32, nkh * 128), _ptr(workspace, "workspace"),
                                workspace.numel() * workspace.element_size(), _stream(stream)),
           "hydra_attn_bwd")


def attn_bwd_noalloc(p: Problem, q, k, v, o_final_bf16, lse_final, d_o, dq_acc, dk_acc, dv_acc, stream=None):
    """attn_bwd with the library's own per-GPU scratch as the workspace (allocates nothing;
    calls on one GPU must not overlap)."""
    nqh, nkh = p.nq * p.n_heads, p.nk * p.n_kv_heads
    qp, kp, vp = _set_rows(p, q, k, v)
    _check(lib().hydra_attn_bwd_noalloc(p.ref, qp, kp, vp, _ptr(o_final_bf16, "o_final", _BF16, nqh * 128),
                                        _ptr(lse_final, "lse_final", _F32, nqh), _ptr(d_o, "d_o", _BF16, nqh * 128),
                                        _ptr(dq_acc, "dq_acc", _F32, nqh * 192),
                                        _ptr(dk_acc, "dk_acc", _F32, nkh * 192),
                                        _ptr(dv_acc, "dv_acc", _F32, nkh * 128), _stream(stream)),
           "hydra_attn_bwd_noalloc")


def bwd_ds_bytes(p: Problem, kv_heads_per_pass: int) -> int:
    """Bytes of dS scratch attn_bwd_ds needs per pass of that many K/V heads (0: the
    stored-dS path does not apply to p)."""
    return int(lib().hydra_bwd_ds_bytes(p.ref, kv_heads_per_pass))


def attn_bwd_ds(p: Problem, q, k, v, o_final_bf16, lse_final, d_o, dq_acc, dk_acc, dv_acc, ds_buf, workspace,
                stream=None):
    """attn_bwd with dQ from the dS the dK/dV kernel stores into ds_buf (a uint8 device
    tensor; None or too small: the recompute path)."""
    nqh, nkh = p.nq * p.n_heads, p.nk * p.n_kv_heads
    qp, kp, vp = _set_rows(p, q, k, v)
    _check(lib().hydra_attn_bwd_ds(p.ref, qp, kp, vp, _ptr(o_final_bf16, "o_final", _BF16, nqh * 128),
                                   _ptr(lse_final, "lse_final", _F32, nqh), _ptr(d_o, "d_o", _BF16, nqh * 128),
                                   _ptr(dq_acc, "dq_acc", _F32, nqh * 192), _ptr(dk_acc, "dk_acc", _F32, nkh * 192),
                                   _ptr(dv_acc, "dv_acc", _F32, nkh * 128), _ptr(ds_buf, "ds_buf"),
                                   0 if ds_buf is None else ds_buf.numel() * ds_buf.element_size(),
                                   _ptr(workspace, "workspace"), workspace.numel() * workspace.element_size(),
                                   _stream(stream)), "hydra_attn_bwd_ds")


def lse_merge(o_acc, lse_acc, o_part, lse_part, o_bf16=None, stream=None):
    """(o_acc, lse_acc) <- exact merge with (o_part, lse_part), in place."""
    n_rows, n_heads, d_v = o_acc.shape
    n = n_rows * n_heads
    _check(lib().hydra_lse_merge(n_rows, n_heads, d_v, _ptr(o_acc, "o_acc", _F32), _ptr(lse_acc, "lse_acc", _F32, n),
                                 _ptr(o_part, "o_part", _F32, n * d_v), _ptr(lse_part, "lse_part", _F32, n),
                                 _ptr(o_bf16, "o_bf16", _BF16, n * d_v), _stream(stream)), "hydra_lse_merge")


# ------------------------------------------------------------------ Ulysses x ring layout

def pack_heads(src, dst, cp_u: int, stream=None):
    """src [T, H, ...] -> dst [cp_u, T, H/cp_u, ...]: the send buffers of the forward exchange."""
    T, H = src.shape[0], src.shape[1]
    hb = src[0, 0].numel() * src.element_size()
    _check(lib().hydra_pack_heads(T, H, hb, cp_u, _ptr(src, "src"), _ptr(dst, "dst", (_dt(src),), src.numel()),
                                  _stream(stream)), "hydra_pack_heads")


def unpack_heads(src, dst, cp_u: int, stream=None):
    """src [cp_u, T, H/cp_u, ...] -> dst [T, H, ...]: the inverse of pack_heads."""
    T, H = dst.shape[0], dst.shape[1]
    hb = dst[0, 0].numel() * dst.element_size()
    _check(lib().hydra_unpack_heads(T, H, hb, cp_u, _ptr(src, "src", (_dt(dst),), dst.numel()), _ptr(dst, "dst"),
                                    _stream(stream)), "hydra_unpack_heads")


def zigzag_gather(src, dst, cp_r: int, r: int, stream=None):
    """Natural-order rows src [S, ...] -> ring rank r's rows dst [S/cp_r, ...]."""
    S = src.shape[0]
    rb = src[0].numel() * src.element_size()
    n = src.numel() // cp_r if cp_r > 0 else None
    _check(lib().hydra_zigzag_gather(S, rb, cp_r, r, _ptr(src, "src"), _ptr(dst, "dst", (_dt(src),), n),
                                     _stream(stream)), "hydra_zigzag_gather")


def zigzag_scatter(src, dst, cp_r: int, r: int, stream=None):
    """Ring rank r's rows src [S/cp_r, ...] -> their natural positions in dst [S, ...]."""
    S = dst.shape[0]
    rb = dst[0].numel() * dst.element_size()
    n = dst.numel() // cp_r if cp_r > 0 else None
    _check(lib().hydra_zigzag_scatter(S, rb, cp_r, r, _ptr(src, "src", (_dt(dst),), n), _ptr(dst, "dst"),
                                      _stream(stream)), "hydra_zigzag_scatter")


# ------------------------------------------------------------------ gated output

def unpack_heads_gated(recv, gate, y, stream=None):
    """recv [cp_u, T, H/cp_u, d_v] bf16, gate logits [T, H, 1 or d_v] bf16 -> y [T, H, d_v] bf16,
    y = unpacked output * sigmoid(gate)."""
    cp_u = recv.shape[0]
    T, H, d_v = y.shape
    e = gate.shape[-1]
    _check(lib().hydra_unpack_heads_gated(T, H, d_v, e, cp_u, _ptr(recv, "recv", _BF16, T * H * d_v),
                                          _ptr(gate, "gate", _BF16, T * H * e), _ptr(y, "y", _BF16),
                                          _stream(stream)), "hydra_unpack_heads_gated")


def pack_heads_gated_bwd(y, gate, d_y, d_send, d_gate, stream=None):
    """Backward of unpack_heads_gated from the gated output y: d_send [cp_u, T, H/cp_u, d_v] and
    d_gate [T, H, 1 or d_v], all bf16."""
    cp_u = d_send.shape[0]
    T, H, d_v = y.shape
    e, n = gate.shape[-1], T * H * d_v
    _check(lib().hydra_pack_heads_gated_bwd(T, H, d_v, e, cp_u, _ptr(y, "y", _BF16), _ptr(gate, "gate", _BF16, T * H * e),
                                            _ptr(d_y, "d_y", _BF16, n), _ptr(d_send, "d_send", _BF16, n),
                                            _ptr(d_gate, "d_gate", _BF16, T * H * e), _stream(stream)),
           "hydra_pack_heads_gated_bwd")


# ------------------------------------------------------------------ scheduler (host only)

def schedule(lengths, n_ranks: int, token_budget: int, pp: int = 1, theta_over_c: float = 0.0, cap: int = 0,
             balance_ratio: float = 0.0):
    """Load-driven DCP placement of a batch: per sequence (micro-batch, group start, group
    size) as three int32 arrays, plus the targets and counts as a dict."""
    ln = np.ascontiguousarray(np.asarray(lengths, dtype=np.int64))
    n = ln.size
    mb, st, sz = (np.empty(n, np.int32) for _ in range(3))
    cfg = SchedConfig(n_ranks, token_budget, pp, theta_over_c, cap, balance_ratio)
    summ = SchedSummary()
    p32 = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    _check(lib().hydra_schedule(ln.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), n, ctypes.byref(cfg), p32(mb),
                                p32(st), p32(sz), ctypes.byref(summ)), "hydra_schedule")
    info = {f: getattr(summ, f) for f, _ in SchedSummary._fields_}
    info["W"] = (info.pop("w_hi") << 62) + info.pop("w_lo")
    return mb, st, sz, info


def profile_start():
    """Start timing every kernel the library launches (HIP events on the launch stream)."""
    _check(lib().hydra_profile_start(), "hydra_profile_start")


def profile_stop() -> dict:
    """Stop timing; returns {kernel: {launches, total_ms, min_ms, max_ms, avg_ms}}."""
    buf = (KernelStat * 16)()
    n = lib().hydra_profile_stop(buf, 16)
    if n < 0:
        raise HydraError(n, "hydra_profile_stop")
    out = {}
    for i in range(min(n, 16)):
        k = buf[i]
        out[k.name.decode()] = dict(launches=k.launches, total_ms=k.total_ms, min_ms=k.min_ms,
                                    max_ms=k.max_ms, avg_ms=k.total_ms / max(k.launches, 1))
    return out
