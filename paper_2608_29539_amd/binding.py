"""ctypes binding for liblogo.so (argument marshalling only).

Each ``logo_*`` function takes torch tensors on the current CUDA/HIP device,
checks dtype / shape / contiguity, allocates outputs and workspace with torch
when the caller does not pass them, and calls the C entry point of the same
name on ``torch.cuda.current_stream()``.  No arithmetic of the layer happens
here.  A failing status raises ``LogoError``.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(HERE, "liblogo.so")

LOGO_SEL_THRESHOLD = 0
LOGO_SEL_RATIO = 1
LOGO_SEL_THRESHOLD_DEVICE = 2
LOGO_ENTRY_SELECT = 0
LOGO_ENTRY_LOCAL = 1
LOGO_ENTRY_GLOBAL = 2
LOGO_ENTRY_COMBINE = 3
LOGO_ENTRY_FWD = 4
LOGO_ENTRY_DENSE = 5
LOGO_ENTRY_DECODE = 6
LOGO_ENTRY_FWD_TRAIN = 7
LOGO_ENTRY_BWD = 8
LOGO_ENTRY_DENSE_BWD = 9
LOGO_ENTRY_GLOBAL_BWD = 10
LOGO_ENTRY_FWD_QPHI = 11
LOGO_PHI_LP = 0
LOGO_PHI_SO = 1

#: every symbol include/logo.h declares
EXPORTS = (
    "logo_select", "logo_local_attn", "logo_global_attn_sparse_q", "logo_combine",
    "logo_attn_fwd", "logo_attn_fwd_profiled", "logo_dense_causal_attn", "logo_workspace_bytes",
    "logo_ratio_capacity", "logo_status_str", "logo_version", "logo_budget_update",
    "logo_pmask_initial_threshold", "logo_decode", "logo_gate_proj", "logo_branch_transform",
    "logo_attn_fwd_train", "logo_attn_bwd", "logo_dense_causal_attn_fwd_train",
    "logo_dense_causal_attn_bwd", "logo_global_attn_sparse_q_fwd_train",
    "logo_global_attn_sparse_q_bwd", "logo_decode_noalloc", "logo_attn_fwd_qphi",
    "logo_attn_fwd_launches",
)

_lib = None


class LogoError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {logo_status_str(status)} ({status})")
        self.status = status


class _Problem(ctypes.Structure):
    _fields_ = [
        ("num_seqs", ctypes.c_int32),
        ("total_tokens", ctypes.c_int32),
        ("max_seqlen", ctypes.c_int32),
        ("cu_seqlens", ctypes.c_void_p),
        ("cu_seqlens_host", ctypes.c_void_p),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("window", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
    ]


def library_path() -> str:
    return _LIB_PATH


def library():
    """Load liblogo.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(
            f"{_LIB_PATH} is missing: build it with "
            "`python -m paper_2608_29539_amd.build` (hipcc, gfx950)")
    lib = ctypes.CDLL(_LIB_PATH)
    P, i32, i64, f32, f64, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                 ctypes.c_float, ctypes.c_double, ctypes.c_size_t)
    PP = ctypes.POINTER(_Problem)
    sigs = {
        "logo_select": [PP, P, i32, f32, f64, P, i32, P, P, P, P, sz, P],
        "logo_local_attn": [PP, P, P, P, P, P],
        "logo_global_attn_sparse_q": [PP, P, P, P, P, P, i32, P, P, sz, P],
        "logo_combine": [PP, P, P, P, P, P, P, f32, ctypes.c_int, P, P],
        "logo_attn_fwd_qphi": [PP, P, P, P, i32, P, P, P, P, P, P, i32, f32, f64, P, P, f32, P,
                               P, i32, P, P, P, P, sz, P],
        "logo_attn_fwd": [PP, P, P, P, P, P, P, P, i32, f32, f64, P, P, f32, P, P, i32, P, P,
                          P, P, sz, P],
        "logo_attn_fwd_profiled": [PP, P, P, P, P, P, P, P, i32, f32, f64, P, P, f32, P, P, i32,
                                   P, P, P, P, sz, P, P],
        "logo_dense_causal_attn": [PP, P, P, P, P, P],
        "logo_budget_update": [PP, P, f64, f32, P, P, P],
        "logo_decode": [PP, P, P, P, P, P, P, P, i32, f32, P, P, P, f32, P, P, P, P, sz, P],
        "logo_decode_noalloc": [PP, P, P, P, P, P, P, P, i32, f32, P, P, P, f32, P, P, P, P],
        "logo_gate_proj": [i64, i32, P, P, P, P],
        "logo_branch_transform": [i64, i32, i32, ctypes.c_int, P, P, P, P, P, i64, P, P, P],
        "logo_attn_fwd_train": [PP, P, P, P, P, P, P, P, i32, f32, f64, P, P, f32, P, P, i32, P,
                                P, P, P, P, P, P, P, sz, P],
        "logo_dense_causal_attn_fwd_train": [PP, P, P, P, P, P, P],
        "logo_global_attn_sparse_q_fwd_train": [PP, P, P, P, P, P, i32, P, P, P, sz, P],
        "logo_global_attn_sparse_q_bwd": [PP, P, P, P, P, P, i32, P, P, P, P, P, P, P, sz, P],
        "logo_dense_causal_attn_bwd": [PP, P, P, P, P, P, P, P, P, P, P, sz, P],
        "logo_attn_bwd": [PP, P, P, P, P, P, P, P, P, P, f32, P, i32, P, P, P, P, P, P, P, P, P,
                          P, P, P, P, P, P, P, P, sz, P],
    }
    for name, args in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.logo_workspace_bytes.argtypes = [PP, ctypes.c_int, i32]
    lib.logo_workspace_bytes.restype = sz
    lib.logo_ratio_capacity.argtypes = [PP, f64]
    lib.logo_ratio_capacity.restype = i64
    lib.logo_attn_fwd_launches.argtypes = [PP]
    lib.logo_attn_fwd_launches.restype = ctypes.c_int
    lib.logo_status_str.argtypes = [ctypes.c_int]
    lib.logo_status_str.restype = ctypes.c_char_p
    lib.logo_version.restype = ctypes.c_char_p
    lib.logo_pmask_initial_threshold.argtypes = [f32, i64]
    lib.logo_pmask_initial_threshold.restype = f32
    _lib = lib
    return lib


def exported_symbols() -> dict:
    """Which declared symbols the built library exports (name -> bool)."""
    lib = library()
    return {name: hasattr(lib, name) for name in EXPORTS}


def logo_status_str(status: int) -> str:
    return library().logo_status_str(int(status)).decode()


def logo_version() -> str:
    return library().logo_version().decode()


class Problem:
    """Host description of a packed varlen problem (mirrors ``logo_problem``).

    ``cu_seqlens`` is an int32 device tensor; ``cu_seqlens_host`` an optional
    host copy (a list or CPU tensor) used for validation and the ratio-mode
    selection bound.
    """

    def __init__(self, cu_seqlens, num_q_heads: int, num_kv_heads: int, head_dim: int,
                 window: int, *, total_tokens: Optional[int] = None,
                 max_seqlen: Optional[int] = None, cu_seqlens_host: Optional[Sequence[int]] = None,
                 softmax_scale: float = 0.0):
        import numpy as np
        self.cu_seqlens = cu_seqlens
        host = None
        if cu_seqlens_host is not None:
            host = np.ascontiguousarray(np.asarray(
                cu_seqlens_host.cpu() if hasattr(cu_seqlens_host, "cpu") else cu_seqlens_host),
                dtype=np.int32)
        self._host = host
        B = int(cu_seqlens.numel()) - 1
        if total_tokens is None or max_seqlen is None:
            if host is None:
                raise ValueError("give total_tokens and max_seqlen, or cu_seqlens_host")
            total_tokens = int(host[-1]) if total_tokens is None else total_tokens
            max_seqlen = int(np.max(np.diff(host))) if max_seqlen is None and B > 0 else max_seqlen
        self.num_seqs = B
        self.total_tokens = int(total_tokens)
        self.max_seqlen = int(max_seqlen)
        self.num_q_heads, self.num_kv_heads, self.head_dim = num_q_heads, num_kv_heads, head_dim
        self.window = int(window)
        self.softmax_scale = float(softmax_scale)
        self._c = _Problem(B, self.total_tokens, self.max_seqlen,
                           ctypes.c_void_p(cu_seqlens.data_ptr()),
                           None if host is None else host.ctypes.data_as(ctypes.c_void_p),
                           num_q_heads, num_kv_heads, head_dim, self.window, self.softmax_scale)

    @property
    def c(self):
        return ctypes.byref(self._c)


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t) -> Optional[ctypes.c_void_p]:
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _check(t, dtype, shape, name):
    import torch
    if t is None:
        raise ValueError(f"{name} is required")
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    return t


def _ws(prob: Problem, entry: int, cap: int, ws):
    import torch
    need = library().logo_workspace_bytes(prob.c, entry, cap)
    if need == 0:
        return None, 0
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=prob.cu_seqlens.device)
    return ws, int(ws.numel())


def _call(name: str, *args):
    st = getattr(library(), name)(*args)
    if st != 0:
        raise LogoError(name, st)


def logo_workspace_bytes(prob: Problem, entry: int, sel_capacity: int = 0) -> int:
    return int(library().logo_workspace_bytes(prob.c, entry, sel_capacity))


def logo_ratio_capacity(prob: Problem, ratio: float) -> int:
    return int(library().logo_ratio_capacity(prob.c, ratio))


def logo_attn_fwd_launches(prob: Problem) -> int:
    return int(library().logo_attn_fwd_launches(prob.c))


def _sel_mode(ratio, threshold, threshold_device, B):
    """(mode, thr_out override) for exactly one of ratio / threshold /
    threshold_device (a device fp32 tensor of >= B elements holding b_th in
    element 0; it also receives the thresholds used)."""
    import torch
    if sum(x is not None for x in (ratio, threshold, threshold_device)) != 1:
        raise ValueError("give exactly one of ratio / threshold / threshold_device")
    if threshold_device is not None:
        if (threshold_device.dtype != torch.float32 or not threshold_device.is_cuda
                or threshold_device.numel() < B or not threshold_device.is_contiguous()):
            raise ValueError("threshold_device: contiguous device float32 tensor of >= B values")
        return LOGO_SEL_THRESHOLD_DEVICE, threshold_device
    return (LOGO_SEL_RATIO if ratio is not None else LOGO_SEL_THRESHOLD), None


def logo_select(prob: Problem, gate, *, ratio: Optional[float] = None,
                threshold: Optional[float] = None, threshold_device=None,
                sel_capacity: Optional[int] = None, sel_idx=None, cu_sel=None, tok2sel=None,
                thr_out=None, ws=None):
    """Hard routing + compaction.  Returns (sel_idx, cu_sel, tok2sel, thr_out)."""
    import torch
    N, B = prob.total_tokens, prob.num_seqs
    mode, thr_dev = _sel_mode(ratio, threshold, threshold_device, B)
    if thr_dev is not None:
        thr_out = thr_dev
    dev = prob.cu_seqlens.device
    _check(gate, torch.float32, (N,), "gate")
    if sel_capacity is None:
        sel_capacity = logo_ratio_capacity(prob, ratio) if ratio is not None else N
    if sel_idx is None:
        sel_idx = torch.empty(max(sel_capacity, 1), dtype=torch.int32, device=dev)
    if cu_sel is None:
        cu_sel = torch.empty(B + 1, dtype=torch.int32, device=dev)
    if tok2sel is None:
        tok2sel = torch.empty(max(N, 1), dtype=torch.int32, device=dev)
    if thr_out is None:
        thr_out = torch.empty(B, dtype=torch.float32, device=dev)
    ws, nbytes = _ws(prob, LOGO_ENTRY_SELECT, 0, ws)
    _call("logo_select", prob.c, _ptr(gate), mode,
          float(threshold if threshold is not None else 0.0),
          float(ratio if ratio is not None else 0.0), _ptr(sel_idx), int(sel_capacity),
          _ptr(cu_sel), _ptr(tok2sel), _ptr(thr_out), _ptr(ws), nbytes, _stream())
    return sel_idx, cu_sel, tok2sel, thr_out


def logo_local_attn(prob: Problem, q, k, v, o_local=None):
    """Local branch, raw fp32 output [N, Hq, d]."""
    import torch
    N, Hq, Hkv, d = prob.total_tokens, prob.num_q_heads, prob.num_kv_heads, prob.head_dim
    _check(q, torch.bfloat16, (N, Hq, d), "q")
    _check(k, torch.bfloat16, (N, Hkv, d), "k")
    _check(v, torch.bfloat16, (N, Hkv, d), "v")
    if o_local is None:
        o_local = torch.empty((N, Hq, d), dtype=torch.float32, device=q.device)
    _check(o_local, torch.float32, (N, Hq, d), "o_local")
    _call("logo_local_attn", prob.c, _ptr(q), _ptr(k), _ptr(v), _ptr(o_local), _stream())
    return o_local


def logo_global_attn_sparse_q(prob: Problem, q, k, v, sel_idx, cu_sel, sel_capacity: int,
                              o_global=None, ws=None):
    """Query-sparse global branch, compact fp32 output [sel_capacity, Hq, d]."""
    import torch
    N, Hq, Hkv, d = prob.total_tokens, prob.num_q_heads, prob.num_kv_heads, prob.head_dim
    _check(q, torch.bfloat16, (N, Hq, d), "q")
    _check(k, torch.bfloat16, (N, Hkv, d), "k")
    _check(v, torch.bfloat16, (N, Hkv, d), "v")
    _check(cu_sel, torch.int32, (prob.num_seqs + 1,), "cu_sel")
    _check(sel_idx, torch.int32, None, "sel_idx")
    if sel_idx.numel() < sel_capacity:
        raise ValueError("sel_idx is smaller than sel_capacity")
    if o_global is None:
        o_global = torch.empty((max(sel_capacity, 1), Hq, d), dtype=torch.float32, device=q.device)
    _check(o_global, torch.float32, None, "o_global")
    if o_global.numel() < sel_capacity * Hq * d:
        raise ValueError("o_global is smaller than sel_capacity rows")
    ws, nbytes = _ws(prob, LOGO_ENTRY_GLOBAL, max(sel_capacity, 1), ws)
    _call("logo_global_attn_sparse_q", prob.c, _ptr(q), _ptr(k), _ptr(v), _ptr(sel_idx),
          _ptr(cu_sel), int(sel_capacity), _ptr(o_global), _ptr(ws), nbytes, _stream())
    return o_global


def logo_combine(prob: Problem, o_local, o_global, gate, tok2sel, *, gain_local=None,
                 gain_global=None, eps: float = 1e-6, apply_norm: bool = True, out=None):
    """ContextNorm + fusion, bf16 output [N, Hq, d]."""
    import torch
    N, Hq, d = prob.total_tokens, prob.num_q_heads, prob.head_dim
    _check(o_local, torch.float32, (N, Hq, d), "o_local")
    _check(gate, torch.float32, (N,), "gate")
    _check(tok2sel, torch.int32, None, "tok2sel")
    if o_global is not None:
        _check(o_global, torch.float32, None, "o_global")
    for g, nm in ((gain_local, "gain_local"), (gain_global, "gain_global")):
        if g is not None:
            _check(g, torch.float32, (Hq, d), nm)
    if out is None:
        out = torch.empty((N, Hq, d), dtype=torch.bfloat16, device=o_local.device)
    _check(out, torch.bfloat16, (N, Hq, d), "out")
    _call("logo_combine", prob.c, _ptr(o_local), _ptr(o_global), _ptr(gate), _ptr(tok2sel),
          _ptr(gain_local), _ptr(gain_global), float(eps), 1 if apply_norm else 0, _ptr(out),
          _stream())
    return out


def logo_attn_fwd(prob: Problem, q, k, v, gate, *, ratio: Optional[float] = None,
                  threshold: Optional[float] = None, threshold_device=None, q_g=None, k_g=None,
                  v_g=None,
                  gain_local=None, gain_global=None, eps: float = 1e-6, out=None,
                  sel_capacity: Optional[int] = None, sel_idx=None, cu_sel=None, tok2sel=None,
                  thr_out=None, ws=None, events=None):
    """The whole layer.  Returns (out, sel_idx, cu_sel, tok2sel, thr_out).

    ``events``: optional sequence of five recorded-once ``torch.cuda.Event``
    objects; when given, ``logo_attn_fwd_profiled`` records them at the stage
    boundaries (see include/logo.h).
    """
    import torch
    N, Hq, Hkv, d, B = (prob.total_tokens, prob.num_q_heads, prob.num_kv_heads, prob.head_dim,
                        prob.num_seqs)
    mode, thr_dev = _sel_mode(ratio, threshold, threshold_device, B)
    if thr_dev is not None:
        thr_out = thr_dev
    dev = q.device
    _check(q, torch.bfloat16, (N, Hq, d), "q")
    _check(k, torch.bfloat16, (N, Hkv, d), "k")
    _check(v, torch.bfloat16, (N, Hkv, d), "v")
    for t, nm, shp in ((q_g, "q_g", (N, Hq, d)), (k_g, "k_g", (N, Hkv, d)),
                       (v_g, "v_g", (N, Hkv, d))):
        if t is not None:
            _check(t, torch.bfloat16, shp, nm)
    _check(gate, torch.float32, (N,), "gate")
    if sel_capacity is None:
        sel_capacity = logo_ratio_capacity(prob, ratio) if ratio is not None else N
    if sel_idx is None:
        sel_idx = torch.empty(max(sel_capacity, 1), dtype=torch.int32, device=dev)
    if cu_sel is None:
        cu_sel = torch.empty(B + 1, dtype=torch.int32, device=dev)
    if tok2sel is None:
        tok2sel = torch.empty(max(N, 1), dtype=torch.int32, device=dev)
    if thr_out is None:
        thr_out = torch.empty(B, dtype=torch.float32, device=dev)
    if out is None:
        out = torch.empty((N, Hq, d), dtype=torch.bfloat16, device=dev)
    _check(out, torch.bfloat16, (N, Hq, d), "out")
    ws, nbytes = _ws(prob, LOGO_ENTRY_FWD, max(sel_capacity, 1), ws)
    args = [prob.c, _ptr(q), _ptr(k), _ptr(v), _ptr(q_g), _ptr(k_g), _ptr(v_g), _ptr(gate), mode,
            float(threshold if threshold is not None else 0.0),
            float(ratio if ratio is not None else 0.0), _ptr(gain_local), _ptr(gain_global),
            float(eps), _ptr(out), _ptr(sel_idx), int(max(sel_capacity, 1)), _ptr(cu_sel),
            _ptr(tok2sel), _ptr(thr_out), _ptr(ws), nbytes, _stream()]
    if events is None:
        _call("logo_attn_fwd", *args)
    else:
        if len(events) != 5:
            raise ValueError("events: five torch.cuda.Event objects")
        handles = (ctypes.c_void_p * 5)(*[ctypes.c_void_p(e.cuda_event) for e in events])
        _call("logo_attn_fwd_profiled", *args, handles)
    return out, sel_idx, cu_sel, tok2sel, thr_out


def logo_attn_fwd_qphi(prob: Problem, q, k, v, gate, q_phi: int, *, A=None, s=None, b=None,
                       ratio: Optional[float] = None, threshold: Optional[float] = None,
                       threshold_device=None, k_g=None, v_g=None, gain_local=None,
                       gain_global=None, eps: float = 1e-6, out=None,
                       sel_capacity: Optional[int] = None, sel_idx=None, cu_sel=None,
                       tok2sel=None, thr_out=None, ws=None):
    """The layer with the global branch's queries transformed inside the
    query-sparse kernel: ``q_phi`` LOGO_PHI_LP with ``A`` [Hq, d, d] bf16, or
    LOGO_PHI_SO with ``s``, ``b`` [Hq, d] float32.  Returns (out, sel_idx,
    cu_sel, tok2sel, thr_out)."""
    import torch
    N, Hq, Hkv, d, B = (prob.total_tokens, prob.num_q_heads, prob.num_kv_heads, prob.head_dim,
                        prob.num_seqs)
    mode, thr_dev = _sel_mode(ratio, threshold, threshold_device, B)
    if thr_dev is not None:
        thr_out = thr_dev
    dev = q.device
    _check(q, torch.bfloat16, (N, Hq, d), "q")
    _check(k, torch.bfloat16, (N, Hkv, d), "k")
    _check(v, torch.bfloat16, (N, Hkv, d), "v")
    for t, nm in ((k_g, "k_g"), (v_g, "v_g")):
        if t is not None:
            _check(t, torch.bfloat16, (N, Hkv, d), nm)
    if q_phi == LOGO_PHI_LP:
        _check(A, torch.bfloat16, (Hq, d, d), "A")
    elif q_phi == LOGO_PHI_SO:
        _check(s, torch.float32, (Hq, d), "s")
        _check(b, torch.float32, (Hq, d), "b")
    else:
        raise ValueError("q_phi: LOGO_PHI_LP or LOGO_PHI_SO")
    _check(gate, torch.float32, (N,), "gate")
    if sel_capacity is None:
        sel_capacity = logo_ratio_capacity(prob, ratio) if ratio is not None else N
    if sel_idx is None:
        sel_idx = torch.empty(max(sel_capacity, 1), dtype=torch.int32, device=dev)
    if cu_sel is None:
        cu_sel = torch.empty(B + 1, dtype=torch.int32, device=dev)
    if tok2sel is None:
        tok2sel = torch.empty(max(N, 1), dtype=torch.int32, device=dev)
    if thr_out is None:
        thr_out = torch.empty(B, dtype=torch.float32, device=dev)
    if out is None:
        out = torch.empty((N, Hq, d), dtype=torch.bfloat16, device=dev)
    _check(out, torch.bfloat16, (N, Hq, d), "out")
    ws, nbytes = _ws(prob, LOGO_ENTRY_FWD_QPHI, max(sel_capacity, 1), ws)
    _call("logo_attn_fwd_qphi", prob.c, _ptr(q), _ptr(k), _ptr(v), int(q_phi), _ptr(A), _ptr(s),
          _ptr(b), _ptr(k_g), _ptr(v_g), _ptr(gate), mode,
          float(threshold if threshold is not None else 0.0),
          float(ratio if ratio is not None else 0.0), _ptr(gain_local), _ptr(gain_global),
          float(eps), _ptr(out), _ptr(sel_idx), int(max(sel_capacity, 1)), _ptr(cu_sel),
          _ptr(tok2sel), _ptr(thr_out), _ptr(ws), nbytes, _stream())
    return out, sel_idx, cu_sel, tok2sel, thr_out


def logo_attn_fwd_train(prob: Problem, q, k, v, gate, *, ratio: Optional[float] = None,
                        threshold: Optional[float] = None, threshold_device=None, q_g=None,
                        k_g=None, v_g=None, gain_local=None, gain_global=None,
                        eps: float = 1e-6, sel_capacity: Optional[int] = None, ws=None) -> dict:
    """Training forward of the layer.  Returns a dict with ``out`` and the
    saved state the backward needs: sel_idx, cu_sel, tok2sel, thr_out,
    o_local, lse_local, o_global, lse_global, sel_capacity."""
    import torch
    N, Hq, Hkv, d, B = (prob.total_tokens, prob.num_q_heads, prob.num_kv_heads, prob.head_dim,
                        prob.num_seqs)
    mode, thr_dev = _sel_mode(ratio, threshold, threshold_device, B)
    dev = q.device
    _check(q, torch.bfloat16, (N, Hq, d), "q")
    _check(k, torch.bfloat16, (N, Hkv, d), "k")
    _check(v, torch.bfloat16, (N, Hkv, d), "v")
    for t, nm, shp in ((q_g, "q_g", (N, Hq, d)), (k_g, "k_g", (N, Hkv, d)),
                       (v_g, "v_g", (N, Hkv, d))):
        if t is not None:
            _check(t, torch.bfloat16, shp, nm)
    _check(gate, torch.float32, (N,), "gate")
    if sel_capacity is None:
        sel_capacity = logo_ratio_capacity(prob, ratio) if ratio is not None else N
    cap = max(int(sel_capacity), 1)
    f32 = dict(dtype=torch.float32, device=dev)
    st = dict(
        out=torch.empty((N, Hq, d), dtype=torch.bfloat16, device=dev),
        sel_idx=torch.empty(cap, dtype=torch.int32, device=dev),
        cu_sel=torch.empty(B + 1, dtype=torch.int32, device=dev),
        tok2sel=torch.empty(max(N, 1), dtype=torch.int32, device=dev),
        thr_out=thr_dev if thr_dev is not None else torch.empty(B, **f32),
        o_local=torch.empty((max(N, 1), Hq, d), **f32),
        lse_local=torch.empty((Hq, max(N, 1)), **f32),
        o_global=torch.empty((cap, Hq, d), **f32),
        lse_global=torch.empty((Hq, cap), **f32),
        sel_capacity=cap)
    ws, nbytes = _ws(prob, LOGO_ENTRY_FWD_TRAIN, cap, ws)
    _call("logo_attn_fwd_train", prob.c, _ptr(q), _ptr(k), _ptr(v), _ptr(q_g), _ptr(k_g),
          _ptr(v_g), _ptr(gate), mode, float(threshold if threshold is not None else 0.0),
          float(ratio if ratio is not None else 0.0), _ptr(gain_local), _ptr(gain_global),
          float(eps), _ptr(st["out"]), _ptr(st["sel_idx"]), cap, _ptr(st["cu_sel"]),
          _ptr(st["tok2sel"]), _ptr(st["thr_out"]), _ptr(st["o_local"]), _ptr(st["lse_local"]),
          _ptr(st["o_global"]), _ptr(st["lse_global"]), _ptr(ws), nbytes, _stream())
    return st


def logo_attn_bwd(prob: Problem, q, k, v, gate, saved: dict, dout, *, q_g=None, k_g=None,
                  v_g=None, gain_local=None, gain_global=None, eps: float = 1e-6,
                  dgain: bool = True, ws=None) -> dict:
    """Gradients of the layer given dout = dL/d out (bf16 [N, Hq, d]) and the
    ``saved`` dict of ``logo_attn_fwd_train``.  Returns fp32 dq, dk, dv (the
    global branch's share added in where its tensor is not given), dq_g /
    dk_g / dv_g for the given global tensors, dgate and (with ``dgain``)
    dgain_local / dgain_global."""
    import torch
    N, Hq, Hkv, d = prob.total_tokens, prob.num_q_heads, prob.num_kv_heads, prob.head_dim
    dev = q.device
    _check(dout, torch.bfloat16, (N, Hq, d), "dout")
    f32 = dict(dtype=torch.float32, device=dev)
    g = dict(dq=torch.empty((N, Hq, d), **f32), dk=torch.empty((N, Hkv, d), **f32),
             dv=torch.empty((N, Hkv, d), **f32), dgate=torch.empty(max(N, 1), **f32))
    for t, nm, shp in ((q_g, "dq_g", (N, Hq, d)), (k_g, "dk_g", (N, Hkv, d)),
                       (v_g, "dv_g", (N, Hkv, d))):
        g[nm] = torch.empty(shp, **f32) if t is not None else None
    if dgain:
        g["dgain_local"] = torch.empty((Hq, d), **f32)
        g["dgain_global"] = torch.empty((Hq, d), **f32)
    cap = int(saved["sel_capacity"])
    ws, nbytes = _ws(prob, LOGO_ENTRY_BWD, cap, ws)
    _call("logo_attn_bwd", prob.c, _ptr(q), _ptr(k), _ptr(v), _ptr(q_g), _ptr(k_g), _ptr(v_g),
          _ptr(gate), _ptr(gain_local), _ptr(gain_global), float(eps), _ptr(saved["sel_idx"]),
          cap, _ptr(saved["cu_sel"]), _ptr(saved["tok2sel"]), _ptr(saved["o_local"]),
          _ptr(saved["lse_local"]), _ptr(saved["o_global"]), _ptr(saved["lse_global"]),
          _ptr(dout), _ptr(g["dq"]), _ptr(g["dk"]), _ptr(g["dv"]), _ptr(g["dq_g"]),
          _ptr(g["dk_g"]), _ptr(g["dv_g"]), _ptr(g["dgate"]), _ptr(g.get("dgain_local")),
          _ptr(g.get("dgain_global")), _ptr(ws), nbytes, _stream())
    g["dgate"] = g["dgate"][:N]
    return {kk: vv for kk, vv in g.items() if vv is not None}


def logo_dense_causal_attn(prob: Problem, q, k, v, out=None):
    """Dense causal attention for every token (the baseline), bf16 [N, Hq, d]."""
    import torch
    N, Hq, Hkv, d = prob.total_tokens, prob.num_q_heads, prob.num_kv_heads, prob.head_dim
    _check(q, torch.bfloat16, (N, Hq, d), "q")
    _check(k, torch.bfloat16, (N, Hkv, d), "k")
    _check(v, torch.bfloat16, (N, Hkv, d), "v")
    if out is None:
        out = torch.empty((N, Hq, d), dtype=torch.bfloat16, device=q.device)
    _check(out, torch.bfloat16, (N, Hq, d), "out")
    _call("logo_dense_causal_attn", prob.c, _ptr(q), _ptr(k), _ptr(v), _ptr(out), _stream())
    return out


def logo_global_attn_sparse_q_fwd_train(prob: Problem, q, k, v, sel_idx, cu_sel,
                                        sel_capacity: int, o_global=None, lse_global=None,
                                        ws=None):
    """Query-sparse global attention keeping the base-2 LSE: (o_global fp32
    [cap, Hq, d], lse_global fp32 [Hq, cap]), compact in rank order."""
    import torch
    N, Hq, Hkv, d = prob.total_tokens, prob.num_q_heads, prob.num_kv_heads, prob.head_dim
    _check(q, torch.bfloat16, (N, Hq, d), "q")
    _check(k, torch.bfloat16, (N, Hkv, d), "k")
    _check(v, torch.bfloat16, (N, Hkv, d), "v")
    cap = int(sel_capacity)
    if o_global is None:
        o_global = torch.empty((max(cap, 1), Hq, d), dtype=torch.float32, device=q.device)
    if lse_global is None:
        lse_global = torch.empty((Hq, max(cap, 1)), dtype=torch.float32, device=q.device)
    ws, nbytes = _ws(prob, LOGO_ENTRY_GLOBAL, max(cap, 1), ws)
    _call("logo_global_attn_sparse_q_fwd_train", prob.c, _ptr(q), _ptr(k), _ptr(v),
          _ptr(sel_idx), _ptr(cu_sel), cap, _ptr(o_global), _ptr(lse_global), _ptr(ws), nbytes,
          _stream())
    return o_global, lse_global


def logo_global_attn_sparse_q_bwd(prob: Problem, q, k, v, sel_idx, cu_sel, sel_capacity: int,
                                  o_global, lse_global, dout, *, ws=None) -> dict:
    """Gradients of the query-sparse global attention alone given dout =
    dL/d o_global (bf16 [cap, Hq, d], compact): fp32 dq (zero rows for
    unselected tokens), dk, dv."""
    import torch
    N, Hq, Hkv, d = prob.total_tokens, prob.num_q_heads, prob.num_kv_heads, prob.head_dim
    cap = int(sel_capacity)
    _check(dout, torch.bfloat16, (max(cap, 1), Hq, d), "dout")
    f32 = dict(dtype=torch.float32, device=q.device)
    g = dict(dq=torch.empty((N, Hq, d), **f32), dk=torch.empty((N, Hkv, d), **f32),
             dv=torch.empty((N, Hkv, d), **f32))
    ws, nbytes = _ws(prob, LOGO_ENTRY_GLOBAL_BWD, max(cap, 1), ws)
    _call("logo_global_attn_sparse_q_bwd", prob.c, _ptr(q), _ptr(k), _ptr(v), _ptr(sel_idx),
          _ptr(cu_sel), cap, _ptr(o_global), _ptr(lse_global), _ptr(dout), _ptr(g["dq"]),
          _ptr(g["dk"]), _ptr(g["dv"]), _ptr(ws), nbytes, _stream())
    return g


def logo_dense_causal_attn_fwd_train(prob: Problem, q, k, v, out=None, lse=None):
    """Dense causal attention keeping the base-2 LSE: (out bf16 [N, Hq, d],
    lse fp32 [Hq, N])."""
    import torch
    N, Hq, Hkv, d = prob.total_tokens, prob.num_q_heads, prob.num_kv_heads, prob.head_dim
    _check(q, torch.bfloat16, (N, Hq, d), "q")
    _check(k, torch.bfloat16, (N, Hkv, d), "k")
    _check(v, torch.bfloat16, (N, Hkv, d), "v")
    if out is None:
        out = torch.empty((N, Hq, d), dtype=torch.bfloat16, device=q.device)
    if lse is None:
        lse = torch.empty((Hq, max(N, 1)), dtype=torch.float32, device=q.device)
    _check(out, torch.bfloat16, (N, Hq, d), "out")
    _call("logo_dense_causal_attn_fwd_train", prob.c, _ptr(q), _ptr(k), _ptr(v), _ptr(out),
          _ptr(lse), _stream())
    return out, lse


def logo_dense_causal_attn_bwd(prob: Problem, q, k, v, out, lse, dout, *, ws=None) -> dict:
    """Gradients of dense causal attention: fp32 dq, dk, dv."""
    import torch
    N, Hq, Hkv, d = prob.total_tokens, prob.num_q_heads, prob.num_kv_heads, prob.head_dim
    _check(dout, torch.bfloat16, (N, Hq, d), "dout")
    _check(out, torch.bfloat16, (N, Hq, d), "out")
    f32 = dict(dtype=torch.float32, device=q.device)
    g = dict(dq=torch.empty((N, Hq, d), **f32), dk=torch.empty((N, Hkv, d), **f32),
             dv=torch.empty((N, Hkv, d), **f32))
    ws, nbytes = _ws(prob, LOGO_ENTRY_DENSE_BWD, 0, ws)
    _call("logo_dense_causal_attn_bwd", prob.c, _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse),
          _ptr(dout), _ptr(g["dq"]), _ptr(g["dk"]), _ptr(g["dv"]), _ptr(ws), nbytes, _stream())
    return g


def logo_budget_update(prob: Problem, cu_sel, rho: float, gamma: float, b_th, realized=None):
    """One controller step b_th <- b_th + gamma sign(F - rho), F = cu_sel[B] / N,
    on the device (b_th: device fp32 tensor, element 0 updated in place)."""
    import torch
    _check(cu_sel, torch.int32, (prob.num_seqs + 1,), "cu_sel")
    if b_th.dtype != torch.float32 or not b_th.is_cuda or b_th.numel() < 1:
        raise ValueError("b_th: device float32 tensor")
    if realized is not None and (realized.dtype != torch.float32 or not realized.is_cuda):
        raise ValueError("realized: device float32 tensor")
    _call("logo_budget_update", prob.c, _ptr(cu_sel), float(rho), float(gamma), _ptr(b_th),
          _ptr(realized), _stream())
    return b_th


def logo_pmask_initial_threshold(gamma: float, pmask_steps: int) -> float:
    """Starting threshold of the P-mask schedule (host value)."""
    return float(library().logo_pmask_initial_threshold(float(gamma), int(pmask_steps)))


def logo_decode(prob: Problem, q, k, v, gate, *, threshold: Optional[float] = None,
                threshold_device=None, q_g=None, k_g=None, v_g=None, gain_local=None,
                gain_global=None, eps: float = 1e-6, out=None, active=None, n_active=None,
                ws=None):
    """One decoding step: ``prob.cu_seqlens`` bounds the KV caches (each
    sequence's last cached row is its new token), ``q`` [B, Hq, d] the new
    tokens' queries, ``gate`` [B].  Exactly one of ``threshold`` (host value)
    and ``threshold_device`` (device fp32, element 0) gives b_th.  Returns
    (out, active, n_active)."""
    import torch
    N, Hq, Hkv, d, B = (prob.total_tokens, prob.num_q_heads, prob.num_kv_heads, prob.head_dim,
                        prob.num_seqs)
    if (threshold is None) == (threshold_device is None):
        raise ValueError("give exactly one of threshold / threshold_device")
    if threshold_device is not None:
        if (threshold_device.dtype != torch.float32 or not threshold_device.is_cuda
                or threshold_device.numel() < 1):
            raise ValueError("threshold_device: device float32 tensor")
        mode = LOGO_SEL_THRESHOLD_DEVICE
    else:
        mode = LOGO_SEL_THRESHOLD
    dev = q.device
    _check(q, torch.bfloat16, (B, Hq, d), "q")
    _check(k, torch.bfloat16, (N, Hkv, d), "k")
    _check(v, torch.bfloat16, (N, Hkv, d), "v")
    for t, nm, shp in ((q_g, "q_g", (B, Hq, d)), (k_g, "k_g", (N, Hkv, d)),
                       (v_g, "v_g", (N, Hkv, d))):
        if t is not None:
            _check(t, torch.bfloat16, shp, nm)
    _check(gate, torch.float32, (B,), "gate")
    if out is None:
        out = torch.empty((B, Hq, d), dtype=torch.bfloat16, device=dev)
    _check(out, torch.bfloat16, (B, Hq, d), "out")
    if active is None:
        active = torch.empty(B, dtype=torch.int32, device=dev)
    if n_active is None:
        n_active = torch.empty(1, dtype=torch.int32, device=dev)
    ws, nbytes = _ws(prob, LOGO_ENTRY_DECODE, 0, ws)
    _call("logo_decode", prob.c, _ptr(q), _ptr(k), _ptr(v), _ptr(q_g), _ptr(k_g), _ptr(v_g),
          _ptr(gate), mode, float(threshold if threshold is not None else 0.0),
          _ptr(threshold_device), _ptr(gain_local), _ptr(gain_global), float(eps), _ptr(out),
          _ptr(active), _ptr(n_active), _ptr(ws), nbytes, _stream())
    return out, active, n_active


def logo_decode_noalloc(prob: Problem, q, k, v, gate, out, *, threshold: Optional[float] = None,
                        threshold_device=None, q_g=None, k_g=None, v_g=None, gain_local=None,
                        gain_global=None, eps: float = 1e-6, active=None, n_active=None):
    """``logo_decode`` without a workspace: the library's fixed device scratch
    array holds the partial results (and the selected list and count when
    ``active`` / ``n_active`` are None).  ``out`` [B, Hq, d] bf16 must be
    given; nothing is allocated.  Returns (out, active, n_active), the last
    two None when not given."""
    import torch
    N, Hq, Hkv, d, B = (prob.total_tokens, prob.num_q_heads, prob.num_kv_heads, prob.head_dim,
                        prob.num_seqs)
    if (threshold is None) == (threshold_device is None):
        raise ValueError("give exactly one of threshold / threshold_device")
    if threshold_device is not None:
        if (threshold_device.dtype != torch.float32 or not threshold_device.is_cuda
                or threshold_device.numel() < 1):
            raise ValueError("threshold_device: device float32 tensor")
        mode = LOGO_SEL_THRESHOLD_DEVICE
    else:
        mode = LOGO_SEL_THRESHOLD
    _check(q, torch.bfloat16, (B, Hq, d), "q")
    _check(k, torch.bfloat16, (N, Hkv, d), "k")
    _check(v, torch.bfloat16, (N, Hkv, d), "v")
    for t, nm, shp in ((q_g, "q_g", (B, Hq, d)), (k_g, "k_g", (N, Hkv, d)),
                       (v_g, "v_g", (N, Hkv, d))):
        if t is not None:
            _check(t, torch.bfloat16, shp, nm)
    _check(gate, torch.float32, (B,), "gate")
    _check(out, torch.bfloat16, (B, Hq, d), "out")
    if active is not None:
        _check(active, torch.int32, (B,), "active")
    if n_active is not None:
        _check(n_active, torch.int32, (1,), "n_active")
    _call("logo_decode_noalloc", prob.c, _ptr(q), _ptr(k), _ptr(v), _ptr(q_g), _ptr(k_g),
          _ptr(v_g), _ptr(gate), mode, float(threshold if threshold is not None else 0.0),
          _ptr(threshold_device), _ptr(gain_local), _ptr(gain_global), float(eps), _ptr(out),
          _ptr(active), _ptr(n_active), _stream())
    return out, active, n_active


def logo_gate_proj(x, w_g, out=None):
    """p = sigmoid(x . w_g) per token (fp32): x [N, d_model] and w_g [d_model]
    bf16 device tensors, d_model a multiple of 8."""
    import torch
    if x.dim() != 2:
        raise ValueError("x: [N, d_model]")
    N, dm = x.shape
    _check(x, torch.bfloat16, (N, dm), "x")
    _check(w_g, torch.bfloat16, (dm,), "w_g")
    if out is None:
        out = torch.empty(N, dtype=torch.float32, device=x.device)
    _check(out, torch.float32, (N,), "out")
    _call("logo_gate_proj", int(N), int(dm), _ptr(x), _ptr(w_g), _ptr(out), _stream())
    return out


def logo_branch_transform(u, kind: int, *, A=None, s=None, b=None, rows=None, n_rows=None,
                          n_rows_dev=None, out=None):
    """Eq. branch-transform per head: LP (``A`` [H, d, d] bf16) or SO (``s``,
    ``b`` [H, d] fp32) of ``u`` [N, H, d] bf16 into ``out`` (same shape; only
    the rows listed in ``rows`` -- int32 token indices -- when given)."""
    import torch
    N, H, d = u.shape
    _check(u, torch.bfloat16, (N, H, d), "u")
    if kind == LOGO_PHI_LP:
        _check(A, torch.bfloat16, (H, d, d), "A")
    else:
        _check(s, torch.float32, (H, d), "s")
        _check(b, torch.float32, (H, d), "b")
    if rows is not None:
        _check(rows, torch.int32, None, "rows")
        n_rows = rows.numel() if n_rows is None else n_rows
    else:
        n_rows = N
    if n_rows_dev is not None:
        _check(n_rows_dev, torch.int32, None, "n_rows_dev")
    if out is None:
        out = torch.empty_like(u)
    _check(out, torch.bfloat16, (N, H, d), "out")
    _call("logo_branch_transform", int(N), int(H), int(d), int(kind), _ptr(u), _ptr(A), _ptr(s),
          _ptr(b), _ptr(rows), int(n_rows), _ptr(n_rows_dev), _ptr(out), _stream())
    return out
