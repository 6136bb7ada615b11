"""ctypes marshalling for the C oracle (``logo_oracle.c``).

Test infrastructure: see the package docstring.  Every function here converts
numpy arguments and calls one C function; none does arithmetic of its own.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, Optional

import numpy as np

SEL_THRESHOLD = 0
SEL_RATIO = 1

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "logo_oracle.c")
_LIB = os.path.join(_HERE, "liblogo_oracle.so")
_lib = None


def library_path() -> str:
    return _LIB


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, IEEE semantics, no FMA contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
               "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra",
               "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    override = os.environ.get("LOGO_ORACLE_LIB")  # mutation tests load a planted variant
    if override:
        lib = ctypes.CDLL(override)
    else:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    i32, i64, f32, f64 = ctypes.c_int, ctypes.c_int64, ctypes.c_float, ctypes.c_double
    lib.oracle_num_threads.restype = i32
    lib.oracle_set_num_threads.argtypes = [i32]
    lib.oracle_thresholds.argtypes = [P, P, i32, i32, f32, f64, P]
    lib.oracle_select.argtypes = [P, P, i32, P, P, P, P]
    lib.oracle_select.restype = i64
    lib.oracle_attn_rows.argtypes = [P, P, P, i32, i32, i32, P, i32, P, i64, i32, f64, P]
    lib.oracle_contextnorm.argtypes = [P, i64, i32, i32, P, f64]
    lib.oracle_fuse.argtypes = [P, P, P, P, i64, i32, i32, P]
    lib.oracle_logo_fwd.argtypes = [P, P, P, P, P, P, P, P, i32, i32, i32, i32, i32, f64,
                                    i32, f32, f64, P, P, f64, i32, P, P, P, P, P, P, P]
    lib.oracle_logo_fwd.restype = i64
    lib.oracle_realized_ratio.argtypes = [i64, i64]
    lib.oracle_realized_ratio.restype = f64
    lib.oracle_budget_update.argtypes = [f32, i64, i64, f64, f32]
    lib.oracle_budget_update.restype = f32
    lib.oracle_pmask_initial_threshold.argtypes = [f32, i64]
    lib.oracle_pmask_initial_threshold.restype = f32
    lib.oracle_decode.argtypes = [P, P, P, P, P, P, P, P, i32, i32, i32, i32, i32, f64, f32,
                                  P, P, f64, P, P, P, P]
    lib.oracle_decode.restype = i64
    lib.oracle_gate_proj.argtypes = [P, P, i64, i32, P]
    lib.oracle_logo_bwd.argtypes = [P, P, P, P, P, P, P, P, i32, i32, i32, i32, i32, f64, i32,
                                    f32, f64, P, P, f64, P, P, P, P, P, P, P, P, P, P]
    lib.oracle_logo_bwd.restype = i64
    lib.oracle_logo_bwd_sample.argtypes = [P, P, P, P, P, P, P, P, i32, i32, i32, i32, i32, f64,
                                           P, P, P, f64, P, i64, P, i64, P, P, P, P, P, P, P,
                                           P]
    lib.oracle_logo_bwd_sample.restype = None
    lib.oracle_attn_bwd.argtypes = [P, P, P, P, i32, i32, i32, i32, i32, f64, P, P, P, P]
    lib.oracle_attn_bwd.restype = None
    lib.oracle_fusion_bwd.argtypes = [P, P, P, P, i64, i32, i32, P, P, f64, P, P, P, P, P, P, P,
                                      P]
    lib.oracle_branch_transform.argtypes = [P, i32, i32, i32, P, P, P, P, i64, P]
    _lib = lib
    return lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    _load().oracle_set_num_threads(int(n))


def thresholds(gate, cu_seqlens, mode: int, threshold: float = 0.0, ratio: float = 0.0):
    gate, cu = _c(gate, np.float32), _c(cu_seqlens, np.int32)
    B = cu.size - 1
    thr = np.empty(B, dtype=np.float32)
    _load().oracle_thresholds(_ptr(gate), _ptr(cu), B, mode, threshold, ratio, _ptr(thr))
    return thr


def select(gate, cu_seqlens, thr):
    gate, cu, thr = _c(gate, np.float32), _c(cu_seqlens, np.int32), _c(thr, np.float32)
    B = cu.size - 1
    N = int(cu[-1])
    sel = np.empty(max(N, 1), dtype=np.int32)
    cu_sel = np.empty(B + 1, dtype=np.int32)
    tok2sel = np.empty(max(N, 1), dtype=np.int32)
    n = _load().oracle_select(_ptr(gate), _ptr(cu), B, _ptr(thr), _ptr(sel), _ptr(cu_sel),
                              _ptr(tok2sel))
    return sel[:n].copy(), cu_sel, tok2sel[:N].copy()


def attn_rows(q, k, v, cu_seqlens, rows, window: int, scale: float = 0.0):
    """fp64 attention rows: [len(rows), Hq, d].  window <= 0 means global."""
    q, k, v = _c(q, np.uint16), _c(k, np.uint16), _c(v, np.uint16)
    cu, rows = _c(cu_seqlens, np.int32), _c(rows, np.int32)
    N, Hq, d = q.shape
    Hkv = k.shape[1]
    if scale <= 0:
        scale = 1.0 / np.sqrt(d)
    out = np.empty((rows.size, Hq, d), dtype=np.float64)
    _load().oracle_attn_rows(_ptr(q), _ptr(k), _ptr(v), Hq, Hkv, d, _ptr(cu), cu.size - 1,
                             _ptr(rows), rows.size, int(window), float(scale), _ptr(out))
    return out


def contextnorm(o, gain=None, eps: float = 1e-6):
    o = np.array(o, dtype=np.float64, copy=True, order="C")
    n, Hq, d = o.shape
    _load().oracle_contextnorm(_ptr(o), n, Hq, d, _ptr(_c(gain, np.float32)), eps)
    return o


def fuse(ol, og, gate, tok2sel):
    ol, og = _c(ol, np.float64), _c(og, np.float64)
    gate, tok2sel = _c(gate, np.float32), _c(tok2sel, np.int32)
    N, Hq, d = ol.shape
    if og.size == 0:
        og = np.zeros((1, Hq, d))
    out = np.empty_like(ol)
    _load().oracle_fuse(_ptr(ol), _ptr(og), _ptr(gate), _ptr(tok2sel), N, Hq, d, _ptr(out))
    return out


def realized_ratio(n_selected: int, n_valid: int) -> float:
    """F of Eq. realized-ratio (Sec. 3.1)."""
    return float(_load().oracle_realized_ratio(int(n_selected), int(n_valid)))


def budget_update(b_th: float, n_selected: int, n_valid: int, rho: float, gamma: float) -> float:
    """One step of Eq. threshold-update (Sec. 3.2); fp32 result."""
    return float(_load().oracle_budget_update(float(b_th), int(n_selected), int(n_valid),
                                              float(rho), float(gamma)))


def pmask_initial_threshold(gamma: float, pmask_steps: int) -> float:
    """Starting threshold of the P-mask schedule (Sec. 3.2); fp32 result."""
    return float(_load().oracle_pmask_initial_threshold(float(gamma), int(pmask_steps)))


def logo_fwd(q, k, v, gate, cu_seqlens, window: int, *, ratio: Optional[float] = None,
             threshold: Optional[float] = None, q_g=None, k_g=None, v_g=None,
             gain_local=None, gain_global=None, eps: float = 1e-6, apply_norm: bool = True,
             scale: float = 0.0) -> Dict[str, np.ndarray]:
    """The whole layer in fp64.  Exactly one of ``ratio``/``threshold`` is given."""
    if (ratio is None) == (threshold is None):
        raise ValueError("give exactly one of ratio / threshold")
    q, k, v = _c(q, np.uint16), _c(k, np.uint16), _c(v, np.uint16)
    q_g, k_g, v_g = _c(q_g, np.uint16), _c(k_g, np.uint16), _c(v_g, np.uint16)
    gate, cu = _c(gate, np.float32), _c(cu_seqlens, np.int32)
    N, Hq, d = q.shape
    Hkv = k.shape[1]
    B = cu.size - 1
    mode = SEL_RATIO if ratio is not None else SEL_THRESHOLD
    thr = np.empty(B, dtype=np.float32)
    sel = np.empty(max(N, 1), dtype=np.int32)
    cu_sel = np.empty(B + 1, dtype=np.int32)
    tok2sel = np.empty(max(N, 1), dtype=np.int32)
    ol = np.empty((max(N, 1), Hq, d), dtype=np.float64)
    og = np.empty((max(N, 1), Hq, d), dtype=np.float64)
    out = np.empty((max(N, 1), Hq, d), dtype=np.float64)
    n = _load().oracle_logo_fwd(
        _ptr(q), _ptr(k), _ptr(v), _ptr(q_g), _ptr(k_g), _ptr(v_g), _ptr(gate), _ptr(cu), B,
        Hq, Hkv, d, int(window), float(scale), mode,
        float(threshold if threshold is not None else 0.0),
        float(ratio if ratio is not None else 0.0),
        _ptr(_c(gain_local, np.float32)), _ptr(_c(gain_global, np.float32)), float(eps),
        1 if apply_norm else 0, _ptr(thr), _ptr(sel), _ptr(cu_sel), _ptr(tok2sel), _ptr(ol),
        _ptr(og), _ptr(out))
    return dict(thr=thr, sel_idx=sel[:n].copy(), cu_sel=cu_sel, tok2sel=tok2sel[:N].copy(),
                o_local=ol[:N], o_global=og[:n].copy(), out=out[:N], n_sel=int(n))


def logo_rows(x: Dict[str, np.ndarray], window: int, rows, *, ratio: Optional[float] = None,
              threshold: Optional[float] = None, gain_local=None, gain_global=None,
              eps: float = 1e-6) -> Dict[str, np.ndarray]:
    """The layer output for the packed token indices ``rows`` only.

    Thresholds and selection are computed over the whole sequences (as the
    layer does); attention, ContextNorm and fusion only for ``rows``.  ``x``
    holds q, k, v (and optionally q_g, k_g, v_g), gate and cu_seqlens.  The
    result equals ``logo_fwd(...)["out"][rows]``; this composition of the C
    functions only avoids computing the other rows.
    """
    if (ratio is None) == (threshold is None):
        raise ValueError("give exactly one of ratio / threshold")
    mode = SEL_RATIO if ratio is not None else SEL_THRESHOLD
    thr = thresholds(x["gate"], x["cu_seqlens"], mode,
                     threshold=threshold if threshold is not None else 0.0,
                     ratio=ratio if ratio is not None else 0.0)
    sel_idx, cu_sel, tok2sel = select(x["gate"], x["cu_seqlens"], thr)
    rows = np.asarray(rows, dtype=np.int32)
    qg, kg, vg = x.get("q_g", x["q"]), x.get("k_g", x["k"]), x.get("v_g", x["v"])
    ol = attn_rows(x["q"], x["k"], x["v"], x["cu_seqlens"], rows, window)
    selected_rows = rows[tok2sel[rows] >= 0]
    og = attn_rows(qg, kg, vg, x["cu_seqlens"], selected_rows, 0)
    sub_t2s = np.full(rows.size, -1, np.int32)
    sub_t2s[tok2sel[rows] >= 0] = np.arange(selected_rows.size, dtype=np.int32)
    nl = contextnorm(ol, gain_local, eps)
    ng = contextnorm(og, gain_global, eps) if og.size else og
    out = fuse(nl, ng, x["gate"][rows], sub_t2s)
    return dict(out=out, o_local=ol, o_global=og, selected_rows=selected_rows, thr=thr,
                sel_idx=sel_idx, cu_sel=cu_sel, tok2sel=tok2sel)


def decode(q_new, k, v, gate_new, cu_cache, window: int, threshold: float, *, q_g_new=None,
           k_g=None, v_g=None, gain_local=None, gain_global=None, eps: float = 1e-6,
           scale: float = 0.0) -> Dict[str, np.ndarray]:
    """One decoding step in fp64 (Sec. 3.3, Autoregressive Decoding): q_new is
    [B, Hq, d] (the new tokens), k/v the packed caches [cu_cache[B], Hkv, d]
    whose last row per sequence is the new token's own key/value."""
    q_new, k, v = _c(q_new, np.uint16), _c(k, np.uint16), _c(v, np.uint16)
    q_g_new, k_g, v_g = _c(q_g_new, np.uint16), _c(k_g, np.uint16), _c(v_g, np.uint16)
    gate_new, cu = _c(gate_new, np.float32), _c(cu_cache, np.int32)
    B, Hq, d = q_new.shape
    Hkv = k.shape[1]
    ol = np.empty((B, Hq, d), dtype=np.float64)
    og = np.empty((B, Hq, d), dtype=np.float64)
    out = np.empty((B, Hq, d), dtype=np.float64)
    z = np.empty(B, dtype=np.int32)
    n = _load().oracle_decode(
        _ptr(q_new), _ptr(q_g_new), _ptr(k), _ptr(v), _ptr(k_g), _ptr(v_g), _ptr(gate_new),
        _ptr(cu), B, Hq, Hkv, d, int(window), float(scale), float(threshold),
        _ptr(_c(gain_local, np.float32)), _ptr(_c(gain_global, np.float32)), float(eps),
        _ptr(ol), _ptr(og), _ptr(out), _ptr(z))
    return dict(out=out, o_local=ol, o_global=og, z=z.astype(bool), n_sel=int(n))


def gate_proj(x, w_g) -> np.ndarray:
    """p = sigmoid(x . w_g) per token (Eq. gate-routing), fp32: x [N, dm] and
    w_g [dm] are bf16 bits."""
    x, w_g = _c(x, np.uint16), _c(w_g, np.uint16)
    N, dm = x.shape
    p = np.empty(N, dtype=np.float32)
    _load().oracle_gate_proj(_ptr(x), _ptr(w_g), N, dm, _ptr(p))
    return p


LP, SO = 0, 1


def branch_transform(u, kind: int, *, A=None, s=None, b=None, rows=None) -> np.ndarray:
    """Eq. branch-transform for the rows ``rows`` (all when None): LP with
    A [H, d, d] (bf16 bits) or SO with s, b [H, d] (fp32); fp64 result
    [len(rows), H, d]."""
    u = _c(u, np.uint16)
    N, H, d = u.shape
    rows = _c(rows, np.int32)
    n = N if rows is None else rows.size
    out = np.empty((n, H, d), dtype=np.float64)
    _load().oracle_branch_transform(_ptr(u), H, d, int(kind), _ptr(_c(A, np.uint16)),
                                    _ptr(_c(s, np.float32)), _ptr(_c(b, np.float32)),
                                    _ptr(rows), n, _ptr(out))
    return out


def logo_bwd(q, k, v, gate, cu_seqlens, window: int, dout, *, ratio: Optional[float] = None,
             threshold: Optional[float] = None, q_g=None, k_g=None, v_g=None, gain_local=None,
             gain_global=None, eps: float = 1e-6, scale: float = 0.0) -> Dict[str, np.ndarray]:
    """Gradients of the layer (fp64) given dout = dL/d out [N, Hq, d], the
    selection held fixed.  With aliased global tensors (q_g etc. None) the
    returned dq / dk / dv include both branches; otherwise the global-branch
    gradients are dq_g / dk_g / dv_g."""
    if (ratio is None) == (threshold is None):
        raise ValueError("give exactly one of ratio / threshold")
    alias = q_g is None and k_g is None and v_g is None
    q, k, v = _c(q, np.uint16), _c(k, np.uint16), _c(v, np.uint16)
    q_g, k_g, v_g = _c(q_g, np.uint16), _c(k_g, np.uint16), _c(v_g, np.uint16)
    gate, cu = _c(gate, np.float32), _c(cu_seqlens, np.int32)
    dout = _c(dout, np.float64)
    N, Hq, d = q.shape
    Hkv = k.shape[1]
    B = cu.size - 1
    mode = SEL_RATIO if ratio is not None else SEL_THRESHOLD
    n1 = max(N, 1)
    dq, dq_g = np.empty((n1, Hq, d)), np.empty((n1, Hq, d))
    dk, dv, dk_g, dv_g = (np.empty((n1, Hkv, d)) for _ in range(4))
    dgate = np.empty(n1)
    dgl, dgg = np.empty((Hq, d)), np.empty((Hq, d))
    n = _load().oracle_logo_bwd(
        _ptr(q), _ptr(k), _ptr(v), _ptr(q_g), _ptr(k_g), _ptr(v_g), _ptr(gate), _ptr(cu), B,
        Hq, Hkv, d, int(window), float(scale), mode,
        float(threshold if threshold is not None else 0.0),
        float(ratio if ratio is not None else 0.0),
        _ptr(_c(gain_local, np.float32)), _ptr(_c(gain_global, np.float32)), float(eps),
        _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dq_g), _ptr(dk_g), _ptr(dv_g),
        _ptr(dgate), _ptr(dgl), _ptr(dgg))
    r = dict(dgate=dgate[:N], dgain_local=dgl, dgain_global=dgg, n_sel=int(n))
    if alias:
        r.update(dq=(dq + dq_g)[:N], dk=(dk + dk_g)[:N], dv=(dv + dv_g)[:N])
    else:
        r.update(dq=dq[:N], dk=dk[:N], dv=dv[:N], dq_g=dq_g[:N], dk_g=dk_g[:N], dv_g=dv_g[:N])
    return r


def fusion_bwd(o_local, o_global_by_token, gate, z, dout, *, gain_local=None, gain_global=None,
               eps: float = 1e-6) -> Dict[str, np.ndarray]:
    """Backward of ContextNorm + fusion only: raw branch outputs [N, Hq, d]
    (the global one indexed by token, used where z), gate [N], z [N] bool,
    dout [N, Hq, d] -> dol, dog, delta_l, delta_g, dgate, dgain_local/global."""
    ol, og = _c(o_local, np.float64), _c(o_global_by_token, np.float64)
    gate, zz = _c(gate, np.float32), _c(np.asarray(z).astype(np.int32), np.int32)
    dout = _c(dout, np.float64)
    N, Hq, d = ol.shape
    dol, dog = np.empty_like(ol), np.empty_like(ol)
    dl, dg = np.empty((N, Hq)), np.empty((N, Hq))
    dgate = np.empty(N)
    gl, gg = np.empty((Hq, d)), np.empty((Hq, d))
    _load().oracle_fusion_bwd(_ptr(ol), _ptr(og), _ptr(gate), _ptr(zz), N, Hq, d,
                              _ptr(_c(gain_local, np.float32)), _ptr(_c(gain_global, np.float32)),
                              float(eps), _ptr(dout), _ptr(dol), _ptr(dog), _ptr(dl), _ptr(dg),
                              _ptr(dgate), _ptr(gl), _ptr(gg))
    return dict(dol=dol, dog=dog, delta_l=dl, delta_g=dg, dgate=dgate, dgain_local=gl,
                dgain_global=gg)


def attn_bwd(q, k, v, cu_seqlens, window: int, dout, *, scale: float = 0.0
             ) -> Dict[str, np.ndarray]:
    """Gradients of plain causal attention (window <= 0: full causal) given
    dout = dL/do [N, Hq, d] -> dq [N, Hq, d], dk, dv [N, Hkv, d] (fp64)."""
    q, k, v = _c(q, np.uint16), _c(k, np.uint16), _c(v, np.uint16)
    cu = _c(cu_seqlens, np.int32)
    dout = _c(dout, np.float64)
    N, Hq, d = q.shape
    Hkv = k.shape[1]
    n1 = max(N, 1)
    dq, dk, dv = np.empty((n1, Hq, d)), np.empty((n1, Hkv, d)), np.empty((n1, Hkv, d))
    _load().oracle_attn_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(cu), cu.size - 1, Hq, Hkv, d,
                            int(window), float(scale), _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv))
    return dict(dq=dq[:N], dk=dk[:N], dv=dv[:N])


def logo_bwd_sample(x: Dict[str, np.ndarray], window: int, dout, qrows, keys, *,
                    ratio: Optional[float] = None, threshold: Optional[float] = None,
                    gain_local=None, gain_global=None, eps: float = 1e-6,
                    scale: float = 0.0) -> Dict[str, np.ndarray]:
    """The layer backward (fp64) at sampled places only: dq / dq_g / dgate of
    the query tokens ``qrows`` and dk / dv / dk_g / dv_g of the key tokens
    ``keys`` (selection over the whole sequences, as the layer does).  With
    aliased global tensors (no q_g / k_g / v_g in ``x``) dq, dk, dv include
    both branches.  The cost grows with the rows that see a sampled key:
    sample global-branch keys near the end of their sequence."""
    if (ratio is None) == (threshold is None):
        raise ValueError("give exactly one of ratio / threshold")
    mode = SEL_RATIO if ratio is not None else SEL_THRESHOLD
    thr = thresholds(x["gate"], x["cu_seqlens"], mode,
                     threshold=threshold if threshold is not None else 0.0,
                     ratio=ratio if ratio is not None else 0.0)
    _, _, tok2sel = select(x["gate"], x["cu_seqlens"], thr)
    alias = "q_g" not in x and "k_g" not in x and "v_g" not in x
    q, k, v = _c(x["q"], np.uint16), _c(x["k"], np.uint16), _c(x["v"], np.uint16)
    qg, kg, vg = (_c(x.get(n), np.uint16) for n in ("q_g", "k_g", "v_g"))
    gate, cu = _c(x["gate"], np.float32), _c(x["cu_seqlens"], np.int32)
    qrows, keys = _c(np.asarray(qrows), np.int32), _c(np.asarray(keys), np.int32)
    dout = _c(dout, np.float64)
    N, Hq, d = q.shape
    Hkv = k.shape[1]
    nq, nk = qrows.size, keys.size
    dq, dqg = np.empty((max(nq, 1), Hq, d)), np.empty((max(nq, 1), Hq, d))
    dgate = np.empty(max(nq, 1))
    dk, dv, dkg, dvg = (np.empty((max(nk, 1), Hkv, d)) for _ in range(4))
    _load().oracle_logo_bwd_sample(
        _ptr(q), _ptr(k), _ptr(v), _ptr(qg), _ptr(kg), _ptr(vg), _ptr(gate), _ptr(cu),
        cu.size - 1, Hq, Hkv, d, int(window), float(scale), _ptr(_c(tok2sel, np.int32)),
        _ptr(_c(gain_local, np.float32)), _ptr(_c(gain_global, np.float32)), float(eps),
        _ptr(dout), nq, _ptr(qrows), nk, _ptr(keys), _ptr(dq), _ptr(dqg), _ptr(dgate), _ptr(dk),
        _ptr(dv), _ptr(dkg), _ptr(dvg))
    r = dict(dgate=dgate[:nq], tok2sel=tok2sel)
    if alias:
        r.update(dq=(dq + dqg)[:nq], dk=(dk + dkg)[:nk], dv=(dv + dvg)[:nk])
    else:
        r.update(dq=dq[:nq], dk=dk[:nk], dv=dv[:nk], dq_g=dqg[:nq], dk_g=dkg[:nk],
                 dv_g=dvg[:nk])
    return r
