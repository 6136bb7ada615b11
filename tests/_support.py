"""Helpers shared by the GPU tests: moving synthetic inputs to the device,
oracle evaluation on a subset of rows, and the error metrics used by the
parity bar.  Expected values always come from ``oracle`` (never from the HIP
path)."""
from __future__ import annotations

import numpy as np

import oracle
import synth


def bf16_to_torch(a: np.ndarray, device):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(torch.bfloat16)


def to_device(x: dict, device="cuda"):
    import torch
    out = {}
    for k, v in x.items():
        if v.dtype == np.uint16:
            out[k] = bf16_to_torch(v, device)
        else:
            out[k] = torch.from_numpy(np.ascontiguousarray(v)).to(device)
    return out


def torch_bf16_to_f64(t) -> np.ndarray:
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """fp64 -> nearest-even bf16 (via fp32), widened back: the output format's floor."""
    b = synth.bf16_bits_from_f32(np.asarray(x, np.float64).astype(np.float32))
    return synth.f32_from_bf16_bits(b).reshape(np.shape(x)).astype(np.float64)


def oracle_layer_rows(x: dict, window: int, rows: np.ndarray, **kw):
    """Oracle layer output for the token rows ``rows`` (see ``oracle.logo_rows``)."""
    return oracle.logo_rows(x, window, rows, **kw)


def err_stats(got: np.ndarray, ref: np.ndarray) -> dict:
    e = np.abs(np.asarray(got, np.float64) - np.asarray(ref, np.float64))
    floor = np.abs(bf16_round(ref) - ref)
    return dict(max_abs=float(e.max()) if e.size else 0.0,
                mean_abs=float(e.mean()) if e.size else 0.0,
                n_over=int((e > 2e-2).sum()),
                floor_max=float(floor.max()) if floor.size else 0.0,
                floor_mean=float(floor.mean()) if floor.size else 0.0)


def rel_rms_err(got: np.ndarray, ref: np.ndarray) -> dict:
    """Error of raw attention rows measured in units of each (row, head) RMS."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    rms = np.sqrt((ref ** 2).mean(axis=-1, keepdims=True))
    e = np.abs(got - ref) / rms
    return dict(max_rel=float(e.max()) if e.size else 0.0,
                mean_rel=float(e.mean()) if e.size else 0.0)


def sample_rows(cu: np.ndarray, tok2sel: np.ndarray, n_sel_rows: int, n_other: int,
                seed: int) -> np.ndarray:
    """A spread of token rows: selected and unselected, including each
    sequence's first and last tokens and the latest selected tokens (the
    longest global rows)."""
    rng = np.random.default_rng(seed)
    N = int(cu[-1])
    sel = np.nonzero(tok2sel >= 0)[0]
    uns = np.nonzero(tok2sel < 0)[0]
    picks = []
    if sel.size:
        picks.append(rng.choice(sel, size=min(n_sel_rows, sel.size), replace=False))
        picks.append(sel[-min(8, sel.size):])
    if uns.size:
        picks.append(rng.choice(uns, size=min(n_other, uns.size), replace=False))
    for b in range(cu.size - 1):
        if cu[b + 1] > cu[b]:
            picks.append(np.array([cu[b], cu[b + 1] - 1, min(cu[b] + 63, cu[b + 1] - 1)]))
    r = np.unique(np.concatenate(picks)) if picks else np.zeros(0, np.int64)
    return r[(r >= 0) & (r < N)].astype(np.int32)


def over_bar_elements(bits: np.ndarray, ref: np.ndarray, bar: float):
    """Elements of a bf16 output (raw bits, the shape of ``ref``) more than
    ``bar`` from the fp64 oracle, and how many of them are not a faithful
    rounding, i.e. neither of the two bf16 values that bracket the oracle
    value (bf16 is sign-magnitude: the fp32 value's top half truncates toward
    zero, and the next code up is the next magnitude)."""
    bits = np.asarray(bits, np.uint16).reshape(ref.shape)
    got = synth.f32_from_bf16_bits(bits.reshape(-1)).reshape(ref.shape).astype(np.float64)
    big = np.argwhere(np.abs(got - ref) > bar)
    unfaithful = 0
    for bi in big:
        lo = np.uint16(np.float32(ref[tuple(bi)]).view(np.uint32) >> 16)
        unfaithful += int(bits[tuple(bi)] not in (lo, np.uint16(lo + 1)))
    return big, unfaithful

