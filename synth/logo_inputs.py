"""Seeded synthetic workloads shaped like the paper's attention benchmarks.

The paper benchmarks its query-sparse operator at batch 1, 8 heads, head
dim 128 and 4k-64k tokens (Sec. 4.3, Fig. "efficiency").  The workloads below
keep those shapes and extend them with GQA, varlen packing and the target
global ratios the method is run at (Sec. 3.2, Eq. realized-ratio).  All data
is synthetic: Q/K/V are normal draws, the gate is a probability per token.

Recipe (identical on every machine):
  * ``numpy.random.SeedSequence(seed).spawn(4)`` gives four independent
    PCG64 streams, used for Q, K, V and the gate in that order.
  * Normals are drawn as float32 (``standard_normal(dtype=float32)``),
    optionally multiplied by a float32 scale, then rounded to bf16 by
    round-to-nearest-even on the raw bits.
  * Gate probabilities are float32.  A logit gate applies the logistic
    function in float64 and rounds once to float32, so both sides of a
    comparison receive the same probability bits.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence

import numpy as np


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest-even) and return the raw uint16 bits.

    For finite inputs ``u + 0x7FFF + lsb`` cannot overflow 32 bits (the largest
    finite magnitude is 0x7F7FFFFF); NaNs are mapped to the quiet NaN 0x7FC0.
    """
    x = np.ascontiguousarray(x, dtype=np.float32).reshape(-1)
    u = x.view(np.uint32)
    r = (u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) >> np.uint32(16)
    out = r.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = np.uint16(0x7FC0)
    return out


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    """Widen raw bf16 bits to float32 (exact)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def markov_burst_gate(rng: np.random.Generator, T: int, p_stay_on: float,
                      p_turn_on: float, pi_on: float) -> np.ndarray:
    """Bursty gate: a two-state Markov chain s_t decides each token's band.

    s_0 ~ Bernoulli(pi_on); P(s_{t+1}=0 | s_t=1) = 1 - p_stay_on and
    P(s_{t+1}=1 | s_t=0) = p_turn_on.  The probability is 0.5 + 0.5u for an
    "on" token and 0.5u otherwise, u ~ U(0,1) float32.
    """
    trans = rng.random(T)                  # float64 uniforms for the chain
    u = rng.random(T, dtype=np.float32)    # float32 uniforms for the value
    if T == 0:
        return np.zeros(0, dtype=np.float32)
    s = np.empty(T, dtype=np.bool_)
    state = bool(trans[0] < pi_on)
    for t in range(T):
        if t > 0:
            if state:
                state = bool(trans[t] < p_stay_on)
            else:
                state = bool(trans[t] < p_turn_on)
        s[t] = state
    half = np.float32(0.5)
    return np.where(s, half + half * u, half * u).astype(np.float32)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    seqlens: Sequence[int]
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    window: int
    ratio: float
    seed: int
    qkv_scale: Optional[float] = None   # multiply the N(0,1) draws (float32) before bf16
    gate: str = "uniform"               # "uniform" | "logit_normal" | "markov_burst"
    note: str = ""

    @property
    def total_tokens(self) -> int:
        return int(sum(self.seqlens))

    @property
    def max_seqlen(self) -> int:
        return int(max(self.seqlens)) if len(self.seqlens) else 0

    def with_ratio(self, ratio: float, seed: int) -> "Workload":
        return dataclasses.replace(self, ratio=ratio, seed=seed,
                                   name=f"{self.name}-r{ratio:g}")


def _ratio_sweep() -> List[Workload]:
    base = Workload("varlen-4seq", (4096, 12288, 16384, 32768), 16, 4, 128, 512,
                    0.0, 1005, note="packed varlen, ratio sweep")
    return [base.with_ratio(r, 1005 + i) for i, r in
            enumerate((0.0, 1.0 / 32, 1.0 / 8, 1.0 / 2, 1.0))]


#: Named workloads.  "T32k-gqa" is the headline configuration.
WORKLOADS: Dict[str, Workload] = {
    "T1k-tiny": Workload("T1k-tiny", (1024,), 4, 4, 64, 128, 0.25, 1001,
                         qkv_scale=1.0 / 8.0, note="N(0,1)/sqrt(d) inputs"),
    "T8k-b2": Workload("T8k-b2", (8192, 8192), 16, 16, 128, 512, 1.0 / 8, 1002,
                       gate="logit_normal"),
    "T32k-gqa": Workload("T32k-gqa", (32768,), 32, 8, 128, 1024, 1.0 / 8, 1003,
                         gate="markov_burst"),
    "T128k-gqa": Workload("T128k-gqa", (131072,), 32, 8, 128, 4096, 1.0 / 16, 1004),
}
for _w in _ratio_sweep():
    WORKLOADS[_w.name] = _w

#: Decoding workloads: `seqlens` are the KV-cache lengths (each sequence's
#: last cached row is its new token), `ratio` the expected selected fraction
#: of the new tokens (gates U(0,1), threshold 1 - ratio).
DECODE_WORKLOADS: Dict[str, Workload] = {
    "decode-B16-32k-gqa": Workload("decode-B16-32k-gqa", (32768,) * 16, 32, 8, 128, 1024,
                                   1.0 / 8, 2001, note="16 caches of 32K tokens"),
}


def _normal_bf16(rng: np.random.Generator, shape, scale: Optional[float],
                 chunk: int = 1 << 20) -> np.ndarray:
    """N(0, scale^2) draws rounded to bf16 bits.  Drawn in cache-sized chunks:
    the generator's state carries over between calls, so the bytes equal one
    draw of the whole array, without its multi-GB float32 temporaries."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16)
    for s in range(0, n, chunk):
        x = rng.standard_normal(size=min(chunk, n - s), dtype=np.float32)
        if scale is not None:
            x *= np.float32(scale)
        out[s:s + x.size] = bf16_bits_from_f32(x)
    return out.reshape(shape)


def make_gate(rng: np.random.Generator, seqlens: Sequence[int], kind: str) -> np.ndarray:
    parts = []
    for T in seqlens:
        if kind == "uniform":
            parts.append(rng.random(T, dtype=np.float32))
        elif kind == "logit_normal":
            z = rng.standard_normal(T, dtype=np.float32).astype(np.float64)
            parts.append((1.0 / (1.0 + np.exp(-z))).astype(np.float32))
        elif kind == "markov_burst":
            # mean "on" run 8, mean "off" run 56 -> stationary on-fraction 1/8
            parts.append(markov_burst_gate(rng, T, p_stay_on=1.0 - 1.0 / 8,
                                           p_turn_on=1.0 / 56, pi_on=1.0 / 8))
        else:
            raise ValueError(f"unknown gate kind {kind!r}")
    if not parts:
        return np.zeros(0, dtype=np.float32)
    return np.concatenate(parts).astype(np.float32)


def make_inputs(w: Workload, *, distinct_global: bool = False) -> Dict[str, np.ndarray]:
    """Draw the inputs of one workload.

    Returns a dict with ``q`` [N,Hq,d], ``k``/``v`` [N,Hkv,d] (uint16 bf16
    bits), ``gate`` [N] float32 and ``cu_seqlens`` [B+1] int32.  With
    ``distinct_global`` it also returns separate global-branch tensors
    ``q_g``/``k_g``/``v_g`` drawn after the others from the same streams.
    """
    ss = np.random.SeedSequence(w.seed).spawn(4)
    rq, rk, rv, rg = (np.random.Generator(np.random.PCG64(s)) for s in ss)
    N = w.total_tokens
    q = _normal_bf16(rq, (N, w.num_q_heads, w.head_dim), w.qkv_scale)
    k = _normal_bf16(rk, (N, w.num_kv_heads, w.head_dim), w.qkv_scale)
    v = _normal_bf16(rv, (N, w.num_kv_heads, w.head_dim), w.qkv_scale)
    gate = make_gate(rg, w.seqlens, w.gate)
    cu = np.zeros(len(w.seqlens) + 1, dtype=np.int32)
    cu[1:] = np.cumsum(np.asarray(w.seqlens, dtype=np.int64)).astype(np.int32)
    out = dict(q=q, k=k, v=v, gate=gate, cu_seqlens=cu)
    if distinct_global:
        out["q_g"] = _normal_bf16(rq, q.shape, w.qkv_scale)
        out["k_g"] = _normal_bf16(rk, k.shape, w.qkv_scale)
        out["v_g"] = _normal_bf16(rv, v.shape, w.qkv_scale)
    return out


def make_dout(w: Workload, seed: int) -> np.ndarray:
    """Upstream gradient dL/d out for a backward pass: bf16 bits [N, Hq, d]
    of N(0,1) draws from its own seeded stream."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([w.seed, seed])))
    return _normal_bf16(rng, (w.total_tokens, w.num_q_heads, w.head_dim), None)


def make_gate_only(w: Workload) -> Dict[str, np.ndarray]:
    """The gate and cu_seqlens of a workload, without drawing Q/K/V.

    The gate uses its own spawned stream, so these are the same bytes as the
    ``gate`` returned by ``make_inputs``.
    """
    ss = np.random.SeedSequence(w.seed).spawn(4)
    rg = np.random.Generator(np.random.PCG64(ss[3]))
    cu = np.zeros(len(w.seqlens) + 1, dtype=np.int32)
    cu[1:] = np.cumsum(np.asarray(w.seqlens, dtype=np.int64)).astype(np.int32)
    return dict(gate=make_gate(rg, w.seqlens, w.gate), cu_seqlens=cu)


def small_workload(seqlens: Sequence[int], hq: int, hkv: int, d: int, window: int,
                   ratio: float, seed: int, gate: str = "uniform",
                   qkv_scale: Optional[float] = None) -> Workload:
    """An ad-hoc workload for tests (ragged lengths, edge cases)."""
    return Workload(f"adhoc-{seed}", tuple(int(t) for t in seqlens), hq, hkv, d,
                    window, ratio, seed, qkv_scale=qkv_scale, gate=gate)


def expected_selected(seqlens: Sequence[int], ratio: float) -> int:
    """Number of tokens a ratio-mode selection keeps when gate values are distinct."""
    return int(sum(min(T, math.floor(ratio * T)) for T in seqlens))


def make_decode_inputs(w: Workload, *, distinct_global: bool = False) -> Dict[str, np.ndarray]:
    """Inputs of one decoding step: the caches ``k``/``v`` [N,Hkv,d] (N = sum
    of the cache lengths), the new tokens' queries ``q`` [B,Hq,d] and gates
    ``gate`` [B] (float32), and ``cu_seqlens`` [B+1] of the caches.  Same
    seeded streams as ``make_inputs``; with ``distinct_global`` also
    ``q_g``/``k_g``/``v_g``."""
    ss = np.random.SeedSequence(w.seed).spawn(4)
    rq, rk, rv, rg = (np.random.Generator(np.random.PCG64(s)) for s in ss)
    N, B = w.total_tokens, len(w.seqlens)
    k = _normal_bf16(rk, (N, w.num_kv_heads, w.head_dim), w.qkv_scale)
    v = _normal_bf16(rv, (N, w.num_kv_heads, w.head_dim), w.qkv_scale)
    q = _normal_bf16(rq, (B, w.num_q_heads, w.head_dim), w.qkv_scale)
    gate = make_gate(rg, (B,), w.gate)
    cu = np.zeros(B + 1, dtype=np.int32)
    cu[1:] = np.cumsum(np.asarray(w.seqlens, dtype=np.int64)).astype(np.int32)
    out = dict(q=q, k=k, v=v, gate=gate, cu_seqlens=cu)
    if distinct_global:
        out["q_g"] = _normal_bf16(rq, q.shape, w.qkv_scale)
        out["k_g"] = _normal_bf16(rk, k.shape, w.qkv_scale)
        out["v_g"] = _normal_bf16(rv, v.shape, w.qkv_scale)
    return out
