"""Pins for the fp64 oracle (CPU only).

The oracle is the definition the GPU path is checked against, so it is pinned
here to things other than itself: a hand-derived example (tests/golden),
closed forms, invariants the paper states, and an independent numpy brute
force on tiny inputs that builds the full score matrix with explicit masks.
Each test names the passage it follows.
"""
import json
import math
import os

import numpy as np
import pytest

import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def bf16(x):
    """Exact bf16 bits for values that are representable (asserted)."""
    x = np.asarray(x, dtype=np.float32)
    b = synth.bf16_bits_from_f32(x).reshape(x.shape)
    assert np.array_equal(synth.f32_from_bf16_bits(b).reshape(x.shape), x), "not bf16-exact"
    return b


def wide(b):
    return synth.f32_from_bf16_bits(b).reshape(b.shape).astype(np.float64)


# ---------------------------------------------------------------------------
# Independent brute force (numpy, full T x T score matrix, explicit masks).
# ---------------------------------------------------------------------------
def brute_layer(q, k, v, gate, seqlens, window, *, ratio=None, threshold=None,
                q_g=None, k_g=None, v_g=None, gain_l=None, gain_g=None, eps=1e-6,
                scale=None):
    qf, kf, vf = wide(q), wide(k), wide(v)
    qg = wide(q_g) if q_g is not None else qf
    kg = wide(k_g) if k_g is not None else kf
    vg = wide(v_g) if v_g is not None else vf
    N, Hq, d = qf.shape
    Hkv = kf.shape[1]
    G = Hq // Hkv
    sc = 1.0 / math.sqrt(d) if scale is None else scale
    heads = np.arange(Hq) // G
    ol = np.zeros((N, Hq, d))
    og_full = np.zeros((N, Hq, d))
    selected = np.zeros(N, dtype=bool)
    thr_list = []
    start = 0
    for T in seqlens:
        sl = slice(start, start + T)
        p = gate[sl]
        if ratio is not None:
            kk = math.floor(ratio * T)
            thr = -np.inf if kk >= T else np.sort(p)[T - kk - 1]
        else:
            thr = threshold
        thr_list.append(thr)
        if T == 0:
            continue
        selected[sl] = np.array([p[i] > np.float32(thr) for i in range(T)], dtype=bool)
        i = np.arange(T)[:, None]
        j = np.arange(T)[None, :]
        causal = j <= i
        local = causal & (j > i - window)
        for h in range(Hq):
            for (Q, K, V, mask, dst) in ((qf, kf, vf, local, ol), (qg, kg, vg, causal, og_full)):
                S = sc * (Q[sl, h, :] @ K[sl, heads[h], :].T)
                S = np.where(mask, S, -np.inf)
                W = np.exp(S - S.max(axis=1, keepdims=True))
                W = W / W.sum(axis=1, keepdims=True)
                dst[sl, h, :] = W @ V[sl, heads[h], :]
        start += T

    def rms(o, g):
        r = np.sqrt((o ** 2).mean(axis=-1, keepdims=True) + eps)
        return o / r * (1.0 if g is None else g.astype(np.float64)[None])

    nl, ng = rms(ol, gain_l), rms(og_full, gain_g)
    pw = gate.astype(np.float64)[:, None, None]
    out = np.where(selected[:, None, None], (1 - pw) * nl + pw * ng, nl)
    sel_idx = np.nonzero(selected)[0]
    return dict(o_local=ol, o_global=og_full[sel_idx], out=out, sel_idx=sel_idx,
                thr=np.array(thr_list, dtype=np.float32), selected=selected)


def test_hand_example_threshold(oracle_lib):
    """Hand-derived T=3 example (tests/golden/hand_t3_d4.json), threshold mode."""
    g = json.load(open(os.path.join(GOLDEN, "hand_t3_d4.json")))
    inp = g["inputs"]
    q = bf16(np.array(inp["q"], np.float32)[:, None, :])
    k = bf16(np.array(inp["k"], np.float32)[:, None, :])
    v = bf16(np.array(inp["v"], np.float32)[:, None, :])
    gate = np.array(inp["gate"], np.float32)
    cu = np.array([0, 3], np.int32)
    r = oracle_lib.logo_fwd(q, k, v, gate, cu, inp["window"], threshold=0.5, eps=inp["eps"])
    e = g["threshold_0.5"]
    assert r["sel_idx"].tolist() == e["sel_idx"]
    assert r["cu_sel"].tolist() == e["cu_sel"]
    assert r["tok2sel"].tolist() == e["tok2sel"]
    np.testing.assert_allclose(r["o_local"][:, 0, :], e["o_local"], rtol=0, atol=1e-14)
    np.testing.assert_allclose(r["o_global"][:, 0, :], e["o_global"], rtol=0, atol=1e-14)
    np.testing.assert_allclose(r["out"][:, 0, :], e["out"], rtol=0, atol=1e-14)


def test_hand_example_ratio(oracle_lib):
    """Same example in ratio mode: strict '>' leaves the tie at the threshold out."""
    g = json.load(open(os.path.join(GOLDEN, "hand_t3_d4.json")))
    inp = g["inputs"]
    q = bf16(np.array(inp["q"], np.float32)[:, None, :])
    k = bf16(np.array(inp["k"], np.float32)[:, None, :])
    v = bf16(np.array(inp["v"], np.float32)[:, None, :])
    gate = np.array(inp["gate"], np.float32)
    cu = np.array([0, 3], np.int32)
    r = oracle_lib.logo_fwd(q, k, v, gate, cu, inp["window"], ratio=0.5, eps=inp["eps"])
    e = g["ratio_0.5"]
    assert float(r["thr"][0]) == e["thr"]
    assert r["sel_idx"].tolist() == e["sel_idx"]
    assert r["cu_sel"].tolist() == e["cu_sel"]
    assert r["tok2sel"].tolist() == e["tok2sel"]
    np.testing.assert_allclose(r["out"][:, 0, :], e["out"], rtol=0, atol=1e-14)


def test_contextnorm_hand(oracle_lib):
    """Eq. contextnorm: (3,4) has rms sqrt(12.5), so it maps to (3,4)/sqrt(12.5)."""
    o = np.array([[[3.0, 4.0]]])
    r = oracle_lib.contextnorm(o, eps=0.0)
    np.testing.assert_allclose(r[0, 0], [0.848528137423857, 1.131370849898476], atol=1e-15)
    gain = np.array([[2.0, -0.5]], np.float32)
    r = oracle_lib.contextnorm(o, gain=gain, eps=0.0)
    np.testing.assert_allclose(r[0, 0], [1.697056274847714, -0.565685424949238], atol=1e-15)
    # eps is added to the mean square, not to the rms
    r = oracle_lib.contextnorm(np.array([[[1.0, 1.0]]]), eps=3.0)
    np.testing.assert_allclose(r[0, 0], [0.5, 0.5], atol=1e-15)


CASES = [
    # seqlens, Hq, Hkv, d, window, mode, value
    ((16,), 2, 2, 8, 4, "ratio", 0.25),
    ((5, 11), 4, 2, 8, 3, "ratio", 0.5),
    ((9, 0, 7), 4, 1, 16, 1, "threshold", 0.4),
    ((13,), 2, 1, 4, 16, "ratio", 1.0),
    ((12, 4), 2, 2, 8, 6, "threshold", 0.7),
    ((1, 15), 6, 3, 8, 2, "ratio", 0.34),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_bruteforce_tiny(oracle_lib, case):
    """Whole layer on T <= 16 against the numpy brute force (Sec. 3.1-3.2)."""
    seqlens, Hq, Hkv, d, w, mode, val = CASES[case]
    wl = synth.small_workload(seqlens, Hq, Hkv, d, w, val if mode == "ratio" else 0.0,
                              seed=700 + case)
    x = synth.make_inputs(wl, distinct_global=(case % 2 == 1))
    rng = np.random.default_rng(case)
    gain_l = rng.uniform(0.5, 1.5, (Hq, d)).astype(np.float32) if case % 3 == 0 else None
    gain_g = rng.uniform(0.5, 1.5, (Hq, d)).astype(np.float32) if case % 3 == 0 else None
    kw = dict(ratio=val) if mode == "ratio" else dict(threshold=val)
    extra = {}
    if case % 2 == 1:
        extra = dict(q_g=x["q_g"], k_g=x["k_g"], v_g=x["v_g"])
    r = oracle_lib.logo_fwd(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], w,
                            gain_local=gain_l, gain_global=gain_g, **kw, **extra)
    b = brute_layer(x["q"], x["k"], x["v"], x["gate"], seqlens, w, gain_l=gain_l,
                    gain_g=gain_g, **kw, **extra)
    assert r["sel_idx"].tolist() == b["sel_idx"].tolist()
    assert np.array_equal(r["thr"], b["thr"])
    exp_cu = np.concatenate([[0], np.cumsum([b["selected"][s:s + T].sum() for s, T in
                                             zip(np.cumsum((0,) + seqlens[:-1]), seqlens)])])
    assert r["cu_sel"].tolist() == exp_cu.tolist()
    exp_t2s = np.full(sum(seqlens), -1)
    exp_t2s[b["sel_idx"]] = np.arange(b["sel_idx"].size)
    assert r["tok2sel"].tolist() == exp_t2s.tolist()
    np.testing.assert_allclose(r["o_local"], b["o_local"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(r["o_global"], b["o_global"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(r["out"], b["out"], rtol=0, atol=1e-12)


def _rows(N):
    return np.arange(N, dtype=np.int32)


def test_window_one_is_value(oracle_lib):
    """w = 1: the local context is the token itself, so O^L_t = v_t (Sec. 3.1)."""
    wl = synth.small_workload((37, 20), 4, 2, 16, 1, 0.0, seed=11)
    x = synth.make_inputs(wl)
    o = oracle_lib.attn_rows(x["q"], x["k"], x["v"], x["cu_seqlens"], _rows(57), window=1)
    vv = np.repeat(wide(x["v"]), 2, axis=1)
    np.testing.assert_allclose(o, vv, rtol=0, atol=1e-15)


def test_zero_query_is_window_mean(oracle_lib):
    """q = 0: all scores are equal, so the output is the mean of the context values.

    Local: mean of v over the last min(t, w) tokens (exactly w keys with self).
    Global: mean over the whole prefix.
    """
    wl = synth.small_workload((50, 31), 2, 1, 8, 7, 0.0, seed=12)
    x = synth.make_inputs(wl)
    q = np.zeros_like(x["q"])
    vv = wide(x["v"])[:, 0, :]
    for window in (7, 0):
        o = oracle_lib.attn_rows(q, x["k"], x["v"], x["cu_seqlens"], _rows(81), window=window)
        for t in range(81):
            base = 0 if t < 50 else 50
            pos = t - base
            lo = base + (max(0, pos - window + 1) if window > 0 else 0)
            ref = vv[lo:t + 1].mean(axis=0)
            for h in range(2):
                np.testing.assert_allclose(o[t, h], ref, rtol=0, atol=1e-14)


def test_window_ge_T_is_dense(oracle_lib):
    """w >= T: the local context is the whole causal prefix (Sec. 3.1)."""
    wl = synth.small_workload((40,), 4, 2, 16, 40, 0.0, seed=13)
    x = synth.make_inputs(wl)
    for w in (40, 41, 1000):
        a = oracle_lib.attn_rows(x["q"], x["k"], x["v"], x["cu_seqlens"], _rows(40), window=w)
        g = oracle_lib.attn_rows(x["q"], x["k"], x["v"], x["cu_seqlens"], _rows(40), window=0)
        np.testing.assert_array_equal(a, g)
    a = oracle_lib.attn_rows(x["q"], x["k"], x["v"], x["cu_seqlens"], _rows(40), window=39)
    assert not np.array_equal(a[39:], g[39:])


def test_ratio_one_is_dense_and_ratio_zero_is_local(oracle_lib):
    """rho = 1 selects every token, so O^G is dense causal attention on all rows;
    rho = 0 selects none, so the output is Norm^L(O^L) (Sec. 3.2, Eq. output-fusion)."""
    wl = synth.small_workload((64, 33), 4, 2, 16, 8, 1.0, seed=14)
    x = synth.make_inputs(wl)
    r1 = oracle_lib.logo_fwd(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], 8, ratio=1.0)
    assert r1["n_sel"] == 97 and r1["sel_idx"].tolist() == list(range(97))
    assert np.all(np.isneginf(r1["thr"]))
    dense = oracle_lib.attn_rows(x["q"], x["k"], x["v"], x["cu_seqlens"], _rows(97), window=0)
    np.testing.assert_array_equal(r1["o_global"], dense)
    r0 = oracle_lib.logo_fwd(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], 8, ratio=0.0)
    assert r0["n_sel"] == 0 and np.all(r0["tok2sel"] == -1)
    np.testing.assert_array_equal(r0["out"], oracle_lib.contextnorm(r0["o_local"]))


def test_shift_invariance(oracle_lib):
    """Adding one vector c to every key of a head shifts each query's scores by
    q.c, which the softmax cancels (Eq. attention).  Values are chosen so the
    shifted keys stay bf16-exact."""
    rng = np.random.default_rng(5)
    N, H, d = 30, 2, 8
    q = bf16(rng.integers(-4, 5, (N, H, d)) / 4.0)
    k = bf16(rng.integers(-8, 9, (N, H, d)) / 8.0)
    v = synth.bf16_bits_from_f32(rng.standard_normal((N, H, d)).astype(np.float32))
    v = v.reshape(N, H, d)
    c = rng.integers(-8, 9, (1, H, d)) / 8.0
    k2 = bf16(wide(k) + c)
    cu = np.array([0, N], np.int32)
    for w in (5, 0):
        a = oracle_lib.attn_rows(q, k, v, cu, _rows(N), window=w)
        b = oracle_lib.attn_rows(q, k2, v, cu, _rows(N), window=w)
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_gqa_equals_repeated_mha(oracle_lib):
    """Query head h reads kv head floor(h/G): repeating each kv head G times
    (contiguous grouping) gives the MHA result."""
    wl = synth.small_workload((45,), 8, 2, 16, 9, 0.0, seed=15)
    x = synth.make_inputs(wl)
    krep = np.repeat(x["k"], 4, axis=1)
    vrep = np.repeat(x["v"], 4, axis=1)
    for w in (9, 0):
        a = oracle_lib.attn_rows(x["q"], x["k"], x["v"], x["cu_seqlens"], _rows(45), window=w)
        b = oracle_lib.attn_rows(x["q"], krep, vrep, x["cu_seqlens"], _rows(45), window=w)
        np.testing.assert_array_equal(a, b)


def test_head_permutation(oracle_lib):
    """Permuting heads (MHA) permutes the outputs of both branches and the fusion."""
    wl = synth.small_workload((33,), 4, 4, 8, 5, 0.25, seed=16)
    x = synth.make_inputs(wl)
    perm = np.array([2, 0, 3, 1])
    a = oracle_lib.logo_fwd(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], 5, ratio=0.25)
    b = oracle_lib.logo_fwd(x["q"][:, perm], x["k"][:, perm], x["v"][:, perm], x["gate"],
                            x["cu_seqlens"], 5, ratio=0.25)
    np.testing.assert_array_equal(a["out"][:, perm], b["out"])


def test_varlen_is_separate_runs(oracle_lib):
    """Packed sequences do not see each other: packing = running each alone."""
    wl = synth.small_workload((19, 26, 7), 2, 1, 8, 6, 0.3, seed=17)
    x = synth.make_inputs(wl)
    r = oracle_lib.logo_fwd(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], 6, ratio=0.3)
    cu = x["cu_seqlens"]
    for b in range(3):
        s, e = cu[b], cu[b + 1]
        rb = oracle_lib.logo_fwd(x["q"][s:e], x["k"][s:e], x["v"][s:e], x["gate"][s:e],
                                 np.array([0, e - s], np.int32), 6, ratio=0.3)
        np.testing.assert_array_equal(r["out"][s:e], rb["out"])
        assert (r["sel_idx"][r["cu_sel"][b]:r["cu_sel"][b + 1]] - s).tolist() == \
            rb["sel_idx"].tolist()


def test_selection_order_statistic_and_ties(oracle_lib):
    """Ratio mode keeps the k = floor(rho T) largest gates when they are distinct;
    with ties at the threshold the strict '>' keeps fewer (Eq. gate-routing)."""
    rng = np.random.default_rng(3)
    for T, rho in ((100, 0.25), (64, 1 / 8), (7, 0.5), (10, 0.99), (1, 0.5), (2, 1.0)):
        g = rng.permutation(T).astype(np.float32) / T
        cu = np.array([0, T], np.int32)
        thr = oracle_lib.thresholds(g, cu, oracle_lib.SEL_RATIO, ratio=rho)
        sel, cu_sel, t2s = oracle_lib.select(g, cu, thr)
        kk = math.floor(rho * T)
        assert sel.size == kk
        assert sorted(sel.tolist()) == sorted(np.argsort(-g, kind="stable")[:kk].tolist())
        assert sel.tolist() == sorted(sel.tolist())
    g = np.array([0.1, 0.5, 0.5, 0.5, 0.9, 0.2], np.float32)
    cu = np.array([0, 6], np.int32)
    thr = oracle_lib.thresholds(g, cu, oracle_lib.SEL_RATIO, ratio=0.5)  # k = 3
    assert thr[0] == np.float32(0.5)
    sel, _, _ = oracle_lib.select(g, cu, thr)
    assert sel.tolist() == [4]
    # threshold mode: +inf selects nothing, -inf selects every finite gate
    for t, n in ((np.inf, 0), (-np.inf, 6), (0.5, 1), (0.1, 5), (0.2, 4)):
        thr = oracle_lib.thresholds(g, cu, oracle_lib.SEL_THRESHOLD, threshold=t)
        sel, _, _ = oracle_lib.select(g, cu, thr)
        assert sel.size == n


def test_fusion_weights(oracle_lib):
    """Eq. output-fusion: a selected token with p = 1 takes Norm^G, one with p
    just above a threshold of 0 takes (1-p) Norm^L + p Norm^G; unselected
    tokens take Norm^L."""
    wl = synth.small_workload((24,), 2, 2, 8, 3, 0.0, seed=18)
    x = synth.make_inputs(wl)
    gate = np.where(np.arange(24) % 3 == 0, 1.0, 0.0).astype(np.float32)
    gate[5] = np.float32(0.125)
    r = oracle_lib.logo_fwd(x["q"], x["k"], x["v"], gate, x["cu_seqlens"], 3, threshold=0.0)
    nl = oracle_lib.contextnorm(r["o_local"])
    ng = oracle_lib.contextnorm(r["o_global"])
    for t in range(24):
        if t % 3 == 0:
            np.testing.assert_allclose(r["out"][t], ng[r["tok2sel"][t]], atol=1e-15)
        elif t == 5:
            np.testing.assert_allclose(
                r["out"][t], 0.875 * nl[t] + 0.125 * ng[r["tok2sel"][t]], atol=1e-15)
        else:
            assert r["tok2sel"][t] == -1
            np.testing.assert_array_equal(r["out"][t], nl[t])


def test_scale_argument(oracle_lib):
    """Doubling q (exact in bf16) equals doubling the softmax scale."""
    wl = synth.small_workload((20,), 2, 2, 8, 0, 0.0, seed=19)
    x = synth.make_inputs(wl)
    q2 = bf16(2.0 * wide(x["q"]))
    a = oracle_lib.attn_rows(q2, x["k"], x["v"], x["cu_seqlens"], _rows(20), 0)
    b = oracle_lib.attn_rows(x["q"], x["k"], x["v"], x["cu_seqlens"], _rows(20), 0,
                             scale=2.0 / math.sqrt(8))
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-13)


def test_logo_rows_matches_whole_layer(oracle_lib):
    """The row-subset composition used for large workloads equals the whole
    layer on those rows."""
    wl = synth.small_workload((200, 57), 4, 2, 16, 9, 0.3, seed=20)
    x = synth.make_inputs(wl)
    full = oracle_lib.logo_fwd(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], 9, ratio=0.3)
    rows = np.array([0, 5, 17, 199, 200, 201, 256, 120], np.int32)
    sub = oracle_lib.logo_rows(x, 9, rows, ratio=0.3)
    np.testing.assert_allclose(sub["out"], full["out"][rows], rtol=0, atol=1e-15)


# ---------------------------------------------------------------------------
# budget controller (Sec. 3.2, Eq. threshold-update; Sec. 3.1, Eq.
# realized-ratio; P-mask paragraph).  Dyadic values keep every fp32 step exact.
# ---------------------------------------------------------------------------
def test_realized_ratio_hand(oracle_lib):
    assert oracle_lib.realized_ratio(3, 8) == 0.375
    assert oracle_lib.realized_ratio(0, 5) == 0.0
    assert oracle_lib.realized_ratio(7, 7) == 1.0


def test_budget_update_sign_cases(oracle_lib):
    # F = 3/8 > rho = 1/4: too many global tokens, the threshold rises
    assert oracle_lib.budget_update(0.25, 3, 8, 0.25, 0.125) == 0.375
    # F = 1/8 < rho: it falls
    assert oracle_lib.budget_update(0.25, 1, 8, 0.25, 0.125) == 0.125
    # F == rho exactly: sign(0) = 0, no change
    assert oracle_lib.budget_update(0.25, 2, 8, 0.25, 0.125) == 0.25
    # no valid token: no change
    assert oracle_lib.budget_update(0.25, 0, 0, 0.25, 0.125) == 0.25


def test_pmask_reaches_gate_centre(oracle_lib):
    # gamma = 2^-10, 1024 P-mask steps: b0 = 0.5 - 1 = -0.5; while b_th < every
    # gate in (0,1) all tokens are selected (F = 1 > rho), each step adds gamma,
    # and after exactly 1024 steps the threshold sits at 0.5
    gamma, S = 2.0 ** -10, 1024
    b = oracle_lib.pmask_initial_threshold(gamma, S)
    assert b == -0.5
    rng = np.random.default_rng(5)
    gate = rng.uniform(0.0, 1.0, 4096).astype(np.float32)
    cu = np.array([0, gate.size], np.int32)
    for step in range(S):
        thr = oracle_lib.thresholds(gate, cu, oracle_lib.SEL_THRESHOLD, threshold=b)
        _, cu_sel, _ = oracle_lib.select(gate, cu, thr)
        if b < 0:
            assert int(cu_sel[-1]) == gate.size        # P-mask: everything global
        b = oracle_lib.budget_update(b, int(cu_sel[-1]), gate.size, 0.25, gamma)
        if b > 0.0:
            break
    # the first 512 steps (b from -0.5 up to 0) select everything
    assert step >= 511


def test_pmask_start_printed_in_paper(oracle_lib):
    # App. C (training details of the 1.5B comparison): gamma = 0.0005 and a
    # P-mask of S = 5000 steps (20% of 100B tokens at 4M tokens per step)
    # give the printed starting threshold b_th,0 = 0.5 - gamma S = -2.0.
    # gamma is an fp32 argument: 0.0005 in fp32 is 0.00050000002374...,
    # so 0.5 - gamma S = -2.0000001187 in double, 1.187e-7 from -2, less
    # than half an fp32 ulp at 2 (1.192e-7): the fp32 result is exactly -2.
    assert oracle_lib.pmask_initial_threshold(0.0005, 5000) == -2.0


def test_controller_settles_at_target_quantile(oracle_lib):
    # gates on the grid (i + 0.5)/N: the fraction above t is 1 - t, so with
    # rho = 1/4 the controller must settle within gamma of t = 0.75 and then
    # keep F within the mass of one gamma-band of rho
    N, rho, gamma = 4096, 0.25, 2.0 ** -6
    gate = ((np.arange(N) + 0.5) / N).astype(np.float32)
    cu = np.array([0, N], np.int32)
    b = 0.0
    for _ in range(200):
        thr = oracle_lib.thresholds(gate, cu, oracle_lib.SEL_THRESHOLD, threshold=b)
        _, cu_sel, _ = oracle_lib.select(gate, cu, thr)
        b = oracle_lib.budget_update(b, int(cu_sel[-1]), N, rho, gamma)
    assert abs(b - 0.75) <= gamma
    thr = oracle_lib.thresholds(gate, cu, oracle_lib.SEL_THRESHOLD, threshold=b)
    _, cu_sel, _ = oracle_lib.select(gate, cu, thr)
    assert abs(int(cu_sel[-1]) / N - rho) <= gamma


# ---------------------------------------------------------------------------
# One decoding step (Sec. 3.3 and App. B, Autoregressive Decoding): the new
# token is the last row of its sequence's cache.
# ---------------------------------------------------------------------------
DECODE_CASES = [
    # seqlens (cache lengths), Hq, Hkv, d, window, threshold, distinct global, gains
    ((5, 1, 9, 16), 4, 2, 8, 4, 0.5, False, False),
    ((12, 3, 7), 2, 2, 4, 16, 0.3, True, True),
    ((1, 2, 6, 11, 4), 8, 2, 8, 1, 0.6, True, False),
    ((16,), 4, 1, 4, 5, -1.0, False, True),
]


def _decode_inputs(case, seed):
    seqlens, Hq, Hkv, d, window, thr, distinct, gains = case
    rng = np.random.default_rng(seed)
    N = int(sum(seqlens))
    mk = lambda *s: bf16(np.round(rng.standard_normal(s) * 8) / 8)  # noqa: E731
    x = dict(q=mk(N, Hq, d), k=mk(N, Hkv, d), v=mk(N, Hkv, d),
             gate=rng.uniform(0, 1, N).astype(np.float32),
             cu_seqlens=np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int32))
    if distinct:
        x.update(q_g=mk(N, Hq, d), k_g=mk(N, Hkv, d), v_g=mk(N, Hkv, d))
    gl = rng.uniform(0.5, 1.5, (Hq, d)).astype(np.float32) if gains else None
    gg = rng.uniform(0.5, 1.5, (Hq, d)).astype(np.float32) if gains else None
    last = x["cu_seqlens"][1:] - 1
    return x, last, window, thr, gl, gg


@pytest.mark.parametrize("ci", range(len(DECODE_CASES)))
def test_decode_equals_layer_last_rows(oracle_lib, ci):
    """The decoding step reproduces the layer's output at each sequence's last
    position (threshold mode): same local window, same strict gate, same
    global context, same ContextNorm and fusion."""
    x, last, window, thr, gl, gg = _decode_inputs(DECODE_CASES[ci], 700 + ci)
    ref = oracle_lib.logo_fwd(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], window,
                              threshold=thr, q_g=x.get("q_g"), k_g=x.get("k_g"),
                              v_g=x.get("v_g"), gain_local=gl, gain_global=gg)
    dq_g = x["q_g"][last] if "q_g" in x else None
    r = oracle_lib.decode(x["q"][last], x["k"], x["v"], x["gate"][last], x["cu_seqlens"], window,
                          thr, q_g_new=dq_g, k_g=x.get("k_g"), v_g=x.get("v_g"),
                          gain_local=gl, gain_global=gg)
    np.testing.assert_array_equal(r["z"], ref["tok2sel"][last] >= 0)
    np.testing.assert_allclose(r["o_local"], ref["o_local"][last], rtol=0, atol=1e-13)
    np.testing.assert_allclose(r["out"], ref["out"][last], rtol=0, atol=1e-13)
    sel = np.nonzero(r["z"])[0]
    np.testing.assert_allclose(r["o_global"][sel], ref["o_global"][ref["tok2sel"][last[sel]]],
                               rtol=0, atol=1e-13)
    assert not r["o_global"][~r["z"]].any()


@pytest.mark.parametrize("ci", range(len(DECODE_CASES)))
def test_decode_bruteforce(oracle_lib, ci):
    """Independent numpy: the last query row against the cache, explicit masks."""
    x, last, window, thr, gl, gg = _decode_inputs(DECODE_CASES[ci], 800 + ci)
    seqlens = np.diff(x["cu_seqlens"])
    b = brute_layer(x["q"], x["k"], x["v"], x["gate"], seqlens, window, threshold=thr,
                    q_g=x.get("q_g"), k_g=x.get("k_g"), v_g=x.get("v_g"), gain_l=gl, gain_g=gg)
    dq_g = x["q_g"][last] if "q_g" in x else None
    r = oracle_lib.decode(x["q"][last], x["k"], x["v"], x["gate"][last], x["cu_seqlens"], window,
                          thr, q_g_new=dq_g, k_g=x.get("k_g"), v_g=x.get("v_g"),
                          gain_local=gl, gain_global=gg)
    np.testing.assert_array_equal(r["z"], b["selected"][last])
    np.testing.assert_allclose(r["out"], b["out"][last], rtol=0, atol=1e-12)


def test_decode_zero_query_closed_form(oracle_lib):
    """q = 0 gives uniform weights: the local output is the mean of the last w
    cached values, the global one the mean of all of them; an unselected
    token's output is Norm^L of the former, a selected one's the fusion."""
    rng = np.random.default_rng(5)
    seqlens, Hq, Hkv, d, w = (9, 3), 2, 1, 4, 4
    N = sum(seqlens)
    v = bf16(np.round(rng.standard_normal((N, Hkv, d)) * 4) / 4)
    k = bf16(np.round(rng.standard_normal((N, Hkv, d)) * 4) / 4)
    q = np.zeros((2, Hq, d), np.uint16)
    cu = np.array([0, 9, 12], np.int32)
    gate = np.array([0.25, 0.75], np.float32)
    r = oracle_lib.decode(q, k, v, gate, cu, w, 0.5, eps=0.0)
    # strict '>': a gate equal to the threshold stays local
    tie = oracle_lib.decode(q, k, v, np.array([0.5, 0.5], np.float32), cu, w, 0.5, eps=0.0)
    assert tie["z"].tolist() == [False, False] and tie["n_sel"] == 0
    vf = wide(v)[:, 0, :]
    loc = [vf[5:9].mean(0), vf[9:12].mean(0)]
    glo = vf[9:12].mean(0)
    rms = lambda a: a / np.sqrt((a ** 2).mean())  # noqa: E731
    np.testing.assert_allclose(r["o_local"][0, 0], loc[0], atol=1e-15)
    np.testing.assert_allclose(r["o_local"][1, 1], loc[1], atol=1e-15)
    np.testing.assert_allclose(r["o_global"][1, 0], glo, atol=1e-15)
    assert r["z"].tolist() == [False, True]
    np.testing.assert_allclose(r["out"][0, 0], rms(loc[0]), atol=1e-14)
    np.testing.assert_allclose(r["out"][1, 0], 0.25 * rms(loc[1]) + 0.75 * rms(glo), atol=1e-14)


# ---------------------------------------------------------------------------
# Gate projection (Eq. gate-routing) and branch transforms (Eq.
# branch-transform).
# ---------------------------------------------------------------------------
def test_gate_proj_hand_and_init(oracle_lib):
    """Hand values: x.w = 0 gives exactly 1/2; x.w = 1 gives 1/(1+e^-1); a zero
    gate vector (the near-zero initialisation) centres every p at 1/2."""
    x = bf16(np.array([[1.0, 2.0], [2.0, 0.0], [-3.0, 4.0]], np.float32))
    w = bf16(np.array([0.5, -0.25], np.float32))
    p = oracle_lib.gate_proj(x, w)
    assert p.dtype == np.float32
    assert p[0] == np.float32(0.5)
    assert p[1] == np.float32(0.7310585786300049)
    assert p[2] == np.float32(1.0 / (1.0 + math.exp(2.5)))
    z = oracle_lib.gate_proj(x, bf16(np.zeros(2, np.float32)))
    assert (z == np.float32(0.5)).all()


def test_gate_proj_bruteforce(oracle_lib):
    rng = np.random.default_rng(11)
    x = bf16(np.round(rng.standard_normal((37, 96)) * 16) / 16)
    w = bf16(np.round(rng.standard_normal(96) * 16) / 64)
    ref = (1.0 / (1.0 + np.exp(-(wide(x) @ wide(w))))).astype(np.float32)
    np.testing.assert_array_equal(oracle_lib.gate_proj(x, w), ref)


def test_branch_transform_identity_and_permutation(oracle_lib):
    """Both transforms start as identities (Sec. 3.2): LP with A = I and SO with
    s = 1, b = 0 return U; a permutation matrix permutes the channels."""
    rng = np.random.default_rng(12)
    N, H, d = 9, 3, 8
    u = bf16(np.round(rng.standard_normal((N, H, d)) * 8) / 8)
    eye = bf16(np.broadcast_to(np.eye(d, dtype=np.float32), (H, d, d)).copy())
    np.testing.assert_array_equal(oracle_lib.branch_transform(u, oracle_lib.LP, A=eye), wide(u))
    ones, zeros = np.ones((H, d), np.float32), np.zeros((H, d), np.float32)
    np.testing.assert_array_equal(oracle_lib.branch_transform(u, oracle_lib.SO, s=ones, b=zeros),
                                  wide(u))
    perm = [rng.permutation(d) for _ in range(H)]
    P = np.zeros((H, d, d), np.float32)
    for h in range(H):
        P[h, perm[h], np.arange(d)] = 1.0          # out[:, j] = u[:, perm[j]]
    out = oracle_lib.branch_transform(u, oracle_lib.LP, A=bf16(P))
    for h in range(H):
        np.testing.assert_array_equal(out[:, h, :], wide(u)[:, h, perm[h]])


def test_branch_transform_bruteforce_and_rows(oracle_lib):
    rng = np.random.default_rng(13)
    N, H, d = 11, 4, 16
    u = bf16(np.round(rng.standard_normal((N, H, d)) * 8) / 8)
    A = bf16(np.round(rng.standard_normal((H, d, d)) * 8) / 64)
    s = rng.uniform(0.5, 2.0, (H, d)).astype(np.float32)
    b = rng.standard_normal((H, d)).astype(np.float32)
    lp = np.stack([wide(u)[:, h, :] @ wide(A)[h] for h in range(H)], axis=1)
    so = wide(u) * s.astype(np.float64)[None] + b.astype(np.float64)[None]
    np.testing.assert_allclose(oracle_lib.branch_transform(u, oracle_lib.LP, A=A), lp,
                               rtol=0, atol=1e-12)
    np.testing.assert_allclose(oracle_lib.branch_transform(u, oracle_lib.SO, s=s, b=b), so,
                               rtol=0, atol=1e-12)
    rows = np.array([10, 0, 7, 7], np.int32)
    np.testing.assert_allclose(oracle_lib.branch_transform(u, oracle_lib.LP, A=A, rows=rows),
                               lp[rows], rtol=0, atol=1e-12)
    np.testing.assert_allclose(oracle_lib.branch_transform(u, oracle_lib.SO, s=s, b=b, rows=rows),
                               so[rows], rtol=0, atol=1e-12)


# ---------------------------------------------------------------------------
# Backward pass (training; Sec. 3.3 / App. B): the oracle's analytic
# gradients against central finite differences of an independent fp64 numpy
# forward, with the selection held fixed.
# ---------------------------------------------------------------------------
def np_layer_f64(qf, kf, vf, qgf, kgf, vgf, p, seqlens, window, z, gl, gg, eps, scale):
    """The layer in fp64 from float inputs (explicit masks, full score matrix)."""
    N, Hq, d = qf.shape
    G = Hq // kf.shape[1]
    out = np.zeros((N, Hq, d))
    start = 0
    for T in seqlens:
        sl = slice(start, start + T)
        start += T
        if T == 0:
            continue
        i = np.arange(T)[:, None]
        j = np.arange(T)[None, :]
        causal = j <= i
        local = causal & (j > i - window)
        for h in range(Hq):
            ys = []
            for (Q, K, V, mask, g) in ((qf, kf, vf, local, gl), (qgf, kgf, vgf, causal, gg)):
                S = scale * (Q[sl, h, :] @ K[sl, h // G, :].T)
                S = np.where(mask, S, -np.inf)
                W = np.exp(S - S.max(axis=1, keepdims=True))
                O = (W / W.sum(axis=1, keepdims=True)) @ V[sl, h // G, :]
                r = np.sqrt((O ** 2).mean(axis=1, keepdims=True) + eps)
                ys.append(O / r * (1.0 if g is None else g[h][None, :]))
            pw = p[sl][:, None]
            out[sl, h, :] = np.where(z[sl][:, None], (1 - pw) * ys[0] + pw * ys[1], ys[0])
    return out


BWD_CASES = [
    # seqlens, Hq, Hkv, d, window, distinct global tensors, gains, eps
    ((5, 7), 2, 1, 4, 3, False, False, 1e-6),
    ((9,), 4, 2, 8, 4, True, True, 1e-3),
    ((3, 0, 6), 2, 2, 4, 16, False, True, 0.0),
]


@pytest.mark.parametrize("ci", range(len(BWD_CASES)))
def test_backward_finite_differences(oracle_lib, ci):
    seqlens, Hq, Hkv, d, window, distinct, gains, eps = BWD_CASES[ci]
    rng = np.random.default_rng(900 + ci)
    N = sum(seqlens)
    mk = lambda *s: bf16(np.round(rng.standard_normal(s) * 8) / 8)  # noqa: E731
    q, k, v = mk(N, Hq, d), mk(N, Hkv, d), mk(N, Hkv, d)
    qg, kg, vg = (mk(N, Hq, d), mk(N, Hkv, d), mk(N, Hkv, d)) if distinct else (None,) * 3
    # gates kept away from the threshold so no finite step changes the selection
    gate = rng.choice([0.15, 0.3, 0.7, 0.85], N).astype(np.float32)
    gl = rng.uniform(0.5, 1.5, (Hq, d)).astype(np.float32) if gains else None
    gg = rng.uniform(0.5, 1.5, (Hq, d)).astype(np.float32) if gains else None
    cu = np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int32)
    dout = rng.standard_normal((N, Hq, d))
    scale = 1.0 / math.sqrt(d)
    r = oracle_lib.logo_bwd(q, k, v, gate, cu, window, dout, threshold=0.5, q_g=qg, k_g=kg,
                            v_g=vg, gain_local=gl, gain_global=gg, eps=eps)
    z = gate > np.float32(0.5)
    base = dict(qf=wide(q), kf=wide(k), vf=wide(v),
                qgf=wide(qg) if distinct else wide(q), kgf=wide(kg) if distinct else wide(k),
                vgf=wide(vg) if distinct else wide(v), p=gate.astype(np.float64),
                gl=None if gl is None else gl.astype(np.float64),
                gg=None if gg is None else gg.astype(np.float64))

    def loss(**over):
        a = dict(base)
        a.update(over)
        if not distinct:       # aliased global tensors move with the local ones
            for lk, gk in (("qf", "qgf"), ("kf", "kgf"), ("vf", "vgf")):
                if lk in over:
                    a[gk] = a[lk]
        o = np_layer_f64(a["qf"], a["kf"], a["vf"], a["qgf"], a["kgf"], a["vgf"], a["p"],
                         seqlens, window, z, a["gl"], a["gg"], eps, scale)
        return float((dout * o).sum())

    targets = [("qf", "dq"), ("kf", "dk"), ("vf", "dv"), ("p", "dgate")]
    if distinct:
        targets += [("qgf", "dq_g"), ("kgf", "dk_g"), ("vgf", "dv_g")]
    if gains:
        targets += [("gl", "dgain_local"), ("gg", "dgain_global")]
    h = 1e-6
    for name, gname in targets:
        for _ in range(2):
            U = rng.standard_normal(base[name].shape)
            fd = (loss(**{name: base[name] + h * U}) - loss(**{name: base[name] - h * U})) / (2 * h)
            an = float((r[gname] * U).sum())
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, fd, an)


def test_backward_invariants(oracle_lib):
    """Softmax shift invariance makes each branch's key gradients sum to zero
    over a sequence's keys (per KV head); with eps = 0, ContextNorm removes any
    positive scale of v, so <dv, v> = 0."""
    rng = np.random.default_rng(950)
    seqlens, Hq, Hkv, d, w = (12, 7), 4, 2, 8, 5
    N = sum(seqlens)
    mk = lambda *s: bf16(np.round(rng.standard_normal(s) * 8) / 8)  # noqa: E731
    q, k, v = mk(N, Hq, d), mk(N, Hkv, d), mk(N, Hkv, d)
    qg, kg, vg = mk(N, Hq, d), mk(N, Hkv, d), mk(N, Hkv, d)
    gate = rng.uniform(0, 1, N).astype(np.float32)
    cu = np.array([0, 12, 19], np.int32)
    dout = rng.standard_normal((N, Hq, d))
    r = oracle_lib.logo_bwd(q, k, v, gate, cu, w, dout, ratio=0.4, q_g=qg, k_g=kg, v_g=vg, eps=0.0)
    for key in ("dk", "dk_g"):
        for b in range(2):
            np.testing.assert_allclose(r[key][cu[b]:cu[b + 1]].sum(axis=0), 0.0, atol=1e-10)
    assert abs(float((r["dv"] * wide(v)).sum())) < 1e-9
    assert abs(float((r["dv_g"] * wide(vg)).sum())) < 1e-9
    # unselected tokens get no gradient through the fusion weight or the global query
    sel = r["n_sel"]
    assert 0 < sel < N
    t2s = oracle_lib.logo_fwd(q, k, v, gate, cu, w, ratio=0.4)["tok2sel"]
    assert not r["dgate"][t2s < 0].any() and not r["dq_g"][t2s < 0].any()


def test_fusion_bwd_finite_differences(oracle_lib):
    """ContextNorm + fusion backward against central differences of a numpy
    fp64 forward of Eqs. contextnorm / output-fusion."""
    rng = np.random.default_rng(960)
    N, Hq, d, eps = 7, 3, 8, 1e-3
    ol, og = rng.standard_normal((N, Hq, d)), rng.standard_normal((N, Hq, d))
    gate = rng.uniform(0.1, 0.9, N).astype(np.float32)
    z = np.array([1, 0, 1, 1, 0, 0, 1], bool)
    gl = rng.uniform(0.5, 1.5, (Hq, d)).astype(np.float32)
    gg = rng.uniform(0.5, 1.5, (Hq, d)).astype(np.float32)
    dout = rng.standard_normal((N, Hq, d))
    r = oracle_lib.fusion_bwd(ol, og, gate, z, dout, gain_local=gl, gain_global=gg, eps=eps)

    def fwd(ol_, og_, p_, gl_, gg_):
        nl = ol_ / np.sqrt((ol_ ** 2).mean(-1, keepdims=True) + eps) * gl_[None]
        ng = og_ / np.sqrt((og_ ** 2).mean(-1, keepdims=True) + eps) * gg_[None]
        pw = p_[:, None, None]
        return np.where(z[:, None, None], (1 - pw) * nl + pw * ng, nl)

    base = [ol, og, gate.astype(np.float64), gl.astype(np.float64), gg.astype(np.float64)]
    names = ["dol", "dog", "dgate", "dgain_local", "dgain_global"]
    h = 1e-6
    for idx, name in enumerate(names):
        U = rng.standard_normal(base[idx].shape)
        plus, minus = list(base), list(base)
        plus[idx] = base[idx] + h * U
        minus[idx] = base[idx] - h * U
        fd = ((dout * fwd(*plus)).sum() - (dout * fwd(*minus)).sum()) / (2 * h)
        an = float((r[name] * U).sum())
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, fd, an)
    np.testing.assert_allclose(r["delta_l"], (r["dol"] * ol).sum(-1), atol=1e-12)
    np.testing.assert_allclose(r["delta_g"], (r["dog"] * og).sum(-1), atol=1e-12)
    assert not r["dog"][~z].any() and not r["dgate"][~z].any()


def np_attn_f64(qf, kf, vf, seqlens, window, scale):
    """Plain causal attention in fp64 (window <= 0: full causal)."""
    N, Hq, d = qf.shape
    G = Hq // kf.shape[1]
    out = np.zeros((N, Hq, d))
    start = 0
    for T in seqlens:
        sl = slice(start, start + T)
        start += T
        if T == 0:
            continue
        i = np.arange(T)[:, None]
        j = np.arange(T)[None, :]
        mask = (j <= i) & ((j > i - window) if window >= 1 else True)
        for h in range(Hq):
            S = np.where(mask, scale * (qf[sl, h] @ kf[sl, h // G].T), -np.inf)
            W = np.exp(S - S.max(axis=1, keepdims=True))
            out[sl, h] = (W / W.sum(axis=1, keepdims=True)) @ vf[sl, h // G]
    return out


@pytest.mark.parametrize("window", [0, 3])
def test_attn_bwd_finite_differences(oracle_lib, window):
    """Plain attention backward (the dense baseline's) against central
    differences of a numpy fp64 forward, GQA and two sequences."""
    rng = np.random.default_rng(970 + window)
    seqlens, Hq, Hkv, d = (6, 9), 4, 2, 8
    N = sum(seqlens)
    mk = lambda *s: bf16(np.round(rng.standard_normal(s) * 8) / 8)  # noqa: E731
    q, k, v = mk(N, Hq, d), mk(N, Hkv, d), mk(N, Hkv, d)
    cu = np.array([0, 6, 15], np.int32)
    dout = rng.standard_normal((N, Hq, d))
    scale = 0.4
    r = oracle_lib.attn_bwd(q, k, v, cu, window, dout, scale=scale)
    base = dict(q=wide(q), k=wide(k), v=wide(v))

    def loss(**over):
        a = dict(base, **over)
        return float((dout * np_attn_f64(a["q"], a["k"], a["v"], seqlens, window, scale)).sum())

    h = 1e-6
    for name in ("q", "k", "v"):
        for _ in range(2):
            U = rng.standard_normal(base[name].shape)
            fd = (loss(**{name: base[name] + h * U}) - loss(**{name: base[name] - h * U})) / (2 * h)
            an = float((r["d" + name] * U).sum())
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, fd, an)


def test_attn_bwd_window_one(oracle_lib):
    """With one key per row the softmax is constant: dq = dk = 0 and dv_j is
    the sum of dout_j over the query heads of the KV head."""
    rng = np.random.default_rng(975)
    N, Hq, Hkv, d = 11, 6, 2, 4
    mk = lambda *s: bf16(np.round(rng.standard_normal(s) * 8) / 8)  # noqa: E731
    q, k, v = mk(N, Hq, d), mk(N, Hkv, d), mk(N, Hkv, d)
    dout = rng.standard_normal((N, Hq, d))
    r = oracle_lib.attn_bwd(q, k, v, np.array([0, 4, 11], np.int32), 1, dout)
    assert not r["dq"].any() and not r["dk"].any()
    np.testing.assert_allclose(r["dv"], dout.reshape(N, Hkv, Hq // Hkv, d).sum(axis=2),
                               atol=1e-12)


@pytest.mark.parametrize("distinct", [False, True])
def test_backward_sample_matches_full(oracle_lib, distinct):
    """The sampled backward equals the full backward (itself pinned by finite
    differences above) at the sampled queries and keys."""
    rng = np.random.default_rng(990 + distinct)
    seqlens, Hq, Hkv, d, w = (40, 1, 57), 4, 2, 8, 7
    N = sum(seqlens)
    mk = lambda *s: bf16(np.round(rng.standard_normal(s) * 8) / 8)  # noqa: E731
    x = dict(q=mk(N, Hq, d), k=mk(N, Hkv, d), v=mk(N, Hkv, d),
             gate=rng.uniform(0, 1, N).astype(np.float32),
             cu_seqlens=np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int32))
    if distinct:
        x.update(q_g=mk(N, Hq, d), k_g=mk(N, Hkv, d), v_g=mk(N, Hkv, d))
    gl = rng.uniform(0.5, 1.5, (Hq, d)).astype(np.float32)
    dout = rng.standard_normal((N, Hq, d))
    full = oracle_lib.logo_bwd(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], w, dout,
                               ratio=0.3, q_g=x.get("q_g"), k_g=x.get("k_g"), v_g=x.get("v_g"),
                               gain_local=gl, eps=1e-4)
    qrows = np.array([0, 5, 39, 40, 41, 60, 97])
    keys = np.array([0, 3, 39, 40, 44, 80, 97])
    smp = oracle_lib.logo_bwd_sample(x, w, dout, qrows, keys, ratio=0.3, gain_local=gl,
                                     eps=1e-4)
    names = [("dq", qrows), ("dgate", qrows), ("dk", keys), ("dv", keys)]
    if distinct:
        names += [("dq_g", qrows), ("dk_g", keys), ("dv_g", keys)]
    for nm, idx in names:
        np.testing.assert_allclose(smp[nm], full[nm][idx], rtol=1e-11, atol=1e-12, err_msg=nm)
