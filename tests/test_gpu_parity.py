"""GPU parity: the HIP path (called through the C ABI) against the fp64 oracle.

Bars (fixed here, not tuned per run):
  * selection (sel_idx, cu_sel, tok2sel, thresholds): bit-exact;
  * raw branch outputs O^L / O^G / dense (fp32): error relative to each
    (row, head) RMS, max <= 2e-2 and mean <= 2e-3 -- the layer bar expressed
    before ContextNorm (which divides by that RMS);
  * layer output (bf16): max-abs <= 2e-2 and mean-abs <= 2e-3 against the
    fp64 oracle;
  * combine on identical fp32 inputs: within one bf16 rounding of the oracle.
Small cases compare every element; full-size workloads compare a spread of
sampled rows that the oracle computes one by one.
"""
import math

import numpy as np
import pytest

import oracle
import synth
from _support import (bf16_round, err_stats, oracle_layer_rows, rel_rms_err, sample_rows,
                      to_device, torch_bf16_to_f64)

pytestmark = pytest.mark.gpu

MAX_ABS, MEAN_ABS = 2e-2, 2e-3


@pytest.fixture(scope="module")
def pk():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible: the gpu tests need an MI355X")
    import paper_2608_29539_amd as pk
    pk.library()   # raises if liblogo.so is missing
    oracle.build(force=False)
    return pk


def problem(pk, x, dev, w: synth.Workload, window=None, scale=0.0):
    return pk.Problem(dev["cu_seqlens"], w.num_q_heads, w.num_kv_heads, w.head_dim,
                      w.window if window is None else window,
                      cu_seqlens_host=x["cu_seqlens"], softmax_scale=scale)


def report(tag, st):
    print(f"[{tag}] " + " ".join(f"{k}={v:.3g}" if isinstance(v, float) else f"{k}={v}"
                                 for k, v in st.items()), flush=True)


# ---------------------------------------------------------------------------
# selection
# ---------------------------------------------------------------------------
SELECT_CASES = [
    # (name, seqlens, gate kind, mode, value)
    ("T1k-ratio", (1024,), "uniform", "ratio", 0.25),
    ("ragged-ratio", (0, 1, 63, 64, 65, 5000, 0), "uniform", "ratio", 0.3),
    ("ragged-kT-1", (7, 100, 4097), "uniform", "ratio", 0.999),
    ("ratio0", (300, 700), "uniform", "ratio", 0.0),
    ("ratio1", (300, 700), "uniform", "ratio", 1.0),
    ("thr-half", (513, 2048, 1), "uniform", "threshold", 0.5),
    ("thr-neginf", (513, 100), "uniform", "threshold", -math.inf),
    ("thr-posinf", (513, 100), "uniform", "threshold", math.inf),
    ("burst-ratio", (20000,), "markov_burst", "ratio", 1 / 8),
    ("many-seqs", tuple(range(0, 3000, 7)), "uniform", "ratio", 0.125),
]


def _select_and_compare(pk, gate, cu, mode, val, tag):
    import torch
    dev_gate = torch.from_numpy(gate).cuda()
    dev_cu = torch.from_numpy(cu).cuda()
    prob = pk.Problem(dev_cu, 4, 4, 64, 16, cu_seqlens_host=cu)
    kw = dict(ratio=val) if mode == "ratio" else dict(threshold=val)
    sel, cu_sel, t2s, thr = pk.logo_select(prob, dev_gate, **kw)
    torch.cuda.synchronize()
    omode = oracle.SEL_RATIO if mode == "ratio" else oracle.SEL_THRESHOLD
    ethr = oracle.thresholds(gate, cu, omode, threshold=val if mode != "ratio" else 0.0,
                             ratio=val if mode == "ratio" else 0.0)
    esel, ecu, et2s = oracle.select(gate, cu, ethr)
    n = int(ecu[-1])
    assert np.array_equal(thr.cpu().numpy().view(np.uint32), ethr.view(np.uint32)), tag
    assert cu_sel.cpu().numpy().tolist() == ecu.tolist(), tag
    assert sel.cpu().numpy()[:n].tolist() == esel.tolist(), tag
    N = int(cu[-1])
    assert t2s.cpu().numpy()[:N].tolist() == et2s.tolist(), tag
    print(f"[select {tag}] n_sel={n} N={N}", flush=True)


@pytest.mark.parametrize("ci", range(len(SELECT_CASES)), ids=[c[0] for c in SELECT_CASES])
def test_select_bit_exact(pk, ci):
    name, seqlens, kind, mode, val = SELECT_CASES[ci]
    w = synth.small_workload(seqlens, 4, 4, 64, 16, val if mode == "ratio" else 0.0,
                             seed=900 + ci, gate=kind)
    x = synth.make_gate_only(w)
    _select_and_compare(pk, x["gate"], x["cu_seqlens"], mode, val, name)


def test_select_ties_and_nan(pk):
    rng = np.random.default_rng(4)
    cu = np.array([0, 4000, 4000, 9000], np.int32)
    gate = (rng.integers(0, 16, 9000) / 16.0).astype(np.float32)   # heavy ties
    for r in (0.1, 0.5, 0.9):
        _select_and_compare(pk, gate, cu, "ratio", r, f"ties-{r}")
    g2 = gate.copy()
    g2[::97] = np.nan
    g2[5] = -0.0
    g2[6] = 0.0
    _select_and_compare(pk, g2, cu, "threshold", 0.4375, "nan-thr")
    _select_and_compare(pk, g2, cu, "threshold", -0.0, "zero-thr")
    g3 = (rng.standard_normal(9000) * 3).astype(np.float32)         # negative values too
    g3[10:20] = -0.0
    g3[20:30] = 0.0
    for r in (0.05, 0.5, 0.97):
        _select_and_compare(pk, g3, cu, "ratio", r, f"signed-{r}")


def test_select_probability_bin_paths(pk):
    """Ratio mode through each path of the threshold search: the threshold's
    probability bin (width 1/4096) holding a few values, exactly 1024 (the
    most ranked directly), 1025 (radix passes instead) and thousands of equal
    values; gates in [0, 1] throughout."""
    rng = np.random.default_rng(21)
    T = 20000
    base = rng.random(T, dtype=np.float32)
    cases = []
    for n_in_bin in (7, 1024, 1025, 6000):
        g = base.copy()
        idx = rng.choice(T, n_in_bin, replace=False)
        # n_in_bin distinct or equal values inside one bin [0.75, 0.75 + 1/4096)
        if n_in_bin == 6000:
            g[idx] = np.float32(0.75)
        else:
            g[idx] = (np.float32(0.75) + rng.random(n_in_bin, dtype=np.float32)
                      * np.float32(1.0 / 4096 * 0.999)).astype(np.float32)
        # keep every other value out of that bin
        other = np.setdiff1d(np.arange(T), idx)
        inb = (g[other] >= np.float32(0.75)) & (g[other] < np.float32(0.75 + 1.0 / 4096))
        g[other[inb]] = np.float32(0.5)
        cases.append((n_in_bin, g))
    cu = np.array([0, T], np.int32)
    for n_in_bin, g in cases:
        n_above = int((g >= np.float32(0.75 + 1.0 / 4096)).sum())
        # a ratio whose threshold rank falls inside the bin
        k = n_above + n_in_bin // 2
        _select_and_compare(pk, g, cu, "ratio", (k + 0.5) / T, f"bin-{n_in_bin}")


@pytest.mark.parametrize("name", ["T1k-tiny", "T8k-b2", "T32k-gqa", "T128k-gqa",
                                  "varlen-4seq-r0", "varlen-4seq-r0.03125", "varlen-4seq-r0.125",
                                  "varlen-4seq-r0.5", "varlen-4seq-r1"])
def test_select_workloads(pk, name):
    w = synth.WORKLOADS[name]
    x = synth.make_gate_only(w)
    _select_and_compare(pk, x["gate"], x["cu_seqlens"], "ratio", w.ratio, name)


def _select_sweep_cases(n=40, seed=7171):
    """Seeded random selections: 1-40 sequences whose lengths straddle the
    kernel's part (4096) and chunk (32768) edges, gates uniform, logit-normal,
    bursty, heavily tied (multiples of 1/64) or signed normal (outside
    [0, 1]), ratio mode at a random ratio or threshold mode at a random value
    (an exact gate value half the time, to exercise the strict comparison)."""
    rng = np.random.default_rng(seed)
    sizes = [0, 1, 2, 63, 64, 65, 1023, 1024, 1025, 4095, 4096, 4097, 5000, 32767, 32768,
             32769, 70000]
    cases = []
    for i in range(n):
        B = int(rng.choice([1, 1, 2, 3, 7, 40]))
        lens = [int(t) for t in rng.choice(sizes, size=B)]
        if B == 40:
            lens = [min(t, 5000) for t in lens]
        kind = ("uniform", "logit_normal", "markov_burst", "ties", "signed")[i % 5]
        mode = "ratio" if rng.random() < 0.6 else "threshold"
        cases.append((tuple(lens), kind, mode, float(rng.random()), int(rng.integers(1 << 30))))
    return cases


SELECT_SWEEP = _select_sweep_cases()


@pytest.mark.parametrize("ci", range(len(SELECT_SWEEP)))
def test_select_random_sweep(pk, ci):
    lens, kind, mode, u, gseed = SELECT_SWEEP[ci]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    N = int(cu[-1])
    rng = np.random.default_rng(gseed)
    if kind in ("uniform", "logit_normal", "markov_burst"):
        w = synth.small_workload(lens, 4, 4, 64, 16, 0.125, seed=gseed % 100000, gate=kind)
        gate = synth.make_gate_only(w)["gate"]
    elif kind == "ties":
        gate = (rng.integers(0, 65, N) / 64.0).astype(np.float32)
    else:
        gate = (rng.standard_normal(N) * 2.0).astype(np.float32)
    if mode == "ratio":
        val = u
    elif N and u < 0.5:
        val = float(gate[int(u * 2 * N) % N])     # a gate value itself
    else:
        val = float(np.float32(u if kind != "signed" else 4.0 * u - 2.0))
    _select_and_compare(pk, gate, cu, mode, val, f"sweep{ci}-{kind}-{mode}")


def test_select_overflow_threshold_mode(pk):
    """Threshold mode with a small capacity: the first sel_capacity selections
    are kept, the rest are marked -1, and cu_sel still counts them all."""
    import torch
    rng = np.random.default_rng(8)
    cu = np.array([0, 1000, 2500], np.int32)
    gate = rng.random(2500, dtype=np.float32)
    prob = pk.Problem(torch.from_numpy(cu).cuda(), 4, 4, 64, 16, cu_seqlens_host=cu)
    cap = 300
    sel, cu_sel, t2s, _ = pk.logo_select(prob, torch.from_numpy(gate).cuda(), threshold=0.5,
                                         sel_capacity=cap)
    ethr = oracle.thresholds(gate, cu, oracle.SEL_THRESHOLD, threshold=0.5)
    esel, ecu, et2s = oracle.select(gate, cu, ethr)
    assert cu_sel.cpu().numpy().tolist() == ecu.tolist()
    assert sel.cpu().numpy()[:cap].tolist() == esel[:cap].tolist()
    exp = np.where(et2s < cap, et2s, -1)
    assert t2s.cpu().numpy().tolist() == exp.tolist()


# ---------------------------------------------------------------------------
# branches (raw fp32 outputs), every element
# ---------------------------------------------------------------------------
BRANCH_CASES = [
    # (seqlens, Hq, Hkv, d, window)
    ((1000,), 4, 4, 64, 128),
    ((1023, 65), 8, 2, 128, 63),
    ((777,), 8, 1, 128, 64),
    ((700, 1, 129), 2, 1, 64, 65),
    ((513,), 4, 2, 128, 1),
    ((600,), 4, 4, 128, 600),
    ((450, 300), 16, 2, 128, 5000),
    ((2100,), 8, 8, 64, 256),
]


@pytest.mark.parametrize("ci", range(len(BRANCH_CASES)))
def test_local_branch(pk, ci):
    seqlens, hq, hkv, d, win = BRANCH_CASES[ci]
    w = synth.small_workload(seqlens, hq, hkv, d, win, 0.25, seed=1200 + ci)
    x = synth.make_inputs(w)
    dev = to_device(x)
    prob = problem(pk, x, dev, w)
    o = pk.logo_local_attn(prob, dev["q"], dev["k"], dev["v"]).cpu().numpy()
    ref = oracle.attn_rows(x["q"], x["k"], x["v"], x["cu_seqlens"],
                           np.arange(w.total_tokens, dtype=np.int32), win)
    st = rel_rms_err(o, ref)
    report(f"local {ci}", st)
    assert st["max_rel"] <= MAX_ABS and st["mean_rel"] <= MEAN_ABS


@pytest.mark.parametrize("ci", range(len(BRANCH_CASES)))
def test_global_branch(pk, ci):
    import torch
    seqlens, hq, hkv, d, win = BRANCH_CASES[ci]
    ratio = (0.25, 0.5, 0.125, 1.0, 0.05, 0.3, 0.75, 0.2)[ci]
    w = synth.small_workload(seqlens, hq, hkv, d, win, ratio, seed=1300 + ci)
    x = synth.make_inputs(w)
    dev = to_device(x)
    prob = problem(pk, x, dev, w)
    sel, cu_sel, t2s, thr = pk.logo_select(prob, dev["gate"], ratio=ratio)
    cap = pk.logo_ratio_capacity(prob, ratio)
    og = pk.logo_global_attn_sparse_q(prob, dev["q"], dev["k"], dev["v"], sel, cu_sel, cap)
    torch.cuda.synchronize()
    ethr = oracle.thresholds(x["gate"], x["cu_seqlens"], oracle.SEL_RATIO, ratio=ratio)
    esel, ecu, _ = oracle.select(x["gate"], x["cu_seqlens"], ethr)
    n = int(ecu[-1])
    assert int(cu_sel[-1]) == n
    ref = oracle.attn_rows(x["q"], x["k"], x["v"], x["cu_seqlens"], esel, 0)
    got = og.cpu().numpy()[:n]
    st = rel_rms_err(got, ref)
    report(f"global {ci} n={n}", st)
    assert st["max_rel"] <= MAX_ABS and st["mean_rel"] <= MEAN_ABS


@pytest.mark.parametrize("seqlens,hkv,d,ratio", [((6000, 2500), 2, 128, 0.05),
                                                  ((9000,), 8, 64, 0.02),
                                                  ((4100, 33, 4100), 1, 128, 0.5)])
def test_global_branch_long_rows(pk, seqlens, hkv, d, ratio):
    """Few selected rows far into long sequences: the tile plan cuts their KV
    ranges into several entries whose partials are merged (rows whose
    positions lie before an entry's KV range see only masked keys there)."""
    import torch
    w = synth.small_workload(seqlens, 8, hkv, d, 64, ratio, seed=1350 + len(seqlens) + d)
    x = synth.make_inputs(w)
    dev = to_device(x)
    prob = problem(pk, x, dev, w)
    sel, cu_sel, _, _ = pk.logo_select(prob, dev["gate"], ratio=ratio)
    cap = pk.logo_ratio_capacity(prob, ratio)
    og = pk.logo_global_attn_sparse_q(prob, dev["q"], dev["k"], dev["v"], sel, cu_sel, cap)
    og2 = pk.logo_global_attn_sparse_q(prob, dev["q"], dev["k"], dev["v"], sel, cu_sel, cap)
    torch.cuda.synchronize()
    ethr = oracle.thresholds(x["gate"], x["cu_seqlens"], oracle.SEL_RATIO, ratio=ratio)
    esel, ecu, _ = oracle.select(x["gate"], x["cu_seqlens"], ethr)
    n = int(ecu[-1])
    ref = oracle.attn_rows(x["q"], x["k"], x["v"], x["cu_seqlens"], esel, 0)
    got = og.cpu().numpy()[:n]
    st = rel_rms_err(got, ref)
    report(f"global long n={n}", st)
    assert st["max_rel"] <= MAX_ABS and st["mean_rel"] <= MEAN_ABS
    # the merge order is fixed: repeated calls agree bit for bit
    assert torch.equal(og[:n], og2[:n])


@pytest.mark.parametrize("ci", [0, 1, 2, 3, 7])
def test_dense_causal(pk, ci):
    seqlens, hq, hkv, d, win = BRANCH_CASES[ci]
    w = synth.small_workload(seqlens, hq, hkv, d, win, 0.0, seed=1400 + ci)
    x = synth.make_inputs(w)
    dev = to_device(x)
    prob = problem(pk, x, dev, w)
    o = torch_bf16_to_f64(pk.logo_dense_causal_attn(prob, dev["q"], dev["k"], dev["v"]))
    ref = oracle.attn_rows(x["q"], x["k"], x["v"], x["cu_seqlens"],
                           np.arange(w.total_tokens, dtype=np.int32), 0)
    st = rel_rms_err(o, ref)
    report(f"dense {ci}", st)
    # bf16 output: add one bf16 rounding (2^-9 relative) to the raw-branch bar
    assert st["max_rel"] <= MAX_ABS + 2 ** -8 and st["mean_rel"] <= MEAN_ABS + 2 ** -9


def test_combine_on_identical_inputs(pk):
    """logo_combine fed the oracle's branch outputs (rounded to fp32) against
    the oracle's ContextNorm + fusion of those same fp32 values."""
    import torch
    rng = np.random.default_rng(21)
    N, hq, d = 700, 6, 128
    cu = np.array([0, 300, 700], np.int32)
    ol = rng.standard_normal((N, hq, d)).astype(np.float32) * rng.uniform(0.1, 3, (N, hq, 1)).astype(np.float32)
    t2s = np.full(N, -1, np.int32)
    selected = np.sort(rng.choice(N, 200, replace=False))
    t2s[selected] = np.arange(200)
    og = rng.standard_normal((200, hq, d)).astype(np.float32)
    gate = rng.random(N, dtype=np.float32)
    gl = rng.uniform(0.5, 1.5, (hq, d)).astype(np.float32)
    gg = rng.uniform(0.5, 1.5, (hq, d)).astype(np.float32)
    prob = pk.Problem(torch.from_numpy(cu).cuda(), hq, hq, d, 16, cu_seqlens_host=cu)
    T = lambda a: torch.from_numpy(a).cuda()
    for norm, gains in ((True, False), (True, True), (False, False)):
        out = pk.logo_combine(prob, T(ol), T(og), T(gate), T(t2s),
                              gain_local=T(gl) if gains else None,
                              gain_global=T(gg) if gains else None, apply_norm=norm)
        got = torch_bf16_to_f64(out)
        nl = oracle.contextnorm(ol, gl if gains else None) if norm else ol.astype(np.float64)
        ng = oracle.contextnorm(og, gg if gains else None) if norm else og.astype(np.float64)
        ref = oracle.fuse(nl, ng, gate, t2s)
        # one bf16 rounding (<= 2^-9 relative) plus fp32 evaluation error
        assert np.all(np.abs(got - ref) <= np.abs(ref) * 2.0 ** -8 + 1e-6), (norm, gains)
        assert np.mean(got == bf16_round(ref)) > 0.99, (norm, gains)


# ---------------------------------------------------------------------------
# whole layer
# ---------------------------------------------------------------------------
def _layer(pk, w: synth.Workload, x=None, n_sel_rows=96, n_other=96, full=False, **kw):
    import torch
    x = synth.make_inputs(w) if x is None else x
    dev = to_device(x)
    prob = problem(pk, x, dev, w)
    extra = {k: dev[k] for k in ("q_g", "k_g", "v_g") if k in dev}
    out, sel, cu_sel, t2s, thr = pk.logo_attn_fwd(prob, dev["q"], dev["k"], dev["v"], dev["gate"],
                                                  ratio=w.ratio, **extra, **kw)
    torch.cuda.synchronize()
    ethr = oracle.thresholds(x["gate"], x["cu_seqlens"], oracle.SEL_RATIO, ratio=w.ratio)
    esel, ecu, et2s = oracle.select(x["gate"], x["cu_seqlens"], ethr)
    n = int(ecu[-1])
    assert cu_sel.cpu().numpy().tolist() == ecu.tolist()
    assert sel.cpu().numpy()[:n].tolist() == esel.tolist()
    assert t2s.cpu().numpy()[:w.total_tokens].tolist() == et2s.tolist()
    rows = (np.arange(w.total_tokens, dtype=np.int32) if full else
            sample_rows(x["cu_seqlens"], et2s, n_sel_rows, n_other, seed=w.seed))
    ref = oracle_layer_rows(x, w.window, rows, ratio=w.ratio)
    got = torch_bf16_to_f64(out[torch.from_numpy(rows).long().cuda()])
    st = err_stats(got, ref["out"])
    report(f"layer {w.name} rows={rows.size} n_sel={n}", st)
    assert st["max_abs"] <= MAX_ABS and st["mean_abs"] <= MEAN_ABS
    return out


def test_layer_tiny_full(pk, fwd_launches):
    _layer(pk, synth.WORKLOADS["T1k-tiny"], full=True)


@pytest.mark.parametrize("name", ["T8k-b2", "T32k-gqa", "varlen-4seq-r0", "varlen-4seq-r0.03125",
                                  "varlen-4seq-r0.125", "varlen-4seq-r0.5", "varlen-4seq-r1"])
def test_layer_workloads_sampled(pk, name):
    _layer(pk, synth.WORKLOADS[name])


def test_layer_longest_sampled(pk):
    _layer(pk, synth.WORKLOADS["T128k-gqa"], n_sel_rows=40, n_other=64)


@pytest.mark.parametrize("ci", range(4))
def test_layer_small_full(pk, ci, fwd_launches):
    cases = [((1000, 23, 1), 8, 2, 128, 100, 0.3), ((513,), 4, 4, 64, 1, 0.9),
             ((640, 0, 300), 8, 8, 128, 2000, 0.5), ((129, 257), 16, 2, 64, 64, 1.0)]
    seqlens, hq, hkv, d, win, r = cases[ci]
    w = synth.small_workload(seqlens, hq, hkv, d, win, r, seed=1500 + ci)
    _layer(pk, w, full=True)


def _sweep_cases(n=32, seed=4242):
    """Seeded random layer shapes inside the documented domain: 1-3 ragged
    sequences (empty, one token, tile edges, several tiles), each G in
    {1, 2, 4, 8} with each d in {64, 128} four times, 1-8 KV heads, windows
    from 1 to beyond T, ratios from 0 to 1."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        B = int(rng.integers(1, 4))
        seqlens = [int(t) for t in rng.choice([0, 1, 63, 64, 65, 255, 700, 1500, 2900], size=B)]
        if sum(seqlens) == 0:
            seqlens[-1] = 300
        hkv = int(rng.choice([1, 2, 4, 8]))
        G = (1, 2, 4, 8)[i % 4]
        if hkv * G > 32:
            hkv = 32 // G
        d = (64, 128)[(i // 4) % 2]
        win = int(rng.choice([1, 16, 64, 65, 200, 1024, 5000]))
        r = float(rng.choice([0.0, 0.02, 0.125, 0.3, 0.75, 1.0]))
        cases.append((tuple(seqlens), hkv * G, hkv, d, win, r))
    return cases


SWEEP_CASES = _sweep_cases()


def test_layer_random_sweep_full(pk, fwd_launches):
    """Every element of every sweep case against the oracle, selection bit for
    bit.  The whole sweep is held to the criterion of the full-output tests:
    each case within the mean bar; an element above 2e-2 only where the
    output's one bf16 rounding (spacing 2^-5 at |out| >= 4) falls on the far
    side of a rounding midpoint after the noise of the bf16 softmax weights
    in the PV product, so it must still be one of the two bf16 values that
    bracket the oracle value; and such elements at most one in 10^7 of the
    sweep's elements (one, 4.4688 against 4.4479, in 4.4e7 as measured)."""
    import torch
    total = over = 0
    for ci, (seqlens, hq, hkv, d, win, r) in enumerate(SWEEP_CASES):
        w = synth.small_workload(seqlens, hq, hkv, d, win, r, seed=1700 + ci)
        tag = f"sweep {ci}: T={seqlens} Hq={hq} Hkv={hkv} d={d} w={win} ratio={r}"
        print(f"[{tag}]", flush=True)
        x = synth.make_inputs(w)
        dev = to_device(x)
        prob = problem(pk, x, dev, w)
        out, sel, cu_sel, t2s, _ = pk.logo_attn_fwd(prob, dev["q"], dev["k"], dev["v"],
                                                    dev["gate"], ratio=r)
        torch.cuda.synchronize()
        ethr = oracle.thresholds(x["gate"], x["cu_seqlens"], oracle.SEL_RATIO, ratio=r)
        esel, ecu, et2s = oracle.select(x["gate"], x["cu_seqlens"], ethr)
        n = int(ecu[-1])
        assert cu_sel.cpu().numpy().tolist() == ecu.tolist(), tag
        assert sel.cpu().numpy()[:n].tolist() == esel.tolist(), tag
        assert t2s.cpu().numpy()[:w.total_tokens].tolist() == et2s.tolist(), tag
        ref = oracle_layer_rows(x, win, np.arange(w.total_tokens, dtype=np.int32), ratio=r)["out"]
        bits = out.view(torch.int16).cpu().numpy().view(np.uint16)[:w.total_tokens]
        got = synth.f32_from_bf16_bits(bits.reshape(-1)).reshape(ref.shape).astype(np.float64)
        st = err_stats(got, ref)
        report(tag, st)
        assert st["mean_abs"] <= MEAN_ABS, (tag, st)
        big = np.argwhere(np.abs(got - ref) > MAX_ABS)
        for bi in big:
            # bf16 is sign-magnitude: the fp32 value's top half truncates
            # toward zero, and the next code up is the next magnitude
            lo = np.uint16(np.float32(ref[tuple(bi)]).view(np.uint32) >> 16)
            hit = bits.reshape(ref.shape)[tuple(bi)]
            assert hit in (lo, np.uint16(lo + 1)), (tag, tuple(int(v) for v in bi),
                                                    float(ref[tuple(bi)]), float(got[tuple(bi)]))
        total += ref.size
        over += int(big.shape[0])
    print(f"[sweep] {over} of {total} elements above {MAX_ABS}", flush=True)
    assert over <= total * 1e-7


def test_profiled_entry_matches_plain(pk, fwd_launches):
    """logo_attn_fwd_profiled runs the same launches as logo_attn_fwd and
    records five caller-created HIP events at the stage boundaries: the
    output and the selection are bit-identical, every stage time is >= 0 and
    the stage times add up to the first-to-last elapsed time."""
    import torch
    w = synth.small_workload((3000, 1200), 16, 4, 128, 256, 0.2, seed=1800)
    x = synth.make_inputs(w)
    dev = to_device(x)
    prob = problem(pk, x, dev, w)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
    for e in evs:
        e.record()                      # creates the HIP event behind each object
    torch.cuda.synchronize()
    a = pk.logo_attn_fwd(prob, dev["q"], dev["k"], dev["v"], dev["gate"], ratio=w.ratio)
    b = pk.logo_attn_fwd(prob, dev["q"], dev["k"], dev["v"], dev["gate"], ratio=w.ratio,
                         events=evs)
    torch.cuda.synchronize()
    n = int(a[2][-1])
    assert torch.equal(a[0].view(torch.int16), b[0].view(torch.int16))
    assert torch.equal(a[1][:n], b[1][:n]) and torch.equal(a[2], b[2])
    assert torch.equal(a[3], b[3])
    stages = [evs[j].elapsed_time(evs[j + 1]) for j in range(4)]
    total = evs[0].elapsed_time(evs[4])
    print(f"[profiled] stages ms {[round(t, 4) for t in stages]} total {total:.4f}", flush=True)
    assert all(t >= 0.0 for t in stages)
    assert abs(sum(stages) - total) <= 1e-3 + 1e-3 * total


def test_layer_distinct_global_tensors(pk, fwd_launches):
    w = synth.small_workload((900, 400), 8, 2, 128, 96, 0.4, seed=1600)
    x = synth.make_inputs(w, distinct_global=True)
    _layer(pk, w, x=x, full=True)


def test_layer_all_sequences_empty(pk):
    """A batch whose every sequence is empty (N = 0): the layer and its
    training forward / backward return OK, cu_sel is all zeros, ratio mode's
    threshold is -inf (k = T = 0) and threshold mode's is the given value."""
    import torch
    cu_host = np.zeros(4, np.int32)
    prob = pk.Problem(torch.zeros(4, dtype=torch.int32, device="cuda"), 8, 2, 64, 16,
                      cu_seqlens_host=cu_host)
    e = lambda h: torch.empty(0, h, 64, dtype=torch.bfloat16, device="cuda")
    q, k, v = e(8), e(2), e(2)
    gate = torch.empty(0, dtype=torch.float32, device="cuda")
    for kw, thr_ref in ((dict(ratio=0.5), -math.inf), (dict(threshold=0.2), np.float32(0.2))):
        out, sel_idx, cu_sel, tok2sel, thr = pk.logo_attn_fwd(prob, q, k, v, gate, **kw)
        torch.cuda.synchronize()
        assert out.shape == (0, 8, 64)
        assert cu_sel.cpu().tolist() == [0, 0, 0, 0], kw
        assert thr.cpu().tolist() == [thr_ref] * 3, kw
    saved = pk.logo_attn_fwd_train(prob, q, k, v, gate, ratio=0.5)
    g = pk.logo_attn_bwd(prob, q, k, v, gate, saved, e(8))
    torch.cuda.synchronize()
    assert saved["cu_sel"].cpu().tolist() == [0, 0, 0, 0]
    assert g["dq"].shape == (0, 8, 64) and g["dk"].shape == (0, 2, 64)
    assert g["dgate"].shape == (0,)
    # the standalone steps and the dense baseline
    sel_idx, cu_sel, tok2sel, thr = pk.logo_select(prob, gate, ratio=0.25)
    o_l = pk.logo_local_attn(prob, q, k, v)
    o_g = pk.logo_global_attn_sparse_q(prob, q, k, v, sel_idx, cu_sel, 0)
    o = pk.logo_combine(prob, o_l, o_g, gate, tok2sel)
    dense = pk.logo_dense_causal_attn(prob, q, k, v)
    torch.cuda.synchronize()
    assert cu_sel.cpu().tolist() == [0, 0, 0, 0]
    assert o_l.shape == (0, 8, 64) and o.shape == (0, 8, 64) and dense.shape == (0, 8, 64)


def test_single_selected_at_position_zero(pk, fwd_launches):
    import torch
    w = synth.small_workload((300,), 4, 2, 128, 32, 0.0, seed=1700)
    x = synth.make_inputs(w)
    x["gate"][:] = 0.1
    x["gate"][0] = 0.9
    dev = to_device(x)
    prob = problem(pk, x, dev, w)
    out, sel, cu_sel, t2s, _ = pk.logo_attn_fwd(prob, dev["q"], dev["k"], dev["v"], dev["gate"],
                                                threshold=0.5)
    assert cu_sel.cpu().tolist() == [0, 1] and int(sel[0]) == 0
    ref = oracle.logo_fwd(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], 32, threshold=0.5)
    st = err_stats(torch_bf16_to_f64(out), ref["out"])
    report("single-at-0", st)
    assert st["max_abs"] <= MAX_ABS and st["mean_abs"] <= MEAN_ABS


@pytest.mark.parametrize("case", ["late-rows-split", "none-selected", "many-seqs"])
def test_layer_launch_cases(pk, case, fwd_launches):
    """Both launch plans of the layer (Hq / Hkv a multiple of 4), every output
    element against the oracle: a long sequence whose few selected rows all
    sit near its end (in one launch their global tiles are longer than the
    launch's mean load, so the work table splits each over four KV ranges
    whose partials are merged inside the launch), a threshold no gate passes
    (no global item: the local items alone), and a batch of 40 short ragged
    sequences (empty ones included)."""
    import torch
    if case == "late-rows-split":
        w = synth.small_workload((20000,), 8, 2, 128, 256, 0.0, seed=2100)
        x = synth.make_inputs(w)
        x["gate"][:] = x["gate"] * 0.5
        x["gate"][-100:] = 0.9
        kw = dict(threshold=0.5)
    elif case == "none-selected":
        w = synth.small_workload((3000, 1000), 8, 2, 64, 128, 0.0, seed=2101)
        x = synth.make_inputs(w)
        kw = dict(threshold=2.0)
    else:
        lens = np.random.default_rng(2102).integers(0, 600, 40)
        lens[[3, 17]] = 0
        w = synth.small_workload(tuple(int(t) for t in lens), 16, 4, 64, 100, 0.3, seed=2102)
        x = synth.make_inputs(w)
        kw = dict(ratio=0.3)
    dev = to_device(x)
    prob = problem(pk, x, dev, w)
    out, sel, cu_sel, t2s, _ = pk.logo_attn_fwd(prob, dev["q"], dev["k"], dev["v"], dev["gate"],
                                                **kw)
    torch.cuda.synchronize()
    ref = oracle.logo_fwd(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], w.window, **kw)
    assert cu_sel.cpu().numpy().tolist() == ref["cu_sel"].tolist()
    n = int(ref["cu_sel"][-1])
    assert n == {"late-rows-split": 100, "none-selected": 0}.get(case, n)
    assert sel.cpu().numpy()[:n].tolist() == ref["sel_idx"][:n].tolist()
    st = err_stats(torch_bf16_to_f64(out), ref["out"])
    assert pk.logo_attn_fwd_launches(prob) == fwd_launches
    report(f"launches={fwd_launches} {case} n_sel={n}", st)
    assert st["max_abs"] <= MAX_ABS and st["mean_abs"] <= MEAN_ABS


def test_fwd_launch_plan(pk, monkeypatch):
    """logo_attn_fwd_launches: one launch where both branches use the same
    workgroups and the local work covers building the work table, two
    otherwise; LOGO_FWD_LAUNCHES forces the choice only where both plans
    apply."""
    import torch
    monkeypatch.delenv("LOGO_FWD_LAUNCHES", raising=False)

    def plan(seqlens, hq, hkv, d, win):
        cu = np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int32)
        prob = pk.Problem(torch.from_numpy(cu).cuda(), hq, hkv, d, win, cu_seqlens_host=cu)
        return pk.logo_attn_fwd_launches(prob)
    assert plan((32768,), 32, 8, 128, 1024) == 1          # T32k-gqa
    assert plan((8192, 8192), 16, 16, 128, 512) == 1      # T8k-b2 (MHA)
    assert plan((1024,), 4, 4, 64, 128) == 2              # T1k-tiny: too little local work
    assert plan((32768,), 32, 16, 128, 1024) == 2         # G = 2: different workgroups
    monkeypatch.setenv("LOGO_FWD_LAUNCHES", "1")
    assert plan((1024,), 4, 4, 64, 128) == 1
    assert plan((32768,), 32, 16, 128, 1024) == 2
    monkeypatch.setenv("LOGO_FWD_LAUNCHES", "2")
    assert plan((32768,), 32, 8, 128, 1024) == 2


def test_determinism(pk, fwd_launches):
    import torch
    w = synth.small_workload((3000, 1500), 8, 2, 128, 256, 0.25, seed=1800)
    x = synth.make_inputs(w)
    dev = to_device(x)
    prob = problem(pk, x, dev, w)
    a = pk.logo_attn_fwd(prob, dev["q"], dev["k"], dev["v"], dev["gate"], ratio=0.25)[0].clone()
    b = pk.logo_attn_fwd(prob, dev["q"], dev["k"], dev["v"], dev["gate"], ratio=0.25)[0].clone()
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_layer_gains_fused_epilogue(pk, fwd_launches):
    """Per-branch ContextNorm gains through the fused epilogues of logo_attn_fwd."""
    import torch
    w = synth.small_workload((1100, 333), 8, 2, 128, 160, 0.3, seed=1900)
    x = synth.make_inputs(w, distinct_global=True)
    rng = np.random.default_rng(19)
    gl = rng.uniform(0.5, 1.5, (8, 128)).astype(np.float32)
    gg = rng.uniform(0.5, 1.5, (8, 128)).astype(np.float32)
    dev = to_device(x)
    prob = problem(pk, x, dev, w)
    out = pk.logo_attn_fwd(prob, dev["q"], dev["k"], dev["v"], dev["gate"], ratio=w.ratio,
                           q_g=dev["q_g"], k_g=dev["k_g"], v_g=dev["v_g"],
                           gain_local=torch.from_numpy(gl).cuda(),
                           gain_global=torch.from_numpy(gg).cuda(), eps=1e-5)[0]
    torch.cuda.synchronize()
    ref = oracle.logo_fwd(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], w.window,
                          ratio=w.ratio, q_g=x["q_g"], k_g=x["k_g"], v_g=x["v_g"],
                          gain_local=gl, gain_global=gg, eps=1e-5)
    st = err_stats(torch_bf16_to_f64(out), ref["out"])
    report("gains-fused", st)
    # the bar is stated for unit-RMS rows; gains scale the rows (and so the
    # bf16 rounding of the output) by at most max(gain)
    gmax = float(max(gl.max(), gg.max()))
    assert st["max_abs"] <= MAX_ABS * gmax and st["mean_abs"] <= MEAN_ABS * gmax


def test_layer_threshold_overflow(pk, fwd_launches):
    """Threshold mode with a capacity below the number of passing tokens:
    the first sel_capacity selections are fused, the rest are treated as
    unselected, cu_sel still counts them all."""
    import torch
    w = synth.small_workload((900, 500), 4, 4, 64, 64, 0.0, seed=2000)
    x = synth.make_inputs(w)
    dev = to_device(x)
    prob = problem(pk, x, dev, w)
    cap = 200
    out, sel, cu_sel, t2s, _ = pk.logo_attn_fwd(prob, dev["q"], dev["k"], dev["v"], dev["gate"],
                                                threshold=0.5, sel_capacity=cap)
    torch.cuda.synchronize()
    full = oracle.logo_fwd(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], w.window,
                           threshold=0.5)
    assert cu_sel.cpu().numpy().tolist() == full["cu_sel"].tolist()
    assert int(cu_sel[-1]) > cap
    # expected: tokens with rank >= cap behave as unselected (gate forced below threshold)
    g2 = x["gate"].copy()
    g2[full["sel_idx"][cap:]] = 0.0
    ref = oracle.logo_fwd(x["q"], x["k"], x["v"], g2, x["cu_seqlens"], w.window, threshold=0.5)
    st = err_stats(torch_bf16_to_f64(out), ref["out"])
    report("thr-overflow", st)
    assert st["max_abs"] <= MAX_ABS and st["mean_abs"] <= MEAN_ABS
