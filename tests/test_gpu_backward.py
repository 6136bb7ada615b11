"""GPU parity of the training forward and the backward pass of the layer
(selection held fixed): logo_attn_fwd_train and logo_attn_bwd through the C
ABI against the fp64 oracle's forward and backward.

Bars.  Training forward: the bf16 output within the layer's bar (max-abs
2e-2, mean-abs 2e-3, times max(gain) when gains are given).  Backward: for every gradient tensor G (dq, dk, dv, the
global-branch ones, dgate, the gain gradients), against the oracle's G_ref:
  relative L2 error  ||G - G_ref|| / ||G_ref||  <= 1e-2
  max-abs error      max |G - G_ref|            <= 2e-2 max |G_ref|
The kernels round dO, P and dS to bf16 (relative error <= 2^-9 each) for the
matrix products and accumulate in fp32; a gradient element is a sum of
products of two or three such rounded factors, so its per-term relative
error is below 3 * 2^-9 = 0.6%, and sums of many terms with independent
rounding errors sit well under that in L2.  The bars leave about a factor 2
over the worst case measured here.
"""
import math

import numpy as np
import pytest

import oracle
import synth
from _support import to_device, torch_bf16_to_f64, err_stats

pytestmark = pytest.mark.gpu

REL_L2, REL_MAX = 1e-2, 2e-2


@pytest.fixture(scope="module")
def pk():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible: the gpu tests need an MI355X")
    import paper_2608_29539_amd as pk
    pk.library()
    oracle.build(force=False)
    return pk


def grad_err(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    nref = np.linalg.norm(ref)
    mref = np.abs(ref).max() if ref.size else 0.0
    if nref == 0.0:
        return dict(rel_l2=float(np.linalg.norm(got)), rel_max=float(np.abs(got).max()
                                                                      if got.size else 0.0))
    return dict(rel_l2=float(np.linalg.norm(got - ref) / nref),
                rel_max=float(np.abs(got - ref).max() / mref))


def run_case(pk, w, *, ratio=None, threshold=None, distinct=False, gains=False, tag=""):
    import torch
    x = synth.make_inputs(w, distinct_global=distinct)
    dout = synth.make_dout(w, 1)
    rng = np.random.default_rng(w.seed + 17)
    gl = rng.uniform(0.5, 1.5, (w.num_q_heads, w.head_dim)).astype(np.float32) if gains else None
    gg = rng.uniform(0.5, 1.5, (w.num_q_heads, w.head_dim)).astype(np.float32) if gains else None
    dev = to_device(dict(x, dout=dout))
    prob = pk.Problem(dev["cu_seqlens"], w.num_q_heads, w.num_kv_heads, w.head_dim, w.window,
                      cu_seqlens_host=x["cu_seqlens"])
    tg = lambda a: torch.from_numpy(a).cuda() if a is not None else None  # noqa: E731
    kw = dict(q_g=dev.get("q_g"), k_g=dev.get("k_g"), v_g=dev.get("v_g"), gain_local=tg(gl),
              gain_global=tg(gg), eps=1e-6)
    print(f"[bwd {tag}] seqlens={w.seqlens} H={w.num_q_heads}/{w.num_kv_heads} "
          f"d={w.head_dim} w={w.window} ratio={ratio} thr={threshold}", flush=True)
    saved = pk.logo_attn_fwd_train(prob, dev["q"], dev["k"], dev["v"], dev["gate"], ratio=ratio,
                                   threshold=threshold, **kw)
    grads = pk.logo_attn_bwd(prob, dev["q"], dev["k"], dev["v"], dev["gate"], saved,
                             dev["dout"], **kw)
    torch.cuda.synchronize()

    # forward output against the oracle
    okw = dict(ratio=ratio, threshold=threshold, q_g=x.get("q_g"), k_g=x.get("k_g"),
               v_g=x.get("v_g"), gain_local=gl, gain_global=gg, eps=1e-6)
    fref = oracle.logo_fwd(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], w.window, **okw)
    st = err_stats(torch_bf16_to_f64(saved["out"]), fref["out"])
    # the layer's bar is stated for unit-RMS rows; gains scale the rows (and
    # so the bf16 rounding of the output) by at most max(gain)
    gmax = max(float(gl.max()), float(gg.max())) if gains else 1.0
    assert st["max_abs"] <= 2e-2 * gmax and st["mean_abs"] <= 2e-3 * gmax, (tag, "fwd", st)
    n_sel = int(saved["cu_sel"].cpu()[-1])
    assert n_sel == fref["n_sel"], (tag, n_sel, fref["n_sel"])

    dout64 = synth.f32_from_bf16_bits(dout).reshape(dout.shape).astype(np.float64)
    ref = oracle.logo_bwd(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], w.window, dout64,
                          **okw)
    names = ["dq", "dk", "dv", "dgate", "dgain_local", "dgain_global"]
    if distinct:
        names += ["dq_g", "dk_g", "dv_g"]
    worst = {}
    for nm in names:
        e = grad_err(grads[nm].cpu().numpy(), ref[nm])
        if nm == "dgate" and n_sel and not np.any(ref[nm]):
            # identical branches (window >= T, the same tensors, no gains):
            # dL/dp_t = dout . (Norm^G - Norm^L) is 0 in exact arithmetic, and
            # the GPU's value is the rounding difference of its two branch
            # kernels; measured against the size of one term, sum |dout * out|
            term = np.abs(dout64 * fref["out"]).sum(axis=(1, 2))
            got = grads[nm].cpu().numpy().astype(np.float64)
            e = dict(rel_l2=float(np.linalg.norm(got) / np.linalg.norm(term)),
                     rel_max=float(np.abs(got).max() / term.max()))
        worst[nm] = e
        print(f"[bwd {tag}] {nm}: rel_l2={e['rel_l2']:.3g} rel_max={e['rel_max']:.3g}",
              flush=True)
    for nm, e in worst.items():
        assert e["rel_l2"] <= REL_L2 and e["rel_max"] <= REL_MAX, (tag, nm, e)
    return grads, ref


BWD_CASES = [
    # (seqlens, Hq, Hkv, d, window, ratio, threshold, distinct, gains)
    ((300, 1000), 8, 2, 128, 257, 0.25, None, False, True),
    ((64, 65, 700), 4, 4, 64, 64, None, 0.5, True, False),
    ((2048,), 16, 2, 128, 1, 0.125, None, False, False),
    ((129,), 4, 1, 128, 4096, 0.0, None, False, True),
    ((513, 200), 4, 2, 64, 100, 1.0, None, True, True),
    ((3000,), 6, 2, 64, 512, 0.5, None, False, False),
    ((1024, 77), 32, 8, 128, 256, 0.125, None, False, True),
    ((1, 2, 3, 190), 2, 2, 128, 3, None, -math.inf, False, False),
    ((1, 0, 37, 2, 0, 65), 4, 2, 64, 16, None, 0.5, True, True),
]


@pytest.mark.parametrize("ci", range(len(BWD_CASES)))
def test_backward_small(pk, ci):
    lens, hq, hkv, d, win, ratio, thr, distinct, gains = BWD_CASES[ci]
    w = synth.small_workload(lens, hq, hkv, d, win, ratio or 0.0, seed=5000 + ci)
    run_case(pk, w, ratio=ratio, threshold=thr, distinct=distinct, gains=gains, tag=f"case{ci}")


def _bwd_sweep_cases(n=16, seed=5151):
    """Seeded random shapes for the training forward + backward: 1-3 ragged
    sequences (empty, one token, tile edges, several tiles), each G in
    {1, 2, 4, 8} with each d in {64, 128} twice, 1-4 KV heads, windows from 1
    to beyond T, ratio or threshold mode, distinct global tensors and gains
    drawn at random."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        B = int(rng.integers(1, 4))
        lens = [int(t) for t in rng.choice([0, 1, 63, 64, 65, 255, 700, 1500], size=B)]
        if sum(lens) == 0:
            lens[-1] = 200
        hkv = int(rng.choice([1, 2, 4]))
        G = (1, 2, 4, 8)[i % 4]
        d = (64, 128)[(i // 4) % 2]
        win = int(rng.choice([1, 16, 64, 65, 200, 1024, 5000]))
        if rng.random() < 0.75:
            ratio, thr = float(rng.choice([0.0, 0.02, 0.125, 0.3, 0.75, 1.0])), None
        else:
            ratio, thr = None, float(rng.choice([0.25, 0.5, 0.9]))
        cases.append((tuple(lens), hkv * G, hkv, d, win, ratio, thr, bool(rng.random() < 0.5),
                      bool(rng.random() < 0.5)))
    return cases


BWD_SWEEP = _bwd_sweep_cases()


@pytest.mark.parametrize("ci", range(len(BWD_SWEEP)),
                         ids=[f"T{'-'.join(map(str, c[0]))}_h{c[1]}-{c[2]}_d{c[3]}_w{c[4]}"
                              f"_{'r' + str(c[5]) if c[6] is None else 'thr' + str(c[6])}"
                              f"{'_distinct' if c[7] else ''}{'_gains' if c[8] else ''}"
                              for c in BWD_SWEEP])
def test_backward_random_sweep(pk, ci):
    lens, hq, hkv, d, win, ratio, thr, distinct, gains = BWD_SWEEP[ci]
    w = synth.small_workload(lens, hq, hkv, d, win, ratio or 0.0, seed=5200 + ci)
    run_case(pk, w, ratio=ratio, threshold=thr, distinct=distinct, gains=gains,
             tag=f"sweep{ci}")


DENSE_CASES = [
    # (seqlens, Hq, Hkv, d)
    ((300, 1000), 8, 2, 128),
    ((64, 65, 700), 4, 4, 64),
    ((2048,), 16, 2, 128),
]


@pytest.mark.parametrize("ci", range(len(DENSE_CASES)))
def test_dense_backward(pk, ci):
    """The dense baseline's backward against the oracle's plain-attention
    backward (same bars; dout . out is formed from the bf16 output)."""
    import torch
    lens, hq, hkv, d = DENSE_CASES[ci]
    w = synth.small_workload(lens, hq, hkv, d, 1, 0.0, seed=5100 + ci)
    x = synth.make_inputs(w)
    dout = synth.make_dout(w, 2)
    dev = to_device(dict(x, dout=dout))
    prob = pk.Problem(dev["cu_seqlens"], hq, hkv, d, max(lens), cu_seqlens_host=x["cu_seqlens"])
    print(f"[dense bwd case{ci}] seqlens={lens} H={hq}/{hkv} d={d}", flush=True)
    out, lse = pk.logo_dense_causal_attn_fwd_train(prob, dev["q"], dev["k"], dev["v"])
    g = pk.logo_dense_causal_attn_bwd(prob, dev["q"], dev["k"], dev["v"], out, lse, dev["dout"])
    torch.cuda.synchronize()
    dout64 = synth.f32_from_bf16_bits(dout).reshape(dout.shape).astype(np.float64)
    ref = oracle.attn_bwd(x["q"], x["k"], x["v"], x["cu_seqlens"], 0, dout64)
    for nm in ("dq", "dk", "dv"):
        e = grad_err(g[nm].cpu().numpy(), ref[nm])
        print(f"[dense bwd case{ci}] {nm}: rel_l2={e['rel_l2']:.3g} rel_max={e['rel_max']:.3g}",
              flush=True)
        assert e["rel_l2"] <= REL_L2 and e["rel_max"] <= REL_MAX, (ci, nm, e)


SPARSE_CASES = [
    # (seqlens, Hq, Hkv, d, ratio)
    ((300, 1000), 8, 2, 128, 0.25),
    ((64, 700, 33), 4, 4, 64, 0.5),
    ((2048,), 8, 8, 128, 0.5),
    ((129, 5), 4, 1, 128, 0.0),
]


@pytest.mark.parametrize("ci", range(len(SPARSE_CASES)))
def test_sparse_global_backward(pk, ci):
    """The query-sparse global attention alone (training forward + backward)
    against the oracle's attention backward with dout zero on unselected
    rows (the operator's loss sees only the selected rows)."""
    import torch
    lens, hq, hkv, d, ratio = SPARSE_CASES[ci]
    w = synth.small_workload(lens, hq, hkv, d, 1, ratio, seed=5200 + ci)
    x = synth.make_inputs(w)
    dout = synth.make_dout(w, 3)
    thr = oracle.thresholds(x["gate"], x["cu_seqlens"], oracle.SEL_RATIO, ratio=ratio)
    sel = oracle.select(x["gate"], x["cu_seqlens"], thr)[0]
    n = sel.size
    dev = to_device(x)
    prob = pk.Problem(dev["cu_seqlens"], hq, hkv, d, max(lens), cu_seqlens_host=x["cu_seqlens"])
    cap = max(pk.logo_ratio_capacity(prob, ratio), 1)
    print(f"[sparse bwd case{ci}] seqlens={lens} H={hq}/{hkv} d={d} n_sel={n}", flush=True)
    sel_idx, cu_sel, _, _ = pk.logo_select(prob, dev["gate"], ratio=ratio, sel_capacity=cap)
    assert sel_idx[:n].cpu().numpy().tolist() == sel.tolist()
    o, lse = pk.logo_global_attn_sparse_q_fwd_train(prob, dev["q"], dev["k"], dev["v"], sel_idx,
                                                    cu_sel, cap)
    dc = np.zeros((cap,) + dout.shape[1:], np.uint16)
    dc[:n] = dout[sel]
    g = pk.logo_global_attn_sparse_q_bwd(prob, dev["q"], dev["k"], dev["v"], sel_idx, cu_sel,
                                         cap, o, lse, to_device(dict(d=dc))["d"])
    torch.cuda.synchronize()
    full = np.zeros(dout.shape)
    full[sel] = synth.f32_from_bf16_bits(dout[sel]).reshape((n,) + dout.shape[1:])
    ref = oracle.attn_bwd(x["q"], x["k"], x["v"], x["cu_seqlens"], 0, full)
    for nm in ("dq", "dk", "dv"):
        got = g[nm].cpu().numpy()
        if n == 0:
            assert not got.any(), (ci, nm)
            continue
        e = grad_err(got, ref[nm])
        print(f"[sparse bwd case{ci}] {nm}: rel_l2={e['rel_l2']:.3g} rel_max={e['rel_max']:.3g}",
              flush=True)
        assert e["rel_l2"] <= REL_L2 and e["rel_max"] <= REL_MAX, (ci, nm, e)
    unsel = np.setdiff1d(np.arange(w.total_tokens), sel)
    assert not g["dq"].cpu().numpy()[unsel].any()


def test_backward_deterministic(pk):
    """Two backward passes on the same inputs are bit-identical (no float
    atomics; fixed-order reductions)."""
    import torch
    w = synth.small_workload((700, 1500), 8, 2, 128, 200, 0.25, seed=5300)
    x = synth.make_inputs(w)
    dev = to_device(dict(x, dout=synth.make_dout(w, 4)))
    prob = pk.Problem(dev["cu_seqlens"], 8, 2, 128, 200, cu_seqlens_host=x["cu_seqlens"])
    saved = pk.logo_attn_fwd_train(prob, dev["q"], dev["k"], dev["v"], dev["gate"], ratio=0.25)
    g1 = pk.logo_attn_bwd(prob, dev["q"], dev["k"], dev["v"], dev["gate"], saved, dev["dout"])
    g2 = pk.logo_attn_bwd(prob, dev["q"], dev["k"], dev["v"], dev["gate"], saved, dev["dout"])
    torch.cuda.synchronize()
    for nm in g1:
        assert torch.equal(g1[nm], g2[nm]), nm


@pytest.mark.parametrize("name, n_sel_rows, n_uns_rows, n_keys",
                         [("T32k-gqa", 14, 20, 3), ("T128k-gqa", 4, 4, 0)])
def test_backward_full_size_sampled(pk, name, n_sel_rows, n_uns_rows, n_keys):
    """A full-size workload (T32k-gqa: 32768 tokens, 32/8 heads, d 128, w 1024,
    ratio 1/8, bursty gate; T128k-gqa: 131072 tokens, w 4096, ratio 1/16) in
    the launch configuration the benchmark times, checked against the oracle
    at sampled places: dq and dgate of query rows (selected and unselected,
    sequence edges, the latest selected rows) and dk / dv of keys near the
    sequence end (their gradient sums over every row that sees them), plus
    the key-gradient sum over all keys, which softmax shift invariance makes
    zero for each KV head."""
    import torch
    w = synth.WORKLOADS[name]
    x = synth.make_inputs(w)
    dout = synth.make_dout(w, 1)
    dev = to_device(dict(x, dout=dout))
    prob = pk.Problem(dev["cu_seqlens"], w.num_q_heads, w.num_kv_heads, w.head_dim, w.window,
                      cu_seqlens_host=x["cu_seqlens"])
    print(f"[bwd full] {name}", flush=True)
    saved = pk.logo_attn_fwd_train(prob, dev["q"], dev["k"], dev["v"], dev["gate"],
                                   ratio=w.ratio)
    g = pk.logo_attn_bwd(prob, dev["q"], dev["k"], dev["v"], dev["gate"], saved, dev["dout"])
    torch.cuda.synchronize()
    N = w.total_tokens
    t2s = saved["tok2sel"].cpu().numpy()
    sel = np.nonzero(t2s >= 0)[0]
    uns = np.nonzero(t2s < 0)[0]
    rng = np.random.default_rng(77)
    qrows = np.unique(np.concatenate([
        [0, 1, w.window - 1, w.window, N - 1], sel[:3], sel[-6:],
        rng.choice(sel, n_sel_rows, replace=False), rng.choice(uns, n_uns_rows, replace=False)]))
    keys = np.unique(np.concatenate([[N - 1, N - 2, N - 64, N - 65, N - 300][:2 + n_keys],
                                     rng.integers(N - 600, N, n_keys)]))
    d64 = synth.f32_from_bf16_bits(dout).reshape(dout.shape).astype(np.float64)
    ref = oracle.logo_bwd_sample(x, w.window, d64, qrows, keys, ratio=w.ratio)
    assert np.array_equal(ref["tok2sel"], t2s)
    for nm, idx in (("dq", qrows), ("dgate", qrows), ("dk", keys), ("dv", keys)):
        e = grad_err(g[nm].cpu().numpy()[idx], ref[nm])
        print(f"[bwd full] {nm}: rel_l2={e['rel_l2']:.3g} rel_max={e['rel_max']:.3g}", flush=True)
        assert e["rel_l2"] <= REL_L2 and e["rel_max"] <= REL_MAX, (nm, e)
    dk = g["dk"].double()
    rms = dk.pow(2).mean(dim=0).sqrt()                      # [Hkv, d]
    zero_sum = dk.sum(dim=0).abs() / (rms * math.sqrt(N))
    print(f"[bwd full] key-gradient sum / (sqrt(N) rms): max {float(zero_sum.max()):.3g}",
          flush=True)
    assert float(zero_sum.max()) <= 0.05
