"""GPU parity of one decoding step (Sec. 3.3 and App. B, Autoregressive
Decoding): logo_decode through the C ABI against the fp64 oracle's decode.

Bars: the selected-sequence list and its count bit-exact; the bf16 output
within max-abs 2e-2 and mean-abs 2e-3 of the oracle (the layer's bar).  Every
element is compared, including the 16 x 32K-token GQA decoding workload.
"""
import math

import numpy as np
import pytest

import oracle
import synth
from _support import err_stats, to_device, torch_bf16_to_f64

pytestmark = pytest.mark.gpu

MAX_ABS, MEAN_ABS = 2e-2, 2e-3


@pytest.fixture(scope="module")
def pk():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible: the gpu tests need an MI355X")
    import paper_2608_29539_amd as pk
    pk.library()
    oracle.build(force=False)
    return pk


def run_case(pk, w, threshold, *, distinct=False, gains=False, gate=None, tag=""):
    import torch
    x = synth.make_decode_inputs(w, distinct_global=distinct)
    if gate is not None:
        x["gate"] = np.asarray(gate, np.float32)
    rng = np.random.default_rng(w.seed)
    gl = rng.uniform(0.5, 1.5, (w.num_q_heads, w.head_dim)).astype(np.float32) if gains else None
    gg = rng.uniform(0.5, 1.5, (w.num_q_heads, w.head_dim)).astype(np.float32) if gains else None
    dev = to_device(x)
    prob = pk.Problem(dev["cu_seqlens"], w.num_q_heads, w.num_kv_heads, w.head_dim, w.window,
                      cu_seqlens_host=x["cu_seqlens"])
    dgl = torch.from_numpy(gl).cuda() if gains else None
    dgg = torch.from_numpy(gg).cuda() if gains else None
    out, active, n_active = pk.logo_decode(prob, dev["q"], dev["k"], dev["v"], dev["gate"],
                                           threshold=threshold, q_g=dev.get("q_g"),
                                           k_g=dev.get("k_g"), v_g=dev.get("v_g"),
                                           gain_local=dgl, gain_global=dgg)
    torch.cuda.synchronize()
    ref = oracle.decode(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], w.window, threshold,
                        q_g_new=x.get("q_g"), k_g=x.get("k_g"), v_g=x.get("v_g"),
                        gain_local=gl, gain_global=gg)
    n = int(n_active.cpu()[0])
    assert n == ref["n_sel"], (tag, n, ref["n_sel"])
    assert active.cpu().numpy()[:n].tolist() == np.nonzero(ref["z"])[0].tolist(), tag
    st = err_stats(torch_bf16_to_f64(out), ref["out"])
    print(f"[decode {tag}] n_active={n} " + " ".join(f"{k}={v:.3g}" for k, v in st.items()),
          flush=True)
    assert st["max_abs"] <= MAX_ABS and st["mean_abs"] <= MEAN_ABS, (tag, st)
    return out, ref


DECODE_CASES = [
    # (cache lengths, Hq, Hkv, d, window, threshold, distinct global tensors, gains)
    ((1, 7, 300, 1000, 2500), 8, 2, 128, 257, 0.5, False, False),
    ((64, 65, 4097), 4, 4, 64, 64, 0.3, True, True),
    ((513, 2048), 16, 2, 128, 1, 0.6, False, False),
    ((3000, 3000, 3000), 6, 2, 64, 5000, 0.2, False, True),
    ((700, 1, 40000), 8, 8, 128, 512, 0.4, True, False),
    ((1000, 2000, 255, 256, 257), 8, 2, 128, 128, -math.inf, False, False),
    ((1000, 2000), 8, 2, 128, 128, math.inf, False, False),
    # group sizes 2 and 4 at d 64 and group size 2 at d 128 (GH = 2, 4, 2)
    ((333, 1500, 70), 8, 4, 64, 200, 0.4, False, True),
    ((2049, 5), 4, 1, 64, 1024, 0.1, True, False),
    ((800, 4000), 4, 2, 128, 300, 0.05, False, False),
]


@pytest.mark.parametrize("ci", range(len(DECODE_CASES)))
def test_decode_small(pk, ci):
    lens, hq, hkv, d, win, thr, distinct, gains = DECODE_CASES[ci]
    w = synth.small_workload(lens, hq, hkv, d, win, 0.0, seed=3000 + ci)
    run_case(pk, w, thr, distinct=distinct, gains=gains, tag=f"case{ci}")


def _decode_sweep_cases(n=24, seed=6161):
    """Seeded random decoding steps: 1-12 caches of 1 to 9000 tokens (tile
    edges included), each G in {1, 2, 4, 8} with each d in {64, 128} three
    times, 1-8 KV heads, windows from 1 to beyond the cache, thresholds from
    -inf to +inf, distinct global tensors and gains drawn at random."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        B = int(rng.integers(1, 13))
        lens = tuple(int(t) for t in rng.choice([1, 2, 63, 64, 65, 255, 256, 257, 1000, 4097,
                                                 9000], size=B))
        hkv = int(rng.choice([1, 2, 4, 8]))
        G = (1, 2, 4, 8)[i % 4]
        if hkv * G > 32:
            hkv = 32 // G
        d = (64, 128)[(i // 4) % 2]
        win = int(rng.choice([1, 16, 64, 257, 1024, 5000]))
        thr = float(rng.choice([-math.inf, 0.1, 0.5, 0.9, math.inf]))
        cases.append((lens, hkv * G, hkv, d, win, thr, bool(rng.random() < 0.5),
                      bool(rng.random() < 0.5)))
    return cases


DECODE_SWEEP = _decode_sweep_cases()


@pytest.mark.parametrize("ci", range(len(DECODE_SWEEP)),
                         ids=[f"B{len(c[0])}_h{c[1]}-{c[2]}_d{c[3]}_w{c[4]}_thr{c[5]}"
                              f"{'_distinct' if c[6] else ''}{'_gains' if c[7] else ''}"
                              for c in DECODE_SWEEP])
def test_decode_random_sweep(pk, ci):
    lens, hq, hkv, d, win, thr, distinct, gains = DECODE_SWEEP[ci]
    w = synth.small_workload(lens, hq, hkv, d, win, 0.0, seed=3300 + ci)
    run_case(pk, w, thr, distinct=distinct, gains=gains, tag=f"sweep{ci}")


def test_decode_gate_edges(pk):
    """NaN gates are never selected, a gate equal to the threshold stays local,
    and -0 / +0 compare equal."""
    w = synth.small_workload((100, 200, 300, 400, 500, 600), 8, 2, 128, 64, 0.0, seed=3100)
    gate = [float("nan"), 0.5, 0.5000001, 0.25, -0.0, 0.75]
    _, ref = run_case(pk, w, 0.5, gate=gate, tag="edges")
    assert ref["z"].tolist() == [False, False, True, False, False, True]
    _, ref0 = run_case(pk, w, 0.0, gate=gate, tag="zero-threshold")
    assert ref0["z"].tolist() == [False, True, True, True, False, True]


def test_decode_device_threshold_matches_host(pk):
    import torch
    w = synth.small_workload((900, 3000, 77), 8, 2, 128, 256, 0.0, seed=3200)
    x = synth.make_decode_inputs(w)
    dev = to_device(x)
    prob = pk.Problem(dev["cu_seqlens"], 8, 2, 128, 256, cu_seqlens_host=x["cu_seqlens"])
    thr = float(np.sort(x["gate"])[1])
    a, act_a, n_a = pk.logo_decode(prob, dev["q"], dev["k"], dev["v"], dev["gate"], threshold=thr)
    t = torch.tensor([thr], dtype=torch.float32, device="cuda")
    b, act_b, n_b = pk.logo_decode(prob, dev["q"], dev["k"], dev["v"], dev["gate"],
                                   threshold_device=t)
    torch.cuda.synchronize()
    assert int(n_a.cpu()[0]) == int(n_b.cpu()[0]) == 1
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_decode_workload_full(pk):
    """The 16 x 32K-token GQA decoding workload, every output element."""
    w = synth.DECODE_WORKLOADS["decode-B16-32k-gqa"]
    run_case(pk, w, 1.0 - w.ratio, tag=w.name)


def test_decode_deterministic(pk):
    import torch
    w = synth.small_workload((5000, 3000), 8, 2, 128, 512, 0.0, seed=3300)
    x = synth.make_decode_inputs(w)
    dev = to_device(x)
    prob = pk.Problem(dev["cu_seqlens"], 8, 2, 128, 512, cu_seqlens_host=x["cu_seqlens"])
    a = pk.logo_decode(prob, dev["q"], dev["k"], dev["v"], dev["gate"], threshold=0.0)[0].clone()
    b = pk.logo_decode(prob, dev["q"], dev["k"], dev["v"], dev["gate"], threshold=0.0)[0]
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
