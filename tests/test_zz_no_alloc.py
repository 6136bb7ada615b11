"""The allocation-free decoding step (logo_decode_noalloc, through the C ABI)
against logo_decode on the same inputs: two calls in a row on one GPU, the
second with a smaller problem, so the second reuses the scratch array the
first filled.  Both entry points run the same kernels with the same
arithmetic, so outputs, the selected list and its count must agree bit for
bit; the first call is also held to the layer bar against the fp64 oracle."""
import numpy as np
import pytest

import oracle
import synth
from _support import err_stats, to_device, torch_bf16_to_f64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pk():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible: the gpu tests need an MI355X")
    import paper_2608_29539_amd as pk
    pk.library()
    oracle.build(force=False)
    return pk


def _case(pk, w, threshold, lists_given: bool, tag: str):
    import torch
    x = synth.make_decode_inputs(w)
    dev = to_device(x)
    prob = pk.Problem(dev["cu_seqlens"], w.num_q_heads, w.num_kv_heads, w.head_dim, w.window,
                      cu_seqlens_host=x["cu_seqlens"])
    B = len(w.seqlens)
    print(f"[noalloc {tag}] B={B} caches={list(w.seqlens)} Hq={w.num_q_heads} "
          f"Hkv={w.num_kv_heads} d={w.head_dim} w={w.window}", flush=True)
    ref_out, ref_act, ref_n = pk.logo_decode(prob, dev["q"], dev["k"], dev["v"], dev["gate"],
                                             threshold=threshold)
    out = torch.empty((B, w.num_q_heads, w.head_dim), dtype=torch.bfloat16, device="cuda")
    act = torch.full((B,), -7, dtype=torch.int32, device="cuda") if lists_given else None
    n_act = torch.full((1,), -7, dtype=torch.int32, device="cuda") if lists_given else None
    got, act, n_act = pk.logo_decode_noalloc(prob, dev["q"], dev["k"], dev["v"], dev["gate"],
                                             out, threshold=threshold, active=act,
                                             n_active=n_act)
    torch.cuda.synchronize()
    assert torch.equal(got.view(torch.int16), ref_out.view(torch.int16)), tag
    n = int(ref_n.cpu()[0])
    if lists_given:
        assert int(n_act.cpu()[0]) == n, tag
        assert act.cpu().tolist()[:n] == ref_act.cpu().tolist()[:n], tag
    ref = oracle.decode(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], w.window, threshold)
    st = err_stats(torch_bf16_to_f64(got), ref["out"])
    print(f"[noalloc {tag}] n_active={n} " + " ".join(f"{k}={v:.3g}" for k, v in st.items()),
          flush=True)
    assert st["max_abs"] <= 2e-2 and st["mean_abs"] <= 2e-3, (tag, st)


def test_noalloc_matches_decode_two_calls(pk):
    big = synth.small_workload((4000, 1, 777, 2048, 65, 3000, 1500), 8, 2, 128, 256, 0.5,
                               seed=2101)
    small = synth.small_workload((300, 17, 129), 4, 4, 64, 32, 0.5, seed=2102)
    _case(pk, big, 0.5, True, "first")
    _case(pk, small, 0.3, False, "second, smaller")
