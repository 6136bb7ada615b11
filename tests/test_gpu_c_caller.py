"""The layer driven from a plain C program (tests/c/layer_from_c.c): device
memory from the HIP runtime, one logo_attn_fwd call in ratio mode, no Python
or torch in that process.  Its selection must equal the oracle's bit for bit
and its bf16 output must meet the layer bar (max-abs 2e-2, mean-abs 2e-3)
against the fp64 oracle layer."""
import os
import subprocess

import numpy as np
import pytest

import oracle
import synth
from _support import err_stats

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BIN = os.path.join(ROOT, "tests", "c", "layer_from_c.bin")

CASES = [
    # (seqlens, Hq, Hkv, d, window, ratio)
    ((1000, 333), 8, 2, 128, 100, 0.3),
    ((2500,), 16, 4, 128, 1024, 0.125),
    ((64, 0, 777), 4, 4, 64, 65, 0.5),
]


def _write_inputs(path, w, x, ratio):
    B, N = len(w.seqlens), w.total_tokens
    with open(path, "wb") as f:
        np.array([B, N, w.num_q_heads, w.num_kv_heads, w.head_dim, w.window, w.max_seqlen, 0],
                 dtype="<i4").tofile(f)
        np.array([ratio], dtype="<f8").tofile(f)
        x["cu_seqlens"].astype("<i4").tofile(f)
        for k in ("q", "k", "v"):
            np.ascontiguousarray(x[k]).astype("<u2").tofile(f)
        x["gate"].astype("<f4").tofile(f)


@pytest.mark.parametrize("ci", range(len(CASES)))
def test_layer_from_c_program(ci, tmp_path):
    if not os.path.exists(BIN):
        pytest.fail("tests/c/layer_from_c.bin is not built (run __graft_entry__.build())")
    seqlens, hq, hkv, d, win, ratio = CASES[ci]
    w = synth.small_workload(seqlens, hq, hkv, d, win, ratio, seed=9100 + ci)
    x = synth.make_inputs(w)
    inp, outp = str(tmp_path / "in.bin"), str(tmp_path / "out.bin")
    _write_inputs(inp, w, x, ratio)
    print(f"[c caller {ci}] T={seqlens} Hq={hq} Hkv={hkv} d={d} w={win} ratio={ratio}",
          flush=True)
    r = subprocess.run([BIN, inp, outp], capture_output=True, text=True, timeout=120)
    print(r.stdout + r.stderr, flush=True)
    assert r.returncode == 0, r.stderr

    B, N = len(seqlens), w.total_tokens
    raw = np.fromfile(outp, dtype=np.uint8)
    cu_sel = raw[: 4 * (B + 1)].view("<i4")
    cap = int(raw[4 * (B + 1): 4 * (B + 2)].view("<i4")[0])
    o = 4 * (B + 2)
    sel = raw[o: o + 4 * cap].view("<i4")
    out_bits = raw[o + 4 * cap:].view("<u2")
    assert out_bits.size == N * hq * d

    ethr = oracle.thresholds(x["gate"], x["cu_seqlens"], oracle.SEL_RATIO, ratio=ratio)
    esel, ecu, _ = oracle.select(x["gate"], x["cu_seqlens"], ethr)
    n = int(ecu[-1])
    assert cu_sel.tolist() == ecu.tolist()
    assert sel[:n].tolist() == esel.tolist()
    ref = oracle.logo_fwd(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], win, ratio=ratio)
    got = synth.f32_from_bf16_bits(out_bits).reshape(N, hq, d).astype(np.float64)
    st = err_stats(got, ref["out"])
    print(f"[c caller {ci}] n_sel={n} " + " ".join(f"{k}={v:.3g}" for k, v in st.items()),
          flush=True)
    assert st["max_abs"] <= 2e-2 and st["mean_abs"] <= 2e-3
