"""CPU checks of the seeded input generators (`synth`), which both the oracle
and the HIP path take their inputs from: the bursty gate's chain statistics,
empty sequences, bf16 draws, determinism, and that the gate-only draw gives
the same bytes as the full draw."""
import numpy as np
import pytest

import synth


def test_markov_burst_statistics():
    """The bursty gate of the T32k workload: stationary on-fraction 1/8 and
    mean on-run length 8 (so mean off-run 56), values in the upper half of
    [0, 1] exactly on the on tokens."""
    rng = np.random.default_rng(123)
    T = 2_000_000
    g = synth.markov_burst_gate(rng, T, p_stay_on=1.0 - 1.0 / 8, p_turn_on=1.0 / 56,
                                pi_on=1.0 / 8)
    on = g >= 0.5
    frac = on.mean()
    assert abs(frac - 1.0 / 8) < 0.01, frac
    # run lengths of the on state
    d = np.diff(np.concatenate([[0], on.astype(np.int8), [0]]))
    starts, ends = np.nonzero(d == 1)[0], np.nonzero(d == -1)[0]
    runs = ends - starts
    assert abs(runs.mean() - 8.0) < 0.2, runs.mean()
    assert g.dtype == np.float32 and g.min() >= 0.0 and g.max() < 1.0


@pytest.mark.parametrize("kind", ["uniform", "logit_normal", "markov_burst"])
def test_gate_kinds_take_empty_sequences(kind):
    w = synth.small_workload((0, 5, 0, 3, 0), 4, 4, 64, 16, 0.25, seed=77, gate=kind)
    x = synth.make_gate_only(w)
    assert x["gate"].shape == (8,) and x["gate"].dtype == np.float32
    assert x["cu_seqlens"].tolist() == [0, 0, 5, 5, 8, 8]
    assert np.all((x["gate"] >= 0) & (x["gate"] <= 1))


def test_draws_are_seeded_and_gate_only_matches():
    w = synth.small_workload((300, 0, 129), 8, 2, 64, 32, 0.25, seed=4321, gate="markov_burst")
    a = synth.make_inputs(w)
    b = synth.make_inputs(w)
    for k in ("q", "k", "v", "gate", "cu_seqlens"):
        assert np.array_equal(a[k], b[k]), k
    g = synth.make_gate_only(w)
    assert np.array_equal(g["gate"], a["gate"])
    assert np.array_equal(g["cu_seqlens"], a["cu_seqlens"])
    other = synth.make_inputs(synth.small_workload((300, 0, 129), 8, 2, 64, 32, 0.25, seed=4322,
                                                   gate="markov_burst"))
    assert not np.array_equal(other["q"], a["q"])


def test_bf16_normal_draws():
    """Q/K/V are N(0, scale^2) rounded to bf16: the bits widen to float32
    exactly, with the moments of the draw."""
    w = synth.small_workload((4096,), 4, 4, 128, 16, 0.25, seed=99)
    x = synth.make_inputs(w)
    q = synth.f32_from_bf16_bits(x["q"].reshape(-1)).astype(np.float64)
    assert x["q"].dtype == np.uint16 and x["q"].shape == (4096, 4, 128)
    assert abs(q.mean()) < 0.01 and abs(q.std() - 1.0) < 0.01
    w2 = synth.small_workload((4096,), 4, 4, 64, 16, 0.25, seed=99, qkv_scale=1.0 / 8.0)
    q2 = synth.f32_from_bf16_bits(synth.make_inputs(w2)["q"].reshape(-1)).astype(np.float64)
    assert abs(q2.std() - 1.0 / 8.0) < 0.002
    # rounding to bf16 is to nearest: re-rounding the widened values is exact
    assert np.array_equal(synth.bf16_bits_from_f32(q.astype(np.float32)), x["q"].reshape(-1))
