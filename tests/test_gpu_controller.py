"""GPU parity of the global-budget controller (Sec. 3.2, Eq. threshold-update;
Sec. 3.1, Eq. realized-ratio; the P-mask paragraph) and of the selection
mode that reads the controller's threshold on the device.  Everything here is
integer or a single fp32 add, so the bar is bit-exact against the oracle."""
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


def f32_bits(x):
    return np.array([x], np.float32).view(np.uint32)[0]


def _prob(pk, seqlens, hq=4, hkv=4, d=64, w=16):
    import torch
    cu = np.zeros(len(seqlens) + 1, np.int32)
    cu[1:] = np.cumsum(seqlens)
    return pk.Problem(torch.from_numpy(cu).cuda(), hq, hkv, d, w, cu_seqlens_host=cu), cu


@pytest.mark.parametrize("case", [
    # (seqlens, per-sequence selected counts, rho, gamma, b_th)
    ((8,), (3,), 0.25, 0.125, 0.25),          # F > rho: up
    ((8,), (1,), 0.25, 0.125, 0.25),          # F < rho: down
    ((8,), (2,), 0.25, 0.125, 0.25),          # F == rho: unchanged
    ((1000, 0, 24), (100, 0, 3), 0.1, 0.01, 0.6180339),
    ((4096,), (4096,), 0.5, 2.0 ** -10, -0.5),
    ((5, 7, 11), (0, 0, 0), 0.0, 0.3, 0.1),   # F == rho == 0
    ((5, 7, 11), (5, 7, 11), 1.0, 0.3, 0.9),  # F == rho == 1
])
def test_budget_update_matches_oracle(pk, case):
    import torch
    seqlens, counts, rho, gamma, b0 = case
    prob, cu = _prob(pk, seqlens)
    cu_sel = np.zeros(len(seqlens) + 1, np.int32)
    cu_sel[1:] = np.cumsum(counts)
    b = torch.tensor([b0], dtype=torch.float32, device="cuda")
    realized = torch.empty(1, dtype=torch.float32, device="cuda")
    pk.logo_budget_update(prob, torch.from_numpy(cu_sel).cuda(), rho, gamma, b, realized)
    torch.cuda.synchronize()
    n, N = int(cu_sel[-1]), int(cu[-1])
    exp_b = oracle.budget_update(np.float32(b0), n, N, rho, gamma)
    assert f32_bits(float(b.cpu()[0])) == f32_bits(exp_b)
    assert f32_bits(float(realized.cpu()[0])) == f32_bits(oracle.realized_ratio(n, N))


def test_pmask_initial_threshold_host(pk):
    for gamma, S in ((2.0 ** -10, 1024), (1e-3, 700), (0.05, 3), (0.0, 100)):
        assert f32_bits(pk.logo_pmask_initial_threshold(gamma, S)) == \
            f32_bits(oracle.pmask_initial_threshold(gamma, S))


@pytest.mark.parametrize("seqlens", [(1000,), (700, 0, 333, 64)])
@pytest.mark.parametrize("b_th", [0.5, 0.0, -0.0, 0.999, float("inf"), float("-inf")])
def test_device_threshold_selection_equals_host(pk, seqlens, b_th):
    import torch
    prob, cu = _prob(pk, seqlens)
    rng = np.random.default_rng(31)
    N = int(cu[-1])
    gate = rng.uniform(0, 1, N).astype(np.float32)
    gate[::97] = 0.5                              # ties at the threshold
    g = torch.from_numpy(gate).cuda()
    h = pk.logo_select(prob, g, threshold=b_th)
    dev_thr = torch.full((len(seqlens),), float("nan"), dtype=torch.float32, device="cuda")
    dev_thr[0] = b_th
    d = pk.logo_select(prob, g, threshold_device=dev_thr)
    torch.cuda.synchronize()
    n = int(h[1][-1])
    assert d[1].cpu().tolist() == h[1].cpu().tolist()
    assert d[0].cpu()[:n].tolist() == h[0].cpu()[:n].tolist()
    assert d[2].cpu().tolist() == h[2].cpu().tolist()
    assert d[3].cpu().view(torch.int32).tolist() == h[3].cpu().view(torch.int32).tolist()


def test_device_threshold_nan_selects_nothing(pk):
    import torch
    prob, cu = _prob(pk, (300, 200))
    gate = torch.rand(500, dtype=torch.float32, device="cuda")
    for nan_bits in (0x7FC00000, 0xFFC00000):     # positive and negative quiet NaN
        thr = torch.tensor(np.array([nan_bits, 0], np.uint32).view(np.float32)).cuda()
        _, cu_sel, t2s, _ = pk.logo_select(prob, gate, threshold_device=thr)
        torch.cuda.synchronize()
        assert cu_sel.cpu().tolist() == [0, 0, 0]
        assert (t2s.cpu() == -1).all()


def test_controller_loop_matches_oracle(pk):
    """Selection with the device threshold, then the controller step, 120
    times from the P-mask start: the threshold trajectory is bit-identical
    to the oracle's (the first 64 steps are the P-mask phase)."""
    import torch
    seqlens = (3000, 1096)
    prob, cu = _prob(pk, seqlens)
    rng = np.random.default_rng(7)
    N = int(cu[-1])
    gate = rng.uniform(0, 1, N).astype(np.float32)
    g = torch.from_numpy(gate).cuda()
    rho, gamma, S = 0.2, 2.0 ** -7, 64
    b0 = oracle.pmask_initial_threshold(gamma, S)
    b_dev = torch.tensor([b0, 0.0], dtype=torch.float32, device="cuda")
    b = np.float32(b0)
    traj_dev, traj_ref = [], []
    for step in range(120):
        _, cu_sel, _, _ = pk.logo_select(prob, g, threshold_device=b_dev)
        pk.logo_budget_update(prob, cu_sel, rho, gamma, b_dev)
        thr = oracle.thresholds(gate, cu, oracle.SEL_THRESHOLD, threshold=float(b))
        _, ecu, _ = oracle.select(gate, cu, thr)
        b = np.float32(oracle.budget_update(float(b), int(ecu[-1]), N, rho, gamma))
        traj_ref.append(f32_bits(b))
        traj_dev.append(f32_bits(float(b_dev.cpu()[0])))
    assert traj_dev == traj_ref
    # settled near the rho-quantile of the gates
    assert abs(float(b) - np.quantile(gate, 1 - rho)) <= 2 * gamma


def test_layer_with_device_threshold_equals_host(pk):
    import torch
    w = synth.small_workload((900, 400), 8, 2, 128, 96, 0.25, seed=2100)
    x = synth.make_inputs(w)
    dev = to_device(x)
    prob = pk.Problem(dev["cu_seqlens"], 8, 2, 128, 96, cu_seqlens_host=x["cu_seqlens"])
    a = pk.logo_attn_fwd(prob, dev["q"], dev["k"], dev["v"], dev["gate"], threshold=0.625)
    thr = torch.tensor([0.625, 0.0], dtype=torch.float32, device="cuda")
    b = pk.logo_attn_fwd(prob, dev["q"], dev["k"], dev["v"], dev["gate"], threshold_device=thr)
    torch.cuda.synchronize()
    assert torch.equal(a[0].view(torch.int16), b[0].view(torch.int16))
    assert a[2].cpu().tolist() == b[2].cpu().tolist()
    ref = oracle.logo_fwd(x["q"], x["k"], x["v"], x["gate"], x["cu_seqlens"], 96, threshold=0.625)
    st = err_stats(torch_bf16_to_f64(b[0]), ref["out"])
    assert st["max_abs"] <= 2e-2 and st["mean_abs"] <= 2e-3
