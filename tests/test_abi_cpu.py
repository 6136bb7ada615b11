"""C ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and rejects every invalid argument with its documented
status before launching anything (no call here reaches a kernel launch)."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "logo.h")

OK, ERR_NULL, ERR_SHAPE, ERR_UNSUPPORTED, ERR_ARG, ERR_WORKSPACE, ERR_HIP, ERR_SCRATCH_LIMIT = \
    range(8)


@pytest.fixture(scope="module")
def lib():
    import paper_2608_29539_amd as pk
    if not os.path.exists(pk.library_path()):
        from paper_2608_29539_amd.build import build_library
        build_library()
    return pk.library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(logo_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert "logo_attn_fwd" in names and len(names) >= 10
    for n in names:
        assert hasattr(lib, n), f"liblogo.so does not export {n}"


def test_status_strings_and_version(lib):
    import paper_2608_29539_amd as pk
    assert pk.logo_status_str(0) == "LOGO_OK"
    assert pk.logo_status_str(5) == "LOGO_ERR_WORKSPACE"
    assert pk.logo_status_str(7) == "LOGO_ERR_SCRATCH_LIMIT"
    assert pk.logo_version().count(".") == 2


class Prob:
    """A logo_problem whose cu_seqlens points at HOST memory: validation never
    dereferences the device pointer, so this is safe for argument checks."""

    def __init__(self, seqlens=(100, 50), hq=8, hkv=2, d=128, window=16, scale=0.0,
                 host=True, max_seqlen=None):
        import paper_2608_29539_amd.binding as b
        cu = np.zeros(len(seqlens) + 1, np.int32)
        cu[1:] = np.cumsum(seqlens)
        self.cu = cu
        self.s = b._Problem(len(seqlens), int(cu[-1]),
                            int(max(seqlens)) if max_seqlen is None else max_seqlen,
                            cu.ctypes.data_as(ctypes.c_void_p),
                            cu.ctypes.data_as(ctypes.c_void_p) if host else None,
                            hq, hkv, d, window, scale)

    @property
    def c(self):
        return ctypes.byref(self.s)


FAKE = ctypes.c_void_p(0x1000)   # never dereferenced: every call below fails validation


def test_problem_validation(lib):
    def local(p):
        return lib.logo_local_attn(p.c, FAKE, FAKE, FAKE, FAKE, None)

    assert lib.logo_local_attn(None, FAKE, FAKE, FAKE, FAKE, None) == ERR_NULL
    p = Prob()
    p.s.cu_seqlens = None
    assert local(p) == ERR_NULL
    assert local(Prob(hq=6, hkv=4)) == ERR_SHAPE
    assert local(Prob(hq=0)) == ERR_SHAPE
    assert local(Prob(d=96)) == ERR_UNSUPPORTED
    assert local(Prob(d=256)) == ERR_UNSUPPORTED
    assert local(Prob(window=0)) == ERR_ARG
    assert local(Prob(scale=float("nan"))) == ERR_ARG
    assert local(Prob(max_seqlen=60)) == ERR_SHAPE          # host copy shows T = 100
    p = Prob()
    p.s.total_tokens = 149                                  # cu[B] = 150
    assert local(p) == ERR_SHAPE
    p = Prob()
    p.s.num_seqs = 0
    assert local(p) == ERR_SHAPE
    p = Prob()
    assert lib.logo_local_attn(p.c, None, FAKE, FAKE, FAKE, None) == ERR_NULL


def test_fwd_launches_rejects_invalid_problems(lib):
    """logo_attn_fwd_launches validates the problem before any device query:
    -1 for a NULL or invalid problem (the plan itself needs the GPU's CU
    count and is checked in the GPU suite)."""
    assert lib.logo_attn_fwd_launches(None) == -1
    assert lib.logo_attn_fwd_launches(Prob(hq=6, hkv=4).c) == -1
    assert lib.logo_attn_fwd_launches(Prob(d=96).c) == -1
    assert lib.logo_attn_fwd_launches(Prob(window=0).c) == -1


def test_select_validation(lib):
    p = Prob()
    ws_need = lib.logo_workspace_bytes(p.c, 0, 0)
    assert ws_need > 0

    def sel(mode=1, thr=0.0, ratio=0.25, sel_idx=FAKE, cap=150, cu_sel=FAKE, ws=FAKE,
            ws_bytes=None, gate=FAKE):
        return lib.logo_select(p.c, gate, mode, thr, ratio, sel_idx, cap, cu_sel, None, None, ws,
                               ws_need if ws_bytes is None else ws_bytes, None)

    assert sel(gate=None) == ERR_NULL
    assert sel(cu_sel=None) == ERR_NULL
    assert sel(sel_idx=None) == ERR_NULL
    assert sel(ratio=-0.1) == ERR_ARG
    assert sel(ratio=1.5) == ERR_ARG
    assert sel(ratio=float("nan")) == ERR_ARG
    assert sel(mode=0, thr=float("nan")) == ERR_ARG
    assert sel(mode=7) == ERR_ARG
    assert sel(cap=-1) == ERR_SHAPE
    # ratio 0.25 of (100, 50) needs floor(25) + floor(12.5) = 37 rows
    assert lib.logo_ratio_capacity(p.c, 0.25) == 37
    assert sel(cap=36) == ERR_SHAPE
    assert sel(ws=None) == ERR_WORKSPACE
    assert sel(ws_bytes=ws_need - 1) == ERR_WORKSPACE
    assert sel(ws=ctypes.c_void_p(0x1008)) == ERR_WORKSPACE   # misaligned
    # without a host copy the bound is N
    q = Prob(host=False)
    assert lib.logo_ratio_capacity(q.c, 0.25) == 150
    assert lib.logo_select(q.c, FAKE, 1, 0.0, 0.25, FAKE, 149, FAKE, None, None, FAKE,
                           ws_need, None) == ERR_SHAPE


def test_global_combine_fwd_validation(lib):
    p = Prob()
    need = lib.logo_workspace_bytes(p.c, 2, 64)
    assert need > 0
    g = lib.logo_global_attn_sparse_q
    assert g(p.c, FAKE, FAKE, FAKE, FAKE, FAKE, -1, FAKE, FAKE, need, None) == ERR_SHAPE
    assert g(p.c, FAKE, FAKE, FAKE, FAKE, None, 64, FAKE, FAKE, need, None) == ERR_NULL
    assert g(p.c, FAKE, FAKE, FAKE, None, FAKE, 64, FAKE, FAKE, need, None) == ERR_NULL
    assert g(p.c, FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, FAKE, need - 1, None) == ERR_WORKSPACE
    c = lib.logo_combine
    assert c(p.c, FAKE, FAKE, FAKE, FAKE, None, None, ctypes.c_float(-1.0), 1, FAKE,
             None) == ERR_ARG
    assert c(p.c, None, FAKE, FAKE, FAKE, None, None, ctypes.c_float(1e-6), 1, FAKE,
             None) == ERR_NULL
    f = lib.logo_attn_fwd
    need_f = lib.logo_workspace_bytes(p.c, 4, 150)
    args = [p.c, FAKE, FAKE, FAKE, None, None, None, FAKE, 1, 0.0, 0.25, None, None, 1e-6, FAKE,
            FAKE, 150, FAKE, FAKE, FAKE, FAKE, need_f, None]
    bad = list(args)
    bad[1] = None
    assert f(*bad) == ERR_NULL
    bad = list(args)
    bad[10] = 2.0
    assert f(*bad) == ERR_ARG
    bad = list(args)
    bad[21] = need_f - 1
    assert f(*bad) == ERR_WORKSPACE
    bad = list(args)
    bad[13] = float("inf")
    assert f(*bad) == ERR_ARG
    # the profiled entry: the five events are required, then the same checks
    fp = lib.logo_attn_fwd_profiled
    assert fp(*args, None) == ERR_NULL
    ev = (ctypes.c_void_p * 5)(*([FAKE.value] * 4 + [None]))
    assert fp(*args, ev) == ERR_NULL
    ev = (ctypes.c_void_p * 5)(*([FAKE.value] * 5))
    bad = list(args)
    bad[1] = None
    assert fp(*bad, ev) == ERR_NULL
    bad = list(args)
    bad[21] = need_f - 1
    assert fp(*bad, ev) == ERR_WORKSPACE
    d = lib.logo_dense_causal_attn
    assert d(Prob(d=32).c, FAKE, FAKE, FAKE, FAKE, None) == ERR_UNSUPPORTED
    assert d(p.c, FAKE, None, FAKE, FAKE, None) == ERR_NULL


def test_workspace_sizes(lib):
    p = Prob(seqlens=(32768,), hq=32, hkv=8, d=128, window=1024)
    fwd = lib.logo_workspace_bytes(p.c, 4, 4096)
    # the compact fp32 (1-p) Norm^L rows of the selected tokens dominate;
    # no full-size fp32 branch buffer is needed by the fused path
    assert 4096 * 32 * 128 * 4 <= fwd < 32768 * 32 * 128 * 4
    assert lib.logo_workspace_bytes(p.c, 1, 0) == 0
    assert lib.logo_workspace_bytes(p.c, 5, 0) == 0
    assert lib.logo_workspace_bytes(p.c, 2, 4096) % 256 == 0
    bad = Prob(d=48)
    assert lib.logo_workspace_bytes(bad.c, 4, 10) == 0


def test_budget_controller_validation(lib):
    p = Prob()
    f = lib.logo_budget_update          # argument types set by the binding
    assert f(None, FAKE, 0.5, 0.1, FAKE, None, None) == ERR_NULL
    assert f(p.c, None, 0.5, 0.1, FAKE, None, None) == ERR_NULL
    assert f(p.c, FAKE, 0.5, 0.1, None, None, None) == ERR_NULL
    assert f(p.c, FAKE, 1.5, 0.1, FAKE, None, None) == ERR_ARG
    assert f(p.c, FAKE, float("nan"), 0.1, FAKE, None, None) == ERR_ARG
    assert f(p.c, FAKE, 0.5, -0.1, FAKE, None, None) == ERR_ARG
    assert f(p.c, FAKE, 0.5, float("inf"), FAKE, None, None) == ERR_ARG
    g = lib.logo_pmask_initial_threshold
    assert g(2.0 ** -10, 1024) == -0.5
    assert g(0.25, 0) == 0.5
    # the value App. C prints for gamma = 0.0005 and S = 5000 steps
    assert g(0.0005, 5000) == -2.0


def test_device_threshold_mode_needs_thr_out(lib):
    p = Prob()
    ws_need = lib.logo_workspace_bytes(p.c, 0, 0)
    assert lib.logo_select(p.c, FAKE, 2, 0.0, 0.0, FAKE, 150, FAKE, None, None, FAKE, ws_need,
                           None) == ERR_NULL


def test_decode_noalloc_validation(lib):
    """logo_decode_noalloc checks its arguments as logo_decode does, and
    refuses a step whose scratch exceeds the fixed array, before any HIP
    call (64 caches of 32K tokens, 32 / 8 heads of d = 128: ~70 MB)."""
    f = lib.logo_decode_noalloc
    p = Prob(seqlens=(100, 50), hq=8, hkv=2, d=128, window=16)
    assert f(p.c, None, FAKE, FAKE, None, None, None, FAKE, 0, 0.5, None, None, None, 1e-6,
             FAKE, None, None, None) == ERR_NULL
    assert f(p.c, FAKE, FAKE, FAKE, None, None, None, FAKE, 0, float("nan"), None, None, None,
             1e-6, FAKE, None, None, None) == ERR_ARG
    assert f(p.c, FAKE, FAKE, FAKE, None, None, None, FAKE, 1, 0.5, None, None, None, 1e-6,
             FAKE, None, None, None) == ERR_ARG          # ratio mode: not for decoding
    big = Prob(seqlens=(32768,) * 64, hq=32, hkv=8, d=128, window=1024)
    assert lib.logo_workspace_bytes(big.c, 6, 0) > (64 << 20)
    assert f(big.c, FAKE, FAKE, FAKE, None, None, None, FAKE, 0, 0.5, None, None, None, 1e-6,
             FAKE, None, None, None) == ERR_SCRATCH_LIMIT


def test_decode_validation(lib):
    """logo_decode rejects bad arguments before any launch."""
    p = Prob(seqlens=(100, 50), hq=8, hkv=2, d=128, window=16)
    need = lib.logo_workspace_bytes(p.c, 6, 0)
    assert need > 0 and need % 256 == 0
    f = lib.logo_decode
    args = [p.c, FAKE, FAKE, FAKE, None, None, None, FAKE, 0, 0.5, None, None, None, 1e-6, FAKE,
            None, None, FAKE, need, None]

    def call(**kw):
        a = list(args)
        for i, v in kw.items():
            a[int(i[1:])] = v
        return f(*a)

    assert call(a1=None) == ERR_NULL                 # q
    assert call(a7=None) == ERR_NULL                 # gate
    assert call(a14=None) == ERR_NULL                # out
    assert call(a9=float("nan")) == ERR_ARG          # NaN threshold
    assert call(a8=1) == ERR_ARG                     # ratio mode
    assert call(a8=2) == ERR_NULL                    # device threshold without thr_dev
    assert call(a13=-1.0) == ERR_ARG                 # eps
    assert call(a18=need - 1) == ERR_WORKSPACE
    assert call(a17=None) == ERR_WORKSPACE
    empty = Prob(seqlens=(10, 0, 5), hq=8, hkv=2, d=128, window=16)
    need_e = lib.logo_workspace_bytes(empty.c, 6, 0)
    a = list(args)
    a[0], a[18] = empty.c, need_e
    assert f(*a) == ERR_SHAPE                        # a sequence with an empty cache
    assert f(Prob(d=96).c, *args[1:]) == ERR_UNSUPPORTED
    # the partial-result slots grow with the cache (chunks of >= 256 keys)
    big = Prob(seqlens=(32768,) * 4, hq=32, hkv=8, d=128, window=1024)
    nb = lib.logo_workspace_bytes(big.c, 6, 0)
    assert 4 * 32 * (128 + 4) * 4 * 4 <= nb < 64 << 20


def test_gate_and_transform_validation(lib):
    g = lib.logo_gate_proj
    assert g(-1, 64, FAKE, FAKE, FAKE, None) == ERR_SHAPE
    assert g(10, 60, FAKE, FAKE, FAKE, None) == ERR_UNSUPPORTED      # d_model % 8
    assert g(10, 64, None, FAKE, FAKE, None) == ERR_NULL
    assert g(10, 64, ctypes.c_void_p(0x1008), FAKE, FAKE, None) == ERR_ARG   # misaligned x
    assert g(0, 64, None, None, None, None) == OK                    # nothing to do
    t = lib.logo_branch_transform
    assert t(10, 4, 96, 0, FAKE, FAKE, None, None, None, 10, None, FAKE, None) == ERR_UNSUPPORTED
    assert t(10, 4, 128, 2, FAKE, FAKE, None, None, None, 10, None, FAKE, None) == ERR_ARG
    assert t(10, 4, 128, 0, FAKE, None, None, None, None, 10, None, FAKE, None) == ERR_NULL
    assert t(10, 4, 128, 1, FAKE, None, FAKE, None, None, 10, None, FAKE, None) == ERR_NULL
    assert t(10, 4, 128, 0, FAKE, FAKE, None, None, None, 9, None, FAKE, None) == ERR_SHAPE
    assert t(10, 0, 128, 0, FAKE, FAKE, None, None, None, 10, None, FAKE, None) == ERR_SHAPE
    assert t(10, 4, 128, 0, FAKE, FAKE, None, None, None, 10, None, None, None) == ERR_NULL


def _caller(f, args):
    def call(**kw):
        a = list(args)
        for i, v in kw.items():
            a[int(i[1:])] = v
        return f(*a)
    return call


def test_train_and_backward_validation(lib):
    """logo_attn_fwd_train, logo_attn_bwd and the dense training entry points
    reject bad arguments before any launch."""
    p = Prob(seqlens=(100, 50), hq=8, hkv=2, d=128, window=16)
    need = lib.logo_workspace_bytes(p.c, 7, 150)
    assert need > 0 and need % 256 == 0
    call = _caller(lib.logo_attn_fwd_train,
                   [p.c, FAKE, FAKE, FAKE, None, None, None, FAKE, 0, 0.5, 0.0, None, None, 1e-6,
                    FAKE, FAKE, 150, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, need, None])
    for i in (1, 7, 14, 15, 17, 18, 20, 21, 22, 23):
        assert call(**{f"a{i}": None}) == ERR_NULL, i
    assert call(a16=-1) == ERR_SHAPE
    assert call(a13=-1.0) == ERR_ARG
    assert call(a8=1, a10=2.0) == ERR_ARG
    assert call(a9=float("nan")) == ERR_ARG
    assert call(a25=need - 1) == ERR_WORKSPACE

    need_b = lib.logo_workspace_bytes(p.c, 8, 150)
    # the backward holds dO^L (bf16) and the row sums at least
    assert need_b >= 150 * 8 * 128 * 2 + 8 * 150 * 4
    args = [p.c, FAKE, FAKE, FAKE, None, None, None, FAKE, None, None, 1e-6, FAKE, 150, FAKE,
            FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, None, FAKE, None,
            None, FAKE, need_b, None]
    call = _caller(lib.logo_attn_bwd, args)
    assert call(a4=FAKE) == ERR_ARG                  # q_g without dq_g
    assert call(a23=FAKE) == ERR_ARG                 # dq_g without q_g
    assert call(a6=FAKE) == ERR_ARG                  # v_g without dv_g
    for i in (1, 7, 14, 15, 16, 19, 20, 21, 22, 13):
        assert call(**{f"a{i}": None}) == ERR_NULL, i
    for i in (11, 17, 18):                           # needed when sel_capacity > 0
        assert call(**{f"a{i}": None}) == ERR_NULL, i
    assert call(a12=-1) == ERR_SHAPE
    assert call(a10=float("nan")) == ERR_ARG
    assert call(a30=need_b - 1) == ERR_WORKSPACE
    wide = Prob(seqlens=(100,), hq=48, hkv=8, d=128, window=16)   # Hq d / 8 = 768
    a = list(args)
    a[0], a[30] = wide.c, lib.logo_workspace_bytes(wide.c, 8, 150)
    assert lib.logo_attn_bwd(*a) == ERR_UNSUPPORTED

    need_d = lib.logo_workspace_bytes(p.c, 9, 0)
    assert need_d == 8 * 150 * 4 + (-8 * 150 * 4) % 256
    call = _caller(lib.logo_dense_causal_attn_bwd,
                   [p.c, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, need_d, None])
    for i in range(1, 10):
        assert call(**{f"a{i}": None}) == ERR_NULL, i
    assert call(a11=need_d - 4) == ERR_WORKSPACE
    assert lib.logo_dense_causal_attn_fwd_train(p.c, None, FAKE, FAKE, FAKE, None, None) == ERR_NULL


def test_sparse_operator_training_validation(lib):
    """The standalone query-sparse training entry points reject bad
    arguments before any launch."""
    p = Prob(seqlens=(100, 50), hq=8, hkv=2, d=128, window=16)
    need_f = lib.logo_workspace_bytes(p.c, 2, 40)
    call = _caller(lib.logo_global_attn_sparse_q_fwd_train,
                   [p.c, FAKE, FAKE, FAKE, FAKE, FAKE, 40, FAKE, FAKE, FAKE, need_f, None])
    for i in (1, 2, 3, 4, 5, 7, 8):
        assert call(**{f"a{i}": None}) == ERR_NULL, i
    assert call(a6=-1) == ERR_SHAPE
    assert call(a10=need_f - 1) == ERR_WORKSPACE
    need_b = lib.logo_workspace_bytes(p.c, 10, 40)
    assert need_b >= 40 * 8 * 128 * 2 + 8 * 40 * 4
    call = _caller(lib.logo_global_attn_sparse_q_bwd,
                   [p.c, FAKE, FAKE, FAKE, FAKE, FAKE, 40, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                    FAKE, need_b, None])
    for i in (1, 2, 3, 4, 5, 7, 8, 9, 10, 11, 12):
        assert call(**{f"a{i}": None}) == ERR_NULL, i
    assert call(a6=-1) == ERR_SHAPE
    assert call(a14=need_b - 1) == ERR_WORKSPACE
    assert call(a13=ctypes.c_void_p(0x1010)) == ERR_WORKSPACE      # misaligned


def test_header_is_c99_and_callable_from_c(lib, tmp_path):
    """include/logo.h compiles as strict C99 (no C++ in the interface) and a
    C program linked against liblogo.so gets the documented answers from its
    host-side paths (tests/c/abi_from_c.c; nothing there reaches the GPU)."""
    import shutil
    import subprocess
    import paper_2608_29539_amd as pk
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not found")
    libdir = os.path.dirname(pk.library_path())
    exe = str(tmp_path / "abi_from_c")
    cmd = [gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
           "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "c", "abi_from_c.c"),
           "-L", libdir, "-llogo", f"-Wl,-rpath,{libdir}", "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "0 failure(s)" in r.stdout
