"""The C-ABI library on the CPU host (no GPU): it loads, exports every
function include/llmv.h declares, computes the same shape constants as the
oracle, and rejects bad host arguments before touching the device."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
import tracegen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "llmv.h")


@pytest.fixture(scope="module")
def llmv():
    from paper_2608_08382_amd import build, llmv as mod
    if build.is_stale():
        build.build()
    mod.load()
    return mod


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(llmv_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_function(llmv):
    names = declared_functions()
    assert set(names) == set(llmv.EXPORTS)
    lib = llmv.load()
    for n in names:
        assert hasattr(lib, n)
    out = subprocess.run(["nm", "-D", "--defined-only", llmv.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (llmv_\w+)", out))
    assert set(names) <= exported
    # nothing else with the llmv_ prefix leaks out
    assert exported == set(names)


def test_library_is_gfx950_code_object(llmv):
    # the offload bundle inside the library names its target
    data = open(llmv.LIB_PATH, "rb").read()
    assert b"amdgcn-amd-amdhsa--gfx950" in data


@pytest.mark.parametrize("name", sorted(tracegen.SHAPES))
def test_shape_constants_match_oracle(llmv, name):
    sh = tracegen.SHAPES[name]
    assert llmv.llmv_shape_constants(sh) == list(oracle.shape_constants(sh))


@settings(max_examples=50, deadline=None)
@given(st.lists(st.integers(1, 1 << 12), min_size=9, max_size=9))
def test_shape_constants_random(llmv, v):
    sh = dict(zip(tracegen.SHAPE_FIELDS, v))
    try:
        want = list(oracle.shape_constants(sh))
    except oracle.OracleError:
        with pytest.raises(llmv.LlmvError):
            llmv.llmv_shape_constants(sh)
        return
    assert llmv.llmv_shape_constants(sh) == want


def test_shape_constants_unit_and_errors(llmv):
    assert llmv.llmv_shape_constants(None) == [1.0, 1.0, 1.0, 1.0]
    bad = dict(tracegen.SHAPES["llama3.1-8b"], head_dim=0)
    with pytest.raises(llmv.LlmvError) as ei:
        llmv.llmv_shape_constants(bad)
    assert ei.value.code == llmv.LLMV_EINVAL
    assert "field" in llmv.llmv_last_error()
    huge = dict(tracegen.SHAPES["llama3.1-8b"], n_layers=1 << 30, hidden=1 << 30)
    with pytest.raises(llmv.LlmvError):
        llmv.llmv_shape_constants(huge)


FAKE = 0x100000  # never dereferenced: every call below fails its host checks first


def _trace(llmv, nB=4, N=8, off=FAKE, p=FAKE, c=FAKE, t=FAKE):
    return llmv.llmv_trace(nB, N, off, p, c, t)


def _attr(llmv, tr, coeffs=None, share=None, T=1, tsum=None, ws=None, wsb=0):
    lib = llmv.load()
    co = (ctypes.c_float * 20)(*(coeffs if coeffs is not None else [1.0] * 20))
    return lib.llmv_attribute(None if tr is None else ctypes.byref(tr), None, co, None, None,
                              share, T, tsum, ws, wsb, None)


def test_host_argument_errors(llmv):
    lib = llmv.load()
    E = llmv.LLMV_EINVAL
    assert _attr(llmv, None) == E
    assert _attr(llmv, _trace(llmv, nB=-1)) == E
    assert _attr(llmv, _trace(llmv, N=-5)) == E
    assert _attr(llmv, _trace(llmv, off=0)) == E
    assert _attr(llmv, _trace(llmv, p=0)) == E
    assert _attr(llmv, _trace(llmv, p=FAKE + 4)) == E  # misaligned
    assert _attr(llmv, _trace(llmv), coeffs=[float("nan")] + [1.0] * 19) == E
    assert _attr(llmv, _trace(llmv), coeffs=[1.0] * 19 + [float("inf")]) == E
    assert _attr(llmv, _trace(llmv), share=FAKE + 8) == E
    # tenant sums need tenant ids and a tenant count
    assert _attr(llmv, _trace(llmv, t=0), tsum=FAKE) == E
    assert _attr(llmv, _trace(llmv), T=0, tsum=FAKE) == E
    assert _attr(llmv, _trace(llmv), T=(1 << 24) + 1, tsum=FAKE) == E
    assert "n_tenants" in llmv.llmv_last_error()
    # features / tenant sums / validate
    assert lib.llmv_features(None, None, None, None, None, 0, None) == E
    assert lib.llmv_tenant_sums(FAKE, FAKE, -1, 4, FAKE, None, 0, None) == E
    assert lib.llmv_tenant_sums(FAKE, FAKE, 10, 0, FAKE, None, 0, None) == E
    assert lib.llmv_tenant_sums(FAKE, FAKE, 10, 4, None, None, 0, None) == E
    assert lib.llmv_tenant_sums(None, FAKE, 10, 4, FAKE, None, 0, None) == E
    assert lib.llmv_validate(None, 0, None, 0, None) == E
    tr = _trace(llmv)
    assert lib.llmv_validate(ctypes.byref(tr), 0, None, 0, None) == E  # tenant without count
    # sweep: argument checks
    co = (ctypes.c_float * 40)(*([1.0] * 40))
    sw = lib.llmv_attribute_sweep
    assert sw(ctypes.byref(tr), None, 2, co, 2, 4, FAKE, None, 0, None) == E  # NULL shapes, 2
    assert sw(ctypes.byref(tr), None, 1, co, 0, 4, FAKE, None, 0, None) == E  # no coeffs
    assert sw(ctypes.byref(tr), None, 1, None, 2, 4, FAKE, None, 0, None) == E
    assert sw(ctypes.byref(tr), None, 1, co, 2, 4097, FAKE, None, 0, None) == E  # LDS limit
    assert sw(ctypes.byref(tr), None, 1, co, 2, 4, None, None, 0, None) == E  # no out
    co[25] = float("nan")
    assert sw(ctypes.byref(tr), None, 1, co, 2, 4, FAKE, None, 0, None) == E
    assert sw(ctypes.byref(_trace(llmv, t=0)), None, 1, co, 2, 4, FAKE, None, 0, None) == E
    # the extended sweep: the same checks, 28 coefficients per set
    cx = (ctypes.c_float * 56)(*([1.0] * 56))
    sx = lib.llmv_attribute_sweep_ext
    assert sx(ctypes.byref(tr), None, 2, cx, 2, 4, FAKE, None, 0, None) == E
    assert sx(ctypes.byref(tr), None, 1, cx, 0, 4, FAKE, None, 0, None) == E
    assert sx(ctypes.byref(tr), None, 1, None, 2, 4, FAKE, None, 0, None) == E
    assert sx(ctypes.byref(tr), None, 1, cx, 2, 4097, FAKE, None, 0, None) == E
    assert sx(ctypes.byref(tr), None, 1, cx, 2, 4, None, None, 0, None) == E
    cx[55] = float("inf")  # the last coefficient of the second set
    assert sx(ctypes.byref(tr), None, 1, cx, 2, 4, FAKE, None, 0, None) == E
    assert "coeffs[55]" in lib.llmv_last_error().decode()
    assert sx(ctypes.byref(_trace(llmv, t=0)), None, 1, cx, 2, 4, FAKE, None, 0, None) == E


def test_batch_sums_and_admit_argument_errors(llmv):
    """Host-side checks only: every call below fails (or returns) before any
    launch."""
    lib = llmv.load()
    E = llmv.LLMV_EINVAL
    assert lib.llmv_batch_sums(None, FAKE, FAKE, None, 0, None) == E
    assert lib.llmv_batch_sums(ctypes.byref(_trace(llmv, nB=-1)), FAKE, FAKE, None, 0, None) == E
    assert lib.llmv_batch_sums(ctypes.byref(_trace(llmv, p=0)), FAKE, FAKE, None, 0, None) == E
    co = (ctypes.c_float * 20)(*([1.0] * 20))
    adm = lib.llmv_admit
    #       sums  phase  nB  shape coeffs  cb    cp    cc    m   outputs x4               stream
    assert adm(FAKE, FAKE, -1, None, co, FAKE, FAKE, FAKE, 4, None, None, None, None, None) == E
    assert adm(FAKE, FAKE, 8, None, co, FAKE, FAKE, FAKE, -4, None, None, None, None, None) == E
    assert adm(FAKE, FAKE, 8, None, None, FAKE, FAKE, FAKE, 4, None, None, None, None, None) == E
    assert adm(FAKE, FAKE, 8, None, co, None, FAKE, FAKE, 4, None, None, None, None, None) == E
    assert adm(FAKE, FAKE, 8, None, co, FAKE, FAKE, None, 4, None, None, None, None, None) == E
    assert adm(None, FAKE, 8, None, co, FAKE, FAKE, FAKE, 4, None, None, None, None, None) == E
    bad = llmv.llmv_shape(n_layers=0)
    assert adm(FAKE, FAKE, 8, ctypes.byref(bad), co, FAKE, FAKE, FAKE, 4, None, None, None, None,
               None) == E
    co[7] = float("nan")
    assert adm(FAKE, FAKE, 8, None, co, FAKE, FAKE, FAKE, 4, None, None, None, None, None) == E
    co[7] = 1.0
    # no candidates: nothing to do, nothing launched
    assert adm(None, None, 0, None, co, None, None, None, 0, None, None, None, None, None) == 0


def test_fit_argument_errors(llmv):
    """Host-side checks of llmv_fit / llmv_fit_metrics: every call below fails
    before any launch (the workspace check is the last one)."""
    lib = llmv.load()
    E, EW = llmv.LLMV_EINVAL, llmv.LLMV_EWORKSPACE
    th0 = (ctypes.c_double * 20)(*([1.0] * 20))
    fit = lib.llmv_fit
    #          sums  phase  nB  shape  y    theta0 rounds theta counts ws   bytes stream
    assert fit(FAKE, FAKE, -1, None, FAKE, th0, 1, FAKE, None, None, 0, None) == E
    assert fit(FAKE, FAKE, (1 << 31) + 1, None, FAKE, th0, 1, FAKE, None, None, 0, None) == E
    assert fit(None, FAKE, 8, None, FAKE, th0, 1, FAKE, None, None, 0, None) == E
    assert fit(FAKE, None, 8, None, FAKE, th0, 1, FAKE, None, None, 0, None) == E
    assert fit(FAKE, FAKE, 8, None, None, th0, 1, FAKE, None, None, 0, None) == E
    assert fit(FAKE, FAKE, 8, None, FAKE, None, 1, FAKE, None, None, 0, None) == E
    assert fit(FAKE, FAKE, 8, None, FAKE, th0, -1, FAKE, None, None, 0, None) == E
    assert fit(FAKE, FAKE, 8, None, FAKE, th0, 1025, FAKE, None, None, 0, None) == E
    assert fit(FAKE, FAKE, 8, None, FAKE, th0, 1, None, None, None, 0, None) == E
    bad = llmv.llmv_shape(n_layers=0)
    assert fit(FAKE, FAKE, 8, ctypes.byref(bad), FAKE, th0, 1, FAKE, None, None, 0, None) == E
    th0[3] = float("inf")
    assert fit(FAKE, FAKE, 8, None, FAKE, th0, 1, FAKE, None, None, 0, None) == E
    th0[3] = 1.0
    need = lib.llmv_fit_workspace_size(8)
    assert fit(FAKE, FAKE, 8, None, FAKE, th0, 1, FAKE, None, None, 0, None) == EW
    assert fit(FAKE, FAKE, 8, None, FAKE, th0, 1, FAKE, None, FAKE, need - 1, None) == EW
    assert fit(FAKE, FAKE, 8, None, FAKE, th0, 1, FAKE, None, FAKE + 16,
               need, None) == EW
    co = (ctypes.c_float * 20)(*([1.0] * 20))
    met = lib.llmv_fit_metrics
    #          sums  phase  nB  shape coeffs  y   rel_err out   ws   bytes stream
    assert met(FAKE, FAKE, -1, None, co, FAKE, None, FAKE, None, 0, None) == E
    assert met(None, FAKE, 8, None, co, FAKE, None, FAKE, None, 0, None) == E
    assert met(FAKE, FAKE, 8, None, co, None, None, FAKE, None, 0, None) == E
    assert met(FAKE, FAKE, 8, None, None, FAKE, None, FAKE, None, 0, None) == E
    assert met(FAKE, FAKE, 8, None, co, FAKE, None, None, None, 0, None) == E
    co[19] = float("nan")
    assert met(FAKE, FAKE, 8, None, co, FAKE, None, FAKE, None, 0, None) == E
    co[19] = 1.0
    assert met(FAKE, FAKE, 8, None, co, FAKE, None, FAKE, None, 0, None) == EW
    assert met(FAKE, FAKE, 8, None, co, FAKE, None, FAKE, FAKE, need - 1, None) == EW


@pytest.mark.parametrize("name", sorted(tracegen.SHAPES))
def test_shape_constants_ext_match_oracle(llmv, name):
    sh = tracegen.SHAPES[name]
    assert llmv.llmv_shape_constants_ext(sh) == list(oracle.shape_constants_ext(sh))
    assert llmv.llmv_shape_constants_ext(None) == [1.0] * 6


def test_attribute_ext_argument_errors(llmv):
    """Host-side checks of llmv_attribute_ext; every call fails before any
    launch."""
    lib = llmv.load()
    E = llmv.LLMV_EINVAL
    co = (ctypes.c_float * 28)(*([1.0] * 28))
    tr = ctypes.byref(_trace(llmv))
    out = FAKE
    ext = lib.llmv_attribute_ext
    assert ext(None, None, co, out, None, None, 0, None, None, 0, None) == E
    assert ext(tr, None, None, out, None, None, 0, None, None, 0, None) == E
    co[27] = float("nan")
    assert ext(tr, None, co, out, None, None, 0, None, None, 0, None) == E
    co[27] = 1.0
    assert ext(tr, None, co, None, None, None, 0, FAKE, None, 0, None) == E  # n_tenants 0
    assert ext(tr, None, co, None, None, FAKE + 4, 0, None, None, 0, None) == E  # share misaligned
    bad = llmv.llmv_shape(n_layers=0)
    assert ext(tr, ctypes.byref(bad), co, out, None, None, 0, None, None, 0, None) == E
    S = (ctypes.c_double * 6)()
    assert lib.llmv_shape_constants_ext(ctypes.byref(bad), S) == E
    assert lib.llmv_shape_constants_ext(None, None) == E


def test_fit_workspace_size(llmv):
    """Fixed part plus 4 bytes per batch (the relative errors), 256-aligned."""
    lib = llmv.load()
    a, b = lib.llmv_fit_workspace_size(0), lib.llmv_fit_workspace_size(1 << 20)
    assert a % 256 == 0 and b % 256 == 0
    assert b - a == 4 << 20
    assert lib.llmv_fit_workspace_size(1) == a + 256


def test_sweep_workspace_size(llmv):
    """The sweep's workspace: the common one (with a tenant histogram per
    setting of a pass) plus 20 bytes per request for the (batch, tenant)
    groups, 40 bytes per batch for their offsets, the exact batch sums and
    the count of zero-context requests.  The common part grows with the
    requests by its chunk table and the lists of batches larger than a wave
    tile (8 bytes per 1,533 requests; 40 per 14,337 and their segments, 8
    per 8,192 plus 16 per listed batch)."""
    lib = llmv.load()
    nB, N, T = 10_000, 1 << 24, 1024  # N large enough for the largest grid
    base = lib.llmv_sweep_workspace_size(nB, N, T)
    assert base % 256 == 0
    assert base >= lib.llmv_workspace_size(nB, N, T) + 20 * N
    d = 1 << 20
    dn = lib.llmv_sweep_workspace_size(nB, N + d, T) - base
    lists = 8 * (d // 1533 + 1) + 56 * (d // 14337 + 1) + 8 * (d // 8192 + 1)
    assert 20 << 20 <= dn <= (20 << 20) + 3 * 8 * (d // 2048) + lists + 8 * 256
    db = lib.llmv_sweep_workspace_size(nB + (1 << 16), N, T) - base
    assert 40 << 16 <= db <= (40 << 16) + 3 * 256
    assert lib.llmv_sweep_workspace_size(0, 0, 1) > 0
    assert lib.llmv_sweep_workspace_size(-5, -5, -5) == lib.llmv_sweep_workspace_size(0, 0, 0)


def test_sweep_workspace_size_ext(llmv):
    """The extended sweep's workspace: the Eq. 1 sweep's plus the groups'
    sums of p*c (4 bytes per request) and one more row of exact batch sums
    (8 bytes per batch)."""
    lib = llmv.load()
    nB, N, T = 10_000, 1 << 24, 1024
    for n_b, n in ((nB, N), (nB + (1 << 16), N), (nB, N + (1 << 20))):
        d = lib.llmv_sweep_workspace_size_ext(n_b, n, T) - lib.llmv_sweep_workspace_size(n_b, n, T)
        assert 4 * n + 8 * n_b <= d <= 4 * n + 8 * n_b + 4 * 1024 + 2 * 256, (n_b, n, d)
    assert lib.llmv_sweep_workspace_size_ext(-5, -5, -5) == \
        lib.llmv_sweep_workspace_size_ext(0, 0, 0) > 0


def test_python_binding_refuses_without_library(tmp_path):
    from paper_2608_08382_amd import llmv as mod
    saved = mod._lib
    try:
        mod._lib = None
        with pytest.raises(RuntimeError, match="build the HIP library"):
            mod.load(str(tmp_path / "missing.so"))
    finally:
        mod._lib = saved
