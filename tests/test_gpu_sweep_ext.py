"""GPU parity of the what-if sweep under the extended model
(llmv_attribute_sweep_ext through the C ABI) against the oracle's tenant
sums of the extended model (oracle.attribute_ext), setting by setting:
within 1e-5 relative.  With a5 = a6 = 0 the sweep is the Eq. 1 sweep up to
the order of its fp64 sums; and a single llmv_attribute_ext call agrees
with it up to fp32 rounding."""
import numpy as np
import pytest

import oracle
import parity
import tracegen

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module")
def L():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_08382_amd import llmv
    llmv.load()
    torch.cuda.set_device(0)
    return llmv


def ext_variants(n, seed0=600):
    """[n, 28] positive coefficient sets of the extended model."""
    return np.stack([tracegen.ext_coeffs(seed0 + j) for j in range(n)])


def run_sweep(L, tr, shapes, co, ext=True):
    import torch
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    out = L.attribute_sweep(dt, shapes, co, tr.n_tenants, ext=ext)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def check_against_oracle(tr, shapes, co, out, pairs, tag):
    for s, v in pairs:
        ref = oracle.attribute_ext(tr.offsets, tr.p, tr.c, tr.tenant,
                                   None if shapes is None else shapes[s], co[v], tr.n_tenants,
                                   ("tenant_sums",))["tenant_sums"]
        assert np.array_equal(out[s, v][ref == 0], ref[ref == 0]), (tag, s, v)
        e = parity.rel_err(out[s, v], ref)
        assert e.max() <= parity.RTOL, (tag, s, v, e.max())


def chunked_fill(rng, sizes, n_tenants, skew=None):
    """Batches of three kinds: prefill chunks over cached prefixes (p > 1 and
    c > 0, where sum p*c is neither sum c nor 0), fresh prefills (c = 0) and
    decode steps (p = 1)."""
    off = np.zeros(len(sizes) + 1, np.int64)
    off[1:] = np.cumsum(sizes)
    N = int(off[-1])
    p = np.ones(N, np.int32)
    c = rng.integers(1, 131072, N).astype(np.int32)
    kind = rng.integers(0, 3, len(sizes))
    for b in range(len(sizes)):
        lo, hi = off[b], off[b + 1]
        if kind[b] == 0:
            p[lo:hi] = rng.integers(2, 4096, hi - lo)
            c[lo:hi] = rng.integers(1, 65536, hi - lo)
        elif kind[b] == 1:
            p[lo:hi] = rng.integers(1, 8192, hi - lo)
            c[lo:hi] = 0
    if skew:
        w = 1.0 / np.arange(1, n_tenants + 1) ** skew
        t = rng.choice(n_tenants, N, p=w / w.sum()).astype(np.int32)
    else:
        t = rng.integers(0, n_tenants, N).astype(np.int32)
    return tracegen.Trace(off, p, c, t, n_tenants, None)


def test_sweep_ext_small(L):
    tr = tracegen.config_trace("whatif-sweep", 1500)
    co = ext_variants(5)
    shapes = [tracegen.SHAPES[k] for k in ("llama3.1-8b", "70b-like")]
    out = run_sweep(L, tr, shapes, co)
    assert out.shape == (2, 5, tr.n_tenants)
    check_against_oracle(tr, shapes, co, out, [(s, v) for s in range(2) for v in range(5)],
                         "small")
    # one llmv_attribute_ext call: there each share is 5 fp32 operations
    # (<= 5 ulp) before the fp64 sum; the sweep rounds a group's 5 sums to
    # fp32 (1 ulp) and evaluates its 5 terms in 5 fp32 operations (<= 5 ulp);
    # with nonnegative terms both stay within 6 * 2^-24 of the exact sum
    import torch
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    one = L.attribute_ext(dt, shapes[1], co[3], tr.n_tenants, ("tenant_sums",))["tenant_sums"]
    torch.cuda.synchronize()
    np.testing.assert_allclose(out[1, 3], one.cpu().numpy(), rtol=12 * 2.0**-24)


@pytest.mark.parametrize("T,skew", [(1, None), (3, 1.2), (1024, 1.2), (1025, None),
                                    (2049, 1.2), (4096, None)])
def test_sweep_ext_chunked_prefill(L, T, skew):
    """Prefill chunks with prefixes at every tenant count (8, 4 and 2
    settings per pass) and a partial last pass (2 x 11 settings)."""
    rng = np.random.default_rng(900 + T)
    sizes = rng.integers(0, 300, 700)
    sizes[::89] = 2000  # a few batches with more groups than a sweep tile
    tr = chunked_fill(rng, sizes, T, skew)
    co = ext_variants(11, 700)
    shapes = [tracegen.SHAPES["qwen2.5-14b"], tracegen.SHAPES["llama3.1-8b"]]
    say(f"[sweep ext] T={T}: nB={tr.n_batches} N={tr.n_requests}")
    out = run_sweep(L, tr, shapes, co)
    check_against_oracle(tr, shapes, co, out, [(s, v) for s in range(2) for v in range(11)],
                         f"T{T}")


def test_sweep_ext_unit_shape(L):
    rng = np.random.default_rng(31)
    tr = chunked_fill(rng, rng.integers(1, 200, 400), 17)
    co = ext_variants(3, 800)
    out = run_sweep(L, tr, None, co)
    check_against_oracle(tr, None, co, out, [(0, v) for v in range(3)], "unit")


@pytest.mark.parametrize("case", ["split-batches", "slice-aligned", "no-requests",
                                  "many-tenants-per-batch"])
def test_sweep_ext_group_edges(L, case):
    """Batches split by the 2048-request build slices (one of 300000
    requests), slices ending on a batch end, empty batches at both ends, no
    requests, and more distinct tenants in a batch than a build wave's hash
    table holds."""
    rng = np.random.default_rng(sum(map(ord, case)) + 5)
    if case == "split-batches":
        sizes = np.array([0, 0, 2048, 0, 4095, 1, 300000, 0, 0]
                         + list(rng.integers(0, 400, 300)) + [0, 0])
        tr = chunked_fill(rng, sizes, 1024, 1.2)
    elif case == "slice-aligned":
        tr = chunked_fill(rng, np.array([2048, 1024, 1024, 0, 2048, 0, 0]), 7)
    elif case == "no-requests":
        tr = chunked_fill(rng, np.zeros(40, np.int64), 5)
    else:
        tr = chunked_fill(rng, np.array([5000] * 30), 4096)
    co = ext_variants(5, 900)
    shapes = [tracegen.SHAPES["qwen2.5-32b"]]
    say(f"[sweep ext edge] {case}: nB={tr.n_batches} N={tr.n_requests} T={tr.n_tenants}")
    out = run_sweep(L, tr, shapes, co)
    if tr.n_requests == 0:
        assert np.array_equal(out, np.zeros_like(out))
        return
    check_against_oracle(tr, shapes, co, out, [(0, v) for v in range(5)], case)


def test_sweep_ext_zero_extension_is_the_eq1_sweep(L):
    """a5 = a6 = 0: every group term and every regime equals the Eq. 1
    sweep's; only the order of the fp64 tenant sums may differ."""
    rng = np.random.default_rng(41)
    tr = chunked_fill(rng, rng.integers(0, 400, 600), 1024, 1.2)
    co20 = tracegen.sweep_coeffs(tracegen.base_coeffs(79), 9)
    co28 = np.zeros((9, 28), np.float32)
    for g in range(4):
        co28[:, g * 7:g * 7 + 5] = co20[:, g * 5:(g + 1) * 5]
    shapes = [tracegen.SHAPES["llama3.1-8b"]]
    a = run_sweep(L, tr, shapes, co20, ext=False)
    b = run_sweep(L, tr, shapes, co28, ext=True)
    np.testing.assert_allclose(b, a, rtol=1e-11, atol=0)


def test_sweep_ext_refuses_the_eq1_workspace(L):
    """llmv_sweep_workspace_size's bytes do not hold the groups' sums of
    p*c: EWORKSPACE, and the output is left alone."""
    import torch
    tr = tracegen.config_trace("whatif-sweep", 300)
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    co = ext_variants(2)
    out = torch.full((1, 2, tr.n_tenants), -1.0, dtype=torch.float64, device="cuda")
    ws = L.sweep_workspace(tr.n_batches, tr.n_requests, tr.n_tenants)
    with pytest.raises(L.LlmvError) as e:
        L.llmv_attribute_sweep(dt, [tr.shape], co, tr.n_tenants, out, ws, ext=True)
    assert e.value.code == L.LLMV_EWORKSPACE
    torch.cuda.synchronize()
    assert bool((out == -1.0).all())


def test_sweep_ext_full_size_sampled(L):
    """The what-if workload at full size (100k batches, 1024 tenants) under 4
    shapes x 256 extended settings; sampled settings against the oracle."""
    tr = tracegen.config_trace("whatif-sweep")
    co = ext_variants(256)
    names = ["llama3.1-8b", "qwen2.5-14b", "qwen2.5-32b", "70b-like"]
    shapes = [tracegen.SHAPES[k] for k in names]
    say(f"[sweep ext] N={tr.n_requests} variants={4 * 256}")
    out = run_sweep(L, tr, shapes, co)
    assert np.all(np.isfinite(out))
    check_against_oracle(tr, shapes, co, out, [(0, 0), (1, 17), (2, 128), (3, 255), (0, 201)],
                         "full")
