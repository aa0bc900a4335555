"""GPU parity for batches larger than a wave tile at the edges of the
input limits (Sec. 2.1, Eq. 1: exact sums of p, c and p^2 per batch and the
phase they imply).  A batch of more than 65,535 zero-context requests and a
decode batch whose sum of c passes 2^48 must keep the exact sums and the
phase, through every entry point that forms batch sums: attribution (Eq. 1
and the extended model), feature rows, batch sums, and the what-if sweep."""
import sys

import numpy as np
import pytest

import oracle
import parity
import tracegen

pytestmark = pytest.mark.gpu

C_MAX = (1 << 31) - 1


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def L():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_08382_amd import llmv
    llmv.load()
    torch.cuda.set_device(0)
    return llmv


def fill(kind, n, rng):
    """(p, c) of one batch of n requests."""
    p = np.ones(n, np.int32)
    if kind == "zero-context":        # prefill-type requests (c == 0): PREFILL
        c = np.zeros(n, np.int32)
    elif kind == "max-context":       # decode at the largest context: sum c >= 2^48
        c = np.full(n, C_MAX, np.int32)
    elif kind == "one-zero-last":     # decode except the last request: PREFILL
        c = np.full(n, C_MAX, np.int32)
        c[-1] = 0
    elif kind == "decode":
        c = rng.integers(1, 1 << 17, n).astype(np.int32)
    elif kind == "prefill":
        p = rng.integers(1, 4096, n).astype(np.int32)
        c = np.zeros(n, np.int32)
    else:
        raise KeyError(kind)
    return p, c


# (kind, size): 65,536 and 131,072 zero-context requests (the count of
# c == 0 is a multiple of 2^16), 131,073 requests at c = 2^31 - 1 (sum c =
# 2^48 + 2^17 - ... > 2^48), small neighbours on both sides
LAYOUTS = {
    "zero-65536": [("decode", 3), ("zero-context", 65536), ("prefill", 5)],
    "zero-131072": [("zero-context", 131072), ("decode", 2)],
    "max-context-131073": [("decode", 7), ("max-context", 131073), ("decode", 1)],
    "mixed-giants": [("prefill", 2), ("zero-context", 65536), ("decode", 4),
                     ("max-context", 131073), ("one-zero-last", 70000), ("decode", 3)],
}


def make_trace(key, n_tenants=3):
    rng = np.random.default_rng(sum(map(ord, key)))
    ps, cs, sizes = [], [], []
    for kind, n in LAYOUTS[key]:
        p, c = fill(kind, n, rng)
        ps.append(p)
        cs.append(c)
        sizes.append(n)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    p = np.concatenate(ps)
    c = np.concatenate(cs)
    t = rng.integers(0, n_tenants, len(p)).astype(np.int32)
    return tracegen.Trace(off, p, c, t, n_tenants, None)


def expected_phases(key):
    want = []
    for kind, _ in LAYOUTS[key]:
        want.append(1 if kind in ("decode", "max-context") else 0)
    return np.array(want, np.uint8)


@pytest.mark.parametrize("key", sorted(LAYOUTS))
def test_big_batch_sums_exact(L, key):
    import torch
    tr = make_trace(key)
    say(f"[big] batch sums {key}: sizes {tr.sizes().tolist()}")
    ref_s, ref_p = oracle.batch_sums(tr.offsets, tr.p, tr.c)
    assert np.array_equal(ref_p, expected_phases(key))
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, None)
    for ext in (False, True):
        sums, phase = L.batch_sums(dt, ext=ext)
        torch.cuda.synchronize()
        want_s = oracle.batch_sums_ext(tr.offsets, tr.p, tr.c)[0] if ext else ref_s
        assert np.array_equal(sums.cpu().numpy(), want_s), (key, ext)
        assert np.array_equal(phase.cpu().numpy(), ref_p), (key, ext)
    if "max-context" in key:
        assert ref_s[2].max() >= 1 << 48


@pytest.mark.parametrize("key", sorted(LAYOUTS))
def test_big_batch_attribute(L, key):
    import torch
    tr = make_trace(key)
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    for shape, co in ((None, tracegen.base_coeffs(91)),
                      (tracegen.SHAPES["llama3.1-8b"], tracegen.config_coeffs("heavy-tailed"))):
        out = L.attribute(dt, shape, co, tr.n_tenants)
        torch.cuda.synchronize()
        g = {k: v.cpu().numpy() for k, v in out.items()}
        ref = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, shape, co, tr.n_tenants)
        assert np.array_equal(g["regime"] // 2, expected_phases(key)), key
        st = parity.compare(ref, tr.offsets, g["latency"], g["regime"], g["share"],
                            g["tenant_sums"])
        say(f"[big] attribute {key} shape={shape is not None}: {st}")


@pytest.mark.parametrize("key", sorted(LAYOUTS))
def test_big_batch_attribute_ext(L, key):
    import torch
    tr = make_trace(key)
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    shape = tracegen.SHAPES["qwen2.5-14b"]
    co = tracegen.ext_coeffs(104)
    out = L.attribute_ext(dt, shape, co, tr.n_tenants,
                          ws=L.workspace(tr.n_batches, tr.n_requests, tr.n_tenants))
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in out.items()}
    ref = oracle.attribute_ext(tr.offsets, tr.p, tr.c, tr.tenant, shape, co, tr.n_tenants)
    assert np.array_equal(g["regime"] // 2, expected_phases(key)), key
    st = parity.compare(ref, tr.offsets, g["latency"], g["regime"], g["share"], g["tenant_sums"])
    say(f"[big] attribute_ext {key}: {st}")


@pytest.mark.parametrize("key", sorted(LAYOUTS))
def test_big_batch_features(L, key):
    import torch
    tr = make_trace(key)
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c)
    shape = tracegen.SHAPES["70b-like"]
    xr, xb = L.features(dt, shape)
    torch.cuda.synchronize()
    rr, rb = oracle.features(tr.offsets, tr.p, tr.c, shape)
    assert parity.rel_err(xr.cpu().numpy(), rr).max() <= parity.RTOL
    assert parity.rel_err(xb.cpu().numpy(), rb).max() <= 1e-12


@pytest.mark.parametrize("ext", [False, True])
def test_big_batch_sweep(L, ext):
    """The sweep's exact batch sums (built per 2048-request slice and added
    across slices) on every layout at once: 10 settings, two passes."""
    import torch
    rng = np.random.default_rng(5)
    parts = [make_trace(k) for k in sorted(LAYOUTS)]
    sizes = np.concatenate([t.sizes() for t in parts])
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    tr = tracegen.Trace(off, np.concatenate([t.p for t in parts]),
                        np.concatenate([t.c for t in parts]),
                        rng.integers(0, 5, int(off[-1])).astype(np.int32), 5, None)
    shapes = [tracegen.SHAPES["llama3.1-8b"], tracegen.SHAPES["qwen2.5-32b"]]
    if ext:
        co = np.stack([tracegen.ext_coeffs(700 + j) for j in range(5)])
    else:
        co = tracegen.sweep_coeffs(tracegen.config_coeffs("heavy-tailed"), 5)
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    out = L.attribute_sweep(dt, shapes, co, tr.n_tenants, ext=ext)
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    attr = oracle.attribute_ext if ext else oracle.attribute
    for s in range(2):
        for v in range(5):
            ref = attr(tr.offsets, tr.p, tr.c, tr.tenant, shapes[s], co[v], tr.n_tenants,
                       ("tenant_sums",))["tenant_sums"]
            e = parity.rel_err(out[s, v], ref)
            assert e.max() <= parity.RTOL, (ext, s, v, e.max())


def long_trace(case, n_tenants):
    """Batches larger than a wave tile between ordinary ones: p, c of decode
    batches (p = 1, c > 0) and prefill batches (c = 0), random tenants."""
    rng = np.random.default_rng(sum(map(ord, case)) + n_tenants)
    if case == "many-just-over":      # two tiles each: held whole by a k_long wave
        sizes = rng.choice([1790, 1791, 1792, 1793, 1794, 1795, 1796, 1537, 2000, 3], 700)
    elif case == "mixed-sizes":       # two tiles, several tiles, listed with segments
        sizes = np.concatenate([rng.integers(1, 300, 300), rng.integers(1793, 40000, 60)])
        rng.shuffle(sizes)
    elif case == "huge-and-small":    # segments over the whole grid
        sizes = np.array([5, 3_000_000, 1, 0, 17, 1_000_001, 2] + list(rng.integers(0, 200, 100)))
    elif case == "listed-runs":       # runs of listed batches next to runs of k_long ones
        sizes = np.concatenate([rng.integers(114_689, 200_000, 12), rng.integers(1793, 114_688, 12),
                                rng.integers(0, 100, 40), [114_688, 114_689, 114_690]])
        sizes = np.concatenate([sizes[:20], np.sort(sizes[20:])])
    elif case == "small-trace":       # one workgroup for the tiles, then k_long
        sizes = np.array([3, 5000, 7, 2500, 1, 0, 1793, 2])
    else:
        raise KeyError(case)
    sizes = np.asarray(sizes, np.int64)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    N = int(off[-1])
    p = np.ones(N, np.int32)
    c = rng.integers(1, 1 << 17, N).astype(np.int32)
    for b in np.nonzero(rng.random(len(sizes)) < 0.4)[0]:
        p[off[b]:off[b + 1]] = rng.integers(1, 3000, sizes[b])
        c[off[b]:off[b + 1]] = 0
    t = rng.integers(0, n_tenants, N).astype(np.int32)
    return tracegen.Trace(off, p, c, t, n_tenants, None)


@pytest.mark.parametrize("case", ["many-just-over", "mixed-sizes", "huge-and-small", "listed-runs",
                                  "small-trace"])
@pytest.mark.parametrize("n_tenants", [7, 5000])
def test_long_batches(L, case, n_tenants):
    """Eq. 1 attribution of batches larger than a wave tile: listed by the
    tile kernel for k_long (one wave each, held whole over two tiles,
    streamed beyond) or, above 64 wide tiles (114,688 requests), with their
    segments for the whole grid; more of them than the grid has waves, and
    more in a row than a wave buffers; the LDS histogram (7 tenants) and the
    tenant cache (5000); every output against the oracle, and output
    subsets agreeing with the full call."""
    import torch
    tr = long_trace(case, n_tenants)
    off, p, c, t = tr.offsets, tr.p, tr.c, tr.tenant
    say(f"[big] long {case} T={n_tenants}: nB={tr.n_batches} N={tr.n_requests}")
    dt = L.DeviceTrace.from_host(off, p, c, t)
    shape = tracegen.SHAPES["llama3.1-8b"]
    co = tracegen.config_coeffs("heavy-tailed")
    out = L.attribute(dt, shape, co, n_tenants)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in out.items()}
    ref = oracle.attribute(off, p, c, t, shape, co, n_tenants)
    st = parity.compare(ref, off, g["latency"], g["regime"], g["share"], g["tenant_sums"])
    say(f"[big] {st}")
    for outs in (("latency", "regime"), ("share",), ("tenant_sums",)):
        part = L.attribute(dt, shape, co, n_tenants, outs)
        torch.cuda.synchronize()
        for k in outs:
            if k == "tenant_sums":
                np.testing.assert_allclose(part[k].cpu().numpy(), g[k], rtol=1e-12)
            else:
                assert np.array_equal(part[k].cpu().numpy(), g[k]), (outs, k)


@pytest.mark.parametrize("case", ["many-just-over", "mixed-sizes", "small-trace"])
def test_long_batches_other_modes(L, case):
    """The feature rows, the exact batch sums and the extended model over
    batches larger than a wave tile (k_long's waves for every size)."""
    import torch
    tr = long_trace(case, 11)
    off, p, c, t = tr.offsets, tr.p, tr.c, tr.tenant
    say(f"[big] long modes {case}: nB={tr.n_batches} N={tr.n_requests}")
    dt = L.DeviceTrace.from_host(off, p, c, t)
    shape = tracegen.SHAPES["qwen2.5-14b"]
    xr, xb = L.features(dt, shape)
    torch.cuda.synchronize()
    rr, rb = oracle.features(off, p, c, shape)
    assert parity.rel_err(xr.cpu().numpy(), rr).max() <= parity.RTOL
    assert parity.rel_err(xb.cpu().numpy(), rb).max() <= 1e-12
    for ext in (False, True):
        sums, phase = L.batch_sums(dt, ext=ext)
        torch.cuda.synchronize()
        want_s, want_p = (oracle.batch_sums_ext if ext else oracle.batch_sums)(off, p, c)[:2]
        assert np.array_equal(sums.cpu().numpy(), want_s), ext
        assert np.array_equal(phase.cpu().numpy(), want_p), ext
    co = tracegen.ext_coeffs(105)
    out = L.attribute_ext(dt, shape, co, 11,
                          ws=L.workspace(tr.n_batches, tr.n_requests, 11))
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in out.items()}
    ref = oracle.attribute_ext(off, p, c, t, shape, co, 11)
    st = parity.compare(ref, off, g["latency"], g["regime"], g["share"], g["tenant_sums"])
    say(f"[big] ext {case}: {st}")


def test_long_mean_full_size(L):
    """Batches of 1793 requests (one more than a wave tile) over the
    decode-only trace's 128M requests: the mean batch is larger than a tile,
    so the tile kernel's work is one static chunk per wave plus claimed
    chunks (a wave's share passes 32 tiles), listing every batch for k_long.
    Every latency, regime, share and tenant sum against the oracle."""
    import torch
    tr = tracegen.config_trace("decode-only")
    n = tr.n_requests
    assert n > 2048 * 32 * 1792
    off = np.append(np.arange(0, n, 1793, dtype=np.int64), n)
    say(f"[big] long mean: nB={len(off) - 1} N={n}")
    dt = L.DeviceTrace.from_host(off, tr.p, tr.c, tr.tenant)
    shape = tracegen.SHAPES["qwen2.5-14b"]
    co = tracegen.config_coeffs("decode-only")
    out = L.attribute(dt, shape, co, tr.n_tenants)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in out.items()}
    ref = oracle.attribute(off, tr.p, tr.c, tr.tenant, shape, co, tr.n_tenants)
    st = parity.compare(ref, off, g["latency"], g["regime"], g["share"], g["tenant_sums"])
    say(f"[big] long mean: {st}")
