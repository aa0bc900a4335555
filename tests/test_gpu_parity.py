"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs.  Rules and tolerances: tests/parity.py."""
import json
import os
import sys

import numpy as np
import pytest

import oracle
import parity
import tracegen

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HAND = json.load(open(os.path.join(ROOT, "tests", "golden", "hand_examples.json")))


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


def run_gpu(L, tr, shape, coeffs, n_tenants, outputs=("latency", "regime", "share", "tenant_sums")):
    import torch
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant if "tenant_sums" in outputs else None)
    out = L.attribute(dt, shape, coeffs, n_tenants, outputs)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def check(L, tr, shape, coeffs, n_tenants, name=""):
    say(f"[parity] {name}: nB={tr.n_batches} N={tr.n_requests} T={n_tenants}")
    g = run_gpu(L, tr, shape, coeffs, n_tenants)
    ref = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, shape, coeffs, n_tenants)
    return parity.compare(ref, tr.offsets, g["latency"], g["regime"], g["share"],
                          g["tenant_sums"]), g, ref


def coeff_vec(d):
    return np.array(d["prefill_mem"] + d["prefill_comp"] + d["decode_mem"] + d["decode_comp"],
                    np.float32)


# ----------------------------------------------------------- hand examples


def test_hand_examples_exact(L):
    th = coeff_vec(HAND["base_coeffs"])
    for ex in HAND["unit_shape_examples"]:
        t = th.copy()
        if ex["coeff_override"]:
            t[ex["coeff_override"]["index"]] = ex["coeff_override"]["value"]
        tr = tracegen.from_batches([(ex["p"], ex["c"])], [[0] * len(ex["p"])], 1)
        g = run_gpu(L, tr, None, t, 1)
        say(f"[hand] {ex['name']}")
        assert g["latency"][0] == ex["T"], ex["name"]
        assert g["regime"][0] == ex["regime"], ex["name"]
        assert list(g["share"]) == ex["shares"], ex["name"]
        assert g["tenant_sums"][0] == sum(ex["shares"]), ex["name"]
    se = HAND["shaped_examples"]
    for ex in se["examples"]:
        tr = tracegen.from_batches([(ex["p"], ex["c"])], [[0] * len(ex["p"])], 1)
        g = run_gpu(L, tr, se["shape"], coeff_vec(se["coeffs"]), 1)
        assert g["latency"][0] == ex["T"] and g["regime"][0] == ex["regime"], ex["name"]
        assert list(g["share"]) == ex["shares"], ex["name"]


def test_hand_tenant_trace_exact(L):
    tt = HAND["tenant_trace"]
    by = {e["name"]: e for e in HAND["unit_shape_examples"]}
    tr = tracegen.from_batches([(by[n]["p"], by[n]["c"]) for n in tt["batches"]], tt["tenants"],
                               tt["n_tenants"])
    g = run_gpu(L, tr, None, coeff_vec(HAND["base_coeffs"]), tt["n_tenants"])
    assert list(g["tenant_sums"]) == tt["tenant_sums"]
    assert list(g["latency"]) == [by[n]["T"] for n in tt["batches"]]


# ------------------------------------------------------- workload recipes


@pytest.mark.parametrize("name,nb", [("tiny-mixed", None), ("decode-only", 3000),
                                     ("chunked-prefill", 2000), ("heavy-tailed", 3000),
                                     ("whatif-sweep", 2000)])
def test_config_recipes(L, name, nb):
    tr = tracegen.config_trace(name, nb)
    st, g, ref = check(L, tr, tr.shape, tracegen.config_coeffs(name), tr.n_tenants, name)
    say(f"[parity] {name}: {st}")
    # every regime the recipe produces is exercised
    assert len(set(g["regime"].tolist())) >= 2


def test_all_four_regimes(L):
    """A trace built to land in every (phase, segment) pair."""
    rng = np.random.default_rng(7)
    batches = []
    for _ in range(50):
        batches.append(([1] * int(rng.integers(1, 8)), list(rng.integers(1, 100, 1))))
    batches = [(b[0], [int(rng.integers(1, 50)) for _ in b[0]]) for b in batches]  # decode, small
    batches += [([1] * 300, [int(x) for x in rng.integers(1, 50, 300)]) for _ in range(20)]
    batches += [([int(x) for x in rng.integers(2, 6, 3)], [0, 0, 0]) for _ in range(20)]
    batches += [([int(x) for x in rng.integers(1000, 4000, 3)], [0, 0, 0]) for _ in range(20)]
    tr = tracegen.from_batches(batches, [[i % 3 for i in range(len(b[0]))] for b in batches], 3)
    th = coeff_vec(HAND["base_coeffs"])
    st, g, ref = check(L, tr, None, th, 3, "four regimes")
    assert set(ref["regime"].tolist()) == {0, 1, 2, 3}


# ------------------------------------------------------------- edge cases


def random_fill(rng, sizes, n_tenants=5, p_hi=5000, c_hi=200000):
    off = np.zeros(len(sizes) + 1, np.int64)
    off[1:] = np.cumsum(sizes)
    N = int(off[-1])
    pre = rng.random(len(sizes)) < 0.3
    p = np.ones(N, np.int32)
    c = rng.integers(1, c_hi, N).astype(np.int32)
    for b in np.nonzero(pre)[0]:
        p[off[b]:off[b + 1]] = rng.integers(1, p_hi, off[b + 1] - off[b])
        c[off[b]:off[b + 1]] = 0
    t = rng.integers(0, n_tenants, N).astype(np.int32)
    return tracegen.Trace(off, p, c, t, n_tenants, None)


SIZE_SETS = {
    "wave-edges": [1, 63, 64, 65, 127, 128, 129, 255, 256, 257, 511, 512, 513],
    "tile-edges": [767, 768, 769, 1023, 1024, 1025, 3068, 3069, 3070, 3071, 3072, 3073],
    "wave-tile-edges": [1787, 1788, 1789, 1790, 1791, 1792, 1793, 1, 3583, 3584, 3585, 2,
                        1795, 1796, 1797, 3, 1791, 1],
    "old-tile-edges": [1531, 1532, 1533, 1534, 1535, 1536, 1537, 1, 2044, 2045, 2046, 2047,
                       2048, 2049, 2, 1280, 1281, 1279],
    "big": [5000, 1, 2, 3, 100000, 7, 3075],
    "tiny": [1] * 700 + [2] * 300 + [3] * 100,
    "unaligned": [3, 5, 7, 1, 9, 11, 13, 2, 6, 10] * 50,
}


@pytest.mark.parametrize("key", sorted(SIZE_SETS))
def test_batch_size_edges(L, key):
    rng = np.random.default_rng(hash(key) % 1000)
    tr = random_fill(rng, SIZE_SETS[key])
    for shape in (None, tracegen.SHAPES["qwen2.5-14b"]):
        co = tracegen.base_coeffs(31)
        st, _, _ = check(L, tr, shape, co, tr.n_tenants, key)
        say(f"[edge] {key}: {st}")


@pytest.mark.parametrize("pattern", ["leading", "trailing", "long-run", "all-empty", "no-batches",
                                     "interleaved"])
def test_empty_batches(L, pattern):
    rng = np.random.default_rng(11)
    if pattern == "leading":
        sizes = [0] * 5 + list(rng.integers(1, 200, 50))
    elif pattern == "trailing":
        sizes = list(rng.integers(1, 200, 50)) + [0] * 7
    elif pattern == "long-run":
        sizes = list(rng.integers(1, 200, 20)) + [0] * 700 + list(rng.integers(1, 200, 20)) + \
            [0] * 300
    elif pattern == "all-empty":
        sizes = [0] * 1000
    elif pattern == "no-batches":
        sizes = []
    else:
        sizes = [int(x) if i % 2 else 0 for i, x in enumerate(rng.integers(1, 50, 600))]
    tr = random_fill(rng, np.array(sizes, np.int64))
    check(L, tr, tracegen.SHAPES["llama3.1-8b"], tracegen.base_coeffs(32), tr.n_tenants, pattern)


@pytest.mark.parametrize("N", [1, 2, 3, 4, 5, 6, 7, 8, 9, 4097, 4098, 4099])
def test_request_count_tails(L, N):
    """N not a multiple of 4: the last 16-byte group runs past the array."""
    rng = np.random.default_rng(N)
    sizes = []
    left = N
    while left > 0:
        s = int(min(left, rng.integers(1, 40)))
        sizes.append(s)
        left -= s
    tr = random_fill(rng, sizes)
    check(L, tr, None, tracegen.base_coeffs(33), tr.n_tenants, f"N={N}")


@pytest.mark.parametrize("N", [1, 12287, 12288, 12289, 14335, 14336, 14337])
def test_single_launch_boundary(L, N):
    """Traces of up to 14336 requests (two 1792-slot tiles per wave) run as
    one workgroup in one launch; one more request takes the partitioned
    multi-workgroup path."""
    rng = np.random.default_rng(N)
    sizes = []
    while sum(sizes) < N:
        sizes.append(int(min(rng.integers(0, 400), N - sum(sizes))))
    tr = random_fill(rng, np.array(sizes), n_tenants=37)
    assert tr.n_requests == N
    check(L, tr, tracegen.SHAPES["llama3.1-8b"], tracegen.base_coeffs(61), 37, f"N={N}")


# 1..1024 tenants: 4 LDS histogram replicas, 2048: 2, 3000 and 4096: 1,
# above 4096: the LDS tenant cache with global atomics for the rest
@pytest.mark.parametrize("n_tenants", [1, 2, 1024, 2048, 3000, 4096, 4097, 100000])
def test_tenant_counts(L, n_tenants):
    rng = np.random.default_rng(n_tenants)
    tr = random_fill(rng, rng.integers(1, 300, 400), n_tenants=n_tenants)
    if n_tenants in (1024, 2048):  # skewed, so that lanes of one atomic share tenants
        tr = tracegen.Trace(tr.offsets, tr.p, tr.c, skewed_tenants(rng, tr.n_requests, n_tenants),
                            n_tenants, None)
    check(L, tr, tracegen.SHAPES["qwen2.5-32b"], tracegen.base_coeffs(34), n_tenants,
          f"T={n_tenants}")


@pytest.mark.parametrize("n_tenants", [4097, 1 << 16, 1 << 20, 1 << 24])
def test_tenant_cache_under_skew(L, n_tenants):
    """More tenants than an LDS histogram holds, Zipf(1.2) ids (a few
    tenants take most requests, most tenants are seen once): the tenant
    cache keeps the frequent ones, the rest go to global atomics; every
    tenant's sum against the oracle.  200k batches (~2.5e7 requests), so each
    workgroup's cache fills and overflows."""
    tr = tracegen.generate(tracegen.KIND_HEAVY_TAILED, 200_000, 41, n_tenants,
                           tracegen.SHAPES["llama3.1-8b"], "skewed")
    st, g, ref = check(L, tr, tr.shape, tracegen.base_coeffs(36), n_tenants, f"T={n_tenants}")
    say(f"[tenant cache] T={n_tenants}: {st}, tenants with requests "
        f"{np.count_nonzero(np.bincount(tr.tenant, minlength=n_tenants))}")


def test_single_tenant_all_requests(L):
    """Every request on one tenant: maximal LDS atomic contention."""
    rng = np.random.default_rng(5)
    tr = random_fill(rng, rng.integers(1, 1024, 300), n_tenants=64)
    tr.tenant[:] = 17
    st, g, ref = check(L, tr, None, tracegen.base_coeffs(35), 64, "one tenant")
    assert np.count_nonzero(g["tenant_sums"]) == 1


def test_extreme_values(L):
    """Largest p (2^20) over a full tile and c near 2^31: the packed 32-bit
    prompt sums and 64-bit context sums stay exact."""
    sizes = [3072, 3069, 1, 5000, 2]
    off = np.zeros(len(sizes) + 1, np.int64)
    off[1:] = np.cumsum(sizes)
    N = int(off[-1])
    p = np.full(N, 1 << 20, np.int32)
    c = np.full(N, (1 << 31) - 1, np.int32)
    c[off[1]:off[2]] = 0
    t = (np.arange(N) % 3).astype(np.int32)
    tr = tracegen.Trace(off, p, c, t, 3, None)
    th = np.ones(20, np.float32)
    check(L, tr, None, th, 3, "extreme")
    check(L, tr, tracegen.SHAPES["70b-like"], tracegen.base_coeffs(36), 3, "extreme shaped")


def test_exact_ties_choose_mem(L):
    """Constructed exact ties (example A with decode-COMP a1 raised to 16)."""
    ex = [e for e in HAND["unit_shape_examples"] if e["name"] == "A_tie"][0]
    th = coeff_vec(HAND["base_coeffs"])
    th[16] = 16
    tr = tracegen.from_batches([(ex["p"], ex["c"])] * 500, [[0] * 4] * 500, 1)
    g = run_gpu(L, tr, None, th, 1)
    assert np.all(g["regime"] == 2)
    assert np.all(g["latency"] == 352)


def test_output_subsets_agree(L):
    tr = tracegen.config_trace("heavy-tailed", 800)
    co = tracegen.config_coeffs("heavy-tailed")
    full = run_gpu(L, tr, tr.shape, co, tr.n_tenants)
    for outs in (("latency",), ("regime",), ("share",), ("tenant_sums",), ("latency", "share"),
                 ("regime", "tenant_sums")):
        part = run_gpu(L, tr, tr.shape, co, tr.n_tenants, outs)
        for k in outs:
            if k == "tenant_sums":
                np.testing.assert_allclose(part[k], full[k], rtol=1e-12)
            else:
                assert np.array_equal(part[k], full[k]), (outs, k)


def test_deterministic(L):
    tr = tracegen.config_trace("decode-only", 4000)
    co = tracegen.config_coeffs("decode-only")
    a = run_gpu(L, tr, tr.shape, co, tr.n_tenants)
    b = run_gpu(L, tr, tr.shape, co, tr.n_tenants)
    for k in ("latency", "regime", "share"):
        assert np.array_equal(a[k], b[k]), k
    np.testing.assert_allclose(a["tenant_sums"], b["tenant_sums"], rtol=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_random_traces(L, seed):
    rng = np.random.default_rng(1000 + seed)
    kind = seed % 3
    nb = int(rng.integers(1, 3000))
    if kind == 0:
        sizes = rng.integers(0, 50, nb)
    elif kind == 1:
        sizes = np.minimum(rng.pareto(1.2, nb) * 30 + 1, 4000).astype(np.int64)
    else:
        sizes = rng.choice([0, 1, 2, 255, 256, 1000, 3071, 3072, 3500], nb)
    tr = random_fill(rng, sizes, n_tenants=int(rng.integers(1, 2000)))
    sh = tracegen.SHAPES[sorted(tracegen.SHAPES)[seed % 4]]
    check(L, tr, sh, tracegen.base_coeffs(40 + seed), tr.n_tenants, f"random {seed}")


# ---------------------------------------------------------------- features


@pytest.mark.parametrize("name,nb", [("tiny-mixed", None), ("heavy-tailed", 1500)])
def test_features(L, name, nb):
    import torch
    tr = tracegen.config_trace(name, nb)
    rng = np.random.default_rng(3)
    sizes = tr.sizes().copy()
    sizes[rng.integers(0, len(sizes), 20)] = 0  # some empty batches
    off = np.zeros(len(sizes) + 1, np.int64)
    off[1:] = np.cumsum(sizes)
    N = int(off[-1])
    p, c = tr.p[:N], tr.c[:N]
    for shape in (None, tr.shape):
        dt = L.DeviceTrace.from_host(off, p, c)
        xr, xb = L.features(dt, shape)
        torch.cuda.synchronize()
        rr, rb = oracle.features(off, p, c, shape)
        e_r = parity.rel_err(xr.cpu().numpy(), rr)
        e_b = parity.rel_err(xb.cpu().numpy(), rb)
        say(f"[features] {name} shape={shape is not None}: req {e_r.max():.2e} batch {e_b.max():.2e}")
        assert e_r.max() <= parity.RTOL
        assert e_b.max() <= 1e-12


@pytest.mark.parametrize("N", [14336, 14337])
def test_features_single_launch_boundary(L, N):
    """The feature rows on both sides of the single-launch boundary (two
    1792-slot tiles per wave), with batches larger than a tile among them."""
    import torch
    rng = np.random.default_rng(N)
    sizes = [2000, 0, 1792, 1793]
    while sum(sizes) < N:
        sizes.append(int(min(rng.integers(0, 500), N - sum(sizes))))
    tr = random_fill(rng, np.array(sizes), n_tenants=1)
    assert tr.n_requests == N
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c)
    shape = tracegen.SHAPES["qwen2.5-14b"]
    xr, xb = L.features(dt, shape)
    torch.cuda.synchronize()
    rr, rb = oracle.features(tr.offsets, tr.p, tr.c, shape)
    assert parity.rel_err(xr.cpu().numpy(), rr).max() <= parity.RTOL
    assert parity.rel_err(xb.cpu().numpy(), rb).max() <= 1e-12


# --------------------------------------------------------- tenant sums API


@pytest.mark.parametrize("n,T", [(0, 3), (1, 1), (12345, 16), (1_000_003, 1024), (200_000, 5000),
                                 (3_000_000, 1 << 20)])
def test_tenant_sums_standalone(L, n, T):
    import torch
    rng = np.random.default_rng(n + T)
    t = rng.integers(0, T, n).astype(np.int32)
    if T > 4096:  # skewed ids: the tenant cache's frequent and rare tenants
        t = (tracegen.zipf(n + T, 7, 0, n, T, 1.2)).astype(np.int32)
    s = (rng.random(n) * 100).astype(np.float32)
    out = L.tenant_sums(torch.from_numpy(t).cuda(), torch.from_numpy(s).cuda(), T)
    torch.cuda.synchronize()
    want = oracle.tenant_sums(t, s.astype(np.float64), T)
    e = parity.rel_err(out.cpu().numpy(), want)
    assert e.max() <= 1e-12 if e.size else True


# ---------------------------------------------------------------- validate


def test_validate(L):
    tr = tracegen.config_trace("tiny-mixed")
    ws = L.workspace(tr.n_batches, tr.n_requests, tr.n_tenants)

    def v(off, p, c, t, T=tr.n_tenants):
        return L.llmv_validate(L.DeviceTrace.from_host(off, p, c, t), T, ws)

    assert v(tr.offsets, tr.p, tr.c, tr.tenant) == L.LLMV_OK
    bad = [
        (np.concatenate([[1], tr.offsets[1:]]), tr.p, tr.c, tr.tenant),
        (tr.offsets, np.where(np.arange(len(tr.p)) == 7, 0, tr.p), tr.c, tr.tenant),
        (tr.offsets, np.where(np.arange(len(tr.p)) == 9, L.LLMV_P_MAX + 1, tr.p), tr.c, tr.tenant),
        (tr.offsets, tr.p, np.where(np.arange(len(tr.c)) == 3, -1, tr.c), tr.tenant),
        (tr.offsets, tr.p, tr.c, np.where(np.arange(len(tr.c)) == 5, tr.n_tenants, tr.tenant)),
    ]
    off2 = tr.offsets.copy()
    off2[10], off2[11] = off2[11], off2[10]  # decreasing
    bad.append((off2, tr.p, tr.c, tr.tenant))
    for i, args in enumerate(bad):
        assert v(*args) == L.LLMV_ERANGE, i
    # n_requests disagreeing with offsets[nB]
    assert v(tr.offsets[:-1], tr.p, tr.c, tr.tenant) == L.LLMV_ERANGE


# ------------------------------------------------- full-size workloads


def full_size(L, name):
    """Every output of the whole trace against the oracle: latency and regime
    of every batch, every share (copied back in slices of whole batches; each
    batch's shares also add up to its latency), every tenant sum.  Outputs
    start as NaN (regime 0xEE), so an unwritten one fails.  The traces of
    ~1e8 requests and more run the static pieces and the claimed chunks of
    the tile kernel's work split."""
    import torch
    tr = tracegen.config_trace(name)
    co = tracegen.config_coeffs(name)
    say(f"[full] {name}: nB={tr.n_batches} N={tr.n_requests}")
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    dev = dt.p.device
    lat_d = torch.full((tr.n_batches,), float("nan"), dtype=torch.float32, device=dev)
    reg_d = torch.full((tr.n_batches,), 0xEE, dtype=torch.uint8, device=dev)
    share = torch.full((tr.n_requests,), float("nan"), dtype=torch.float32, device=dev)
    ts_d = torch.full((tr.n_tenants,), float("nan"), dtype=torch.float64, device=dev)
    ws = L.workspace(tr.n_batches, tr.n_requests, tr.n_tenants)
    L.llmv_attribute(dt, tr.shape, co, lat_d, reg_d, share, tr.n_tenants, ts_d, ws)
    torch.cuda.synchronize()
    lat = lat_d.cpu().numpy()
    reg = reg_d.cpu().numpy()
    ts = ts_d.cpu().numpy()
    del dt, ws
    ref = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, tr.shape, co, tr.n_tenants,
                           ("T", "TM", "TC", "phase", "regime", "share", "tenant_sums"))
    st = parity.compare(ref, tr.offsets, lat, reg, None, ts)

    def alt_shares(bids):
        off, p, c, t = parity.sub_trace(tr.offsets, tr.p, tr.c, tr.tenant, bids)
        return oracle.attribute(off, p, c, t, tr.shape, co, tr.n_tenants,
                                ("share_alt",))["share_alt"]

    st.update(parity.compare_all_shares(tr.offsets, lambda lo, hi: share[lo:hi].cpu().numpy(),
                                        ref["share"], ref["TM"], ref["TC"], ref["regime"], reg,
                                        lat, alt_shares))
    tot = lat.astype(np.float64).sum()
    assert abs(ts.sum() - tot) / tot <= parity.RTOL
    say(f"[full] {name}: {st}")


@pytest.mark.parametrize("name", ["decode-only", "chunked-prefill", "heavy-tailed"])
def test_full_size(L, name):
    full_size(L, name)


# ---------------------------------------------------------- what-if sweep


def run_sweep(L, tr, shapes, co):
    import torch
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    out = L.attribute_sweep(dt, shapes, co, tr.n_tenants)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def test_sweep_small(L):
    tr = tracegen.config_trace("whatif-sweep", 1500)
    co = tracegen.sweep_coeffs(tracegen.config_coeffs("whatif-sweep"), 5)
    shapes = [tracegen.SHAPES[k] for k in ("llama3.1-8b", "70b-like")]
    out = run_sweep(L, tr, shapes, co)
    assert out.shape == (2, 5, tr.n_tenants)
    for s, sh in enumerate(shapes):
        for v in range(5):
            ref = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, sh, co[v], tr.n_tenants,
                                   ("tenant_sums",))["tenant_sums"]
            e = parity.rel_err(out[s, v], ref)
            assert e.max() <= parity.RTOL, (s, v, e.max())
    # single attribution calls give the same sums up to fp32 rounding: there
    # each share is 4 fp32 operations (<= 4 ulp) before the fp64 sum; the sweep
    # rounds a group's sums to fp32 (1 ulp) and evaluates k0*n + k1*P + k2*C +
    # k3*Q in 4 fp32 operations (<= 4 ulp); with nonnegative terms both stay
    # within 5 * 2^-24 of the exact sum over the same fp32 constants
    import torch
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    one = L.attribute(dt, shapes[1], co[3], tr.n_tenants, ("tenant_sums",))["tenant_sums"]
    torch.cuda.synchronize()
    np.testing.assert_allclose(out[1, 3], one.cpu().numpy(), rtol=10 * 2.0**-24)


def skewed_tenants(rng, N, T, s=1.2):
    """Tenant ids with Zipf-like skew over T ids, most frequent first (the
    top ids collect a large share, as in the what-if workload)."""
    w = 1.0 / np.arange(1, T + 1) ** s
    return rng.choice(T, N, p=w / w.sum()).astype(np.int32)


SWEEP_CASES = {
    # name: (n_tenants, skewed) -- 1024 tenants run 8 variants per pass,
    # up to 2048 four, up to 4096 two; 1 and 3 tenants have fewer tenants
    # than the replicated hot set
    "T1": (1, False),
    "T3-skewed": (3, True),
    "T1024-skewed": (1024, True),
    "T1025-uniform": (1025, False),
    "T2049-skewed": (2049, True),
    "T4096-uniform": (4096, False),
}


@pytest.mark.parametrize("case", sorted(SWEEP_CASES))
def test_sweep_tenant_counts(L, case):
    T, skewed = SWEEP_CASES[case]
    rng = np.random.default_rng(sum(map(ord, case)))
    sizes = rng.integers(0, 300, 900)
    sizes[::97] = 2000  # a few batches larger than a wave tile
    tr = random_fill(rng, sizes, n_tenants=T)
    if skewed:
        tr = tracegen.Trace(tr.offsets, tr.p, tr.c, skewed_tenants(rng, tr.n_requests, T), T, None)
    co = tracegen.sweep_coeffs(tracegen.base_coeffs(77), 11)  # 22 variants: a partial last pass
    shapes = [tracegen.SHAPES["qwen2.5-14b"], tracegen.SHAPES["llama3.1-8b"]]
    out = run_sweep(L, tr, shapes, co)
    for s_ in range(2):
        for v in range(11):
            ref = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, shapes[s_], co[v], T,
                                   ("tenant_sums",))["tenant_sums"]
            e = parity.rel_err(out[s_, v], ref)
            assert e.max() <= parity.RTOL, (case, s_, v, e.max())


@pytest.mark.parametrize("ext", [False, True])
def test_sweep_tiny_batches(L, ext):
    """Batches of 0 to 3 requests (1 to 3 groups each), so that a lane's
    run of groups spans many batches: the pass kernel reads the constants of
    a lane's first two batches ahead and every later batch inside its loop.
    Every setting's tenant sums against the oracle."""
    import torch
    rng = np.random.default_rng(404 + ext)
    sizes = rng.integers(0, 4, 6000)
    tr = random_fill(rng, sizes, n_tenants=37)
    shapes = [tracegen.SHAPES["llama3.1-8b"]]
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    if ext:
        co = np.stack([tracegen.ext_coeffs(700 + j) for j in range(9)])
        out = L.attribute_sweep(dt, shapes, co, tr.n_tenants, ext=True)
    else:
        co = tracegen.sweep_coeffs(tracegen.base_coeffs(78), 9)
        out = L.attribute_sweep(dt, shapes, co, tr.n_tenants)
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    for v in range(9):
        f = oracle.attribute_ext if ext else oracle.attribute
        ref = f(tr.offsets, tr.p, tr.c, tr.tenant, shapes[0], co[v], tr.n_tenants,
                ("tenant_sums",))["tenant_sums"]
        e = parity.rel_err(out[0, v], ref)
        assert e.max() <= parity.RTOL, (ext, v, e.max())


def test_sweep_unit_shape_and_hand_coeffs(L):
    tt = HAND["tenant_trace"]
    by = {e["name"]: e for e in HAND["unit_shape_examples"]}
    tr = tracegen.from_batches([(by[n]["p"], by[n]["c"]) for n in tt["batches"]], tt["tenants"],
                               tt["n_tenants"])
    th = coeff_vec(HAND["base_coeffs"])
    out = run_sweep(L, tr, None, np.stack([th, th]))
    assert list(out[0, 0]) == tt["tenant_sums"] and list(out[0, 1]) == tt["tenant_sums"]


def sweep_edge_trace(case):
    """Traces for the sweep's (batch, tenant) groups: batches split by the
    2048-request build slices (a 300000-request one among them), slices
    that end exactly on a batch end, empty batches at both ends, no
    requests at all, and batches with more distinct tenants than the
    per-wave hash table holds."""
    rng = np.random.default_rng(sum(map(ord, case)) + 11)
    if case == "split-batches-skewed":
        sizes = np.array([0, 0, 2048, 0, 4095, 1, 300000, 0, 0]
                         + list(rng.integers(0, 400, 500)) + [0, 0, 0])
        tr = random_fill(rng, sizes, n_tenants=1024)
        return tracegen.Trace(tr.offsets, tr.p, tr.c, skewed_tenants(rng, tr.n_requests, 1024),
                              1024, None)
    if case == "slice-aligned":
        return random_fill(rng, np.array([2048, 1024, 1024, 0, 2048, 0, 0]), n_tenants=7)
    if case == "no-requests":
        return random_fill(rng, np.zeros(40, np.int64), n_tenants=5)
    if case == "many-tenants-per-batch":
        return random_fill(rng, np.array([5000] * 40), n_tenants=4096)
    raise KeyError(case)


@pytest.mark.parametrize("case", ["split-batches-skewed", "slice-aligned", "no-requests",
                                  "many-tenants-per-batch"])
def test_sweep_group_edges(L, case):
    tr = sweep_edge_trace(case)
    co = tracegen.sweep_coeffs(tracegen.base_coeffs(78), 5)
    shapes = [tracegen.SHAPES["qwen2.5-32b"]]
    say(f"[sweep edge] {case}: nB={tr.n_batches} N={tr.n_requests} T={tr.n_tenants}")
    out = run_sweep(L, tr, shapes, co)
    for v in range(5):
        ref = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, shapes[0], co[v], tr.n_tenants,
                               ("tenant_sums",))["tenant_sums"]
        assert np.array_equal(out[0, v][ref == 0], ref[ref == 0]), (case, v)
        if tr.n_requests:
            e = parity.rel_err(out[0, v], ref)
            assert e.max() <= parity.RTOL, (case, v, e.max())


def test_sweep_refuses_a_small_workspace(L):
    """llmv_workspace_size's bytes do not hold the groups: EWORKSPACE, and
    the output is left alone."""
    import torch
    tr = tracegen.config_trace("whatif-sweep", 300)
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    co = tracegen.sweep_coeffs(tracegen.config_coeffs("whatif-sweep"), 2)
    out = torch.full((1, 2, tr.n_tenants), -1.0, dtype=torch.float64, device="cuda")
    ws = L.workspace(tr.n_batches, tr.n_requests, tr.n_tenants)
    with pytest.raises(L.LlmvError) as e:
        L.llmv_attribute_sweep(dt, [tr.shape], co, tr.n_tenants, out, ws)
    assert e.value.code == L.LLMV_EWORKSPACE
    torch.cuda.synchronize()
    assert bool((out == -1.0).all())


def test_sweep_claimed_chunks_two_passes(L):
    """The decode-only trace (1.28e8 requests) under 10 settings: the pass
    kernel's work split then has claimed chunks (a worker's share of the
    requests passes 32 narrow tiles, 49,152 requests, at 2048 wave workers
    and more), and the second pass starts at claim n_chunks.  Every setting's
    tenant sums against the oracle."""
    tr = tracegen.config_trace("decode-only")
    assert tr.n_requests > 2048 * 49152
    co = tracegen.sweep_coeffs(tracegen.config_coeffs("decode-only"), 10)
    shapes = [tracegen.SHAPES["qwen2.5-14b"]]
    say(f"[sweep] claimed chunks: N={tr.n_requests} settings=10")
    out = run_sweep(L, tr, shapes, co)
    for v in range(10):
        ref = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, shapes[0], co[v], tr.n_tenants,
                               ("tenant_sums",))["tenant_sums"]
        e = parity.rel_err(out[0, v], ref)
        say(f"[sweep] claimed chunks, setting {v}: max rel err {e.max():.2e}")
        assert e.max() <= parity.RTOL, (v, e.max())


def test_sweep_full_size_sampled(L):
    tr = tracegen.config_trace("whatif-sweep")
    co = tracegen.sweep_coeffs(tracegen.config_coeffs("whatif-sweep"), 256)
    names = ["llama3.1-8b", "qwen2.5-14b", "qwen2.5-32b", "70b-like"]
    shapes = [tracegen.SHAPES[k] for k in names]
    say(f"[sweep] N={tr.n_requests} variants={4 * 256}")
    out = run_sweep(L, tr, shapes, co)
    assert np.all(np.isfinite(out))
    for s, v in [(0, 0), (1, 17), (2, 128), (3, 255), (3, 1), (0, 200)]:
        ref = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, shapes[s], co[v], tr.n_tenants,
                               ("tenant_sums",))["tenant_sums"]
        e = parity.rel_err(out[s, v], ref)
        say(f"[sweep] shape {names[s]} variant {v}: max rel err {e.max():.2e}")
        assert e.max() <= parity.RTOL
