"""GPU parity of llmv_attribute_ext (the extended model: Eq. 1 plus the
cross term a5*S5*sum p*c and the per-request term a6*S6*|B|) through the C
ABI, against orc_attribute_ext, under the rules of parity.py.  Plus the
reduction to llmv_attribute: with a5 = a6 = 0 latency, regime and shares are
bit-identical to the Eq. 1 path's, and tenant sums equal up to the order of
their fp64 additions (LDS atomics of four waves, claimed chunks)."""
import json
import os
import sys

import numpy as np
import pytest

import oracle
import parity
import tracegen

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
from test_gpu_parity import SIZE_SETS, random_fill  # noqa: E402

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXT = json.load(open(os.path.join(ROOT, "tests", "golden", "ext_examples.json")))
SETS = ("prefill_mem", "prefill_comp", "decode_mem", "decode_comp")
OUTS = ("latency", "regime", "share", "tenant_sums")


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


def coeffs28(sets):
    th = np.zeros(28, np.float32)
    for g, name in enumerate(SETS):
        if name in sets:
            th[g * 7:(g + 1) * 7] = sets[name]
    return th


def widen(co20):
    th = np.zeros(28, np.float32)
    for g in range(4):
        th[g * 7:g * 7 + 5] = co20[g * 5:(g + 1) * 5]
    return th


def run(L, tr, shape, coeffs, n_tenants, outputs=OUTS, ext=True):
    import torch
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c,
                                 tr.tenant if "tenant_sums" in outputs else None)
    fn = L.attribute_ext if ext else L.attribute
    out = fn(dt, shape, coeffs, n_tenants, outputs)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def check(L, tr, shape, coeffs, n_tenants, name="", outputs=OUTS):
    say(f"[ext] {name}: nB={tr.n_batches} N={tr.n_requests} T={n_tenants} outputs={outputs}")
    g = run(L, tr, shape, coeffs, n_tenants, outputs)
    ref = oracle.attribute_ext(tr.offsets, tr.p, tr.c, tr.tenant, shape, coeffs, n_tenants)
    st = parity.compare(ref, tr.offsets, g.get("latency"), g.get("regime"), g.get("share"),
                        g.get("tenant_sums"))
    return st, g, ref


def test_hand_examples_exact(L):
    for ex in EXT["unit_shape_examples"]:
        tr = tracegen.from_batches([(ex["p"], ex["c"])], [[0] * len(ex["p"])], 1)
        g = run(L, tr, None, coeffs28(ex["sets"]), 1)
        say(f"[ext hand] {ex['name']}")
        assert g["latency"][0] == ex["T"] and g["regime"][0] == ex["regime"], ex["name"]
        assert list(g["share"]) == ex["shares"], ex["name"]
        assert g["tenant_sums"][0] == sum(ex["shares"]), ex["name"]
    sh = EXT["shaped"]
    for ex in sh["examples"]:
        tr = tracegen.from_batches([(ex["p"], ex["c"])], [[0] * len(ex["p"])], 1)
        g = run(L, tr, sh["shape"], coeffs28(sh["sets"]), 1)
        assert g["latency"][0] == ex["T"] and g["regime"][0] == ex["regime"]
        assert list(g["share"]) == ex["shares"]


@pytest.mark.parametrize("name,nb", [("tiny-mixed", None), ("chunked-prefill", 2000),
                                     ("heavy-tailed", 3000), ("decode-only", 3000)])
def test_zero_extension_is_the_eq1_path(L, name, nb):
    """a5 = a6 = 0: every share and batch output bit-identical to
    llmv_attribute's; every tenant sum adds the same fp32 shares in fp64, in
    an order that may differ between launches."""
    tr = tracegen.config_trace(name, nb)
    co = tracegen.config_coeffs(name)
    a = run(L, tr, tr.shape, co, tr.n_tenants, ext=False)
    b = run(L, tr, tr.shape, widen(co), tr.n_tenants)
    for k in ("latency", "regime", "share"):
        assert np.array_equal(a[k], b[k]), k
    np.testing.assert_allclose(b["tenant_sums"], a["tenant_sums"], rtol=1e-12, atol=0)


@pytest.mark.parametrize("name,nb", [("tiny-mixed", None), ("chunked-prefill", 2000),
                                     ("heavy-tailed", 3000), ("decode-only", 3000),
                                     ("whatif-sweep", 2000)])
def test_config_recipes(L, name, nb):
    tr = tracegen.config_trace(name, nb)
    co = tracegen.ext_coeffs(100 + tracegen.CONFIG_SEED[name])
    st, g, ref = check(L, tr, tr.shape, co, tr.n_tenants, name)
    say(f"[ext] {name}: {st}")
    assert len(set(g["regime"].tolist())) >= 2


@pytest.mark.parametrize("key", sorted(SIZE_SETS))
def test_batch_size_edges(L, key):
    """Wave and tile edges, the two-pass path for batches larger than a
    tile, ragged and unaligned sizes; prefill batches carry a context."""
    rng = np.random.default_rng(hash(key) % 1000 + 7)
    tr = random_fill(rng, SIZE_SETS[key])
    tr.c = np.where(tr.c == 0, rng.integers(0, 3000, tr.n_requests), tr.c).astype(np.int32)
    for shape in (None, tracegen.SHAPES["qwen2.5-32b"]):
        st, _, _ = check(L, tr, shape, tracegen.ext_coeffs(41), tr.n_tenants, key)
        say(f"[ext edge] {key}: {st}")


@pytest.mark.parametrize("outputs", [("latency", "regime"), ("share",), ("tenant_sums",),
                                     ("latency", "share"), OUTS])
@pytest.mark.parametrize("n_tenants", [3, 5000])
def test_output_subsets(L, outputs, n_tenants):
    """Every kernel instance: with and without shares, no tenant sums, LDS
    (<= 4096 tenants) and global-atomic tenant sums."""
    rng = np.random.default_rng(n_tenants + len(outputs))
    tr = random_fill(rng, rng.integers(0, 300, 400), n_tenants=n_tenants)
    st, _, _ = check(L, tr, tracegen.SHAPES["llama3.1-8b"], tracegen.ext_coeffs(42), n_tenants,
                     f"subset {outputs}", outputs)
    say(f"[ext subset] {st}")


@pytest.mark.parametrize("pattern", ["all-empty", "no-batches", "interleaved"])
def test_empty_batches(L, pattern):
    rng = np.random.default_rng(13)
    if pattern == "all-empty":
        sizes = [0] * 500
    elif pattern == "no-batches":
        sizes = []
    else:
        sizes = [int(x) if i % 2 else 0 for i, x in enumerate(rng.integers(1, 50, 600))]
    tr = random_fill(rng, np.array(sizes, np.int64))
    check(L, tr, None, tracegen.ext_coeffs(43), tr.n_tenants, pattern)


@pytest.mark.parametrize("N", [1, 12289, 14335, 14336, 14337])
def test_single_launch_boundary(L, N):
    rng = np.random.default_rng(N + 5)
    sizes = []
    while sum(sizes) < N:
        sizes.append(int(min(rng.integers(0, 400), N - sum(sizes))))
    tr = random_fill(rng, sizes)
    check(L, tr, tracegen.SHAPES["qwen2.5-14b"], tracegen.ext_coeffs(44), tr.n_tenants, f"N={N}")


def test_large_cross_products(L):
    """p*c near 2^51 per request: the batch sums of p*c stay exact (uint64)
    and convert to fp64 as the oracle's int64 do."""
    big = (2**20, 2**31 - 1)
    batches = [([big[0]] * 4, [big[1]] * 4), ([big[0], 1, 3], [big[1], 5, 2**30]),
               ([2**19] * 1000, [2**31 - 1] * 1000)]
    tr = tracegen.from_batches(batches, [[0] * len(b[0]) for b in batches], 1)
    check(L, tr, None, tracegen.ext_coeffs(45), 1, "large p*c")


def test_full_size_sampled(L):
    """The 1M-batch chunked-prefill workload (2.2e8 requests), where prefill
    chunks carry cached prefixes: latency, regime and tenant sums of every
    batch and tenant; shares of sampled batches."""
    import torch
    tr = tracegen.config_trace("chunked-prefill")
    co = tracegen.ext_coeffs(103)
    say(f"[ext full] chunked-prefill: nB={tr.n_batches} N={tr.n_requests}")
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    out = L.attribute_ext(dt, tr.shape, co, tr.n_tenants)
    torch.cuda.synchronize()
    lat, reg = out["latency"].cpu().numpy(), out["regime"].cpu().numpy()
    ts = out["tenant_sums"].cpu().numpy()
    share = out["share"]
    assert not bool(torch.isnan(share).any())
    rng = np.random.default_rng(17)
    bids = np.unique(np.concatenate([rng.integers(0, tr.n_batches, 1500), np.arange(3),
                                     tr.n_batches - 1 - np.arange(3)]))
    idx = np.concatenate([np.arange(tr.offsets[b], tr.offsets[b + 1]) for b in bids])
    g_share = np.zeros(tr.n_requests, np.float32)
    g_share[idx] = share[torch.from_numpy(idx).cuda()].cpu().numpy()
    del share, out, dt
    torch.cuda.empty_cache()
    off, p, c, t = parity.sub_trace(tr.offsets, tr.p, tr.c, tr.tenant, bids)
    ref = oracle.attribute_ext(off, p, c, t, tr.shape, co, tr.n_tenants,
                               ("T", "TM", "TC", "phase", "regime", "share", "share_alt"))
    st = parity.compare(ref, tr.offsets, lat, reg, g_share, None, batch_ids=bids)
    ref_all = oracle.attribute_ext(tr.offsets, tr.p, tr.c, tr.tenant, tr.shape, co, tr.n_tenants,
                                   ("T", "TM", "TC", "phase", "regime", "tenant_sums"))
    st["all_batches"] = parity.compare(ref_all, tr.offsets, lat, reg, None, ts)
    say(f"[ext full] {st}")
