"""llmv_attribute_host (the library's single-step attributor on host arrays)
against the oracle: exact on the hand-worked batches, within the parity rules
on the workload recipes and random steps, and its argument and data checks.
It runs on the CPU; the GPU tests hold it bit for bit against the GPU."""
import json
import os

import numpy as np
import pytest

import oracle
import parity
import tracegen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HAND = json.load(open(os.path.join(ROOT, "tests", "golden", "hand_examples.json")))


@pytest.fixture(scope="module")
def L():
    from paper_2608_08382_amd import llmv
    llmv.load()
    return llmv


def coeff_vec(d):
    return np.array(d["prefill_mem"] + d["prefill_comp"] + d["decode_mem"] + d["decode_comp"],
                    np.float32)


def host(L, tr, shape, coeffs, n_tenants, outputs=("latency", "regime", "share", "tenant_sums")):
    return L.llmv_attribute_host(tr.offsets, tr.p, tr.c, tr.tenant, shape, coeffs, n_tenants,
                                 outputs)


def test_hand_examples_exact(L):
    th = coeff_vec(HAND["base_coeffs"])
    for ex in HAND["unit_shape_examples"]:
        t = th.copy()
        if ex["coeff_override"]:
            t[ex["coeff_override"]["index"]] = ex["coeff_override"]["value"]
        tr = tracegen.from_batches([(ex["p"], ex["c"])], [[0] * len(ex["p"])], 1)
        g = host(L, tr, None, t, 1)
        assert g["latency"][0] == ex["T"], ex["name"]
        assert g["regime"][0] == ex["regime"], ex["name"]
        assert list(g["share"]) == ex["shares"], ex["name"]
        assert g["tenant_sums"][0] == sum(ex["shares"]), ex["name"]
    se = HAND["shaped_examples"]
    for ex in se["examples"]:
        tr = tracegen.from_batches([(ex["p"], ex["c"])], [[0] * len(ex["p"])], 1)
        g = host(L, tr, se["shape"], coeff_vec(se["coeffs"]), 1)
        assert g["latency"][0] == ex["T"] and g["regime"][0] == ex["regime"], ex["name"]
        assert list(g["share"]) == ex["shares"], ex["name"]


def test_hand_tenant_trace_exact(L):
    tt = HAND["tenant_trace"]
    by = {e["name"]: e for e in HAND["unit_shape_examples"]}
    tr = tracegen.from_batches([(by[n]["p"], by[n]["c"]) for n in tt["batches"]], tt["tenants"],
                               tt["n_tenants"])
    g = host(L, tr, None, coeff_vec(HAND["base_coeffs"]), tt["n_tenants"])
    assert list(g["tenant_sums"]) == tt["tenant_sums"]
    assert list(g["latency"]) == [by[n]["T"] for n in tt["batches"]]


@pytest.mark.parametrize("name,nb", [("tiny-mixed", None), ("decode-only", 40),
                                     ("chunked-prefill", 30), ("heavy-tailed", 60)])
def test_recipes_against_oracle(L, name, nb):
    tr = tracegen.config_trace(name, nb)
    co = tracegen.config_coeffs(name)
    g = host(L, tr, tr.shape, co, tr.n_tenants)
    ref = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, tr.shape, co, tr.n_tenants)
    parity.compare(ref, tr.offsets, g["latency"], g["regime"], g["share"], g["tenant_sums"])


@pytest.mark.parametrize("seed", range(4))
def test_random_steps(L, seed):
    rng = np.random.default_rng(300 + seed)
    sizes = rng.integers(0, 300, int(rng.integers(1, 20)))
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    N = int(off[-1])
    pre = rng.random(len(sizes)) < 0.4
    p = np.ones(N, np.int32)
    c = rng.integers(1, 1 << 17, N).astype(np.int32)
    for b in np.nonzero(pre)[0]:
        p[off[b]:off[b + 1]] = rng.integers(1, 4000, sizes[b])
        c[off[b]:off[b + 1]] = 0
    T = int(rng.integers(1, 50))
    t = rng.integers(0, T, N).astype(np.int32)
    tr = tracegen.Trace(off, p, c, t, T, None)
    sh = tracegen.SHAPES[sorted(tracegen.SHAPES)[seed % 4]]
    co = tracegen.base_coeffs(50 + seed)
    g = host(L, tr, sh, co, T)
    ref = oracle.attribute(off, p, c, t, sh, co, T)
    parity.compare(ref, off, g["latency"], g["regime"], g["share"], g["tenant_sums"])
    # outputs are independent of the others being requested
    part = host(L, tr, sh, co, T, ("share",))
    assert np.array_equal(part["share"], g["share"])


def test_empty_and_degenerate(L):
    co = tracegen.base_coeffs(60)
    # no batches at all
    g = host(L, tracegen.Trace(np.zeros(1, np.int64), np.zeros(0, np.int32),
                               np.zeros(0, np.int32), np.zeros(0, np.int32), 3, None), None, co, 3)
    assert g["latency"].size == 0 and np.all(g["tenant_sums"] == 0)
    # only empty batches
    tr = tracegen.Trace(np.zeros(6, np.int64), np.zeros(0, np.int32), np.zeros(0, np.int32),
                        np.zeros(0, np.int32), 2, None)
    g = host(L, tr, None, co, 2)
    assert np.all(g["latency"] == 0) and np.all(g["regime"] == 255)
    # largest p and c over one batch
    tr = tracegen.from_batches([([1 << 20] * 5, [(1 << 31) - 1] * 5)], [[0] * 5], 1)
    g = host(L, tr, tracegen.SHAPES["70b-like"], co, 1)
    ref = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, tracegen.SHAPES["70b-like"], co, 1)
    parity.compare(ref, tr.offsets, g["latency"], g["regime"], g["share"], g["tenant_sums"])


def test_refuses_bad_arguments_and_data(L):
    co = tracegen.base_coeffs(61)
    tr = tracegen.from_batches([([1, 1], [5, 6])], [[0, 1]], 2)

    def code(offsets=tr.offsets, p=tr.p, c=tr.c, t=tr.tenant, T=2, coeffs=co):
        with pytest.raises(L.LlmvError) as e:
            L.llmv_attribute_host(offsets, p, c, t, None, coeffs, T)
        return e.value.code

    # n_tenants 0 with a tenant-sum output (through the C entry point itself)
    import ctypes
    lib = L.load()
    off, p, c, t = (np.ascontiguousarray(a) for a in (tr.offsets, tr.p, tr.c, tr.tenant))
    ptr = lambda a: ctypes.c_void_p(a.ctypes.data)  # noqa: E731
    out = np.zeros(4, np.float64)
    st = L.llmv_trace(1, 2, ptr(off), ptr(p), ptr(c), ptr(t))
    cof = (ctypes.c_float * 20)(*[float(v) for v in co])
    assert lib.llmv_attribute_host(ctypes.byref(st), None, cof, None, None, None, 0,
                                   ptr(out)) == L.LLMV_EINVAL
    assert lib.llmv_attribute_host(None, None, cof, None, None, None, 0, None) == L.LLMV_EINVAL
    bad = co.copy()
    bad[3] = np.nan
    assert code(coeffs=bad) == L.LLMV_EINVAL
    assert code(p=np.array([0, 1], np.int32)) == L.LLMV_ERANGE
    assert code(p=np.array([1, (1 << 20) + 1], np.int32)) == L.LLMV_ERANGE
    assert code(c=np.array([-1, 1], np.int32)) == L.LLMV_ERANGE
    assert code(t=np.array([0, 2], np.int32)) == L.LLMV_ERANGE
    assert code(offsets=np.array([1, 2], np.int64)) == L.LLMV_ERANGE
    assert code(offsets=np.array([0, 3], np.int64)) == L.LLMV_ERANGE
