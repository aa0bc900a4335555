"""Pins of the extended-model oracle (orc_attribute_ext; no GPU).

The extended model adds two features the paper leaves open to Eq. 1: the
cross term sum p*c (a chunk attending to its cached prefix) and a
per-request term |B| (the output projection, or with the unit shape the
other reading of Eq. 1's a4 term).  The pins: hand-worked batches
(tests/golden/ext_examples.json), brute-force FLOP counts for the two new
constants, the reduction to Eq. 1 when the new coefficients are zero,
closed-form special cases and invariants.
"""
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle
import tracegen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXT = json.load(open(os.path.join(ROOT, "tests", "golden", "ext_examples.json")))
SETS = ("prefill_mem", "prefill_comp", "decode_mem", "decode_comp")


def coeffs28(sets):
    th = np.zeros(28, np.float32)
    for g, name in enumerate(SETS):
        if name in sets:
            th[g * 7:(g + 1) * 7] = sets[name]
    return th


def widen(co20, a5=None, a6=None):
    """28 coefficients from Eq. 1's 20 plus optional a5, a6 per set."""
    th = np.zeros(28, np.float32)
    for g in range(4):
        th[g * 7:g * 7 + 5] = co20[g * 5:(g + 1) * 5]
        if a5 is not None:
            th[g * 7 + 5] = a5[g]
        if a6 is not None:
            th[g * 7 + 6] = a6[g]
    return th


def one_batch(p, c):
    return np.array([0, len(p)], np.int64), np.array(p, np.int32), np.array(c, np.int32)


@pytest.mark.parametrize("ex", EXT["unit_shape_examples"], ids=lambda e: e["name"][:2])
def test_hand_examples_unit_shape(ex):
    off, p, c = one_batch(ex["p"], ex["c"])
    r = oracle.attribute_ext(off, p, c, None, None, coeffs28(ex["sets"]), 0,
                             ("T", "regime", "share"))
    assert r["T"][0] == ex["T"] and r["regime"][0] == ex["regime"]
    assert list(r["share"]) == ex["shares"]


def test_hand_examples_shaped():
    sh = EXT["shaped"]
    assert list(oracle.shape_constants_ext(sh["shape"])) == sh["S"]
    for ex in sh["examples"]:
        off, p, c = one_batch(ex["p"], ex["c"])
        r = oracle.attribute_ext(off, p, c, None, sh["shape"], coeffs28(sh["sets"]), 0,
                                 ("T", "regime", "share"))
        assert r["T"][0] == ex["T"] and r["regime"][0] == ex["regime"]
        assert list(r["share"]) == ex["shares"]


def brute_pair_flops(shape):
    """FLOPs for one processed token against one cached key, counted matrix
    element by matrix element: per layer and query head, the score is a
    head_dim-long dot product (a multiply and an add per element) and the
    value mix a head_dim-long multiply-add."""
    total = 0
    for _layer in range(shape["n_layers"]):
        for _head in range(shape["n_q_heads"]):
            for _e in range(shape["head_dim"]):
                total += 2  # score: q[e] * k[e], accumulated
                total += 2  # output: prob * v[e], accumulated
    return total


def brute_logit_flops(shape):
    """FLOPs of one position's logits: every vocab row dotted with the
    hidden state."""
    return sum(2 * shape["hidden"] for _ in range(shape["vocab"]))


@pytest.mark.parametrize("name", sorted(tracegen.SHAPES))
def test_new_constants_brute_force(name):
    sh = dict(tracegen.SHAPES[name])
    S = oracle.shape_constants_ext(sh)
    assert list(S[:4]) == list(oracle.shape_constants(sh))
    small = dict(sh, n_layers=2, n_q_heads=3, head_dim=5, vocab=7, hidden=11)
    Ss = oracle.shape_constants_ext(small)
    assert Ss[4] == brute_pair_flops(small)
    assert Ss[5] == brute_logit_flops(small)
    # the causal p^2 constant counts half of the pairs of a block
    assert S[4] == 2 * S[3]


def test_llama_constants():
    S = oracle.shape_constants_ext(tracegen.SHAPES["llama3.1-8b"])
    assert S[4] == EXT["llama3_1_8b"]["S5"] and S[5] == EXT["llama3_1_8b"]["S6"]


ALL = ("T", "TM", "TC", "phase", "regime", "share", "share_alt", "tenant_sums")


@pytest.mark.parametrize("name,nb", [("tiny-mixed", None), ("chunked-prefill", 300),
                                     ("decode-only", 500), ("heavy-tailed", 2000)])
def test_reduces_to_eq1(name, nb):
    """With a5 = a6 = 0 every added term is an exact zero: bit-identical to
    the Eq. 1 oracle, every output."""
    tr = tracegen.config_trace(name, nb)
    co = tracegen.config_coeffs(name)
    a = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, tr.shape, co, tr.n_tenants, ALL)
    b = oracle.attribute_ext(tr.offsets, tr.p, tr.c, tr.tenant, tr.shape, widen(co),
                             tr.n_tenants, ALL)
    for k in ALL:
        assert np.array_equal(a[k], b[k]), k


def test_per_request_term_is_the_other_a4_reading():
    """Unit shape, a4 = 0, a6 = a in both segments of a phase: each batch
    gains a*|B| in both segments (so the segment is unchanged) and each
    request gains a."""
    tr = tracegen.config_trace("tiny-mixed")
    co = tracegen.config_coeffs("tiny-mixed").copy()
    for g in range(4):
        co[g * 5 + 4] = 0.0
    a = np.float32(0.375)
    base = oracle.attribute(tr.offsets, tr.p, tr.c, None, None, co, 0, ("T", "regime", "share"))
    ext = oracle.attribute_ext(tr.offsets, tr.p, tr.c, None, None, widen(co, a6=[a] * 4), 0,
                               ("T", "regime", "share"))
    n = np.diff(tr.offsets).astype(np.float64)
    assert np.array_equal(base["regime"], ext["regime"])
    assert np.allclose(ext["T"], base["T"] + a * n, rtol=1e-14, atol=0)
    assert np.allclose(ext["share"], base["share"] + a, rtol=1e-14, atol=0)


def test_cross_term_in_decode_is_the_c_term():
    """In decode every p is 1, so sum p*c = sum c: (a2, a5) acts as
    a2 + a5*S5/S2 with a5 = 0 (unit shape: a2 + a5)."""
    tr = tracegen.config_trace("decode-only", 400)
    co = tracegen.config_coeffs("decode-only").astype(np.float64)
    co = (co * 1e3).astype(np.float32)  # keep the added terms well above rounding
    co[10 + 2], co[15 + 2] = 0.25, 0.25  # decode a2 (sums below are exact in fp32)
    a5 = np.array([0, 0, 0.25, 0.5], np.float32)
    ext = oracle.attribute_ext(tr.offsets, tr.p, tr.c, None, None, widen(co, a5=a5), 0,
                               ("T", "share"))
    co2 = co.copy()
    co2[10 + 2], co2[15 + 2] = 0.5, 0.75
    base = oracle.attribute(tr.offsets, tr.p, tr.c, None, None, co2, 0, ("T", "share"))
    assert np.allclose(ext["T"], base["T"], rtol=1e-13, atol=0)
    assert np.allclose(ext["share"], base["share"], rtol=1e-13, atol=0)


def rand_coeffs(rng):
    return (rng.uniform(0.0, 2.0, 28) * rng.choice([0, 1e-3, 1.0], 28)).astype(np.float32)


@settings(max_examples=60, deadline=None)
@given(st.integers(0, 2**31 - 1))
def test_invariants(seed):
    """Additivity, nonnegativity, T = max(T_M, T_C) with ties to MEM,
    reparameterisation (shape, theta) = (unit, theta * S)."""
    rng = np.random.default_rng(seed)
    batches = []
    for _ in range(int(rng.integers(1, 12))):
        n = int(rng.integers(0, 9))
        batches.append((rng.integers(1, 300, n).tolist(), rng.integers(0, 5000, n).tolist()))
    tr = tracegen.from_batches(batches, None, 1)
    th = rand_coeffs(rng)
    sh = tracegen.SHAPES["qwen2.5-14b"]
    r = oracle.attribute_ext(tr.offsets, tr.p, tr.c, None, sh, th, 0, ("T", "TM", "TC", "share"))
    sums = np.add.reduceat(np.append(r["share"], 0.0), tr.offsets[:-1]) * (np.diff(tr.offsets) > 0)
    assert np.allclose(sums, r["T"], rtol=1e-12, atol=0)
    assert (r["share"] >= 0).all()
    assert np.array_equal(r["T"], np.where(r["TC"] > r["TM"], r["TC"], r["TM"]))
    S = oracle.shape_constants_ext(sh)
    scale = np.array([S[0], S[1], S[2], S[3], 1.0, S[4], S[5]])
    th_unit = (th.astype(np.float64).reshape(4, 7) * scale).reshape(28)
    # unit-shape theta*S is not an fp32 vector: compare through features
    X = []
    for b in range(tr.n_batches):
        lo, hi = tr.offsets[b], tr.offsets[b + 1]
        p, c = tr.p[lo:hi].astype(np.int64), tr.c[lo:hi].astype(np.int64)
        n = hi - lo
        X.append([1.0, p.sum(), c.sum(), (p * p).sum(), n * n, (p * c).sum(), n])
    X = np.array(X, np.float64)
    ph = oracle.attribute(tr.offsets, tr.p, tr.c, None, None, np.zeros(20, np.float32), 0,
                          ("phase",))["phase"]
    for b in range(tr.n_batches):
        if ph[b] == 255:
            assert r["T"][b] == 0.0
            continue
        tm = X[b] @ th_unit[(ph[b] * 2) * 7:(ph[b] * 2 + 1) * 7]
        tc = X[b] @ th_unit[(ph[b] * 2 + 1) * 7:(ph[b] * 2 + 2) * 7]
        assert abs(r["TM"][b] - tm) <= 1e-12 * max(abs(tm), 1e-300)
        assert abs(r["TC"][b] - tc) <= 1e-12 * max(abs(tc), 1e-300)


def test_cross_sum_limit():
    """A batch whose sum of p*c reaches 2^63 is refused (ORC_ERANGE)."""
    n = 5000
    off, p, c = one_batch([2**20] * n, [2**31 - 1] * n)
    with pytest.raises(RuntimeError):
        oracle.attribute_ext(off, p, c, None, None, np.ones(28, np.float32), 0, ("T",))
    off, p, c = one_batch([2**20] * 4000, [2**31 - 1] * 4000)  # 2^62.97: accepted
    oracle.attribute_ext(off, p, c, None, None, np.ones(28, np.float32), 0, ("T",))
