"""Pins for the CPU oracle (no GPU).

The oracle is checked against things fixed from outside its own code:
hand-worked batches (tests/golden/hand_examples.json), published model
parameter counts (tests/golden/model_shapes.json), brute-force counts of
FLOPs and bytes, special cases that reduce to plain numpy reductions, and
closed-form invariants of Eq. 1 (LLMVisor Sec. 2.1) and of the additive
attribution (Sec. 2, Problem formulation).
"""
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st, HealthCheck

import oracle
import tracegen

GOLD = os.path.join(os.path.dirname(__file__), "golden")
HAND = json.load(open(os.path.join(GOLD, "hand_examples.json")))
SHAPE_PINS = json.load(open(os.path.join(GOLD, "model_shapes.json")))

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def coeff_vec(d):
    return np.array(d["prefill_mem"] + d["prefill_comp"] + d["decode_mem"] + d["decode_comp"],
                    np.float32)


def one_batch(p, c):
    off = np.array([0, len(p)], np.int64)
    return off, np.array(p, np.int32), np.array(c, np.int32)


# --------------------------------------------------------------------------
# Hand-worked batches


@pytest.mark.parametrize("ex", HAND["unit_shape_examples"], ids=lambda e: e["name"])
def test_hand_examples_unit_shape(ex):
    th = coeff_vec(HAND["base_coeffs"])
    if ex["coeff_override"]:
        th[ex["coeff_override"]["index"]] = ex["coeff_override"]["value"]
    off, p, c = one_batch(ex["p"], ex["c"])
    r = oracle.attribute(off, p, c, np.zeros(len(p), np.int32), None, th, 1)
    assert r["T"][0] == ex["T"]
    assert r["TM"][0] == ex["T_mem"]
    assert r["TC"][0] == ex["T_comp"]
    assert r["phase"][0] == ex["phase"]
    assert r["regime"][0] == ex["regime"]
    assert list(r["share"]) == ex["shares"]
    # fp32 rounding of an exact binary fraction is exact
    assert list(r["share"].astype(np.float32)) == ex["shares"]


def test_hand_tenant_trace():
    tt = HAND["tenant_trace"]
    by_name = {e["name"]: e for e in HAND["unit_shape_examples"]}
    batches = [(by_name[n]["p"], by_name[n]["c"]) for n in tt["batches"]]
    tr = tracegen.from_batches(batches, tt["tenants"], tt["n_tenants"])
    th = coeff_vec(HAND["base_coeffs"])
    r = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, None, th, tr.n_tenants)
    assert list(r["tenant_sums"]) == tt["tenant_sums"]
    assert list(r["T"]) == [by_name[n]["T"] for n in tt["batches"]]
    assert list(r["regime"]) == [by_name[n]["regime"] for n in tt["batches"]]
    # standalone tenant sums of the same shares agree exactly
    assert list(oracle.tenant_sums(tr.tenant, r["share"], tr.n_tenants)) == tt["tenant_sums"]


def test_hand_shaped_examples():
    se = HAND["shaped_examples"]
    assert list(oracle.shape_constants(se["shape"])) == se["S"]
    th = coeff_vec(se["coeffs"])
    for ex in se["examples"]:
        off, p, c = one_batch(ex["p"], ex["c"])
        r = oracle.attribute(off, p, c, np.zeros(len(p), np.int32), se["shape"], th, 1)
        assert r["T"][0] == ex["T"], ex["name"]
        assert r["TM"][0] == ex["T_mem"], ex["name"]
        assert r["TC"][0] == ex["T_comp"], ex["name"]
        assert r["regime"][0] == ex["regime"], ex["name"]
        assert list(r["share"]) == ex["shares"], ex["name"]


# --------------------------------------------------------------------------
# Shape constants against published counts and brute-force counts


def test_shape_constants_llama_published():
    pin = SHAPE_PINS["llama3_1_8b"]
    sh = tracegen.SHAPES["llama3.1-8b"]
    S = oracle.shape_constants(sh)
    h, L, V = sh["hidden"], sh["n_layers"], sh["vocab"]
    embedding = V * h
    norms = (2 * L + 1) * h
    streamed_params = pin["total_parameters"] - embedding - norms
    assert S[0] == sh["weight_bytes"] * streamed_params
    # linear FLOPs per token: 2 per weight of the decoder layers (output
    # projection excluded: it runs once per request, not per token)
    layer_params = (streamed_params - V * h)
    assert S[1] == 2 * layer_params
    assert S[2] == pin["kv_cache_bytes_per_token_bf16"]


def _matrices(sh):
    """(rows, cols) of every weight matrix of one decoder layer."""
    h, d = sh["hidden"], sh["head_dim"]
    return [(h, sh["n_q_heads"] * d),   # q
            (h, sh["n_kv_heads"] * d),  # k
            (h, sh["n_kv_heads"] * d),  # v
            (sh["n_q_heads"] * d, h),   # o
            (h, sh["ffn"]),             # gate
            (h, sh["ffn"]),             # up
            (sh["ffn"], h)]             # down


def _attention_flops(sh, p):
    """Brute force: FLOPs of causal self-attention over a block of p tokens,
    counting every (query, key<=query) pair: q.k and the weighted value add
    are head_dim multiply-adds each, per head, per layer."""
    pairs = sum(q + 1 for q in range(p))
    return pairs * sh["n_layers"] * sh["n_q_heads"] * 2 * (2 * sh["head_dim"])


def _check_shape(sh):
    S = oracle.shape_constants(sh)
    per_layer = sum(r * c for r, c in _matrices(sh))
    L = sh["n_layers"]
    assert S[0] == sh["weight_bytes"] * (L * per_layer + sh["vocab"] * sh["hidden"])
    assert S[1] == 2 * L * per_layer
    kv_per_token = sum(sh["n_kv_heads"] * sh["head_dim"] for _ in ("K", "V")) * L
    assert S[2] == kv_per_token * sh["kv_bytes"]
    # p^2 coefficient of the brute-force count F(p) = a p^2 + b p
    F1, F2 = _attention_flops(sh, 1), _attention_flops(sh, 2)
    a = (F2 - 2 * F1) / 2
    assert S[3] == a
    assert _attention_flops(sh, 7) == a * 49 + (F1 - a) * 7


@pytest.mark.parametrize("name", sorted(tracegen.SHAPES))
def test_shape_constants_bruteforce(name):
    _check_shape(tracegen.SHAPES[name])


@settings(max_examples=40, deadline=None)
@given(st.lists(st.integers(1, 64), min_size=9, max_size=9))
def test_shape_constants_bruteforce_random(v):
    sh = dict(zip(tracegen.SHAPE_FIELDS, v))
    _check_shape(sh)


def test_shape_constants_reject_bad():
    sh = dict(tracegen.SHAPES["llama3.1-8b"])
    for f in tracegen.SHAPE_FIELDS:
        bad = dict(sh)
        bad[f] = 0
        with pytest.raises(oracle.OracleError):
            oracle.shape_constants(bad)


def test_unit_shape_is_one():
    assert list(oracle.shape_constants(None)) == [1, 1, 1, 1]


# --------------------------------------------------------------------------
# Special cases that reduce to plain reductions: one unit coefficient


def random_trace(rng, nB=40, max_n=12, with_empty=True):
    sizes = rng.integers(0 if with_empty else 1, max_n + 1, nB)
    off = np.zeros(nB + 1, np.int64)
    off[1:] = np.cumsum(sizes)
    N = int(off[-1])
    p = np.where(rng.random(N) < 0.5, 1, rng.integers(1, 3000, N)).astype(np.int32)
    c = np.where(rng.random(N) < 0.3, 0, rng.integers(0, 100000, N)).astype(np.int32)
    t = rng.integers(0, 7, N).astype(np.int32)
    return off, p, c, t


@pytest.mark.parametrize("k", range(5))
@pytest.mark.parametrize("shape", [None, "llama3.1-8b", "qwen2.5-32b"])
def test_single_term_reduces_to_sum(k, shape):
    rng = np.random.default_rng(10 + k)
    off, p, c, t = random_trace(rng)
    sh = None if shape is None else tracegen.SHAPES[shape]
    S = [1, 1, 1, 1] if sh is None else oracle.shape_constants(sh)
    th = np.zeros(20, np.float32)
    for grp in range(4):
        th[grp * 5 + k] = 1.0
    r = oracle.attribute(off, p, c, t, sh, th, 7)
    sizes = np.diff(off)
    nz = sizes > 0
    p64, c64 = p.astype(np.float64), c.astype(np.float64)
    raw = [np.ones_like(p64), p64, c64, p64 * p64]
    if k < 4:
        seg = np.add.reduceat(raw[k], off[:-1][nz]) if len(p) else np.zeros(0)
        expect = np.zeros(len(sizes))
        expect[nz] = S[k] * seg if k > 0 else S[0]
    else:
        expect = sizes.astype(np.float64) ** 2
    np.testing.assert_allclose(r["T"], expect, rtol=1e-15, atol=0)
    n_of = np.repeat(sizes, sizes).astype(np.float64)
    req = [S[0] / n_of, S[1] * p64, S[2] * c64, S[3] * p64 * p64, n_of][k]
    np.testing.assert_allclose(r["share"], req, rtol=1e-15, atol=0)
    # with equal segment coefficients the tie rule always picks MEM
    assert np.all((r["regime"][nz] % 2) == 0)


# --------------------------------------------------------------------------
# Phase: the paper's pure cases


def test_phase_pure_cases():
    th = coeff_vec(HAND["base_coeffs"])
    # decode step: every request processes 1 token over a context c >= 1
    off, p, c = one_batch([1] * 5, [1, 7, 100, 3, 9])
    assert oracle.attribute(off, p, c, None, None, th, 1, ("phase",))["phase"][0] == oracle.DECODE
    # prefill step: c = 0 for every request, any prompt length (even 1)
    for plist in ([1], [1, 1], [5, 1, 300]):
        off, p, c = one_batch(plist, [0] * len(plist))
        assert oracle.attribute(off, p, c, None, None, th, 1, ("phase",))["phase"][0] == oracle.PREFILL


# --------------------------------------------------------------------------
# Invariants (coefficients >= 0)


def trace_strategy(max_batches=8, max_n=6):
    batch = st.lists(st.tuples(st.integers(1, 200), st.integers(0, 5000)), min_size=0,
                     max_size=max_n)
    return st.lists(batch, min_size=1, max_size=max_batches)


coeff_strategy = st.lists(st.floats(0.0, 8.0, allow_nan=False, width=32), min_size=20,
                          max_size=20)
shape_strategy = st.sampled_from([None] + sorted(tracegen.SHAPES))


def _mk(batches):
    tr = tracegen.from_batches([([x[0] for x in b], [x[1] for x in b]) for b in batches])
    return tr


def _rel(a, b):
    return abs(a - b) / max(abs(a), abs(b), 1e-300)


@settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(trace_strategy(), coeff_strategy, shape_strategy, st.integers(1, 5))
def test_invariants_additivity_nonneg_tenants(batches, co, shape, nt):
    tr = _mk(batches)
    rng = np.random.default_rng(len(tr.p))
    tr.tenant = rng.integers(0, nt, len(tr.p)).astype(np.int32)
    sh = None if shape is None else tracegen.SHAPES[shape]
    th = np.array(co, np.float32)
    r = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, sh, th, nt)
    sizes = tr.sizes()
    for b in range(tr.n_batches):
        lo, hi = tr.offsets[b], tr.offsets[b + 1]
        s = r["share"][lo:hi]
        # I5: nonnegative shares
        assert np.all(s >= 0)
        if sizes[b] == 0:
            assert r["T"][b] == 0 and r["regime"][b] == oracle.REGIME_EMPTY
            continue
        # I1: shares sum to the batch latency
        assert _rel(s.sum(), r["T"][b]) <= 1e-13
        # the other segment's shares sum to the other segment's latency
        other = r["TC"][b] if r["regime"][b] % 2 == 0 else r["TM"][b]
        assert _rel(r["share_alt"][lo:hi].sum(), other) <= 1e-13
        # T is the roofline max of the two segments, ties to MEM
        assert r["T"][b] == max(r["TM"][b], r["TC"][b])
        assert (r["regime"][b] % 2 == 1) == (r["TC"][b] > r["TM"][b])
        # I2: a single request carries the whole latency
        if sizes[b] == 1:
            assert _rel(s[0], r["T"][b]) <= 1e-15
    # I6: tenant sums add up to the total latency
    assert _rel(r["tenant_sums"].sum(), r["T"].sum()) <= 1e-12 or r["T"].sum() == 0
    for u in range(nt):
        assert _rel(r["tenant_sums"][u], r["share"][tr.tenant == u].sum()) <= 1e-12 or \
            r["tenant_sums"][u] == 0


@settings(max_examples=80, deadline=None)
@given(st.integers(1, 40), st.integers(1, 3000), st.integers(0, 9000), coeff_strategy,
       shape_strategy)
def test_invariant_homogeneous_equal_shares(n, pv, cv, co, shape):
    """I3: identical requests get T/|B| each."""
    off, p, c = one_batch([pv] * n, [cv] * n)
    sh = None if shape is None else tracegen.SHAPES[shape]
    r = oracle.attribute(off, p, c, None, sh, np.array(co, np.float32), 1)
    assert np.all(r["share"] == r["share"][0])
    assert _rel(r["share"][0] * n, r["T"][0]) <= 1e-14 or r["T"][0] == 0


@settings(max_examples=60, deadline=None)
@given(st.lists(st.integers(1, 20000), min_size=1, max_size=10), coeff_strategy,
       shape_strategy, st.integers(0, 9), st.integers(1, 5000))
def test_invariant_monotone_in_context(cs, co, shape, which, delta):
    """I4: with the phase held (decode: p=1, c>=1), raising one context
    length never lowers the batch latency."""
    n = len(cs)
    which %= n
    off, p, c = one_batch([1] * n, cs)
    sh = None if shape is None else tracegen.SHAPES[shape]
    th = np.array(co, np.float32)
    t0 = oracle.attribute(off, p, c, None, sh, th, 1, ("T",))["T"][0]
    c2 = c.copy()
    c2[which] += delta
    t1 = oracle.attribute(off, p, c2, None, sh, th, 1, ("T",))["T"][0]
    assert t1 >= t0


@settings(max_examples=60, deadline=None)
@given(st.lists(st.integers(2, 5000), min_size=1, max_size=10), coeff_strategy,
       shape_strategy, st.integers(0, 9), st.integers(1, 500))
def test_invariant_monotone_in_prompt(ps, co, shape, which, delta):
    """I4: in a prefill batch, raising one prompt length never lowers T."""
    n = len(ps)
    which %= n
    off, p, c = one_batch(ps, [0] * n)
    sh = None if shape is None else tracegen.SHAPES[shape]
    th = np.array(co, np.float32)
    t0 = oracle.attribute(off, p, c, None, sh, th, 1, ("T",))["T"][0]
    p2 = p.copy()
    p2[which] += delta
    t1 = oracle.attribute(off, p2, c, None, sh, th, 1, ("T",))["T"][0]
    assert t1 >= t0


@settings(max_examples=60, deadline=None)
@given(trace_strategy(), st.lists(st.floats(1 / 64, 8, width=32), min_size=20, max_size=20),
       st.sampled_from(sorted(tracegen.SHAPES)))
def test_invariant_reparameterization(batches, co, shape):
    """I7: scaling features by S is the same as scaling coefficients by S."""
    tr = _mk(batches)
    sh = tracegen.SHAPES[shape]
    S = oracle.shape_constants(sh)
    th = np.array(co, np.float32)
    scale = np.tile(np.array([S[0], S[1], S[2], S[3], 1.0]), 4)
    th_s = (th.astype(np.float64) * scale).astype(np.float32)
    a = oracle.attribute(tr.offsets, tr.p, tr.c, None, sh, th, 1)
    b = oracle.attribute(tr.offsets, tr.p, tr.c, None, None, th_s, 1)
    np.testing.assert_allclose(a["T"], b["T"], rtol=2e-7)
    np.testing.assert_allclose(a["share"], b["share"], rtol=2e-7)
    tie = np.abs(a["TM"] - a["TC"]) <= 1e-6 * np.maximum(a["TM"], a["TC"])
    assert np.all((a["regime"] == b["regime"]) | tie)


def test_invariant_continuity_at_switch():
    """I8: sweeping one context length across the MEM->COMP switch moves T by
    at most the steeper segment's slope per unit step; no jump."""
    th = coeff_vec(HAND["base_coeffs"])
    th[17] = 1.0  # decode COMP a2 (1.0) steeper than decode MEM a2 (0.25)
    n = 4
    ts, regs = [], []
    for cv in range(0, 400):
        off, p, c = one_batch([1] * n, [1, 2, 3, 1 + cv])
        r = oracle.attribute(off, p, c, None, None, th, 1, ("T", "regime"))
        ts.append(r["T"][0])
        regs.append(r["regime"][0])
    assert len(set(regs)) == 2, "sweep must cross the switch"
    steps = np.diff(ts)
    assert np.all(steps >= 0) and np.all(steps <= 1.0 + 1e-12)


@settings(max_examples=60, deadline=None)
@given(trace_strategy(), coeff_strategy, st.randoms(use_true_random=False))
def test_invariant_permutation(batches, co, rnd):
    """I9: permuting requests inside a batch permutes its shares; reordering
    batches leaves the tenant sums unchanged."""
    tr = _mk(batches)
    n = tr.n_requests
    tr.tenant = (np.arange(n) % 3).astype(np.int32)
    th = np.array(co, np.float32)
    a = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, None, th, 3)
    perm = np.arange(n)
    for b in range(tr.n_batches):
        lo, hi = tr.offsets[b], tr.offsets[b + 1]
        seg = list(range(lo, hi))
        rnd.shuffle(seg)
        perm[lo:hi] = seg
    b2 = oracle.attribute(tr.offsets, tr.p[perm], tr.c[perm], tr.tenant[perm], None, th, 3)
    np.testing.assert_array_equal(b2["share"], a["share"][perm])
    np.testing.assert_allclose(b2["T"], a["T"], rtol=1e-15)
    # batch reorder
    order = list(range(tr.n_batches))
    rnd.shuffle(order)
    idx = np.concatenate([np.arange(tr.offsets[b], tr.offsets[b + 1]) for b in order] +
                         [np.zeros(0, np.int64)])
    sizes = tr.sizes()[order]
    off2 = np.zeros(len(order) + 1, np.int64)
    off2[1:] = np.cumsum(sizes)
    c2 = oracle.attribute(off2, tr.p[idx], tr.c[idx], tr.tenant[idx], None, th, 3)
    np.testing.assert_allclose(c2["tenant_sums"], a["tenant_sums"], rtol=1e-13)


@settings(max_examples=60, deadline=None)
@given(st.lists(st.tuples(st.integers(1, 300), st.integers(0, 3000)), min_size=1, max_size=12),
       st.sampled_from([None, "llama3.1-8b"]))
def test_invariant_beta_and_a4_terms(reqs, shape):
    """I10: with only beta set, every request carries beta*S0/|B|; with only
    a4 set, every request carries a4*|B| and the batch a4*|B|^2."""
    p = [x[0] for x in reqs]
    c = [x[1] for x in reqs]
    n = len(p)
    off, p, c = one_batch(p, c)
    sh = None if shape is None else tracegen.SHAPES[shape]
    S0 = oracle.shape_constants(sh)[0]
    th = np.zeros(20, np.float32)
    th[0::5] = 3.0
    r = oracle.attribute(off, p, c, None, sh, th, 1)
    assert np.all(r["share"] == 3.0 * (S0 / n))
    assert r["T"][0] == 3.0 * S0
    th = np.zeros(20, np.float32)
    th[4::5] = 0.5
    r = oracle.attribute(off, p, c, None, sh, th, 1)
    assert np.all(r["share"] == 0.5 * n)
    assert r["T"][0] == 0.5 * n * n


def test_exhaustive_tiny_batches():
    """Brute force over every batch of up to 3 requests with p in {1,2,3} and
    c in {0,1,2}: additivity, the max rule, and the phase rule's pure cases."""
    import itertools
    th = coeff_vec(HAND["base_coeffs"])
    reqs = [(p, c) for p in (1, 2, 3) for c in (0, 1, 2)]
    batches = []
    for n in (1, 2, 3):
        batches.extend(itertools.product(reqs, repeat=n))
    tr = tracegen.from_batches([([x[0] for x in b], [x[1] for x in b]) for b in batches])
    r = oracle.attribute(tr.offsets, tr.p, tr.c, None, None, th, 1)
    for i, b in enumerate(batches):
        lo, hi = tr.offsets[i], tr.offsets[i + 1]
        assert r["share"][lo:hi].sum() == pytest.approx(r["T"][i], rel=1e-15)
        assert r["T"][i] == max(r["TM"][i], r["TC"][i])
        if all(pc[0] == 1 and pc[1] >= 1 for pc in b):
            assert r["phase"][i] == oracle.DECODE
        if all(pc[1] == 0 for pc in b):
            assert r["phase"][i] == oracle.PREFILL


# --------------------------------------------------------------------------
# Input validation


def test_validate_errors():
    off = np.array([0, 2, 3], np.int64)
    p = np.array([1, 2, 3], np.int32)
    c = np.array([0, 5, 9], np.int32)
    t = np.array([0, 1, 1], np.int32)
    assert oracle.validate(off, p, c, t, 2) == oracle.OK
    assert oracle.validate(np.array([1, 2, 3]), p, c, t, 2) == oracle.ERANGE
    assert oracle.validate(np.array([0, 2, 1]), p, c, t, 2) == oracle.ERANGE
    assert oracle.validate(np.array([0, 2, 2]), p, c, t, 2) == oracle.ERANGE
    assert oracle.validate(off, np.array([1, 0, 3]), c, t, 2) == oracle.ERANGE
    assert oracle.validate(off, np.array([1, oracle.P_MAX + 1, 3]), c, t, 2) == oracle.ERANGE
    assert oracle.validate(off, p, np.array([0, -1, 9]), t, 2) == oracle.ERANGE
    assert oracle.validate(off, p, c, np.array([0, 2, 1]), 2) == oracle.ERANGE
    assert oracle.validate(off, p, c, np.array([0, -1, 1]), 2) == oracle.ERANGE
    assert oracle.validate(off, p, c, t, 0) == oracle.EINVAL
    big = np.array([0, oracle.BATCH_MAX + 1], np.int64)
    ones = np.ones(oracle.BATCH_MAX + 1, np.int32)
    assert oracle.validate(big, ones, ones) == oracle.ERANGE
    with pytest.raises(oracle.OracleError):
        oracle.attribute(np.array([0, 2, 1]), p, c, t, None, np.ones(20, np.float32), 2)


def test_empty_trace():
    th = coeff_vec(HAND["base_coeffs"])
    r = oracle.attribute(np.zeros(1, np.int64), np.zeros(0, np.int32), np.zeros(0, np.int32),
                         np.zeros(0, np.int32), None, th, 3)
    assert len(r["T"]) == 0 and list(r["tenant_sums"]) == [0, 0, 0]
    r = oracle.attribute(np.zeros(4, np.int64), np.zeros(0, np.int32), np.zeros(0, np.int32),
                         np.zeros(0, np.int32), None, th, 3)
    assert list(r["T"]) == [0, 0, 0] and list(r["regime"]) == [255] * 3


def test_features_sum_to_batch_features():
    rng = np.random.default_rng(3)
    off, p, c, _ = random_trace(rng, nB=60)
    for sh in (None, tracegen.SHAPES["qwen2.5-14b"]):
        xr, xb = oracle.features(off, p, c, sh)
        sizes = np.diff(off)
        for b in range(len(sizes)):
            lo, hi = off[b], off[b + 1]
            if sizes[b] == 0:
                assert np.all(xb[:, b] == 0)
                continue
            np.testing.assert_allclose(xr[:, lo:hi].sum(axis=1), xb[:, b], rtol=1e-14)
        # a coefficient vector dotted with the features gives the latencies
        th = np.random.default_rng(4).random(20).astype(np.float32)
        r = oracle.attribute(off, p, c, None, sh, th, 1)
        for b in range(len(sizes)):
            if sizes[b] == 0:
                continue
            ph = r["phase"][b]
            tm = float(np.dot(th[(ph * 2) * 5:(ph * 2) * 5 + 5].astype(np.float64), xb[:, b]))
            assert _rel(tm, r["TM"][b]) <= 1e-14
