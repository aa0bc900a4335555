"""Pins of the oracle's batch sums and admission query (no GPU).

The admission query (Sec. 1: admission control that rejects or defers a
request whose share would exceed its budget) is, by definition, the
attribution of the batch with the candidate appended, compared with the
attribution of the batch without it (Sec. 2 Problem formulation, Sec. 2.1
Eq. 1).  Hand-worked values in tests/golden/admission_examples.json pin it;
the properties below hold for any batch.
"""
import json
import os

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ADM = json.load(open(os.path.join(ROOT, "tests", "golden", "admission_examples.json")))
HAND = json.load(open(os.path.join(ROOT, "tests", "golden", "hand_examples.json")))


def base_coeffs():
    d = HAND["base_coeffs"]
    return np.array(d["prefill_mem"] + d["prefill_comp"] + d["decode_mem"] + d["decode_comp"],
                    np.float32)


@pytest.mark.parametrize("ex", ADM["examples"], ids=[e["name"] for e in ADM["examples"]])
def test_admission_hand_examples(ex):
    r = oracle.admit(ex["p"], ex["c"], ex["cand_p"], ex["cand_c"], None, base_coeffs())
    assert r["T_after"] == ex["T_after"]
    assert r["delta"] == ex["delta"]
    assert r["TM_after"] == ex["TM_after"] and r["TC_after"] == ex["TC_after"]
    assert r["regime"] == ex["regime"]
    if "share" in ex:
        assert r["share"] == ex["share"]
    else:  # 4/9 is not a binary fraction: within the fp64 rounding of five terms
        want = ex["share_num"] / ex["share_den"]
        assert abs(r["share"] - want) <= 4e-16 * want


def random_batch(rng, n, prefill):
    if prefill:
        return rng.integers(1, 4000, n).astype(np.int32), np.zeros(n, np.int32)
    return np.ones(n, np.int32), rng.integers(1, 100000, n).astype(np.int32)


@pytest.mark.parametrize("seed", range(8))
def test_admission_properties(seed):
    """For any batch: the delta is the difference of the two latencies; the
    candidate's share and the others' shares in B' add up to f(B')
    (additivity, Sec. 2 Problem formulation); and the shares of B's requests
    in B' are what attribution of B' gives them."""
    rng = np.random.default_rng(seed)
    co = oracle_coeffs(rng)
    shape = {"n_layers": 32, "hidden": 4096, "n_q_heads": 32, "n_kv_heads": 8, "head_dim": 128,
             "ffn": 14336, "vocab": 128256, "weight_bytes": 2, "kv_bytes": 2}
    n = int(rng.integers(0, 40))
    p, c = random_batch(rng, n, seed % 2 == 0)
    cp, cc = (int(rng.integers(1, 3000)), 0) if seed % 3 == 0 else (1, int(rng.integers(1, 50000)))
    r = oracle.admit(p, c, cp, cc, shape, co)
    before = oracle.attribute(np.array([0, n], np.int64), p, c, None, shape, co, 0, ("T",))["T"][0]
    p1, c1 = np.append(p, cp).astype(np.int32), np.append(c, cc).astype(np.int32)
    after = oracle.attribute(np.array([0, n + 1], np.int64), p1, c1, None, shape, co, 0,
                             ("T", "share"))
    assert r["T_after"] == after["T"][0]
    assert r["delta"] == r["T_after"] - before
    assert r["share"] == after["share"][-1]
    assert abs(after["share"].sum() - r["T_after"]) <= 1e-12 * abs(r["T_after"])
    # both segment values bracket the chosen one (roofline max)
    assert r["T_after"] == max(r["TM_after"], r["TC_after"])


def oracle_coeffs(rng):
    """Positive coefficients with the magnitudes of the synthetic workloads."""
    bw, fl = 4e6, 5e8
    mem = [1 / bw, 0.1 / fl, 1 / bw, 0.5 / fl, 0.01]
    comp = [0.1 / bw, 1 / fl, 1 / bw, 1 / fl, 0.01]
    base = np.array(mem + comp + mem + comp, np.float64)
    return (base * np.exp(0.2 * rng.standard_normal(20))).astype(np.float32)


def test_batch_sums_against_numpy():
    """Sums over each batch by numpy's segment reduction; phase by the rule
    of the attribution (prefill iff some request has p > 1 or c = 0)."""
    rng = np.random.default_rng(5)
    sizes = rng.integers(0, 50, 300)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    N = int(off[-1])
    p = np.where(rng.random(N) < 0.2, rng.integers(1, 1 << 20, N), 1).astype(np.int32)
    c = np.where(rng.random(N) < 0.1, 0, rng.integers(0, 1 << 31 - 1, N)).astype(np.int32)
    sums, phase = oracle.batch_sums(off, p, c)
    for b in range(len(sizes)):
        lo, hi = off[b], off[b + 1]
        pp, cc = p[lo:hi].astype(np.int64), c[lo:hi].astype(np.int64)
        assert sums[0, b] == hi - lo
        assert sums[1, b] == pp.sum() and sums[2, b] == cc.sum() and sums[3, b] == (pp * pp).sum()
        if hi == lo:
            assert phase[b] == 255
        else:
            assert phase[b] == (0 if ((pp > 1) | (cc == 0)).any() else 1)
