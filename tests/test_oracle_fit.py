"""Pins of the fitting and metrics oracle (oracle/fit.py; no GPU).

Sec. 2.1 fits Eq. 1's four coefficient sets by OLS on profiled latencies;
Sec. 3 / Appendix A report r^2 and p90/p99 relative error.  The pins below
do not re-run the oracle's own formulas: planted coefficients must be
recovered, the OLS normal equations must hold at the solution, and hand
values fix r^2 and the nearest-rank percentiles.
"""
import numpy as np
import pytest

import oracle
import tracegen
from oracle import fit as F


def planted_trace(seed, nb=600):
    """Mixed prefill/decode batches of varied size, so that with the
    coefficients below both segments of both phases hold many batches."""
    rng = np.random.default_rng(seed)
    batches = []
    for _ in range(nb):
        if rng.random() < 0.4:  # prefill: P from 2 to a few hundred (MEM below ~60)
            n = int(rng.integers(1, 8))
            batches.append((rng.integers(2, 60, n).tolist(), [0] * n))
        else:
            n = int(rng.integers(1, 64))
            batches.append(([1] * n, rng.integers(1, 3000, n).tolist()))
    return tracegen.from_batches(batches, None, 1)


# unit shape: X = (1, P, C, Q, n^2).  Prefill: MEM wins for small P, COMP for
# large; decode: MEM for small batches, COMP for large ones.
THETA_TRUE = np.array([200, 1.0, 0.5, 0.001, 0.5,      # prefill MEM
                       20, 4.0, 0.5, 0.004, 0.5,       # prefill COMP
                       300, 1.0, 0.02, 0.5, 0.1,       # decode MEM
                       10, 12.0, 0.02, 0.5, 0.1],      # decode COMP
                      np.float64)


def test_planted_coefficients_recovered():
    """From a start 25% off: the true segment of every batch, exact
    predictions, every identifiable coefficient (F2); the p^2 coefficient of
    decode and the c coefficient of prefill keep their starting values, and
    decode's a1 takes a1 + a3 - a3_start (sum p = sum p^2 there)."""
    tr = planted_trace(1)
    T = oracle.attribute(tr.offsets, tr.p, tr.c, None, None, THETA_TRUE.astype(np.float32), 0,
                         ("T", "regime"))
    counts_true = np.bincount(T["regime"][T["regime"] != 255], minlength=4)
    assert (counts_true >= 20).all(), counts_true  # every set is exercised
    rng = np.random.default_rng(2)
    truth = THETA_TRUE.astype(np.float32).astype(np.float64)  # y was made with fp32 coefficients
    theta0 = truth * rng.uniform(0.75, 1.25, 20)
    theta, counts = F.fit(tr.offsets, tr.p, tr.c, None, T["T"], theta0, rounds=8)
    assert np.array_equal(counts, counts_true)
    want = truth.copy()
    for g in (0, 1):  # prefill: C == 0 everywhere, a2 keeps its start
        want[g * 5 + 2] = theta0[g * 5 + 2]
    for g in (2, 3):  # decode: Q == P everywhere, a3 keeps its start, a1 absorbs
        want[g * 5 + 3] = theta0[g * 5 + 3]
        want[g * 5 + 1] = truth[g * 5 + 1] + truth[g * 5 + 3] - theta0[g * 5 + 3]
    assert np.max(np.abs(theta - want) / np.abs(want)) < 1e-6


def test_chunked_prefill_identifies_every_coefficient():
    """Prefill batches with cached prefixes (c > 0) and p > 1: all five
    prefill coefficients are determined."""
    rng = np.random.default_rng(4)
    batches = []
    for _ in range(500):
        n = int(rng.integers(1, 8))
        batches.append((rng.integers(2, 60, n).tolist(), rng.integers(0, 500, n).tolist()))
    tr = tracegen.from_batches(batches, None, 1)
    T = oracle.attribute(tr.offsets, tr.p, tr.c, None, None, THETA_TRUE.astype(np.float32), 0,
                         ("T", "regime"))
    truth = THETA_TRUE.astype(np.float32).astype(np.float64)
    theta0 = truth * rng.uniform(0.9, 1.1, 20)
    theta, counts = F.fit(tr.offsets, tr.p, tr.c, None, T["T"], theta0, rounds=8)
    assert counts[0] >= 20 and counts[1] >= 20 and counts[2] == 0 and counts[3] == 0
    assert np.max(np.abs(theta[:10] - truth[:10]) / np.abs(truth[:10])) < 1e-6
    assert np.array_equal(theta[10:], theta0[10:])  # no decode batches: kept


def model_shape_trace(seed, nb=8000):
    """10% small prefill batches (1-3 requests, p < 40: memory-bound under
    the heavy-tailed workload's coefficients), 60% large ones (up to 63
    requests, p < 4096), 30% decode batches (up to 255 requests,
    c < 32768); Llama3.1-8B shape.  The compute-bound prefill set then has
    thousands of batches whose raw columns span ~1e12."""
    rng = np.random.default_rng(seed)
    batches = []
    for _ in range(nb):
        u = rng.random()
        if u < 0.1:
            n = int(rng.integers(1, 4))
            batches.append((rng.integers(2, 40, n).tolist(), [0] * n))
        elif u < 0.7:
            n = int(rng.integers(1, 64))
            batches.append((rng.integers(2, 4096, n).tolist(), [0] * n))
        else:
            n = int(rng.integers(1, 256))
            batches.append(([1] * n, rng.integers(1, 32768, n).tolist()))
    tr = tracegen.from_batches(batches, None, 1)
    tr.shape = tracegen.SHAPES["llama3.1-8b"]
    return tr


def test_planted_recovery_model_shape():
    """Planted recovery under a real model shape (Llama3.1-8B constants):
    the raw feature columns then differ by many orders of magnitude (S1*P
    up to ~1e15, |B|^2 ~ 1), which must not make a well-determined set
    (condition number ~60 on unit-norm columns) look rank deficient (F2)."""
    tr = model_shape_trace(12)
    co = tracegen.config_coeffs("heavy-tailed")
    T = oracle.attribute(tr.offsets, tr.p, tr.c, None, tr.shape, co, 0, ("T", "regime"))
    counts_true = np.bincount(T["regime"][T["regime"] != 255], minlength=4)
    assert (counts_true >= 100).all(), counts_true
    truth = co.astype(np.float64)
    theta0 = truth * np.random.default_rng(6).uniform(0.9, 1.1, 20)
    theta, counts = F.fit(tr.offsets, tr.p, tr.c, tr.shape, T["T"], theta0, rounds=6)
    assert np.array_equal(counts, counts_true)
    want = truth.copy()
    for g in (0, 1):  # prefill: C == 0 everywhere, a2 keeps its start
        want[g * 5 + 2] = theta0[g * 5 + 2]
    S = oracle.shape_constants(tr.shape)
    for g in (2, 3):  # decode: Q == P, a3 keeps its start, a1 absorbs (a3 - a3_0) S3/S1
        want[g * 5 + 3] = theta0[g * 5 + 3]
        want[g * 5 + 1] = truth[g * 5 + 1] + (truth[g * 5 + 3] - theta0[g * 5 + 3]) * S[3] / S[1]
    assert np.max(np.abs(theta - want) / np.abs(want)) < 1e-6, np.abs(theta - want) / np.abs(want)


@pytest.mark.parametrize("seed", range(4))
def test_ols_normal_equations_hold(seed):
    """With noise, each set's solution makes the residuals orthogonal to its
    batches' features (the defining property of least squares)."""
    tr = planted_trace(10 + seed)
    T = oracle.attribute(tr.offsets, tr.p, tr.c, None, None, THETA_TRUE.astype(np.float32), 0,
                         ("T",))["T"]
    rng = np.random.default_rng(seed)
    y = T * np.exp(0.05 * rng.standard_normal(len(T)))
    theta, _ = F.fit(tr.offsets, tr.p, tr.c, None, y, THETA_TRUE, rounds=1)
    X, phase, ne = F.design(tr.offsets, tr.p, tr.c, None)
    tm, tc = F.segment_values(X, phase, THETA_TRUE)
    seg = np.where(tc > tm, 1, 0)
    for g, (ph, s) in enumerate(F.GROUPS):
        idx = ne & (phase == ph) & (seg == s)
        assert idx.sum() >= 20, (g, idx.sum())
        Xg, yg = X[idx], y[idx]
        r = yg - Xg @ theta[g * 5:(g + 1) * 5]
        grad = Xg.T @ r
        scale = np.abs(Xg).T @ np.abs(yg)
        assert np.all(np.abs(grad) <= 1e-8 * scale), (g, grad / scale)


def test_ties_go_to_mem():
    """Identical MEM and COMP starting sets: every batch ties, and ties take
    the memory-bound segment (the evaluation rule, F1)."""
    tr = planted_trace(5, nb=100)
    th = THETA_TRUE.copy()
    th[5:10] = th[0:5]
    th[15:20] = th[10:15]
    T = oracle.attribute(tr.offsets, tr.p, tr.c, None, None, THETA_TRUE.astype(np.float32), 0,
                         ("T", "phase"))
    _, counts = F.fit(tr.offsets, tr.p, tr.c, None, T["T"], th, rounds=1)
    assert counts[1] == 0 and counts[3] == 0
    assert counts[0] == np.sum(T["phase"] == 0) and counts[2] == np.sum(T["phase"] == 1)


def test_small_set_keeps_its_coefficients():
    tr = tracegen.from_batches([([1, 1], [10, 20]), ([1], [5]), ([3, 4], [0, 0])], None, 1)
    y = np.array([50.0, 20.0, 70.0])
    theta0 = np.arange(1, 21, dtype=np.float64)
    theta, counts = F.fit(tr.offsets, tr.p, tr.c, None, y, theta0, rounds=3)
    assert np.array_equal(theta, theta0)  # no set has 5 batches
    assert counts.sum() == 3


def only_c():
    """Decode MEM = (0, 0, 1, 0, 0), everything else 0: a decode batch's
    prediction is its context sum C (COMP is 0, so MEM is taken); prefill
    MEM = (0, 1, 0, 0, 0): a prefill batch's prediction is P."""
    th = np.zeros(20, np.float32)
    th[2 * 5 + 2] = 1.0
    th[0 * 5 + 1] = 1.0
    return th


def test_metrics_hand_values():
    # decode batches with C = 2, 4, 6, 9 against y = 2, 4, 6, 8:
    #   SSE = 1, mean 5, SS_tot = 9 + 1 + 1 + 9 = 20, r^2 = 0.95;
    #   relative errors 0, 0, 0, 1/8: p90 = 4th smallest (ceil 3.6), p99 = 4th (ceil 3.96)
    # prefill batches with P = 10 .. 100 against y = 10 .. 100 except the last (y = 50):
    #   relative errors nine 0s and 1.0: p90 = 9th smallest = 0, p99 = 10th = 1
    dec = [([1], [2]), ([1], [4]), ([1], [6]), ([1], [9])]
    pre = [([p], [0]) for p in range(10, 101, 10)]
    tr = tracegen.from_batches(dec + pre + [([], [])], None, 1)
    y = np.array([2, 4, 6, 8] + list(range(10, 100, 10)) + [50, 7], np.float64)
    m = F.metrics(tr.offsets, tr.p, tr.c, None, only_c(), y)
    assert m["decode"]["n"] == 4 and m["prefill"]["n"] == 10 and m["all"]["n"] == 14
    assert m["decode"]["r2"] == 0.95
    assert m["decode"]["p90"] == np.float32(0.125) and m["decode"]["p99"] == np.float32(0.125)
    assert m["prefill"]["p90"] == 0.0 and m["prefill"]["p99"] == 1.0
    # prefill: SSE = 50^2, SS_tot = sum (y - mean)^2 with y = 10..90, 50
    yp = np.array(list(range(10, 100, 10)) + [50], np.float64)
    assert abs(m["prefill"]["r2"] - (1 - 2500 / np.sum((yp - yp.mean()) ** 2))) < 1e-15


def test_metrics_perfect_fit():
    tr = planted_trace(3, nb=200)
    T = oracle.attribute(tr.offsets, tr.p, tr.c, None, None, THETA_TRUE.astype(np.float32), 0,
                         ("T",))["T"]
    m = F.metrics(tr.offsets, tr.p, tr.c, None, THETA_TRUE.astype(np.float32), T)
    for g in ("prefill", "decode", "all"):
        assert m[g]["r2"] == 1.0 and m[g]["p90"] == 0.0 and m[g]["p99"] == 0.0
