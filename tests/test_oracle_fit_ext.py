"""Pins of the extended-model fit (oracle/fit.py with ext=True; no GPU).

The extended model adds a5*S5*sum p*c and a6*S6*|B| to Eq. 1 (the feature
variants the paper leaves open); its four seven-term sets are fitted like
Eq. 1's (Sec. 2.1, OLS per phase and segment) with the identifiability
reading F5: a5 is kept where sum p*c equals sum c in every batch of a set, a6
where sum p equals |B|.  The pins: planted recovery (with the exact
absorptions the kept columns imply), hand-derived free columns, the
reduction to the Eq. 1 fit on Eq. 1 data, the least-squares normal
equations, and exact metrics of an exact model.
"""
import numpy as np
import pytest

import oracle
import tracegen
from oracle import fit as F


def ext_trace(seed, nb=1500):
    """Prefill chunks with cached prefixes (p > 1, c > 0: every prefill
    column identifiable) and decode batches of varied size."""
    rng = np.random.default_rng(seed)
    batches = []
    for _ in range(nb):
        if rng.random() < 0.5:
            n = int(rng.integers(1, 8))
            batches.append((rng.integers(2, 60, n).tolist(), rng.integers(0, 500, n).tolist()))
        else:
            n = int(rng.integers(1, 64))
            batches.append(([1] * n, rng.integers(1, 3000, n).tolist()))
    return tracegen.from_batches(batches, None, 1)


# unit shape: X = (1, P, C, Q, n^2, R, n); both segments of both phases
# are taken by many batches
THETA_EXT = np.array([200, 1.0, 0.5, 0.001, 0.5, 0.002, 3.0,     # prefill MEM
                      20, 4.0, 0.5, 0.004, 0.5, 0.004, 1.0,      # prefill COMP
                      300, 1.0, 0.02, 0.5, 0.1, 0.01, 2.0,       # decode MEM
                      10, 12.0, 0.02, 0.5, 0.1, 0.01, 2.0],      # decode COMP
                     np.float32).astype(np.float64)


def planted(seed, nb=1500):
    tr = ext_trace(seed, nb)
    T = oracle.attribute_ext(tr.offsets, tr.p, tr.c, None, None, THETA_EXT.astype(np.float32), 0,
                             ("T", "regime"))
    return tr, T


def test_free_columns_by_hand():
    """The exact tests of F2 and F5 on hand-made batch sums."""
    # rows: n, P, C, Q, R
    decode = np.array([[3, 2], [3, 2], [700, 90], [3, 2], [700, 90]], np.int64)
    assert F.free_columns(decode, np.ones(2, bool), ext=True) == [0, 1, 2, 4]
    fresh_prefill = np.array([[2, 1], [9, 40], [0, 0], [41, 1600], [0, 0]], np.int64)
    assert F.free_columns(fresh_prefill, np.ones(2, bool), ext=True) == [0, 1, 3, 4, 6]
    chunked = np.array([[2, 1], [9, 40], [30, 5], [41, 1600], [120, 200]], np.int64)
    assert F.free_columns(chunked, np.ones(2, bool), ext=True) == [0, 1, 2, 3, 4, 5, 6]
    # a decode request with a context beside a fresh prefill: R == C, the
    # cross term is the c term
    mixed = np.array([[2, 2], [6, 9], [100, 7], [26, 65], [100, 7]], np.int64)
    assert F.free_columns(mixed, np.ones(2, bool), ext=True) == [0, 1, 2, 3, 4, 6]
    # one batch of the set breaking the pattern frees the column
    assert F.free_columns(np.concatenate([decode, chunked], axis=1), np.ones(4, bool),
                          ext=True) == [0, 1, 2, 3, 4, 5, 6]
    # Eq. 1 only tests its two columns
    assert F.free_columns(decode, np.ones(2, bool)) == [0, 1, 2, 4]


def test_planted_recovery():
    """From a start 10% off: the true segment of every batch and every
    identifiable coefficient.  Prefill (p > 1 with prefixes): all seven.
    Decode: sum p^2 = sum p = |B| and sum p*c = sum c, so a3, a5 and a6 keep
    their starting values, a1 absorbs a3 and a6, a2 absorbs a5 (unit shape)."""
    tr, T = planted(21)
    counts_true = np.bincount(T["regime"][T["regime"] != 255], minlength=4)
    assert (counts_true >= 50).all(), counts_true
    rng = np.random.default_rng(22)
    theta0 = THETA_EXT * rng.uniform(0.9, 1.1, 28)
    theta, counts = F.fit(tr.offsets, tr.p, tr.c, None, T["T"], theta0, rounds=8, ext=True)
    assert np.array_equal(counts, counts_true)
    want = THETA_EXT.copy()
    for g in (2, 3):
        o = g * 7
        for k in (3, 5, 6):
            want[o + k] = theta0[o + k]
        want[o + 1] = THETA_EXT[o + 1] + (THETA_EXT[o + 3] - theta0[o + 3]) + \
            (THETA_EXT[o + 6] - theta0[o + 6])
        want[o + 2] = THETA_EXT[o + 2] + (THETA_EXT[o + 5] - theta0[o + 5])
    err = np.abs(theta - want) / np.abs(want)
    assert np.max(err) < 1e-6, err


def test_planted_recovery_model_shape():
    """Under Llama3.1-8B constants (S5 = 2 S3, S6 = 2 vocab hidden): the
    same recovery, with the absorptions scaled by the shape constants."""
    tr = ext_trace(31, nb=4000)
    sh = tracegen.SHAPES["llama3.1-8b"]
    co = tracegen.ext_coeffs(104)
    T = oracle.attribute_ext(tr.offsets, tr.p, tr.c, None, sh, co, 0, ("T", "regime"))
    counts_true = np.bincount(T["regime"][T["regime"] != 255], minlength=4)
    truth = co.astype(np.float64)
    theta0 = truth * np.random.default_rng(32).uniform(0.9, 1.1, 28)
    theta, counts = F.fit(tr.offsets, tr.p, tr.c, sh, T["T"], theta0, rounds=6, ext=True)
    assert np.array_equal(counts, counts_true)
    S = oracle.shape_constants_ext(sh)  # S0, S1, S2, S3, S5, S6
    want = truth.copy()
    for g in (0, 1, 2, 3):
        if counts_true[g] == 0:
            want[g * 7:(g + 1) * 7] = theta0[g * 7:(g + 1) * 7]
    for g in (2, 3):
        if counts_true[g] == 0:
            continue
        o = g * 7
        for k in (3, 5, 6):
            want[o + k] = theta0[o + k]
        want[o + 1] = truth[o + 1] + (truth[o + 3] - theta0[o + 3]) * S[3] / S[1] + \
            (truth[o + 6] - theta0[o + 6]) * S[5] / S[1]
        want[o + 2] = truth[o + 2] + (truth[o + 5] - theta0[o + 5]) * S[4] / S[2]
    live = np.repeat(counts_true > 0, 7)
    err = np.abs(theta - want)[live] / np.abs(want)[live]
    assert np.max(err) < 1e-6, err
    assert np.array_equal(theta[~live], theta0[~live])


def test_reduces_to_the_eq1_fit():
    """On Eq. 1 data (prefill without prefixes, decode): the extended fit
    finds a6 = 0 in prefill (free there), keeps a5 and the decode a5, a6,
    and agrees with the Eq. 1 fit on the other coefficients."""
    rng = np.random.default_rng(41)
    batches = []
    for _ in range(1200):
        if rng.random() < 0.4:
            n = int(rng.integers(1, 8))
            batches.append((rng.integers(2, 60, n).tolist(), [0] * n))
        else:
            n = int(rng.integers(1, 64))
            batches.append(([1] * n, rng.integers(1, 3000, n).tolist()))
    tr = tracegen.from_batches(batches, None, 1)
    th20 = np.delete(THETA_EXT.reshape(4, 7), [5, 6], axis=1).reshape(20)
    T = oracle.attribute(tr.offsets, tr.p, tr.c, None, None, th20.astype(np.float32), 0, ("T",))["T"]
    theta0_20 = th20 * np.random.default_rng(42).uniform(0.9, 1.1, 20)
    theta0 = np.zeros(28)
    for g in range(4):
        theta0[g * 7:g * 7 + 5] = theta0_20[g * 5:(g + 1) * 5]
    t20, c20 = F.fit(tr.offsets, tr.p, tr.c, None, T, theta0_20, rounds=6)
    t28, c28 = F.fit(tr.offsets, tr.p, tr.c, None, T, theta0, rounds=6, ext=True)
    assert np.array_equal(c20, c28)
    for g in range(4):
        np.testing.assert_allclose(t28[g * 7:g * 7 + 5], t20[g * 5:(g + 1) * 5], rtol=1e-6)
    # prefill a6 is free and fitted to (almost) 0; every other a5, a6 stays 0
    for g in (0, 1):
        assert abs(t28[g * 7 + 6]) < 1e-6 * THETA_EXT[g * 7 + 1]
        assert t28[g * 7 + 5] == 0.0
    for g in (2, 3):
        assert t28[g * 7 + 5] == 0.0 and t28[g * 7 + 6] == 0.0


@pytest.mark.parametrize("seed", range(3))
def test_ols_normal_equations_hold(seed):
    """With noise: in every set the residuals are orthogonal to the free
    columns at the solution."""
    tr, T = planted(50 + seed, nb=1200)
    rng = np.random.default_rng(seed)
    y = T["T"] * np.exp(0.05 * rng.standard_normal(len(T["T"])))
    theta, _ = F.fit(tr.offsets, tr.p, tr.c, None, y, THETA_EXT, rounds=1, ext=True)
    X, phase, ne = F.design(tr.offsets, tr.p, tr.c, None, ext=True)
    sums, _ = oracle.batch_sums_ext(tr.offsets, tr.p, tr.c)
    tm, tc = F.segment_values(X, phase, THETA_EXT)
    seg = np.where(tc > tm, 1, 0)
    for g, (ph, s) in enumerate(F.GROUPS):
        idx = ne & (phase == ph) & (seg == s)
        assert idx.sum() >= 20, (g, idx.sum())
        free = F.free_columns(sums, idx, ext=True)
        Xg, yg = X[idx], y[idx]
        r = yg - Xg @ theta[g * 7:(g + 1) * 7]
        grad = Xg[:, free].T @ r
        scale = np.abs(Xg[:, free]).T @ np.abs(yg)
        assert np.all(np.abs(grad) <= 1e-8 * scale), (g, grad / scale)


def test_metrics_of_the_exact_model():
    tr, T = planted(61, nb=300)
    m = F.metrics(tr.offsets, tr.p, tr.c, None, THETA_EXT.astype(np.float32), T["T"], ext=True)
    for g in ("prefill", "decode", "all"):
        assert m[g]["r2"] == 1.0 and m[g]["p90"] == 0.0 and m[g]["p99"] == 0.0
    # the Eq. 1 part alone misses the a5, a6 terms
    th20 = np.delete(THETA_EXT.reshape(4, 7), [5, 6], axis=1).reshape(20)
    m20 = F.metrics(tr.offsets, tr.p, tr.c, None, th20.astype(np.float32), T["T"])
    assert m20["all"]["p90"] > 0.0 and m20["all"]["r2"] < 1.0


def test_batch_sums_ext_brute_force():
    rng = np.random.default_rng(7)
    tr = ext_trace(71, nb=200)
    sums, phase = oracle.batch_sums_ext(tr.offsets, tr.p, tr.c)
    s4, ph4 = oracle.batch_sums(tr.offsets, tr.p, tr.c)
    assert np.array_equal(sums[:4], s4) and np.array_equal(phase, ph4)
    for b in rng.integers(0, tr.n_batches, 40):
        lo, hi = tr.offsets[b], tr.offsets[b + 1]
        assert sums[4][b] == sum(int(a) * int(c) for a, c in zip(tr.p[lo:hi], tr.c[lo:hi]))
