"""GPU parity of llmv_fit and llmv_fit_metrics (through the C ABI) against
the fitting oracle (oracle/fit.py).

Fitting (Sec. 2.1: OLS per phase and segment).  The library solves the
normal equations by a Cholesky factorisation after column scaling; the
oracle calls a least-squares routine on the design matrix.  Both are
backward stable for the scaled problem up to a factor kappa^2, kappa being
the condition number of a set's column-scaled free features, so the
comparison is made on the scaled coefficients D*theta (D = column norms):
|D (theta_gpu - theta_oracle)| <= tol * |D theta_oracle| with
tol = 1e-9 + 100 * eps * kappa^2, for sets with kappa < 1e4.  Exactly rank
deficient sets (the oracle's rank below the free count) must keep their
coefficients on both sides.  Segment counts are exact (no batch of these
inputs lies in the tie zone).

Metrics (Sec. 3 / Appendix A): r^2 within 1e-9; p90 / p99 within 2 fp32
ulp (the fp32 rounding of an fp64 relative error can differ by one ulp when
the two fp64 predictions differ in the last place); per-batch relative
errors within 1e-6, NaN exactly where the oracle has none; batch counts
exact.
"""
import os
import sys

import numpy as np
import pytest

import oracle
import parity
import tracegen
from oracle import fit as F

pytestmark = pytest.mark.gpu

EPS = np.finfo(np.float64).eps


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


def measured(tr, coeffs, seed, sigma=0.05):
    """Synthetic measured latencies: the model's T under `coeffs` (oracle)
    times a lognormal factor exp(sigma * Z), Z from the seeded generator."""
    T = oracle.attribute(tr.offsets, tr.p, tr.c, None, tr.shape, coeffs, 0, ("T",))["T"]
    z = tracegen.normal(seed, 21, 0, tr.n_batches)
    return T * np.exp(sigma * z)


def gpu_state(L, tr, y):
    import torch
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, None)
    sums, phase = L.batch_sums(dt)
    y_d = torch.as_tensor(np.ascontiguousarray(y, np.float64), device=sums.device)
    torch.cuda.synchronize()
    return sums, phase, y_d


def gpu_fit(L, tr, y, theta0, rounds):
    import torch
    sums, phase, y_d = gpu_state(L, tr, y)
    theta = torch.full((20,), float("nan"), dtype=torch.float64, device=y_d.device)
    counts = torch.full((4,), -7, dtype=torch.int64, device=y_d.device)
    L.llmv_fit(sums, phase, tr.shape, y_d, theta0, rounds, theta, counts)
    torch.cuda.synchronize()
    return theta.cpu().numpy(), counts.cpu().numpy()


def set_checks(tr, y, theta0, theta_o, theta_g):
    """Per set of the last round's assignment (that of theta0 after one
    round): the scaled comparison, or exact keeping for a rank-deficient
    set.  Returns {set: (batches, kappa, scaled error)}."""
    X, phase, ne = F.design(tr.offsets, tr.p, tr.c, tr.shape)
    sums, _ = oracle.batch_sums(tr.offsets, tr.p, tr.c)
    tm, tc = F.segment_values(X, phase, theta0)
    seg = np.where(tc > tm, 1, 0)
    out = {}
    for g, (ph, s) in enumerate(F.GROUPS):
        idx = ne & (phase == ph) & (seg == s)
        sl = slice(g * 5, g * 5 + 5)
        if idx.sum() == 0:
            assert np.array_equal(theta_g[sl], theta0[sl]), g
            continue
        free = F.free_columns(sums, idx)
        kept = [k for k in range(5) if k not in free]
        assert np.array_equal(theta_g[sl][kept], theta0[sl][kept]), (g, kept)
        Xg = X[idx][:, free]
        D = np.linalg.norm(Xg, axis=0)
        kappa = np.linalg.cond(Xg / D) if idx.sum() >= len(free) else np.inf
        if kappa > 1e14 or idx.sum() < len(free):
            assert np.array_equal(theta_g[sl], theta0[sl]), (g, kappa)
            assert np.array_equal(theta_o[sl], theta0[sl]), (g, kappa)
            out[g] = (int(idx.sum()), kappa, 0.0)
            continue
        assert kappa < 1e4, (g, kappa)  # no case between the two regimes
        a = D * theta_g[g * 5 + np.array(free)]
        b = D * theta_o[g * 5 + np.array(free)]
        err = np.linalg.norm(a - b) / np.linalg.norm(b)
        tol = 1e-9 + 100 * EPS * kappa * kappa
        assert err <= tol, (g, err, tol, kappa)
        out[g] = (int(idx.sum()), float(kappa), float(err))
    return out


FIT_CASES = [("tiny-mixed", None), ("chunked-prefill", 5000), ("heavy-tailed", 20000),
             ("decode-only", 5000)]


@pytest.mark.parametrize("name,nb", FIT_CASES)
def test_fit_one_round_matches_oracle(L, name, nb):
    tr = tracegen.config_trace(name, nb)
    co = tracegen.config_coeffs(name)
    y = measured(tr, co, seed=7)
    theta0 = tracegen.perturbed_coeffs(co, 77).astype(np.float64)
    say(f"[fit] {name} nB={tr.n_batches} rounds=1")
    theta_o, counts_o = F.fit(tr.offsets, tr.p, tr.c, tr.shape, y, theta0, rounds=1)
    theta_g, counts_g = gpu_fit(L, tr, y, theta0, 1)
    assert np.array_equal(counts_g, counts_o), (counts_g, counts_o)
    st = set_checks(tr, y, theta0, theta_o, theta_g)
    say(f"[fit] {name}: {st}")


@pytest.mark.parametrize("name,nb", [("tiny-mixed", None), ("heavy-tailed", 20000)])
def test_fit_rounds_match_oracle(L, name, nb):
    """Several rounds: each round's assignment follows the previous round's
    fitted coefficients on both sides."""
    tr = tracegen.config_trace(name, nb)
    co = tracegen.config_coeffs(name)
    y = measured(tr, co, seed=8, sigma=0.02)
    theta0 = tracegen.perturbed_coeffs(co, 78).astype(np.float64)
    theta_o, counts_o = F.fit(tr.offsets, tr.p, tr.c, tr.shape, y, theta0, rounds=4)
    theta_g, counts_g = gpu_fit(L, tr, y, theta0, 4)
    assert np.array_equal(counts_g, counts_o), (counts_g, counts_o)
    # the last round's start is theta after 3 rounds (oracle)
    theta3, _ = F.fit(tr.offsets, tr.p, tr.c, tr.shape, y, theta0, rounds=3)
    # kept coefficients come from theta0 through every round
    st = set_checks(tr, y, theta3, theta_o, theta_g)
    say(f"[fit rounds] {name}: {st}")


def planted_trace(seed, nb=600):
    """Prefill and decode batches of varied size, so that under THETA_TRUE
    (unit shape) both segments of both phases hold many batches."""
    rng = np.random.default_rng(seed)
    batches = []
    for _ in range(nb):
        if rng.random() < 0.4:
            n = int(rng.integers(1, 8))
            batches.append((rng.integers(2, 60, n).tolist(), [0] * n))
        else:
            n = int(rng.integers(1, 64))
            batches.append(([1] * n, rng.integers(1, 3000, n).tolist()))
    return tracegen.from_batches(batches, None, 1)


THETA_TRUE = np.array([200, 1.0, 0.5, 0.001, 0.5, 20, 4.0, 0.5, 0.004, 0.5,
                       300, 1.0, 0.02, 0.5, 0.1, 10, 12.0, 0.02, 0.5, 0.1], np.float64)


def test_fit_planted_recovery(L):
    """Noise-free latencies of planted coefficients, fitted from a start 25%
    off in 8 rounds: the true segment counts and every identifiable
    coefficient; a2 of prefill and a3 of decode keep their start (Q == P in
    decode, so decode's a1 absorbs a3's error)."""
    tr = planted_trace(1)
    truth = THETA_TRUE.astype(np.float32)
    T = oracle.attribute(tr.offsets, tr.p, tr.c, None, None, truth, 0, ("T", "regime"))
    counts_true = np.bincount(T["regime"][T["regime"] != 255], minlength=4)
    truth = truth.astype(np.float64)
    theta0 = truth * np.random.default_rng(2).uniform(0.75, 1.25, 20)
    theta, counts = gpu_fit(L, tr, T["T"], theta0, 8)
    assert np.array_equal(counts, counts_true)
    want = truth.copy()
    for g in (0, 1):
        want[g * 5 + 2] = theta0[g * 5 + 2]
    for g in (2, 3):
        want[g * 5 + 3] = theta0[g * 5 + 3]
        want[g * 5 + 1] = truth[g * 5 + 1] + truth[g * 5 + 3] - theta0[g * 5 + 3]
    assert np.max(np.abs(theta - want) / np.abs(want)) < 1e-6


def test_fit_planted_recovery_model_shape(L):
    """Planted recovery under the Llama3.1-8B shape (raw feature columns
    spanning ~12 orders of magnitude, thousands of batches per set): the
    column-scaled solve must recover every identifiable coefficient, as the
    oracle pin with the same trace does."""
    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    from test_oracle_fit import model_shape_trace
    tr = model_shape_trace(12)
    co = tracegen.config_coeffs("heavy-tailed")
    T = oracle.attribute(tr.offsets, tr.p, tr.c, None, tr.shape, co, 0, ("T", "regime"))
    counts_true = np.bincount(T["regime"][T["regime"] != 255], minlength=4)
    truth = co.astype(np.float64)
    theta0 = truth * np.random.default_rng(6).uniform(0.9, 1.1, 20)
    theta, counts = gpu_fit(L, tr, T["T"], theta0, 6)
    assert np.array_equal(counts, counts_true)
    want = truth.copy()
    for g in (0, 1):
        want[g * 5 + 2] = theta0[g * 5 + 2]
    S = oracle.shape_constants(tr.shape)
    for g in (2, 3):
        want[g * 5 + 3] = theta0[g * 5 + 3]
        want[g * 5 + 1] = truth[g * 5 + 1] + (truth[g * 5 + 3] - theta0[g * 5 + 3]) * S[3] / S[1]
    assert np.max(np.abs(theta - want) / np.abs(want)) < 1e-6


def test_fit_edge_cases(L):
    import torch
    theta0 = np.arange(1, 21, dtype=np.float64)
    # rounds = 0: theta0 copied, counts zero
    tr = planted_trace(3, nb=100)
    y = np.ones(tr.n_batches)
    theta, counts = gpu_fit(L, tr, y, theta0, 0)
    assert np.array_equal(theta, theta0) and not counts.any()
    # no batches at all
    sums = torch.zeros((4, 0), dtype=torch.int64, device="cuda")
    phase = torch.zeros(0, dtype=torch.uint8, device="cuda")
    yd = torch.zeros(0, dtype=torch.float64, device="cuda")
    th, ct = L.fit(sums, phase, None, yd, theta0, 3)
    torch.cuda.synchronize()
    assert np.array_equal(th.cpu().numpy(), theta0) and not ct.cpu().numpy().any()
    # only empty batches
    tr = tracegen.from_batches([([], [])] * 5, None, 1)
    theta, counts = gpu_fit(L, tr, np.ones(5), theta0, 2)
    assert np.array_equal(theta, theta0) and not counts.any()
    # sets with fewer batches than free coefficients keep theirs
    tr = tracegen.from_batches([([1, 1], [10, 20]), ([1], [5]), ([3, 4], [0, 0])], None, 1)
    y = np.array([50.0, 20.0, 70.0])
    theta_o, counts_o = F.fit(tr.offsets, tr.p, tr.c, None, y, theta0, rounds=3)
    theta, counts = gpu_fit(L, tr, y, theta0, 3)
    assert np.array_equal(theta, theta_o) and np.array_equal(theta, theta0)
    assert np.array_equal(counts, counts_o)
    # every decode batch of one size: |B|^2 and sum p are constant, the set
    # is rank deficient and keeps its coefficients (as in the oracle)
    rng = np.random.default_rng(5)
    tr = tracegen.from_batches([([1] * 8, rng.integers(1, 900, 8).tolist()) for _ in range(50)],
                               None, 1)
    y = rng.uniform(100, 200, 50)
    theta_o, counts_o = F.fit(tr.offsets, tr.p, tr.c, None, y, theta0, rounds=1)
    theta, counts = gpu_fit(L, tr, y, theta0, 1)
    assert np.array_equal(theta, theta_o) and np.array_equal(theta, theta0)
    assert np.array_equal(counts, counts_o)


def test_fit_ties_go_to_mem(L):
    tr = planted_trace(5, nb=100)
    th = THETA_TRUE.copy()
    th[5:10] = th[0:5]
    th[15:20] = th[10:15]
    T = oracle.attribute(tr.offsets, tr.p, tr.c, None, None, THETA_TRUE.astype(np.float32), 0,
                         ("T", "phase"))
    _, counts = gpu_fit(L, tr, T["T"], th, 1)
    assert counts[1] == 0 and counts[3] == 0
    assert counts[0] == np.sum(T["phase"] == 0) and counts[2] == np.sum(T["phase"] == 1)


# ------------------------------------------------------------------ metrics


def gpu_metrics(L, tr, coeffs, y):
    import torch
    sums, phase, y_d = gpu_state(L, tr, y)
    m = L.fit_metrics(sums, phase, tr.shape, coeffs, y_d, rel_err=True)
    torch.cuda.synchronize()
    m["rel_err"] = m["rel_err"].cpu().numpy()
    return m


def oracle_rel_err(tr, coeffs, y):
    """Per-batch relative errors as the oracle defines them (F4), NaN where
    it has none."""
    X, phase, ne = F.design(tr.offsets, tr.p, tr.c, tr.shape)
    tm, tc = F.segment_values(X, phase, np.asarray(coeffs, np.float32).astype(np.float64))
    yhat = np.where(tc > tm, tc, tm)
    e = np.full(len(y), np.nan, np.float32)
    ok = ne & (y > 0)
    e[ok] = (np.abs(yhat[ok] - y[ok]) / y[ok]).astype(np.float32)
    return e


def compare_metrics(mg, mo):
    for g in ("prefill", "decode", "all"):
        a, b = mg[g], mo[g]
        assert a["n"] == b["n"], g
        for k in ("r2", "p90", "p99"):
            if np.isnan(b[k]):
                assert np.isnan(a[k]), (g, k, a[k])
                continue
            tol = 1e-9 if k == "r2" else 2 * np.spacing(np.float32(b[k]))
            assert abs(a[k] - b[k]) <= tol * (1 if k != "r2" else max(1.0, abs(b[k]))), \
                (g, k, a[k], b[k])


@pytest.mark.parametrize("name,nb", FIT_CASES)
def test_metrics_match_oracle(L, name, nb):
    tr = tracegen.config_trace(name, nb)
    co = tracegen.config_coeffs(name)
    y = measured(tr, co, seed=9, sigma=0.1)
    y[::97] = 0.0   # y <= 0: in r^2, not in the relative errors
    y[5::211] = -1.0
    model = tracegen.perturbed_coeffs(co, 79)
    say(f"[metrics] {name} nB={tr.n_batches}")
    mo = F.metrics(tr.offsets, tr.p, tr.c, tr.shape, model, y)
    mg = gpu_metrics(L, tr, model, y)
    compare_metrics(mg, mo)
    e_o = oracle_rel_err(tr, model, y)
    nan = np.isnan(e_o)
    assert np.array_equal(np.isnan(mg["rel_err"]), nan)
    assert parity.rel_err(mg["rel_err"][~nan], e_o[~nan]).max(initial=0) <= 1e-6
    say(f"[metrics] {name}: gpu {({g: mg[g] for g in ('prefill', 'decode', 'all')})}")


def test_metrics_hand_values(L):
    """The oracle's hand example (decode r^2 = 0.95, p90 = p99 = 1/8;
    prefill p90 = 0, p99 = 1), now through the library."""
    th = np.zeros(20, np.float32)
    th[2 * 5 + 2] = 1.0
    th[0 * 5 + 1] = 1.0
    dec = [([1], [2]), ([1], [4]), ([1], [6]), ([1], [9])]
    pre = [([p], [0]) for p in range(10, 101, 10)]
    tr = tracegen.from_batches(dec + pre + [([], [])], None, 1)
    tr.shape = None
    y = np.array([2, 4, 6, 8] + list(range(10, 100, 10)) + [50, 7], np.float64)
    m = gpu_metrics(L, tr, th, y)
    assert m["decode"]["n"] == 4 and m["prefill"]["n"] == 10 and m["all"]["n"] == 14
    assert abs(m["decode"]["r2"] - 0.95) < 1e-15
    assert m["decode"]["p90"] == np.float32(0.125) and m["decode"]["p99"] == np.float32(0.125)
    assert m["prefill"]["p90"] == 0.0 and m["prefill"]["p99"] == 1.0
    assert np.isnan(m["rel_err"][-1])


def test_metrics_edge_cases(L):
    """No nonempty batch of a phase: NaN r^2 and percentiles, n = 0; all y
    equal: NaN r^2; a single error: every percentile is that error."""
    th = tracegen.config_coeffs("tiny-mixed")
    tr = tracegen.from_batches([([1, 1], [100, 200]), ([], []), ([1], [50])], None, 1)
    tr.shape = None
    y = np.array([3.0, 1.0, 3.0])
    mg = gpu_metrics(L, tr, th, y)
    mo = F.metrics(tr.offsets, tr.p, tr.c, None, th, y)
    compare_metrics(mg, mo)
    assert mg["prefill"]["n"] == 0 and np.isnan(mg["prefill"]["r2"])
    assert np.isnan(mg["prefill"]["p90"]) and np.isnan(mg["decode"]["r2"])
    tr = tracegen.from_batches([([5], [0])], None, 1)
    tr.shape = None
    mg = gpu_metrics(L, tr, th, np.array([2.0]))
    mo = F.metrics(tr.offsets, tr.p, tr.c, None, th, np.array([2.0]))
    compare_metrics(mg, mo)
    assert mg["prefill"]["p90"] == mg["prefill"]["p99"] == mo["prefill"]["p90"]


def test_metrics_no_batches(L):
    """No batches at all: every r^2 and percentile NaN, no batches counted."""
    import torch
    sums = torch.zeros((4, 0), dtype=torch.int64, device="cuda")
    phase = torch.zeros(0, dtype=torch.uint8, device="cuda")
    y = torch.zeros(0, dtype=torch.float64, device="cuda")
    m = L.fit_metrics(sums, phase, None, tracegen.config_coeffs("tiny-mixed"), y)
    for g in ("prefill", "decode", "all"):
        assert m[g]["n"] == 0
        assert np.isnan(m[g]["r2"]) and np.isnan(m[g]["p90"]) and np.isnan(m[g]["p99"])


# -------------------------------------------------------- full-size workload


def test_fit_and_metrics_full_size(L):
    """The 4M-batch heavy-tailed workload (about 5e8 requests): one fitting
    round and the metrics of the fitted fp32 coefficients against the
    oracle, every batch."""
    import torch
    tr = tracegen.config_trace("heavy-tailed")
    co = tracegen.config_coeffs("heavy-tailed")
    say(f"[fit full] heavy-tailed nB={tr.n_batches} N={tr.n_requests}")
    X, phase, ne = F.design(tr.offsets, tr.p, tr.c, tr.shape)
    tm, tc = F.segment_values(X, phase, co.astype(np.float64))
    z = tracegen.normal(10, 21, 0, tr.n_batches)
    y = np.where(ne, np.where(tc > tm, tc, tm), 0.0) * np.exp(0.05 * z)
    theta0 = tracegen.perturbed_coeffs(co, 80).astype(np.float64)
    theta_o, counts_o = F.fit(tr.offsets, tr.p, tr.c, tr.shape, y, theta0, rounds=1)
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, None)
    sums, ph = L.batch_sums(dt)
    del dt
    y_d = torch.as_tensor(y, device=sums.device)
    theta_d, counts_d = L.fit(sums, ph, tr.shape, y_d, theta0, 1)
    torch.cuda.synchronize()
    theta_g, counts_g = theta_d.cpu().numpy(), counts_d.cpu().numpy()
    assert np.array_equal(counts_g, counts_o), (counts_g, counts_o)
    st = set_checks(tr, y, theta0, theta_o, theta_g)
    say(f"[fit full] sets: {st}")
    model = theta_o.astype(np.float32)
    mo = F.metrics(tr.offsets, tr.p, tr.c, tr.shape, model, y)
    mg = L.fit_metrics(sums, ph, tr.shape, model, y_d)
    compare_metrics(mg, mo)
    say(f"[fit full] metrics gpu {mg}")
