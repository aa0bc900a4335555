"""GPU parity of the extended model's batch sums, fitting and metrics
(llmv_batch_sums_ext, llmv_fit_ext, llmv_fit_metrics_ext through the C ABI)
against the oracle (orc_batch_sums_ext, oracle/fit.py with ext=True).

The bars are those of test_gpu_fit.py: batch sums bit-exact; fitted sets
compared on the column-scaled coefficients with tol = 1e-9 + 100 eps kappa^2,
kept coefficients and rank-deficient sets exactly; segment counts exact;
r^2 within 1e-9, p90/p99 within 2 fp32 ulp, per-batch errors within 1e-6.
"""
import os
import sys

import numpy as np
import pytest

import oracle
import tracegen
from oracle import fit as F

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
from test_gpu_parity import SIZE_SETS, random_fill  # noqa: E402
from test_oracle_fit_ext import THETA_EXT, ext_trace  # noqa: E402

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


def measured_ext(tr, coeffs28, seed, sigma=0.05):
    """The extended model's T (oracle) times exp(sigma * Z), Z seeded."""
    T = oracle.attribute_ext(tr.offsets, tr.p, tr.c, None, tr.shape, coeffs28, 0, ("T",))["T"]
    z = tracegen.normal(seed, 21, 0, tr.n_batches)
    return T * np.exp(sigma * z)


def gpu_state(L, tr, y):
    import torch
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, None)
    sums, phase = L.batch_sums(dt, ext=True)
    y_d = torch.as_tensor(np.ascontiguousarray(y, np.float64), device=sums.device)
    torch.cuda.synchronize()
    return sums, phase, y_d


def gpu_fit(L, tr, y, theta0, rounds):
    import torch
    sums, phase, y_d = gpu_state(L, tr, y)
    theta = torch.full((28,), float("nan"), dtype=torch.float64, device=y_d.device)
    counts = torch.full((4,), -7, dtype=torch.int64, device=y_d.device)
    L.llmv_fit_ext(sums, phase, tr.shape, y_d, theta0, rounds, theta, counts)
    torch.cuda.synchronize()
    return theta.cpu().numpy(), counts.cpu().numpy()


def set_checks(tr, theta0, theta_o, theta_g):
    """Per set of the assignment under theta0: the scaled comparison, or
    exact keeping for kept columns and rank-deficient sets."""
    X, phase, ne = F.design(tr.offsets, tr.p, tr.c, tr.shape, ext=True)
    sums, _ = oracle.batch_sums_ext(tr.offsets, tr.p, tr.c)
    tm, tc = F.segment_values(X, phase, theta0)
    seg = np.where(tc > tm, 1, 0)
    out = {}
    for g, (ph, s) in enumerate(F.GROUPS):
        idx = ne & (phase == ph) & (seg == s)
        sl = slice(g * 7, g * 7 + 7)
        if idx.sum() == 0:
            assert np.array_equal(theta_g[sl], theta0[sl]), g
            continue
        free = F.free_columns(sums, idx, ext=True)
        kept = [k for k in range(7) if k not in free]
        assert np.array_equal(theta_g[sl][kept], theta0[sl][kept]), (g, kept)
        Xg = X[idx][:, free]
        D = np.linalg.norm(Xg, axis=0)
        kappa = np.linalg.cond(Xg / D) if idx.sum() >= len(free) else np.inf
        if kappa > 1e14 or idx.sum() < len(free):
            assert np.array_equal(theta_g[sl], theta0[sl]), (g, kappa)
            assert np.array_equal(theta_o[sl], theta0[sl]), (g, kappa)
            out[g] = (int(idx.sum()), kappa, 0.0)
            continue
        assert kappa < 1e4, (g, kappa)
        a = D * theta_g[g * 7 + np.array(free)]
        b = D * theta_o[g * 7 + np.array(free)]
        err = np.linalg.norm(a - b) / np.linalg.norm(b)
        tol = 1e-9 + 100 * EPS * kappa * kappa
        assert err <= tol, (g, err, tol, kappa)
        out[g] = (int(idx.sum()), float(kappa), float(err), kept)
    return out


@pytest.mark.parametrize("key", sorted(SIZE_SETS))
def test_batch_sums_ext_exact(L, key):
    """Every batch-size edge (wave, tile, two-pass batches larger than a
    tile); prefill batches carry contexts so that sum p*c differs from
    sum c."""
    rng = np.random.default_rng(hash(key) % 1000 + 3)
    tr = random_fill(rng, SIZE_SETS[key])
    tr.c = np.where(tr.c == 0, rng.integers(0, 3000, tr.n_requests), tr.c).astype(np.int32)
    sums, phase, _ = gpu_state(L, tr, np.zeros(tr.n_batches))
    s_o, ph_o = oracle.batch_sums_ext(tr.offsets, tr.p, tr.c)
    assert np.array_equal(sums.cpu().numpy(), s_o), key
    assert np.array_equal(phase.cpu().numpy(), ph_o), key


@pytest.mark.parametrize("name,nb", [("tiny-mixed", None), ("chunked-prefill", 20000),
                                     ("heavy-tailed", 20000), ("decode-only", 20000)])
def test_batch_sums_ext_config_traces(L, name, nb):
    tr = tracegen.config_trace(name, nb)
    sums, phase, _ = gpu_state(L, tr, np.zeros(tr.n_batches))
    s_o, ph_o = oracle.batch_sums_ext(tr.offsets, tr.p, tr.c)
    assert np.array_equal(sums.cpu().numpy(), s_o) and np.array_equal(phase.cpu().numpy(), ph_o)
    # the first four rows are llmv_batch_sums'
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, None)
    s4, ph4 = L.batch_sums(dt)
    assert np.array_equal(s4.cpu().numpy(), s_o[:4]) and np.array_equal(ph4.cpu().numpy(), ph_o)


FIT_CASES = [("tiny-mixed", None), ("chunked-prefill", 5000), ("heavy-tailed", 20000),
             ("decode-only", 5000)]


@pytest.mark.parametrize("name,nb", FIT_CASES)
def test_fit_ext_one_round_matches_oracle(L, name, nb):
    tr = tracegen.config_trace(name, nb)
    co = tracegen.ext_coeffs(100 + tracegen.CONFIG_SEED[name])
    y = measured_ext(tr, co, seed=9)
    theta0 = co.astype(np.float64) * np.random.default_rng(79).uniform(0.8, 1.2, 28)
    say(f"[fit ext] {name} nB={tr.n_batches}")
    theta_o, counts_o = F.fit(tr.offsets, tr.p, tr.c, tr.shape, y, theta0, rounds=1, ext=True)
    theta_g, counts_g = gpu_fit(L, tr, y, theta0, 1)
    assert np.array_equal(counts_g, counts_o), (counts_g, counts_o)
    say(f"[fit ext] {name}: {set_checks(tr, theta0, theta_o, theta_g)}")


def test_fit_ext_rounds_match_oracle(L):
    tr = tracegen.config_trace("chunked-prefill", 5000)
    co = tracegen.ext_coeffs(103)
    y = measured_ext(tr, co, seed=10, sigma=0.02)
    theta0 = co.astype(np.float64) * np.random.default_rng(80).uniform(0.8, 1.2, 28)
    theta_o, counts_o = F.fit(tr.offsets, tr.p, tr.c, tr.shape, y, theta0, rounds=4, ext=True)
    theta_g, counts_g = gpu_fit(L, tr, y, theta0, 4)
    assert np.array_equal(counts_g, counts_o)
    theta3, _ = F.fit(tr.offsets, tr.p, tr.c, tr.shape, y, theta0, rounds=3, ext=True)
    say(f"[fit ext rounds] {set_checks(tr, theta3, theta_o, theta_g)}")


def test_fit_ext_planted_recovery(L):
    """Noise-free latencies of planted coefficients (unit shape), 8 rounds
    from 10% off: as the oracle pin, the true segments and every
    identifiable coefficient, the decode absorptions exact."""
    tr = ext_trace(21)
    T = oracle.attribute_ext(tr.offsets, tr.p, tr.c, None, None, THETA_EXT.astype(np.float32), 0,
                             ("T", "regime"))
    counts_true = np.bincount(T["regime"][T["regime"] != 255], minlength=4)
    theta0 = THETA_EXT * np.random.default_rng(22).uniform(0.9, 1.1, 28)
    theta, counts = gpu_fit(L, tr, T["T"], theta0, 8)
    assert np.array_equal(counts, counts_true)
    want = THETA_EXT.copy()
    for g in (2, 3):
        o = g * 7
        for k in (3, 5, 6):
            want[o + k] = theta0[o + k]
        want[o + 1] = THETA_EXT[o + 1] + (THETA_EXT[o + 3] - theta0[o + 3]) + \
            (THETA_EXT[o + 6] - theta0[o + 6])
        want[o + 2] = THETA_EXT[o + 2] + (THETA_EXT[o + 5] - theta0[o + 5])
    assert np.max(np.abs(theta - want) / np.abs(want)) < 1e-6


def test_fit_ext_edge_cases(L):
    import torch
    theta0 = np.arange(1, 29, dtype=np.float64)
    tr = ext_trace(3, nb=100)
    theta, counts = gpu_fit(L, tr, np.ones(tr.n_batches), theta0, 0)
    assert np.array_equal(theta, theta0) and not counts.any()
    sums = torch.zeros((5, 0), dtype=torch.int64, device="cuda")
    phase = torch.zeros(0, dtype=torch.uint8, device="cuda")
    yd = torch.zeros(0, dtype=torch.float64, device="cuda")
    th, ct = L.fit(sums, phase, None, yd, theta0, 3, ext=True)
    torch.cuda.synchronize()
    assert np.array_equal(th.cpu().numpy(), theta0) and not ct.cpu().numpy().any()
    # fewer batches than free coefficients: kept on both sides
    tr = tracegen.from_batches([([2, 3], [10, 20]), ([1], [5]), ([3, 4], [7, 0])], None, 1)
    y = np.array([50.0, 20.0, 70.0])
    theta_o, counts_o = F.fit(tr.offsets, tr.p, tr.c, None, y, theta0, rounds=3, ext=True)
    theta, counts = gpu_fit(L, tr, y, theta0, 3)
    assert np.array_equal(theta, theta_o) and np.array_equal(theta, theta0)
    assert np.array_equal(counts, counts_o)


@pytest.mark.parametrize("name,nb", [("chunked-prefill", 20000), ("heavy-tailed", 50000)])
def test_metrics_ext_match_oracle(L, name, nb):
    import torch
    tr = tracegen.config_trace(name, nb)
    co = tracegen.ext_coeffs(100 + tracegen.CONFIG_SEED[name])
    y = measured_ext(tr, co, seed=11)
    coeffs = (co.astype(np.float64) * np.random.default_rng(81).uniform(0.95, 1.05, 28)).astype(
        np.float32)
    m_o = F.metrics(tr.offsets, tr.p, tr.c, tr.shape, coeffs, y, ext=True)
    sums, phase, y_d = gpu_state(L, tr, y)
    m_g = L.fit_metrics(sums, phase, tr.shape, coeffs, y_d, rel_err=True, ext=True)
    torch.cuda.synchronize()
    for g in ("prefill", "decode", "all"):
        assert m_g[g]["n"] == m_o[g]["n"], g
        if np.isnan(m_o[g]["r2"]):
            assert np.isnan(m_g[g]["r2"])
        else:
            assert abs(m_g[g]["r2"] - m_o[g]["r2"]) <= 1e-9, g
        for k in ("p90", "p99"):
            a, b = np.float32(m_g[g][k]), np.float32(m_o[g][k])
            assert abs(int(a.view(np.int32)) - int(b.view(np.int32))) <= 2, (g, k, a, b)
    # per-batch errors
    X, ph, ne = F.design(tr.offsets, tr.p, tr.c, tr.shape, ext=True)
    tm, tc = F.segment_values(X, ph, coeffs.astype(np.float64))
    yhat = np.where(tc > tm, tc, tm)
    e_o = np.where(ne & (y > 0), np.abs(yhat - y) / np.where(y > 0, y, 1.0), np.nan)
    e_g = m_g["rel_err"].cpu().numpy().astype(np.float64)
    assert np.array_equal(np.isnan(e_g), np.isnan(e_o))
    ok = ~np.isnan(e_o)
    assert np.all(np.abs(e_g[ok] - e_o[ok]) <= 1e-6 * np.maximum(e_o[ok], 1e-30) + 1e-12)


def test_fit_ext_full_size(L):
    """The 4M-batch heavy-tailed workload: batch sums of every batch exact,
    one round of the extended fit against the oracle."""
    tr = tracegen.config_trace("heavy-tailed")
    co = tracegen.ext_coeffs(104)
    say(f"[fit ext full] nB={tr.n_batches} N={tr.n_requests}")
    y = measured_ext(tr, co, seed=12)
    theta0 = co.astype(np.float64) * np.random.default_rng(82).uniform(0.9, 1.1, 28)
    sums, phase, y_d = gpu_state(L, tr, y)
    s_o, ph_o = oracle.batch_sums_ext(tr.offsets, tr.p, tr.c)
    assert np.array_equal(sums.cpu().numpy(), s_o) and np.array_equal(phase.cpu().numpy(), ph_o)
    import torch
    theta = torch.full((28,), float("nan"), dtype=torch.float64, device=y_d.device)
    counts = torch.full((4,), -7, dtype=torch.int64, device=y_d.device)
    L.llmv_fit_ext(sums, phase, tr.shape, y_d, theta0, 1, theta, counts)
    torch.cuda.synchronize()
    theta_o, counts_o = F.fit(tr.offsets, tr.p, tr.c, tr.shape, y, theta0, rounds=1, ext=True)
    assert np.array_equal(counts.cpu().numpy(), counts_o)
    say(f"[fit ext full] {set_checks(tr, theta0, theta_o, theta.cpu().numpy())}")
