"""OLS fitting of Eq. 1's coefficient sets and the accuracy metrics: the
plain fp64 CPU oracle (numpy).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: only the test suite,
the smoke check and the benchmark's CPU-baseline leg may import it.  It
shares no code with the HIP library; batch sums and shape constants come
from the C oracle (``orc.c``).

What it computes:
* Sec. 2.1: Eq. 1's coefficients are fitted by ordinary least squares on
  profiled batch latencies, giving four sets (beta, a1..a4): two phases times
  the memory-bound and the compute-bound segment.
* Sec. 3 and Appendix A (Metrics): the accuracy of a coefficient set against
  measured latencies as the coefficient of determination r^2 and the 90th
  and 99th percentiles of the relative error, per phase.

Readings where the paper is silent (each applied in the function below):
* F1 Segment membership while fitting.  The paper fits a two-segment form
  per phase but does not say which profiled batches belong to which segment.
  Fitting proceeds in rounds.  A round assigns every nonempty batch to the
  segment whose prediction under the current coefficients is larger (the
  roofline max used at evaluation, ties to the memory-bound segment), then
  refits each (phase, segment) set by OLS over its batches.  The first round
  starts from coefficients the caller gives.
* F2 Identifiability.  Inside one set a feature can be structurally absent:
  in decode every p is 1, so sum p^2 = sum p for every batch and a1, a3 act
  as one coefficient; without cached prefixes every prefill c is 0, so a2
  has no data.  Tested exactly on the integer sums: when Q == P for every
  batch of the set, the p^2 coefficient a3 keeps its starting value; when
  C == 0 for every batch, a2 does.  The remaining coefficients are fitted by
  OLS to y minus the kept terms.  A set with fewer batches than free
  coefficients, or whose free columns have lower rank, keeps all its
  coefficients; the rank is a property of the columns, not of their units,
  so it is judged (numerically) on the columns scaled to unit norm.
* F3 r^2 = 1 - sum (y - yhat)^2 / sum (y - mean y)^2 over the nonempty
  batches of the group (0 batches: NaN; all y equal: NaN).
* F4 Relative error |yhat - y| / y over the nonempty batches with y > 0,
  rounded to fp32; the p-th percentile is the ceil(p * n)-th smallest (the
  nearest-rank definition), p = 90/100 and 99/100 in exact integer arithmetic.
* F5 The extended model (readings X1-X3: Eq. 1 plus a5*S5*sum p*c and
  a6*S6*|B|) is fitted the same way with seven columns.  Two more columns
  can be structurally absent, tested exactly on the integer sums: when
  R == C for every batch of the set (every request with a context processes
  one token, so the cross term is the c term), a5 keeps its starting value;
  when P == |B| for every batch (every request processes one token, so the
  per-request term is the p term), a6 does.  C == 0 everywhere gives R == 0
  == C, so a5 is kept with a2.
"""
from __future__ import annotations

import numpy as np

import oracle

GROUPS = ((0, 0), (0, 1), (1, 0), (1, 1))  # (phase, segment) = regime order


def batch_state(offsets, p, c, ext=False):
    """Exact per-batch sums (|B|, P, C, Q[, R = sum p*c]) and the phase."""
    return oracle.batch_sums_ext(offsets, p, c) if ext else oracle.batch_sums(offsets, p, c)


def design(offsets, p, c, shape, ext=False):
    """Eq. 1's per-batch feature vector X_b = (S0, S1*P, S2*C, S3*Q, |B|^2)
    (Sec. 2.1), with ext the extended model's (..., S5*R, S6*|B|) (F5); the
    phase of each batch and the nonempty mask."""
    sums, phase = batch_state(offsets, p, c, ext)
    n, P, C, Q = (sums[k].astype(np.float64) for k in range(4))
    if ext:
        S = oracle.shape_constants_ext(shape)
        R = sums[4].astype(np.float64)
        cols = [np.full_like(n, S[0]), S[1] * P, S[2] * C, S[3] * Q, n * n, S[4] * R, S[5] * n]
    else:
        S = oracle.shape_constants(shape)
        cols = [np.full_like(n, S[0]), S[1] * P, S[2] * C, S[3] * Q, n * n]
    return np.stack(cols, axis=1), phase, sums[0] > 0


def segment_values(X, phase, theta):
    """Eq. 1 (or the extended model) under both segment sets of each batch's
    phase: (T_M, T_C), the terms added in order k = 0, 1, ..."""
    K = X.shape[1]
    th = np.asarray(theta, np.float64).reshape(2, 2, K)
    ph = np.where(phase == 1, 1, 0)
    tm = np.zeros(len(X))
    tc = np.zeros(len(X))
    for k in range(K):
        tm = tm + th[ph, 0, k] * X[:, k]
        tc = tc + th[ph, 1, k] * X[:, k]
    return tm, tc


def free_columns(sums, idx, ext=False):
    """F2, F5: the coefficients a set's batches can determine.  Column 3
    (p^2) is dropped when Q == P for every batch, column 2 (c) when C == 0
    for every batch; with ext column 5 (p*c) when R == C and column 6 (|B|)
    when P == |B| for every batch; integer tests on the exact sums."""
    free = list(range(7 if ext else 5))
    if np.all(sums[2][idx] == 0):
        free.remove(2)
    if np.all(sums[3][idx] == sums[1][idx]):
        free.remove(3)
    if ext and np.all(sums[4][idx] == sums[2][idx]):
        free.remove(5)
    if ext and np.all(sums[1][idx] == sums[0][idx]):
        free.remove(6)
    return free


def fit(offsets, p, c, shape, y, theta0, rounds, ext=False):
    """Fitted theta (fp64 [20], layout (phase*2 + segment)*5 + k; with ext
    [28], (phase*2 + segment)*7 + k) and the number of batches of each
    (phase, segment) set in the last round."""
    X, phase, ne = design(offsets, p, c, shape, ext)
    sums, _ = batch_state(offsets, p, c, ext)
    K = X.shape[1]
    y = np.asarray(y, np.float64)
    theta = np.asarray(theta0, np.float64).copy()
    counts = np.zeros(4, np.int64)
    for _ in range(rounds):
        tm, tc = segment_values(X, phase, theta)
        seg = np.where(tc > tm, 1, 0)  # F1: roofline max, ties to MEM
        new = theta.copy()
        for g, (ph, s) in enumerate(GROUPS):
            idx = ne & (phase == ph) & (seg == s)
            counts[g] = int(idx.sum())
            if counts[g] == 0:
                continue
            free = free_columns(sums, idx, ext)  # F2, F5
            kept = [k for k in range(K) if k not in free]
            if counts[g] < len(free):
                continue
            yf = y[idx] - X[idx][:, kept] @ theta[g * K + np.array(kept, int)] if kept else y[idx]
            # The rank of the free columns does not depend on their scale,
            # but a numerical rank on raw columns does (S1*P and |B|^2 differ
            # by up to 17 orders of magnitude): rank and solution are taken on
            # unit-norm columns, then unscaled.  Every free column is nonzero.
            Xf = X[idx][:, free]
            D = np.linalg.norm(Xf, axis=0)
            sol, _, rank, _ = np.linalg.lstsq(Xf / D, yf, rcond=None)
            if rank == len(free):
                new[g * K + np.array(free, int)] = sol / D
        theta = new
    return theta, counts


def metrics(offsets, p, c, shape, coeffs, y, ext=False):
    """{"prefill"|"decode"|"all": {"r2", "p90", "p99", "n"}} for fp32
    coefficients (the model as evaluated everywhere else; [28] with ext)
    against measured latencies y."""
    X, phase, ne = design(offsets, p, c, shape, ext)
    y = np.asarray(y, np.float64)
    tm, tc = segment_values(X, phase, np.asarray(coeffs, np.float32).astype(np.float64))
    yhat = np.where(tc > tm, tc, tm)
    out = {}
    for name, sel in (("prefill", ne & (phase == 0)), ("decode", ne & (phase == 1)),
                      ("all", ne)):
        ys, yh = y[sel], yhat[sel]
        n = len(ys)
        r2 = float("nan")
        if n > 0:
            ss_tot = float(np.sum((ys - ys.mean()) ** 2))
            if ss_tot > 0:
                r2 = 1.0 - float(np.sum((ys - yh) ** 2)) / ss_tot  # F3
        pos = ys > 0
        e = (np.abs(yh[pos] - ys[pos]) / ys[pos]).astype(np.float32)  # F4
        m = len(e)
        srt = np.sort(e)
        pct = {}
        for num, den, key in ((9, 10, "p90"), (99, 100, "p99")):
            k = (num * m + den - 1) // den  # ceil(m * num / den), exact
            pct[key] = float(srt[k - 1]) if m else float("nan")
        out[name] = {"r2": r2, "p90": pct["p90"], "p99": pct["p99"], "n": n}
    return out
