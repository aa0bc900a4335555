"""Planted mistakes in the fitting/metrics oracle must fail its pins (no
GPU).  Each case edits a copy of oracle/fit.py with one plausible mistake,
imports the copy, and runs the pins of test_oracle_fit.py against it."""
import importlib.util
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "fit.py")
sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import test_oracle_fit as pins  # noqa: E402
import test_oracle_fit_ext as ext_pins  # noqa: E402

MUTANTS = [
    ("ties go to COMP", "seg = np.where(tc > tm, 1, 0)", "seg = np.where(tc >= tm, 1, 0)"),
    ("drops the p column instead of p^2", "        free.remove(3)", "        free.remove(1)"),
    ("r2 without 1 -", "r2 = 1.0 - float(np.sum((ys - yh) ** 2)) / ss_tot",
     "r2 = float(np.sum((ys - yh) ** 2)) / ss_tot"),
    ("percentile rank off by one", "pct[key] = float(srt[k - 1]) if m else float(\"nan\")",
     "pct[key] = float(srt[min(k, m - 1)]) if m else float(\"nan\")"),
    ("relative error over the prediction", "e = (np.abs(yh[pos] - ys[pos]) / ys[pos])",
     "e = (np.abs(yh[pos] - ys[pos]) / yh[pos])"),
    ("kept terms not subtracted",
     "yf = y[idx] - X[idx][:, kept] @ theta[g * K + np.array(kept, int)] if kept else y[idx]",
     "yf = y[idx]"),
    ("rank judged on raw columns", "D = np.linalg.norm(Xf, axis=0)", "D = np.ones(Xf.shape[1])"),
    # extended model (F5)
    ("cross term kept only without contexts", "if ext and np.all(sums[4][idx] == sums[2][idx]):",
     "if ext and np.all(sums[4][idx] == 0):"),
    # (Q == P is the same test as P == |B|: both say every p is 1)
    ("per-request term kept without contexts", "if ext and np.all(sums[1][idx] == sums[0][idx]):",
     "if ext and np.all(sums[2][idx] == 0):"),
    ("cross column from C", "S[4] * R", "S[4] * C"),
    ("per-request column |B|^2", "S[5] * n]", "S[5] * n * n]"),
]


def load(path, name):
    spec = importlib.util.spec_from_file_location(name, path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def ext_battery(F):
    saved = ext_pins.F
    try:
        ext_pins.F = F
        ext_pins.test_free_columns_by_hand()
        ext_pins.test_planted_recovery()
        ext_pins.test_planted_recovery_model_shape()
        ext_pins.test_reduces_to_the_eq1_fit()
        ext_pins.test_ols_normal_equations_hold(0)
        ext_pins.test_metrics_of_the_exact_model()
    finally:
        ext_pins.F = saved


def battery(F):
    ext_battery(F)
    saved = pins.F
    try:
        pins.F = F
        pins.test_planted_coefficients_recovered()
        pins.test_chunked_prefill_identifies_every_coefficient()
        pins.test_planted_recovery_model_shape()
        for seed in range(2):
            pins.test_ols_normal_equations_hold(seed)
        pins.test_small_set_keeps_its_coefficients()
        pins.test_ties_go_to_mem()
        pins.test_metrics_hand_values()
        pins.test_metrics_perfect_fit()
    finally:
        pins.F = saved


def test_battery_passes_on_real_source(tmp_path):
    p = tmp_path / "fit_orig.py"
    p.write_text(open(SRC).read())
    battery(load(str(p), "fit_orig"))


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new):
    text = open(SRC).read()
    assert text.count(old) == 1, f"mutation anchor for '{name}' must be unique"
    p = tmp_path / "fit_mut.py"
    p.write_text(text.replace(old, new))
    with pytest.raises((AssertionError, IndexError, ValueError)):
        battery(load(str(p), "fit_mut"))
