"""Pins of the extended model's admission query (orc_admit_ext; no GPU):
the query of Sec. 1 (admission control) under Eq. 1 plus the cross term
a5*S5*sum p*c and the per-request term a6*S6*|B| (readings X1-X3)."""
import numpy as np
import pytest

import oracle


def sets28(pm, pc, dm, dc):
    return np.array(pm + pc + dm + dc, np.float32)


def test_hand_example():
    """Unit shape.  B: one prefill chunk p = 4 over a context c = 8, so
    X = (1, P, C, Q, n^2, R, n) = (1, 4, 8, 16, 1, 32, 1).  Prefill MEM =
    (8, 1, 0.5, 0, 0, 0.25, 2) gives 8 + 4 + 4 + 0 + 0 + 8 + 2 = 26; COMP =
    (1, 2, 0, 0.25, 0, 0, 0) gives 1 + 8 + 4 = 13: f(B) = 26.
    B' adds (p, c) = (2, 4): X' = (1, 6, 12, 20, 4, 40, 2); MEM 8 + 6 + 6 +
    10 + 4 = 34, COMP 1 + 12 + 5 = 18: f(B') = 34 (prefill MEM), delta 8.
    The candidate's terms under MEM with |B'| = 2: 8/2 + 2 + 2 + 0 + 0 +
    0.25*8 + 2 = 12 (the other request's: 4 + 4 + 4 + 8 + 2 = 22; 12 + 22 =
    34); under COMP: 1/2 + 4 + 0 + 1 = 5.5."""
    co = sets28([8, 1, 0.5, 0, 0, 0.25, 2], [1, 2, 0, 0.25, 0, 0, 0], [0] * 7, [0] * 7)
    r = oracle.admit_ext([4], [8], 2, 4, None, co)
    assert r["T_after"] == 34.0 and r["delta"] == 8.0 and r["share"] == 12.0
    assert r["TM_after"] == 34.0 and r["TC_after"] == 18.0 and r["regime"] == 0
    assert r["share_alt"] == 5.5


def test_cross_term_flips_the_segment():
    """Decode batch p = (1, 1), c = (100, 300); candidate (1, 200).  Decode
    MEM = (50, 0, 1, 0, 0, 0, 0): f = 50 + C; COMP = (0, 0, 0, 0, 0, 1.5, 0):
    f = 1.5 R = 1.5 C in decode.  B: MEM 450, COMP 600: f(B) = 600 (COMP).
    B': C = 600: MEM 650, COMP 900: f(B') = 900, delta 300, the candidate's
    share 1.5*200 = 300 (regime decode COMP = 3)."""
    co = sets28([0] * 7, [0] * 7, [50, 0, 1, 0, 0, 0, 0], [0, 0, 0, 0, 0, 1.5, 0])
    r = oracle.admit_ext([1, 1], [100, 300], 1, 200, None, co)
    assert r["T_after"] == 900.0 and r["delta"] == 300.0 and r["share"] == 300.0
    assert r["regime"] == 3


@pytest.mark.parametrize("seed", range(6))
def test_reduces_to_the_eq1_query(seed):
    """With a5 = a6 = 0 every output equals orc_admit's, bit for bit."""
    rng = np.random.default_rng(seed)
    shape = {"n_layers": 32, "hidden": 4096, "n_q_heads": 32, "n_kv_heads": 8, "head_dim": 128,
             "ffn": 14336, "vocab": 128256, "weight_bytes": 2, "kv_bytes": 2}
    co20 = (rng.uniform(0.5, 2.0, 20) * np.repeat([1e-6, 1e-9, 1e-6, 1e-9, 0.01], 4)).astype(
        np.float32)
    co28 = np.zeros(28, np.float32)
    for g in range(4):
        co28[g * 7:g * 7 + 5] = co20[g * 5:(g + 1) * 5]
    n = int(rng.integers(0, 30))
    pre = seed % 2 == 0
    p = rng.integers(1, 3000, n) if pre else np.ones(n, np.int64)
    c = rng.integers(0, 5000, n) if pre else rng.integers(1, 100000, n)
    for cand in ((1, 777), (int(rng.integers(2, 500)), 0), (17, 4096)):
        a = oracle.admit(p, c, cand[0], cand[1], shape, co20)
        b = oracle.admit_ext(p, c, cand[0], cand[1], shape, co28)
        assert a == b, (cand, a, b)


def test_refuses_wrong_coefficient_count():
    with pytest.raises(ValueError):
        oracle.admit_ext([1], [5], 1, 5, None, np.ones(20, np.float32))
