"""GPU parity of the extended model's admission query (llmv_admit_ext
through the C ABI, from llmv_batch_sums_ext's state) against orc_admit_ext:
outputs within 1e-5 relative (a delta against the latency it is a
difference of), regimes exact outside the tie zone; with a5 = a6 = 0 the
outputs equal llmv_admit's bit for bit."""
import numpy as np
import pytest

import oracle
import parity
import tracegen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_08382_amd import llmv
    llmv.load()
    torch.cuda.set_device(0)
    return llmv


def gpu_sums(L, tr, ext=True):
    import torch
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, None)
    sums, phase = L.batch_sums(dt, ext=ext)
    torch.cuda.synchronize()
    return sums, phase


def gpu_admit(L, sums, phase, shape, co, cb, cp, cc, ext=True):
    import torch
    dev = sums.device
    out = L.admit(sums, phase, shape, co, torch.as_tensor(np.asarray(cb, np.int64), device=dev),
                  torch.as_tensor(np.asarray(cp, np.int32), device=dev),
                  torch.as_tensor(np.asarray(cc, np.int32), device=dev), ext=ext)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def test_hand_example(L):
    """The worked query of test_oracle_admission_ext.py: f(B') = 34, delta 8,
    the candidate's share 12, regime prefill MEM."""
    co = np.array([8, 1, 0.5, 0, 0, 0.25, 2, 1, 2, 0, 0.25, 0, 0, 0] + [0] * 14, np.float32)
    tr = tracegen.from_batches([([4], [8])], [[0]], 1)
    sums, phase = gpu_sums(L, tr)
    g = gpu_admit(L, sums, phase, None, co, [0], [2], [4])
    assert g["t_after"][0] == 34.0 and g["delta"][0] == 8.0 and g["share"][0] == 12.0
    assert g["regime"][0] == 0


@pytest.mark.parametrize("seed", range(4))
def test_admit_ext_random(L, seed):
    names = ["tiny-mixed", "decode-only", "chunked-prefill", "heavy-tailed"]
    rng = np.random.default_rng(300 + seed)
    tr = tracegen.config_trace(names[seed], None if seed == 0 else 1500)
    shape = tracegen.SHAPES[sorted(tracegen.SHAPES)[seed]]
    co = tracegen.ext_coeffs(100 + tracegen.CONFIG_SEED[names[seed]])
    m = 2000
    cb = rng.integers(0, tr.n_batches, m)
    pre = rng.random(m) < 0.4
    cp = np.where(pre, rng.integers(1, 8192, m), 1).astype(np.int32)
    cc = np.where(rng.random(m) < 0.5, 0, rng.integers(1, 131072, m)).astype(np.int32)
    sums, phase = gpu_sums(L, tr)
    g = gpu_admit(L, sums, phase, shape, co, cb, cp, cc)
    worst = {"t_after": 0.0, "delta": 0.0, "share": 0.0}
    ties = 0
    for j in range(m):
        b = cb[j]
        lo, hi = tr.offsets[b], tr.offsets[b + 1]
        r = oracle.admit_ext(tr.p[lo:hi], tr.c[lo:hi], cp[j], cc[j], shape, co)
        if parity.tie_zone(np.array([r["TM_after"]]), np.array([r["TC_after"]]))[0]:
            ties += 1
            continue
        assert g["regime"][j] == r["regime"], (seed, j)
        for k, ref in (("t_after", r["T_after"]), ("delta", r["delta"]), ("share", r["share"])):
            if k == "delta":
                e = abs(float(g[k][j]) - ref) / max(abs(ref), abs(r["T_after"]), 1e-30)
            else:
                e = float(parity.rel_err(np.array([g[k][j]], np.float64), np.array([ref]))[0])
            worst[k] = max(worst[k], e)
    print(f"[admit ext] seed {seed}: ties {ties}, max rel err {worst}", flush=True)
    for k, v in worst.items():
        assert v <= parity.RTOL, (seed, k, v)


def test_zero_extension_is_the_eq1_query(L):
    tr = tracegen.config_trace("chunked-prefill", 1000)
    co20 = tracegen.config_coeffs("chunked-prefill")
    co28 = np.zeros(28, np.float32)
    for g in range(4):
        co28[g * 7:g * 7 + 5] = co20[g * 5:(g + 1) * 5]
    rng = np.random.default_rng(5)
    m = 1000
    cb = rng.integers(-2, tr.n_batches + 2, m)  # a few out of range
    cp = rng.integers(1, 500, m).astype(np.int32)
    cc = rng.integers(0, 9000, m).astype(np.int32)
    s5, ph5 = gpu_sums(L, tr, ext=True)
    s4, ph4 = gpu_sums(L, tr, ext=False)
    a = gpu_admit(L, s4, ph4, tr.shape, co20, cb, cp, cc, ext=False)
    b = gpu_admit(L, s5, ph5, tr.shape, co28, cb, cp, cc, ext=True)
    for k in a:
        assert np.array_equal(a[k], b[k], equal_nan=(k != "regime")), k
