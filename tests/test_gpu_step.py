"""GPU parity of one scheduling step (Sec. 1, admission control; Sec. 2.1,
last paragraph): a trace of at most 4096 requests and 1024 batches runs in
the single-workgroup step kernel.  Every output against the oracle, and
latency, regime and shares bit for bit against the library's host
attributor (same operations); on both sides of the step limits the tile
path takes over and must agree as well."""
import sys

import numpy as np
import pytest

import oracle
import parity
import tracegen

pytestmark = pytest.mark.gpu


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


def step_trace(seed, sizes, n_tenants, prefill_frac=0.3):
    rng = np.random.default_rng(seed)
    sizes = np.asarray(sizes, np.int64)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    N = int(off[-1])
    p = np.ones(N, np.int32)
    c = rng.integers(1, 1 << 17, N).astype(np.int32)
    for b in np.nonzero(rng.random(len(sizes)) < prefill_frac)[0]:
        p[off[b]:off[b + 1]] = rng.integers(1, 8192, sizes[b])
        c[off[b]:off[b + 1]] = rng.integers(0, 2, sizes[b]) * rng.integers(0, 4096, sizes[b])
    t = rng.integers(0, n_tenants, N).astype(np.int32)
    return tracegen.Trace(off, p, c, t, n_tenants, None)


def check(L, tr, shape, co, T, ws=None, name=""):
    import torch
    say(f"[step] {name}: nB={tr.n_batches} N={tr.n_requests} T={T}")
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    out = L.attribute(dt, shape, co, T, ws=ws if ws is not None else
                      L.workspace(tr.n_batches, tr.n_requests, T))
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in out.items()}
    ref = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, shape, co, T)
    st = parity.compare(ref, tr.offsets, g["latency"], g["regime"], g["share"], g["tenant_sums"])
    h = L.llmv_attribute_host(tr.offsets, tr.p, tr.c, tr.tenant, shape, co, T)
    for k in ("latency", "regime", "share"):
        assert np.array_equal(g[k], h[k]), (name, k)
    np.testing.assert_allclose(g["tenant_sums"], h["tenant_sums"], rtol=1e-12)
    return st


@pytest.mark.parametrize("n", [1, 2, 63, 64, 65, 256, 1000, 1024, 4095, 4096])
def test_one_batch_steps(L, n):
    tr = step_trace(n, [n], 16, prefill_frac=0.5)
    st = check(L, tr, tracegen.SHAPES["llama3.1-8b"], tracegen.config_coeffs("heavy-tailed"), 16,
               name=f"one batch of {n}")
    say(f"[step] n={n}: {st}")


@pytest.mark.parametrize("case", ["many-small", "ragged", "empties", "max-batches", "one-tenant"])
def test_multi_batch_steps(L, case):
    rng = np.random.default_rng(sum(map(ord, case)))
    T = 37
    if case == "many-small":
        sizes = rng.integers(1, 8, 500)
    elif case == "ragged":
        sizes = rng.integers(0, 300, 13)
    elif case == "empties":
        sizes = [0, 0, 5, 0, 1, 0, 0, 200, 0, 3, 0, 0]
    elif case == "max-batches":
        sizes = rng.integers(0, 5, 1024)
    else:
        sizes = rng.integers(1, 100, 40)
    tr = step_trace(len(sizes), sizes, T)
    if case == "one-tenant":
        tr.tenant[:] = 5
    check(L, tr, tracegen.SHAPES["qwen2.5-32b"], tracegen.base_coeffs(71), T, name=case)


def test_step_without_workspace_and_outputs(L):
    """The step path needs no workspace; each output is independent."""
    import torch
    tr = step_trace(9, [100, 0, 56], 4)
    co = tracegen.base_coeffs(72)
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    full = L.llmv_attribute_host(tr.offsets, tr.p, tr.c, tr.tenant, None, co, 4)
    for outs in (("latency",), ("regime",), ("share",), ("tenant_sums",)):
        o = {k: None for k in ("latency", "regime", "share", "tenant_sums")}
        dev = dt.p.device
        if "latency" in outs:
            o["latency"] = torch.empty(3, dtype=torch.float32, device=dev)
        if "regime" in outs:
            o["regime"] = torch.empty(3, dtype=torch.uint8, device=dev)
        if "share" in outs:
            o["share"] = torch.empty(156, dtype=torch.float32, device=dev)
        if "tenant_sums" in outs:
            o["tenant_sums"] = torch.empty(4, dtype=torch.float64, device=dev)
        L.llmv_attribute(dt, None, co, o["latency"], o["regime"], o["share"], 4,
                         o["tenant_sums"], None)
        torch.cuda.synchronize()
        for k in outs:
            if k == "tenant_sums":
                np.testing.assert_allclose(o[k].cpu().numpy(), full[k], rtol=1e-12)
            else:
                assert np.array_equal(o[k].cpu().numpy(), full[k]), (outs, k)


@pytest.mark.parametrize("N,nB,T", [(4096, 64, 16), (4097, 64, 16), (1500, 1024, 16),
                                    (1500, 1025, 16), (900, 30, 4096), (900, 30, 4097)])
def test_step_limits(L, N, nB, T):
    """Both sides of each step limit (requests, batches, tenants): the step
    kernel on one side, the tile kernels on the other, both against the
    oracle and the host attributor."""
    rng = np.random.default_rng(N + nB + T)
    cuts = np.sort(rng.integers(0, N + 1, nB - 1))
    sizes = np.diff(np.concatenate([[0], cuts, [N]]))
    tr = step_trace(N + T, sizes, T)
    check(L, tr, tracegen.SHAPES["qwen2.5-14b"], tracegen.base_coeffs(73), T,
          name=f"N={N} nB={nB} T={T}")
