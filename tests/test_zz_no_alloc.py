"""llmv_attribute_noalloc (through the C ABI) against llmv_attribute on the
same inputs: the entry point for callers that cannot allocate uses the
library's static scratch instead of a workspace argument.  Two calls in a
row, the second on a smaller trace, each checked against llmv_attribute
(latency, regime and shares bit for bit; tenant sums up to the order of
their fp64 additions) and against the oracle; a trace whose scratch exceeds
the static array is refused before anything runs."""
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


def outputs(L, tr, dev):
    import torch
    return {"latency": torch.full((tr.n_batches,), float("nan"), dtype=torch.float32, device=dev),
            "regime": torch.full((tr.n_batches,), 0xEE, dtype=torch.uint8, device=dev),
            "share": torch.full((tr.n_requests,), float("nan"), dtype=torch.float32, device=dev),
            "tenant_sums": torch.full((tr.n_tenants,), float("nan"), dtype=torch.float64,
                                      device=dev)}


def one_case(L, name, nb):
    import torch
    tr = tracegen.config_trace(name, nb)
    co = tracegen.config_coeffs(name)
    say(f"[noalloc] {name}: nB={tr.n_batches} N={tr.n_requests} T={tr.n_tenants}")
    dt = L.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    a = outputs(L, tr, dt.p.device)
    L.llmv_attribute_noalloc(dt, tr.shape, co, a["latency"], a["regime"], a["share"],
                             tr.n_tenants, a["tenant_sums"])
    b = L.attribute(dt, tr.shape, co, tr.n_tenants)
    torch.cuda.synchronize()
    a = {k: v.cpu().numpy() for k, v in a.items()}
    b = {k: v.cpu().numpy() for k, v in b.items()}
    for k in ("latency", "regime", "share"):
        assert np.array_equal(a[k], b[k]), (name, k)
    np.testing.assert_allclose(a["tenant_sums"], b["tenant_sums"], rtol=1e-12)
    ref = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, tr.shape, co, tr.n_tenants)
    st = parity.compare(ref, tr.offsets, a["latency"], a["regime"], a["share"], a["tenant_sums"])
    say(f"[noalloc] {name}: {st}")


def test_noalloc_two_calls_second_smaller(L):
    # 2.5M requests: the multi-workgroup path (chunk table, claim counter,
    # tenant partials in the static scratch); then 0.4M requests on the same
    # scratch, then a 16k-request trace (the single-launch path)
    one_case(L, "heavy-tailed", 20_000)
    one_case(L, "decode-only", 3_000)
    one_case(L, "tiny-mixed", None)


def test_noalloc_refuses_past_the_scratch(L):
    """4096 tenants over 4M requests: the tenant partials of up to 652
    workgroups alone take 21 MB, more than the static 16 MiB.  EINVAL,
    nothing written."""
    import torch
    N, T = 4_000_000, 4096
    off = np.arange(0, N + 1, 100, dtype=np.int64)
    rng = np.random.default_rng(1)
    dt = L.DeviceTrace.from_host(off, np.ones(N, np.int32), rng.integers(1, 99, N).astype(np.int32),
                                 rng.integers(0, T, N).astype(np.int32))
    assert L.llmv_workspace_size(len(off) - 1, N, T) > 16 << 20
    ts = torch.full((T,), -1.0, dtype=torch.float64, device=dt.p.device)
    with pytest.raises(L.LlmvError) as e:
        L.llmv_attribute_noalloc(dt, None, np.ones(20, np.float32), None, None, None, T, ts)
    assert e.value.code == L.LLMV_EINVAL
    torch.cuda.synchronize()
    assert bool((ts == -1.0).all())
