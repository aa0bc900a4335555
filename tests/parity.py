"""Parity rules between the HIP path and the oracle (shared by the tests,
the smoke check and the benchmark's sampled check).

Rules, for coefficients >= 0 (LLMVisor Sec. 2.1, Eq. 1; Sec. 2, Problem
formulation):
  1. phase bit-exact;
  2. regime bit-exact outside the tie zone |T_C - T_M| <= 1e-6*max(T_M, T_C);
     inside it either segment is accepted, and latency and shares are then
     compared with the oracle's values for the segment the GPU chose;
  3. latency, shares and tenant sums within 1e-5 relative (denominator
     max(|oracle|, 1e-30); an oracle 0 needs an exact 0);
  4. the fp64 sum of a batch's GPU shares within 1e-5 of both the GPU and
     the oracle batch latency.
The 1e-5 bound: shares are evaluated in fp64 and rounded once to fp32
(relative error <= 2^-24 ~ 6e-8) and latencies likewise, so 1e-5 leaves a
margin of two orders of magnitude while catching any wrong term.
"""
import numpy as np

RTOL = 1e-5
TIE = 1e-6


def rel_err(got, want):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    if got.size == 0:
        return np.zeros(0)
    err = np.abs(got - want) / np.maximum(np.abs(want), 1e-30)
    err[(want == 0) & (got == 0)] = 0.0
    err[(want == 0) & (got != 0)] = np.inf
    return err


def tie_zone(TM, TC):
    return np.abs(TC - TM) <= TIE * np.maximum(TM, TC)


def compare(ref, offsets, latency=None, regime=None, share=None, tenant_sums=None,
            batch_ids=None):
    """ref: oracle outputs for the batches `batch_ids` (all when None) of a
    trace with `offsets`; GPU arrays indexed like the full trace (latency,
    regime by batch; share by request).  Returns a dict of max errors."""
    offsets = np.asarray(offsets)
    nB = len(offsets) - 1
    bids = np.arange(nB) if batch_ids is None else np.asarray(batch_ids)
    stats = {}
    ref_T, TM, TC = ref["T"], ref["TM"], ref["TC"]
    sizes = offsets[bids + 1] - offsets[bids]
    nonempty = sizes > 0
    tie = tie_zone(TM, TC) & nonempty
    gpu_seg = None
    if regime is not None:
        g = np.asarray(regime)[bids]
        r = ref["regime"]
        assert np.all(g[~nonempty] == 255), "empty batch regime"
        gph = g[nonempty] // 2
        assert np.array_equal(gph, ref["phase"][nonempty]), \
            f"phase mismatch at batches {bids[nonempty][gph != ref['phase'][nonempty]][:10]}"
        bad = (g != r) & ~tie
        assert not np.any(bad), f"regime mismatch at batches {bids[bad][:10]}"
        stats["ties"] = int(tie.sum())
        gpu_seg = np.where(nonempty, g % 2, 0)
    # expected latency for the segment the GPU chose
    if gpu_seg is not None:
        want_T = np.where(nonempty, np.where(gpu_seg == 1, TC, TM), 0.0)
        same = gpu_seg == (np.asarray(ref["regime"]) % 2)
    else:
        want_T = ref_T
        same = np.ones(len(bids), bool)
    if latency is not None:
        g = np.asarray(latency, np.float64)[bids]
        e = rel_err(g, want_T)
        stats["latency"] = float(e.max()) if e.size else 0.0
        assert stats["latency"] <= RTOL, \
            f"latency rel err {stats['latency']:.3e} at batch {bids[np.argmax(e)]}"
    if share is not None:
        share = np.asarray(share, np.float64)
        worst, worst_sum = 0.0, 0.0
        ref_off = np.zeros(len(bids) + 1, np.int64)
        ref_off[1:] = np.cumsum(sizes)
        lat = None if latency is None else np.asarray(latency, np.float64)
        for k, b in enumerate(bids):
            if sizes[k] == 0:
                continue
            gs = share[offsets[b]:offsets[b + 1]]
            rs = ref["share" if same[k] else "share_alt"][ref_off[k]:ref_off[k + 1]]
            e = rel_err(gs, rs)
            worst = max(worst, float(e.max()))
            tot = gs.sum()
            es = abs(tot - want_T[k]) / max(abs(want_T[k]), 1e-30)
            if lat is not None:
                es = max(es, abs(tot - lat[b]) / max(abs(lat[b]), 1e-30))
            worst_sum = max(worst_sum, es)
            assert worst <= RTOL, f"share rel err {worst:.3e} in batch {b}"
            assert worst_sum <= RTOL, f"shares of batch {b} sum off by {worst_sum:.3e}"
        stats["share"] = worst
        stats["share_sum"] = worst_sum
    if tenant_sums is not None:
        e = rel_err(tenant_sums, ref["tenant_sums"])
        stats["tenant"] = float(e.max()) if e.size else 0.0
        assert stats["tenant"] <= RTOL, \
            f"tenant rel err {stats['tenant']:.3e} at tenant {np.argmax(e)}"
    return stats


def sub_trace(offsets, p, c, tenant, bids):
    """The batches `bids` of a trace as a trace of their own (for running
    the oracle batch by batch on a sample of a large trace)."""
    offsets = np.asarray(offsets)
    sizes = offsets[np.asarray(bids) + 1] - offsets[np.asarray(bids)]
    off = np.zeros(len(bids) + 1, np.int64)
    off[1:] = np.cumsum(sizes)
    idx = np.concatenate([np.arange(offsets[b], offsets[b + 1]) for b in bids] +
                         [np.zeros(0, np.int64)])
    t = None if tenant is None else np.asarray(tenant)[idx]
    return off, np.asarray(p)[idx], np.asarray(c)[idx], t
