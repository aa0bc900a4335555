"""Parity rules between the HIP path and the oracle (shared by the tests,
the smoke check and the benchmark's parity check).

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
The 1e-5 bound.  The GPU path computes the batch sums exactly in integers,
the batch model and the four share constants k0..k3 in fp64, then rounds the
constants to fp32 and forms each share as three fp32 FMAs
(k0 + k1 p + k2 c + k3 p^2, with p^2 itself rounded to fp32 for p > 2^12).
For nonnegative coefficients every term is nonnegative, so each rounding
costs at most 2^-24 relative of the exact result: four constant roundings,
one p^2 rounding and three FMA roundings bound the share's error by about
8 * 2^-24 ~ 5e-7 (measured: 1.7e-7).  Latencies are fp64 rounded once to
fp32 (<= 2^-24); tenant sums add fp32 shares in fp64 (the shares' bound).
1e-5 leaves a margin of more than an order of magnitude while catching any
wrong or missing term.
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


def compare_all_shares(offsets, get_share, ref_share, ref_TM, ref_TC, ref_regime, regime,
                       latency=None, alt_shares=None, chunk=1 << 26):
    """Every share of a (large) trace against the oracle, in slices of whole
    batches of at most `chunk` requests (one batch when it is larger).
    get_share(lo, hi): the GPU shares of requests [lo, hi) as a host array.
    ref_share: the oracle's shares for its own segment choice; regime: the
    GPU's regimes; alt_shares(bids): the oracle's shares of batches `bids`
    for the other segment (tie zone only; needed only when the GPU chose the
    other segment somewhere).  Also checks that every batch's GPU shares add
    up (in fp64) to the oracle's latency for the GPU's segment and to the GPU
    latency.  Returns the max relative errors."""
    offsets = np.asarray(offsets)
    nB = len(offsets) - 1
    regime = np.asarray(regime)
    nonempty = offsets[1:] > offsets[:-1]
    gseg = np.where(nonempty, regime % 2, 0)
    same = ~nonempty | (gseg == np.asarray(ref_regime) % 2)
    want_T = np.where(nonempty, np.where(gseg == 1, ref_TC, ref_TM), 0.0)
    lat = None if latency is None else np.asarray(latency, np.float64)
    worst, worst_sum, checked = 0.0, 0.0, 0
    b0 = 0
    while b0 < nB:
        b1 = int(np.searchsorted(offsets, offsets[b0] + chunk, side="right")) - 1
        b1 = min(max(b1, b0 + 1), nB)
        lo, hi = int(offsets[b0]), int(offsets[b1])
        if hi > lo:
            g = np.asarray(get_share(lo, hi), np.float64)
            sizes = np.diff(offsets[b0:b1 + 1])
            keep = np.repeat(same[b0:b1], sizes)
            e = rel_err(g[keep], np.asarray(ref_share[lo:hi])[keep])
            if e.size:
                k = int(np.argmax(e))
                worst = max(worst, float(e[k]))
                assert worst <= RTOL, \
                    f"share rel err {worst:.3e} at request {lo + np.flatnonzero(keep)[k]}"
            checked += int(keep.sum())
            nz = sizes > 0
            starts = (offsets[b0:b1] - lo)[nz]
            tot = np.add.reduceat(g, starts)
            T = want_T[b0:b1][nz]
            es = np.abs(tot - T) / np.maximum(np.abs(T), 1e-30)
            if lat is not None:
                Lg = lat[b0:b1][nz]
                es = np.maximum(es, np.abs(tot - Lg) / np.maximum(np.abs(Lg), 1e-30))
            if es.size:
                worst_sum = max(worst_sum, float(es.max()))
                assert worst_sum <= RTOL, \
                    f"shares of batch {b0 + np.flatnonzero(nz)[int(np.argmax(es))]} sum off"
            # batches in the tie zone where the GPU took the other segment
            tb = b0 + np.flatnonzero(~same[b0:b1])
            if tb.size:
                assert alt_shares is not None, "tie-zone batches need the oracle's other shares"
                alt = alt_shares(tb)
                idx = np.concatenate([np.arange(offsets[b], offsets[b + 1]) for b in tb])
                e = rel_err(g[idx - lo], alt)
                worst = max(worst, float(e.max()))
                assert worst <= RTOL, f"share rel err {worst:.3e} in a tie-zone batch"
                checked += idx.size
        b0 = b1
    assert checked == int(offsets[-1]), (checked, int(offsets[-1]))
    return {"share": worst, "share_sum": worst_sum, "shares_checked": checked}
