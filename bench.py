#!/usr/bin/env python3
"""Benchmark: batched LLMVisor latency attribution on one MI355X.

One step = one llmv_attribute call over the whole trace (per-request
features, per-batch Eq. 1 evaluation and segment choice, per-request shares,
per-tenant sums), inputs already resident in HBM.  Prints ONE JSON line.

  python bench.py [--steps K] [--warmup W] [--workload heavy-tailed]
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E
PROFILE_COUNTERS = os.path.join(ROOT, "profiles", "k_tiles_heavy-tailed_counters.json")
SWEEP_COUNTERS = os.path.join(ROOT, "profiles", "k_sweep_groups_whatif_counters.json")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_08382_amd", "csrc", f)
                  for f in ("kernels.hpp", "api.hip")]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_sha():
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def algorithmic_bytes(n_requests, n_batches):
    """Bytes the method must move per step: p, c, tenant (int32) in and the
    fp32 share out per request; the int64 offset in and the fp32 latency and
    uint8 regime out per batch (plus the closing offset).  Tenant sums
    (n_tenants doubles) are negligible and left out."""
    return 16 * n_requests + 13 * n_batches + 8


def traffic_from_profile(workload, n_req, n_b):
    """HBM bytes per launch of the tile kernel from committed rocprofv3 PMC
    counters, if they were taken on the current kernel source."""
    try:
        prof = json.load(open(PROFILE_COUNTERS))
    except (OSError, ValueError):
        return None
    if prof.get("kernel_source_sha") != kernel_source_sha() or prof.get("workload") != workload:
        return None
    return prof.get("hbm_bytes_per_launch")


def cpu_info():
    """Host CPU model and logical CPU count (context for the oracle's rate)."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "cpu_model": model}


def cpu_baseline(tr, coeffs, gpu_out, budget_s=30.0):
    """The oracle (single thread, fp64) on the same host arrays, with the same
    outputs as the GPU step, timed.  Its results then check every output of
    the GPU step: latency and regime of every batch, every share (copied back
    in slices), every tenant sum."""
    import numpy as np
    import oracle
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import parity

    nB = tr.n_batches
    # bounded sample: a prefix of the batches sized to the time budget at an
    # assumed ~20 ns per request, never more than the whole trace
    max_req = int(budget_s / 20e-9)
    nb = nB if tr.n_requests <= max_req else int(np.searchsorted(tr.offsets, max_req))
    nb = max(1, min(nb, nB))
    off = tr.offsets[:nb + 1]
    nreq = int(off[-1])
    log(f"[bench] oracle on {nb} batches / {nreq} requests ...")
    t0 = time.perf_counter()
    ref = oracle.attribute(off, tr.p[:nreq], tr.c[:nreq], tr.tenant[:nreq], tr.shape, coeffs,
                           tr.n_tenants, ("T", "TM", "TC", "phase", "regime", "share",
                                          "tenant_sums"))
    dt = time.perf_counter() - t0
    rate = nreq / dt
    stats = parity.compare(ref, off, gpu_out["latency"][:nb], gpu_out["regime"][:nb], None,
                           gpu_out["tenant_sums"] if nb == nB else None)

    def alt_shares(bids):
        so, sp, sc, st = parity.sub_trace(off, tr.p, tr.c, tr.tenant, bids)
        return oracle.attribute(so, sp, sc, st, tr.shape, coeffs, tr.n_tenants,
                                ("share_alt",))["share_alt"]

    stats.update(parity.compare_all_shares(off, gpu_out["share_slice"], ref["share"], ref["TM"],
                                           ref["TC"], ref["regime"], gpu_out["regime"][:nb],
                                           gpu_out["latency"][:nb], alt_shares))
    sample = (f"full trace ({nreq} requests)" if nb == nB
              else f"first {nb} of {nB} batches ({nreq} requests)")
    return {"value": rate, "unit": "requests/s", "cores": 1, "kind": "oracle",
            "sample": sample, "seconds": round(dt, 3), **cpu_info()}, stats


def calibration(hip, stream, dt, share, reps=5):
    """STREAM-style rates of the attribution step's access mix on this GPU:
    plain coalesced kernels (libllmv_calib) reading the trace's own p, c and
    tenant arrays and writing the share array, over the same request count.
    For each access kind (read 12 B, write 4 B, read 12 B + write 4 B per
    request, the last also as wave tiles dealt round-robin) and each choice
    of plain or non-temporal loads and stores, the best of a few launch
    shapes (grid, elements per thread, tiles per chunk) is reported, in GB/s
    of bytes moved."""
    import ctypes
    import torch
    from paper_2608_08382_amd import build as hipbuild

    lib = ctypes.CDLL(hipbuild.CALIB_OUT)
    P = ctypes.c_void_p
    lib.llmv_calib_stream.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                      P, P, P, P, ctypes.c_int64, P, P, ctypes.c_int]
    lib.llmv_calib_stream.restype = ctypes.c_int
    n4 = dt.n_requests // 4
    sink = torch.zeros(4, dtype=torch.int32, device=share.device)
    cus = torch.cuda.get_device_properties(share.device).multi_processor_count
    ptrs = [P(x.data_ptr()) for x in (dt.p, dt.c, dt.tenant, share)]

    def run(mode, flags, unroll, grid, chunk):
        rc = lib.llmv_calib_stream(mode, flags, unroll, grid, *ptrs, n4, P(sink.data_ptr()),
                                   P(stream), chunk)
        if rc != 0:
            raise RuntimeError("llmv_calib_stream failed")

    # kind: (mode, bytes per request, flag choices, launch shapes (unroll,
    # workgroups per CU, chunk))
    grid_stride = [(u, w, 1) for u in (1, 2, 4) for w in (4, 8)]
    wave_tiles = [(2, 2, 2), (2, 4, 2), (4, 2, 1), (4, 2, 8), (7, 2, 1), (2, 2, 8)]
    kinds = {"read": (0, 12, (0, 1), grid_stride), "write": (1, 4, (0, 2), grid_stride),
             "mix_12r_4w": (2, 16, (0, 1, 2, 3), grid_stride),
             "mix_12r_4w_wave_tiles": (3, 16, (0, 3), wave_tiles)}
    flag_names = {0: "plain", 1: "nt_loads", 2: "nt_stores", 3: "nt_loads_stores"}
    out = {}
    for kind, (mode, bpr, flag_set, shapes) in kinds.items():
        for flags in flag_set:
            best = None
            for unroll, per_cu, chunk in shapes:
                grid = cus * per_cu
                run(mode, flags, unroll, grid, chunk)
                torch.cuda.synchronize()
                ev = [(hip.create(), hip.create()) for _ in range(reps)]
                for a, b in ev:
                    hip.record(a, stream)
                    run(mode, flags, unroll, grid, chunk)
                    hip.record(b, stream)
                torch.cuda.synchronize()
                ms = sorted(hip.elapsed_ms(a, b) for a, b in ev)[reps // 2]
                gbps = bpr * 4 * n4 / (ms / 1e3) / 1e9
                if best is None or gbps > best["gbps"]:
                    best = {"gbps": gbps, "ms": ms, "unroll": unroll, "grid": grid, "chunk": chunk}
            name = f"{kind}_{flag_names[flags]}"
            out[name] = best
            log(f"[bench] calibration {name}: {best['gbps']:.0f} GB/s "
                f"(grid {best['grid']}, unroll {best['unroll']}, chunk {best['chunk']})")
    best_mix = max(v["gbps"] for k, v in out.items() if k.startswith("mix"))
    best_grid_stride = max(v["gbps"] for k, v in out.items()
                           if k.startswith("mix") and "wave_tiles" not in k)
    return {"unit": "GB/s", "bytes_per_request": {"read": 12, "write": 4, "mix_12r_4w": 16},
            "n_requests": 4 * n4, "kinds": out, "best_mix_gbps": best_mix,
            "best_mix_frac_of_peak": best_mix / PEAK_HBM_GBPS,
            "best_grid_stride_mix_gbps": best_grid_stride}


def bench_configs(hip, stream, steps, with_oracle):
    """The attribution step on the other single-GPU workloads: the tiny mixed
    trace (1k batches; launch-bound, L2-resident, no roofline claim), the
    decode-only trace (1M batches, Qwen2.5-14B) and the chunked-prefill trace
    (1M batches, Qwen2.5-32B).  Each step between HIP events (the median
    step), the tile kernel between the library's own events, and, with the
    oracle, every output checked."""
    import numpy as np
    import torch
    import tracegen
    from paper_2608_08382_amd import llmv

    res = {}
    for name in ("tiny-mixed", "decode-only", "chunked-prefill"):
        tr = tracegen.config_trace(name)
        co = tracegen.config_coeffs(name)
        dt = llmv.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
        dev = dt.p.device
        lat = torch.empty(tr.n_batches, dtype=torch.float32, device=dev)
        reg = torch.empty(tr.n_batches, dtype=torch.uint8, device=dev)
        share = torch.empty(tr.n_requests, dtype=torch.float32, device=dev)
        tsum = torch.empty(tr.n_tenants, dtype=torch.float64, device=dev)
        ws = llmv.workspace(tr.n_batches, tr.n_requests, tr.n_tenants)

        def step():
            llmv.llmv_attribute(dt, tr.shape, co, lat, reg, share, tr.n_tenants, tsum, ws)

        for _ in range(3):
            step()
        torch.cuda.synchronize()
        # each step between its own HIP events (GPU clock; a pause of the
        # host between two enqueues is not counted), the median reported
        evs = [(hip.create(), hip.create()) for _ in range(steps)]
        sevs = [(hip.create(), hip.create()) for _ in range(steps)]
        for i in range(steps):
            hip.record(sevs[i][0], stream)
            llmv.llmv_set_kernel_events(*evs[i])
            step()
            hip.record(sevs[i][1], stream)
        llmv.llmv_set_kernel_events(None, None)
        torch.cuda.synchronize()
        ms = sorted(hip.elapsed_ms(a, b) for a, b in sevs)[steps // 2]
        k_ms = sum(hip.elapsed_ms(a, b) for a, b in evs) / steps
        nbytes = algorithmic_bytes(tr.n_requests, tr.n_batches)
        gbps = nbytes / (k_ms / 1e3) / 1e9
        r = {"n_requests": tr.n_requests, "n_batches": tr.n_batches, "n_tenants": tr.n_tenants,
             "shape": tracegen.CONFIGS[name][2], "ms_per_step": ms,
             "value": tr.n_requests / (ms / 1e3), "unit": "requests/s", "kernel_ms": k_ms,
             "algorithmic_bytes": nbytes}
        if name == "tiny-mixed":
            r["note"] = ("launch-bound: 0.27 MB, one workgroup in one launch; not a roofline "
                         "number")
        else:
            r["roofline"] = {"bound": "hbm", "achieved": gbps, "peak": PEAK_HBM_GBPS,
                             "unit": "GB/s", "frac": gbps / PEAK_HBM_GBPS, "kernel": "k_tiles"}
        log(f"[bench] {name}: {ms:.4f} ms/step, tile kernel {k_ms:.4f} ms, {gbps:.0f} GB/s")
        if with_oracle:
            import oracle
            sys.path.insert(0, os.path.join(ROOT, "tests"))
            import parity
            ref = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, tr.shape, co,
                                   tr.n_tenants, ("T", "TM", "TC", "phase", "regime", "share",
                                                  "tenant_sums"))
            lat_h, reg_h = lat.cpu().numpy(), reg.cpu().numpy()
            st = parity.compare(ref, tr.offsets, lat_h, reg_h, None, tsum.cpu().numpy())

            def alt_shares(bids):
                so, sp, sc, stt = parity.sub_trace(tr.offsets, tr.p, tr.c, tr.tenant, bids)
                return oracle.attribute(so, sp, sc, stt, tr.shape, co, tr.n_tenants,
                                        ("share_alt",))["share_alt"]

            st.update(parity.compare_all_shares(
                tr.offsets, lambda lo, hi: share[lo:hi].cpu().numpy(), ref["share"], ref["TM"],
                ref["TC"], ref["regime"], reg_h, lat_h, alt_shares))
            r["parity"] = st
        res[name] = r
        del dt, lat, reg, share, tsum, ws
        torch.cuda.empty_cache()
    return res


def bench_sweep(hip, stream, with_oracle):
    """What-if sweep: tenant sums of the 100k-batch mixed trace under 4 model
    shapes x 256 coefficient vectors, one llmv_attribute_sweep call; then the
    same under 4 x 256 settings of the extended model
    (llmv_attribute_sweep_ext)."""
    import numpy as np
    import torch
    import tracegen
    from paper_2608_08382_amd import llmv

    tr = tracegen.config_trace("whatif-sweep")
    co = tracegen.sweep_coeffs(tracegen.config_coeffs("whatif-sweep"), 256)
    names = ["llama3.1-8b", "qwen2.5-14b", "qwen2.5-32b", "70b-like"]
    shapes = [tracegen.SHAPES[k] for k in names]
    dt = llmv.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    out = torch.empty((4, 256, tr.n_tenants), dtype=torch.float64, device=dt.p.device)
    ws = llmv.sweep_workspace(tr.n_batches, tr.n_requests, tr.n_tenants)
    llmv.llmv_attribute_sweep(dt, shapes, co, tr.n_tenants, out, ws)
    torch.cuda.synchronize()
    reps = 3
    evs = [(hip.create(), hip.create()) for _ in range(reps)]
    for a, b in evs:
        hip.record(a, stream)
        llmv.llmv_attribute_sweep(dt, shapes, co, tr.n_tenants, out, ws)
        hip.record(b, stream)
    torch.cuda.synchronize()
    ms = sorted(hip.elapsed_ms(a, b) for a, b in evs)[reps // 2]
    variants = 4 * 256
    res = {"metric": "attributed request-variants/sec", "value": tr.n_requests * variants / (ms / 1e3),
           "unit": "request-variants/s", "ms": ms, "variants": variants,
           "n_requests": tr.n_requests, "n_batches": tr.n_batches, "n_tenants": tr.n_tenants}
    # the pass kernel's limiting resource, from the committed rocprofv3 counters
    try:
        prof = json.load(open(SWEEP_COUNTERS))
        res["bound"] = {"resource": "lds", "kernel": prof["kernel"],
                        "frac": prof["lds_busy_frac"],
                        "frac_definition": "SQ_LDS_IDX_ACTIVE / SQ_BUSY_CU_CYCLES per pass (LDS busy "
                                           "with the fp64 histogram atomics while the CUs are busy)",
                        "valu_busy_frac": prof["valu_busy_frac"], "pass_us": prof["pass_us"],
                        "source": os.path.relpath(SWEEP_COUNTERS, ROOT)}
    except (OSError, ValueError, KeyError):
        res["bound"] = None
    log(f"[bench] what-if sweep: {variants} variants in {ms:.2f} ms, "
        f"{res['value']:.3e} request-variants/s")
    if with_oracle:
        import oracle
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        import parity
        host = out.cpu().numpy()
        sample = [(0, 0), (1, 64), (2, 128), (3, 255)]
        t0 = time.perf_counter()
        worst = 0.0
        for s, v in sample:
            ref = oracle.attribute(tr.offsets, tr.p, tr.c, tr.tenant, shapes[s], co[v],
                                   tr.n_tenants, ("tenant_sums",))["tenant_sums"]
            worst = max(worst, float(parity.rel_err(host[s, v], ref).max()))
        dt_o = time.perf_counter() - t0
        assert worst <= parity.RTOL, worst
        res["cpu_baseline"] = {"value": tr.n_requests * len(sample) / dt_o,
                               "unit": "request-variants/s", "cores": 1, "kind": "oracle",
                               "sample": f"{len(sample)} of {variants} variants, full trace"}
        res["parity_tenant_max_rel_err"] = worst
    # the extended model: 28 coefficients per setting
    del ws
    co28 = np.stack([tracegen.ext_coeffs(600 + j) for j in range(256)])
    wsx = llmv.sweep_workspace(tr.n_batches, tr.n_requests, tr.n_tenants, ext=True)
    llmv.llmv_attribute_sweep_ext(dt, shapes, co28, tr.n_tenants, out, wsx)
    torch.cuda.synchronize()
    evs = [(hip.create(), hip.create()) for _ in range(reps)]
    for a, b in evs:
        hip.record(a, stream)
        llmv.llmv_attribute_sweep_ext(dt, shapes, co28, tr.n_tenants, out, wsx)
        hip.record(b, stream)
    torch.cuda.synchronize()
    msx = sorted(hip.elapsed_ms(a, b) for a, b in evs)[reps // 2]
    res["extended"] = {"ms": msx, "value": tr.n_requests * variants / (msx / 1e3),
                       "unit": "request-variants/s"}
    log(f"[bench] what-if sweep (extended model): {variants} variants in {msx:.2f} ms, "
        f"{res['extended']['value']:.3e} request-variants/s")
    if with_oracle:
        host = out.cpu().numpy()
        worst_x = 0.0
        for s, v in [(0, 3), (3, 250)]:
            ref = oracle.attribute_ext(tr.offsets, tr.p, tr.c, tr.tenant, shapes[s], co28[v],
                                       tr.n_tenants, ("tenant_sums",))["tenant_sums"]
            worst_x = max(worst_x, float(parity.rel_err(host[s, v], ref).max()))
        assert worst_x <= parity.RTOL, worst_x
        res["extended"]["parity_tenant_max_rel_err"] = worst_x
    return res


def bench_admission(hip, stream, dt, tr, coeffs, ws, with_oracle):
    """Admission queries on the trace's batches: llmv_batch_sums over every
    batch, then 2^20 candidate requests (20% prefill-type) in one llmv_admit
    call; plus the host-side latency of one query and of one single-batch
    attribution step (median of 50 synchronous calls).  Then the same
    queries under the extended model."""
    import numpy as np
    import torch
    import tracegen
    from paper_2608_08382_amd import llmv

    dev = dt.p.device
    sums = torch.empty((4, tr.n_batches), dtype=torch.int64, device=dev)
    phase = torch.empty(tr.n_batches, dtype=torch.uint8, device=dev)
    rng = np.random.default_rng(11)
    m = 1 << 20
    cb_h = rng.integers(0, tr.n_batches, m)
    pre = rng.random(m) < 0.2
    cp_h = np.where(pre, rng.integers(1, 16384, m), 1).astype(np.int32)
    cc_h = np.where(pre, 0, rng.integers(1, 131072, m)).astype(np.int32)
    cb = torch.as_tensor(cb_h, device=dev)
    cp = torch.as_tensor(cp_h, device=dev)
    cc = torch.as_tensor(cc_h, device=dev)
    out = {k: torch.empty(m, dtype=torch.float32, device=dev) for k in ("t_after", "delta", "share")}
    out["regime"] = torch.empty(m, dtype=torch.uint8, device=dev)

    def timed(fn, reps=5):
        fn()
        torch.cuda.synchronize()
        ev = [(hip.create(), hip.create()) for _ in range(reps)]
        for a, b in ev:
            hip.record(a, stream)
            fn()
            hip.record(b, stream)
        torch.cuda.synchronize()
        return sorted(hip.elapsed_ms(a, b) for a, b in ev)[reps // 2]

    ms_sums = timed(lambda: llmv.llmv_batch_sums(dt, sums, phase, ws))
    ms_admit = timed(lambda: llmv.llmv_admit(sums, phase, tr.n_batches, tr.shape, coeffs, cb, cp,
                                             cc, out["t_after"], out["delta"], out["share"],
                                             out["regime"]))
    # host-side latency of a single query (launch + completion)
    one = [x[:1] for x in (cb, cp, cc)]
    lat_q = []
    for _ in range(50):
        t0 = time.perf_counter()
        llmv.llmv_admit(sums, phase, tr.n_batches, tr.shape, coeffs, *one, out["t_after"][:1],
                        out["delta"][:1], out["share"][:1], out["regime"][:1])
        torch.cuda.synchronize()
        lat_q.append(time.perf_counter() - t0)
    # the same query on the GPU's clock (HIP events around the call)
    gq = timed(lambda: llmv.llmv_admit(sums, phase, tr.n_batches, tr.shape, coeffs, *one,
                                       out["t_after"][:1], out["delta"][:1], out["share"][:1],
                                       out["regime"][:1]), reps=21)
    res = {"metric": "admission queries/sec", "value": m / (ms_admit / 1e3), "unit": "queries/s",
           "n_candidates": m, "admit_ms": ms_admit, "n_batches": tr.n_batches,
           "batch_sums_ms": ms_sums,
           "batch_sums_gbps": (8 * tr.n_requests + 41 * tr.n_batches) / (ms_sums / 1e3) / 1e9,
           "single_query_us": float(np.median(lat_q)) * 1e6,
           "single_query_gpu_us": gq * 1e3,
           "single_step": bench_steps(hip, stream, tr.shape, coeffs, timed)}
    s256 = res["single_step"]["256"]
    res["single_step_256_us"] = s256["host_sync_us"]
    res["single_step_256_gpu_us"] = s256["gpu_clock_us"]
    log(f"[bench] admission: batch sums {ms_sums:.3f} ms, {m} queries in {ms_admit:.3f} ms "
        f"({res['value']:.3e}/s); one query {res['single_query_us']:.1f} us host-synchronous, "
        f"{res['single_query_gpu_us']:.1f} us on the GPU's clock")
    # the same 2^20 queries under the extended model, from llmv_batch_sums_ext's state
    sums5 = torch.empty((5, tr.n_batches), dtype=torch.int64, device=dev)
    llmv.llmv_batch_sums_ext(dt, sums5, phase, ws)
    co28 = tracegen.ext_coeffs(104)
    ox = {k: torch.empty_like(v) for k, v in out.items()}
    ms_ax = timed(lambda: llmv.llmv_admit_ext(sums5, phase, tr.n_batches, tr.shape, co28, cb, cp,
                                              cc, ox["t_after"], ox["delta"], ox["share"],
                                              ox["regime"]))
    del sums5
    res["extended"] = {"admit_ms": ms_ax, "value": m / (ms_ax / 1e3), "unit": "queries/s"}
    log(f"[bench] admission (extended model): {m} queries in {ms_ax:.3f} ms "
        f"({res['extended']['value']:.3e}/s)")
    if with_oracle:
        import oracle
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        import parity
        host = {k: v.cpu().numpy() for k, v in out.items()}
        idx = rng.choice(m, 300, replace=False)
        worst = 0.0
        t0 = time.perf_counter()
        for j in idx:
            b = cb_h[j]
            lo, hi = tr.offsets[b], tr.offsets[b + 1]
            r = oracle.admit(tr.p[lo:hi], tr.c[lo:hi], cp_h[j], cc_h[j], tr.shape, coeffs)
            if parity.tie_zone(np.array([r["TM_after"]]), np.array([r["TC_after"]]))[0]:
                continue
            worst = max(worst, abs(float(host["t_after"][j]) - r["T_after"]) / r["T_after"],
                        abs(float(host["share"][j]) - r["share"]) / abs(r["share"]))
        dt_o = time.perf_counter() - t0
        assert worst <= parity.RTOL, worst
        hx = {k: v.cpu().numpy() for k, v in ox.items()}
        worst_x = 0.0
        for j in idx[:100]:
            b = cb_h[j]
            lo, hi = tr.offsets[b], tr.offsets[b + 1]
            r = oracle.admit_ext(tr.p[lo:hi], tr.c[lo:hi], cp_h[j], cc_h[j], tr.shape, co28)
            if parity.tie_zone(np.array([r["TM_after"]]), np.array([r["TC_after"]]))[0]:
                continue
            worst_x = max(worst_x, abs(float(hx["t_after"][j]) - r["T_after"]) / r["T_after"],
                          abs(float(hx["share"][j]) - r["share"]) / abs(r["share"]))
        assert worst_x <= parity.RTOL, worst_x
        res["extended"]["parity_max_rel_err"] = worst_x
        res["cpu_baseline"] = {"value": len(idx) / dt_o, "unit": "queries/s", "cores": 1,
                               "kind": "oracle", "sample": f"{len(idx)} of {m} queries"}
        res["parity_max_rel_err"] = worst
    return res


def bench_fit(hip, stream, dt, tr, lat, with_oracle):
    """Fitting and accuracy metrics on the trace's batches: llmv_batch_sums,
    then llmv_fit (4 rounds) and llmv_fit_metrics against synthetic measured
    latencies, the model's latency times exp(0.05 Z)."""
    import numpy as np
    import torch
    import tracegen
    from paper_2608_08382_amd import llmv

    dev = dt.p.device
    sums, phase = llmv.batch_sums(dt)
    z = torch.as_tensor(tracegen.normal(10, 21, 0, tr.n_batches), device=dev)
    y = lat.double() * torch.exp(0.05 * z)
    del z
    theta0 = tracegen.perturbed_coeffs(tracegen.config_coeffs(tr.name), 80).astype(np.float64)
    theta = torch.empty(20, dtype=torch.float64, device=dev)
    counts = torch.empty(4, dtype=torch.int64, device=dev)
    out = torch.empty((3, 4), dtype=torch.float64, device=dev)
    err = torch.empty(tr.n_batches, dtype=torch.float32, device=dev)
    fws = llmv.fit_workspace(tr.n_batches, dev)
    rounds = 4

    def timed(fn, reps=5):
        fn()
        torch.cuda.synchronize()
        ev = [(hip.create(), hip.create()) for _ in range(reps)]
        for a, b in ev:
            hip.record(a, stream)
            fn()
            hip.record(b, stream)
        torch.cuda.synchronize()
        return sorted(hip.elapsed_ms(a, b) for a, b in ev)[reps // 2]

    ms_fit = timed(lambda: llmv.llmv_fit(sums, phase, tr.shape, y, theta0, rounds, theta, counts,
                                         fws))
    fitted = theta.cpu().numpy().astype(np.float32)
    ms_met = timed(lambda: llmv.llmv_fit_metrics(sums, phase, tr.shape, fitted, y, out, err, fws))
    o = out.cpu().numpy()
    # bytes a round must move per batch: the four sums, the phase and y
    round_bytes = 41 * tr.n_batches
    res = {"metric": "fitting rounds/sec", "value": rounds / (ms_fit / 1e3), "unit": "rounds/s",
           "n_batches": tr.n_batches, "rounds": rounds, "fit_ms": ms_fit,
           "round_ms": ms_fit / rounds,
           "round_gbps": round_bytes / (ms_fit / rounds / 1e3) / 1e9,
           "metrics_ms": ms_met, "counts": counts.cpu().tolist(),
           "r2": {"prefill": o[0, 0], "decode": o[1, 0], "all": o[2, 0]},
           "p90": {"prefill": o[0, 1], "decode": o[1, 1], "all": o[2, 1]},
           "p99": {"prefill": o[0, 2], "decode": o[1, 2], "all": o[2, 2]}}
    log(f"[bench] fit: {rounds} rounds over {tr.n_batches} batches in {ms_fit:.3f} ms "
        f"({res['round_gbps']:.0f} GB/s per round); metrics {ms_met:.3f} ms; r2 {res['r2']}")
    # the extended model: batch sums with sum p*c, fit of the 28 coefficients,
    # metrics, on the same measured latencies
    del sums
    ws = llmv.workspace(tr.n_batches, tr.n_requests, 0, dev)
    sums5 = torch.empty((5, tr.n_batches), dtype=torch.int64, device=dev)
    ms_bs = timed(lambda: llmv.llmv_batch_sums_ext(dt, sums5, phase, ws), reps=3)
    del ws
    theta0x = tracegen.ext_coeffs(104).astype(np.float64) * \
        np.random.default_rng(83).uniform(0.9, 1.1, 28)
    thetax = torch.empty(28, dtype=torch.float64, device=dev)
    ms_fx = timed(lambda: llmv.llmv_fit_ext(sums5, phase, tr.shape, y, theta0x, rounds, thetax,
                                            counts, fws))
    fittedx = thetax.cpu().numpy().astype(np.float32)
    ms_mx = timed(lambda: llmv.llmv_fit_metrics_ext(sums5, phase, tr.shape, fittedx, y, out, err,
                                                    fws))
    ox = out.cpu().numpy()
    res["extended"] = {"batch_sums_ms": ms_bs, "fit_ms": ms_fx, "round_ms": ms_fx / rounds,
                       "round_gbps": 49 * tr.n_batches / (ms_fx / rounds / 1e3) / 1e9,
                       "metrics_ms": ms_mx, "counts": counts.cpu().tolist(),
                       "r2": {"prefill": ox[0, 0], "decode": ox[1, 0], "all": ox[2, 0]}}
    log(f"[bench] fit (extended model): batch sums {ms_bs:.3f} ms; {rounds} rounds in "
        f"{ms_fx:.3f} ms; metrics {ms_mx:.3f} ms; r2 {res['extended']['r2']}")
    if with_oracle:
        from oracle import fit as F
        nb = 200_000
        n = int(tr.offsets[nb])
        y_h = y[:nb].cpu().numpy()
        t0 = time.perf_counter()
        F.fit(tr.offsets[:nb + 1], tr.p[:n], tr.c[:n], tr.shape, y_h, theta0, rounds=1)
        dt_o = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": 1.0 / dt_o * nb / tr.n_batches, "unit": "rounds/s",
                               "cores": 1, "kind": "oracle",
                               "sample": f"one round over the first {nb} batches, scaled to "
                                         f"{tr.n_batches}"}
    return res


def bench_ext(hip, stream, dt, tr, bufs, ws, steps, with_oracle):
    """The extended model (Eq. 1 plus the cross term sum p*c and the
    per-request term) on the same trace and outputs: llmv_attribute_ext
    steps between HIP events, the tile kernel on its own, and the oracle's
    extended model on sampled batches and every tenant."""
    import numpy as np
    import torch
    import tracegen
    from paper_2608_08382_amd import llmv

    lat, reg, share, tsum = bufs
    co = tracegen.ext_coeffs(100 + tracegen.CONFIG_SEED.get(tr.name, 0))

    def step():
        llmv.llmv_attribute_ext(dt, tr.shape, co, lat, reg, share, tr.n_tenants, tsum, ws)

    step()
    torch.cuda.synchronize()
    evs = [(hip.create(), hip.create()) for _ in range(steps)]
    start, stop = hip.create(), hip.create()
    hip.record(start, stream)
    for i in range(steps):
        llmv.llmv_set_kernel_events(*evs[i])
        step()
    llmv.llmv_set_kernel_events(None, None)
    hip.record(stop, stream)
    torch.cuda.synchronize()
    ms = hip.elapsed_ms(start, stop) / steps
    k_ms = sum(hip.elapsed_ms(a, b) for a, b in evs) / steps
    nbytes = algorithmic_bytes(tr.n_requests, tr.n_batches)
    gbps = nbytes / (k_ms / 1e3) / 1e9
    res = {"metric": "attributed requests/sec, extended model", "value": tr.n_requests / (ms / 1e3),
           "unit": "requests/s", "ms_per_step": ms, "kernel_ms": k_ms, "achieved_gbps": gbps,
           "frac": gbps / PEAK_HBM_GBPS, "steps": steps}
    log(f"[bench] extended model: {ms:.4f} ms/step, tile kernel {k_ms:.4f} ms, {gbps:.0f} GB/s")
    if with_oracle:
        import oracle
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        import parity
        t0 = time.perf_counter()
        ref_all = oracle.attribute_ext(tr.offsets, tr.p, tr.c, tr.tenant, tr.shape, co,
                                       tr.n_tenants, ("T", "TM", "TC", "phase", "regime",
                                                      "tenant_sums"))
        dt_o = time.perf_counter() - t0
        st = parity.compare(ref_all, tr.offsets, lat.cpu().numpy(), reg.cpu().numpy(), None,
                            tsum.cpu().numpy())
        rng = np.random.default_rng(23)
        bids = np.unique(rng.integers(0, tr.n_batches, 500))
        off, p, c, t = parity.sub_trace(tr.offsets, tr.p, tr.c, tr.tenant, bids)
        ref = oracle.attribute_ext(off, p, c, t, tr.shape, co, tr.n_tenants,
                                   ("T", "TM", "TC", "phase", "regime", "share", "share_alt"))
        idx = np.concatenate([np.arange(tr.offsets[b], tr.offsets[b + 1]) for b in bids])
        g_share = np.zeros(tr.n_requests, np.float32)
        g_share[idx] = share[torch.from_numpy(idx).to(share.device)].cpu().numpy()
        st["sampled"] = parity.compare(ref, tr.offsets, lat.cpu().numpy(), reg.cpu().numpy(),
                                       g_share, None, batch_ids=bids)
        res["cpu_baseline"] = {"value": tr.n_requests / dt_o, "unit": "requests/s", "cores": 1,
                               "kind": "oracle", "sample": "full trace, batch outputs and "
                                                           "tenant sums"}
        res["parity"] = st
    return res


def bench_many_tenants(hip, stream, dt, tr, coeffs, bufs, with_oracle, n_tenants=1 << 20):
    """The same trace with 2^20 tenants (Zipf(1.2) ids from the generator):
    tenant sums through the LDS tenant cache and global atomics instead of
    an LDS histogram.  Five llmv_attribute steps between HIP events."""
    import numpy as np
    import torch
    import tracegen
    from paper_2608_08382_amd import llmv

    lat, reg, share = bufs
    big = tracegen.generate(tracegen.KIND_HEAVY_TAILED, tr.n_batches,
                            tracegen.CONFIG_SEED.get(tr.name, 4), n_tenants, tr.shape, "many")
    assert np.array_equal(big.offsets, tr.offsets)
    ten = torch.as_tensor(big.tenant, device=dt.p.device)
    saved = dt.tenant
    dt.tenant = ten
    tsum = torch.empty(n_tenants, dtype=torch.float64, device=dt.p.device)
    ws = llmv.workspace(tr.n_batches, tr.n_requests, n_tenants)

    def step():
        llmv.llmv_attribute(dt, tr.shape, coeffs, lat, reg, share, n_tenants, tsum, ws)

    step()
    torch.cuda.synchronize()
    evs = [(hip.create(), hip.create()) for _ in range(5)]
    for a, b in evs:
        hip.record(a, stream)
        step()
        hip.record(b, stream)
    torch.cuda.synchronize()
    ms = sorted(hip.elapsed_ms(a, b) for a, b in evs)[2]
    res = {"metric": "attributed requests/sec, 2^20 tenants", "value": tr.n_requests / (ms / 1e3),
           "unit": "requests/s", "ms_per_step": ms, "n_tenants": n_tenants,
           "tenants_with_requests": int(np.count_nonzero(np.bincount(big.tenant,
                                                                     minlength=n_tenants)))}
    log(f"[bench] {n_tenants} tenants: {ms:.3f} ms/step")
    if with_oracle:
        import oracle
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        import parity
        ref = oracle.attribute(tr.offsets, tr.p, tr.c, big.tenant, tr.shape, coeffs, n_tenants,
                               ("T", "TM", "TC", "phase", "regime", "tenant_sums"))
        res["parity"] = parity.compare(ref, tr.offsets, lat.cpu().numpy(), reg.cpu().numpy(), None,
                                       tsum.cpu().numpy())
    dt.tenant = saved
    del ten, tsum, ws
    return res


def bench_big_batches(hip, stream, dt, tr, coeffs, ws, with_oracle, steps=5):
    """Batches larger than a wave tile, on the heavy-tailed trace's own
    request arrays cut into other batches: uniform batches of 1792 requests
    (one full tile), of 1793 (one request past it: every batch is held whole
    by a k_long wave), of 3585 and 16384 (streamed by a k_long wave), of
    131072 (spread over the grid in segments), and 124 batches of 4M
    requests (segments).  ms per
    llmv_attribute step (HIP events), and with the oracle every batch's
    latency and regime and every tenant sum checked."""
    import numpy as np
    import torch
    from paper_2608_08382_amd import llmv

    dev = dt.p.device
    res = {}
    cases = {"uniform_1792": (1792, tr.n_requests), "uniform_1793": (1793, tr.n_requests),
             "uniform_3585": (3585, tr.n_requests), "uniform_16384": (16384, tr.n_requests),
             "uniform_131072": (131072, tr.n_requests),
             "124_x_4M": (4_000_000, 124 * 4_000_000)}
    for name, (size, n) in cases.items():
        off = np.arange(0, n, size, dtype=np.int64)
        off = np.append(off, n)
        bt = llmv.DeviceTrace(torch.as_tensor(off, device=dev), dt.p[:n], dt.c[:n],
                              dt.tenant[:n])
        nb = len(off) - 1
        lat = torch.empty(nb, dtype=torch.float32, device=dev)
        reg = torch.empty(nb, dtype=torch.uint8, device=dev)
        share = torch.empty(n, dtype=torch.float32, device=dev)
        tsum = torch.empty(tr.n_tenants, dtype=torch.float64, device=dev)
        bws = llmv.workspace(nb, n, tr.n_tenants)

        def step():
            llmv.llmv_attribute(bt, tr.shape, coeffs, lat, reg, share, tr.n_tenants, tsum, bws)

        step()
        torch.cuda.synchronize()
        ev = [(hip.create(), hip.create()) for _ in range(steps)]
        for a, b in ev:
            hip.record(a, stream)
            step()
            hip.record(b, stream)
        torch.cuda.synchronize()
        ms = sorted(hip.elapsed_ms(a, b) for a, b in ev)[steps // 2]
        r = {"batch_size": size, "n_batches": nb, "n_requests": n, "ms_per_step": ms,
             "value": n / (ms / 1e3), "unit": "requests/s"}
        log(f"[bench] big batches {name}: {ms:.3f} ms/step ({nb} batches of {size})")
        if with_oracle:
            import oracle
            sys.path.insert(0, os.path.join(ROOT, "tests"))
            import parity
            ref = oracle.attribute(off, tr.p[:n], tr.c[:n], tr.tenant[:n], tr.shape, coeffs,
                                   tr.n_tenants, ("T", "TM", "TC", "phase", "regime",
                                                  "tenant_sums"))
            r["parity"] = parity.compare(ref, off, lat.cpu().numpy(), reg.cpu().numpy(), None,
                                         tsum.cpu().numpy())
        res[name] = r
        del bt, lat, reg, share, tsum, bws
        torch.cuda.empty_cache()
    res["ratio_1793_over_1792"] = res["uniform_1793"]["ms_per_step"] / \
        res["uniform_1792"]["ms_per_step"]
    return res


def tracegen_single_batch(n):
    """One decode batch of n requests (context U[128, 8192]), 16 tenants."""
    import numpy as np
    import tracegen
    rng = np.random.default_rng(3)
    c = rng.integers(128, 8193, n).tolist()
    t = rng.integers(0, 16, n).tolist()
    return tracegen.from_batches([([1] * n, c)], [t], 16)


def bench_steps(hip, stream, shape, coeffs, timed, sizes=(1, 64, 256, 1024)):
    """One scheduler step (one decode batch of n requests, 16 tenants):
    llmv_attribute's step kernel host-synchronous (launch to completion, the
    median of 50 calls) and on the GPU's clock (HIP events around the call),
    and the library's host attributor on the same step (median of 200
    calls); the GPU outputs checked against the host attributor's."""
    import numpy as np
    import torch
    from paper_2608_08382_amd import llmv

    res = {}
    for n in sizes:
        st = tracegen_single_batch(n)
        sdt = llmv.DeviceTrace.from_host(st.offsets, st.p, st.c, st.tenant)
        o = llmv.attribute(sdt, shape, coeffs, st.n_tenants, ws=torch.empty(0, device="cuda"))

        def call():
            llmv.llmv_attribute(sdt, shape, coeffs, o["latency"], o["regime"], o["share"],
                                st.n_tenants, o["tenant_sums"], None)

        call()
        torch.cuda.synchronize()
        lat = []
        for _ in range(50):
            t0 = time.perf_counter()
            call()
            torch.cuda.synchronize()
            lat.append(time.perf_counter() - t0)
        g = timed(call, reps=21)
        per_step = graph_step_time(hip, stream, call, o)
        h = llmv.llmv_attribute_host(st.offsets, st.p, st.c, st.tenant, shape, coeffs,
                                     st.n_tenants)
        # the C entry point called directly (arguments built once: the time
        # is the attribution plus one ctypes call)
        hl = host_step_times(llmv, st, shape, coeffs, 200)
        same = all(np.array_equal(o[k].cpu().numpy(), h[k]) for k in ("latency", "regime", "share"))
        assert same, f"step of {n}: GPU and host attributor differ"
        res[str(n)] = {"host_sync_us": float(np.median(lat)) * 1e6, "gpu_clock_us": g * 1e3,
                       "gpu_clock_us_back_to_back": per_step,
                       "host_attributor_us": float(np.median(hl)) * 1e6,
                       "gpu_equals_host_attributor": same}
        log(f"[bench] step of {n} requests: {res[str(n)]['host_sync_us']:.1f} us "
            f"host-synchronous, {res[str(n)]['gpu_clock_us']:.1f} us on the GPU's clock "
            f"({per_step:.1f} us per step back to back); host attributor "
            f"{res[str(n)]['host_attributor_us']:.1f} us")
    return res


def graph_step_time(hip, stream, call, outs, n_calls=100, replays=5):
    """GPU time per step when steps are issued back to back: n_calls calls
    captured in one HIP graph, each replay between HIP events (median);
    between replays an eager call and a synchronisation, and after each
    replay every output checked against the eager call's."""
    import numpy as np
    import torch
    call()
    torch.cuda.synchronize()
    ref = {k: v.cpu().numpy().copy() for k, v in outs.items()}
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(n_calls):
            call()
    torch.cuda.synchronize()
    per = []
    for _ in range(replays):
        call()
        torch.cuda.synchronize()
        a, b = hip.create(), hip.create()
        hip.record(a, stream)
        graph.replay()
        hip.record(b, stream)
        torch.cuda.synchronize()
        per.append(hip.elapsed_ms(a, b) * 1e3 / n_calls)
        for k, v in outs.items():
            got = v.cpu().numpy()
            if k == "tenant_sums":
                assert np.allclose(got, ref[k], rtol=1e-12, atol=0.0), "graph replay: " + k
            else:
                assert np.array_equal(got, ref[k]), "graph replay: " + k
    del graph
    return float(np.median(per))


def host_step_times(llmv, st, shape, coeffs, reps):
    """Seconds per llmv_attribute_host call on one step's host arrays."""
    import ctypes
    import numpy as np
    off = np.ascontiguousarray(st.offsets, np.int64)
    p = np.ascontiguousarray(st.p, np.int32)
    c = np.ascontiguousarray(st.c, np.int32)
    t = np.ascontiguousarray(st.tenant, np.int32)
    lat = np.zeros(st.n_batches, np.float32)
    reg = np.zeros(st.n_batches, np.uint8)
    share = np.zeros(st.n_requests, np.float32)
    ts = np.zeros(st.n_tenants, np.float64)
    ptr = [ctypes.c_void_p(a.ctypes.data) for a in (off, p, c, t, lat, reg, share, ts)]
    tr = llmv.llmv_trace(st.n_batches, st.n_requests, *ptr[:4])
    sh = llmv.make_shape(shape)
    co = (ctypes.c_float * 20)(*[float(v) for v in coeffs])
    lib = llmv.load()
    args = (ctypes.byref(tr), ctypes.byref(sh) if sh is not None else None, co, ptr[4], ptr[5],
            ptr[6], int(st.n_tenants), ptr[7])
    out = []
    for _ in range(reps):
        t0 = time.perf_counter()
        rc = lib.llmv_attribute_host(*args)
        out.append(time.perf_counter() - t0)
        assert rc == 0
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="heavy-tailed")
    ap.add_argument("--n-batches", type=int, default=None, help="override the batch count")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--breakdown", action="store_true",
                    help="also time the step with subsets of the outputs (stderr)")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the what-if sweep measurement (4 shapes x 256 coefficient vectors)")
    ap.add_argument("--no-tenants", action="store_true",
                    help="skip the 2^20-tenant measurement")
    ap.add_argument("--no-ext", action="store_true",
                    help="skip the extended-model measurement")
    ap.add_argument("--no-fit", action="store_true",
                    help="skip the fitting and metrics measurement")
    ap.add_argument("--no-admission", action="store_true",
                    help="skip the admission-query measurement")
    ap.add_argument("--no-calibration", action="store_true",
                    help="skip the STREAM-style bandwidth calibration")
    ap.add_argument("--no-big", action="store_true",
                    help="skip the batches-larger-than-a-tile measurement")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the tiny, decode-only and chunked-prefill workloads")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="also run a plain device copy of this many bytes (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the attribution path "
              "is built and measured on a single MI355X", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import tracegen
    from paper_2608_08382_amd import llmv

    llmv.load()
    torch.cuda.set_device(0)
    t0 = time.perf_counter()
    tr = tracegen.config_trace(args.workload, args.n_batches)
    coeffs = tracegen.config_coeffs(args.workload)
    log(f"[bench] {args.workload}: {tr.n_batches} batches, {tr.n_requests} requests, "
        f"generated in {time.perf_counter() - t0:.1f}s")
    dt = llmv.DeviceTrace.from_host(tr.offsets, tr.p, tr.c, tr.tenant)
    dev = dt.p.device
    lat = torch.empty(tr.n_batches, dtype=torch.float32, device=dev)
    reg = torch.empty(tr.n_batches, dtype=torch.uint8, device=dev)
    share = torch.empty(tr.n_requests, dtype=torch.float32, device=dev)
    tsum = torch.empty(tr.n_tenants, dtype=torch.float64, device=dev)
    ws = llmv.workspace(tr.n_batches, tr.n_requests, tr.n_tenants)
    torch.cuda.synchronize()

    def step():
        llmv.llmv_attribute(dt, tr.shape, coeffs, lat, reg, share, tr.n_tenants, tsum, ws)

    hip = HipEvents()
    stream = torch.cuda.current_stream().cuda_stream
    # bandwidth calibration on the same arrays (it overwrites the shares,
    # so it runs before the steps)
    calib = None if args.no_calibration else calibration(hip, stream, dt, share)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: K steps, HIP events on the stream the kernels run on:
    # one pair around the whole region, one pair around each step's tile
    # kernel (recorded by the library right before / after that launch)
    evs = [(hip.create(), hip.create()) for _ in range(args.steps)]
    start, stop = hip.create(), hip.create()
    torch.cuda.synchronize()
    hip.record(start, stream)
    for i in range(args.steps):
        llmv.llmv_set_kernel_events(*evs[i])
        step()
    llmv.llmv_set_kernel_events(None, None)
    hip.record(stop, stream)
    torch.cuda.synchronize()
    total_ms = hip.elapsed_ms(start, stop)
    kern_ms = [hip.elapsed_ms(a, b) for a, b in evs]
    ms_per_step = total_ms / args.steps
    k_avg_ms = sum(kern_ms) / len(kern_ms)
    value = tr.n_requests * args.steps / (total_ms / 1e3)
    nbytes = algorithmic_bytes(tr.n_requests, tr.n_batches)
    achieved = nbytes / (k_avg_ms / 1e3) / 1e9
    log(f"[bench] {ms_per_step:.4f} ms/step, tile kernel {k_avg_ms:.4f} ms "
        f"(min {min(kern_ms):.4f}), {achieved:.0f} GB/s algorithmic")

    if args.breakdown:
        variants = {"latency+regime": (lat, reg, None, None), "share": (None, None, share, None),
                    "tenant_sums": (None, None, None, tsum),
                    "latency+regime+share": (lat, reg, share, None)}
        for name, (a, b, c, d) in variants.items():
            ev = [(hip.create(), hip.create()) for _ in range(5)]
            for i in range(5):
                llmv.llmv_set_kernel_events(*ev[i])
                llmv.llmv_attribute(dt, tr.shape, coeffs, a, b, c, tr.n_tenants, d, ws)
            llmv.llmv_set_kernel_events(None, None)
            torch.cuda.synchronize()
            ms = min(hip.elapsed_ms(x, y) for x, y in ev)
            log(f"[bench] breakdown {name}: tile kernel {ms:.4f} ms")
    if args.copy_bytes:
        # plain device copy of known size (counter calibration): torch.neg
        # reads copy_bytes and writes copy_bytes in one elementwise kernel
        src = torch.ones(args.copy_bytes // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        ev = [(hip.create(), hip.create()) for _ in range(3)]
        for x, y in ev:
            hip.record(x, stream)
            torch.neg(src, out=dst)
            hip.record(y, stream)
        torch.cuda.synchronize()
        ms = min(hip.elapsed_ms(x, y) for x, y in ev)
        log(f"[bench] copy (neg) of {args.copy_bytes} bytes: {ms:.4f} ms, "
            f"{2 * args.copy_bytes / ms / 1e6:.0f} GB/s read+write")
        del src, dst

    reg_host = reg.cpu().numpy()
    regimes = np.bincount(reg_host[reg_host != 255], minlength=4)[:4]
    gpu_out = {"latency": lat.cpu().numpy(), "regime": reg_host,
               "tenant_sums": tsum.cpu().numpy(),
               "share_slice": lambda lo, hi: share[lo:hi].cpu().numpy()}

    traffic = traffic_from_profile(args.workload, tr.n_requests, tr.n_batches)
    result = {
        "metric": "attributed requests/sec on 1 MI355X; achieved HBM GB/s vs peak",
        "value": value,
        "unit": "requests/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i64+f64+f32",
        "dtype_detail": ("exact integer batch sums; fp64 batch model and share constants; "
                         "fp32 per-request shares (three FMAs on fp32-rounded constants); fp64 "
                         "tenant sums"),
        "data": "synthetic",
        "config": {"workload": args.workload, "n_batches": tr.n_batches,
                   "n_requests": tr.n_requests, "shape": tracegen.CONFIGS[args.workload][2],
                   "n_tenants": tr.n_tenants, "outputs": "latency,regime,share,tenant_sums"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBPS,
                     "unit": "GB/s", "frac": achieved / PEAK_HBM_GBPS,
                     "traffic": traffic, "kernel": "k_tiles",
                     "kernel_ms": k_avg_ms, "algorithmic_bytes": nbytes},
        "regime_mix": {"prefill_mem": int(regimes[0]), "prefill_comp": int(regimes[1]),
                       "decode_mem": int(regimes[2]), "decode_comp": int(regimes[3])},
    }
    if calib is not None:
        result["calibration"] = calib
        result["roofline"]["frac_of_calibrated_mix"] = achieved / calib["best_mix_gbps"]
    if not args.no_cpu_baseline:
        cb, stats = cpu_baseline(tr, coeffs, gpu_out)
        result["cpu_baseline"] = cb
        result["parity"] = {k: v for k, v in stats.items()}
        log(f"[bench] oracle {cb['value']:.3e} req/s on {cb['cores']} core; parity {stats}")
    if not args.no_configs:
        # the heavy-tailed trace stays resident; the others come and go
        result["configs"] = bench_configs(hip, stream, args.steps, not args.no_cpu_baseline)
    if not args.no_big:
        result["big_batches"] = bench_big_batches(hip, stream, dt, tr, coeffs, ws,
                                                  not args.no_cpu_baseline)
        result["big_batches"]["ratio_4M_over_step"] = \
            result["big_batches"]["124_x_4M"]["ms_per_step"] / ms_per_step
    if not args.no_ext:
        result["extended_model"] = bench_ext(hip, stream, dt, tr, (lat, reg, share, tsum), ws,
                                             max(5, args.steps // 2), not args.no_cpu_baseline)
        step()  # the Eq. 1 outputs again, for the blocks below
        torch.cuda.synchronize()
    if not args.no_tenants:
        result["many_tenants"] = bench_many_tenants(hip, stream, dt, tr, coeffs, (lat, reg, share),
                                                    not args.no_cpu_baseline)
        step()  # the Eq. 1 outputs again, for the blocks below
        torch.cuda.synchronize()
    if not args.no_admission:
        del share
        torch.cuda.empty_cache()
        result["admission"] = bench_admission(hip, stream, dt, tr, coeffs, ws,
                                              not args.no_cpu_baseline)
    if not args.no_fit:
        result["fit"] = bench_fit(hip, stream, dt, tr, lat, not args.no_cpu_baseline)
        torch.cuda.empty_cache()
    if not args.no_sweep:
        del gpu_out, dt, lat, reg, tsum, ws
        torch.cuda.empty_cache()
        result["whatif_sweep"] = bench_sweep(hip, stream, not args.no_cpu_baseline)
    print(json.dumps(result), flush=True)


class HipEvents:
    """hipEvent_t handles through the HIP runtime (ctypes)."""

    def __init__(self):
        import ctypes
        self.ct = ctypes
        self.lib = ctypes.CDLL("libamdhip64.so")
        self.lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float),
                                                 ctypes.c_void_p, ctypes.c_void_p]
        self.lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.events = []

    def _ok(self, rc, what):
        if rc != 0:
            raise RuntimeError(f"{what} failed with HIP error {rc}")

    def create(self):
        ev = self.ct.c_void_p()
        self._ok(self.lib.hipEventCreate(self.ct.byref(ev)), "hipEventCreate")
        self.events.append(ev)
        return ev

    def record(self, ev, stream):
        self._ok(self.lib.hipEventRecord(ev, self.ct.c_void_p(stream)), "hipEventRecord")

    def elapsed_ms(self, a, b):
        ms = self.ct.c_float()
        self._ok(self.lib.hipEventElapsedTime(self.ct.byref(ms), a, b), "hipEventElapsedTime")
        return ms.value


if __name__ == "__main__":
    main()
