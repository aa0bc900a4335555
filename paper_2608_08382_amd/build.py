"""Builds libllmv.so in-tree with hipcc for gfx950."""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SOURCES = [os.path.join(PKG, "csrc", "api.hip"), os.path.join(PKG, "csrc", "fit.hip")]
DEPS = SOURCES + [os.path.join(PKG, "csrc", h) for h in ("kernels.hpp", "groups.hpp", "fit.hpp", "host.hpp", "model.hpp", "step.hpp")] + [
    os.path.join(ROOT, "include", "llmv.h")]
OUT = os.path.join(PKG, "libllmv.so")
# bandwidth calibration kernels (measurement context for the benchmark; not
# part of libllmv's C ABI)
CALIB_SOURCES = [os.path.join(PKG, "csrc", "calib.hip")]
CALIB_OUT = os.path.join(PKG, "libllmv_calib.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # no packed-FP32 instructions in generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # fp64 atomic adds as hardware instructions, not CAS loops
    "-munsafe-fp-atomics",
    # products rounded before their adds (no contraction into fused
    # multiply-adds), on the device and the host alike; the shares' fused
    # multiply-adds are written out as fmaf
    "-ffp-contract=off",
    "-Wall",
]


def build(out: str = OUT, verbose: bool = False, sources=None) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    sources = SOURCES if sources is None else sources
    cmd = [hipcc, *HIPCC_FLAGS, "-I", os.path.join(ROOT, "include"), *sources, "-o", out + ".tmp"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    if verbose and r.stderr:
        print(r.stderr)
    os.replace(out + ".tmp", out)
    return out


def is_stale(out: str = OUT) -> bool:
    if not os.path.exists(out):
        return True
    t = os.path.getmtime(out)
    return any(os.path.getmtime(d) > t for d in DEPS)


def build_calib(verbose: bool = False) -> str:
    return build(CALIB_OUT, verbose, CALIB_SOURCES)


if __name__ == "__main__":
    print(build(verbose=True))
    print(build_calib(verbose=True))
