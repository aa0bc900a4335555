"""Seeded synthetic inputs for LLMVisor batched latency attribution.

This module produces INPUTS only: model shapes, coefficient vectors and
traces of co-batched scheduling steps (CSR batch offsets plus per-request
prompt/context lengths and tenant ids).  It holds none of the attribution
arithmetic, and both the HIP library's tests/benchmark and the oracle consume
the same arrays it returns.

The paper's own workloads are synthetic (Appendix A, "Workloads"); the
recipes here stand in for them.  Heavy generation runs in ``tracegen.c``
(counter-based SplitMix64, OpenMP): a value depends only on
(seed, stream, index), never on the thread count.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "libtracegen.so")
_SRC = os.path.join(_HERE, "tracegen.c")
CFLAGS = ["-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra"]

# Model shapes of the models the paper evaluates (Sec. 3.1, Appendix A) and a
# 70B-class shape for what-if sweeps.  Values follow the public model
# configurations; weights and KV cache in bf16 (2 bytes per element).
SHAPES = {
    "llama3.1-8b": dict(n_layers=32, hidden=4096, n_q_heads=32, n_kv_heads=8,
                        head_dim=128, ffn=14336, vocab=128256, weight_bytes=2, kv_bytes=2),
    "qwen2.5-14b": dict(n_layers=48, hidden=5120, n_q_heads=40, n_kv_heads=8,
                        head_dim=128, ffn=13824, vocab=152064, weight_bytes=2, kv_bytes=2),
    "qwen2.5-32b": dict(n_layers=64, hidden=5120, n_q_heads=40, n_kv_heads=8,
                        head_dim=128, ffn=27648, vocab=152064, weight_bytes=2, kv_bytes=2),
    "70b-like": dict(n_layers=80, hidden=8192, n_q_heads=64, n_kv_heads=8,
                     head_dim=128, ffn=28672, vocab=128256, weight_bytes=2, kv_bytes=2),
}
SHAPE_FIELDS = ("n_layers", "hidden", "n_q_heads", "n_kv_heads", "head_dim", "ffn",
                "vocab", "weight_bytes", "kv_bytes")

_lock = threading.Lock()
_lib = None


def build(out: str = _SO) -> str:
    subprocess.run(["gcc", *CFLAGS, _SRC, "-o", out, "-lm"], check=True)
    return out


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_SO):
                build()
            lib = ctypes.CDLL(_SO)
            P = ctypes.c_void_p
            i64, i32, u64, f64 = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64, ctypes.c_double
            lib.tg_sizes.argtypes = [i32, u64, i64, P]
            lib.tg_sizes.restype = ctypes.c_int
            lib.tg_fill.argtypes = [i32, u64, i64, P, P, P, P, i32]
            lib.tg_fill.restype = ctypes.c_int
            lib.tg_uniform.argtypes = [u64, u64, i64, i64, P]
            lib.tg_uniform.restype = None
            lib.tg_normal.argtypes = [u64, u64, i64, i64, P]
            lib.tg_normal.restype = None
            lib.tg_zipf.argtypes = [u64, u64, i64, i64, i32, f64, P]
            lib.tg_zipf.restype = ctypes.c_int
            _lib = lib
    return _lib


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p)


# ---------------------------------------------------------------------------
# Primitive draws (exposed for tests of the generator itself)

def uniform(seed: int, stream: int, start: int, n: int) -> np.ndarray:
    """U in [0, 1): (u >> 11) * 2^-53 of SplitMix64 output (seed, stream, i)."""
    out = np.empty(n, np.float64)
    _load().tg_uniform(seed, stream, start, n, _p(out))
    return out


def normal(seed: int, stream: int, start: int, n: int) -> np.ndarray:
    """N(0,1) by Box-Muller from the uniforms at indices 2i and 2i+1."""
    out = np.empty(n, np.float64)
    _load().tg_normal(seed, stream, start, n, _p(out))
    return out


def zipf(seed: int, stream: int, start: int, n: int, n_items: int, s: float) -> np.ndarray:
    """Zipf(s) over 0..n_items-1: P(k) proportional to (k+1)^-s, inverse CDF."""
    out = np.empty(n, np.int32)
    rc = _load().tg_zipf(seed, stream, start, n, n_items, s, _p(out))
    if rc != 0:
        raise ValueError("bad zipf arguments")
    return out


# ---------------------------------------------------------------------------
# Coefficients (the paper prints none; these are synthetic, in microseconds
# per feature unit)

# Anchors: a bandwidth of 4e6 bytes/us and a compute rate of 5e8 FLOP/us.
_BW, _FL = 4.0e6, 5.0e8
_MEM_ANCHOR = (1 / _BW, 0.1 / _FL, 1 / _BW, 0.5 / _FL, 0.01)
_COMP_ANCHOR = (0.1 / _BW, 1 / _FL, 1 / _BW, 1 / _FL, 0.01)
_SIGMA = (0.2, 0.2, 0.02, 0.2, 0.02)
STREAM_COEFF = 11
STREAM_PERTURB = 12


def base_coeffs(seed: int) -> np.ndarray:
    """20 positive fp32 coefficients, index (phase*2+segment)*5+k: each is its
    anchor times exp(sigma_k * Z), Z ~ N(0,1) drawn per (phase, segment, k)."""
    z = normal(seed, STREAM_COEFF, 0, 20)
    out = np.empty(20, np.float64)
    for ph in range(2):
        for seg in range(2):
            anchor = _MEM_ANCHOR if seg == 0 else _COMP_ANCHOR
            for k in range(5):
                i = (ph * 2 + seg) * 5 + k
                out[i] = anchor[k] * np.exp(_SIGMA[k] * z[i])
    return out.astype(np.float32)


# Extended model: a5 (per processed-token/cached-key pair, attention FLOPs)
# and a6 (per request, output-projection FLOPs), anchored like a3 and a1.
_EXT_MEM_ANCHOR = (0.5 / _FL, 0.1 / _FL)
_EXT_COMP_ANCHOR = (1 / _FL, 1 / _FL)
_EXT_SIGMA = (0.2, 0.2)
STREAM_EXT = 13


def ext_coeffs(seed: int) -> np.ndarray:
    """28 positive fp32 coefficients, index (phase*2+segment)*7+k: k < 5 are
    base_coeffs(seed); a5, a6 are anchor * exp(sigma * Z), Z ~ N(0,1) drawn
    per (phase, segment, k) from their own stream."""
    base = base_coeffs(seed)
    z = normal(seed, STREAM_EXT, 0, 8)
    out = np.empty(28, np.float64)
    for g in range(4):
        anchor = _EXT_MEM_ANCHOR if g % 2 == 0 else _EXT_COMP_ANCHOR
        out[g * 7:g * 7 + 5] = base[g * 5:(g + 1) * 5]
        for j in range(2):
            out[g * 7 + 5 + j] = anchor[j] * np.exp(_EXT_SIGMA[j] * z[g * 2 + j])
    return out.astype(np.float32)


def perturbed_coeffs(base: np.ndarray, seed: int) -> np.ndarray:
    """Each of the 20 coefficients times U[0.8, 1.2]."""
    u = uniform(seed, STREAM_PERTURB, 0, 20)
    return (base.astype(np.float64) * (0.8 + 0.4 * u)).astype(np.float32)


def sweep_coeffs(base: np.ndarray, n: int = 256) -> np.ndarray:
    """[n, 20]: variant 0 is the base draw, variant j >= 1 uses seed 5000 + j."""
    out = np.empty((n, 20), np.float32)
    out[0] = base
    for j in range(1, n):
        out[j] = perturbed_coeffs(base, 5000 + j)
    return out


# ---------------------------------------------------------------------------
# Traces

class Trace:
    """CSR trace: offsets [nB+1] int64, p/c/tenant [N] int32."""

    def __init__(self, offsets, p, c, tenant, n_tenants, shape, name=""):
        self.offsets = offsets
        self.p = p
        self.c = c
        self.tenant = tenant
        self.n_tenants = int(n_tenants)
        self.shape = shape
        self.name = name

    @property
    def n_batches(self):
        return len(self.offsets) - 1

    @property
    def n_requests(self):
        return len(self.p)

    def sizes(self):
        return np.diff(self.offsets)


# Recipes: kind ids shared with tracegen.c.
KIND_TINY_MIXED = 1
KIND_DECODE_ONLY = 2
KIND_CHUNKED_PREFILL = 3
KIND_HEAVY_TAILED = 4
KIND_SWEEP_MIXED = 5

# name -> (kind, n_batches, shape, n_tenants, description)
CONFIGS = {
    "tiny-mixed": (KIND_TINY_MIXED, 1000, "llama3.1-8b", 16,
                   "1k batches, size U[1,32]; 30% prefill batches (prompt lognormal "
                   "median 512 sigma 1 clipped [16,8192], c=0), decode p=1 c~U[128,8192]; "
                   "16 tenants uniform; Llama3.1-8B"),
    "decode-only": (KIND_DECODE_ONLY, 1_000_000, "qwen2.5-14b", 64,
                    "1M batches, size U[1,256]; p=1, c lognormal median 2048 sigma 1.2 "
                    "clipped [1,32768]; 64 tenants Zipf(1.1); Qwen2.5-14B"),
    "chunked-prefill": (KIND_CHUNKED_PREFILL, 1_000_000, "qwen2.5-32b", 256,
                        "1M batches, 8192-token budget: 0-4 prefill chunks (length "
                        "U[64,4096], prefix U[0,16384], truncated to the budget) then "
                        "decodes (p=1, c lognormal median 1024 sigma 1.2 clipped "
                        "[1,32768]) up to 256 sequences; 256 tenants uniform; Qwen2.5-32B"),
    "heavy-tailed": (KIND_HEAVY_TAILED, 4_000_000, "llama3.1-8b", 1024,
                     "4M batches, size min(1024, 1+floor(86*(U^(-1/1.5)-1))) (Lomax, "
                     "alpha 1.5); 20% prefill batches (p lognormal median 256 sigma 1 "
                     "clipped [1,16384], c=0), decode p=1 c~U[1,131072]; 1024 tenants "
                     "Zipf(1.2); Llama3.1-8B"),
    "whatif-sweep": (KIND_SWEEP_MIXED, 100_000, "llama3.1-8b", 1024,
                     "100k batches, size U[1,256]; 30% prefill batches (as tiny-mixed); "
                     "1024 tenants Zipf(1.2); evaluated under 4 shapes x 256 coefficient "
                     "vectors"),
}
CONFIG_SEED = {"tiny-mixed": 1, "decode-only": 2, "chunked-prefill": 3,
               "heavy-tailed": 4, "whatif-sweep": 5}


def generate(kind: int, n_batches: int, seed: int, n_tenants: int, shape=None,
             name: str = "") -> Trace:
    """Two passes: batch sizes, then the per-request fields."""
    lib = _load()
    sizes = np.empty(n_batches, np.int64)
    if lib.tg_sizes(kind, seed, n_batches, _p(sizes)) != 0:
        raise ValueError(f"unknown trace kind {kind}")
    offsets = np.zeros(n_batches + 1, np.int64)
    np.cumsum(sizes, out=offsets[1:])
    N = int(offsets[-1])
    p = np.empty(N, np.int32)
    c = np.empty(N, np.int32)
    t = np.empty(N, np.int32)
    if lib.tg_fill(kind, seed, n_batches, _p(offsets), _p(p), _p(c), _p(t), n_tenants) != 0:
        raise ValueError(f"trace fill failed for kind {kind}")
    return Trace(offsets, p, c, t, n_tenants, shape, name)


def config_trace(name: str, n_batches: int | None = None) -> Trace:
    """The named workload; ``n_batches`` overrides the batch count (a prefix
    of the same recipe: batch b depends only on (seed, b))."""
    kind, nb, shape, nt, _ = CONFIGS[name]
    return generate(kind, nb if n_batches is None else n_batches, CONFIG_SEED[name], nt,
                    SHAPES[shape], name)


def config_coeffs(name: str) -> np.ndarray:
    return base_coeffs(100 + CONFIG_SEED[name])


def from_batches(batches, tenants=None, n_tenants=1) -> Trace:
    """Build a trace from a list of (p_list, c_list) pairs."""
    sizes = [len(b[0]) for b in batches]
    offsets = np.zeros(len(batches) + 1, np.int64)
    offsets[1:] = np.cumsum(sizes)
    p = np.array([v for b in batches for v in b[0]], np.int32)
    c = np.array([v for b in batches for v in b[1]], np.int32)
    if tenants is None:
        t = np.zeros(len(p), np.int32)
    else:
        t = np.array([v for tb in tenants for v in tb], np.int32)
    return Trace(offsets, p, c, t, n_tenants, None)
