"""Plain fp64 CPU oracle for LLMVisor batched latency attribution.

TEST INFRASTRUCTURE ONLY.  The oracle exists to check the HIP library; only
the test suite, the smoke check and the benchmark's CPU-baseline leg may
import it.  The C source (``orc.c``) shares no code with the HIP library.

This module is a thin ctypes wrapper: argument marshalling from numpy arrays
to the C functions declared in ``orc.h``, nothing else.  What the functions
compute, and which reading of the paper each applies, is documented in
``orc.h`` / ``orc.c`` (LLMVisor Sec. 2 "Problem formulation", Sec. 2.1, Eq. 1).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liborc.so")
_SRC = os.path.join(_HERE, "orc.c")
# -ffp-contract=off: no fused multiply-add, so every product and sum rounds
# once, in the order written.
CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fPIC", "-shared", "-Wall", "-Wextra"]

OK, EINVAL, ERANGE = 0, -1, -2
PREFILL, DECODE = 0, 1
MEM, COMP = 0, 1
REGIME_EMPTY = 255
P_MAX = 1 << 20
BATCH_MAX = 1 << 22

_lock = threading.Lock()
_default = None


def build(out: str = _SO, src: str = _SRC) -> str:
    """Compile an oracle C source with gcc into ``out``."""
    cmd = ["gcc", *CFLAGS, src, "-o", out]
    subprocess.run(cmd, check=True)
    return out


class _Shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "hidden", "n_q_heads", "n_kv_heads", "head_dim", "ffn",
        "vocab", "weight_bytes", "kv_bytes")]


SHAPE_FIELDS = [f[0] for f in _Shape._fields_]


def _shape_ptr(shape):
    """shape: None (unit shape), a mapping with the nine field names, or a
    sequence of nine ints in field order."""
    if shape is None:
        return None, None
    if isinstance(shape, dict):
        vals = [int(shape[f]) for f in SHAPE_FIELDS]
    else:
        vals = [int(v) for v in shape]
    s = _Shape(*vals)
    return s, ctypes.cast(ctypes.pointer(s), ctypes.c_void_p)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _arr(a, dtype):
    if a is None:
        return None
    return np.ascontiguousarray(a, dtype=dtype)


class OracleError(RuntimeError):
    def __init__(self, code, what):
        super().__init__(f"oracle {what} returned {code}")
        self.code = code


def _check(rc, what):
    if rc != OK:
        raise OracleError(rc, what)


ALL_OUTPUTS = ("T", "TM", "TC", "phase", "regime", "share", "share_alt", "tenant_sums")


class Oracle:
    """The oracle functions bound to one built copy of orc.c."""

    def __init__(self, so_path: str = _SO):
        lib = ctypes.CDLL(so_path)
        P = ctypes.c_void_p
        i64, i32 = ctypes.c_int64, ctypes.c_int32
        lib.orc_shape_constants.argtypes = [P, P]
        lib.orc_validate.argtypes = [i64, i64, P, P, P, P, i32]
        lib.orc_features.argtypes = [i64, i64, P, P, P, P, P, P]
        lib.orc_attribute.argtypes = [i64, i64, P, P, P, P, P, P, i32,
                                      P, P, P, P, P, P, P, P]
        lib.orc_tenant_sums.argtypes = [P, P, i64, i32, P]
        lib.orc_batch_sums.argtypes = [i64, i64, P, P, P, P, P]
        lib.orc_batch_sums_ext.argtypes = [i64, i64, P, P, P, P, P]
        lib.orc_admit.argtypes = [i64, P, P, i32, i32, P, P, P, P, P, P, P, P, P]
        lib.orc_admit_ext.argtypes = [i64, P, P, i32, i32, P, P, P, P, P, P, P, P, P]
        lib.orc_shape_constants_ext.argtypes = [P, P]
        lib.orc_attribute_ext.argtypes = [i64, i64, P, P, P, P, P, P, i32,
                                          P, P, P, P, P, P, P, P]
        for f in ("orc_shape_constants", "orc_validate", "orc_features",
                  "orc_attribute", "orc_tenant_sums", "orc_batch_sums", "orc_batch_sums_ext",
                  "orc_admit", "orc_admit_ext",
                  "orc_shape_constants_ext", "orc_attribute_ext"):
            getattr(lib, f).restype = ctypes.c_int
        self.lib = lib
        self.path = so_path

    def shape_constants(self, shape=None) -> np.ndarray:
        S = np.zeros(4, np.float64)
        keep, sp = _shape_ptr(shape)
        _check(self.lib.orc_shape_constants(sp, _ptr(S)), "shape_constants")
        del keep
        return S

    def validate(self, offsets, p, c, tenant=None, n_tenants=0) -> int:
        off = _arr(offsets, np.int64)
        p, c, t = _arr(p, np.int32), _arr(c, np.int32), _arr(tenant, np.int32)
        return int(self.lib.orc_validate(len(off) - 1, len(p), _ptr(off), _ptr(p),
                                         _ptr(c), _ptr(t), int(n_tenants)))

    def features(self, offsets, p, c, shape=None):
        """Returns (x_req [5, N], x_batch [5, nB]) in fp64."""
        off = _arr(offsets, np.int64)
        p, c = _arr(p, np.int32), _arr(c, np.int32)
        nB, N = len(off) - 1, len(p)
        xr = np.zeros((5, N), np.float64)
        xb = np.zeros((5, nB), np.float64)
        keep, sp = _shape_ptr(shape)
        _check(self.lib.orc_features(nB, N, _ptr(off), _ptr(p), _ptr(c), sp, _ptr(xr),
                                     _ptr(xb)), "features")
        del keep
        return xr, xb

    def shape_constants_ext(self, shape=None) -> np.ndarray:
        """(S0, S1, S2, S3, S5, S6) of the extended model."""
        S = np.zeros(6, np.float64)
        keep, sp = _shape_ptr(shape)
        _check(self.lib.orc_shape_constants_ext(sp, _ptr(S)), "shape_constants_ext")
        del keep
        return S

    def attribute(self, offsets, p, c, tenant, shape, coeffs, n_tenants,
                  outputs=ALL_OUTPUTS, ext=False) -> dict:
        """Runs the oracle; returns a dict with the requested outputs.  With
        ext=True, the extended model (28 coefficients)."""
        off = _arr(offsets, np.int64)
        p, c, t = _arr(p, np.int32), _arr(c, np.int32), _arr(tenant, np.int32)
        co = _arr(coeffs, np.float32)
        if co.shape != ((28,) if ext else (20,)):
            raise ValueError("coeffs must hold 28 (extended) or 20 fp32 values")
        nB, N = len(off) - 1, len(p)
        out = {}
        for name, n, dt in (("T", nB, np.float64), ("TM", nB, np.float64),
                            ("TC", nB, np.float64), ("phase", nB, np.uint8),
                            ("regime", nB, np.uint8), ("share", N, np.float64),
                            ("share_alt", N, np.float64)):
            if name in outputs:
                out[name] = np.zeros(n, dt)
        if "tenant_sums" in outputs and t is not None:
            out["tenant_sums"] = np.zeros(int(n_tenants), np.float64)
        keep, sp = _shape_ptr(shape)
        g = out.get
        fn = self.lib.orc_attribute_ext if ext else self.lib.orc_attribute
        rc = fn(
            nB, N, _ptr(off), _ptr(p), _ptr(c), _ptr(t), sp, _ptr(co), int(n_tenants),
            _ptr(g("T")), _ptr(g("TM")), _ptr(g("TC")), _ptr(g("phase")),
            _ptr(g("regime")), _ptr(g("share")), _ptr(g("share_alt")),
            _ptr(g("tenant_sums")))
        del keep
        _check(rc, "attribute")
        return out

    def batch_sums(self, offsets, p, c):
        """Returns (sums [4, nB] int64 = (|B|, sum p, sum c, sum p^2), phase [nB] uint8)."""
        off = _arr(offsets, np.int64)
        p, c = _arr(p, np.int32), _arr(c, np.int32)
        nB, N = len(off) - 1, len(p)
        sums = np.zeros((4, nB), np.int64)
        phase = np.zeros(nB, np.uint8)
        _check(self.lib.orc_batch_sums(nB, N, _ptr(off), _ptr(p), _ptr(c), _ptr(sums),
                                       _ptr(phase)), "batch_sums")
        return sums, phase

    def batch_sums_ext(self, offsets, p, c):
        """Returns (sums [5, nB] int64 = (|B|, sum p, sum c, sum p^2, sum p*c),
        phase [nB] uint8)."""
        off = _arr(offsets, np.int64)
        p, c = _arr(p, np.int32), _arr(c, np.int32)
        nB, N = len(off) - 1, len(p)
        sums = np.zeros((5, nB), np.int64)
        phase = np.zeros(nB, np.uint8)
        _check(self.lib.orc_batch_sums_ext(nB, N, _ptr(off), _ptr(p), _ptr(c), _ptr(sums),
                                           _ptr(phase)), "batch_sums_ext")
        return sums, phase

    def admit(self, p, c, cand_p, cand_c, shape, coeffs, ext=False) -> dict:
        """Admission query for the batch of requests (p, c) and one candidate
        request (cand_p, cand_c): T_after, delta, share, share_alt, TM_after,
        TC_after, regime.  With ext=True, the extended model (28 coefficients)."""
        p, c = _arr(p, np.int32), _arr(c, np.int32)
        co = _arr(coeffs, np.float32)
        if co.shape != ((28,) if ext else (20,)):
            raise ValueError("coeffs must hold 20 (28 with ext) fp32 values")
        vals = [ctypes.c_double() for _ in range(6)]
        reg = ctypes.c_uint8()
        keep, sp = _shape_ptr(shape)
        fn = self.lib.orc_admit_ext if ext else self.lib.orc_admit
        rc = fn(len(p), _ptr(p), _ptr(c), int(cand_p), int(cand_c), sp, _ptr(co),
                *[ctypes.addressof(v) for v in vals], ctypes.addressof(reg))
        del keep
        _check(rc, "admit")
        names = ("T_after", "delta", "share", "share_alt", "TM_after", "TC_after")
        out = {k: v.value for k, v in zip(names, vals)}
        out["regime"] = reg.value
        return out

    def tenant_sums(self, tenant, share, n_tenants) -> np.ndarray:
        t = _arr(tenant, np.int32)
        s = _arr(share, np.float64)
        out = np.zeros(int(n_tenants), np.float64)
        _check(self.lib.orc_tenant_sums(_ptr(t), _ptr(s), len(t), int(n_tenants),
                                        _ptr(out)), "tenant_sums")
        return out


def default() -> Oracle:
    """The oracle built from orc.c next to this file (built on first use)."""
    global _default
    with _lock:
        if _default is None:
            if not os.path.exists(_SO):
                build()
            _default = Oracle(_SO)
    return _default


def shape_constants(shape=None):
    return default().shape_constants(shape)


def validate(offsets, p, c, tenant=None, n_tenants=0):
    return default().validate(offsets, p, c, tenant, n_tenants)


def features(offsets, p, c, shape=None):
    return default().features(offsets, p, c, shape)


def attribute(offsets, p, c, tenant, shape, coeffs, n_tenants, outputs=ALL_OUTPUTS):
    return default().attribute(offsets, p, c, tenant, shape, coeffs, n_tenants, outputs)


def shape_constants_ext(shape=None):
    return default().shape_constants_ext(shape)


def attribute_ext(offsets, p, c, tenant, shape, coeffs, n_tenants, outputs=ALL_OUTPUTS):
    """The extended model: coeffs [28], index (phase*2 + segment)*7 + k."""
    return default().attribute(offsets, p, c, tenant, shape, coeffs, n_tenants, outputs, ext=True)


def tenant_sums(tenant, share, n_tenants):
    return default().tenant_sums(tenant, share, n_tenants)


def batch_sums(offsets, p, c):
    return default().batch_sums(offsets, p, c)


def batch_sums_ext(offsets, p, c):
    return default().batch_sums_ext(offsets, p, c)


def admit(p, c, cand_p, cand_c, shape, coeffs):
    return default().admit(p, c, cand_p, cand_c, shape, coeffs)


def admit_ext(p, c, cand_p, cand_c, shape, coeffs):
    """The admission query under the extended model: coeffs [28]."""
    return default().admit(p, c, cand_p, cand_c, shape, coeffs, ext=True)
