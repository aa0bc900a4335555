"""ctypes binding of libllmv (include/llmv.h).

Argument marshalling only: torch tensors are passed as device pointers, the
current torch stream as the hipStream_t, and every step of the computation
runs in the library's HIP kernels.  There is no CPU fallback: if the built
library is missing, loading fails with an error.
"""
from __future__ import annotations

import ctypes
import os
import threading

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libllmv.so")

LLMV_OK, LLMV_EINVAL, LLMV_ERANGE, LLMV_EDEVICE, LLMV_EWORKSPACE = 0, -1, -2, -3, -4
LLMV_PREFILL, LLMV_DECODE = 0, 1
LLMV_MEM, LLMV_COMP = 0, 1
LLMV_REGIME_EMPTY = 255
LLMV_P_MAX = 1 << 20
LLMV_BATCH_MAX = 1 << 22
LLMV_TENANTS_MAX = 1 << 24

EXPORTS = ("llmv_shape_constants", "llmv_workspace_size", "llmv_sweep_workspace_size",
           "llmv_sweep_workspace_size_ext", "llmv_attribute", "llmv_attribute_sweep",
           "llmv_attribute_sweep_ext", "llmv_features", "llmv_tenant_sums", "llmv_validate",
           "llmv_batch_sums", "llmv_batch_sums_ext", "llmv_admit", "llmv_admit_ext", "llmv_fit_workspace_size", "llmv_fit",
           "llmv_fit_metrics", "llmv_fit_ext", "llmv_fit_metrics_ext", "llmv_shape_constants_ext",
           "llmv_attribute_ext", "llmv_attribute_noalloc", "llmv_attribute_host",
           "llmv_last_error", "llmv_set_kernel_events")


class LlmvError(RuntimeError):
    def __init__(self, code: int, func: str, msg: str):
        super().__init__(f"{func} failed ({code}): {msg}")
        self.code = code


class llmv_shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "hidden", "n_q_heads", "n_kv_heads", "head_dim", "ffn", "vocab",
        "weight_bytes", "kv_bytes")]


class llmv_trace(ctypes.Structure):
    _fields_ = [("n_batches", ctypes.c_int64), ("n_requests", ctypes.c_int64),
                ("offsets", ctypes.c_void_p), ("p", ctypes.c_void_p), ("c", ctypes.c_void_p),
                ("tenant", ctypes.c_void_p)]


_lock = threading.Lock()
_lib = None


def load(path: str = LIB_PATH):
    """Loads libllmv; raises if it has not been built."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(path):
                raise RuntimeError(
                    f"{path} is missing: build the HIP library first (__graft_entry__.build())")
            lib = ctypes.CDLL(path)
            P, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
            lib.llmv_shape_constants.argtypes = [P, P]
            lib.llmv_workspace_size.argtypes = [i64, i64, i32]
            lib.llmv_workspace_size.restype = sz
            lib.llmv_sweep_workspace_size.argtypes = [i64, i64, i32]
            lib.llmv_sweep_workspace_size.restype = sz
            lib.llmv_sweep_workspace_size_ext.argtypes = [i64, i64, i32]
            lib.llmv_sweep_workspace_size_ext.restype = sz
            lib.llmv_attribute.argtypes = [P, P, P, P, P, P, i32, P, P, sz, P]
            lib.llmv_attribute_sweep.argtypes = [P, P, i32, P, i32, i32, P, P, sz, P]
            lib.llmv_attribute_sweep_ext.argtypes = [P, P, i32, P, i32, i32, P, P, sz, P]
            lib.llmv_features.argtypes = [P, P, P, P, P, sz, P]
            lib.llmv_tenant_sums.argtypes = [P, P, i64, i32, P, P, sz, P]
            lib.llmv_batch_sums.argtypes = [P, P, P, P, sz, P]
            lib.llmv_batch_sums_ext.argtypes = [P, P, P, P, sz, P]
            lib.llmv_admit.argtypes = [P, P, i64, P, P, P, P, P, i64, P, P, P, P, P]
            lib.llmv_admit_ext.argtypes = [P, P, i64, P, P, P, P, P, i64, P, P, P, P, P]
            lib.llmv_validate.argtypes = [P, i32, P, sz, P]
            lib.llmv_shape_constants_ext.argtypes = [P, P]
            lib.llmv_attribute_ext.argtypes = [P, P, P, P, P, P, i32, P, P, sz, P]
            lib.llmv_attribute_noalloc.argtypes = [P, P, P, P, P, P, i32, P, P]
            lib.llmv_attribute_host.argtypes = [P, P, P, P, P, P, i32, P]
            lib.llmv_fit_workspace_size.argtypes = [i64]
            lib.llmv_fit_workspace_size.restype = sz
            lib.llmv_fit.argtypes = [P, P, i64, P, P, P, i32, P, P, P, sz, P]
            lib.llmv_fit_metrics.argtypes = [P, P, i64, P, P, P, P, P, P, sz, P]
            lib.llmv_fit_ext.argtypes = [P, P, i64, P, P, P, i32, P, P, P, sz, P]
            lib.llmv_fit_metrics_ext.argtypes = [P, P, i64, P, P, P, P, P, P, sz, P]
            lib.llmv_last_error.argtypes = []
            lib.llmv_last_error.restype = ctypes.c_char_p
            lib.llmv_set_kernel_events.argtypes = [P, P]
            lib.llmv_set_kernel_events.restype = ctypes.c_int
            for f in ("llmv_shape_constants", "llmv_attribute", "llmv_attribute_sweep",
                      "llmv_attribute_sweep_ext",
                      "llmv_features", "llmv_tenant_sums", "llmv_validate", "llmv_batch_sums",
                      "llmv_batch_sums_ext", "llmv_admit", "llmv_admit_ext", "llmv_fit",
                      "llmv_fit_metrics",
                      "llmv_fit_ext", "llmv_fit_metrics_ext", "llmv_shape_constants_ext",
                      "llmv_attribute_ext", "llmv_attribute_noalloc", "llmv_attribute_host"):
                getattr(lib, f).restype = ctypes.c_int
            _lib = lib
    return _lib


def _check(rc: int, func: str):
    if rc != LLMV_OK:
        raise LlmvError(rc, func, load().llmv_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("expected a torch tensor")
    if t.numel() and not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return ctypes.c_void_p(t.data_ptr()) if t.numel() else None


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def make_shape(shape) -> llmv_shape | None:
    """shape: None, a dict with the nine field names, or llmv_shape."""
    if shape is None or isinstance(shape, llmv_shape):
        return shape
    return llmv_shape(*[int(shape[f[0]]) for f in llmv_shape._fields_])


def _shape_ref(sh):
    return None if sh is None else ctypes.byref(sh)


class DeviceTrace:
    """A trace resident in device memory (torch tensors on the current device)."""

    def __init__(self, offsets, p, c, tenant=None):
        self.offsets = offsets
        self.p = p
        self.c = c
        self.tenant = tenant
        self.n_batches = offsets.numel() - 1
        self.n_requests = p.numel()

    @classmethod
    def from_host(cls, offsets, p, c, tenant=None, device="cuda"):
        f = lambda a, dt: torch.as_tensor(a).to(device=device, dtype=dt).contiguous()
        return cls(f(offsets, torch.int64), f(p, torch.int32), f(c, torch.int32),
                   None if tenant is None else f(tenant, torch.int32))

    def struct(self, with_tenant=True) -> llmv_trace:
        return llmv_trace(self.n_batches, self.n_requests, _ptr(self.offsets), _ptr(self.p),
                          _ptr(self.c), _ptr(self.tenant) if with_tenant else None)


# ---------------------------------------------------------------- C ABI

def llmv_shape_constants(shape=None):
    S = (ctypes.c_double * 4)()
    sh = make_shape(shape)
    _check(load().llmv_shape_constants(_shape_ref(sh), S), "llmv_shape_constants")
    return [S[i] for i in range(4)]


def llmv_workspace_size(n_batches: int, n_requests: int, n_tenants: int) -> int:
    return int(load().llmv_workspace_size(n_batches, n_requests, n_tenants))


def llmv_sweep_workspace_size(n_batches: int, n_requests: int, n_tenants: int) -> int:
    return int(load().llmv_sweep_workspace_size(n_batches, n_requests, n_tenants))


def llmv_sweep_workspace_size_ext(n_batches: int, n_requests: int, n_tenants: int) -> int:
    return int(load().llmv_sweep_workspace_size_ext(n_batches, n_requests, n_tenants))


def llmv_attribute(trace: DeviceTrace, shape, coeffs, latency=None, regime=None, share=None,
                   n_tenants: int = 0, tenant_sums=None, ws=None, stream=None):
    co = (ctypes.c_float * 20)(*[float(v) for v in coeffs])
    sh = make_shape(shape)
    tr = trace.struct(with_tenant=tenant_sums is not None)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(load().llmv_attribute(ctypes.byref(tr), _shape_ref(sh), co, _ptr(latency),
                                 _ptr(regime), _ptr(share), int(n_tenants), _ptr(tenant_sums),
                                 _ptr(ws), nbytes, _stream(stream)), "llmv_attribute")


def llmv_attribute_noalloc(trace: DeviceTrace, shape, coeffs, latency=None, regime=None,
                           share=None, n_tenants: int = 0, tenant_sums=None, stream=None):
    """llmv_attribute without a workspace (the library's static scratch)."""
    co = (ctypes.c_float * 20)(*[float(v) for v in coeffs])
    sh = make_shape(shape)
    tr = trace.struct(with_tenant=tenant_sums is not None)
    _check(load().llmv_attribute_noalloc(ctypes.byref(tr), _shape_ref(sh), co, _ptr(latency),
                                         _ptr(regime), _ptr(share), int(n_tenants),
                                         _ptr(tenant_sums), _stream(stream)),
           "llmv_attribute_noalloc")


def llmv_attribute_host(offsets, p, c, tenant, shape, coeffs, n_tenants: int = 0,
                        outputs=("latency", "regime", "share", "tenant_sums")):
    """llmv_attribute_host on host (numpy) arrays: returns the requested
    outputs as numpy arrays.  The arrays are passed to the library as they
    are (contiguous, converted to int64 / int32 first)."""
    import numpy as np
    off = np.ascontiguousarray(offsets, dtype=np.int64)
    pp = np.ascontiguousarray(p, dtype=np.int32)
    cc = np.ascontiguousarray(c, dtype=np.int32)
    want_t = "tenant_sums" in outputs
    tt = np.ascontiguousarray(tenant, dtype=np.int32) if (want_t and tenant is not None) else None
    nB, N = len(off) - 1, len(pp)

    def hp(a):
        return None if a is None or a.size == 0 else ctypes.c_void_p(a.ctypes.data)

    tr = llmv_trace(nB, N, hp(off), hp(pp), hp(cc), hp(tt))
    out = {}
    if "latency" in outputs:
        out["latency"] = np.zeros(nB, np.float32)
    if "regime" in outputs:
        out["regime"] = np.zeros(nB, np.uint8)
    if "share" in outputs:
        out["share"] = np.zeros(N, np.float32)
    if want_t:
        out["tenant_sums"] = np.zeros(int(n_tenants), np.float64)
    co = (ctypes.c_float * 20)(*[float(v) for v in coeffs])
    sh = make_shape(shape)
    _check(load().llmv_attribute_host(ctypes.byref(tr), _shape_ref(sh), co,
                                      hp(out.get("latency")), hp(out.get("regime")),
                                      hp(out.get("share")), int(n_tenants),
                                      hp(out.get("tenant_sums"))), "llmv_attribute_host")
    return out


def llmv_attribute_sweep(trace: DeviceTrace, shapes, coeffs, n_tenants: int, out, ws=None,
                         stream=None, ext: bool = False):
    """shapes: list of shape dicts (or [None] for the unit shape); coeffs:
    array-like [n_coeffs, 20] ([n_coeffs, 28] with ext: llmv_attribute_sweep_ext);
    out: device fp64 [n_shapes, n_coeffs, n_tenants]."""
    import numpy as np
    co = np.ascontiguousarray(coeffs, dtype=np.float32).reshape(-1, 28 if ext else 20)
    if shapes == [None] or shapes is None:
        arr, n_sh = None, 1
    else:
        arr = (llmv_shape * len(shapes))(*[make_shape(s) for s in shapes])
        n_sh = len(shapes)
    tr = trace.struct(with_tenant=True)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    name = "llmv_attribute_sweep_ext" if ext else "llmv_attribute_sweep"
    _check(getattr(load(), name)(
        ctypes.byref(tr), None if arr is None else ctypes.cast(arr, ctypes.c_void_p), n_sh,
        co.ctypes.data_as(ctypes.c_void_p), co.shape[0], int(n_tenants), _ptr(out), _ptr(ws),
        nbytes, _stream(stream)), name)


def llmv_attribute_sweep_ext(trace: DeviceTrace, shapes, coeffs, n_tenants: int, out, ws=None,
                             stream=None):
    llmv_attribute_sweep(trace, shapes, coeffs, n_tenants, out, ws, stream, ext=True)


def llmv_batch_sums_ext(trace: DeviceTrace, sums=None, phase=None, ws=None, stream=None):
    """sums: device int64 [5, n_batches] (with sum p*c); phase: device uint8 [n_batches]."""
    tr = trace.struct(with_tenant=False)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(load().llmv_batch_sums_ext(ctypes.byref(tr), _ptr(sums), _ptr(phase), _ptr(ws), nbytes,
                                      _stream(stream)), "llmv_batch_sums_ext")


def llmv_batch_sums(trace: DeviceTrace, sums=None, phase=None, ws=None, stream=None):
    """sums: device int64 [4, n_batches]; phase: device uint8 [n_batches]."""
    tr = trace.struct(with_tenant=False)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(load().llmv_batch_sums(ctypes.byref(tr), _ptr(sums), _ptr(phase), _ptr(ws), nbytes,
                                  _stream(stream)), "llmv_batch_sums")


def llmv_admit(sums, phase, n_batches: int, shape, coeffs, cand_batch, cand_p, cand_c,
               t_after=None, delta=None, share=None, regime=None, stream=None, ext=False):
    """Device tensors: sums int64 [4, n_batches], phase uint8 [n_batches],
    cand_batch int64 [m], cand_p / cand_c int32 [m]; outputs fp32 / uint8 [m].
    With ext the extended model (llmv_admit_ext): sums [5, n_batches], 28
    coefficients."""
    k = 28 if ext else 20
    co = (ctypes.c_float * k)(*[float(v) for v in coeffs])
    sh = make_shape(shape)
    m = int(cand_p.numel())
    fn, name = (load().llmv_admit_ext, "llmv_admit_ext") if ext else (load().llmv_admit,
                                                                     "llmv_admit")
    _check(fn(_ptr(sums), _ptr(phase), int(n_batches), _shape_ref(sh), co, _ptr(cand_batch),
              _ptr(cand_p), _ptr(cand_c), m, _ptr(t_after), _ptr(delta), _ptr(share), _ptr(regime),
              _stream(stream)), name)


def llmv_admit_ext(sums, phase, n_batches: int, shape, coeffs, cand_batch, cand_p, cand_c,
                   t_after=None, delta=None, share=None, regime=None, stream=None):
    """llmv_admit for the extended model: sums [5, n_batches], 28 coefficients."""
    llmv_admit(sums, phase, n_batches, shape, coeffs, cand_batch, cand_p, cand_c, t_after, delta,
               share, regime, stream, ext=True)


def llmv_shape_constants_ext(shape=None):
    """(S0, S1, S2, S3, S5, S6) of the extended model (host only)."""
    S = (ctypes.c_double * 6)()
    sh = make_shape(shape)
    _check(load().llmv_shape_constants_ext(_shape_ref(sh), S), "llmv_shape_constants_ext")
    return list(S)


def llmv_attribute_ext(trace: DeviceTrace, shape, coeffs, latency=None, regime=None, share=None,
                       n_tenants: int = 0, tenant_sums=None, ws=None, stream=None):
    """llmv_attribute under the extended model: coeffs holds 28 numbers,
    index (phase*2 + segment)*7 + k, k = (beta, a1, ..., a6)."""
    vals = [float(v) for v in coeffs]
    if len(vals) != 28:
        raise ValueError("the extended model takes 28 coefficients")
    co = (ctypes.c_float * 28)(*vals)
    sh = make_shape(shape)
    if ws is None:
        ws = workspace(trace.n_batches, trace.n_requests, n_tenants, trace.p.device)
    tr = trace.struct(with_tenant=tenant_sums is not None)
    nbytes = ws.numel() * ws.element_size()
    _check(load().llmv_attribute_ext(ctypes.byref(tr), _shape_ref(sh), co, _ptr(latency),
                                     _ptr(regime), _ptr(share), int(n_tenants), _ptr(tenant_sums),
                                     _ptr(ws), nbytes, _stream(stream)),
           "llmv_attribute_ext")


def llmv_fit_workspace_size(n_batches: int) -> int:
    return int(load().llmv_fit_workspace_size(int(n_batches)))


def llmv_fit(sums, phase, shape, y, theta0, rounds: int, theta, counts=None, ws=None,
             stream=None, ext=False):
    """Device tensors: sums int64 [4, n_batches], phase uint8 [n_batches],
    y fp64 [n_batches]; outputs theta fp64 [20], counts int64 [4] (or None).
    theta0: 20 host numbers.  With ext the extended model (llmv_fit_ext):
    sums [5, n_batches], theta0 and theta 28 values."""
    n = int(phase.numel())
    k = 28 if ext else 20
    th0 = (ctypes.c_double * k)(*[float(v) for v in theta0])
    sh = make_shape(shape)
    if ws is None:
        ws = fit_workspace(n, theta.device)
    fn, name = (load().llmv_fit_ext, "llmv_fit_ext") if ext else (load().llmv_fit, "llmv_fit")
    _check(fn(_ptr(sums), _ptr(phase), n, _shape_ref(sh), _ptr(y), th0, int(rounds), _ptr(theta),
              _ptr(counts), _ptr(ws), ws.numel(), _stream(stream)), name)


def llmv_fit_metrics(sums, phase, shape, coeffs, y, out, rel_err=None, ws=None, stream=None,
                     ext=False):
    """Device tensors as for llmv_fit; out fp64 [3, 4] (prefill, decode, all)
    x (r2, p90, p99, batches); rel_err fp32 [n_batches] or None.  With ext the
    extended model (llmv_fit_metrics_ext, 28 coefficients)."""
    n = int(phase.numel())
    k = 28 if ext else 20
    co = (ctypes.c_float * k)(*[float(v) for v in coeffs])
    sh = make_shape(shape)
    if ws is None:
        ws = fit_workspace(n, out.device)
    fn, name = ((load().llmv_fit_metrics_ext, "llmv_fit_metrics_ext") if ext
                else (load().llmv_fit_metrics, "llmv_fit_metrics"))
    _check(fn(_ptr(sums), _ptr(phase), n, _shape_ref(sh), co, _ptr(y), _ptr(rel_err), _ptr(out),
              _ptr(ws), ws.numel(), _stream(stream)), name)


def llmv_fit_ext(sums, phase, shape, y, theta0, rounds: int, theta, counts=None, ws=None,
                 stream=None):
    """llmv_fit for the extended model: sums [5, n_batches], theta0/theta 28 values."""
    llmv_fit(sums, phase, shape, y, theta0, rounds, theta, counts, ws, stream, ext=True)


def llmv_fit_metrics_ext(sums, phase, shape, coeffs, y, out, rel_err=None, ws=None, stream=None):
    """llmv_fit_metrics for the extended model: sums [5, n_batches], 28 coefficients."""
    llmv_fit_metrics(sums, phase, shape, coeffs, y, out, rel_err, ws, stream, ext=True)


def llmv_features(trace: DeviceTrace, shape, x_req=None, x_batch=None, ws=None, stream=None):
    sh = make_shape(shape)
    tr = trace.struct(with_tenant=False)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(load().llmv_features(ctypes.byref(tr), _shape_ref(sh), _ptr(x_req), _ptr(x_batch),
                                _ptr(ws), nbytes, _stream(stream)), "llmv_features")


def llmv_tenant_sums(tenant, share, n_tenants: int, tenant_sums, ws=None, stream=None):
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(load().llmv_tenant_sums(_ptr(tenant), _ptr(share), int(share.numel()),
                                   int(n_tenants), _ptr(tenant_sums), _ptr(ws), nbytes,
                                   _stream(stream)), "llmv_tenant_sums")


def llmv_validate(trace: DeviceTrace, n_tenants: int = 0, ws=None, stream=None) -> int:
    """Returns LLMV_OK or LLMV_ERANGE; raises on argument / device errors."""
    tr = trace.struct(with_tenant=trace.tenant is not None)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    rc = load().llmv_validate(ctypes.byref(tr), int(n_tenants), _ptr(ws), nbytes,
                              _stream(stream))
    if rc not in (LLMV_OK, LLMV_ERANGE):
        _check(rc, "llmv_validate")
    return rc


def llmv_last_error() -> str:
    return load().llmv_last_error().decode()


def llmv_set_kernel_events(before=None, after=None):
    """before/after: hipEvent_t handles (ctypes.c_void_p or int), or None."""
    _check(load().llmv_set_kernel_events(before, after), "llmv_set_kernel_events")


# ---------------------------------------------------------------- helpers

def workspace(n_batches: int, n_requests: int, n_tenants: int, device="cuda"):
    """A device workspace tensor of llmv_workspace_size bytes (256-aligned)."""
    n = llmv_workspace_size(n_batches, n_requests, n_tenants)
    return torch.empty(max(n, 1), dtype=torch.uint8, device=device)


def sweep_workspace(n_batches: int, n_requests: int, n_tenants: int, device="cuda",
                    ext: bool = False):
    """A device workspace tensor of llmv_sweep_workspace_size(_ext) bytes."""
    size = llmv_sweep_workspace_size_ext if ext else llmv_sweep_workspace_size
    n = size(n_batches, n_requests, n_tenants)
    return torch.empty(max(n, 1), dtype=torch.uint8, device=device)


def attribute(trace: DeviceTrace, shape, coeffs, n_tenants: int = 0,
              outputs=("latency", "regime", "share", "tenant_sums"), ws=None):
    """Allocates the requested outputs and runs llmv_attribute."""
    dev = trace.p.device
    out = {}
    if "latency" in outputs:
        out["latency"] = torch.empty(trace.n_batches, dtype=torch.float32, device=dev)
    if "regime" in outputs:
        out["regime"] = torch.empty(trace.n_batches, dtype=torch.uint8, device=dev)
    if "share" in outputs:
        out["share"] = torch.empty(trace.n_requests, dtype=torch.float32, device=dev)
    if "tenant_sums" in outputs:
        out["tenant_sums"] = torch.empty(n_tenants, dtype=torch.float64, device=dev)
    if ws is None:
        ws = workspace(trace.n_batches, trace.n_requests, n_tenants, dev)
    llmv_attribute(trace, shape, coeffs, out.get("latency"), out.get("regime"), out.get("share"),
                   n_tenants, out.get("tenant_sums"), ws)
    return out


def attribute_sweep(trace: DeviceTrace, shapes, coeffs, n_tenants: int, ws=None,
                    ext: bool = False):
    """Allocates out [n_shapes, n_coeffs, n_tenants] and runs the sweep (under
    the extended model with ext, coeffs [n_coeffs, 28])."""
    import numpy as np
    n_sh = 1 if shapes is None else len(shapes)
    n_co = int(np.asarray(coeffs).reshape(-1, 28 if ext else 20).shape[0])
    out = torch.empty((n_sh, n_co, n_tenants), dtype=torch.float64, device=trace.p.device)
    if ws is None:
        ws = sweep_workspace(trace.n_batches, trace.n_requests, n_tenants, trace.p.device, ext)
    llmv_attribute_sweep(trace, shapes if shapes is not None else [None], coeffs, n_tenants,
                         out, ws, ext=ext)
    return out


def features(trace: DeviceTrace, shape, ws=None):
    dev = trace.p.device
    x_req = torch.empty((5, trace.n_requests), dtype=torch.float32, device=dev)
    x_batch = torch.empty((5, trace.n_batches), dtype=torch.float64, device=dev)
    if ws is None:
        ws = workspace(trace.n_batches, trace.n_requests, 0, dev)
    llmv_features(trace, shape, x_req, x_batch, ws)
    return x_req, x_batch


def tenant_sums(tenant, share, n_tenants: int, ws=None):
    out = torch.empty(n_tenants, dtype=torch.float64, device=share.device)
    if ws is None:
        ws = workspace(0, share.numel(), n_tenants, share.device)
    llmv_tenant_sums(tenant, share, n_tenants, out, ws)
    return out


def batch_sums(trace: DeviceTrace, ws=None, ext=False):
    """Allocates and returns (sums int64 [4, n_batches], phase uint8
    [n_batches]); with ext the sums have a fifth row, sum p*c."""
    dev = trace.p.device
    sums = torch.empty((5 if ext else 4, trace.n_batches), dtype=torch.int64, device=dev)
    phase = torch.empty(trace.n_batches, dtype=torch.uint8, device=dev)
    if ws is None:
        ws = workspace(trace.n_batches, trace.n_requests, 0, dev)
    (llmv_batch_sums_ext if ext else llmv_batch_sums)(trace, sums, phase, ws)
    return sums, phase


def admit(sums, phase, shape, coeffs, cand_batch, cand_p, cand_c, ext=False):
    """Allocates the outputs (t_after, delta, share fp32; regime uint8) and
    runs llmv_admit (llmv_admit_ext with ext); returns them in a dict."""
    m = int(cand_p.numel())
    dev = cand_p.device
    out = {"t_after": torch.empty(m, dtype=torch.float32, device=dev),
           "delta": torch.empty(m, dtype=torch.float32, device=dev),
           "share": torch.empty(m, dtype=torch.float32, device=dev),
           "regime": torch.empty(m, dtype=torch.uint8, device=dev)}
    llmv_admit(sums, phase, int(phase.numel()), shape, coeffs, cand_batch, cand_p, cand_c,
               out["t_after"], out["delta"], out["share"], out["regime"], ext=ext)
    return out


def fit_workspace(n_batches: int, device="cuda"):
    """A device workspace tensor of llmv_fit_workspace_size bytes."""
    return torch.empty(max(llmv_fit_workspace_size(n_batches), 1), dtype=torch.uint8,
                       device=device)


def fit(sums, phase, shape, y, theta0, rounds: int, ws=None, ext=False):
    """Allocates the outputs and runs llmv_fit (llmv_fit_ext with ext);
    returns (theta fp64 [20] or [28], counts int64 [4]) as device tensors."""
    dev = y.device
    theta = torch.empty(28 if ext else 20, dtype=torch.float64, device=dev)
    counts = torch.empty(4, dtype=torch.int64, device=dev)
    llmv_fit(sums, phase, shape, y, theta0, rounds, theta, counts, ws, ext=ext)
    return theta, counts


METRIC_GROUPS = ("prefill", "decode", "all")


def fit_metrics(sums, phase, shape, coeffs, y, ws=None, rel_err=False, ext=False):
    """Runs llmv_fit_metrics (llmv_fit_metrics_ext with ext); returns
    {"prefill"|"decode"|"all": {"r2", "p90", "p99", "n"}} (waits for the
    result), plus the per-batch relative errors under "rel_err" when asked
    for."""
    dev = y.device
    out = torch.empty((3, 4), dtype=torch.float64, device=dev)
    err = torch.empty(int(phase.numel()), dtype=torch.float32, device=dev) if rel_err else None
    llmv_fit_metrics(sums, phase, shape, coeffs, y, out, err, ws, ext=ext)
    o = out.cpu().tolist()
    res = {g: {"r2": o[i][0], "p90": o[i][1], "p99": o[i][2], "n": int(o[i][3])}
           for i, g in enumerate(METRIC_GROUPS)}
    if rel_err:
        res["rel_err"] = err
    return res


def attribute_ext(trace: DeviceTrace, shape, coeffs, n_tenants: int = 0,
                  outputs=("latency", "regime", "share", "tenant_sums"), ws=None):
    """Allocates the requested outputs and runs llmv_attribute_ext."""
    dev = trace.p.device
    out = {}
    if "latency" in outputs:
        out["latency"] = torch.empty(trace.n_batches, dtype=torch.float32, device=dev)
    if "regime" in outputs:
        out["regime"] = torch.empty(trace.n_batches, dtype=torch.uint8, device=dev)
    if "share" in outputs:
        out["share"] = torch.empty(trace.n_requests, dtype=torch.float32, device=dev)
    if "tenant_sums" in outputs:
        out["tenant_sums"] = torch.empty(n_tenants, dtype=torch.float64, device=dev)
    llmv_attribute_ext(trace, shape, coeffs, out.get("latency"), out.get("regime"),
                       out.get("share"), n_tenants, out.get("tenant_sums"), ws)
    return out
