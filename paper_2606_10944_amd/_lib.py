"""ctypes binding of libthin.so (see include/thin.h).

Argument marshalling only: every step of the path runs in the HIP library.
Tensors are PyTorch tensors on the GPU (PyTorch provides device memory and the
current HIP stream).  The library must have been built (``__graft_entry__.
build()`` or ``python paper_2606_10944_amd/build.py``); importing works without
it, but every call fails loudly if it is missing.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libthin.so")

THIN_OK, THIN_EINVAL, THIN_EDTYPE, THIN_EUNIFORMS, THIN_EWORKSPACE, THIN_EHIP = range(6)
THIN_FP32, THIN_BF16 = 0, 1
THIN_STATUS_WAIT_EXHAUSTED = 1

# Every symbol include/thin.h declares.
EXPORTS = ("thin_plan", "thin_compress", "thin_compress_static", "thin_compress_traced", "thin_compress_ex", "thin_attention",
           "thin_attention_ex", "thin_express_plan", "thin_express_create", "thin_express_step",
           "thin_express_cache", "thin_express_next", "thin_express_destroy",
           "thin_express_prefill_plan", "thin_express_prefill",
           "thin_selftest_gram16", "thin_status_str", "thin_workspace_status",
           "thin_set_launch_hook")

# thin_kernel_t
KERNEL_NAMES = {0: "trace_clear", 1: "subsample", 2: "fill", 3: "vmax", 4: "scores",
                5: "decide", 6: "attention", 7: "local", 8: "uniform", 9: "assemble",
                10: "express", 11: "status"}
HALVE = {"kh": 0, "uniform": 1}  # thin_halve_t
LaunchHook = C.CFUNCTYPE(None, C.c_void_p, C.c_int32, C.c_int32, C.c_int32, C.c_void_p)


class ThinError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {thin_status_str(status)} (status {status})")


class ExpressPlan(C.Structure):
    _fields_ = [("uniforms_per_slice", C.c_int64), ("max_keys", C.c_int64),
                ("workspace_bytes", C.c_size_t), ("subsample_draws", C.c_int64)]


class PrefillPlan(C.Structure):
    _fields_ = [("uniforms_per_slice", C.c_int64), ("subsample_draws", C.c_int64),
                ("workspace_bytes", C.c_size_t), ("attention_keys", C.c_int64),
                ("staged_keys", C.c_int64), ("host_staging_bytes", C.c_size_t)]


class CompressOpts(C.Structure):
    _fields_ = [("halve", C.c_int32), ("delta", C.c_void_p), ("n_sinks", C.c_int64),
                ("n_window", C.c_int64), ("logw_out", C.c_void_p)]


class Plan(C.Structure):
    _fields_ = [
        ("n_kept", C.c_int64),
        ("rounds", C.c_int32),
        ("compress_levels", C.c_int32),
        ("uniforms_per_slice", C.c_int64),
        ("uniforms_total", C.c_int64),
        ("max_bucket", C.c_int64),
        ("workspace_bytes", C.c_size_t),
    ]


_lib = None


def lib():
    """Load libthin.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    L = C.CDLL(LIB_PATH)
    P, I64, I32, SZ = C.c_void_p, C.c_int64, C.c_int32, C.c_size_t
    L.thin_plan.argtypes = [I64, I64, I64, I64, I64, I32, C.POINTER(Plan)]
    L.thin_compress.argtypes = [P, P, I32, I64, I64, I64, I64, I64, I32, P, I64, P, P, SZ, P]
    L.thin_compress_static.argtypes = [P, P, I32, I64, I64, I64, I64, I64, I32, P, I64, P, P, P]
    L.thin_compress_traced.argtypes = [P, P, I32, I64, I64, I64, I64, I64, I32, P, I64, P, P,
                                       SZ, P, I64, P]
    L.thin_compress_ex.argtypes = [P, P, I32, I64, I64, I64, I64, I64, I32, P, I64, P, P, SZ,
                                   C.POINTER(CompressOpts), P, I64, P]
    L.thin_attention.argtypes = [P, P, P, I32, I64, I64, I64, I64, I64, P, I64, P, I32, P]
    L.thin_attention_ex.argtypes = [P, P, P, I32, I64, I64, I64, I64, I64, P, P, I64, P, I32, P]
    L.thin_express_plan.argtypes = [I64, I64, I64, I64, I32, I64, C.POINTER(ExpressPlan)]
    L.thin_express_create.argtypes = [I32, I64, I64, I64, I64, I32, C.c_double, I32, I64, P, SZ,
                                      C.POINTER(C.c_void_p)]
    L.thin_express_step.argtypes = [P, P, P, P, P, I64, P, I64, P, I32, P, P]
    L.thin_express_cache.argtypes = [P, P, P, C.POINTER(C.c_int64), C.POINTER(C.c_int32), P]
    L.thin_express_next.argtypes = [P, C.POINTER(C.c_int64), C.POINTER(C.c_int64)]
    L.thin_express_destroy.argtypes = [P]
    L.thin_express_prefill_plan.argtypes = [I64, I64, I64, I64, I64, I32, C.POINTER(PrefillPlan)]
    L.thin_express_prefill.argtypes = [I32, I64, I64, I64, I64, I64, I32, C.c_double, I32, P, P,
                                       P, P, I64, P, I64, P, I32, P, SZ, P, SZ, P, P]
    L.thin_workspace_status.argtypes = [P, P, P]
    L.thin_selftest_gram16.argtypes = [I32, I64, P, P, P]
    L.thin_status_str.argtypes = [C.c_int]
    L.thin_status_str.restype = C.c_char_p
    L.thin_set_launch_hook.argtypes = [LaunchHook, P]
    L.thin_set_launch_hook.restype = C.c_int
    for f in ("thin_plan", "thin_compress", "thin_compress_static", "thin_compress_traced",
              "thin_compress_ex",
              "thin_attention", "thin_attention_ex", "thin_selftest_gram16", "thin_express_plan",
              "thin_express_create", "thin_express_step", "thin_express_cache",
              "thin_express_next", "thin_express_destroy", "thin_express_prefill_plan",
              "thin_express_prefill", "thin_workspace_status"):
        getattr(L, f).restype = C.c_int
    _lib = L
    return L


def thin_status_str(status: int) -> str:
    return lib().thin_status_str(int(status)).decode()


def _dtype_code(t: torch.dtype) -> int:
    if t == torch.float32:
        return THIN_FP32
    if t == torch.bfloat16:
        return THIN_BF16
    raise ThinError(THIN_EDTYPE, f"dtype {t}")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream) -> C.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def _check(rc: int, where: str):
    if rc != THIN_OK:
        raise ThinError(rc, where)


def workspace_status(workspace: torch.Tensor, stream=None) -> int:
    """The device status word of a workspace once the work enqueued on
    `stream` so far has run (this synchronises that stream): 0, or
    THIN_STATUS_WAIT_EXHAUSTED if a decision pass's bounded wait gave up."""
    out = torch.zeros(1, dtype=torch.int32, pin_memory=True)
    _check(lib().thin_workspace_status(_ptr(workspace), _ptr(out), _stream(stream)),
           "thin_workspace_status")
    (stream if stream is not None else torch.cuda.current_stream()).synchronize()
    return int(out[0])


# Pinned host buffers handed to asynchronous calls, each kept until an event
# recorded after its call has completed.
_pending = []


def _keep_until_done(buf: torch.Tensor, stream) -> None:
    global _pending
    _pending = [(e, b) for e, b in _pending if not e.query()]
    ev = torch.cuda.Event()
    ev.record(stream if stream is not None else torch.cuda.current_stream())
    _pending.append((ev, buf))


def thin_plan(B: int, H: int, n: int, d: int, n_out: int, g: int) -> dict:
    p = Plan()
    _check(lib().thin_plan(B, H, n, d, n_out, g, C.byref(p)), "thin_plan")
    return {k: getattr(p, k) for k, _ in Plan._fields_}


def _shape4(t: torch.Tensor, name: str) -> Tuple[int, int, int, int]:
    if t.dim() != 4 or not t.is_contiguous():
        raise ThinError(THIN_EINVAL, f"{name} must be a contiguous [B,H,rows,d] tensor")
    return tuple(t.shape)


def thin_compress(K: torch.Tensor, V: torch.Tensor, n_out: int, g: int,
                  uniforms: torch.Tensor, *, idx_out: Optional[torch.Tensor] = None,
                  workspace: Optional[torch.Tensor] = None, trace: bool = False,
                  halve: str = "kh", delta=None, n_sinks: int = 0, n_window: int = 0,
                  return_logw: bool = False, logw_out: Optional[torch.Tensor] = None,
                  stream=None):
    """Compress of every slice; returns idx [B,H,n_out] int32, then the uint8
    swap trace when trace=True, then the float32 log-weights [B,H,m] when
    return_logw=True (a tuple when either is asked for).  halve="kh" (kernel
    halving, KH's delta per round in `delta`, default 1/2) or "uniform".  With
    n_sinks / n_window the first / last rows of every slice are kept exactly
    and the rows between them thinned to n_out: idx is then [B,H,m] with
    m = n_sinks + n_out + n_window, and the uniforms and workspace are those of
    thin_plan for n - n_sinks - n_window rows.  logw_out (float32 [B,H,m]) is
    filled with the log-weights and returned as with return_logw=True.
    Anything but the defaults goes through thin_compress_ex."""
    B, H, n, d = _shape4(K, "K")
    if tuple(V.shape) != (B, H, n, d) or V.dtype != K.dtype or not V.is_contiguous():
        raise ThinError(THIN_EINVAL, "V must match K")
    if uniforms.dtype != torch.float32 or not uniforms.is_contiguous():
        raise ThinError(THIN_EINVAL, "uniforms must be contiguous float32")
    if n_sinks < 0 or n_window < 0 or n_sinks + n_window >= n:
        raise ThinError(THIN_EINVAL, "n_sinks and n_window must leave rows to thin")
    plan = thin_plan(B, H, n - n_sinks - n_window, d, n_out, g)
    dev = K.device
    m = n_sinks + n_out + n_window
    if idx_out is None:
        idx_out = torch.empty((B, H, m), dtype=torch.int32, device=dev)
    elif tuple(idx_out.shape) != (B, H, m) or idx_out.dtype != torch.int32 \
            or not idx_out.is_contiguous():
        raise ThinError(THIN_EINVAL, "idx_out must be contiguous int32 [B,H,m]")
    lw = None
    if logw_out is not None:
        if tuple(logw_out.shape) != (B, H, m) or logw_out.dtype != torch.float32 \
                or not logw_out.is_contiguous():
            raise ThinError(THIN_EINVAL, "logw_out must be contiguous float32 [B,H,m]")
        lw, return_logw = logw_out, True
    elif return_logw:
        lw = torch.empty((B, H, m), dtype=torch.float32, device=dev)
    if workspace is None:
        workspace = torch.empty(max(plan["workspace_bytes"], 256), dtype=torch.uint8, device=dev)
    tr = None
    args = [_ptr(K), _ptr(V), _dtype_code(K.dtype), B, H, n, d, n_out, g, _ptr(uniforms),
            uniforms.numel(), _ptr(idx_out), _ptr(workspace), workspace.numel()]
    if halve != "kh" or delta is not None or n_sinks or n_window or return_logw:
        if halve not in HALVE:
            raise ThinError(THIN_EINVAL, f"unknown halving {halve!r}")
        dl = None
        if delta is not None:
            dl = (C.c_double * max(len(delta), 1))(*[float(x) for x in delta])
            if len(delta) < plan["rounds"]:
                raise ThinError(THIN_EINVAL, "delta needs one value per round")
        opts = CompressOpts(HALVE[halve], C.cast(dl, C.c_void_p) if dl is not None else None,
                            n_sinks, n_window, _ptr(lw) if return_logw else None)
        if trace:
            tr = torch.empty(max(plan["uniforms_total"], 1), dtype=torch.uint8, device=dev)
        rc = lib().thin_compress_ex(*args, C.byref(opts), _ptr(tr) if trace else None,
                                    tr.numel() if trace else 0, _stream(stream))
        _check(rc, "thin_compress_ex")
        out = [idx_out] + ([tr[: plan["uniforms_total"]]] if trace else []) \
            + ([lw] if return_logw else [])
        return out[0] if len(out) == 1 else tuple(out)
    if trace:
        tr = torch.empty(max(plan["uniforms_total"], 1), dtype=torch.uint8, device=dev)
        rc = lib().thin_compress_traced(*args, _ptr(tr), tr.numel(), _stream(stream))
        _check(rc, "thin_compress_traced")
        return idx_out, tr[: plan["uniforms_total"]]
    _check(lib().thin_compress(*args, _stream(stream)), "thin_compress")
    return idx_out


def thin_attention(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, idx: torch.Tensor, *,
                   logw: Optional[torch.Tensor] = None, out_dtype: torch.dtype = torch.float32,
                   O: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Attention of every query over its slice's coreset rows idx[b,h,:]; with
    logw (float32 [B,H,n_out]) key j weighs exp(logw[b,h,j]) (thin_attention_ex)."""
    B, H, n_q, d = _shape4(Q, "Q")
    Bk, Hk, n, dk = _shape4(K, "K")
    if (Bk, Hk, dk) != (B, H, d) or tuple(V.shape) != tuple(K.shape):
        raise ThinError(THIN_EINVAL, "Q/K/V shapes disagree")
    if K.dtype != Q.dtype or V.dtype != Q.dtype:
        raise ThinError(THIN_EDTYPE, "Q, K, V must share a dtype")
    if idx.dtype != torch.int32 or idx.dim() != 3 or tuple(idx.shape[:2]) != (B, H):
        raise ThinError(THIN_EINVAL, "idx must be int32 [B,H,n_out]")
    idx = idx.contiguous()
    n_out = idx.shape[2]
    if O is None:
        O = torch.empty((B, H, n_q, d), dtype=out_dtype, device=Q.device)
    if logw is not None:
        if logw.dtype != torch.float32 or tuple(logw.shape) != (B, H, n_out):
            raise ThinError(THIN_EINVAL, "logw must be float32 [B,H,n_out]")
        logw = logw.contiguous()
        rc = lib().thin_attention_ex(_ptr(Q), _ptr(K), _ptr(V), _dtype_code(Q.dtype), B, H, n_q,
                                     n, d, _ptr(idx), _ptr(logw), n_out, _ptr(O),
                                     _dtype_code(O.dtype), _stream(stream))
        _check(rc, "thin_attention_ex")
        return O
    rc = lib().thin_attention(_ptr(Q), _ptr(K), _ptr(V), _dtype_code(Q.dtype), B, H, n_q, n, d,
                              _ptr(idx), n_out, _ptr(O), _dtype_code(O.dtype), _stream(stream))
    _check(rc, "thin_attention")
    return O


def thin_express_plan(B: int, H: int, d: int, n_out: int, mbar: int, n_max: int) -> dict:
    p = ExpressPlan()
    _check(lib().thin_express_plan(B, H, d, n_out, mbar, n_max, C.byref(p)), "thin_express_plan")
    return {k: getattr(p, k) for k, _ in ExpressPlan._fields_}


class ExpressCache:
    """Thinformer decoding over an Express cache for B*H slices in lockstep
    (thin_express_*): ``step(Q_t, K, V, U)`` attends point t = ``self.n``
    (query Q_t [B,H,d]; K, V [B,H,n_max,d] caches holding rows 0..t) over the
    cache plus itself and then adds it to the cache.  ``draws`` (host float32
    array of plan["subsample_draws"] values, one per Subsample stratum, shared
    by all slices) is needed once a level above mbar is reached."""

    def __init__(self, B: int, H: int, d: int, n_out: int, mbar: int, n_max: int, *,
                 dtype: torch.dtype = torch.bfloat16, delta: float = 0.5, halve: str = "kh",
                 device="cuda"):
        if halve not in HALVE:
            raise ThinError(THIN_EINVAL, f"unknown halving {halve!r}")
        self.plan = thin_express_plan(B, H, d, n_out, mbar, n_max)
        self.B, self.H, self.d, self.n_out, self.n_max = B, H, d, n_out, n_max
        self.dtype = dtype
        self.ws = torch.empty(max(self.plan["workspace_bytes"], 256), dtype=torch.uint8,
                              device=device)
        h = C.c_void_p()
        _check(lib().thin_express_create(_dtype_code(dtype), B, H, d, n_out, mbar, delta,
                                         HALVE[halve], n_max, _ptr(self.ws), self.ws.numel(),
                                         C.byref(h)), "thin_express_create")
        self._h = h
        self.n = 0

    def step(self, Q_t: torch.Tensor, K: torch.Tensor, V: torch.Tensor, uniforms, *,
             draws=None, O: Optional[torch.Tensor] = None,
             out_dtype: torch.dtype = torch.float32, trace: Optional[torch.Tensor] = None,
             stream=None) -> torch.Tensor:
        B, H, d = self.B, self.H, self.d
        if tuple(Q_t.shape) != (B, H, d) or not Q_t.is_contiguous() or Q_t.dtype != self.dtype:
            raise ThinError(THIN_EINVAL, "Q_t must be contiguous [B,H,d] of the cache's dtype")
        for t, nm in ((K, "K"), (V, "V")):
            if tuple(t.shape) != (B, H, self.n_max, d) or not t.is_contiguous() \
                    or t.dtype != self.dtype:
                raise ThinError(THIN_EINVAL, f"{nm} must be contiguous [B,H,n_max,d]")
        if uniforms is not None and (uniforms.dtype != torch.float32
                                     or not uniforms.is_contiguous()):
            raise ThinError(THIN_EINVAL, "uniforms must be contiguous float32")
        if O is None:
            O = torch.empty((B, H, d), dtype=out_dtype, device=Q_t.device)
        elif tuple(O.shape) != (B, H, d) or not O.is_contiguous():
            raise ThinError(THIN_EINVAL, "O must be contiguous [B,H,d]")
        nU = 0 if uniforms is None else uniforms.numel()
        if draws is not None and (not isinstance(draws, torch.Tensor) or draws.is_cuda
                                  or draws.dtype != torch.float32 or not draws.is_contiguous()):
            raise ThinError(THIN_EINVAL, "draws must be a contiguous float32 CPU tensor")
        nD = 0 if draws is None else draws.numel()
        rc = lib().thin_express_step(self._h, _ptr(Q_t), _ptr(K), _ptr(V),
                                     None if uniforms is None else _ptr(uniforms), nU,
                                     None if draws is None else _ptr(draws), nD, _ptr(O),
                                     _dtype_code(O.dtype), None if trace is None else _ptr(trace),
                                     _stream(stream))
        _check(rc, "thin_express_step")
        self.n += 1
        return O

    def status(self, stream=None) -> int:
        """The object's device status word (see workspace_status)."""
        return workspace_status(self.ws, stream)

    def next_keys(self) -> int:
        """Keys the next step attends over (host-only)."""
        k, t = C.c_int64(0), C.c_int64(0)
        _check(lib().thin_express_next(self._h, C.byref(k), C.byref(t)), "thin_express_next")
        return k.value

    def cache(self, stream=None):
        """(idx [B,H,len] int32, logw [B,H,len] float32, m): the current
        weighted cache in the order C_0, C_1, .., C_mp, E."""
        k = self.plan["max_keys"]
        idx = torch.empty((self.B, self.H, k), dtype=torch.int32, device=self.ws.device)
        lw = torch.empty((self.B, self.H, k), dtype=torch.float32, device=self.ws.device)
        ln = C.c_int64(0)
        m = C.c_int32(0)
        _check(lib().thin_express_cache(self._h, _ptr(idx), _ptr(lw), C.byref(ln), C.byref(m),
                                        _stream(stream)), "thin_express_cache")
        return idx[..., :ln.value], lw[..., :ln.value], m.value

    def close(self):
        if self._h:
            lib().thin_express_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def thin_express_prefill_plan(B: int, H: int, n: int, d: int, n_out: int, mbar: int) -> dict:
    p = PrefillPlan()
    _check(lib().thin_express_prefill_plan(B, H, n, d, n_out, mbar, C.byref(p)),
           "thin_express_prefill_plan")
    return {k: getattr(p, k) for k, _ in PrefillPlan._fields_}


def thin_express_prefill(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, n_out: int,
                         mbar: int, uniforms, *, draws=None, delta: float = 0.5,
                         halve: str = "kh", out_dtype: torch.dtype = torch.float32,
                         O: Optional[torch.Tensor] = None, workspace=None,
                         trace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Masked prefill (thin_express_prefill): every point's Thinformer output
    over the Express cache of the points before it plus itself, O [B,H,n,d]."""
    B, H, n, d = _shape4(Q, "Q")
    for t, nm in ((K, "K"), (V, "V")):
        if tuple(t.shape) != (B, H, n, d) or not t.is_contiguous() or t.dtype != Q.dtype:
            raise ThinError(THIN_EINVAL, f"{nm} must match Q")
    if halve not in HALVE:
        raise ThinError(THIN_EINVAL, f"unknown halving {halve!r}")
    plan = thin_express_prefill_plan(B, H, n, d, n_out, mbar)
    if workspace is None:
        workspace = torch.empty(max(plan["workspace_bytes"], 256), dtype=torch.uint8,
                                device=Q.device)
    if O is None:
        O = torch.empty((B, H, n, d), dtype=out_dtype, device=Q.device)
    if draws is not None and (not isinstance(draws, torch.Tensor) or draws.is_cuda
                              or draws.dtype != torch.float32 or not draws.is_contiguous()):
        raise ThinError(THIN_EINVAL, "draws must be a contiguous float32 CPU tensor")
    nU = 0 if uniforms is None else uniforms.numel()
    staging = torch.empty(max(plan["host_staging_bytes"], 1), dtype=torch.uint8, pin_memory=True)
    rc = lib().thin_express_prefill(
        _dtype_code(Q.dtype), B, H, n, d, n_out, mbar, delta, HALVE[halve], _ptr(Q), _ptr(K),
        _ptr(V), None if uniforms is None else _ptr(uniforms), nU,
        None if draws is None else _ptr(draws), 0 if draws is None else draws.numel(), _ptr(O),
        _dtype_code(O.dtype), _ptr(workspace), workspace.numel(), _ptr(staging),
        staging.numel(), None if trace is None else _ptr(trace), _stream(stream))
    _check(rc, "thin_express_prefill")
    _keep_until_done(staging, stream)
    return O


def thin_selftest_gram16(rows: torch.Tensor, stream=None) -> torch.Tensor:
    """<rows[m], rows[16+n]> for m, n < 16 through the MFMA fragment path."""
    if rows.dim() != 2 or rows.shape[0] != 32 or not rows.is_contiguous():
        raise ThinError(THIN_EINVAL, "rows must be a contiguous [32, d] tensor")
    out = torch.empty((16, 16), dtype=torch.float32, device=rows.device)
    rc = lib().thin_selftest_gram16(_dtype_code(rows.dtype), rows.shape[1], _ptr(rows),
                                    _ptr(out), _stream(stream))
    _check(rc, "thin_selftest_gram16")
    return out


class LaunchTimer:
    """Times every kernel launch of the library on one stream with HIP events
    (thin_set_launch_hook): inside ``with LaunchTimer(stream) as lt:`` each
    launch is bracketed by two events recorded on ``stream``; after
    synchronising, ``lt.records()`` lists (kernel name, round, milliseconds)
    in launch order.  Events come from a pool created up front, so the hook
    only records."""

    def __init__(self, stream, capacity: int = 4096):
        self.stream = stream
        self._raw = stream.cuda_stream
        self._events = [torch.cuda.Event(enable_timing=True) for _ in range(2 * capacity)]
        self._n = 0
        self._meta = []
        self._cb = LaunchHook(self._hook)

    def _hook(self, ctx, kernel, rnd, phase, stream_ptr):
        if (stream_ptr or 0) != self._raw:
            raise RuntimeError("LaunchTimer: launch on another stream")
        if self._n >= len(self._events):
            raise RuntimeError("LaunchTimer: event pool exhausted")
        self._events[self._n].record(self.stream)
        self._n += 1
        if phase == 1:
            self._meta.append((kernel, rnd))

    def __enter__(self):
        _check(lib().thin_set_launch_hook(self._cb, None), "thin_set_launch_hook")
        return self

    def __exit__(self, *exc):
        lib().thin_set_launch_hook(LaunchHook(), None)
        return False

    def records(self):
        ev = self._events
        return [(KERNEL_NAMES.get(k, str(k)), r, ev[2 * i].elapsed_time(ev[2 * i + 1]))
                for i, (k, r) in enumerate(self._meta)]
