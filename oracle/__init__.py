"""CPU oracle for the thinning hot path -- TEST INFRASTRUCTURE ONLY.

A plain, single-threaded float64 C implementation (``oracle.c``) of kernel
halving under kappa_att, the Compress level structure, stratified subsampling
and softmax attention, written from the paper ("Express Language Modeling").
This wrapper only marshals numpy arrays.  Only ``tests/``, the smoke check and
the benchmark's CPU-baseline leg may import it; the HIP library never does.

Pinned by ``tests/test_oracle_pins.py`` (closed forms, invariants, special
cases, an explicit feature-space route and brute force on tiny inputs).
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liboracle.so")
_lib = None

KERNELS = {"katt": 0, "linear": 1}


class Stats(C.Structure):
    _fields_ = [
        ("decisions", C.c_int64),
        ("swaps", C.c_int64),
        ("near_ties", C.c_int64),
        ("hard_mismatch", C.c_int64),
        ("zero_threshold", C.c_int64),
        ("min_abs_rho", C.c_double),
    ]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class Plan(C.Structure):
    _fields_ = [
        ("n_kept", C.c_int64),
        ("rounds", C.c_int32),
        ("compress_levels", C.c_int32),
        ("uniforms", C.c_int64),
        ("subsample", C.c_int32),
    ]


def build() -> str:
    """Compile liboracle.so with gcc (no fast-math: IEEE float64 throughout)."""
    src = os.path.join(_HERE, "oracle.c")
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-o", _SO, src, "-lm"]
    subprocess.run(cmd, check=True)
    return _SO


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(
                os.path.join(_HERE, "oracle.c")):
            build()
        L = C.CDLL(_SO)
        P = C.c_void_p
        L.or_plan.argtypes = [C.c_int64, C.c_int64, C.c_int32, C.POINTER(Plan)]
        L.or_plan.restype = C.c_int
        L.or_vmax2.argtypes = [P, C.c_int64, C.c_int64]
        L.or_vmax2.restype = C.c_double
        L.or_subsample.argtypes = [C.c_int64, C.c_int64, P, P]
        L.or_subsample.restype = None
        L.or_kernel_halving.argtypes = [P, P, C.c_int64, C.c_double, C.c_int, C.c_double, P,
                                        C.c_int64, P, P, P, C.c_double, P, P, P, P,
                                        C.POINTER(Stats)]
        L.or_kernel_halving.restype = C.c_int
        L.or_compress.argtypes = [P, P, C.c_int64, C.c_int64, C.c_int64, C.c_int32, C.c_int, P,
                                  P, P, C.c_double, P, P, C.POINTER(Stats)]
        L.or_compress.restype = C.c_int
        L.or_compress_ex.argtypes = [P, P, C.c_int64, C.c_int64, C.c_int64, C.c_int32, C.c_int,
                                     C.c_int, P, P, P, P, C.c_double, P, P, C.POINTER(Stats)]
        L.or_attention_weighted.argtypes = [P, P, P, C.c_int64, C.c_int64, P, P, C.c_int64, P]
        L.or_attention_weighted.restype = None
        L.or_express_decode.argtypes = [P, P, P, C.c_int64, C.c_int64, C.c_int64, C.c_int,
                                        C.c_double, C.c_int, P, P, P, C.c_double, P, P, P, P, P,
                                        P, C.POINTER(Stats)]
        L.or_express_decode.restype = C.c_int
        L.or_express_uniforms.argtypes = [C.c_int64, C.c_int64, C.c_int, C.POINTER(C.c_int64)]
        L.or_express_uniforms.restype = C.c_int64
        L.or_express_keys.argtypes = [C.c_int64, C.c_int64, C.c_int, P, P]
        L.or_express_keys.restype = C.c_int
        L.or_express_delta.argtypes = [C.c_int, C.c_int, C.c_int, C.c_double]
        L.or_express_delta.restype = C.c_double
        L.or_compress_ex.restype = C.c_int
        L.or_uniform_halving.argtypes = [P, C.c_int64, P, P, P, C.POINTER(Stats)]
        L.or_uniform_halving.restype = C.c_int
        L.or_attention.argtypes = [P, P, P, C.c_int64, C.c_int64, P, C.c_int64, P]
        L.or_attention.restype = None
        _lib = L
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _f64(a) -> np.ndarray:
    if hasattr(a, "detach"):  # torch tensor: exact upcast
        import torch
        a = a.detach().to("cpu", torch.float64).numpy()
    return np.ascontiguousarray(a, dtype=np.float64)


def _f32(a) -> np.ndarray:
    if hasattr(a, "detach"):
        a = a.detach().cpu().numpy()
    return np.ascontiguousarray(a, dtype=np.float32)


def plan(n: int, n_out: int, g: int) -> Optional[dict]:
    p = Plan()
    if lib().or_plan(n, n_out, g, C.byref(p)) != 0:
        return None
    return {k: getattr(p, k) for k, _ in Plan._fields_}


def vmax2(V) -> float:
    V = _f64(V)
    return lib().or_vmax2(_p(V), V.shape[0], V.shape[1])


def subsample(n: int, n_kept: int, u) -> np.ndarray:
    u = _f32(u)
    assert u.size >= n_kept
    out = np.empty(n_kept, dtype=np.int32)
    lib().or_subsample(n, n_kept, _p(u), _p(out))
    return out


def kernel_halving(K, V, rows, u, *, vmax2_value: Optional[float] = None,
                   kernel: str = "katt", delta: float = 0.5, follow=None,
                   tol: float = 1e-5) -> dict:
    """KH(delta) on one bucket `rows` (indices into K/V rows)."""
    K, V = _f64(K), _f64(V)
    rows = np.ascontiguousarray(rows, dtype=np.int32)
    u = _f32(u)
    N = rows.size
    h = N // 2
    assert u.size >= h
    vm = vmax2(V) if vmax2_value is None else float(vmax2_value)
    out = np.empty(h, dtype=np.int32)
    bits = np.empty(h, dtype=np.uint8)
    rho = np.empty(h)
    alpha = np.empty(h)
    thresh = np.empty(h)
    fol = None if follow is None else np.ascontiguousarray(follow, dtype=np.uint8)
    st = Stats()
    rc = lib().or_kernel_halving(_p(K), _p(V), K.shape[1], vm, KERNELS[kernel], delta,
                                 _p(rows), N, _p(u), _p(out), _p(fol), tol, _p(bits),
                                 _p(rho), _p(alpha), _p(thresh), C.byref(st))
    if rc != 0:
        raise ValueError(f"or_kernel_halving failed ({rc})")
    return {"out": out, "bits": bits, "rho": rho, "alpha": alpha, "thresh": thresh,
            "stats": st.as_dict()}


HALVES = {"kh": 0, "uniform": 1}


def uniform_halving(rows, u) -> dict:
    """One bucket: pair i keeps rows[2i+1] iff u[i] < 1/2, else rows[2i]."""
    rows = np.ascontiguousarray(rows, dtype=np.int32)
    u = _f32(u)
    N = rows.size
    out = np.empty(N // 2, dtype=np.int32)
    bits = np.zeros(N // 2, dtype=np.uint8)
    st = Stats()
    rc = lib().or_uniform_halving(_p(rows), N, _p(u), _p(out), _p(bits), C.byref(st))
    if rc != 0:
        raise ValueError(f"or_uniform_halving failed ({rc})")
    return {"out": out, "bits": bits, "stats": st.as_dict()}


def compress(K, V, n_out: int, g: int, U, *, kernel: str = "katt", follow=None,
             tol: float = 1e-5, halve: str = "kh", delta=None, n_sinks: int = 0,
             n_window: int = 0) -> dict:
    """One slice: K, V [n, d]; U = this slice's uniforms.  halve: "kh" (KH(delta),
    delta[r] per round, default 1/2) or "uniform" (one point of each pair, each
    with probability 1/2).  With n_sinks / n_window the first and last rows are
    kept exactly and the n_mid rows between them are thinned to n_out as a
    dataset of their own (v_max of eq. eq:katt over those rows, U drawn for a
    slice of n_mid rows); "idx" is then sinks + coreset + window and "logw"
    their log-weights for eq. def:att_approx: 0 for an exact row and
    log(n_mid / n_out) for a coreset row, which stands for that many rows."""
    K, V = _f64(K), _f64(V)
    if n_sinks or n_window:
        n = K.shape[0]
        mid = slice(n_sinks, n - n_window)
        r = _compress_rows(K[mid], V[mid], n_out, g, U, kernel, follow, tol, halve, delta)
        n_mid = n - n_sinks - n_window
        r["idx"] = np.concatenate([np.arange(n_sinks, dtype=np.int32), r["idx"] + n_sinks,
                                   np.arange(n - n_window, n, dtype=np.int32)])
        r["logw"] = np.concatenate([np.zeros(n_sinks), np.full(n_out, np.log(n_mid / n_out)),
                                    np.zeros(n_window)])
        return r
    return _compress_rows(K, V, n_out, g, U, kernel, follow, tol, halve, delta)


def _compress_rows(K, V, n_out, g, U, kernel, follow, tol, halve, delta):
    n, d = K.shape
    pl = plan(n, n_out, g)
    if pl is None:
        raise ValueError("no valid level structure for these arguments")
    U = _f32(U)
    assert U.size >= pl["uniforms"], (U.size, pl["uniforms"])
    cnt = max(int(pl["uniforms"]), 1)
    idx = np.empty(n_out, dtype=np.int32)
    bits = np.zeros(cnt, dtype=np.uint8)
    rho = np.zeros(cnt)
    fol = None if follow is None else np.ascontiguousarray(follow, dtype=np.uint8)
    if fol is not None:
        assert fol.size >= pl["uniforms"]
    st = Stats()
    dl = None
    if delta is not None:
        dl = np.ascontiguousarray(delta, dtype=np.float64)
        assert dl.size >= pl["rounds"]
    rc = lib().or_compress_ex(_p(K), _p(V), n, d, n_out, g, KERNELS[kernel], HALVES[halve],
                              _p(dl), _p(U), _p(idx), _p(fol), tol, _p(bits), _p(rho),
                              C.byref(st))
    if rc != 0:
        raise ValueError(f"or_compress_ex failed ({rc})")
    return {"idx": idx, "bits": bits, "rho": rho, "stats": st.as_dict(), "plan": pl}


def attention(Q, K, V, rows) -> np.ndarray:
    """Softmax attention of every query over the rows `rows` of K/V (float64)."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    rows = np.ascontiguousarray(rows, dtype=np.int32)
    n_q, d = Q.shape
    O = np.empty((n_q, d))
    lib().or_attention(_p(Q), _p(K), _p(V), n_q, d, _p(rows), rows.size, _p(O))
    return O


def weighted_attention(Q, K, V, rows, logw) -> np.ndarray:
    """Weighted attention (eq. def:att_approx): key rows[j] weighs exp(logw[j])."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    rows = np.ascontiguousarray(rows, dtype=np.int32)
    lw = np.ascontiguousarray(logw, dtype=np.float64)
    assert lw.size == rows.size
    n_q, d = Q.shape
    O = np.empty((n_q, d))
    lib().or_attention_weighted(_p(Q), _p(K), _p(V), n_q, d, _p(rows), _p(lw), rows.size, _p(O))
    return O


def express_uniforms(n: int, n_out: int, mbar: int) -> int:
    """Uniforms a Thinformer decode of n points consumes at most (Halve calls)."""
    u = lib().or_express_uniforms(n, n_out, mbar, None)
    if u < 0:
        raise ValueError("no Express structure for these sizes")
    return u


def express_draws(n: int, n_out: int, mbar: int) -> int:
    """Subsample draws (one per stratum above mbar) a decode of n points needs."""
    k = C.c_int64(0)
    if lib().or_express_uniforms(n, n_out, mbar, C.byref(k)) < 0:
        raise ValueError("no Express structure for these sizes")
    return k.value


def express_keys(n: int, n_out: int, mbar: int, sub_u=None) -> np.ndarray:
    """Keys every point attends over in Thinformer decoding of n points (its
    weighted cache plus itself), int64 [n]; sub_u as in express_decode."""
    keys = np.zeros(max(n, 1), np.int64)
    su = None if sub_u is None else np.ascontiguousarray(sub_u, dtype=np.float32)
    if lib().or_express_keys(n, n_out, mbar, _p(su), _p(keys)) != 0:
        raise ValueError("no Express structure for these sizes")
    return keys[:n]


def express_delta(m: int, i: int, mbar: int, delta: float = 0.5) -> float:
    """Cor. 2: delta_{m,i} for i >= 0, delta_m / 2 (the Halve phase) for i < 0."""
    return lib().or_express_delta(m, i, mbar, delta)


def express_decode(Q, K, V, n_out: int, mbar: int, U, *, delta: float = 0.5,
                   halve: str = "kh", follow=None, tol: float = 1e-5,
                   outputs: bool = True, sub_u=None) -> dict:
    """Thinformer decoding of one slice (Alg. 4 over the Express cache of
    Alg. 1): "O" [n, d] (every point attends over the cache of the points
    before it plus itself), then the final weighted cache ("idx", "logw", in
    the order C_0..C_mp, E), the final thinning factor "m", the swap "bits"
    (indexed like U) and KH "stats".  sub_u: Subsample's draws, one per
    stratum above mbar (None: 0 each, the first point of every stratum)."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    n, d = K.shape
    U = np.ascontiguousarray(U, dtype=np.float32)
    need = express_uniforms(n, n_out, mbar)
    assert U.size >= need
    fol = None if follow is None else np.ascontiguousarray(follow, dtype=np.uint8)
    su = None if sub_u is None else np.ascontiguousarray(sub_u, dtype=np.float32)
    if su is not None:
        assert su.size >= express_draws(n, n_out, mbar)
    bits = np.zeros(max(need, 1), np.uint8)
    O = np.zeros((n, d)) if outputs else None
    cap = 8 * n_out + 2
    rows = np.zeros(cap, np.int32)
    logw = np.zeros(cap)
    klen = C.c_int64(0)
    mfin = C.c_int(0)
    st = Stats()
    rc = lib().or_express_decode(_p(Q), _p(K), _p(V), n, d, n_out, mbar, delta, HALVES[halve],
                                 _p(U), _p(su), _p(fol), tol, _p(bits), _p(O), _p(rows), _p(logw),
                                 C.byref(klen), C.byref(mfin), C.byref(st))
    if rc != 0:
        raise ValueError(f"or_express_decode failed ({rc})")
    k = klen.value
    return {"O": O, "idx": rows[:k].copy(), "logw": logw[:k].copy(), "m": mfin.value,
            "bits": bits[:need], "stats": {f: getattr(st, f) for f, _ in Stats._fields_}}


def exact_attention(Q, K, V) -> np.ndarray:
    K = _f64(K)
    return attention(Q, K, V, np.arange(K.shape[0], dtype=np.int32))
