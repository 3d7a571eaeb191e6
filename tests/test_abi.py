"""C-ABI library checks that need no GPU: it loads, exports every declared
symbol, plans like the oracle, and rejects bad arguments before launching."""
import ctypes as C
import os
import re

import pytest

import oracle
from paper_2606_10944_amd import _lib
from paper_2606_10944_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = C.c_void_p(0x10000)  # never dereferenced: every call below fails validation


def _declared_symbols():
    with open(os.path.join(ROOT, "include", "thin.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:int|const char\*)\s+(thin_\w+)\(", text, re.M)))


def test_library_exports_every_declared_symbol():
    L = _lib.lib()
    declared = _declared_symbols()
    assert set(declared) == set(_lib.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name


def test_status_strings():
    for s in range(6):
        assert _lib.thin_status_str(s).startswith("THIN_")
    assert "unknown" in _lib.thin_status_str(99)


@pytest.mark.parametrize("n,n_out,g", [
    (1024, 32, 2), (3136, 64, 2), (1024, 64, 3), (16384, 128, 3), (65536, 256, 4),
    (1000, 7, 3), (96, 96, 1), (97, 48, 0), (5000, 40, 5), (2, 1, 0), (130, 64, 0),
])
def test_plan_agrees_with_oracle(n, n_out, g):
    p = _lib.thin_plan(3, 2, n, 64, n_out, g)
    o = oracle.plan(n, n_out, g)
    assert o is not None
    assert p["n_kept"] == o["n_kept"]
    assert p["rounds"] == o["rounds"]
    assert p["compress_levels"] == o["compress_levels"]
    assert p["uniforms_per_slice"] == o["uniforms"]
    assert p["uniforms_total"] == 6 * o["uniforms"]
    assert p["workspace_bytes"] >= 6 * p["n_kept"] * 4


@pytest.mark.parametrize("n,n_out,g", [(1024, 1, 0), (1024, 1, 4), (10, 11, 1), (10, 0, 1),
                                       (10, 2, -1), (1000, 7, 2), (200, 3, 2)])
def test_plan_rejects_what_the_oracle_rejects(n, n_out, g):
    with pytest.raises(_lib.ThinError) as e:
        _lib.thin_plan(1, 1, n, 64, n_out, g)
    assert e.value.status == _lib.THIN_EINVAL
    if n_out >= 1 and g >= 0:
        assert oracle.plan(n, n_out, g) is None


def test_plan_rejects_unsupported_head_dim_and_oversized_buckets():
    for d in (16, 48, 256):
        with pytest.raises(_lib.ThinError):
            _lib.thin_plan(1, 1, 1024, d, 32, 2)
    with pytest.raises(_lib.ThinError):           # one bucket of 32768 rows
        _lib.thin_plan(1, 1, 65536, 64, 16384, 0)


def _compress(**kw):
    a = dict(K=FAKE, V=FAKE, dtype=1, B=1, H=2, n=1024, d=64, n_out=32, g=2, U=FAKE,
             nU=2 * 992, idx=FAKE, ws=C.c_void_p(0x100000), wsb=1 << 20)
    a.update(kw)
    return _lib.lib().thin_compress(a["K"], a["V"], a["dtype"], a["B"], a["H"], a["n"], a["d"],
                                    a["n_out"], a["g"], a["U"], a["nU"], a["idx"], a["ws"],
                                    a["wsb"], None)


def test_compress_validates_before_launch():
    assert _compress(n_out=2000) == _lib.THIN_EINVAL
    assert _compress(d=96) == _lib.THIN_EINVAL
    assert _compress(K=None) == _lib.THIN_EINVAL
    assert _compress(idx=None) == _lib.THIN_EINVAL
    assert _compress(dtype=5) == _lib.THIN_EDTYPE
    assert _compress(nU=2 * 992 - 1) == _lib.THIN_EUNIFORMS
    assert _compress(U=None) == _lib.THIN_EINVAL
    assert _compress(wsb=100) == _lib.THIN_EWORKSPACE
    assert _compress(ws=None) == _lib.THIN_EWORKSPACE
    assert _compress(ws=C.c_void_p(0x100010)) == _lib.THIN_EWORKSPACE   # misaligned
    assert _compress(B=0) == _lib.THIN_EINVAL
    assert _compress(B=65536) == _lib.THIN_EINVAL      # more slices than grid y holds


def test_compress_ex_validates_options_before_launch():
    L = _lib.lib()

    def call(halve, delta, opts=True):
        dl = None if delta is None else (C.c_double * len(delta))(*delta)
        o = _lib.CompressOpts(halve, C.cast(dl, C.c_void_p) if dl is not None else None)
        return L.thin_compress_ex(FAKE, FAKE, 1, 1, 1, 1024, 64, 32, 2, FAKE, 992, FAKE,
                                  C.c_void_p(0x100000), 1 << 20, C.byref(o) if opts else None,
                                  None, 0, None)

    assert call(0, None, opts=False) == _lib.THIN_EINVAL
    assert call(2, None) == _lib.THIN_EINVAL
    assert call(-1, None) == _lib.THIN_EINVAL
    assert call(0, [0.5, 0.5, 0.0, 0.5, 0.5]) == _lib.THIN_EINVAL      # delta = 0
    assert call(0, [0.5, 1.5, 0.5, 0.5, 0.5]) == _lib.THIN_EINVAL      # delta > 1
    assert call(0, [0.5, 0.5, 0.5, 0.5, float("nan")]) == _lib.THIN_EINVAL


def test_compress_ex_validates_sinks_and_window_before_launch():
    L = _lib.lib()

    def call(ns, nw):
        o = _lib.CompressOpts(0, None, ns, nw, None)
        return L.thin_compress_ex(FAKE, FAKE, 1, 1, 1, 1024, 64, 32, 2, FAKE, 1 << 20, FAKE,
                                  C.c_void_p(0x100000), 1 << 30, C.byref(o), None, 0, None)

    assert call(-1, 0) == _lib.THIN_EINVAL
    assert call(0, -1) == _lib.THIN_EINVAL
    assert call(1025, 0) == _lib.THIN_EINVAL
    assert call(500, 500) == _lib.THIN_EINVAL   # 24 rows left for n_out = 32
    assert call(0, 1024) == _lib.THIN_EINVAL


def test_traced_compress_checks_trace_length():
    L = _lib.lib()
    rc = L.thin_compress_traced(FAKE, FAKE, 1, 1, 1, 1024, 64, 32, 2, FAKE, 992, FAKE,
                                C.c_void_p(0x100000), 1 << 20, FAKE, 991, None)
    assert rc == _lib.THIN_EINVAL
    rc = L.thin_compress_traced(FAKE, FAKE, 1, 1, 1, 1024, 64, 32, 2, FAKE, 992, FAKE,
                                C.c_void_p(0x100000), 1 << 20, None, 992, None)
    assert rc == _lib.THIN_EINVAL


def test_attention_validates_before_launch():
    L = _lib.lib()

    def call(**kw):
        a = dict(Q=FAKE, K=FAKE, V=FAKE, dtype=1, B=1, H=1, n_q=8, n=16, d=64, idx=FAKE,
                 n_out=4, O=FAKE, od=0)
        a.update(kw)
        return L.thin_attention(a["Q"], a["K"], a["V"], a["dtype"], a["B"], a["H"], a["n_q"],
                                a["n"], a["d"], a["idx"], a["n_out"], a["O"], a["od"], None)

    assert call(d=80) == _lib.THIN_EINVAL
    assert call(n_out=0) == _lib.THIN_EINVAL
    assert call(n_q=0) == _lib.THIN_EINVAL
    assert call(O=None) == _lib.THIN_EINVAL
    assert call(dtype=3) == _lib.THIN_EDTYPE
    assert call(od=2) == _lib.THIN_EDTYPE


def test_weighted_attention_validates_before_launch():
    L = _lib.lib()

    def call(**kw):
        a = dict(dtype=1, n_q=8, d=64, n_out=4, od=0)
        a.update(kw)
        return L.thin_attention_ex(FAKE, FAKE, FAKE, a["dtype"], 1, 1, a["n_q"], 16, a["d"], FAKE,
                                   FAKE, a["n_out"], FAKE, a["od"], None)

    assert call(d=80) == _lib.THIN_EINVAL
    assert call(n_out=0) == _lib.THIN_EINVAL
    assert call(n_q=0) == _lib.THIN_EINVAL
    assert call(dtype=7) == _lib.THIN_EDTYPE
    assert call(od=2) == _lib.THIN_EDTYPE


def test_workloads_are_seeded_and_shaped():
    w = W.WORKLOADS["tiny"]
    Q1, K1, V1 = W.make_qkv(w)
    Q2, K2, V2 = W.make_qkv(w)
    assert tuple(K1.shape) == (1, 1, 1024, 64) and K1.dtype.is_floating_point
    assert (K1 == K2).all() and (Q1 == Q2).all() and (V1 == V2).all()
    u = W.make_uniforms(w, 992)
    assert u.numel() == 992 and float(u.min()) >= 0 and float(u.max()) < 1
    assert ((u.double() * 2 ** 24) % 1 == 0).all()
    w3 = W.WORKLOADS["imggen"].with_(B=2)
    Q, K, V = W.make_qkv(w3)
    assert tuple(Q.shape) == (2, 1, 4096, 64) and tuple(K.shape) == (2, 1, 1024, 64)
    assert float(V.abs().max()) <= 1.0


def test_launch_hook_can_be_set_and_cleared():
    L = _lib.lib()
    calls = []
    cb = _lib.LaunchHook(lambda *a: calls.append(a))
    assert L.thin_set_launch_hook(cb, None) == _lib.THIN_OK
    # a call rejected during validation launches nothing, so the hook is silent
    assert _compress(dtype=5) == _lib.THIN_EDTYPE
    assert L.thin_set_launch_hook(_lib.LaunchHook(), None) == _lib.THIN_OK
    assert calls == []


@pytest.mark.parametrize("n_out,mbar,n_max", [(8, 4, 512), (8, 4, 300), (16, 4, 1000),
                                              (128, 6, 16384), (128, 8, 100000), (4, 2, 64),
                                              (32, 5, 2000), (8, 2, 2000), (8, 4, 5000),
                                              (128, 5, 40000)])
def test_express_plan_counts_the_oracles_uniforms(n_out, mbar, n_max):
    p = _lib.thin_express_plan(2, 3, 64, n_out, mbar, n_max)
    assert p["uniforms_per_slice"] == oracle.express_uniforms(n_max, n_out, mbar)
    assert p["subsample_draws"] == oracle.express_draws(n_max, n_out, mbar)
    assert 1 <= p["max_keys"] <= 6 * n_out + 1 and p["workspace_bytes"] > 0


def test_express_rejects_unsupported_sizes():
    L = _lib.lib()
    plan = _lib.ExpressPlan()

    def rc(B=1, H=1, d=64, n_out=8, mbar=4, n_max=512):
        return L.thin_express_plan(B, H, d, n_out, mbar, n_max, C.byref(plan))

    assert rc() == _lib.THIN_OK
    assert rc(n_max=5000) == _lib.THIN_OK             # m = 6 > mbar: Subsample, groups of 2
    assert rc(mbar=5, n_max=512) == _lib.THIN_OK
    assert rc(mbar=5, n_max=513) == _lib.THIN_EINVAL  # m = 6: groups of 4*8/2^5 = 1 point
    assert rc(n_out=4, mbar=4, n_max=300) == _lib.THIN_EINVAL  # groups of 4*4/16 = 1 point
    assert rc(d=80) == _lib.THIN_EINVAL
    assert rc(n_out=4096) == _lib.THIN_EINVAL         # 4 n_out above the largest bucket
    assert rc(n_max=0) == _lib.THIN_EINVAL
    h = C.c_void_p()
    assert L.thin_express_create(1, 1, 1, 64, 8, 4, 0.0, 0, 512, FAKE, 1 << 30,
                                 C.byref(h)) == _lib.THIN_EINVAL   # delta = 0
    assert L.thin_express_create(1, 1, 1, 64, 8, 4, 0.5, 0, 512, None, 1 << 30,
                                 C.byref(h)) == _lib.THIN_EWORKSPACE
    assert L.thin_express_create(1, 1, 1, 64, 8, 4, 0.5, 0, 512, C.c_void_p(0x100010), 1 << 30,
                                 C.byref(h)) == _lib.THIN_EWORKSPACE  # not 256-byte aligned


@pytest.mark.parametrize("n_out,mbar,n", [(8, 4, 512), (8, 2, 1500), (128, 5, 9000), (16, 4, 1000)])
def test_prefill_plan_matches_decoding(n_out, mbar, n):
    p = _lib.thin_express_prefill_plan(1, 2, n, 64, n_out, mbar)
    assert p["uniforms_per_slice"] == oracle.express_uniforms(n, n_out, mbar)
    assert p["subsample_draws"] == oracle.express_draws(n, n_out, mbar)
    assert p["workspace_bytes"] > 0 and p["host_staging_bytes"] > 0
    # App. G's per-point key counts (Subsample draws of 0), summed
    assert p["attention_keys"] == int(oracle.express_keys(n, n_out, mbar).sum())
    L = _lib.lib()
    assert L.thin_express_prefill(1, 1, 2, n, 64, n_out, mbar, 0.5, 0, FAKE, FAKE, FAKE, FAKE,
                                  1 << 30, None, 0, FAKE, 0, None, 0, None, 0, None, None) in (
        _lib.THIN_EWORKSPACE, _lib.THIN_EINVAL)
    assert L.thin_express_prefill(1, 1, 2, n, 64, n_out, mbar, 1.5, 0, FAKE, FAKE, FAKE, FAKE,
                                  1 << 30, None, 0, FAKE, 0, FAKE, 1 << 40, FAKE, 1 << 40, None,
                                  None) == _lib.THIN_EINVAL


def test_prefill_plan_is_kept_per_size():
    """The prefill's layout is computed once per size: a repeated plan is
    identical, and a cached size does not let arguments that differ from it
    (negative batch and heads of the same product, another d) past the checks."""
    a = _lib.thin_express_prefill_plan(1, 2, 777, 64, 16, 4)
    b = _lib.thin_express_prefill_plan(1, 2, 777, 64, 16, 4)
    assert a == b
    for args in [(-1, -2, 777, 64, 16, 4), (2, 1, 777, 48, 16, 4), (1, 2, 0, 64, 16, 4)]:
        with pytest.raises(_lib.ThinError):
            _lib.thin_express_prefill_plan(*args)
    # another slice count of the same sequence: same uniforms per slice, larger workspace
    c = _lib.thin_express_prefill_plan(2, 2, 777, 64, 16, 4)
    assert c["uniforms_per_slice"] == a["uniforms_per_slice"]
    assert c["workspace_bytes"] > a["workspace_bytes"]


def test_prefill_requires_host_staging():
    n_out, mbar, n = 8, 4, 512
    p = _lib.thin_express_prefill_plan(1, 2, n, 64, n_out, mbar)
    L = _lib.lib()
    draws = (C.c_float * 1)()
    args = [1, 1, 2, n, 64, n_out, mbar, 0.5, 0, FAKE, FAKE, FAKE, FAKE, 1 << 30, draws, 1,
            FAKE, 0, FAKE, 1 << 40]
    assert L.thin_express_prefill(*args, None, 0, None, None) == _lib.THIN_EWORKSPACE
    assert L.thin_express_prefill(*args, FAKE, p["host_staging_bytes"] - 1, None, None) == \
        _lib.THIN_EWORKSPACE


def test_workspace_status_validates_pointers():
    L = _lib.lib()
    st = C.c_int32(0)
    assert L.thin_workspace_status(None, C.byref(st), None) == _lib.THIN_EINVAL
    assert L.thin_workspace_status(FAKE, None, None) == _lib.THIN_EINVAL


def test_shared_mean_workload_reaches_large_cross_exponents():
    """The heavy_tail_mean recipe is a parity case for kappa_att's range: some
    cross exponent <k_i,k_q>/sqrt(d) of an earlier row i against a row q of a
    pair exceeds that pair's larger diagonal exponent ||k||^2/sqrt(d) by more
    than 64 log(2) = 44.4 (natural units), i.e. by more than 2^64 in kappa."""
    import numpy as np
    w = W.custom("hm", B=1, H=1, n=1024, d=128, dtype="bf16", kind="heavy_tail_mean", seed=3)
    _, K, _ = W.make_qkv(w)
    k = K[0, 0].double().numpy()
    X = k @ k.T / np.sqrt(w.d)
    e = np.diag(X)
    worst = -np.inf
    for p in range(1, w.n // 2):
        hp = max(e[2 * p], e[2 * p + 1])
        worst = max(worst, X[: 2 * p, 2 * p: 2 * p + 2].max() - hp)
    assert worst > 64 * np.log(2.0), worst
    assert abs(np.linalg.norm(k.mean(axis=0)) ** 2 / (2 * w.d) - 1.0) < 0.5


def test_static_compress_rejects_what_does_not_fit_before_any_launch():
    """thin_compress_static checks sizes against its fixed array before it
    touches a device: B*H = 256 slices of 65536 rows need more than it holds."""
    L = _lib.lib()
    rc = L.thin_compress_static(FAKE, FAKE, 1, 8, 32, 65536, 128, 256, 4, FAKE, 1 << 40, FAKE,
                                None, None)
    assert rc == _lib.THIN_EWORKSPACE
    assert L.thin_compress_static(FAKE, FAKE, 1, 1, 1, 1000, 80, 8, 1, FAKE, 1 << 20, FAKE,
                                  None, None) == _lib.THIN_EINVAL  # d unsupported
