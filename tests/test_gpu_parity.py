"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Indices: bit-exact, except decisions whose margin |alpha/a - (1 - 2u)| is
below 1e-5 (relative to the threshold a), where either branch is correct; the
oracle then follows the GPU's branch ("follow mode") and counts it.  Any other
disagreement is a hard mismatch and fails.  Attention: max-abs error 2e-3
(bf16 inputs, fp32 accumulation) and 1e-5 (fp32 inputs) against the float64
oracle on the same coreset.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from paper_2606_10944_amd import (LaunchTimer, thin_attention, thin_compress, thin_plan,
                                  thin_selftest_gram16, workspace_status)
from paper_2606_10944_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
MARGIN = 1e-5


def _pmap(fn, items):
    """fn over items on CPU threads (the oracle's C calls release the GIL)."""
    items = list(items)
    with ThreadPoolExecutor(max_workers=min(8, max(len(items), 1))) as ex:
        return list(ex.map(fn, items))


def _tol(w):
    return 2e-3 if w.dtype == "bf16" else 1e-5


def _compress_gpu(w, Q, K, V):
    plan = thin_plan(w.B, w.H, w.n, w.d, w.n_out, w.g)
    U = W.make_uniforms(w, plan["uniforms_total"])
    ws = torch.empty(max(plan["workspace_bytes"], 256), dtype=torch.uint8, device=DEV)
    idx, tr = thin_compress(K.to(DEV), V.to(DEV), w.n_out, w.g, U.to(DEV), trace=True,
                            workspace=ws)
    # every bounded wait of the decision passes completed
    assert workspace_status(ws) == 0
    torch.cuda.synchronize()
    return plan, U, idx.cpu().numpy(), tr.cpu().numpy()


def _check_compress(w, K, V, U, idx, tr, slices):
    Us = U.numpy().reshape(w.S, -1) if U.numel() else np.zeros((w.S, 1), np.float32)
    ts = tr.reshape(w.S, -1) if tr.size else np.zeros((w.S, 1), np.uint8)
    # cheap invariants on every slice: n_out strictly increasing rows in range
    assert idx.shape == (w.B, w.H, w.n_out)
    flat = idx.reshape(w.S, w.n_out)
    assert np.all(np.diff(flat, axis=-1) > 0) and flat.min() >= 0 and flat.max() < w.n

    def one(s):
        b, h = divmod(s, w.H)
        r = oracle.compress(K[b, h], V[b, h], w.n_out, w.g, Us[s], follow=ts[s], tol=MARGIN)
        return s, r

    near = 0
    for s, r in _pmap(one, slices):
        b, h = divmod(s, w.H)
        st = r["stats"]
        assert st["hard_mismatch"] == 0, (w.name, s, st)
        assert np.array_equal(r["idx"], idx[b, h]), (w.name, s)
        near += st["near_ties"]
    return near


def _check_attention(w, Q, K, V, idx, O, slices, rows=None):
    tol = _tol(w)
    q = np.arange(w.n_q) if rows is None else rows

    def one(s):
        b, h = divmod(s, w.H)
        ref = oracle.attention(Q[b, h][q], K[b, h], V[b, h], idx[b, h])
        return float(np.abs(ref - O[b, h][q].astype(np.float64)).max())

    worst = max(_pmap(one, slices))
    assert worst <= tol, (w.name, worst)
    return worst


# ---------------------------------------------------------------------------
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("d", [32, 64, 128])
def test_mfma_fragment_gram_matches_matmul(dtype, d):
    g = torch.Generator().manual_seed(d)
    rows = torch.randn(32, d, generator=g).to(dtype)
    got = thin_selftest_gram16(rows.to(DEV)).cpu().double()
    r = rows.double()
    want = r[:16] @ r[16:].T
    assert torch.allclose(got, want, rtol=1e-5, atol=1e-4 * d), (got - want).abs().max()


@pytest.mark.parametrize("name", ["tiny", "vit", "imggen"])
def test_named_workload_full_parity(name):
    w = W.WORKLOADS[name]
    Q, K, V = W.make_qkv(w)
    plan, U, idx, tr = _compress_gpu(w, Q, K, V)
    near = _check_compress(w, K, V, U, idx, tr, range(w.S))
    O = thin_attention(Q.to(DEV), K.to(DEV), V.to(DEV), torch.from_numpy(idx).to(DEV))
    torch.cuda.synchronize()
    err = _check_attention(w, Q, K, V, idx, O.cpu().numpy(), range(w.S))
    print(f"{name}: near-ties {near}, attention max err {err:.3g}")


# 16 of the long workload's 64 slices: every batch, first / last / two inner heads
LONG_SLICES = [0, 5, 10, 15, 16, 21, 26, 31, 32, 37, 42, 47, 48, 53, 58, 63]


def test_long_workload_sampled_parity():
    """Full-size long-sequence workload (the benchmark's configuration):
    compress parity on 16 slices, attention on sampled queries."""
    w = W.WORKLOADS["long"]
    Q, K, V = W.make_qkv(w)
    plan, U, idx, tr = _compress_gpu(w, Q, K, V)
    near = _check_compress(w, K, V, U, idx, tr, LONG_SLICES)
    O = thin_attention(Q.to(DEV), K.to(DEV), V.to(DEV), torch.from_numpy(idx).to(DEV))
    torch.cuda.synchronize()
    rows = np.random.default_rng(0).choice(w.n_q, 512, replace=False)
    err = _check_attention(w, Q, K, V, idx, O.cpu().numpy(), LONG_SLICES, rows)
    print(f"long: near-ties {near}, attention max err {err:.3g}")


def test_long_shared_key_mean_parity():
    """The long workload's shape and recipe with a key mean shared by each
    slice's rows (||mu||^2 = 2d, then 5% of the rows x4): cross exponents of
    the large rows exceed small pairs' diagonal exponents by ~90 natural
    units, which no float32 exponent can hold unscaled."""
    w = W.WORKLOADS["long"].with_(name="long_mean", kind="heavy_tail_mean")
    Q, K, V = W.make_qkv(w)
    plan, U, idx, tr = _compress_gpu(w, Q, K, V)
    near = _check_compress(w, K, V, U, idx, tr, LONG_SLICES[::2])
    O = thin_attention(Q.to(DEV), K.to(DEV), V.to(DEV), torch.from_numpy(idx).to(DEV))
    torch.cuda.synchronize()
    rows = np.random.default_rng(2).choice(w.n_q, 256, replace=False)
    err = _check_attention(w, Q, K, V, idx, O.cpu().numpy(), LONG_SLICES[::4], rows)
    print(f"long, shared key mean: near-ties {near}, attention max err {err:.3g}")


def test_stress_workload_sampled_parity():
    """Stress workload: compress parity on the first, the last and two inner
    slices (the oracle takes ~25 s per slice, run on CPU threads)."""
    w = W.WORKLOADS["stress"]
    Q, K, V = W.make_qkv(w)
    plan, U, idx, tr = _compress_gpu(w, Q, K, V)
    slices = [0, 11, 22, 31]
    near = _check_compress(w, K, V, U, idx, tr, slices)
    O = thin_attention(Q.to(DEV), K.to(DEV), V.to(DEV), torch.from_numpy(idx).to(DEV))
    torch.cuda.synchronize()
    rows = np.random.default_rng(1).choice(w.n_q, 256, replace=False)
    err = _check_attention(w, Q, K, V, idx, O.cpu().numpy(), slices, rows)
    print(f"stress: near-ties {near}, attention max err {err:.3g}")


CUSTOM = [
    # ragged buckets (40 rows < one 64-row block), subsample, bf16 d=64
    dict(B=1, H=2, n=5000, n_out=40, g=2, d=64, dtype="bf16", kind="gauss"),
    # single 2560-row bucket (eight-wave kernel), subsample
    dict(B=1, H=1, n=5000, n_out=40, g=5, d=64, dtype="bf16", kind="layernorm"),
    # odd n_out, d=32, many tiny buckets
    dict(B=2, H=3, n=1000, n_out=7, g=3, d=32, dtype="bf16", kind="gauss"),
    dict(B=1, H=1, n=1000, n_out=7, g=4, d=32, dtype="fp32", kind="gauss_d4"),
    # one round, subsample of 97 rows to 96
    dict(B=2, H=1, n=97, n_out=48, g=0, d=64, dtype="fp32", kind="gauss_d4"),
    # smallest case: two rows
    dict(B=3, H=1, n=2, n_out=1, g=0, d=64, dtype="fp32", kind="gauss"),
    dict(B=1, H=2, n=130, n_out=64, g=0, d=128, dtype="bf16", kind="gauss"),
    # fp32 with d = 128 (32-row blocks)
    dict(B=1, H=2, n=600, n_out=32, g=1, d=128, dtype="fp32", kind="gauss_d4"),
    # heavy-tailed keys at a small size
    dict(B=2, H=1, n=2048, n_out=32, g=2, d=128, dtype="bf16", kind="heavy_tail"),
    # clustered keys, one bucket per round
    dict(B=2, H=1, n=512, n_out=16, g=4, d=64, dtype="fp32", kind="mixture"),
    # fp32 d = 128 with buckets above its 128-row local size: score launches
    # with streamed chunks from round 0 on (own chunks first, then the rest)
    dict(B=1, H=1, n=1024, n_out=64, g=2, d=128, dtype="fp32", kind="gauss_d4"),
    # bf16 d = 32: local rounds, then 512- and 1024-row buckets
    dict(B=1, H=2, n=4096, n_out=8, g=6, d=32, dtype="bf16", kind="gauss"),
    # 64 slices: rounds of 16384, 4096 and 1024 buckets of 16, 32 and 64 rows
    # (one wavefront per bucket), then the local and score kernels
    dict(B=4, H=16, n=4096, n_out=16, g=3, d=32, dtype="bf16", kind="heavy_tail"),
    # keys with a shared mean and 5% of rows x4 (cross exponents far above
    # small pairs' diagonal ones): local rounds, then 512-row buckets
    dict(B=2, H=1, n=4096, n_out=64, g=2, d=128, dtype="bf16", kind="heavy_tail_mean"),
    dict(B=2, H=1, n=8192, n_out=16, g=5, d=64, dtype="bf16", kind="heavy_tail_mean"),
    dict(B=1, H=2, n=2048, n_out=32, g=3, d=64, dtype="fp32", kind="heavy_tail_mean"),
]


@pytest.mark.parametrize("cfg", CUSTOM, ids=lambda c: f"n{c['n']}-o{c['n_out']}-g{c['g']}-d{c['d']}-{c['dtype']}")
def test_custom_shapes_parity(cfg):
    w = W.custom("custom", seed=11, **cfg)
    Q, K, V = W.make_qkv(w)
    plan, U, idx, tr = _compress_gpu(w, Q, K, V)
    _check_compress(w, K, V, U, idx, tr, range(w.S))
    O = thin_attention(Q.to(DEV), K.to(DEV), V.to(DEV), torch.from_numpy(idx).to(DEV))
    torch.cuda.synchronize()
    _check_attention(w, Q, K, V, idx, O.cpu().numpy(), range(w.S))


# Decision passes whose buckets' early rows are added by helper workgroups
# (rounds of at most 128 buckets, a multiple of 8, of at least 4096 rows):
# every slice, or four of the 8192-row case, against the oracle.
HELPER_CASES = [
    # one round of 8 buckets of 4096 rows (seven helpers per bucket)
    (dict(B=1, H=8, n=4096, n_out=32, g=6, d=64, dtype="bf16", kind="gauss"), range(8)),
    # fp32, d = 128: 8 buckets of 4096 rows
    (dict(B=1, H=8, n=4096, n_out=64, g=5, d=128, dtype="fp32", kind="gauss_d4"), range(8)),
    # 16 buckets of 8192 rows, then 16 of 4096
    (dict(B=2, H=8, n=8192, n_out=64, g=6, d=64, dtype="bf16", kind="heavy_tail"), (0, 5, 10, 15)),
]


@pytest.mark.parametrize("cfg,slices", HELPER_CASES,
                         ids=lambda c: f"S{c['B'] * c['H']}-n{c['n']}-d{c['d']}-{c['dtype']}"
                         if isinstance(c, dict) else "")
def test_decision_helpers_parity(cfg, slices):
    w = W.custom("helpers", seed=13, **cfg)
    Q, K, V = W.make_qkv(w)
    plan, U, idx, tr = _compress_gpu(w, Q, K, V)
    _check_compress(w, K, V, U, idx, tr, slices)


def test_nout_equal_n_is_identity_and_exact_attention():
    w = W.custom("ident", B=2, H=1, n=96, n_out=96, g=1, d=64, dtype="fp32")
    Q, K, V = W.make_qkv(w)
    plan, U, idx, tr = _compress_gpu(w, Q, K, V)
    assert plan["rounds"] == 0
    assert np.array_equal(idx, np.broadcast_to(np.arange(96, dtype=np.int32), idx.shape))
    O = thin_attention(Q.to(DEV), K.to(DEV), V.to(DEV), torch.from_numpy(idx).to(DEV)).cpu()
    for s in range(2):
        ref = oracle.exact_attention(Q[s, 0], K[s, 0], V[s, 0])
        assert np.abs(ref - O[s, 0].numpy()).max() <= 1e-5


def test_compress_is_deterministic_and_stream_ordered():
    w = W.custom("det", B=2, H=2, n=3000, n_out=32, g=2, d=128, dtype="bf16", kind="gauss")
    Q, K, V = W.make_qkv(w)
    plan = thin_plan(w.B, w.H, w.n, w.d, w.n_out, w.g)
    U = W.make_uniforms(w, plan["uniforms_total"]).to(DEV)
    Kd, Vd = K.to(DEV), V.to(DEV)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        a, ta = thin_compress(Kd, Vd, w.n_out, w.g, U, trace=True, stream=side)
        b, tb = thin_compress(Kd, Vd, w.n_out, w.g, U, trace=True, stream=side)
    side.synchronize()
    assert torch.equal(a, b) and torch.equal(ta, tb)


def test_attention_edge_cases():
    w = W.custom("edge", B=1, H=2, n=700, n_q=333, d=64, dtype="bf16", kind="gauss")
    Q, K, V = W.make_qkv(w)
    Qd, Kd, Vd = Q.to(DEV), K.to(DEV), V.to(DEV)
    rng = np.random.default_rng(3)
    cases = {
        "one key": np.array([[[5], [600]]], np.int32),
        "many chunks, ragged": np.sort(rng.choice(700, size=(1, 2, 301)), axis=-1).astype(np.int32),
        "duplicates": np.full((1, 2, 70), 3, np.int32),
    }
    for name, idx in cases.items():
        O = thin_attention(Qd, Kd, Vd, torch.from_numpy(idx).to(DEV)).cpu().numpy()
        for h in range(2):
            ref = oracle.attention(Q[0, h], K[0, h], V[0, h], idx[0, h])
            assert np.abs(ref - O[0, h]).max() <= 2e-3, name
    O = thin_attention(Qd, Kd, Vd, torch.from_numpy(cases["one key"]).to(DEV)).cpu().numpy()
    assert np.array_equal(O[0, 0], np.repeat(V[0, 0, 5:6].float().numpy(), 333, axis=0))


def test_attention_bf16_output():
    w = W.custom("bo", B=2, H=1, n=1024, n_q=1000, d=128, dtype="bf16", kind="gauss")
    Q, K, V = W.make_qkv(w)
    idx = np.sort(np.random.default_rng(4).choice(1024, size=(2, 1, 128), replace=False),
                  axis=-1).astype(np.int32)
    O = thin_attention(Q.to(DEV), K.to(DEV), V.to(DEV), torch.from_numpy(idx).to(DEV),
                       out_dtype=torch.bfloat16)
    O = O.float().cpu().numpy()
    for s in range(2):
        ref = oracle.attention(Q[s, 0], K[s, 0], V[s, 0], idx[s, 0])
        # fp32 accumulation error plus one bf16 rounding of the output
        assert np.all(np.abs(ref - O[s, 0]) <= 2e-3 + 2.0 ** -8 * np.abs(ref))


def test_launch_timer_sees_every_kernel_in_order():
    w = W.custom("lt", B=1, H=2, n=5000, n_out=40, g=2, d=64, dtype="bf16", kind="gauss")
    Q, K, V = W.make_qkv(w)
    plan = thin_plan(w.B, w.H, w.n, w.d, w.n_out, w.g)
    U = W.make_uniforms(w, plan["uniforms_total"]).to(DEV)
    stream = torch.cuda.current_stream()
    with LaunchTimer(stream) as lt:
        idx = thin_compress(K.to(DEV), V.to(DEV), w.n_out, w.g, U, stream=stream)
        thin_attention(Q.to(DEV), K.to(DEV), V.to(DEV), idx, stream=stream)
        torch.cuda.synchronize()
    rec = lt.records()
    L = plan["rounds"]
    got = [(k, r) for k, r, _ in rec]
    assert got[:2] == [("subsample", -1), ("vmax", -1)] and got[-1] == ("attention", -1)
    # each round is either one local launch (buckets of 40..160 rows here) or
    # pair scores + decisions (the 320-row round)
    body, i, kinds = got[2:-1], 0, []
    for r in range(L):
        if body[i] == ("local", r):
            i += 1
            kinds.append("local")
        else:
            assert body[i:i + 2] == [("scores", r), ("decide", r)]
            i += 2
            kinds.append("split")
    assert i == len(body)
    assert "local" in kinds and "split" in kinds
    assert all(ms > 0 for _, _, ms in rec)


# ---------------------------------------------------------------------------
# thin_compress_ex: uniform halving and KH's delta per round
# ---------------------------------------------------------------------------
def _compress_gpu_ex(w, K, V, **kw):
    plan = thin_plan(w.B, w.H, w.n, w.d, w.n_out, w.g)
    U = W.make_uniforms(w, plan["uniforms_total"])
    idx, tr = thin_compress(K.to(DEV), V.to(DEV), w.n_out, w.g, U.to(DEV), trace=True, **kw)
    torch.cuda.synchronize()
    return plan, U, idx.cpu().numpy(), tr.cpu().numpy()


@pytest.mark.parametrize("name", ["tiny", "vit", "imggen", "long", "stress"])
def test_uniform_halving_parity(name):
    """Uniform halving (no floating point but u < 1/2): indices and swap bits
    bit-exact against the oracle."""
    w = W.WORKLOADS[name]
    Q, K, V = W.make_qkv(w)
    plan, U, idx, tr = _compress_gpu_ex(w, K, V, halve="uniform")
    Us = U.numpy().reshape(w.S, -1)
    ts = tr.reshape(w.S, -1)
    # (every round in one launch up to 32768 kept rows per slice, one launch
    # per round beyond: the stress workload keeps 65536)
    slices = range(w.S) if w.S <= 16 else [0, w.S // 2 + 5, w.S - 1]
    for s in slices:
        b, h = divmod(s, w.H)
        r = oracle.compress(K[b, h], V[b, h], w.n_out, w.g, Us[s], halve="uniform")
        assert np.array_equal(r["idx"], idx[b, h]), (name, s)
        assert np.array_equal(r["bits"], ts[s]), (name, s)


@pytest.mark.parametrize("name", ["tiny", "imggen"])
def test_kh_delta_schedule_parity(name):
    """KH with a different delta in every round, against the oracle with the
    same schedule (same margin rule as the default path)."""
    w = W.WORKLOADS[name]
    Q, K, V = W.make_qkv(w)
    L = thin_plan(w.B, w.H, w.n, w.d, w.n_out, w.g)["rounds"]
    delta = [1e-4 + (1.0 - 1e-4) * r / max(L - 1, 1) for r in range(L)]
    plan, U, idx, tr = _compress_gpu_ex(w, K, V, delta=delta)
    Us = U.numpy().reshape(w.S, -1)
    ts = tr.reshape(w.S, -1)
    for s in range(w.S):
        b, h = divmod(s, w.H)
        r = oracle.compress(K[b, h], V[b, h], w.n_out, w.g, Us[s], delta=delta, follow=ts[s],
                            tol=MARGIN)
        assert r["stats"]["hard_mismatch"] == 0, (name, s, r["stats"])
        assert np.array_equal(r["idx"], idx[b, h]), (name, s)


def test_uniform_halving_runs_every_round_in_one_launch():
    w = W.custom("lu", B=1, H=2, n=5000, n_out=40, g=2, d=64, dtype="bf16", kind="gauss")
    Q, K, V = W.make_qkv(w)
    plan = thin_plan(w.B, w.H, w.n, w.d, w.n_out, w.g)
    U = W.make_uniforms(w, plan["uniforms_total"]).to(DEV)
    stream = torch.cuda.current_stream()
    with LaunchTimer(stream) as lt:
        thin_compress(K.to(DEV), V.to(DEV), w.n_out, w.g, U, halve="uniform", stream=stream)
        torch.cuda.synchronize()
    got = [(k, r) for k, r, _ in lt.records()]
    assert got == [("subsample", -1), ("status", -1), ("uniform", -1)]


# ---------------------------------------------------------------------------
# Exact sink / window rows and weighted attention (eq. def:att_approx)
# ---------------------------------------------------------------------------
SINKS = [
    # the n_sinks = n_window = 32 setting of the long-context experiments, full size
    dict(name="long", ns=32, nw=32, halve="kh", slices=[0, 37, 63], q_rows=512),
    # a few sinks and a longer window
    dict(name="imggen", ns=4, nw=64, halve="kh", slices=None, q_rows=None),
    dict(name="vit", ns=1, nw=0, halve="kh", slices=[0, 17, 31], q_rows=None),
    dict(name="tiny", ns=0, nw=9, halve="uniform", slices=None, q_rows=None),
]


def _check_sinks_case(w, ns, nw, halve, slices, q_rows):
    Q, K, V = W.make_qkv(w)
    nm = w.n - ns - nw
    plan = thin_plan(w.B, w.H, nm, w.d, w.n_out, w.g)
    U = W.make_uniforms(w, plan["uniforms_total"])
    Kd, Vd = K.to(DEV), V.to(DEV)
    idx, tr, lw = thin_compress(Kd, Vd, w.n_out, w.g, U.to(DEV), trace=True, halve=halve,
                                n_sinks=ns, n_window=nw, return_logw=True)
    O = thin_attention(Q.to(DEV), Kd, Vd, idx, logw=lw)
    torch.cuda.synchronize()
    idx, tr, lw, O = idx.cpu().numpy(), tr.cpu().numpy(), lw.cpu().numpy(), O.cpu().numpy()
    m = ns + w.n_out + nw
    assert idx.shape == (w.B, w.H, m)
    Us = U.numpy().reshape(w.S, -1) if U.numel() else np.zeros((w.S, 1), np.float32)
    ts = tr.reshape(w.S, -1) if tr.size else np.zeros((w.S, 1), np.uint8)
    q = np.arange(w.n_q) if q_rows is None else \
        np.random.default_rng(5).choice(w.n_q, q_rows, replace=False)
    worst = 0.0
    for s in (range(w.S) if slices is None else slices):
        b, h = divmod(s, w.H)
        r = oracle.compress(K[b, h], V[b, h], w.n_out, w.g, Us[s], halve=halve, follow=ts[s],
                            tol=MARGIN, n_sinks=ns, n_window=nw)
        assert r["stats"]["hard_mismatch"] == 0, (w.name, s, r["stats"])
        assert np.array_equal(r["idx"], idx[b, h]), (w.name, s)
        np.testing.assert_allclose(lw[b, h], r["logw"].astype(np.float32), rtol=1e-7, atol=0)
        ref = oracle.weighted_attention(Q[b, h][q], K[b, h], V[b, h], r["idx"], r["logw"])
        worst = max(worst, float(np.abs(ref - O[b, h][q]).max()))
    assert worst <= _tol(w), (w.name, worst)
    return worst


@pytest.mark.parametrize("case", SINKS, ids=lambda c: f"{c['name']}-s{c['ns']}-w{c['nw']}-{c['halve']}")
def test_sinks_window_compress_and_weighted_attention_parity(case):
    w = W.WORKLOADS[case["name"]]
    err = _check_sinks_case(w, case["ns"], case["nw"], case["halve"], case["slices"],
                            case["q_rows"])
    print(f"{case['name']} sinks {case['ns']} window {case['nw']}: attention max err {err:.3g}")


SINKS_EDGE = [
    # nothing left to thin: the coreset is every middle row, no round runs
    dict(B=2, H=1, n=96, n_out=64, g=1, d=64, dtype="fp32", ns=16, nw=16),
    # no round, subsample of 69 middle rows to 64
    dict(B=2, H=1, n=101, n_out=64, g=1, d=128, dtype="bf16", ns=16, nw=16),
    # odd offsets, ragged buckets, generic attention kernel (d = 32)
    dict(B=2, H=2, n=1000, n_out=7, g=3, d=32, dtype="bf16", ns=7, nw=13),
    # fp32 d = 128 with streamed score chunks, weighted generic kernel
    dict(B=1, H=1, n=1100, n_out=64, g=2, d=128, dtype="fp32", ns=40, nw=36),
]


@pytest.mark.parametrize("cfg", SINKS_EDGE, ids=lambda c: f"n{c['n']}-o{c['n_out']}-s{c['ns']}-w{c['nw']}-d{c['d']}-{c['dtype']}")
def test_sinks_window_edge_cases(cfg):
    cfg = dict(cfg)
    ns, nw = cfg.pop("ns"), cfg.pop("nw")
    w = W.custom("sinks", seed=17, **cfg)
    _check_sinks_case(w, ns, nw, "kh", None, None)


def test_sinks_window_launch_sequence_ends_with_the_layout():
    w = W.custom("sl", B=1, H=2, n=5000, n_out=40, g=2, d=64, dtype="bf16", kind="gauss")
    Q, K, V = W.make_qkv(w)
    plan = thin_plan(w.B, w.H, w.n - 64, w.d, w.n_out, w.g)
    U = W.make_uniforms(w, plan["uniforms_total"]).to(DEV)
    stream = torch.cuda.current_stream()
    with LaunchTimer(stream) as lt:
        thin_compress(K.to(DEV), V.to(DEV), w.n_out, w.g, U, n_sinks=32, n_window=32,
                      stream=stream)
        torch.cuda.synchronize()
    got = [k for k, _, _ in lt.records()]
    assert got[:2] == ["subsample", "vmax"] and got[-1] == "assemble"
    assert got.count("assemble") == 1


@pytest.mark.parametrize("dtype,d,n_out", [("bf16", 128, 192), ("bf16", 64, 29), ("bf16", 32, 300),
                                           ("bf16", 128, 300), ("fp32", 64, 130)])
def test_weighted_attention_edge_cases(dtype, d, n_out):
    """Random log-weights with dropped keys, over the resident kernel (bf16,
    d = 64 / 128, up to 256 keys) and the chunked one (others); the first 64
    keys all dropped, so a whole chunk carries no weight."""
    w = W.custom("wa", B=1, H=2, n=700, n_q=333, d=d, dtype=dtype, kind="gauss")
    Q, K, V = W.make_qkv(w)
    rng = np.random.default_rng(d + n_out)
    idx = rng.integers(0, 700, size=(1, 2, n_out)).astype(np.int32)
    logw = (rng.standard_normal((1, 2, n_out)) * 3).astype(np.float32)
    logw[rng.random((1, 2, n_out)) < 0.2] = -np.inf
    if n_out > 64:
        logw[:, :, :64] = -np.inf
    logw[:, :, -1] = 1.0
    O = thin_attention(Q.to(DEV), K.to(DEV), V.to(DEV), torch.from_numpy(idx).to(DEV),
                       logw=torch.from_numpy(logw).to(DEV)).cpu().numpy()
    for h in range(2):
        ref = oracle.weighted_attention(Q[0, h], K[0, h], V[0, h], idx[0, h],
                                        logw[0, h].astype(np.float64))
        assert np.abs(ref - O[0, h]).max() <= _tol(w), (dtype, d, n_out, h)


def test_equal_log_weights_match_unweighted_attention():
    w = W.custom("eq", B=2, H=1, n=1024, n_q=1000, d=128, dtype="bf16", kind="gauss")
    Q, K, V = W.make_qkv(w)
    idx = np.sort(np.random.default_rng(6).choice(1024, size=(2, 1, 128), replace=False),
                  axis=-1).astype(np.int32)
    Qd, Kd, Vd, Id = Q.to(DEV), K.to(DEV), V.to(DEV), torch.from_numpy(idx).to(DEV)
    a = thin_attention(Qd, Kd, Vd, Id)
    b = thin_attention(Qd, Kd, Vd, Id, logw=torch.full((2, 1, 128), 2.5, device=DEV))
    torch.cuda.synchronize()
    assert (a - b).abs().max().item() <= 1e-5


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("n_out", [17, 64, 90, 96, 128, 150, 192, 256])
def test_resident_attention_tiers(d, n_out):
    """Every coreset size tier of the resident bf16 kernel (16-key tiles padded
    to 2, 4, 6, 8, 12, 16), unweighted and weighted."""
    w = W.custom("rt", B=1, H=2, n=900, n_q=777, d=d, dtype="bf16", kind="gauss")
    Q, K, V = W.make_qkv(w)
    rng = np.random.default_rng(n_out * d)
    idx = rng.integers(0, 900, size=(1, 2, n_out)).astype(np.int32)
    logw = (rng.standard_normal((1, 2, n_out)) * 2).astype(np.float32)
    Qd, Kd, Vd, Id = Q.to(DEV), K.to(DEV), V.to(DEV), torch.from_numpy(idx).to(DEV)
    O = thin_attention(Qd, Kd, Vd, Id).cpu().numpy()
    Ow = thin_attention(Qd, Kd, Vd, Id, logw=torch.from_numpy(logw).to(DEV)).cpu().numpy()
    for h in range(2):
        ref = oracle.attention(Q[0, h], K[0, h], V[0, h], idx[0, h])
        assert np.abs(ref - O[0, h]).max() <= 2e-3, (d, n_out, h)
        ref = oracle.weighted_attention(Q[0, h], K[0, h], V[0, h], idx[0, h],
                                        logw[0, h].astype(np.float64))
        assert np.abs(ref - Ow[0, h]).max() <= 2e-3, (d, n_out, h, "weighted")
