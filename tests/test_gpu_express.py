"""Thinformer decoding over the Express cache (thin_express_*) against the
CPU oracle: every point's output (max-abs 2e-3 for bf16 inputs, 1e-5 for
fp32) and the final weighted cache (indices bit-exact, KH decisions in
follow mode at a 1e-5 relative margin as for the compress path; uniform
halving bit-exact including its swap bits)."""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from paper_2606_10944_amd import (ExpressCache, thin_express_plan, thin_express_prefill,
                                  thin_express_prefill_plan, workspace_status)
from paper_2606_10944_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
MARGIN = 1e-5

CASES = [
    # exact phase, levels 0, 2, 4 and their Halve phases (all KH calls local)
    dict(B=2, H=2, d=64, dtype="bf16", n_out=8, mbar=4, n=512, halve="kh"),
    dict(B=1, H=3, d=32, dtype="bf16", n_out=8, mbar=4, n=400, halve="uniform"),
    dict(B=1, H=2, d=128, dtype="fp32", n_out=16, mbar=4, n=1024, halve="kh"),
    # n_out = 128: Halve phase on 512 points (pair scores + decisions), a partial level 2
    dict(B=1, H=2, d=128, dtype="bf16", n_out=128, mbar=6, n=1800, halve="kh"),
    # Subsample above mbar (strata of 4 and 16 points)
    dict(B=1, H=2, d=64, dtype="bf16", n_out=8, mbar=2, n=1500, halve="kh"),
    dict(B=2, H=1, d=64, dtype="fp32", n_out=8, mbar=2, n=2100, halve="uniform"),
    # the decoding experiments' setting mbar = log2(n_out) - 2, past 8192 points
    dict(B=1, H=2, d=128, dtype="bf16", n_out=128, mbar=5, n=9000, halve="kh"),
    # fewer points than n_out (exact phase only, no uniforms), and exactly the
    # points that end in the first Halve phase
    dict(B=1, H=2, d=64, dtype="fp32", n_out=8, mbar=2, n=5, halve="kh"),
    dict(B=2, H=1, d=64, dtype="bf16", n_out=8, mbar=2, n=32, halve="kh"),
]


def _run(c):
    w = W.custom("ex", B=c["B"], H=c["H"], n=c["n"], d=c["d"], dtype=c["dtype"], kind="gauss")
    Q, K, V = W.make_qkv(w)
    plan = thin_express_plan(w.B, w.H, w.d, c["n_out"], c["mbar"], w.n)
    U = W.make_uniforms(w, w.S * plan["uniforms_per_slice"])
    nd = plan["subsample_draws"]
    draws = torch.from_numpy(np.random.default_rng(7).random(max(nd, 1)).astype(np.float32))
    dt = torch.bfloat16 if c["dtype"] == "bf16" else torch.float32
    ex = ExpressCache(w.B, w.H, w.d, c["n_out"], c["mbar"], w.n, dtype=dt, halve=c["halve"])
    Qd, Kd, Vd, Ud = Q.to(DEV), K.to(DEV), V.to(DEV), U.to(DEV)
    tr = torch.zeros(max(U.numel(), 1), dtype=torch.uint8, device=DEV)
    O = torch.empty((w.B, w.H, w.n, w.d), dtype=torch.float32, device=DEV)
    for t in range(w.n):
        O[:, :, t] = ex.step(Qd[:, :, t].contiguous(), Kd, Vd, Ud, draws=draws, trace=tr)
    idx, lw, m = ex.cache()
    torch.cuda.synchronize()
    assert ex.status() == 0  # every bounded wait of every Halve call completed
    ex.close()
    return w, Q, K, V, U, O.cpu().numpy(), idx.cpu().numpy(), lw.cpu().numpy(), m, \
        tr.cpu().numpy(), plan, draws.numpy()


@pytest.mark.parametrize("c", CASES, ids=lambda c: f"o{c['n_out']}-mbar{c['mbar']}-n{c['n']}-d{c['d']}-{c['dtype']}-{c['halve']}")
def test_express_decode_parity(c):
    w, Q, K, V, U, O, idx, lw, m, tr, plan, draws = _run(c)
    us = plan["uniforms_per_slice"]
    Us = U.numpy().reshape(w.S, -1) if us else np.zeros((w.S, 1), np.float32)
    ts = tr[: w.S * us].reshape(w.S, -1) if us else np.zeros((w.S, 1), np.uint8)
    tol = 2e-3 if c["dtype"] == "bf16" else 1e-5
    near = 0
    for s in range(w.S):
        b, h = divmod(s, w.H)
        r = oracle.express_decode(Q[b, h], K[b, h], V[b, h], c["n_out"], c["mbar"], Us[s],
                                  halve=c["halve"], follow=ts[s] if c["halve"] == "kh" else None,
                                  tol=MARGIN, sub_u=draws)
        assert r["stats"]["hard_mismatch"] == 0, (s, r["stats"])
        near += r["stats"]["near_ties"]
        if c["halve"] == "uniform":
            assert np.array_equal(r["bits"], ts[s]), s
        assert r["m"] == m
        assert np.array_equal(r["idx"], idx[b, h]), s
        np.testing.assert_allclose(lw[b, h], r["logw"].astype(np.float32), rtol=1e-6, atol=1e-7)
        err = np.abs(r["O"] - O[b, h]).max()
        assert err <= tol, (s, err)
    print(f"near ties {near}")


@pytest.mark.parametrize("c", CASES, ids=lambda c: f"o{c['n_out']}-mbar{c['mbar']}-n{c['n']}-d{c['d']}-{c['dtype']}-{c['halve']}")
def test_express_prefill_parity(c):
    """Masked prefill: every point's output equals Thinformer decoding's (the
    oracle, following the prefill's own KH decisions at near ties)."""
    w = W.custom("ex", B=c["B"], H=c["H"], n=c["n"], d=c["d"], dtype=c["dtype"], kind="gauss")
    Q, K, V = W.make_qkv(w)
    plan = thin_express_plan(w.B, w.H, w.d, c["n_out"], c["mbar"], w.n)
    us = plan["uniforms_per_slice"]
    U = W.make_uniforms(w, w.S * us)
    draws = torch.from_numpy(np.random.default_rng(7).random(
        max(plan["subsample_draws"], 1)).astype(np.float32))
    _check_prefill(w, Q, K, V, U, c["n_out"], c["mbar"], c["halve"], draws, range(w.S))


def _check_prefill(w, Q, K, V, U, n_out, mbar, halve, draws, slices):
    us = U.numel() // w.S
    pplan = thin_express_prefill_plan(w.B, w.H, w.n, w.d, n_out, mbar)
    ws = torch.empty(max(pplan["workspace_bytes"], 256), dtype=torch.uint8, device=DEV)
    tr = torch.zeros(max(U.numel(), 1), dtype=torch.uint8, device=DEV)
    O = thin_express_prefill(Q.to(DEV), K.to(DEV), V.to(DEV), n_out, mbar, U.to(DEV),
                             draws=draws, halve=halve, trace=tr, workspace=ws)
    assert workspace_status(ws) == 0
    torch.cuda.synchronize()
    O, tr = O.cpu().numpy(), tr.cpu().numpy()
    Us = U.numpy().reshape(w.S, -1) if us else np.zeros((w.S, 1), np.float32)
    ts = tr[: w.S * us].reshape(w.S, -1) if us else np.zeros((w.S, 1), np.uint8)
    tol = 2e-3 if w.dtype == "bf16" else 1e-5

    def one(s):
        b, h = divmod(s, w.H)
        return s, oracle.express_decode(Q[b, h], K[b, h], V[b, h], n_out, mbar, Us[s],
                                        halve=halve, follow=ts[s] if halve == "kh" else None,
                                        tol=MARGIN, sub_u=draws.numpy())

    slices = list(slices)
    with ThreadPoolExecutor(max_workers=min(8, len(slices))) as ex:
        results = list(ex.map(one, slices))
    for s, r in results:
        b, h = divmod(s, w.H)
        assert r["stats"]["hard_mismatch"] == 0, (s, r["stats"])
        if halve == "uniform":
            assert np.array_equal(r["bits"], ts[s]), s
        err = np.abs(r["O"] - O[b, h]).max(axis=-1)
        bad = np.nonzero(err > tol)[0]
        assert bad.size == 0, (s, bad[:10], err[bad[:10]])


def test_express_prefill_parity_at_the_benchmarked_setting():
    """The masked-prefill benchmark's setting (n_out = 256, mbar = 6 = h - 2,
    65536 points, d = 128, bf16) on two slices, every point's output: the
    1024-point Halve phases, the Compress2 depths batched per level, Subsample
    above mbar and attention over n_out = 256 caches."""
    w = W.custom("pf", B=1, H=2, n=65536, d=128, dtype="bf16", kind="gauss", seed=21)
    n_out, mbar = 256, 6
    Q, K, V = W.make_qkv(w)
    plan = thin_express_plan(w.B, w.H, w.d, n_out, mbar, w.n)
    U = W.make_uniforms(w, w.S * plan["uniforms_per_slice"])
    draws = torch.from_numpy(np.random.default_rng(8).random(
        max(plan["subsample_draws"], 1)).astype(np.float32))
    _check_prefill(w, Q, K, V, U, n_out, mbar, "kh", draws, range(w.S))
