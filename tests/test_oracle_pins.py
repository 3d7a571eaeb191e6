"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle by a route other than its own formulas: a worked
example derived by hand, explicit RKHS feature maps, closed forms of the
level structure, library routines and invariants.  All CPU-only.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# Kernel halving
# ---------------------------------------------------------------------------
def test_kh_worked_example_golden():
    """Hand-derived KH example (App. A, Algorithm A.1 under eq. katt, delta=1/2)."""
    with open(os.path.join(GOLDEN, "kh_worked_example.json")) as f:
        ex = json.load(f)
    K = np.array(ex["K"])[:, None]
    V = np.array(ex["V"])[:, None]
    rows = np.arange(4)
    for case in ex["cases"]:
        r = oracle.kernel_halving(K, V, rows, np.array(case["u"], np.float32))
        assert list(r["out"]) == case["out"], case
        assert r["alpha"][0] == 0.0
        ratio = r["alpha"][1] / r["thresh"][1]
        want = ex["ratio_after_swap"] if case["u"][0] < 0.5 else ex["ratio_after_no_swap"]
        assert ratio == pytest.approx(want, rel=1e-13)


def test_kh_size2_bucket_is_a_fair_coin():
    """N = 2: no earlier points, alpha = 0, p = 1/2 -> keep the second iff u < 1/2."""
    rng = np.random.default_rng(0)
    K = rng.standard_normal((2, 8))
    V = rng.standard_normal((2, 8))
    for u in [0.0, 0.1, 0.49999997, 0.5, 0.7, 1 - 2 ** -24]:
        r = oracle.kernel_halving(K, V, [0, 1], np.array([u], np.float32))
        assert r["alpha"][0] == 0.0
        assert r["out"][0] == (1 if np.float32(u) < 0.5 else 0)


def test_kh_first_pair_of_any_bucket_has_zero_score():
    rng = np.random.default_rng(1)
    K = rng.standard_normal((32, 4))
    V = rng.standard_normal((32, 4))
    u = rng.random(16).astype(np.float32)
    r = oracle.kernel_halving(K, V, np.arange(32), u)
    assert r["alpha"][0] == 0.0
    assert np.all(r["alpha"][1:] != 0.0)


@pytest.mark.parametrize("N", [2, 4, 10, 64])
def test_kh_output_is_one_of_each_pair(N):
    rng = np.random.default_rng(N)
    K = rng.standard_normal((N, 3))
    V = rng.standard_normal((N, 3))
    rows = np.sort(rng.choice(1000, size=N, replace=False)).astype(np.int32)
    Kf = np.zeros((1000, 3)); Kf[rows] = K
    Vf = np.zeros((1000, 3)); Vf[rows] = V
    r = oracle.kernel_halving(Kf, Vf, rows, rng.random(N // 2).astype(np.float32),
                              vmax2_value=float(np.abs(V).max() ** 2))
    out = r["out"]
    assert out.size == N // 2                       # Def. 1: halving keeps floor(N/2)
    for i in range(N // 2):
        assert out[i] in (rows[2 * i], rows[2 * i + 1])
    assert np.all(np.diff(out) > 0)


def _kh_feature_space(Phi, u, delta=0.5):
    """KH in an explicit feature space: alpha_i = <psi, f_i>, b_i = ||f_i||,
    psi = sum_{S2} phi - sum_{S1} phi (the RKHS form of App. A's score)."""
    N = Phi.shape[0]
    psi = np.zeros(Phi.shape[1])
    bmax = 0.0
    c = 0.5 + math.log(2 * N / delta)
    out, alphas, ths = [], [], []
    for i in range(N // 2):
        x, xp = 2 * i, 2 * i + 1
        f = Phi[x] - Phi[xp]
        b = math.sqrt(max(float(f @ f), 0.0))
        bmax = max(bmax, b)
        a = b * bmax * c
        alpha = float(psi @ f)
        p = 0.5 if a == 0 else min(1.0, max(0.0, 0.5 * (1 - alpha / a)))
        swap = float(u[i]) < p
        s1, s2 = (xp, x) if swap else (x, xp)
        psi += Phi[s2] - Phi[s1]
        out.append(s1)
        alphas.append(alpha)
        ths.append(a)
    return np.array(out), np.array(alphas), np.array(ths)


def test_kh_linear_kernel_matches_feature_space():
    rng = np.random.default_rng(2)
    N, d = 40, 3
    K = rng.standard_normal((N, d))
    V = rng.standard_normal((N, d))
    u = rng.random(N // 2).astype(np.float32)
    r = oracle.kernel_halving(K, V, np.arange(N), u, kernel="linear")
    out, al, th = _kh_feature_space(np.hstack([K, V]), u)
    assert np.array_equal(r["out"], out)
    np.testing.assert_allclose(r["alpha"], al, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(r["thresh"], th, rtol=1e-12)


def _katt_features(K, V, vmax, terms):
    """Explicit features of kappa_att (eq. katt): the exponential factor by its
    Taylor series over tensor powers, the value factor by [v, v_max]."""
    N, d = K.shape
    blocks = []
    for n in range(terms):
        scale = 1.0 / math.sqrt(math.factorial(n) * d ** (n / 2))
        t = np.ones((N, 1))
        for _ in range(n):
            t = (t[:, :, None] * K[:, None, :]).reshape(N, -1)
        blocks.append(t * scale)
    fk = np.hstack(blocks)
    fv = np.hstack([V, np.full((N, 1), vmax)])
    return (fk[:, :, None] * fv[:, None, :]).reshape(N, -1)


@pytest.mark.parametrize("d,terms,N", [(1, 40, 24), (2, 15, 12)])
def test_kh_katt_matches_feature_space(d, terms, N):
    rng = np.random.default_rng(3 + d)
    K = rng.uniform(-0.8, 0.8, size=(N, d))
    V = rng.standard_normal((N, d))
    vmax = float(np.abs(V).max())
    u = rng.random(N // 2).astype(np.float32)
    r = oracle.kernel_halving(K, V, np.arange(N), u)
    out, al, th = _kh_feature_space(_katt_features(K, V, vmax, terms), u)
    assert np.array_equal(r["out"], out)
    np.testing.assert_allclose(r["alpha"], al, rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(r["thresh"], th, rtol=1e-12)


def test_kh_incremental_pair_scores_match_literal_sums():
    """The pair-score recursion the GPU uses (alpha_p += sgn_i E(i,p)) agrees
    with the literal double sums of App. A, Algorithm A.1."""
    rng = np.random.default_rng(5)
    N, d = 64, 6
    K = rng.standard_normal((N, d)) * 0.6
    V = rng.standard_normal((N, d))
    vm2 = float(np.abs(V).max() ** 2)
    u = rng.random(N // 2).astype(np.float32)
    G = np.exp(K @ K.T / math.sqrt(d)) * (V @ V.T + vm2)
    r = oracle.kernel_halving(K, V, np.arange(N), u)
    P = N // 2
    alpha = np.zeros(P)
    for i in range(P):
        x, xp = 2 * i, 2 * i + 1
        np.testing.assert_allclose(alpha[i], r["alpha"][i], rtol=1e-10, atol=1e-9)
        sgn = -1.0 if r["bits"][i] else 1.0
        for p in range(i + 1, P):
            y, yp = 2 * p, 2 * p + 1
            E = G[xp, y] - G[x, y] - G[xp, yp] + G[x, yp]
            alpha[p] += sgn * E


def _mmd2(G, keep):
    N = G.shape[0]
    w = np.full(N, 1.0 / N)
    w[keep] -= 2.0 / N
    return float(w @ G @ w)


def test_kh_balances_far_better_than_uniform_halving():
    """Sec. 2.1: KH balances the two halves far better than uniform halving.
    In one dimension with the linear kernel the signed sum psi = sum_S2 x -
    sum_S1 x is a self-balancing walk; a wrong sign anywhere in the score or
    the swap rule turns it into an anti-balancing walk."""
    rng = np.random.default_rng(6)
    N = 1024
    kh, uni = [], []
    for _ in range(20):
        K = rng.standard_normal((N, 1))
        V = np.zeros((N, 1))
        u = rng.random(N // 2).astype(np.float32)
        out = oracle.kernel_halving(K, V, np.arange(N), u, kernel="linear")["out"]
        w = np.ones(N)
        w[out] -= 2.0
        kh.append(float(w @ K[:, 0]) ** 2)
        keep = np.arange(0, N, 2) + (rng.random(N // 2) < 0.5)
        w = np.ones(N)
        w[keep] -= 2.0
        uni.append(float(w @ K[:, 0]) ** 2)
    assert np.mean(kh) * 10 < np.mean(uni)


def test_kh_katt_coreset_beats_uniform_halving_on_average():
    rng = np.random.default_rng(6)
    N, d = 512, 2
    kh, uni = [], []
    for _ in range(20):
        K = rng.standard_normal((N, d)) * 0.5
        V = rng.standard_normal((N, d))
        vm2 = float(np.abs(V).max() ** 2)
        G = np.exp(K @ K.T / math.sqrt(d)) * (V @ V.T + vm2)
        u = rng.random(N // 2).astype(np.float32)
        kh.append(_mmd2(G, oracle.kernel_halving(K, V, np.arange(N), u)["out"]))
        uni.append(_mmd2(G, np.arange(0, N, 2) + (rng.random(N // 2) < 0.5)))
    assert np.mean(kh) * 1.5 < np.mean(uni)


def test_kh_value_scaling_leaves_decisions_unchanged():
    """V -> cV multiplies every kappa_att value by c^2 (v_max scales too), so
    every ratio alpha/a and hence every decision is unchanged."""
    rng = np.random.default_rng(7)
    N, d = 48, 5
    K = rng.standard_normal((N, d))
    V = rng.standard_normal((N, d))
    u = rng.random(N // 2).astype(np.float32)
    r1 = oracle.kernel_halving(K, V, np.arange(N), u)
    r2 = oracle.kernel_halving(K, 4.0 * V, np.arange(N), u)
    assert np.array_equal(r1["out"], r2["out"])
    np.testing.assert_allclose(r2["alpha"], 16 * r1["alpha"], rtol=1e-12, atol=1e-300)


# ---------------------------------------------------------------------------
# Alternative halving (uniform) and KH's delta
# ---------------------------------------------------------------------------
def test_uniform_halving_is_kh_where_every_threshold_is_zero():
    """Identical rows give b_i = 0, hence a_i = 0, and KH takes p = 1/2: it
    then is uniform halving, decision for decision.  Ties the uniform rule to
    KH's own a = 0 case (App. A), through a whole compress."""
    rng = np.random.default_rng(11)
    n, d, n_out, g = 256, 4, 8, 2
    K = np.tile(rng.standard_normal((1, d)), (n, 1))
    V = np.tile(rng.standard_normal((1, d)), (n, 1))
    pl = oracle.plan(n, n_out, g)
    U = (rng.integers(0, 1 << 24, pl["uniforms"]) * 2.0 ** -24).astype(np.float32)
    kh = oracle.compress(K, V, n_out, g, U)
    un = oracle.compress(K, V, n_out, g, U, halve="uniform")
    assert kh["stats"]["zero_threshold"] == pl["uniforms"]
    assert np.array_equal(kh["idx"], un["idx"])
    assert np.array_equal(kh["bits"], un["bits"])


def test_uniform_halving_keeps_each_row_of_a_pair_half_the_time():
    rng = np.random.default_rng(12)
    rows = rng.permutation(4096).astype(np.int32)
    u = rng.random(2048).astype(np.float32)
    r = oracle.uniform_halving(rows, u)
    pairs = rows.reshape(-1, 2)
    assert np.all((r["out"] == pairs[:, 0]) | (r["out"] == pairs[:, 1]))
    assert abs(r["bits"].mean() - 0.5) < 0.05


def test_kh_delta_scales_every_threshold_by_the_log_term():
    """a_i = b_i b_max (1/2 + log(2N/delta)): delta enters through one factor
    common to every pair of the call; alpha does not depend on it."""
    rng = np.random.default_rng(13)
    N, d = 64, 3
    K = rng.standard_normal((N, d)) * 0.5
    V = rng.standard_normal((N, d))
    u = rng.random(N // 2).astype(np.float32)
    r0 = oracle.kernel_halving(K, V, np.arange(N), u, delta=0.5)
    for delta in (1e-6, 0.05, 1.0):
        r = oracle.kernel_halving(K, V, np.arange(N), u, delta=delta)
        ratio = (0.5 + math.log(2 * N / delta)) / (0.5 + math.log(4 * N))
        pos = r0["thresh"] > 0
        np.testing.assert_allclose(r["thresh"][pos] / r0["thresh"][pos], ratio, rtol=1e-12)
        # alpha sums the scores of the earlier pairs, whose decisions may differ
        assert r["alpha"][0] == r0["alpha"][0] == 0.0


def test_compress_with_delta_half_every_round_is_the_default():
    rng = np.random.default_rng(14)
    n, d, n_out, g = 512, 4, 16, 2
    K = rng.standard_normal((n, d)) * 0.7
    V = rng.standard_normal((n, d))
    pl = oracle.plan(n, n_out, g)
    U = (rng.integers(0, 1 << 24, pl["uniforms"]) * 2.0 ** -24).astype(np.float32)
    a = oracle.compress(K, V, n_out, g, U)
    b = oracle.compress(K, V, n_out, g, U, delta=[0.5] * pl["rounds"])
    assert np.array_equal(a["idx"], b["idx"]) and np.array_equal(a["bits"], b["bits"])


# ---------------------------------------------------------------------------
# Compress level structure
# ---------------------------------------------------------------------------
def test_plan_uniform_counts_for_the_five_workloads():
    # n_kept - n_out halving draws, plus n_kept subsample draws when n_kept < n
    assert oracle.plan(1024, 32, 2)["uniforms"] == 992
    assert oracle.plan(3136, 64, 2)["uniforms"] == 2048 + 1984
    assert oracle.plan(1024, 64, 3)["uniforms"] == 960
    assert oracle.plan(16384, 128, 3)["uniforms"] == 16256
    assert oracle.plan(65536, 256, 4)["uniforms"] == 65280


def _bucket_sizes_from_trace(res, n_kept, n_out, subsample):
    """Bucket boundaries are where the score is exactly zero (first pair of a
    KH call): there rho = 0 - (1 - 2u) exactly."""
    U = res["U"]
    rho = res["rho"]
    off = n_kept if subsample else 0
    rounds = []
    n_r = n_kept
    while n_r > n_out:
        seg = slice(off, off + n_r // 2)
        zero = rho[seg] == 0.0 - (1.0 - 2.0 * U[seg].astype(np.float64))
        starts = np.flatnonzero(zero)
        sizes = 2 * np.diff(np.append(starts, n_r // 2))
        rounds.append(list(sizes))
        off += n_r // 2
        n_r //= 2
    return rounds


def _run_compress(n, n_out, g, d=3, seed=0):
    rng = np.random.default_rng(seed)
    K = rng.standard_normal((n, d))
    V = rng.standard_normal((n, d))
    pl = oracle.plan(n, n_out, g)
    U = rng.random(pl["uniforms"]).astype(np.float32)
    res = oracle.compress(K, V, n_out, g, U)
    res["U"] = U
    return res, pl


def test_compress2_bucket_counts_match_theorem1_runtime_sum():
    """Thm 1: Compress2(m, 2^m n_out) runs 4^j Halve calls on 2^(1-j) n_out
    points, j = 0..m-1 (g = 0: no trailing halvings)."""
    m, n_out = 3, 16
    res, pl = _run_compress(n_out * 2 ** m, n_out, 0)
    rounds = _bucket_sizes_from_trace(res, pl["n_kept"], n_out, False)
    got = sorted(s for r in rounds for s in r)
    want = sorted([int(2 ** (1 - j) * n_out) for j in range(m) for _ in range(4 ** j)])
    assert got == want


def _shetty_compress_calls(n, g):
    """Halving-call sizes of Compress with oversampling g (base case 4^g
    points returned as they are), followed by g halvings to sqrt(n)."""
    calls = []

    def comp(size):
        if size <= 4 ** g:
            return size
        out = sum(comp(size // 4) for _ in range(4))
        calls.append(out)
        return out // 2

    top = comp(n)
    while top > math.isqrt(n):
        calls.append(top)
        top //= 2
    return calls


@pytest.mark.parametrize("k,g", [(5, 2), (4, 1), (5, 0), (3, 3), (6, 2)])
def test_compress_matches_recursive_compress_with_oversampling(k, g):
    n = 4 ** k
    n_out = 2 ** k
    res, pl = _run_compress(n, n_out, g, seed=k + g)
    rounds = _bucket_sizes_from_trace(res, n, n_out, False)
    got = sorted(s for r in rounds for s in r)
    assert got == sorted(_shetty_compress_calls(n, g))
    if g < k:
        assert rounds[0][0] == 4 ** (g + 1)


def test_compress_output_size_order_and_identity_case():
    res, _ = _run_compress(3000, 40, 2)
    idx = res["idx"]
    assert idx.size == 40 and np.all(np.diff(idx) > 0) and idx.min() >= 0 and idx.max() < 3000
    res, pl = _run_compress(96, 96, 3)
    assert pl["rounds"] == 0 and np.array_equal(res["idx"], np.arange(96))


def test_plan_rejects_buckets_below_two_rows():
    assert oracle.plan(1024, 1, 0) is None       # 4^9 groups of a 1024-row input
    assert oracle.plan(10, 11, 1) is None
    assert oracle.plan(1024, 1, 4) is None       # groups of one row
    assert oracle.plan(1024, 1, 5) is not None   # groups of four rows


# ---------------------------------------------------------------------------
# Stratified subsample
# ---------------------------------------------------------------------------
def test_subsample_equal_groups_is_offline_subsample():
    """Algorithm H.1: one uniform draw from each group of 2^k consecutive points."""
    rng = np.random.default_rng(8)
    n_kept, k = 100, 3
    u = rng.integers(0, 2 ** 24, size=n_kept) * 2.0 ** -24
    out = oracle.subsample(n_kept * 2 ** k, n_kept, u.astype(np.float32))
    t = np.arange(n_kept)
    assert np.array_equal(out, t * 2 ** k + np.floor(u * 2 ** k).astype(np.int64))


def test_subsample_unequal_strata_cover_and_are_uniform():
    n, n_kept = 3136, 2048
    u = np.zeros(n_kept, np.float32)
    lo = oracle.subsample(n, n_kept, u)
    hi = oracle.subsample(n, n_kept, np.full(n_kept, 1 - 2 ** -24, np.float32))
    # first/last element of each stratum; strata tile [0, n)
    assert lo[0] == 0 and hi[-1] == n - 1
    assert np.array_equal(lo[1:], hi[:-1] + 1)
    assert set(np.unique(hi - lo + 1)) == {1, 2}
    # uniformity within a stratum of length 2: half of the u-grid picks each
    grid = (np.arange(1 << 12) * 2.0 ** -12).astype(np.float32)
    s = int(np.flatnonzero(hi - lo == 1)[0])
    picks = [oracle.subsample(n, n_kept, np.full(n_kept, g, np.float32))[s] for g in grid[::64]]
    assert np.bincount(np.array(picks) - lo[s]).tolist() == [32, 32]


def test_vmax2_is_max_abs_squared():
    rng = np.random.default_rng(9)
    V = rng.standard_normal((77, 13))
    assert oracle.vmax2(V) == np.abs(V).max() ** 2


# ---------------------------------------------------------------------------
# Attention
# ---------------------------------------------------------------------------
def test_exact_attention_matches_library_sdpa():
    rng = np.random.default_rng(10)
    Q = rng.standard_normal((37, 16))
    K = rng.standard_normal((53, 16))
    V = rng.standard_normal((53, 16))
    O = oracle.exact_attention(Q, K, V)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(Q)[None], torch.from_numpy(K)[None], torch.from_numpy(V)[None])[0]
    np.testing.assert_allclose(O, ref.numpy(), rtol=1e-12, atol=1e-13)


def test_attention_over_one_key_returns_its_value():
    rng = np.random.default_rng(11)
    Q = rng.standard_normal((5, 8)) * 10
    K = rng.standard_normal((9, 8))
    V = rng.standard_normal((9, 8))
    O = oracle.attention(Q, K, V, [4])
    assert np.array_equal(O, np.repeat(V[4:5], 5, axis=0))


def test_attention_invariant_to_a_common_key_shift():
    rng = np.random.default_rng(12)
    Q = rng.standard_normal((6, 8))
    K = rng.standard_normal((20, 8))
    V = rng.standard_normal((20, 8))
    rows = [1, 3, 4, 9, 15]
    O1 = oracle.attention(Q, K, V, rows)
    O2 = oracle.attention(Q, K + rng.standard_normal(8) * 3, V, rows)
    np.testing.assert_allclose(O1, O2, rtol=1e-11, atol=1e-12)


def test_thinned_attention_with_nout_equal_n_is_exact_attention():
    rng = np.random.default_rng(13)
    n, d = 64, 8
    Q, K, V = (rng.standard_normal((n, d)) for _ in range(3))
    res = oracle.compress(K, V, n, 2, np.zeros(1, np.float32))
    assert np.array_equal(oracle.attention(Q, K, V, res["idx"]), oracle.exact_attention(Q, K, V))


def test_attention_value_scaling_is_linear():
    rng = np.random.default_rng(14)
    Q, K, V = (rng.standard_normal((30, 8)) for _ in range(3))
    rows = np.arange(0, 30, 3)
    np.testing.assert_array_equal(oracle.attention(Q, K, 2 * V, rows),
                                  2 * oracle.attention(Q, K, V, rows))


# ---------------------------------------------------------------------------
# Weighted attention (eq. def:att_approx) and exact sink / window rows
# ---------------------------------------------------------------------------
def test_weighted_attention_matches_library_sdpa_with_an_additive_mask():
    """exp(logw_j) * exp(s_j) = exp(s_j + logw_j): the log-weights are the float
    mask SDPA adds to the scaled scores (including -inf, a dropped key)."""
    rng = np.random.default_rng(20)
    Q = rng.standard_normal((23, 16))
    K = rng.standard_normal((41, 16))
    V = rng.standard_normal((41, 16))
    rows = rng.permutation(41)[:29].astype(np.int32)
    logw = rng.standard_normal(29) * 2
    logw[[3, 17]] = -np.inf
    O = oracle.weighted_attention(Q, K, V, rows, logw)
    mask = torch.from_numpy(np.broadcast_to(logw, (23, 29)).copy())
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(Q)[None], torch.from_numpy(K[rows])[None],
        torch.from_numpy(V[rows])[None], attn_mask=mask[None])[0]
    np.testing.assert_allclose(O, ref.numpy(), rtol=1e-12, atol=1e-13)


def test_weighted_attention_with_equal_weights_is_attention():
    rng = np.random.default_rng(21)
    Q, K, V = (rng.standard_normal((30, 8)) for _ in range(3))
    rows = np.arange(1, 30, 2)
    O = oracle.weighted_attention(Q, K, V, rows, np.full(rows.size, 3.7))
    np.testing.assert_allclose(O, oracle.attention(Q, K, V, rows), rtol=1e-12, atol=1e-13)


def test_integer_weight_is_a_repeated_key():
    """Weight k on a key = that key listed k times with weight 1."""
    rng = np.random.default_rng(22)
    Q, K, V = (rng.standard_normal((12, 8)) for _ in range(3))
    rows = np.array([2, 5, 7, 11])
    mult = np.array([1, 3, 1, 5])
    O = oracle.weighted_attention(Q, K, V, rows, np.log(mult))
    np.testing.assert_allclose(O, oracle.attention(Q, K, V, np.repeat(rows, mult)),
                               rtol=1e-12, atol=1e-13)


def test_minus_inf_weight_drops_the_key():
    rng = np.random.default_rng(23)
    Q, K, V = (rng.standard_normal((12, 8)) for _ in range(3))
    rows = np.array([0, 4, 6, 9, 10])
    logw = np.array([0.0, -np.inf, 0.0, -np.inf, 0.0])
    np.testing.assert_array_equal(oracle.weighted_attention(Q, K, V, rows, logw),
                                  oracle.attention(Q, K, V, rows[np.isfinite(logw)]))


def test_sinks_and_window_are_exact_and_the_weights_sum_to_n():
    rng = np.random.default_rng(24)
    n, d, ns, nw, n_out, g = 300, 8, 20, 24, 16, 1
    K, V = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    pl = oracle.plan(n - ns - nw, n_out, g)
    U = rng.random(pl["uniforms"]).astype(np.float32)
    r = oracle.compress(K, V, n_out, g, U, n_sinks=ns, n_window=nw)
    idx, logw = r["idx"], r["logw"]
    assert idx.size == ns + n_out + nw == logw.size
    assert np.array_equal(idx[:ns], np.arange(ns))
    assert np.array_equal(idx[ns + n_out:], np.arange(n - nw, n))
    core = idx[ns:ns + n_out]
    assert core.min() >= ns and core.max() < n - nw and np.unique(core).size == n_out
    assert np.all(logw[:ns] == 0) and np.all(logw[ns + n_out:] == 0)
    assert np.exp(logw).sum() == pytest.approx(n, rel=1e-12)
    # the middle rows are a dataset of their own: thinning them alone gives the same coreset
    mid = oracle.compress(K[ns:n - nw], V[ns:n - nw], n_out, g, U)
    assert np.array_equal(core, mid["idx"] + ns)


def test_sinks_and_window_with_nothing_to_thin_is_exact_attention():
    """n - n_sinks - n_window = n_out: every row is kept with weight 1."""
    rng = np.random.default_rng(25)
    n, d, ns, nw = 48, 8, 8, 8
    Q, K, V = (rng.standard_normal((n, d)) for _ in range(3))
    r = oracle.compress(K, V, n - ns - nw, 1, np.zeros(1, np.float32), n_sinks=ns, n_window=nw)
    assert np.array_equal(r["idx"], np.arange(n)) and np.all(r["logw"] == 0)
    np.testing.assert_allclose(oracle.weighted_attention(Q, K, V, r["idx"], r["logw"]),
                               oracle.exact_attention(Q, K, V), rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------------------------
# Express (Alg. 1 / 2) and Thinformer decoding (Alg. 4 / 5)
# ---------------------------------------------------------------------------
def _express_inputs(n, d, seed):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((n, d)) for _ in range(3))


def test_thinformer_is_exact_for_the_first_four_n_out_points():
    """The accuracy theorem of Sec. 4: outputs equal exact causal attention
    for every n <= 4 n_out (no point is thinned before the first Halve phase)."""
    n_out, n, d = 8, 32, 8
    Q, K, V = _express_inputs(n, d, 30)
    U = np.random.default_rng(31).random(max(oracle.express_uniforms(n, n_out, 2), 1))
    r = oracle.express_decode(Q, K, V, n_out, 2, U.astype(np.float32))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(Q)[None], torch.from_numpy(K)[None], torch.from_numpy(V)[None],
        is_causal=True)[0].numpy()
    np.testing.assert_allclose(r["O"], ref, rtol=1e-12, atol=1e-13)
    assert r["m"] == 2 and r["idx"].size == n_out  # the cache right after the first Halve phase


@pytest.mark.parametrize("n", [1, 7, 8, 9, 31, 33, 100, 128, 129, 200, 511, 512])
def test_express_cache_weights_count_every_point(n):
    """A cache point of C_i stands for 2^i points and one of E for 2^m, so
    2^m * sum of the weights is the number of points seen (no subsampling
    up to 512 points at mbar = 4)."""
    n_out, mbar, d = 8, 4, 4
    Q, K, V = _express_inputs(n, d, 32)
    U = np.random.default_rng(33).random(max(oracle.express_uniforms(n, n_out, mbar), 1))
    r = oracle.express_decode(Q, K, V, n_out, mbar, U.astype(np.float32), outputs=False)
    assert np.exp(r["logw"]).sum() * 2.0 ** r["m"] == pytest.approx(n, rel=1e-12)
    assert r["idx"].size <= 6 * n_out  # Thm. 1: cache size at most 6 n_out
    assert np.unique(r["idx"]).size == r["idx"].size and (r["idx"].size == 0 or r["idx"].max() < n)


def _keep_first(rows):
    return rows[0::2]


def _offline_compress2(m, rows):
    """Offline Compress2 (App. H): 4^(m-1) groups halved, then recurse on m - 1."""
    if m == 0:
        return rows
    g = 4 ** (m - 1)
    size = rows.size // g
    return _offline_compress2(m - 1, np.concatenate(
        [_keep_first(rows[k * size:(k + 1) * size]) for k in range(g)]))


def _offline_subsample(m, mbar, rows, draws):
    """Offline Subsample: one point of every 2^(m - mbar), at offset floor(u R)."""
    if m <= mbar:
        return rows
    R = 2 ** (m - mbar)
    return np.array([rows[k + min(R - 1, int(np.floor(next(draws) * R)))]
                     for k in range(0, rows.size, R)], dtype=rows.dtype)


def _offline_express(n_out, mbar, rows, m, draws):
    """Offline-Express (App. H, Algorithm H.3, the recursive procedure) on 2^(m+2) n_out points;
    the draws are taken in the order the recursion meets the strata."""
    if rows.size <= n_out:
        return rows
    q = rows.size // 4
    parts = [_offline_express(n_out, mbar, rows[:q], m - 2, draws)]
    for j in (1, 2, 3):
        kept = _offline_subsample(m, mbar, rows[j * q:(j + 1) * q], draws)
        parts.append(_offline_compress2(min(m, mbar), kept))
    return _keep_first(_keep_first(np.concatenate(parts)))


@pytest.mark.parametrize("n_out,mbar,levels", [(4, 2, 2), (8, 4, 3), (16, 6, 3), (16, 4, 2),
                                               (4, 2, 3), (8, 2, 4), (16, 3, 4)])
def test_streaming_express_equals_offline_express(n_out, mbar, levels):
    """The streaming procedure equals the recursive offline one (App. H, Algorithm H.3);
    with a deterministic Halve (uniform halving with every u >= 1/2 keeps
    the first point of each pair) and the same Subsample draws (levels above
    mbar) both must return the same coreset."""
    m = 2 * levels - 2
    n = n_out * 2 ** (m + 2)
    Q, K, V = _express_inputs(n, 2, 34)
    U = np.full(max(oracle.express_uniforms(n, n_out, mbar), 1), 0.75, np.float32)
    nd = oracle.express_draws(n, n_out, mbar)
    draws = (np.random.default_rng(35).integers(0, 1 << 24, max(nd, 1)) * 2.0 ** -24)
    draws = draws.astype(np.float32)
    r = oracle.express_decode(Q, K, V, n_out, mbar, U, halve="uniform", outputs=False,
                              sub_u=draws)
    want = _offline_express(n_out, mbar, np.arange(n, dtype=np.int32), m,
                            iter(draws.astype(np.float64)))
    assert r["m"] == m + 2 and np.array_equal(r["idx"], want)
    assert (m <= mbar) == (nd == 0)


def test_cor2_delta_schedule_meets_the_union_bound():
    """Cor. 2's budgets: the level budgets delta_m telescope to at most delta/2,
    and within level m the two Halve-phase calls and the Compress2 calls
    (4^(m^mbar - i) calls at depth i per group, 3 groups, weighted 3/8 as in
    the theorem) add up to exactly delta_m."""
    delta, mbar = 0.5, 6
    tot = 0.0
    for m in range(0, 40, 2):
        dm = 2 * oracle.express_delta(m, -1, mbar, delta)
        tot += dm
        if m == 0:
            continue
        mp = min(m, mbar)
        s = dm / 2 + 3 / 8 * sum(4 ** (mp - i) * oracle.express_delta(m, i, mbar, delta)
                                 for i in range(mp))
        assert s == pytest.approx(dm, rel=1e-12)
    K = 19
    assert tot == pytest.approx(delta / 2 * (1 - 1 / math.log2(K + 3)), rel=1e-12)
    assert tot < delta / 2


def test_express_subsample_cache_weights_count_whole_strata():
    """Above mbar a kept point stands for its stratum of 2^(m - mbar) points:
    at the end of every level (all strata complete) 2^m * the weight sum
    counts every point, and the cache stays within 6 n_out."""
    n_out, mbar, d = 8, 2, 4
    for levels in (3, 4):
        n = n_out * 4 ** levels
        Q, K, V = _express_inputs(n, d, 36)
        U = np.random.default_rng(37).random(oracle.express_uniforms(n, n_out, mbar))
        nd = oracle.express_draws(n, n_out, mbar)
        draws = np.random.default_rng(38).random(nd).astype(np.float32)
        r = oracle.express_decode(Q, K, V, n_out, mbar, U.astype(np.float32), outputs=False,
                                  sub_u=draws)
        assert np.exp(r["logw"]).sum() * 2.0 ** r["m"] == pytest.approx(n, rel=1e-12)
        assert r["idx"].size == n_out and np.unique(r["idx"]).size == n_out


def _wtd_attention_cost(n, n_out, mbar):
    """App. G, proposition "Cost of WtdAttention" (eq. streaming_express_query),
    in keys (the d factor common to every term dropped): the keys summed over
    the first n queries of Thinformer decoding, m_n = 2 ceil(log4(n / (4 n_out)))."""
    if n <= 4 * n_out:
        return n * (n + 1) // 2
    mn, q = 0, 4 * n_out
    while q < n:
        q *= 4
        mn += 2
    base = 2 * n_out * (4 * n_out + 1)
    if mn <= mbar:
        return base + (7 * n_out * n_out - n_out) * (2 ** (mn + 2) - 4) // 2 \
            - 3 * (mn // 2) * n_out * n_out
    return base + 6 * n_out * (n - 4 * n_out)


@pytest.mark.parametrize("n_out,mbar", [(4, 2), (8, 2), (8, 4), (16, 4), (16, 5), (32, 3), (32, 6)])
def test_wtd_attention_query_cost_proposition(n_out, mbar):
    """The oracle's per-point key counts against App. G's proposition.  Its
    proof counts a thin-phase query's cache without the query's own key (the
    exact phase counts it), while WtdAttention (Alg. 5) adds the query to C_0,
    so with the query counted the sum is the proposition's value plus one per
    thin-phase point: equal in the exact phase and at every level end
    n = n_out 4^k with m_n <= mbar (the proposition's endpoints), below it
    elsewhere; at most the cache bound 6 n_out (+ the query) once m_n > mbar."""
    n_max = n_out * 4 ** (mbar // 2 + 2)
    keys = oracle.express_keys(n_max, n_out, mbar)
    cum = np.concatenate([[0], np.cumsum(keys)])
    assert np.all(keys <= 6 * n_out + 1)
    ends = 0
    for n in range(1, n_max + 1):
        bound = _wtd_attention_cost(n, n_out, mbar) + max(n - 4 * n_out, 0)
        assert cum[n] <= bound, (n, cum[n], bound)
        if n <= 4 * n_out:
            assert cum[n] == n * (n + 1) // 2
        k = round(math.log(n / n_out, 4)) if n >= n_out else -1
        if k >= 2 and n == n_out * 4 ** k and 2 * k - 2 <= mbar:
            assert cum[n] == bound, (n, cum[n], bound)
            ends += 1
    assert ends >= 1
