"""Benchmark of the thinning hot path on one MI355X.

One step = thin_compress (v_max scan + every kernel-halving round: pair
scores, then decisions) + thin_attention (fp32 output) over one batch of the
long-sequence workload (B=4, H=16, n=16384 keys and queries, d=128, bf16,
n_out=128, g=3), inputs resident in HBM.  The K timed steps run with nothing
between kernels; the same K steps then run again with every kernel launch
bracketed by HIP events on its stream (thin_set_launch_hook), which gives the
per-kernel times and the roofline figures.  Prints one JSON line.

  python bench.py [--gpus 1] [--steps 20] [--warmup 100] [--workload long]
                  [--no-cpu-baseline] [--halve kh|uniform] [--sinks S --window W]

With --sinks / --window the first S and last W keys of every slice are kept
exactly, the rows between them are thinned to n_out, and attention runs over
the S + n_out + W weighted keys (eq. def:att_approx).

--mode decode measures Thinformer decoding over the Express cache instead
(Alg. 4): B=1, H=32 slices, d=128, bf16, n_out=128, mbar=5 (log2 n_out - 2,
the decoding experiments' choice: Subsample runs from point 8192 on), 16384
points decoded one at a time (each attends over the cache plus itself, then
enters it); one step = one point of every slice.

--mode prefill measures the masked prefill over the Express cache (every
point's Thinformer output at once): B=1, H=32, d=128, bf16, 65536 points,
n_out=256 (h = 8), mbar=6 (h - 2); one step = one whole prefill.

--mode peaks measures the GPU's own ceilings beside the spec figures the
rooflines use: library GEMM rates (bf16, fp16, fp32) and 1 GiB copy, fill
and read-reduce bandwidth.
"""
import argparse
import collections
import dataclasses
import hashlib
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "thinned-attention (B·H·n)/s incl. Compress; % HBM + MFMA roofline"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_MFMA_PEAK_TFLOPS = 2500.0  # dense
FP32_MFMA_PEAK_TFLOPS = 157.3


def elem_bytes(dtype: str) -> int:
    return 2 if dtype == "bf16" else 4


def compress_bytes(w, plan) -> int:
    """Algorithmic HBM bytes of one compress call: the v_max scan reads V once;
    round r reads the K and V rows of its n_r rows per slice, their int32
    indices (not in round 0 without subsample), one float32 uniform per pair
    and writes n_r/2 int32 indices; the subsample reads n_kept uniforms and
    writes n_kept indices."""
    b = elem_bytes(w.dtype)
    S, n, d = w.S, w.n, w.d
    total = S * n * d * b
    n_kept, L = plan["n_kept"], plan["rounds"]
    sub = n_kept < n
    if sub:
        total += S * n_kept * (4 + 4)
    for r in range(L):
        n_r = n_kept >> r
        total += S * n_r * 2 * d * b
        if r > 0 or sub:
            total += S * n_r * 4
        total += S * (n_r // 2) * (4 + 4)
    return total


def uniform_compress_bytes(w, plan) -> int:
    """Algorithmic HBM bytes of one compress call with uniform halving: the
    subsample (n_kept uniforms read, n_kept indices written), then per slice
    the kept indices read once, one float32 uniform per pair of every round
    and the n_out indices written (no row of K or V is read)."""
    S, n = w.S, w.n
    n_kept, L = plan["n_kept"], plan["rounds"]
    sub = n_kept < n
    total = S * n_kept * (4 + 4 + 4) if sub else 0
    total += S * sum((n_kept >> r) // 2 for r in range(L)) * 4
    total += S * w.n_out * 4
    return total


def kappa_evals(plan, w) -> int:
    """kappa_att evaluations of one compress call: N^2/2 + N/2 per bucket."""
    n_kept, L, g = plan["n_kept"], plan["rounds"], w.g
    tot = 0
    for r in range(L):
        n_r = n_kept >> r
        e = L - g - 1 - r
        G = 4 ** e if e > 0 else 1
        N = n_r // G
        tot += G * (N * N // 2 + N // 2)
    return tot * w.S


def round_bytes(w, plan) -> list:
    """Algorithmic HBM bytes of each Halve round (the per-round term of the
    compress byte model): the round's K and V rows read once and their int32
    indices, S n_r (2 d b + 4)."""
    b = elem_bytes(w.dtype)
    n_kept, L = plan["n_kept"], plan["rounds"]
    return [w.S * (n_kept >> r) * (2 * w.d * b + 4) for r in range(L)]


def score_buffer_bytes(w, plan) -> list:
    """Bytes this design adds to each round's pair-score launch (not part of
    the algorithm): the float32 pair scores written (8 x 32 tiles over each
    64-row block and the columns from its diagonal on) and two float32 pair
    terms per pair; the decision pass reads them back."""
    n_kept, L, g = plan["n_kept"], plan["rounds"], w.g
    out = []
    for r in range(L):
        n_r = n_kept >> r
        e = L - g - 1 - r
        G = 4 ** e if e > 0 else 1
        N = n_r // G
        NT, nb = (N + 15) // 16, (N + 63) // 64
        tiles = nb * NT - 4 * nb * (nb - 1) // 2
        out.append(w.S * (G * tiles * 1024 + (n_r // 2) * 8))
    return out


def kernel_sources_sha256() -> str:
    """Hash of the compress kernels' sources and of the launch sequence (a
    stored traffic measurement is only reported while it matches)."""
    h = hashlib.sha256()
    for f in ("compress.hip", "common.hpp", "launch.hpp", "api.cpp"):
        with open(os.path.join(ROOT, "paper_2606_10944_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def stored_traffic(workload: str):
    """HBM bytes per pair-score launch measured with rocprofv3 counters
    (profiles/pair_scores_<workload>_traffic.md), or None if absent or taken
    on other kernel sources."""
    path = os.path.join(ROOT, "profiles", f"pair_scores_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_sha = re.search(r"^source_sha256:\s*([0-9a-f]{64})", text, re.M)
    m_val = re.search(r"^traffic_bytes_per_launch:\s*([0-9.eE+]+)", text, re.M)
    if not m_sha or not m_val or m_sha.group(1) != kernel_sources_sha256():
        return None
    return float(m_val.group(1))


def attention_bytes(w, out_bytes: int, weighted: bool = False) -> int:
    """Queries read and outputs written once; per coreset key its K and V rows,
    its int32 index and (weighted) its float32 log-weight."""
    b = elem_bytes(w.dtype)
    return w.S * (w.n_q * w.d * (b + out_bytes) + w.n_out * (2 * w.d * b + 4 + 4 * weighted))


def attention_flops(w) -> int:
    return w.S * w.n_q * 4 * w.n_out * w.d


def host_cpu() -> dict:
    """CPU model and logical core count of the host that runs the oracle."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count()
    return {"cpu_model": model, "host_cores": os.cpu_count(), "cores_available": avail}


def cpu_baseline(w, Q, K, V, U, plan, budget_s: float = 20.0, halve: str = "kh",
                 n_sinks: int = 0, n_window: int = 0):
    """The oracle, single-threaded, on as many whole slices as fit the budget."""
    import numpy as np
    import oracle
    oracle.lib()
    Us = U.numpy().reshape(w.S, -1)
    t_used, done = 0.0, 0
    for s in range(w.S):
        b, h = divmod(s, w.H)
        Ks, Vs, Qs = K[b, h], V[b, h], Q[b, h]
        t0 = time.perf_counter()
        if n_sinks or n_window:
            r = oracle.compress(Ks, Vs, w.n_out, w.g, Us[s], halve=halve, n_sinks=n_sinks,
                                n_window=n_window)
            oracle.weighted_attention(Qs, Ks, Vs, r["idx"], r["logw"])
        else:
            r = oracle.compress(Ks, Vs, w.n_out, w.g, Us[s], halve=halve)
            oracle.attention(Qs, Ks, Vs, r["idx"])
        t_used += time.perf_counter() - t0
        done += 1
        if t_used >= budget_s:
            break
    _ = np  # noqa: F841
    return {"value": done * w.n_q / t_used, "unit": "(B·H·n)/s", "cores": 1,
            "kind": "oracle", **host_cpu(),
            "sample": f"{done} of {w.S} slices of the {w.name} workload (compress + "
                      f"attention of all {w.n_q} queries per slice), float64, one thread, "
                      f"{t_used:.1f} s"}


DECODE = dict(B=1, H=32, d=128, dtype="bf16", n_out=128, mbar=5, n=16384)


def decode_main(args):
    """Thinformer decoding over the Express cache (one JSON line)."""
    import numpy as np
    import torch

    from paper_2606_10944_amd import ExpressCache, LaunchTimer, thin_express_plan
    from paper_2606_10944_amd import workloads as W
    c = DECODE
    w = W.custom("decode", B=c["B"], H=c["H"], n=c["n"], d=c["d"], dtype=c["dtype"],
                 kind="heavy_tail")
    Q, K, V = W.make_qkv(w)
    plan = thin_express_plan(w.B, w.H, w.d, c["n_out"], c["mbar"], w.n)
    U = W.make_uniforms(w, w.S * plan["uniforms_per_slice"])
    # Subsample's draws (host, shared by the slices), from their own seeded stream
    draws = torch.from_numpy(np.random.default_rng(w.seed + 1).random(
        max(plan["subsample_draws"], 1)).astype(np.float32))
    dev = torch.device("cuda:0")
    Qd, Kd, Vd, Ud = Q.to(dev), K.to(dev), V.to(dev), U.to(dev)
    Qt = [Qd[:, :, t].contiguous() for t in range(w.n)]
    O = torch.empty((w.B, w.H, w.d), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    def run(n_steps, timer=None, keys=None):
        ex = ExpressCache(w.B, w.H, w.d, c["n_out"], c["mbar"], w.n, dtype=torch.bfloat16)
        for t in range(n_steps):
            if keys is not None:
                keys.append(ex.next_keys())
            ex.step(Qt[t], Kd, Vd, Ud, draws=draws, O=O, stream=stream)
        return ex

    for _ in range(max(args.warmup // 50, 1)):
        run(1024).close()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    ex = run(w.n)
    t1.record(stream)
    torch.cuda.synchronize()
    ex.close()
    ms_total = t0.elapsed_time(t1)
    # per-kernel times over the last 2048 points (where the cache is largest)
    keys = []
    ex = ExpressCache(w.B, w.H, w.d, c["n_out"], c["mbar"], w.n, dtype=torch.bfloat16)
    tail = 2048
    for t in range(w.n - tail):
        ex.step(Qt[t], Kd, Vd, Ud, draws=draws, O=O, stream=stream)
    torch.cuda.synchronize()
    with LaunchTimer(stream, capacity=16 * tail) as lt:
        for t in range(w.n - tail, w.n):
            keys.append(ex.next_keys())
            ex.step(Qt[t], Kd, Vd, Ud, draws=draws, O=O, stream=stream)
        torch.cuda.synchronize()
    ex.close()
    rec = lt.records()
    per = collections.defaultdict(float)
    for name, _, ms in rec:
        per[name] += ms / tail
    att = [ms for name, _, ms in rec if name == "attention"]
    att_ms = statistics.mean(att)
    # algorithmic bytes of one attention launch: per slice the query row, the
    # output row (fp32) and per key its K and V rows, index and log-weight
    kb = elem_bytes(w.dtype)
    att_bytes = w.S * (statistics.mean(keys) * (2 * w.d * kb + 8) + w.d * (kb + 4))
    gbs = att_bytes / (att_ms * 1e-3) / 1e9
    value = w.S * w.n / (ms_total * 1e-3)
    out = {
        "metric": "Thinformer decoding over the Express cache: points/s over B·H slices",
        "value": value, "unit": "points/s", "n_gpus": 1, "steps": w.n, "warmup": args.warmup,
        "ms_per_step": ms_total / w.n, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": "express-decode", "B": w.B, "H": w.H, "n": w.n, "d": w.d,
                   "n_out": c["n_out"], "mbar": c["mbar"], "delta": 0.5, "halve": "kh"},
        "roofline": {
            "kernel": "coreset attention of one query per slice over the weighted cache "
                      "(last 2048 points)",
            "bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": gbs / HBM_PEAK_GBS, "traffic": None,
            "algorithmic_bytes_per_launch": att_bytes, "ms_per_launch": att_ms,
            "mean_keys": statistics.mean(keys)},
        "ms_per_step_by_kernel_last_2048": dict(per),
        "gpu": torch.cuda.get_device_name(0),
    }
    if not args.no_cpu_baseline:
        import oracle
        oracle.lib()
        Us = U.numpy().reshape(w.S, -1)
        t_used, done = 0.0, 0
        for s in range(w.S):
            t_a = time.perf_counter()
            oracle.express_decode(Q[0, s], K[0, s], V[0, s], c["n_out"], c["mbar"], Us[s],
                                  sub_u=draws.numpy())
            t_used += time.perf_counter() - t_a
            done += 1
            if t_used >= 20.0:
                break
        out["cpu_baseline"] = {
            "value": done * w.n / t_used, "unit": "points/s", "cores": 1, "kind": "oracle", **host_cpu(),
            "sample": f"{done} of {w.S} slices decoded over all {w.n} points, float64, one "
                      f"thread, {t_used:.1f} s"}
    _ = np  # noqa: F841
    print(json.dumps(out), flush=True)


PREFILL = dict(B=1, H=32, d=128, dtype="bf16", n_out=256, mbar=6, n=65536)


def prefill_main(args):
    """Masked prefill over the Express cache (one JSON line)."""
    import numpy as np
    import torch

    from paper_2606_10944_amd import LaunchTimer, thin_express_prefill, thin_express_prefill_plan
    from paper_2606_10944_amd import workloads as W
    c = PREFILL
    w = W.custom("prefill", B=c["B"], H=c["H"], n=c["n"], d=c["d"], dtype=c["dtype"],
                 kind="heavy_tail")
    Q, K, V = W.make_qkv(w)
    plan = thin_express_prefill_plan(w.B, w.H, w.n, w.d, c["n_out"], c["mbar"])
    U = W.make_uniforms(w, w.S * plan["uniforms_per_slice"])
    draws = torch.from_numpy(np.random.default_rng(w.seed + 1).random(
        max(plan["subsample_draws"], 1)).astype(np.float32))
    dev = torch.device("cuda:0")
    Qd, Kd, Vd, Ud = Q.to(dev), K.to(dev), V.to(dev), U.to(dev)
    ws = torch.empty(plan["workspace_bytes"], dtype=torch.uint8, device=dev)
    O = torch.empty((w.B, w.H, w.n, w.d), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        thin_express_prefill(Qd, Kd, Vd, c["n_out"], c["mbar"], Ud, draws=draws, O=O,
                             workspace=ws, stream=stream)

    steps, warm = max(args.steps // 4, 3), max(args.warmup // 20, 2)
    for _ in range(warm):
        step()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(steps):
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    with LaunchTimer(stream) as lt:
        step()
        torch.cuda.synchronize()
    per = collections.defaultdict(float)
    for name, _, t in lt.records():
        per[name] += t
    att_ms = per["attention"]
    kb = elem_bytes(w.dtype)
    att_bytes = w.S * (plan["staged_keys"] * 2 * w.d * kb + w.n * w.d * (kb + 4))
    att_flops = 4 * w.d * plan["attention_keys"] * w.S
    gbs = att_bytes / (att_ms * 1e-3) / 1e9
    tfl = att_flops / (att_ms * 1e-3) / 1e12
    out = {
        "metric": "masked prefill over the Express cache: points/s over B·H slices",
        "value": w.S * w.n / (ms * 1e-3), "unit": "points/s", "n_gpus": 1, "steps": steps,
        "warmup": warm, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": "express-prefill", "B": w.B, "H": w.H, "n": w.n, "d": w.d,
                   "n_out": c["n_out"], "mbar": c["mbar"], "delta": 0.5, "halve": "kh"},
        "roofline": {
            "kernel": "prefill_attn_kernel (block-causal weighted attention of every point)",
            "bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": gbs / HBM_PEAK_GBS, "traffic": None, "algorithmic_bytes_per_launch": att_bytes,
            "ms_per_launch": att_ms, "mfma_tflops": tfl,
            "mfma_frac": tfl / BF16_MFMA_PEAK_TFLOPS,
            "keys_per_point": plan["attention_keys"] / w.n},
        "ms_by_kernel": dict(per),
        "gpu": torch.cuda.get_device_name(0),
    }
    if not args.no_cpu_baseline:
        import oracle
        oracle.lib()
        Us = U.numpy().reshape(w.S, -1)
        t_a = time.perf_counter()
        oracle.express_decode(Q[0, 0], K[0, 0], V[0, 0], c["n_out"], c["mbar"], Us[0],
                              sub_u=draws.numpy())
        t_used = time.perf_counter() - t_a
        out["cpu_baseline"] = {
            "value": w.n / t_used, "unit": "points/s", "cores": 1, "kind": "oracle", **host_cpu(),
            "sample": f"1 of {w.S} slices, all {w.n} points, float64, one thread, "
                      f"{t_used:.1f} s"}
    print(json.dumps(out), flush=True)


def peaks_main(args):
    """Measured ceilings of the GPU beside the spec sheet: library GEMMs
    (torch.matmul, hipBLASLt) on square operands and device-wide copy, fill
    and read-reduce over 1 GiB of fp32, each timed with HIP events."""
    import torch
    dev = torch.device("cuda:0")

    def timed(fn, n):
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n * 1e-3

    gemm = {}
    for dt, name in ((torch.bfloat16, "bf16"), (torch.float16, "fp16"), (torch.float32, "fp32")):
        for M in (8192, 16384):
            a = torch.randn(M, M, device=dev, dtype=dt)
            b = torch.randn(M, M, device=dev, dtype=dt)
            t = timed(lambda: torch.matmul(a, b), 10 if M == 16384 else 20)
            gemm[f"{name}_{M}"] = 2 * M ** 3 / t / 1e12
            del a, b
    x = torch.empty(1 << 28, device=dev, dtype=torch.float32)
    y = torch.empty_like(x)
    nb = x.numel() * 4
    bw = {"copy_read_write": 2 * nb / timed(lambda: y.copy_(x), 20) / 1e12,
          "fill_write": nb / timed(lambda: x.fill_(1.0), 20) / 1e12,
          "sum_read": nb / timed(lambda: x.sum(), 20) / 1e12}
    best_bf16 = max(gemm["bf16_8192"], gemm["bf16_16384"])
    print(json.dumps({
        "metric": "measured peaks (library GEMM TFLOP/s, 1 GiB copy/fill/read TB/s)",
        "value": best_bf16, "unit": "TFLOP/s (bf16 GEMM)", "n_gpus": 1,
        "higher_is_better": True, "vs_baseline": None, "data": "synthetic",
        "gemm_tflops": gemm, "bandwidth_tbs": bw,
        "spec": {"bf16_dense_tflops": BF16_MFMA_PEAK_TFLOPS, "fp32_tflops": FP32_MFMA_PEAK_TFLOPS,
                 "hbm_tbs": HBM_PEAK_GBS / 1e3},
        "gpu": torch.cuda.get_device_name(0),
    }), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", default="long")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--halve", choices=["kh", "uniform"], default="kh",
                    help="halving algorithm of compress (kernel halving, the paper's; or "
                         "uniform halving)")
    ap.add_argument("--sinks", type=int, default=0,
                    help="keys kept exactly at the start of every slice")
    ap.add_argument("--window", type=int, default=0,
                    help="keys kept exactly at the end of every slice")
    ap.add_argument("--mode", choices=["compress", "decode", "prefill", "peaks"],
                    default="compress",
                    help="compress + attention (default), Express decoding, masked prefill, or "
                         "the GPU's measured GEMM and bandwidth ceilings")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the thinning path runs each (batch, head) "
              "slice independently and this build has no multi-GPU mode.", file=sys.stderr)
        sys.exit(2)
    if args.mode == "decode":
        decode_main(args)
        return
    if args.mode == "peaks":
        peaks_main(args)
        return
    if args.mode == "prefill":
        prefill_main(args)
        return

    import torch

    from paper_2606_10944_amd import LaunchTimer, thin_attention, thin_compress, thin_plan
    from paper_2606_10944_amd import workloads as W

    w = W.WORKLOADS[args.workload]
    ns, nw = args.sinks, args.window
    weighted = ns > 0 or nw > 0
    # the compress byte models see the thinned rows, attention the m output keys
    wc = dataclasses.replace(w, n=w.n - ns - nw)
    wa = dataclasses.replace(w, n_out=ns + w.n_out + nw)
    Q, K, V = W.make_qkv(w)
    plan = thin_plan(w.B, w.H, wc.n, w.d, w.n_out, w.g)
    U = W.make_uniforms(w, plan["uniforms_total"])
    dev = torch.device("cuda:0")
    Qd, Kd, Vd, Ud = Q.to(dev), K.to(dev), V.to(dev), U.to(dev)
    ws = torch.empty(plan["workspace_bytes"], dtype=torch.uint8, device=dev)
    idx = torch.empty((w.B, w.H, wa.n_out), dtype=torch.int32, device=dev)
    lw = torch.empty((w.B, w.H, wa.n_out), dtype=torch.float32, device=dev) if weighted else None
    O = torch.empty((w.B, w.H, w.n_q, w.d), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        thin_compress(Kd, Vd, w.n_out, w.g, Ud, idx_out=idx, workspace=ws, halve=args.halve,
                      n_sinks=ns, n_window=nw, logw_out=lw, stream=stream)
        thin_attention(Qd, Kd, Vd, idx, logw=lw, O=O, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # Timed region: K steps, nothing recorded between kernels.
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for _ in range(args.steps):
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    # The same K steps again with every kernel launch bracketed by events on
    # its stream (each event adds a few microseconds between kernels, so this
    # pass gives the per-kernel times, not the step time).
    # Launches per step (rounds whose score buffer exceeds the workspace's score
    # region run in several launches), counted on one extra step.
    with LaunchTimer(stream, capacity=4096) as probe:
        step()
    torch.cuda.synchronize()
    launches = len(probe.records())
    with LaunchTimer(stream, capacity=launches * args.steps + 16) as lt:
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
    ms_total = t0.elapsed_time(t1)
    ms_step = ms_total / args.steps
    rec = lt.records()
    per_step = collections.defaultdict(float)
    for name, _, ms in rec:
        per_step[name] += ms / args.steps
    # pair_scores_kernel: the score launches of two-launch rounds and the
    # local launches (scores and decisions in one) of the others
    PS = ("scores", "local")
    score_ms = [ms for name, _, ms in rec if name in PS]
    L = plan["rounds"]
    tc = sum(v for k, v in per_step.items() if k != "attention")
    ta = per_step["attention"]

    cb = compress_bytes(wc, plan) if args.halve == "kh" else uniform_compress_bytes(wc, plan)
    if weighted:  # the layout launch: m indices and m log-weights per slice
        cb += w.S * wa.n_out * 8
    rb = round_bytes(wc, plan)
    ib = score_buffer_bytes(wc, plan)
    ab = attention_bytes(wa, 4, weighted)
    af = attention_flops(wa)
    kev = kappa_evals(plan, wc) if args.halve == "kh" else 0
    # per launch: averages over every score launch of the K steps (a round may
    # take several launches; bytes and time are both summed over the step)
    n_sc = len(score_ms) // args.steps
    sc_rounds = sorted({r for name, r, _ in rec if name in PS})
    two_launch = {r for name, r, _ in rec if name == "scores"}  # rounds with a score buffer
    if n_sc:
        sc_ms_launch = statistics.mean(score_ms)
        sc_bytes_launch = sum(rb[r] for r in sc_rounds) / n_sc
        sc_impl_launch = sum(ib[r] for r in two_launch) / n_sc
        sc_gbs = sc_bytes_launch / (sc_ms_launch * 1e-3) / 1e9
        # per round: its score launches' time per step and the fraction of
        # the HBM roofline its algorithmic bytes reach
        by_round = {}
        for r in sc_rounds:
            ms_r = sum(ms for name, rr, ms in rec if name in PS and rr == r) / args.steps
            by_round[r] = {"ms": ms_r, "frac": rb[r] / (ms_r * 1e-3) / 1e9 / HBM_PEAK_GBS}
    traffic = stored_traffic(w.name) if args.halve == "kh" and not weighted else None
    # bf16 output (half the output bytes; the precision of the parity tests
    # is fp32 output): the same attention timed on its own, after the steps
    Ob = torch.empty((w.B, w.H, w.n_q, w.d), dtype=torch.bfloat16, device=dev)
    thin_attention(Qd, Kd, Vd, idx, logw=lw, O=Ob, stream=stream)
    b0 = torch.cuda.Event(enable_timing=True)
    b1 = torch.cuda.Event(enable_timing=True)
    b0.record(stream)
    for _ in range(args.steps):
        thin_attention(Qd, Kd, Vd, idx, logw=lw, O=Ob, stream=stream)
    b1.record(stream)
    torch.cuda.synchronize()
    ta16 = b0.elapsed_time(b1) / args.steps
    ab16 = attention_bytes(wa, 2, weighted)
    attn_gbs = ab / (ta * 1e-3) / 1e9
    attn_tflops = af / (ta * 1e-3) / 1e12
    value = w.S * w.n_q / (ms_step * 1e-3)

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "(B·H·n)/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "n": w.n, "n_q": w.n_q, "d": w.d,
                   "n_out": w.n_out, "g": w.g, "out_dtype": "fp32", "halve": args.halve,
                   "n_sinks": ns, "n_window": nw},
        "roofline": {
            "kernel": "pair_scores_kernel (one launch per Halve round: the score launch of "
                      "a round above the local bucket size, else the local launch, scores "
                      "and decisions in one)",
            "bound": "hbm", "achieved": sc_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": sc_gbs / HBM_PEAK_GBS,
            "traffic": traffic,
            "traffic_over_algorithmic": traffic / sc_bytes_launch if traffic else None,
            "algorithmic_bytes_per_launch": sc_bytes_launch,
            "impl_bytes_per_launch": sc_impl_launch,
            "ms_per_launch": sc_ms_launch,
            "launches_per_step": n_sc, "rounds": sc_rounds, "by_round": by_round,
        } if n_sc else {
            # uniform halving evaluates no kernel: attention is the dominant kernel
            "kernel": "coreset attention (one launch per step)",
            "bound": "hbm", "achieved": attn_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": attn_gbs / HBM_PEAK_GBS, "traffic": None,
            "algorithmic_bytes_per_launch": ab, "ms_per_launch": ta, "launches_per_step": 1,
        },
        "compress": {"ms": tc, "kappa_evals": kev, "kappa_evals_per_s": kev / (tc * 1e-3),
                     "algorithmic_bytes": cb, "hbm_gbs": cb / (tc * 1e-3) / 1e9,
                     "hbm_frac": cb / (tc * 1e-3) / 1e9 / HBM_PEAK_GBS},
        "attention": {
            "ms": ta, "hbm_gbs": attn_gbs, "hbm_frac": attn_gbs / HBM_PEAK_GBS,
            "mfma_tflops": attn_tflops,
            "mfma_frac": attn_tflops / (BF16_MFMA_PEAK_TFLOPS if w.dtype == "bf16"
                                        else FP32_MFMA_PEAK_TFLOPS),
            "algorithmic_bytes": ab, "flops": af,
        },
        "attention_bf16_out": {
            "ms": ta16, "hbm_gbs": ab16 / (ta16 * 1e-3) / 1e9,
            "hbm_frac": ab16 / (ta16 * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "mfma_tflops": af / (ta16 * 1e-3) / 1e12,
            "mfma_frac": af / (ta16 * 1e-3) / 1e12 / (BF16_MFMA_PEAK_TFLOPS if w.dtype == "bf16"
                                                      else FP32_MFMA_PEAK_TFLOPS),
            "algorithmic_bytes": ab16,
        },
        "ms_per_step_by_kernel": dict(per_step),
        "gpu": torch.cuda.get_device_name(0),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, Q, K, V, U, plan, halve=args.halve, n_sinks=ns,
                                           n_window=nw)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
