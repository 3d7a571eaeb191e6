"""Seeded synthetic workloads for the thinning path.

This module only draws random numbers and shapes them into Q/K/V tensors and
uniform buffers.  It holds none of the method's arithmetic (no kernel, no
halving, no planning formula): the number of uniforms a call consumes is an
argument, computed by whoever plans the call.  Both the HIP path and the CPU
oracle are fed from here, byte for byte.

The five named workloads stand in for the paper's prefill benchmarks (its
single-layer runtime study and LongBench/ViT-style shapes), whose models and
datasets are not available; the recipes are synthetic:

* ``tiny``   B=1  H=1  n=1024  d=64  fp32  Q,K,V ~ N(0,1)/d^(1/4)       n_out=32  g=2
* ``vit``    B=32 H=1  n=3136  d=64  bf16  Q,K,V ~ N(0,1), per-row LayerNorm  n_out=64  g=2
* ``imggen`` B=16 H=1  n=1024 keys, 4096 queries, d=64 fp32; keys from a
             16-centre Gaussian mixture (sigma 0.3), V ~ U[-1,1], Q ~ N(0,1)   n_out=64 g=3
* ``long``   B=4  H=16 n=16384 d=128 bf16  Q,K,V ~ N(0,1), 5% of key rows x4  n_out=128 g=3
* ``stress`` B=1  H=32 n=65536 d=128 bf16  Q,K,V ~ N(0,1)                  n_out=256 g=4

Kind ``heavy_tail_mean`` (a parity case, not a benchmark) is ``long``'s recipe
with a key mean shared by the rows of a slice: k = z + mu_s, ||mu_s||^2 = 2d
exactly (a random direction per slice), then 5% of the rows x4.  Keys with a
common direction are usual in attention layers; here the cross exponents
<k_i,k_j>/sqrt(d) of the large rows exceed a smaller pair's own diagonal
exponents by up to ~90 (natural units).

Workload i (1-based, in the order above) uses seed i-1.  ``SeedSequence(seed)
.spawn(4)`` gives independent PCG64 streams for Q, K, V and the uniforms.
Values are drawn in float64 and cast once (bf16 by torch's round-to-nearest-
even).  Uniforms are ``k * 2**-24`` with k uniform on [0, 2**24), stored as
float32, so every quantity derived from them is exact on both sides.
"""
from __future__ import annotations

from dataclasses import dataclass, replace
from typing import Optional, Tuple

import numpy as np
import torch

KINDS = ("gauss_d4", "layernorm", "mixture", "heavy_tail", "gauss", "heavy_tail_mean")


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    n: int          # key/value rows per slice
    n_q: int        # query rows per slice
    d: int
    dtype: str      # "fp32" or "bf16"
    n_out: int
    g: int
    seed: int
    kind: str

    @property
    def S(self) -> int:
        return self.B * self.H

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


WORKLOADS = {
    "tiny": Workload("tiny", 1, 1, 1024, 1024, 64, "fp32", 32, 2, 0, "gauss_d4"),
    "vit": Workload("vit", 32, 1, 3136, 3136, 64, "bf16", 64, 2, 1, "layernorm"),
    "imggen": Workload("imggen", 16, 1, 1024, 4096, 64, "fp32", 64, 3, 2, "mixture"),
    "long": Workload("long", 4, 16, 16384, 16384, 128, "bf16", 128, 3, 3, "heavy_tail"),
    "stress": Workload("stress", 1, 32, 65536, 65536, 128, "bf16", 256, 4, 4, "gauss"),
}
ORDER = ("tiny", "vit", "imggen", "long", "stress")


def torch_dtype(name: str) -> torch.dtype:
    return {"fp32": torch.float32, "bf16": torch.bfloat16}[name]


def _streams(seed: int):
    ss = np.random.SeedSequence(seed)
    return [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(4)]


def _cast(x: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x))
    return t.to(torch_dtype(dtype))


def _layernorm_rows(x: np.ndarray, eps: float = 1e-5) -> np.ndarray:
    # no affine, population variance, in float64
    mu = x.mean(axis=-1, keepdims=True)
    var = x.var(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def make_qkv(w: Workload) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """Return CPU tensors Q [B,H,n_q,d], K [B,H,n,d], V [B,H,n,d] in w.dtype."""
    gq, gk, gv, _ = _streams(w.seed)
    S, n, nq, d = w.S, w.n, w.n_q, w.d
    shape_q = (w.B, w.H, nq, d)
    shape_kv = (w.B, w.H, n, d)
    if w.kind == "gauss_d4":
        s = d ** -0.25
        q = gq.standard_normal(shape_q) * s
        k = gk.standard_normal(shape_kv) * s
        v = gv.standard_normal(shape_kv) * s
    elif w.kind == "layernorm":
        q = _layernorm_rows(gq.standard_normal(shape_q))
        k = _layernorm_rows(gk.standard_normal(shape_kv))
        v = _layernorm_rows(gv.standard_normal(shape_kv))
    elif w.kind == "mixture":
        q = gq.standard_normal(shape_q)
        centres = gk.standard_normal((S, 16, d))
        which = gk.integers(0, 16, size=(S, n))
        noise = gk.standard_normal((S, n, d))
        k = np.take_along_axis(centres, which[:, :, None], axis=1) + 0.3 * noise
        k = k.reshape(shape_kv)
        v = gv.uniform(-1.0, 1.0, size=shape_kv)
    elif w.kind == "heavy_tail":
        q = gq.standard_normal(shape_q)
        k = gk.standard_normal(shape_kv)
        m = int(0.05 * n)
        k2 = k.reshape(S, n, d)
        for s in range(S):
            rows = gk.choice(n, size=m, replace=False)
            k2[s, rows, :] *= 4.0
        v = gv.standard_normal(shape_kv)
    elif w.kind == "heavy_tail_mean":
        q = gq.standard_normal(shape_q)
        k = gk.standard_normal(shape_kv).reshape(S, n, d)
        mu = gk.standard_normal((S, 1, d))
        mu *= np.sqrt(2.0 * d) / np.linalg.norm(mu, axis=-1, keepdims=True)
        k += mu
        m = int(0.05 * n)
        for s in range(S):
            rows = gk.choice(n, size=m, replace=False)
            k[s, rows, :] *= 4.0
        k = k.reshape(shape_kv)
        v = gv.standard_normal(shape_kv)
    elif w.kind == "gauss":
        q = gq.standard_normal(shape_q)
        k = gk.standard_normal(shape_kv)
        v = gv.standard_normal(shape_kv)
    else:
        raise ValueError(f"unknown workload kind {w.kind!r}")
    return _cast(q, w.dtype), _cast(k, w.dtype), _cast(v, w.dtype)


def make_uniforms(w: Workload, count: int) -> torch.Tensor:
    """`count` float32 uniforms k*2^-24, k ~ Unif{0..2^24-1}, slice-major."""
    _, _, _, gu = _streams(w.seed)
    k = gu.integers(0, 1 << 24, size=int(count), dtype=np.int64)
    return torch.from_numpy((k.astype(np.float64) * 2.0 ** -24).astype(np.float32))


def custom(name: str = "custom", *, B=1, H=1, n=256, n_q: Optional[int] = None,
           d=64, dtype="fp32", n_out=16, g=1, seed=1234, kind="gauss_d4") -> Workload:
    """A small workload of any shape, for tests (ragged sizes, edge cases)."""
    return Workload(name, B, H, n, n if n_q is None else n_q, d, dtype, n_out, g, seed, kind)
