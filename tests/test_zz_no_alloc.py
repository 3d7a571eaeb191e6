"""thin_compress_static (no workspace argument, no allocation) against
thin_compress on the same inputs: the coreset indices bit-exact, on two
calls in a row (the second with a smaller input, so the static workspace
holds the first call's contents), and the status word 0."""
import ctypes as C

import numpy as np
import pytest
import torch

from paper_2606_10944_amd import _lib, thin_compress, thin_plan
from paper_2606_10944_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _static(w, Kd, Vd, Ud):
    idx = torch.full((w.B, w.H, w.n_out), -1, dtype=torch.int32, device=DEV)
    status = torch.full((1,), 7, dtype=torch.int32, device=DEV)
    dtype = _lib.THIN_BF16 if Kd.dtype == torch.bfloat16 else _lib.THIN_FP32
    stream = torch.cuda.current_stream()
    rc = _lib.lib().thin_compress_static(
        C.c_void_p(Kd.data_ptr()), C.c_void_p(Vd.data_ptr()), dtype, w.B, w.H, w.n, w.d,
        w.n_out, w.g, C.c_void_p(Ud.data_ptr()), Ud.numel(), C.c_void_p(idx.data_ptr()),
        C.c_void_p(status.data_ptr()), C.c_void_p(stream.cuda_stream))
    assert rc == _lib.THIN_OK, _lib.thin_status_str(rc)
    return idx, status


def test_static_workspace_compress_matches_thin_compress():
    # the benchmark's workload (its first round's scores exceed what the
    # static array leaves: several score launches), then a smaller one
    for name in ("long", "vit"):
        w = W.WORKLOADS[name]
        print(f"no-alloc compress: {name}", flush=True)
        _, K, V = W.make_qkv(w)
        plan = thin_plan(w.B, w.H, w.n, w.d, w.n_out, w.g)
        U = W.make_uniforms(w, plan["uniforms_total"])
        Kd, Vd, Ud = K.to(DEV), V.to(DEV), U.to(DEV)
        got, status = _static(w, Kd, Vd, Ud)
        want = thin_compress(Kd, Vd, w.n_out, w.g, Ud)
        torch.cuda.synchronize()
        assert int(status.item()) == 0, name
        assert torch.equal(got, want), name
        g = got.cpu().numpy().reshape(w.S, w.n_out)
        assert np.all(np.diff(g, axis=-1) > 0) and g.min() >= 0 and g.max() < w.n
