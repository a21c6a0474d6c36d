"""The allocation-free forward (kdn_forward_diag_noalloc, scratch held by the library) against
the workspace forward (kdn_forward_diag) through the C ABI: two calls in a row, the second with
a smaller input, each equal to the workspace forward's result."""

import ctypes

import numpy as np
import pytest
import torch

from gpu_util import NAMES, TOL, host_f64, rel_l2, to_device
from paper_2609_07816_amd import workloads as W

pytestmark = pytest.mark.gpu


def _call(L, fn, d, x, ws=None):
    from paper_2609_07816_amd import kdn
    B, T, H, dk = x.B, x.T, x.H, x.dk
    dv = x.dv
    N = x.N
    o = torch.empty((B, T, H, dv), dtype=d["k"].dtype, device="cuda")
    S = torch.empty((N, H, dk, dv), dtype=torch.float32, device="cuda")
    P = torch.empty((N, H, dk), dtype=torch.float32, device="cuda")
    dt = kdn.KDN_BF16 if x.dtype == "bf16" else kdn.KDN_F32
    args = [kdn._ptr(d[n]) for n in NAMES] + [kdn._ptr(d["S0"]), kdn._ptr(d["P0"]), kdn._ptr(o),
                                              kdn._ptr(S), kdn._ptr(P), kdn._ptr(d["cu"]), N, B,
                                              T, H, dk, dv, dt, ctypes.c_float(x.mu),
                                              ctypes.c_float(x.scale)]
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if fn == "noalloc":
        st = L.kdn_forward_diag_noalloc(*args, stream)
    else:
        nbytes = L.kdn_forward_workspace_bytes(0, N, B, T, H, dk, dv, dt, int(d["cu"] is not None),
                                               0)
        ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        st = L.kdn_forward_diag(*args, 0, kdn._ptr(ws), nbytes, stream)
    assert st == kdn.KDN_OK, L.kdn_last_error().decode()
    torch.cuda.synchronize()
    return host_f64(o), host_f64(S), host_f64(P)


def test_noalloc_matches_workspace_forward():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2609_07816_amd import kdn
    L = kdn.lib()
    cases = [
        W.draw_inputs("diag", "bf16", 2, 1500, 8, 128, 128, seed=70, random_state=True),
        W.draw_inputs("diag", "bf16", 1, 300, 4, 64, 64, seed=71, lengths=[100, 0, 200],
                      random_state=True),
    ]
    for x in cases:  # the second call is smaller and packed: stale scratch must not matter
        d = to_device(x)
        got = _call(L, "noalloc", d, x)
        ref = _call(L, "workspace", d, x)
        for name, g, r in zip(("o", "S_T", "P_T"), got, ref):
            err = rel_l2(g, r)
            print(f"  {name}: rel-L2 vs workspace forward {err:.3e}", flush=True)
            assert np.all(np.isfinite(g))
            assert err <= TOL[x.dtype]
            assert np.array_equal(g, r), f"{name}: same kernels, same inputs, different bits"
    # sizes beyond the fixed scratch are refused before anything runs
    big = W.draw_inputs("diag", "bf16", 1, 64, 2, 128, 128, seed=72)
    d = to_device(big)
    args = [kdn._ptr(d[n]) for n in NAMES] + [None, None, kdn._ptr(d["v"]), None, None, None,
                                              4, 4, 4096, 16, 128, 128, kdn.KDN_BF16,
                                              ctypes.c_float(128.0), ctypes.c_float(0.088), None]
    assert L.kdn_forward_diag_noalloc(*args) == kdn.KDN_ERR_UNSUPPORTED
    assert "scratch" in L.kdn_last_error().decode()
