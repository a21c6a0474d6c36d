"""Helpers shared by the GPU tests: move seeded inputs to the device, compare with the oracle."""

from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2609_07816_amd import workloads as W

NAMES = ("q", "k", "v", "alpha", "omega", "r")
TOL = {"f32": 1e-5, "bf16": 2e-2}   # rel-L2 bounds fixed for this path (fp32 / bf16 inputs)


def dev_tensor(stored: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(stored).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(stored, dtype=np.float32))
    return t.to(device)


def to_device(x: W.KdnInputs, device="cuda"):
    d = {n: dev_tensor(x.stored[n], x.dtype, device) for n in NAMES}
    d["S0"] = None if x.S0 is None else torch.from_numpy(x.S0).to(device)
    d["P0"] = None if x.P0 is None else torch.from_numpy(x.P0).to(device)
    d["cu"] = None if x.cu_seqlens is None else torch.from_numpy(x.cu_seqlens).to(device)
    return d


def host_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def rel_l2(x: np.ndarray, ref: np.ndarray) -> float:
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref.ravel())
    num = np.linalg.norm((x - ref).ravel())
    return float(num / den) if den > 0 else float(num)


def run_gpu_forward(x: W.KdnInputs, chunk: int = 0):
    from paper_2609_07816_amd import kdn
    d = to_device(x)
    f = kdn.forward_diag if x.variant == "diag" else kdn.forward_iso
    o, S, P = f(d["q"], d["k"], d["v"], d["alpha"], d["omega"], d["r"], S0=d["S0"], P0=d["P0"],
                cu_seqlens=d["cu"], mu=x.mu, scale=x.scale, chunk=chunk)
    torch.cuda.synchronize()
    return host_f64(o), host_f64(S), host_f64(P)


def run_oracle_forward(x: W.KdnInputs, chains=None, traces=False):
    """Oracle on the whole batch (chains None) or on selected (row, head) chains of a
    fixed-length batch: returns arrays restricted to those chains, in the given order."""
    f = oracle.forward_diag if x.variant == "diag" else oracle.forward_iso
    if chains is None:
        arrs = [x.f64(n) for n in NAMES]
        return f(*arrs, S0=x.S0, P0=x.P0, cu_seqlens=x.cu_seqlens, mu=x.mu, scale=x.scale,
                 traces=traces)
    outs = []
    for (b, h) in chains:
        arrs = [x.f64(n)[b:b + 1, :, h:h + 1] for n in NAMES]
        S0 = None if x.S0 is None else x.S0[b:b + 1, h:h + 1]
        P0 = None if x.P0 is None else x.P0[b:b + 1, h:h + 1]
        outs.append(f(*arrs, S0=S0, P0=P0, mu=x.mu, scale=x.scale, traces=traces))
    return outs


def run_oracle_packed_seq(x: W.KdnInputs, n: int, heads):
    """Oracle on sequence n (all listed heads) of a packed batch."""
    f = oracle.forward_diag if x.variant == "diag" else oracle.forward_iso
    t0, t1 = int(x.cu_seqlens[n]), int(x.cu_seqlens[n + 1])
    hs = list(heads)
    arrs = [x.f64(nm)[:, t0:t1][:, :, hs] for nm in NAMES]
    S0 = None if x.S0 is None else x.S0[n:n + 1][:, hs]
    P0 = None if x.P0 is None else x.P0[n:n + 1][:, hs]
    return f(*arrs, S0=S0, P0=P0, mu=x.mu, scale=x.scale)
