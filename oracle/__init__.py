"""KDN CPU oracle -- test infrastructure only.

Plain float64 implementations of the Diagonal and Isotropic KDN recurrences written from the
paper (arXiv 2609.07816; Prop. "Diagonal Kalman Delta Network" and Prop. "Isotropic Kalman Delta
Network"), their reverse-mode adjoint (``backward``, kdn_oracle_bwd.c), plus three Moebius-scan
forms of the variance chain (App. "Hardware-Efficient Chunkwise Algorithm"). Only the tests, ``__graft_entry__.smoke()`` and the benchmark's CPU
baseline may import this package; the GPU library never does.

The C source ``kdn_oracle.c`` is compiled with gcc (``build()``) into ``liboracle.so`` next to
it. Inputs are float64 arrays; bf16/float32 inputs are upcast exactly by the caller.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kdn_oracle.c")
_SRCS = [_SRC, os.path.join(_HERE, "kdn_oracle_bwd.c")]
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile liboracle.so with gcc (-O2, OpenMP, IEEE arithmetic: no fast-math, no FMA)."""
    if not force and os.path.exists(_LIB) and all(
            os.path.getmtime(_LIB) >= os.path.getmtime(src) for src in _SRCS):
        return _LIB
    tmp = _LIB + f".tmp{os.getpid()}"
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
           "-Wall", "-Wextra", "-o", tmp, *_SRCS, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    build(force=False)
    lib = ctypes.CDLL(_LIB)
    d = ctypes.POINTER(ctypes.c_double)
    i32p = ctypes.POINTER(ctypes.c_int32)
    ci, cd = ctypes.c_int, ctypes.c_double
    lib.oracle_kdn_forward_diag.argtypes = [d] * 14 + [i32p] + [ci] * 6 + [cd, cd, ci, d, d]
    lib.oracle_kdn_forward_iso.argtypes = [d] * 14 + [i32p] + [ci] * 7 + [cd, cd, ci, d, d]
    lib.oracle_kdn_decode_step.argtypes = ([ci] + [d] * 8 + [i32p, d] + [ci] * 6 +
                                           [cd, cd, ci, d, d])
    for name in ("oracle_mobius_fold", "oracle_mobius_tree"):
        getattr(lib, name).argtypes = [d, d, d, cd, ctypes.c_int64, ci, d, d]
    lib.oracle_mobius_chunked.argtypes = [d, d, d, cd, ctypes.c_int64, ctypes.c_int64, ci, d, d]
    lib.oracle_kdn_forward_kam.argtypes = [d] * 11 + [i32p] + [ci] * 6 + [cd, ci]
    lib.oracle_kdn_forward_kam.restype = ci
    lib.oracle_kdn_backward.argtypes = ([ci] + [d] * 8 + [i32p] + [ci] * 7 + [cd, cd] +
                                        [d] * 13 + [ci])
    for name in ("oracle_kdn_forward_diag", "oracle_kdn_forward_iso", "oracle_kdn_decode_step",
                 "oracle_mobius_fold", "oracle_mobius_tree", "oracle_mobius_chunked",
                 "oracle_kdn_backward"):
        getattr(lib, name).restype = ci
    _lib = lib
    return lib


def _p(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.dtype == np.float64 and a.flags["C_CONTIGUOUS"], "oracle arrays are C-contiguous f64"
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _pi(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.dtype == np.int32 and a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _f64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def forward_diag(q, k, v, alpha, omega, r, S0=None, P0=None, cu_seqlens=None, mu=None,
                 scale=None, traces=False, nthreads=0, mu_t=None, beta_eff=False):
    """Diagonal KDN forward. Returns dict with o, S_T, P_T (and phat, kappa, p when traces;
    beta_eff = k^T kappa per token when beta_eff). mu_t [B,T,H] replaces mu per token."""
    q, k, v, alpha, omega, r, S0, P0, mu_t = map(_f64, (q, k, v, alpha, omega, r, S0, P0, mu_t))
    B, T, H, dk = k.shape
    dv = v.shape[-1]
    cu = None if cu_seqlens is None else np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    N = B if cu is None else len(cu) - 1
    mu = float(dk if mu is None else mu)
    scale = float(dk ** -0.5 if scale is None else scale)
    out = dict(o=np.zeros((B, T, H, dv)), S_T=np.zeros((N, H, dk, dv)), P_T=np.zeros((N, H, dk)))
    if traces:
        for name in ("phat", "kappa", "p"):
            out[name] = np.zeros((B, T, H, dk))
    if beta_eff:
        out["beta_eff"] = np.zeros((B, T, H))
    rc = _load().oracle_kdn_forward_diag(
        _p(q), _p(k), _p(v), _p(alpha), _p(omega), _p(r), _p(S0), _p(P0), _p(out["o"]),
        _p(out["S_T"]), _p(out["P_T"]), _p(out.get("phat")), _p(out.get("kappa")),
        _p(out.get("p")), _pi(cu), N, B, T, H, dk, dv, mu, scale, nthreads, _p(mu_t),
        _p(out.get("beta_eff")))
    if rc != 0:
        raise ValueError("oracle_kdn_forward_diag rejected its arguments")
    return out


def forward_iso(q, k, v, alpha, omega, r, S0=None, P0=None, cu_seqlens=None, mu=None,
                scale=None, traces=False, nthreads=0, mu_t=None, beta_eff=False):
    """Isotropic KDN forward; alpha [B,T,H,dk] (per channel) or [B,T,H] (per head).
    mu_t [B,T,H] replaces mu per token; beta_eff adds beta ||k||^2 per token."""
    q, k, v, alpha, omega, r, S0, P0, mu_t = map(_f64, (q, k, v, alpha, omega, r, S0, P0, mu_t))
    B, T, H, dk = k.shape
    dv = v.shape[-1]
    per_channel = int(alpha.ndim == 4)
    cu = None if cu_seqlens is None else np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    N = B if cu is None else len(cu) - 1
    mu = float(dk if mu is None else mu)
    scale = float(dk ** -0.5 if scale is None else scale)
    out = dict(o=np.zeros((B, T, H, dv)), S_T=np.zeros((N, H, dk, dv)), P_T=np.zeros((N, H)))
    if traces:
        for name in ("bhat", "beta", "b"):
            out[name] = np.zeros((B, T, H))
    if beta_eff:
        out["beta_eff"] = np.zeros((B, T, H))
    rc = _load().oracle_kdn_forward_iso(
        _p(q), _p(k), _p(v), _p(alpha), _p(omega), _p(r), _p(S0), _p(P0), _p(out["o"]),
        _p(out["S_T"]), _p(out["P_T"]), _p(out.get("bhat")), _p(out.get("beta")),
        _p(out.get("b")), _pi(cu), N, B, T, H, dk, dv, per_channel, mu, scale, nthreads,
        _p(mu_t), _p(out.get("beta_eff")))
    if rc != 0:
        raise ValueError("oracle_kdn_forward_iso rejected its arguments")
    return out


def decode_step(variant, q, k, v, alpha, omega, r, S, P, slot_idx=None, mu=None, scale=None,
                nthreads=0, mu_t=None, beta_eff=None):
    """One decode step; S and P (float64 arrays) are updated in place. Returns o [R,H,dv].
    mu_t [R,H] replaces mu per row; beta_eff (a float64 [R,H] array) receives k^T kappa."""
    q, k, v, alpha, omega, r, mu_t = map(_f64, (q, k, v, alpha, omega, r, mu_t))
    assert S.dtype == np.float64 and S.flags["C_CONTIGUOUS"]
    assert P.dtype == np.float64 and P.flags["C_CONTIGUOUS"]
    R, H, dk = k.shape
    dv = v.shape[-1]
    num_slots = S.shape[0]
    per_channel = int(alpha.ndim == 3)
    vid = {"diag": 0, "iso": 1}[variant]
    o = np.zeros((R, H, dv))
    si = None if slot_idx is None else np.ascontiguousarray(slot_idx, dtype=np.int32)
    mu = float(dk if mu is None else mu)
    scale = float(dk ** -0.5 if scale is None else scale)
    rc = _load().oracle_kdn_decode_step(
        vid, _p(q), _p(k), _p(v), _p(alpha), _p(omega), _p(r), _p(S), _p(P), _pi(si), _p(o),
        R, num_slots, H, dk, dv, per_channel, mu, scale, nthreads, _p(mu_t), _p(beta_eff))
    if rc != 0:
        raise ValueError("oracle_kdn_decode_step rejected its arguments")
    return o


def forward_kam(q, k, v, alpha, omega, r, S0=None, P0=None, cu_seqlens=None, scale=None,
                nthreads=0):
    """Kalman Associative Memory (the exact filter, dense dk x dk covariance per head): returns
    o, S_T and P_T [N,H,dk,dk]. P0 [N,H,dk,dk] (None = identity); alpha, omega [B,T,H,dk]."""
    q, k, v, alpha, omega, r, S0, P0 = map(_f64, (q, k, v, alpha, omega, r, S0, P0))
    B, T, H, dk = k.shape
    dv = v.shape[-1]
    cu = None if cu_seqlens is None else np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    N = B if cu is None else len(cu) - 1
    scale = float(dk ** -0.5 if scale is None else scale)
    out = dict(o=np.zeros((B, T, H, dv)), S_T=np.zeros((N, H, dk, dv)),
               P_T=np.zeros((N, H, dk, dk)))
    rc = _load().oracle_kdn_forward_kam(
        _p(q), _p(k), _p(v), _p(alpha), _p(omega), _p(r), _p(S0), _p(P0), _p(out["o"]),
        _p(out["S_T"]), _p(out["P_T"]), _pi(cu), N, B, T, H, dk, dv, scale, nthreads)
    if rc != 0:
        raise ValueError("oracle_kdn_forward_kam rejected its arguments")
    return out


def backward(variant, q, k, v, alpha, omega, r, S0=None, P0=None, cu_seqlens=None, mu=None,
             scale=None, mu_t=None, dO=None, dS_T=None, dP_T=None, nthreads=0):
    """Reverse-mode adjoint of forward_diag / forward_iso (kdn_oracle_bwd.c): given the adjoints
    of o, S_T and P_T (None = zero), returns a dict of dq, dk, dv, dalpha, domega, dr, dS0, dP0
    (and dmu_t when mu_t is given), each shaped like its input."""
    q, k, v, alpha, omega, r, S0, P0, mu_t, dO, dS_T, dP_T = map(
        _f64, (q, k, v, alpha, omega, r, S0, P0, mu_t, dO, dS_T, dP_T))
    B, T, H, dk = k.shape
    dv = v.shape[-1]
    vid = {"diag": 0, "iso": 1}[variant]
    per_channel = int(vid == 0 or alpha.ndim == 4)
    cu = None if cu_seqlens is None else np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    N = B if cu is None else len(cu) - 1
    mu = float(dk if mu is None else mu)
    scale = float(dk ** -0.5 if scale is None else scale)
    out = dict(dq=np.zeros_like(q), dk=np.zeros_like(k), dv=np.zeros_like(v),
               dalpha=np.zeros_like(alpha), domega=np.zeros_like(omega), dr=np.zeros_like(r),
               dS0=np.zeros((N, H, dk, dv)),
               dP0=np.zeros((N, H, dk) if vid == 0 else (N, H)))
    if mu_t is not None:
        out["dmu_t"] = np.zeros_like(mu_t)
    rc = _load().oracle_kdn_backward(
        vid, _p(q), _p(k), _p(v), _p(alpha), _p(omega), _p(r), _p(S0), _p(P0), _pi(cu), N, B, T,
        H, dk, dv, per_channel, mu, scale, _p(mu_t), _p(dO), _p(dS_T), _p(dP_T), _p(out["dq"]),
        _p(out["dk"]), _p(out["dv"]), _p(out["dalpha"]), _p(out["domega"]), _p(out["dr"]),
        _p(out["dS0"]), _p(out["dP0"]), _p(out.get("dmu_t")), nthreads)
    if rc != 0:
        raise ValueError("oracle_kdn_backward rejected its arguments")
    return out


def _mobius(name, a, w, u, p0, renorm, *extra):
    a, w, u = map(_f64, (a, w, u))
    T = a.shape[0]
    phat, p = np.zeros(T), np.zeros(T)
    rc = getattr(_load(), name)(_p(a), _p(w), _p(u), float(p0), T, *extra, int(renorm),
                                _p(phat), _p(p))
    if rc != 0:
        raise ValueError(name)
    return phat, p


def mobius_fold(a, w, u, p0=1.0, renorm=True):
    """Left fold of the Moebius matrices of one chain; returns (phat, p) per token."""
    return _mobius("oracle_mobius_fold", a, w, u, p0, renorm)


def mobius_tree(a, w, u, p0=1.0, renorm=True):
    """Blelloch exclusive scan of the Moebius matrices; returns (phat, p) per token."""
    return _mobius("oracle_mobius_tree", a, w, u, p0, renorm)


def mobius_chunked(a, w, u, p0=1.0, Cg=256, renorm=True):
    """Three-pass chunked Moebius scan with chunk length Cg; returns (phat, p) per token."""
    return _mobius("oracle_mobius_chunked", a, w, u, p0, renorm, int(Cg))


# ---------------------------------------------------------------------------------------------
# The mixer layer's input maps (Prop. "Diagonal Kalman Delta Network", eq.
# kla-box-parameterization; Prop. "Isotropic Kalman Delta Network", eq.
# iso-kla-box-parameterization): the gates and noise terms come from pre-activations through
# alpha = sigmoid(.), omega = softplus(.), r = r_min + softplus(.); the layer's queries and keys
# are L2-normalised per token and head (Sec. "Experiments", the KDA-style layer).
# ---------------------------------------------------------------------------------------------

def sigmoid(x):
    """1 / (1 + exp(-x)) in float64, evaluated without overflow for either sign."""
    x = np.asarray(x, dtype=np.float64)
    e = np.exp(-np.abs(x))
    return np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def softplus(x):
    """log(1 + exp(x)) in float64, as max(x, 0) + log1p(exp(-|x|))."""
    x = np.asarray(x, dtype=np.float64)
    return np.maximum(x, 0.0) + np.log1p(np.exp(-np.abs(x)))


def l2_normalize(x):
    """x / ||x|| over the last axis (zero rows stay zero)."""
    x = np.asarray(x, dtype=np.float64)
    n = np.sqrt(np.sum(x * x, axis=-1, keepdims=True))
    return np.where(n > 0, x / np.where(n > 0, n, 1.0), 0.0)


def layer_inputs(q, k, a_pre, w_pre, r_pre, r_min, qk_norm=True):
    """The recurrence's inputs from the layer's: (q, k, alpha, omega, r) in float64."""
    qq, kk = (l2_normalize(q), l2_normalize(k)) if qk_norm else (_f64(q), _f64(k))
    return qq, kk, sigmoid(a_pre), softplus(w_pre), float(r_min) + softplus(r_pre)
