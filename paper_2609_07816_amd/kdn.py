"""Thin Python binding of libkdn (C ABI in include/kdn.h).

Argument marshalling only: every step of the computation runs in the HIP kernels of
``libkdn.so``. torch provides device memory (output allocation) and the current stream. If the
library is missing this module raises at import of the first call; there is no fallback.

Functions mirror the C entry points:

* ``forward_diag(q, k, v, alpha, omega, r, S0=None, P0=None, cu_seqlens=None, mu=None,
  scale=None, chunk=0) -> (o, S_T, P_T)``
* ``forward_iso(...)`` -- same, ``alpha`` may be [B,T,H,dk] (per channel) or [B,T,H]
* ``forward_diag_noalloc(...)`` -- ``forward_diag`` on the library's fixed scratch
* ``decode_step(variant, q, k, v, alpha, omega, r, S, P, slot_idx=None, mu=None, scale=None)
  -> o`` (S and P updated in place)
* ``gain_diag(k, alpha, omega, r, P0=None, cu_seqlens=None, mu=None) -> (kappa, phat, P_T)``
* ``gain_iso(...) -> (beta, bhat, P_T)``
* ``forward_layer(variant, q, k, v, alpha, omega, r, ..., gates_preact=False, r_min=0.01,
  qk_l2norm=False, mu_t=None, want_beta_eff=False) -> (o, S_T, P_T, beta_eff or None)``
* ``decode_step_layer(variant, ..., gates_preact=False, r_min=0.01, qk_l2norm=False,
  mu_t=None, beta_eff=None) -> o``
* ``backward(variant, q, k, v, alpha, omega, r, S0=None, P0=None, cu_seqlens=None, mu=None,
  scale=None, dO=None, dS_T=None, dP_T=None) -> dict`` of float32 gradients
* ``forward_kam(q, k, v, alpha, omega, r, S0=None, P0=None, cu_seqlens=None, scale=None)
  -> (o, S_T, P_T)`` -- the dense-covariance Kalman Associative Memory
"""

from __future__ import annotations

import ctypes
import os
import re
from typing import Optional

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkdn.so")
HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "kdn.h")

KDN_OK, KDN_ERR_INVALID_ARG, KDN_ERR_UNSUPPORTED, KDN_ERR_WORKSPACE, KDN_ERR_HIP = range(5)
KDN_F32, KDN_BF16 = 0, 1

_lib = None


class LayerOpts(ctypes.Structure):
    """kdn_layer_opts of include/kdn.h."""
    _fields_ = [("gates_preact", ctypes.c_int32), ("r_min", ctypes.c_float),
                ("qk_l2norm", ctypes.c_int32), ("mu_t", ctypes.c_void_p),
                ("beta_eff", ctypes.c_void_p)]


class KdnError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status} ({detail})")
        self.status = status


def declared_symbols():
    """Names of the entry points declared in include/kdn.h."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(kdn_[a-z_]+)\s*\(", text)))


def lib():
    """Load libkdn.so (raises FileNotFoundError when it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise FileNotFoundError(f"{LIB_PATH} is missing: build it with "
                                "`python -m paper_2609_07816_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
    L.kdn_forward_diag.argtypes = [vp] * 12 + [i32] * 6 + [ctypes.c_int, f32, f32, i32, vp, sz,
                                                            vp]
    L.kdn_forward_iso.argtypes = [vp] * 12 + [i32] * 6 + [ctypes.c_int, i32, f32, f32, i32, vp,
                                                           sz, vp]
    L.kdn_forward_diag_noalloc.argtypes = [vp] * 12 + [i32] * 6 + [ctypes.c_int, f32, f32, vp]
    L.kdn_decode_step.argtypes = [i32] + [vp] * 10 + [i32] * 5 + [ctypes.c_int, i32, f32, f32,
                                                                   vp]
    L.kdn_gain_diag.argtypes = [vp] * 9 + [i32] * 5 + [ctypes.c_int, f32, vp, sz, vp]
    L.kdn_gain_iso.argtypes = [vp] * 9 + [i32] * 5 + [ctypes.c_int, i32, f32, vp, sz, vp]
    L.kdn_forward_layer.argtypes = [i32] + [vp] * 12 + [i32] * 6 + [ctypes.c_int, i32, f32, f32,
                                                                     ctypes.POINTER(LayerOpts),
                                                                     vp, sz, vp]
    L.kdn_decode_step_layer.argtypes = ([i32] + [vp] * 10 + [i32] * 5 +
                                        [ctypes.c_int, i32, f32, f32, ctypes.POINTER(LayerOpts),
                                         vp])
    L.kdn_backward.argtypes = ([i32] + [vp] * 9 + [i32] * 6 + [ctypes.c_int, i32, f32, f32] +
                               [vp] * 11 + [vp, sz, vp])
    L.kdn_forward_kam.argtypes = [vp] * 12 + [i32] * 6 + [ctypes.c_int, f32, vp]
    L.kdn_forward_kam.restype = ctypes.c_int
    L.kdn_backward_workspace_bytes.argtypes = [i32] * 8
    L.kdn_backward_workspace_bytes.restype = sz
    L.kdn_forward_workspace_bytes.argtypes = [i32] * 7 + [ctypes.c_int, i32, i32]
    L.kdn_gain_workspace_bytes.argtypes = [i32] * 6
    for name in ("kdn_forward_diag", "kdn_forward_iso", "kdn_forward_diag_noalloc",
                 "kdn_decode_step", "kdn_gain_diag", "kdn_gain_iso", "kdn_forward_layer",
                 "kdn_decode_step_layer", "kdn_backward"):
        getattr(L, name).restype = ctypes.c_int
    L.kdn_forward_workspace_bytes.restype = sz
    L.kdn_gain_workspace_bytes.restype = sz
    L.kdn_status_string.argtypes = [ctypes.c_int]
    L.kdn_status_string.restype = ctypes.c_char_p
    L.kdn_last_error.restype = ctypes.c_char_p
    L.kdn_version.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(status: int, where: str):
    if status != KDN_OK:
        L = lib()
        raise KdnError(status, where, f"{L.kdn_status_string(status).decode()}: "
                                      f"{L.kdn_last_error().decode()}")


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libkdn must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return KDN_F32
    if t.dtype == torch.bfloat16:
        return KDN_BF16
    raise TypeError(f"unsupported input dtype {t.dtype} (float32 or bfloat16)")


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _same(dtype, *ts):
    for t in ts:
        if t is not None and t.dtype != dtype:
            raise TypeError("q, k, v, alpha, omega and r must share one dtype")


def _f32(t):
    if t is not None and t.dtype != torch.float32:
        raise TypeError("states (S, P) are float32")
    return t


def _forward(variant, q, k, v, alpha, omega, r, S0, P0, cu_seqlens, mu, scale, chunk):
    B, T, H, dk = k.shape
    dv = v.shape[-1]
    _same(k.dtype, q, v, alpha, omega, r)
    dev = k.device
    N = B if cu_seqlens is None else cu_seqlens.numel() - 1
    mu = float(dk if mu is None else mu)
    scale = float(dk ** -0.5 if scale is None else scale)
    o = torch.empty((B, T, H, dv), dtype=k.dtype, device=dev)
    S_T = torch.empty((N, H, dk, dv), dtype=torch.float32, device=dev)
    P_T = torch.empty((N, H, dk) if variant == 0 else (N, H), dtype=torch.float32, device=dev)
    ws_bytes = lib().kdn_forward_workspace_bytes(variant, N, B, T, H, dk, dv, _dtype_code(k),
                                                 int(cu_seqlens is not None), int(chunk))
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev) if ws_bytes else None
    cu = None if cu_seqlens is None else cu_seqlens
    if cu is not None and cu.dtype != torch.int32:
        raise TypeError("cu_seqlens must be int32")
    common = [_ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(omega), _ptr(r), _ptr(_f32(S0)),
              _ptr(_f32(P0)), _ptr(o), _ptr(S_T), _ptr(P_T), _ptr(cu), N, B, T, H, dk, dv,
              _dtype_code(k)]
    tail = [ctypes.c_float(mu), ctypes.c_float(scale), int(chunk), _ptr(ws),
            ws_bytes, _stream(dev)]
    if variant == 0:
        st = lib().kdn_forward_diag(*common, *tail)
        _check(st, "kdn_forward_diag")
    else:
        apc = int(alpha.dim() == 4)
        st = lib().kdn_forward_iso(*common, apc, *tail)
        _check(st, "kdn_forward_iso")
    return o, S_T, P_T


def forward_diag(q, k, v, alpha, omega, r, S0=None, P0=None, cu_seqlens=None, mu=None,
                 scale=None, chunk=0):
    """Diagonal KDN forward; returns (o, S_T, P_T)."""
    return _forward(0, q, k, v, alpha, omega, r, S0, P0, cu_seqlens, mu, scale, chunk)


def forward_diag_noalloc(q, k, v, alpha, omega, r, S0=None, P0=None, cu_seqlens=None, mu=None,
                         scale=None, o=None, S_T=None, P_T=None):
    """Diagonal KDN forward with the library's own fixed scratch (no workspace); outputs may be
    passed in (o, S_T, P_T) so that the call allocates nothing. Returns (o, S_T, P_T)."""
    B, T, H, dk = k.shape
    dv = v.shape[-1]
    _same(k.dtype, q, v, alpha, omega, r)
    dev = k.device
    N = B if cu_seqlens is None else cu_seqlens.numel() - 1
    mu = float(dk if mu is None else mu)
    scale = float(dk ** -0.5 if scale is None else scale)
    if o is None:
        o = torch.empty((B, T, H, dv), dtype=k.dtype, device=dev)
    if S_T is None:
        S_T = torch.empty((N, H, dk, dv), dtype=torch.float32, device=dev)
    if P_T is None:
        P_T = torch.empty((N, H, dk), dtype=torch.float32, device=dev)
    st = lib().kdn_forward_diag_noalloc(
        _ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(omega), _ptr(r), _ptr(_f32(S0)),
        _ptr(_f32(P0)), _ptr(o), _ptr(_f32(S_T)), _ptr(_f32(P_T)), _ptr(cu_seqlens), N, B, T, H,
        dk, dv, _dtype_code(k), ctypes.c_float(mu), ctypes.c_float(scale), _stream(dev))
    _check(st, "kdn_forward_diag_noalloc")
    return o, S_T, P_T


def forward_iso(q, k, v, alpha, omega, r, S0=None, P0=None, cu_seqlens=None, mu=None,
                scale=None, chunk=0):
    """Isotropic KDN forward; returns (o, S_T, P_T)."""
    return _forward(1, q, k, v, alpha, omega, r, S0, P0, cu_seqlens, mu, scale, chunk)


def decode_step(variant, q, k, v, alpha, omega, r, S, P, slot_idx=None, mu=None, scale=None,
                o=None):
    """One decode step (variant "diag" or "iso"); S, P updated in place; returns o."""
    vid = {"diag": 0, "iso": 1}[variant] if isinstance(variant, str) else int(variant)
    R, H, dk = k.shape
    dv = v.shape[-1]
    _same(k.dtype, q, v, alpha, omega, r)
    if o is None:
        o = torch.empty((R, H, dv), dtype=k.dtype, device=k.device)
    if slot_idx is not None and slot_idx.dtype != torch.int32:
        raise TypeError("slot_idx must be int32")
    mu = float(dk if mu is None else mu)
    scale = float(dk ** -0.5 if scale is None else scale)
    apc = int(alpha.dim() == 3)
    st = lib().kdn_decode_step(vid, _ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(omega), _ptr(r),
                               _ptr(_f32(S)), _ptr(_f32(P)), _ptr(slot_idx), _ptr(o), R,
                               S.shape[0], H, dk, dv, _dtype_code(k), apc, ctypes.c_float(mu),
                               ctypes.c_float(scale), _stream(k.device))
    _check(st, "kdn_decode_step")
    return o


def _gain(variant, k, alpha, omega, r, P0, cu_seqlens, mu, want_phat):
    B, T, H, dk = k.shape
    _same(k.dtype, alpha, omega, r)
    dev = k.device
    N = B if cu_seqlens is None else cu_seqlens.numel() - 1
    mu = float(dk if mu is None else mu)
    gshape = (B, T, H, dk) if variant == 0 else (B, T, H)
    gain = torch.empty(gshape, dtype=torch.float32, device=dev)
    phat = torch.empty(gshape, dtype=torch.float32, device=dev) if want_phat else None
    P_T = torch.empty((N, H, dk) if variant == 0 else (N, H), dtype=torch.float32, device=dev)
    ws_bytes = lib().kdn_gain_workspace_bytes(variant, N, B, T, H, dk)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    args = [_ptr(k), _ptr(alpha), _ptr(omega), _ptr(r), _ptr(_f32(P0)), _ptr(gain), _ptr(phat),
            _ptr(P_T), _ptr(cu_seqlens), N, B, T, H, dk, _dtype_code(k)]
    if variant == 0:
        st = lib().kdn_gain_diag(*args, ctypes.c_float(mu), _ptr(ws), ws_bytes, _stream(dev))
        _check(st, "kdn_gain_diag")
    else:
        apc = int(alpha.dim() == 4)
        st = lib().kdn_gain_iso(*args, apc, ctypes.c_float(mu), _ptr(ws), ws_bytes, _stream(dev))
        _check(st, "kdn_gain_iso")
    return gain, phat, P_T


def gain_diag(k, alpha, omega, r, P0=None, cu_seqlens=None, mu=None, want_phat=True):
    """Gain scan alone (diagonal): returns (kappa, phat or None, P_T)."""
    return _gain(0, k, alpha, omega, r, P0, cu_seqlens, mu, want_phat)


def gain_iso(k, alpha, omega, r, P0=None, cu_seqlens=None, mu=None, want_phat=True):
    """Gain scan alone (isotropic): returns (beta, bhat or None, P_T)."""
    return _gain(1, k, alpha, omega, r, P0, cu_seqlens, mu, want_phat)


def _layer_opts(gates_preact, r_min, qk_l2norm, mu_t, beta_eff):
    return LayerOpts(int(bool(gates_preact)), float(r_min), int(bool(qk_l2norm)),
                     None if mu_t is None else mu_t.data_ptr(),
                     None if beta_eff is None else beta_eff.data_ptr())


def forward_layer(variant, q, k, v, alpha, omega, r, S0=None, P0=None, cu_seqlens=None, mu=None,
                  scale=None, gates_preact=False, r_min=0.01, qk_l2norm=False, mu_t=None,
                  want_beta_eff=False):
    """The forward with the layer options (variant "diag" or "iso"); alpha, omega and r are
    pre-activations when gates_preact. Returns (o, S_T, P_T, beta_eff or None)."""
    vid = {"diag": 0, "iso": 1}[variant] if isinstance(variant, str) else int(variant)
    B, T, H, dk = k.shape
    dv = v.shape[-1]
    _same(k.dtype, q, v, alpha, omega, r, mu_t)
    dev = k.device
    N = B if cu_seqlens is None else cu_seqlens.numel() - 1
    mu = float(dk if mu is None else mu)
    scale = float(dk ** -0.5 if scale is None else scale)
    if cu_seqlens is not None and cu_seqlens.dtype != torch.int32:
        raise TypeError("cu_seqlens must be int32")
    if mu_t is not None:
        _ptr(mu_t)
    o = torch.empty((B, T, H, dv), dtype=k.dtype, device=dev)
    S_T = torch.empty((N, H, dk, dv), dtype=torch.float32, device=dev)
    P_T = torch.empty((N, H, dk) if vid == 0 else (N, H), dtype=torch.float32, device=dev)
    beff = torch.empty((B, T, H), dtype=torch.float32, device=dev) if want_beta_eff else None
    ws_bytes = lib().kdn_forward_workspace_bytes(vid, N, B, T, H, dk, dv, _dtype_code(k),
                                                 int(cu_seqlens is not None), 0)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev) if ws_bytes else None
    opts = _layer_opts(gates_preact, r_min, qk_l2norm, mu_t, beff)
    apc = int(vid == 0 or alpha.dim() == 4)
    st = lib().kdn_forward_layer(vid, _ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(omega),
                                 _ptr(r), _ptr(_f32(S0)), _ptr(_f32(P0)), _ptr(o), _ptr(S_T),
                                 _ptr(P_T), _ptr(cu_seqlens), N, B, T, H, dk, dv, _dtype_code(k),
                                 apc, ctypes.c_float(mu), ctypes.c_float(scale),
                                 ctypes.byref(opts), _ptr(ws), ws_bytes, _stream(dev))
    _check(st, "kdn_forward_layer")
    return o, S_T, P_T, beff


def decode_step_layer(variant, q, k, v, alpha, omega, r, S, P, slot_idx=None, mu=None,
                      scale=None, o=None, gates_preact=False, r_min=0.01, qk_l2norm=False,
                      mu_t=None, beta_eff=None):
    """One decode step with the layer options; S, P (and beta_eff [R,H] float32 when given)
    updated in place; returns o."""
    vid = {"diag": 0, "iso": 1}[variant] if isinstance(variant, str) else int(variant)
    R, H, dk = k.shape
    dv = v.shape[-1]
    _same(k.dtype, q, v, alpha, omega, r, mu_t)
    if o is None:
        o = torch.empty((R, H, dv), dtype=k.dtype, device=k.device)
    if slot_idx is not None and slot_idx.dtype != torch.int32:
        raise TypeError("slot_idx must be int32")
    if beta_eff is not None and (beta_eff.dtype != torch.float32 or not beta_eff.is_contiguous()):
        raise TypeError("beta_eff must be a contiguous float32 tensor")
    if mu_t is not None:
        _ptr(mu_t)
    mu = float(dk if mu is None else mu)
    scale = float(dk ** -0.5 if scale is None else scale)
    apc = int(alpha.dim() == 3)
    opts = _layer_opts(gates_preact, r_min, qk_l2norm, mu_t, beta_eff)
    st = lib().kdn_decode_step_layer(vid, _ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(omega),
                                     _ptr(r), _ptr(_f32(S)), _ptr(_f32(P)), _ptr(slot_idx),
                                     _ptr(o), R, S.shape[0], H, dk, dv, _dtype_code(k), apc,
                                     ctypes.c_float(mu), ctypes.c_float(scale),
                                     ctypes.byref(opts), _stream(k.device))
    _check(st, "kdn_decode_step_layer")
    return o


def backward(variant, q, k, v, alpha, omega, r, S0=None, P0=None, cu_seqlens=None, mu=None,
             scale=None, dO=None, dS_T=None, dP_T=None):
    """Gradients of a loss through the forward, given its gradients dO (input dtype), dS_T and
    dP_T (float32); None = zero. Returns a dict of float32 tensors dq, dk, dv, dalpha, domega,
    dr, dS0, dP0 shaped like the inputs (dS0 / dP0 like S_T / P_T)."""
    vid = {"diag": 0, "iso": 1}[variant] if isinstance(variant, str) else int(variant)
    B, T, H, dk = k.shape
    dv = v.shape[-1]
    _same(k.dtype, q, v, alpha, omega, r, dO)
    dev = k.device
    N = B if cu_seqlens is None else cu_seqlens.numel() - 1
    mu = float(dk if mu is None else mu)
    scale = float(dk ** -0.5 if scale is None else scale)
    if cu_seqlens is not None and cu_seqlens.dtype != torch.int32:
        raise TypeError("cu_seqlens must be int32")
    f32 = dict(dtype=torch.float32, device=dev)
    g = dict(dq=torch.empty(q.shape, **f32), dk=torch.empty(k.shape, **f32),
             dv=torch.empty(v.shape, **f32), dalpha=torch.empty(alpha.shape, **f32),
             domega=torch.empty(omega.shape, **f32), dr=torch.empty(r.shape, **f32),
             dS0=torch.empty((N, H, dk, dv), **f32),
             dP0=torch.empty((N, H, dk) if vid == 0 else (N, H), **f32))
    ws_bytes = lib().kdn_backward_workspace_bytes(vid, N, B, T, H, dk, dv,
                                                  int(cu_seqlens is not None))
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    apc = int(vid == 0 or alpha.dim() == 4)
    st = lib().kdn_backward(vid, _ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(omega), _ptr(r),
                            _ptr(_f32(S0)), _ptr(_f32(P0)), _ptr(cu_seqlens), N, B, T, H, dk, dv,
                            _dtype_code(k), apc, ctypes.c_float(mu), ctypes.c_float(scale),
                            _ptr(dO), _ptr(_f32(dS_T)), _ptr(_f32(dP_T)), _ptr(g["dq"]),
                            _ptr(g["dk"]), _ptr(g["dv"]), _ptr(g["dalpha"]), _ptr(g["domega"]),
                            _ptr(g["dr"]), _ptr(g["dS0"]), _ptr(g["dP0"]), _ptr(ws), ws_bytes,
                            _stream(dev))
    _check(st, "kdn_backward")
    return g


def forward_kam(q, k, v, alpha, omega, r, S0=None, P0=None, cu_seqlens=None, scale=None):
    """Kalman Associative Memory (dense dk x dk covariance); returns (o, S_T, P_T)."""
    B, T, H, dk = k.shape
    dv = v.shape[-1]
    _same(k.dtype, q, v, alpha, omega, r)
    dev = k.device
    N = B if cu_seqlens is None else cu_seqlens.numel() - 1
    scale = float(dk ** -0.5 if scale is None else scale)
    if cu_seqlens is not None and cu_seqlens.dtype != torch.int32:
        raise TypeError("cu_seqlens must be int32")
    o = torch.empty((B, T, H, dv), dtype=k.dtype, device=dev)
    S_T = torch.empty((N, H, dk, dv), dtype=torch.float32, device=dev)
    P_T = torch.empty((N, H, dk, dk), dtype=torch.float32, device=dev)
    st = lib().kdn_forward_kam(_ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(omega), _ptr(r),
                               _ptr(_f32(S0)), _ptr(_f32(P0)), _ptr(o), _ptr(S_T), _ptr(P_T),
                               _ptr(cu_seqlens), N, B, T, H, dk, dv, _dtype_code(k),
                               ctypes.c_float(scale), _stream(dev))
    _check(st, "kdn_forward_kam")
    return o, S_T, P_T
