"""Seeded synthetic inputs for the KDN hot path.

This module only draws random numbers and rounds them to the storage dtype. It holds none of the
KDN arithmetic, so both the HIP path and the CPU oracle can consume its output without sharing any
of the method's code.

Workload shapes follow the paper's mixer layers (16 heads of width 128 at d_model = 2048, 4K
training context, throughput probe at batch 4; Sec. "Experiments", mixer-throughput figure). The
paper's data (FineWeb-Edu and its evaluation suites) is not available, so every tensor here is a
synthetic stand-in drawn from fixed laws:

* q, k ~ N(0, 1), then divided by their L2 norm over the key dimension (normalised keys, as in
  the fixed-gain reduction of Sec. 3.3), computed in float64 and only then rounded;
* v ~ N(0, 1);
* transition gates alpha = sigmoid(N(0,1) + 2);
* process and observation noise omega, r = softplus(N(0,1)) + 1e-3;
* optional initial state S0 ~ N(0, 0.02^2) and initial variances P0 ~ U(0.1, 1).

Each tensor comes from its own generator ``numpy.random.default_rng([seed, stream, id])`` so that
changing one shape never perturbs another tensor. bf16 values are rounded to nearest-even on the
host; the float64 view of the rounded bits is exactly what both sides compute on.
"""

from __future__ import annotations

import dataclasses
from typing import Dict, Optional, Sequence

import numpy as np

# stream ids (one independent generator per tensor)
SID_Q, SID_K, SID_V, SID_ALPHA, SID_OMEGA, SID_R, SID_S0, SID_P0, SID_LEN = range(9)


# ---------------------------------------------------------------------------------------------
# bf16 helpers (round-to-nearest-even on the float32 bit pattern)
# ---------------------------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest-even); returns the 16-bit patterns (uint16)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    rounding = 0x7FFF + ((u >> 16) & 1)
    out = ((u + rounding) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 data to the storage dtype; returns the stored array (float32 or uint16)."""
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "bf16":
        return f32_to_bf16_bits(np.asarray(x, dtype=np.float32))
    raise ValueError(f"unknown dtype {dtype!r}")


def to_f64(stored: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 view of stored values (bf16 bits or float32)."""
    if dtype == "bf16":
        return bf16_bits_to_f32(stored).astype(np.float64)
    return np.asarray(stored, dtype=np.float32).astype(np.float64)


# ---------------------------------------------------------------------------------------------
# laws
# ---------------------------------------------------------------------------------------------

def _rng(seed: int, stream: int, sid: int) -> np.random.Generator:
    return np.random.default_rng([seed, stream, sid])


def _softplus(x: np.ndarray) -> np.ndarray:
    return np.maximum(x, 0.0) + np.log1p(np.exp(-np.abs(x)))


def _sigmoid(x: np.ndarray) -> np.ndarray:
    return 1.0 / (1.0 + np.exp(-x))


def _unit_rows(x: np.ndarray) -> np.ndarray:
    n = np.sqrt(np.sum(x * x, axis=-1, keepdims=True))
    return x / n


@dataclasses.dataclass
class KdnInputs:
    """One batch of inputs in storage form plus its float64 view.

    Shapes: q, k [B, T, H, dk]; v [B, T, H, dv]; alpha [B, T, H, dk] or [B, T, H];
    omega [B, T, H, dk] (diagonal) or [B, T, H] (isotropic); r [B, T, H];
    S0 [N, H, dk, dv] or None; P0 [N, H, dk] / [N, H] or None; cu_seqlens [N + 1] or None.
    """

    variant: str
    dtype: str
    B: int
    T: int
    H: int
    dk: int
    dv: int
    alpha_per_channel: bool
    stored: Dict[str, np.ndarray]
    cu_seqlens: Optional[np.ndarray] = None
    S0: Optional[np.ndarray] = None  # float32
    P0: Optional[np.ndarray] = None  # float32
    mu: float = 0.0
    scale: float = 0.0

    @property
    def N(self) -> int:
        return self.B if self.cu_seqlens is None else len(self.cu_seqlens) - 1

    def f64(self, name: str) -> np.ndarray:
        return to_f64(self.stored[name], self.dtype)

    def tokens(self) -> int:
        return self.B * self.T


def _law(rng: np.random.Generator, shape, law, default):
    """Values of one tensor: ``default(rng, shape)`` unless ``law`` overrides it with
    ("uniform", lo, hi), ("const", c) or ("spikes", base, low, frac): ``base`` everywhere except
    a random fraction ``frac`` of the entries, which take the value ``low``."""
    if law is None:
        return default(rng, shape)
    kind = law[0]
    if kind == "uniform":
        return rng.uniform(law[1], law[2], shape)
    if kind == "const":
        return np.full(shape, float(law[1]))
    if kind == "spikes":
        x = np.full(shape, float(law[1]))
        x[rng.random(shape) < law[3]] = float(law[2])
        return x
    raise ValueError(f"unknown law {law!r}")


def draw_inputs(variant: str, dtype: str, B: int, T: int, H: int, dk: int, dv: int, *,
                seed: int, stream: int = 0, alpha_per_channel: bool = True,
                lengths: Optional[Sequence[int]] = None, random_state: bool = False,
                mu: Optional[float] = None, scale: Optional[float] = None,
                alpha_law=None, omega_law=None, r_law=None) -> KdnInputs:
    """Draw one batch.

    ``variant`` is "diag" or "iso". With ``lengths`` the batch is packed (B must be 1 and T the
    total length). ``random_state`` draws S0 ~ N(0, 0.02^2) and P0 ~ U(0.1, 1) per sequence;
    otherwise both are None (the method's defaults S0 = 0 and P0 = 1 apply). ``alpha_law``,
    ``omega_law`` and ``r_law`` replace the default laws of the gates and noise terms (see
    ``_law``; used by the stress tests: small or unit gates, zero process noise, tiny r).
    """
    if variant not in ("diag", "iso"):
        raise ValueError(variant)
    cu = None
    if lengths is not None:
        lengths = [int(x) for x in lengths]
        if B != 1 or sum(lengths) != T:
            raise ValueError("packed batch needs B == 1 and T == sum(lengths)")
        cu = np.zeros(len(lengths) + 1, dtype=np.int32)
        cu[1:] = np.cumsum(lengths)
    N = B if cu is None else len(cu) - 1

    st = {}
    st["q"] = round_to(_unit_rows(_rng(seed, stream, SID_Q).standard_normal((B, T, H, dk))), dtype)
    st["k"] = round_to(_unit_rows(_rng(seed, stream, SID_K).standard_normal((B, T, H, dk))), dtype)
    st["v"] = round_to(_rng(seed, stream, SID_V).standard_normal((B, T, H, dv)), dtype)
    ashape = (B, T, H, dk) if (variant == "diag" or alpha_per_channel) else (B, T, H)
    st["alpha"] = round_to(_law(_rng(seed, stream, SID_ALPHA), ashape, alpha_law,
                                lambda g, sh: _sigmoid(g.standard_normal(sh) + 2.0)), dtype)
    oshape = (B, T, H, dk) if variant == "diag" else (B, T, H)
    st["omega"] = round_to(_law(_rng(seed, stream, SID_OMEGA), oshape, omega_law,
                                lambda g, sh: _softplus(g.standard_normal(sh)) + 1e-3), dtype)
    st["r"] = round_to(_law(_rng(seed, stream, SID_R), (B, T, H), r_law,
                            lambda g, sh: _softplus(g.standard_normal(sh)) + 1e-3), dtype)
    S0 = P0 = None
    if random_state:
        S0 = (0.02 * _rng(seed, stream, SID_S0).standard_normal((N, H, dk, dv))).astype(np.float32)
        pshape = (N, H, dk) if variant == "diag" else (N, H)
        P0 = _rng(seed, stream, SID_P0).uniform(0.1, 1.0, pshape).astype(np.float32)
    return KdnInputs(variant=variant, dtype=dtype, B=B, T=T, H=H, dk=dk, dv=dv,
                     alpha_per_channel=(variant == "diag" or alpha_per_channel), stored=st,
                     cu_seqlens=cu, S0=S0, P0=P0,
                     mu=float(dk if mu is None else mu),
                     scale=float(dk ** -0.5 if scale is None else scale))


SID_MU_T = 9


def draw_layer_inputs(variant: str, dtype: str, B: int, T: int, H: int, dk: int, dv: int, *,
                      seed: int, stream: int = 0, alpha_per_channel: bool = True,
                      lengths: Optional[Sequence[int]] = None, random_state: bool = False,
                      mu_t: bool = False) -> KdnInputs:
    """One batch of the layer's inputs, before the layer's maps: the stored "alpha", "omega"
    and "r" are pre-activations and q, k are not normalised.

    * q, k ~ N(0, 1) per element times a per-(token, head) scale ~ U(0.25, 4), so that rows of
      very different norms reach the normalisation;
    * gate pre-activations ~ N(2, 1) (their sigmoid has the law of the plain workloads' gates);
    * process- and observation-noise pre-activations ~ N(0, 1);
    * with ``mu_t`` a per-token information scale ~ U(dk / 4, 2 dk), stored as "mu_t".
    Everything else (v, lengths, S0, P0, mu, scale) is drawn as in ``draw_inputs``.
    """
    x = draw_inputs(variant, dtype, B, T, H, dk, dv, seed=seed, stream=stream,
                    alpha_per_channel=alpha_per_channel, lengths=lengths,
                    random_state=random_state)
    g = _rng(seed, stream + 1, SID_Q)
    scale_q = g.uniform(0.25, 4.0, (B, T, H, 1))
    x.stored["q"] = round_to(g.standard_normal((B, T, H, dk)) * scale_q, dtype)
    g = _rng(seed, stream + 1, SID_K)
    scale_k = g.uniform(0.25, 4.0, (B, T, H, 1))
    x.stored["k"] = round_to(g.standard_normal((B, T, H, dk)) * scale_k, dtype)
    ashape = x.stored["alpha"].shape
    x.stored["alpha"] = round_to(_rng(seed, stream + 1, SID_ALPHA).standard_normal(ashape) + 2.0,
                                 dtype)
    oshape = x.stored["omega"].shape
    x.stored["omega"] = round_to(_rng(seed, stream + 1, SID_OMEGA).standard_normal(oshape), dtype)
    x.stored["r"] = round_to(_rng(seed, stream + 1, SID_R).standard_normal((B, T, H)), dtype)
    if mu_t:
        x.stored["mu_t"] = round_to(_rng(seed, stream + 1, SID_MU_T).uniform(dk / 4, 2 * dk,
                                                                              (B, T, H)), dtype)
    return x


def draw_lengths(n: int, lo: int, hi: int, seed: int, stream: int = 0) -> np.ndarray:
    """Sequence lengths uniform on the integers [lo, hi]."""
    return _rng(seed, stream, SID_LEN).integers(lo, hi + 1, size=n)


# ---------------------------------------------------------------------------------------------
# the five workloads (seed = 1000 + id)
# ---------------------------------------------------------------------------------------------

WORKLOADS = {
    0: dict(name="tiny-f32", B=1, H=2, T=64, dk=16, dv=16, dtype="f32", chunk=16),
    1: dict(name="iso-fwd-B4-H16-T2048-d128", variant="iso", B=4, H=16, T=2048, dk=128, dv=128,
            dtype="bf16", alpha_per_channel=False),
    2: dict(name="diag-fwd-B4-H16-T4096-d128", variant="diag", B=4, H=16, T=4096, dk=128,
            dv=128, dtype="bf16"),
    3: dict(name="diag-varlen-32seq-U256-8192-H16-d128", variant="diag", n_seq=32, lo=256,
            hi=8192, H=16, dk=128, dv=128, dtype="bf16"),
    4: dict(name="decode-R256-H16-d128-64steps", R=256, H=16, dk=128, dv=128, steps=64,
            prefill_T=1024, dtype="bf16"),
}


def workload_seed(wid: int) -> int:
    return 1000 + wid


def draw_workload(wid: int, variant: Optional[str] = None, alpha_per_channel: bool = True
                  ) -> KdnInputs:
    """Inputs of forward workloads 0-3 (workload 0 needs ``variant``)."""
    w = WORKLOADS[wid]
    seed = workload_seed(wid)
    if wid == 0:
        return draw_inputs(variant or "diag", "f32", w["B"], w["T"], w["H"], w["dk"], w["dv"],
                           seed=seed, alpha_per_channel=alpha_per_channel)
    if wid in (1, 2):
        return draw_inputs(w["variant"], w["dtype"], w["B"], w["T"], w["H"], w["dk"], w["dv"],
                           seed=seed, alpha_per_channel=w.get("alpha_per_channel", True))
    if wid == 3:
        lens = draw_lengths(w["n_seq"], w["lo"], w["hi"], seed)
        return draw_inputs("diag", w["dtype"], 1, int(lens.sum()), w["H"], w["dk"], w["dv"],
                           seed=seed, lengths=lens, random_state=True)
    raise ValueError("workload 4 is drawn with draw_decode_prefill / draw_decode_step")


def draw_decode_prefill(variant: str, R: int = 256, H: int = 16, d: int = 128, T: int = 1024,
                        dtype: str = "bf16", seed: int = 1004) -> KdnInputs:
    """Prefill batch used to initialise the decode states (channel-wise gates for both variants)."""
    return draw_inputs(variant, dtype, R, T, H, d, d, seed=seed, stream=0, alpha_per_channel=True)


def draw_decode_step(variant: str, step: int, R: int = 256, H: int = 16, d: int = 128,
                     dtype: str = "bf16", seed: int = 1004) -> KdnInputs:
    """Inputs of one decode step: a T = 1 batch over R rows (stream 100 + step)."""
    return draw_inputs(variant, dtype, R, 1, H, d, d, seed=seed, stream=100 + step,
                       alpha_per_channel=True)
