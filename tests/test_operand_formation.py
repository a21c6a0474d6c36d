"""The intra-chunk decay products in the float32 form the GPU kernels use (tests/chunk_model.py),
against the exact per-pair products (App. "Hardware-Efficient Chunkwise Algorithm", Sec.
"Chunkwise Memory Scan": the decay ratios gamma_t / gamma_s of the chunkwise WY form).

A single chunk-start factorisation (K_bar = gamma k, P_bar = G k / gamma) overflows once a
channel's decay over the chunk falls below 2^-126 (a gate of 0.2 held for 64 tokens); the block
references the kernels use stay finite and exact for every gate down to the floor documented in
the header (decay over 8 tokens >= 2^-126)."""

import numpy as np
import pytest

from chunk_model import intra_chunk_exact, intra_chunk_f32


def _draw(alpha_fn, seed, dk=16, C=64):
    g = np.random.default_rng(seed)
    k = g.standard_normal((C, dk))
    k /= np.linalg.norm(k, axis=1, keepdims=True)
    q = g.standard_normal((C, dk))
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    G = g.uniform(0.2, 2.0, (C, dk))
    alpha = alpha_fn(g, (C, dk)).astype(np.float32).astype(np.float64)
    return k.astype(np.float32).astype(np.float64), q.astype(np.float32).astype(np.float64), \
        alpha, G.astype(np.float32).astype(np.float64)


def _rel(a, b):
    return np.linalg.norm(a - b) / np.linalg.norm(b)


def test_chunk_start_reference_overflows_for_small_gates():
    k, q, a, G = _draw(lambda g, sh: np.full(sh, 0.2), seed=1)
    M, Mq = intra_chunk_f32(k, q, a, G, "chunk_start")
    assert not np.all(np.isfinite(M)), "0.2^64 underflows float32: the old form must fail here"


@pytest.mark.parametrize("law", ["const0.2", "uniform0.01-0.3", "workload", "ones",
                                 "uniform1e-4-1e-2"])
def test_block_references_are_exact(law):
    fns = {
        "const0.2": lambda g, sh: np.full(sh, 0.2),
        "uniform0.01-0.3": lambda g, sh: g.uniform(0.01, 0.3, sh),
        "workload": lambda g, sh: 1.0 / (1.0 + np.exp(-(g.standard_normal(sh) + 2.0))),
        "ones": lambda g, sh: np.ones(sh),
        "uniform1e-4-1e-2": lambda g, sh: g.uniform(1e-4, 1e-2, sh),
    }
    k, q, a, G = _draw(fns[law], seed=2)
    M, Mq = intra_chunk_f32(k, q, a, G, "blocks")
    Me, Mqe = intra_chunk_exact(k, q, a, G)
    assert np.all(np.isfinite(M)) and np.all(np.isfinite(Mq))
    assert _rel(M.astype(np.float64), Me) < 1e-6
    assert _rel(Mq.astype(np.float64), Mqe) < 1e-6
    # entrywise: every entry is within float32 rounding of the exact value, relative to the
    # magnitude of its row (no cancellation-free entry may be lost)
    scale = np.abs(Me).max(axis=1, keepdims=True) + 1e-300
    assert np.max(np.abs(M - Me) / scale) < 1e-5


def test_block_references_stay_finite_below_the_floor():
    # gates of 1e-6 on a fifth of the tokens: some 8-token decays fall below 2^-126, where the
    # midpoint factors saturate; the products must stay finite
    k, q, a, G = _draw(lambda g, sh: np.where(g.random(sh) < 0.2, 1e-6, 0.9), seed=3)
    M, Mq = intra_chunk_f32(k, q, a, G, "blocks")
    assert np.all(np.isfinite(M)) and np.all(np.isfinite(Mq))
