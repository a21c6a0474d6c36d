"""Pins of the oracle's reverse-mode adjoint (oracle.backward) by central finite differences of
the forward oracle (no GPU).

The loss is L = <W_o, o> + <W_S, S_T> + <W_P, P_T> with fixed random weights, so the adjoints
handed to the backward are dO = W_o, dS_T = W_S, dP_T = W_P. Every element of every input (q, k,
v, the gates, the noise terms, the initial state and variances, the per-token information scale)
is perturbed by +-h, and the centred difference of L is compared with the backward's gradient.
The forward oracle is itself pinned against independent references (test_oracle_pins.py), so a
match here ties the adjoint to the paper's recurrences (Prop. "Diagonal Kalman Delta Network",
Prop. "Isotropic Kalman Delta Network").
"""

import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _inputs(variant, B, T, H, dk, dv, seed, per_channel=True, lengths=None):
    g = np.random.default_rng(seed)
    x = dict(q=g.standard_normal((B, T, H, dk)), k=g.standard_normal((B, T, H, dk)) * 0.6,
             v=g.standard_normal((B, T, H, dv)),
             alpha=g.uniform(0.4, 0.99, (B, T, H, dk) if per_channel else (B, T, H)),
             omega=g.uniform(0.05, 0.6, (B, T, H, dk) if variant == "diag" else (B, T, H)),
             r=g.uniform(0.2, 1.5, (B, T, H)))
    N = B if lengths is None else len(lengths)
    x["S0"] = 0.3 * g.standard_normal((N, H, dk, dv))
    x["P0"] = g.uniform(0.2, 1.2, (N, H, dk) if variant == "diag" else (N, H))
    x["mu_t"] = g.uniform(0.5, 3.0 * dk, (B, T, H))
    return x


def _loss_fn(variant, x, W, cu, mu, use_mu_t):
    f = oracle.forward_diag if variant == "diag" else oracle.forward_iso

    def loss(y):
        out = f(y["q"], y["k"], y["v"], y["alpha"], y["omega"], y["r"], S0=y["S0"], P0=y["P0"],
                cu_seqlens=cu, mu=mu, scale=0.7, mu_t=y["mu_t"] if use_mu_t else None)
        return (np.sum(W["o"] * out["o"]) + np.sum(W["S"] * out["S_T"]) +
                np.sum(W["P"] * out["P_T"]))
    return loss


def _check_fd(variant, x, cu=None, mu=3.0, use_mu_t=False, seed=0, rtol=2e-6):
    g = np.random.default_rng(seed + 1000)
    out = (oracle.forward_diag if variant == "diag" else oracle.forward_iso)(
        x["q"], x["k"], x["v"], x["alpha"], x["omega"], x["r"], S0=x["S0"], P0=x["P0"],
        cu_seqlens=cu, mu=mu, scale=0.7)
    W = dict(o=g.standard_normal(out["o"].shape), S=g.standard_normal(out["S_T"].shape),
             P=g.standard_normal(out["P_T"].shape))
    grads = oracle.backward(variant, x["q"], x["k"], x["v"], x["alpha"], x["omega"], x["r"],
                            S0=x["S0"], P0=x["P0"], cu_seqlens=cu, mu=mu, scale=0.7,
                            mu_t=x["mu_t"] if use_mu_t else None, dO=W["o"], dS_T=W["S"],
                            dP_T=W["P"])
    loss = _loss_fn(variant, x, W, cu, mu, use_mu_t)
    names = ["q", "k", "v", "alpha", "omega", "r", "S0", "P0"] + (["mu_t"] if use_mu_t else [])
    for name in names:
        gk = {"S0": "dS0", "P0": "dP0"}.get(name, "d" + name)
        G = grads[gk]
        X = x[name]
        fd = np.zeros_like(X)
        for idx in np.ndindex(X.shape):
            h = 1e-6 * max(1.0, abs(X[idx]))
            y = dict(x)
            y[name] = X.copy()
            y[name][idx] = X[idx] + h
            lp = loss(y)
            y[name][idx] = X[idx] - h
            lm = loss(y)
            fd[idx] = (lp - lm) / (2 * h)
        scale = max(1.0, np.max(np.abs(fd)))
        err = np.max(np.abs(G - fd)) / scale
        assert err < rtol, f"{variant} d{name}: max error {err:.2e} (scale {scale:.2e})"


@pytest.mark.parametrize("variant,per_channel", [("diag", True), ("iso", True),
                                                 ("iso", False)])
def test_backward_matches_finite_differences(variant, per_channel):
    x = _inputs(variant, 2, 6, 2, 4, 3, seed=80, per_channel=per_channel)
    _check_fd(variant, x, seed=80)


@pytest.mark.parametrize("variant", ["diag", "iso"])
def test_backward_per_token_mu(variant):
    x = _inputs(variant, 1, 5, 2, 3, 2, seed=81)
    _check_fd(variant, x, use_mu_t=True, seed=81)


@pytest.mark.parametrize("variant", ["diag", "iso"])
def test_backward_packed_with_empty_sequence(variant):
    lens = [3, 0, 5, 1]
    x = _inputs(variant, 1, sum(lens), 2, 3, 2, seed=82, lengths=lens)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    _check_fd(variant, x, cu=cu, seed=82)


def test_backward_empty_sequence_passes_state_adjoints_through():
    """A sequence without tokens maps S0 -> S_T and P0 -> P_T by the identity, so its dS0 and
    dP0 are the incoming adjoints themselves."""
    lens = [2, 0]
    x = _inputs("diag", 1, 2, 1, 3, 2, seed=83, lengths=lens)
    cu = np.array([0, 2, 2], dtype=np.int32)
    g = np.random.default_rng(84)
    dS, dP = g.standard_normal((2, 1, 3, 2)), g.standard_normal((2, 1, 3))
    out = oracle.backward("diag", x["q"], x["k"], x["v"], x["alpha"], x["omega"], x["r"],
                          S0=x["S0"], P0=x["P0"], cu_seqlens=cu, dS_T=dS, dP_T=dP)
    np.testing.assert_array_equal(out["dS0"][1], dS[1])
    np.testing.assert_array_equal(out["dP0"][1], dP[1])


def test_backward_of_output_only_is_linear_in_dO():
    """The gradients are linear in the incoming adjoints: backward(a dO1 + b dO2) equals
    a backward(dO1) + b backward(dO2)."""
    x = _inputs("diag", 1, 9, 1, 4, 3, seed=85)
    g = np.random.default_rng(86)
    d1, d2 = g.standard_normal((2, 1, 9, 1, 3))
    args = [x[n] for n in ("q", "k", "v", "alpha", "omega", "r")]
    g1 = oracle.backward("diag", *args, S0=x["S0"], P0=x["P0"], dO=d1)
    g2 = oracle.backward("diag", *args, S0=x["S0"], P0=x["P0"], dO=d2)
    g3 = oracle.backward("diag", *args, S0=x["S0"], P0=x["P0"], dO=2.0 * d1 - 0.5 * d2)
    for name in g1:
        np.testing.assert_allclose(g3[name], 2.0 * g1[name] - 0.5 * g2[name], rtol=1e-12,
                                   atol=1e-12)
