"""Pins of the oracle's layer maps, per-token information scale and effective-write output
(no GPU).

The gate maps are checked against identities of sigmoid and softplus that hold exactly in real
arithmetic (symmetry, inverses, derivatives by central differences), not against a retyped
formula. The per-token information scale is checked against the scalar-mu recurrence run one
token at a time, against the closed-form variance update and its derivatives (App. "Overwrite
and Protection-Write Decoupling", eqs. appendix-protection-scale-update,
appendix-protection-current-invariance and appendix-protection-future-write), and the effective
write against its residual identity (eqs. appendix-effective-write and
appendix-effective-write-residual).
"""

import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def rng(*s):
    return np.random.default_rng(list(s))


# ------------------------------------------------------------------------------------------
# Gate maps (eqs. kla-box-parameterization and iso-kla-box-parameterization).
# ------------------------------------------------------------------------------------------

def test_sigmoid_identities():
    x = np.concatenate([np.linspace(-40, 40, 801), [-745.0, -700.0, 700.0, 0.0]])
    s = oracle.sigmoid(x)
    assert oracle.sigmoid(0.0) == 0.5
    np.testing.assert_allclose(s + oracle.sigmoid(-x), 1.0, rtol=0, atol=4.5e-16)
    assert np.all((s >= 0) & (s <= 1)) and np.all(np.diff(s[:801]) >= 0)
    assert np.all(np.diff(s[100:701]) > 0)
    mid = np.abs(x) < 30
    # sigmoid(x) / sigmoid(-x) = exp(x): the ratio form keeps 1 - s from cancelling
    np.testing.assert_allclose(np.log(s[mid]) - np.log(oracle.sigmoid(-x[mid])), x[mid],
                               rtol=1e-13, atol=1e-13)
    # the tails: sigmoid(x) ~ exp(x) for x -> -inf, no overflow for large |x|
    np.testing.assert_allclose(oracle.sigmoid(-700.0), np.exp(-700.0), rtol=1e-15)
    assert oracle.sigmoid(700.0) == 1.0


def test_softplus_identities():
    x = np.linspace(-40, 40, 801)
    sp = oracle.softplus(x)
    assert oracle.softplus(0.0) == np.log(2.0)
    np.testing.assert_allclose(sp - oracle.softplus(-x), x, rtol=0, atol=1e-13)
    mid = np.abs(x) < 30
    np.testing.assert_allclose(np.exp(sp[mid]), 1 + np.exp(x[mid]), rtol=1e-13)
    assert np.all(sp > 0)
    # large arguments: softplus(x) = x + log1p(exp(-x)) without overflow
    assert oracle.softplus(1000.0) == 1000.0
    np.testing.assert_allclose(oracle.softplus(-700.0), np.exp(-700.0), rtol=1e-15)


def test_softplus_derivative_is_sigmoid():
    x = np.linspace(-12, 12, 97)
    h = 1e-5
    d = (oracle.softplus(x + h) - oracle.softplus(x - h)) / (2 * h)
    np.testing.assert_allclose(d, oracle.sigmoid(x), rtol=0, atol=1e-9)


def test_l2_normalize():
    g = rng(40)
    x = g.standard_normal((5, 7, 3, 16)) * g.uniform(0.01, 100, (5, 7, 3, 1))
    y = oracle.l2_normalize(x)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), 1.0, rtol=1e-15)
    # direction kept: y is a positive multiple of x
    c = np.sum(x * y, axis=-1) / np.linalg.norm(x, axis=-1)
    np.testing.assert_allclose(c, 1.0, rtol=1e-14)
    z = np.zeros((2, 4))
    np.testing.assert_array_equal(oracle.l2_normalize(z), z)


def test_layer_inputs_ranges_and_scale_invariance():
    g = rng(41)
    T, H, dk = 9, 2, 8
    q, k = g.standard_normal((2, 1, T, H, dk))
    a_pre, w_pre = g.standard_normal((2, 1, T, H, dk)) * 3
    r_pre = g.standard_normal((1, T, H)) * 3
    qq, kk, a, w, r = oracle.layer_inputs(q, k, a_pre, w_pre, r_pre, 0.01)
    assert np.all((a > 0) & (a < 1)) and np.all(w > 0) and np.all(r > 0.01)
    # r - r_min is softplus, and r_min is a floor approached as the pre-activation falls
    np.testing.assert_allclose(oracle.layer_inputs(q, k, a_pre, w_pre, np.full_like(r_pre, -60),
                                                   0.01)[4], 0.01, rtol=1e-15)
    # normalised queries and keys make the recurrence blind to their scales
    v = g.standard_normal((1, T, H, 4))
    out1 = oracle.forward_diag(qq, kk, v, a, w, r)
    q2, k2, *_ = oracle.layer_inputs(q * 7.5, k * 0.01, a_pre, w_pre, r_pre, 0.01)
    out2 = oracle.forward_diag(q2, k2, v, a, w, r)
    np.testing.assert_allclose(out2["o"], out1["o"], rtol=1e-12, atol=1e-14)


# ------------------------------------------------------------------------------------------
# Per-token information scale mu_t (eq. appendix-protection-scale-update).
# ------------------------------------------------------------------------------------------

def _draw(g, B, T, H, dk, dv, iso_head_alpha=False):
    q = oracle.l2_normalize(g.standard_normal((B, T, H, dk)))
    k = oracle.l2_normalize(g.standard_normal((B, T, H, dk)))
    v = g.standard_normal((B, T, H, dv))
    a = g.uniform(0.3, 1.0, (B, T, H) if iso_head_alpha else (B, T, H, dk))
    w = g.uniform(0.01, 0.5, (B, T, H, dk))
    r = g.uniform(0.05, 1.0, (B, T, H))
    mu_t = g.uniform(1.0, 2.0 * dk, (B, T, H))
    return q, k, v, a, w, r, mu_t


@pytest.mark.parametrize("variant", ["diag", "iso"])
def test_constant_mu_t_equals_scalar_mu(variant):
    g = rng(42)
    q, k, v, a, w, r, _ = _draw(g, 2, 30, 2, 8, 4)
    if variant == "iso":
        w = w[..., 0]
    f = oracle.forward_diag if variant == "diag" else oracle.forward_iso
    ref = f(q, k, v, a, w, r, mu=5.5)
    out = f(q, k, v, a, w, r, mu=123.0, mu_t=np.full(r.shape, 5.5))
    for name in ("o", "S_T", "P_T"):
        np.testing.assert_array_equal(out[name], ref[name])


@pytest.mark.parametrize("variant", ["diag", "iso"])
def test_per_token_mu_equals_steps_with_that_mu(variant):
    """Running token t with scalar mu = mu_t[t] one decode step at a time gives the forward with
    the per-token array: the array is read at each token's own index."""
    g = rng(43)
    B, T, H, dk, dv = 2, 25, 3, 8, 4
    q, k, v, a, w, r, mu_t = _draw(g, B, T, H, dk, dv)
    if variant == "iso":
        w = w[..., 0]
    f = oracle.forward_diag if variant == "diag" else oracle.forward_iso
    full = f(q, k, v, a, w, r, mu_t=mu_t, beta_eff=True)
    S = np.zeros((B, H, dk, dv))
    P = np.ones((B, H, dk)) if variant == "diag" else np.ones((B, H))
    for t in range(T):
        for h in range(H):
            sl = lambda x: np.ascontiguousarray(x[:, t, h:h + 1])  # noqa: E731
            Sh, Ph = np.ascontiguousarray(S[:, h:h + 1]), np.ascontiguousarray(P[:, h:h + 1])
            for b in range(B):
                Sb, Pb = Sh[b:b + 1].copy(), Ph[b:b + 1].copy()
                be = np.zeros((1, 1))
                o = oracle.decode_step(variant, *(sl(x)[b:b + 1] for x in (q, k, v, a, w, r)),
                                       Sb, Pb, mu=float(mu_t[b, t, h]), beta_eff=be)
                np.testing.assert_allclose(o[0, 0], full["o"][b, t, h], rtol=1e-13, atol=1e-15)
                np.testing.assert_allclose(be[0, 0], full["beta_eff"][b, t, h], rtol=1e-14)
                S[b, h], P[b, h] = Sb[0, 0], Pb[0, 0]
    np.testing.assert_allclose(S, full["S_T"], rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(P, full["P_T"], rtol=1e-13)


def test_mu_t_closed_form_variance_update():
    """p_t = (phat_t^-1 + mu_t k_t^2 / r_t)^-1 channel by channel, with phat_t from the trace."""
    g = rng(44)
    q, k, v, a, w, r, mu_t = _draw(g, 1, 40, 1, 8, 3)
    out = oracle.forward_diag(q, k, v, a, w, r, mu_t=mu_t, traces=True)
    want = 1.0 / (1.0 / out["phat"] + mu_t[..., None] * k * k / r[..., None])
    np.testing.assert_allclose(out["p"], want, rtol=1e-14)
    # and phat_{t+1} = alpha_{t+1}^2 p_t + omega_{t+1} links consecutive tokens
    np.testing.assert_allclose(out["phat"][:, 1:], a[:, 1:] ** 2 * out["p"][:, :-1] + w[:, 1:],
                               rtol=1e-14)


def test_mu_t_current_invariance_and_future_protection():
    """Perturbing mu at one token leaves that token's gain, output and memory unchanged; the
    variance moves with derivative -k^2 p^2 / r, and the next token's z and effective write move
    with the derivatives of eq. appendix-protection-future-write (central differences)."""
    g = rng(45)
    T, dk, dv, t0 = 12, 8, 3, 6
    q, k, v, a, w, r, mu_t = _draw(g, 1, T, 1, dk, dv)
    base = oracle.forward_diag(q, k, v, a, w, r, mu_t=mu_t, traces=True, beta_eff=True)
    h = 1e-4 * mu_t[0, t0, 0]
    runs = []
    for s in (+1, -1):
        m = mu_t.copy()
        m[0, t0, 0] += s * h
        runs.append(oracle.forward_diag(q, k, v, a, w, r, mu_t=m, traces=True, beta_eff=True))
    up, dn = runs
    for name in ("kappa", "o"):
        np.testing.assert_array_equal(up[name][:, :t0 + 1], base[name][:, :t0 + 1])
    dp = (up["p"][0, t0, 0] - dn["p"][0, t0, 0]) / (2 * h)
    kk, pp, rr = k[0, t0, 0], base["p"][0, t0, 0], r[0, t0, 0]
    np.testing.assert_allclose(dp, -kk ** 2 * pp ** 2 / rr, rtol=1e-7)
    z = lambda o: np.sum(o["phat"][0, t0 + 1, 0] * k[0, t0 + 1, 0] ** 2)  # noqa: E731
    dz = (z(up) - z(dn)) / (2 * h)
    want_dz = -np.sum(a[0, t0 + 1, 0] ** 2 * pp ** 2 * kk ** 2 * k[0, t0 + 1, 0] ** 2) / rr
    np.testing.assert_allclose(dz, want_dz, rtol=1e-7)
    assert want_dz <= 0
    r1, z1 = r[0, t0 + 1, 0], z(base)
    db = (up["beta_eff"][0, t0 + 1, 0] - dn["beta_eff"][0, t0 + 1, 0]) / (2 * h)
    np.testing.assert_allclose(db, r1 / (r1 + z1) ** 2 * want_dz, rtol=1e-6)


# ------------------------------------------------------------------------------------------
# Effective write (eqs. appendix-effective-write, appendix-effective-write-residual).
# ------------------------------------------------------------------------------------------

@pytest.mark.parametrize("variant", ["diag", "iso"])
def test_beta_eff_residual_identity(variant):
    """v_t - S_t^T k_t = (1 - beta_eff_t)(v_t - Shat_t^T k_t) with Shat_t = diag(alpha_t) S_{t-1},
    with S_{t-1}, S_t taken from forwards of lengths t and t + 1."""
    g = rng(46)
    T, dk, dv = 10, 8, 5
    q, k, v, a, w, r, _ = _draw(g, 1, T, 1, dk, dv)
    if variant == "iso":
        w = w[..., 0]
    f = oracle.forward_diag if variant == "diag" else oracle.forward_iso
    full = f(q, k, v, a, w, r, beta_eff=True)
    be = full["beta_eff"][0, :, 0]
    assert np.all((be > 0) & (be < 1))
    S_prev = np.zeros((dk, dv))
    for t in range(T):
        S_t = f(*(x[:, :t + 1] for x in (q, k, v, a, w, r)))["S_T"][0, 0]
        kt, vt = k[0, t, 0], v[0, t, 0]
        S_hat = a[0, t, 0][:, None] * S_prev
        np.testing.assert_allclose(vt - S_t.T @ kt, (1 - be[t]) * (vt - S_hat.T @ kt),
                                   rtol=1e-12, atol=1e-14)
        S_prev = S_t


def test_beta_eff_from_variance_traces():
    """Diagonal: beta_eff = z / (r + z) with z = sum_i phat_i k_i^2 (the gain's own
    denominator); isotropic: beta ||k||^2 from the beta trace."""
    g = rng(47)
    q, k, v, a, w, r, _ = _draw(g, 2, 20, 2, 8, 3)
    d = oracle.forward_diag(q, k, v, a, w, r, traces=True, beta_eff=True)
    z = np.sum(d["phat"] * k * k, axis=-1)
    np.testing.assert_allclose(d["beta_eff"], z / (r + z), rtol=1e-14)
    i = oracle.forward_iso(q, k, v, a, w[..., 0], r, traces=True, beta_eff=True)
    np.testing.assert_allclose(i["beta_eff"], i["beta"] * np.sum(k * k, axis=-1), rtol=1e-15)
