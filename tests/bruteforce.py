"""Brute-force references used to pin the oracle (tests only).

None of this is the KDN recurrence. It is textbook Gaussian filtering written in information form
(Bayes' rule for a Gaussian prior and a linear-Gaussian observation), dense linear algebra, and
numerical minimisation of the reverse KL divergence, so that a mistake in the oracle's closed
forms cannot be reproduced here by construction.

Model (paper, Sec. 3.1, eqs. mem-update-dynamics and mem-update-observation): the latent memory
has i.i.d. value columns with a shared key-space covariance; the transition is S~ = D S~ + W with
W ~ N_col(0, Omega); the observation is v = S~^T k + e with e ~ N(0, r I).
"""

from __future__ import annotations

import numpy as np
from scipy import optimize


def predict(S, P, D, Omega):
    """Moments of D X + W for X ~ N_col(S, P), W ~ N_col(0, Omega) (linear map of a Gaussian)."""
    return D @ S, D @ P @ D.T + Omega


def condition(S_hat, P_hat, k, v, r):
    """Posterior of N_col(S_hat, P_hat) given v = S^T k + e, e ~ N(0, r I), via the
    information form: precision Lam = P_hat^-1 + k k^T / r and, column by column,
    mean = Lam^-1 (P_hat^-1 s_hat_j + k v_j / r). Returns (mean, covariance, precision)."""
    Pinv = np.linalg.inv(P_hat)
    Lam = Pinv + np.outer(k, k) / r
    P_post = np.linalg.inv(Lam)
    M = P_post @ (Pinv @ S_hat + np.outer(k, v) / r)
    return M, P_post, Lam


def reverse_kl_cov_part(Sigma_q, Lam_p, logdet_p):
    """Covariance-dependent part of KL(N(m, Sigma_q) || N(m, Lam_p^-1)) for equal means."""
    d = Sigma_q.shape[0]
    sign, logdet_q = np.linalg.slogdet(Sigma_q)
    return 0.5 * (np.trace(Lam_p @ Sigma_q) - d + logdet_p - logdet_q)


def project_diag_kl(P_post):
    """argmin over diagonal covariances of KL(N(0, diag(p)) || N(0, P_post)), found numerically
    (BFGS on log p, objective only)."""
    Lam = np.linalg.inv(P_post)
    _, logdet_p = np.linalg.slogdet(P_post)
    d = P_post.shape[0]

    def f(lp):
        return reverse_kl_cov_part(np.diag(np.exp(lp)), Lam, logdet_p)

    x0 = np.log(np.diag(P_post))
    res = optimize.minimize(f, x0, method="BFGS", options=dict(gtol=1e-12, maxiter=10000))
    # polish with Nelder-Mead-free Newton-like refinement via a few more BFGS restarts
    for _ in range(3):
        res = optimize.minimize(f, res.x, method="BFGS", options=dict(gtol=1e-13, maxiter=10000))
    assert d == res.x.shape[0]
    return np.exp(res.x)


def project_iso_kl(P_post):
    """argmin over b > 0 of KL(N(0, b I) || N(0, P_post)), found numerically (bounded scalar)."""
    Lam = np.linalg.inv(P_post)
    _, logdet_p = np.linalg.slogdet(P_post)
    d = P_post.shape[0]

    def f(lb):
        return reverse_kl_cov_part(np.exp(lb) * np.eye(d), Lam, logdet_p)

    ev = np.linalg.eigvalsh(P_post)
    res = optimize.minimize_scalar(f, bounds=(np.log(ev.min()) - 1, np.log(ev.max()) + 1),
                                   method="bounded", options=dict(xatol=1e-13))
    return float(np.exp(res.x))


def project_iso_frobenius(X):
    """Frobenius-nearest multiple of the identity, by linear least squares on vec(X)."""
    d = X.shape[0]
    coef, *_ = np.linalg.lstsq(np.eye(d).reshape(-1, 1), X.reshape(-1), rcond=None)
    return float(coef[0])


def dense_filter(S0, P0, alphas, omegas, ks, vs, rs, qs, scale):
    """Exact dense Kalman filter over a whole sequence (Prop. "Kalman Associative Memory"), with
    diagonal transitions D_t = diag(alpha_t) and process noise Omega_t = diag(omega_t).
    Returns per-token outputs scale * S_t^T q_t and the final (S, P)."""
    S, P = S0.copy(), P0.copy()
    outs = []
    for a, w, k, v, r, q in zip(alphas, omegas, ks, vs, rs, qs):
        S_hat, P_hat = predict(S, P, np.diag(a), np.diag(w))
        S, P, _ = condition(S_hat, P_hat, k, v, r)
        outs.append(scale * S.T @ q)
    return np.array(outs), S, P


def gated_delta_rule(S0, alphas, betas, ks, vs, qs, scale):
    """Plain delta rule in its transition form S_t = (I - beta k k^T) D_t S_{t-1} + beta k v^T
    (paper eq. unified-delta-rule with D_t = diag(alpha_t)); o_t = scale S_t^T q_t."""
    S = S0.copy()
    dk = S.shape[0]
    outs = []
    for a, b, k, v, q in zip(alphas, betas, ks, vs, qs):
        S = (np.eye(dk) - b * np.outer(k, k)) @ np.diag(a) @ S + b * np.outer(k, v)
        outs.append(scale * S.T @ q)
    return np.array(outs), S


def asym_delta_rule(S0, alphas, kappas, ks, vs, qs, scale):
    """Two-key delta rule S_t = (I - kappa k^T) D_t S_{t-1} + kappa v^T (eq. kla-box-memory)."""
    S = S0.copy()
    dk = S.shape[0]
    outs = []
    for a, kap, k, v, q in zip(alphas, kappas, ks, vs, qs):
        S = (np.eye(dk) - np.outer(kap, k)) @ np.diag(a) @ S + np.outer(kap, v)
        outs.append(scale * S.T @ q)
    return np.array(outs), S
