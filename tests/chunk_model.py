"""Float64 NumPy model of the chunkwise compact-WY memory scan (tests only).

Written from App. "Hardware-Efficient Chunkwise Algorithm", Sec. "Chunkwise Memory Scan"
(eqs. chunk-memory-normalization, chunk-memory-scaled-keys, chunk-memory-wy,
chunk-memory-tail-output, chunk-memory-output-state). Given the gains kappa_t, the memory
recurrence S_t = (I - kappa_t k_t^T) diag(alpha_t) S_{t-1} + kappa_t v_t^T with o_t = tau S_t^T q_t
is evaluated chunk by chunk; only S^in crosses chunk boundaries. It shares nothing with the
oracle and is used to show that the chunked algebra the kernels rely on is exact.
"""

from __future__ import annotations

import numpy as np


def chunk_forward(q, k, v, alpha, kappa, S0, C, scale):
    """One (sequence, head): q, k, alpha, kappa [T, dk]; v [T, dv]; S0 [dk, dv].
    Returns (o [T, dv], S_T [dk, dv])."""
    T, dk = k.shape
    S = np.array(S0, dtype=np.float64, copy=True)
    O = np.zeros((T, v.shape[1]))
    for c0 in range(0, T, C):
        sl = slice(c0, min(c0 + C, T))
        L = sl.stop - sl.start
        gamma = np.cumprod(alpha[sl], axis=0)          # gamma_r = prod_{j <= r} alpha_j
        Kb = gamma * k[sl]                              # K_bar = Gamma (.) K
        Kk = kappa[sl] / gamma                          # K_bar^(kappa) = K^(kappa) (/) Gamma
        Qb = scale * gamma * q[sl]                      # Q_bar = tau Gamma (.) Q
        Tm = np.tril(Kb @ Kk.T, -1)
        A = np.linalg.inv(np.eye(L) + Tm)
        W = A @ Kb
        U = A @ v[sl]
        R = U - W @ S
        Aqk = np.tril(Qb @ Kk.T)                        # diagonal included (read after write)
        O[sl] = Qb @ S + Aqk @ R
        Ktail = (gamma[-1] / gamma) * kappa[sl]
        S = gamma[-1][:, None] * S + Ktail.T @ R
    return O, S


def chunk_forward_lsolve(q, k, v, alpha, gainvec, diag, S0, C, scale):
    """The same recurrence in the form the fused GPU kernel evaluates, with the gain's
    normalisation moved into a lower-triangular solve. Per chunk, with gamma as above,
        K_bar = Gamma (.) K,  Q_bar = tau Gamma (.) Q,  P_bar = G (.) K (/) Gamma,
        L = diag(c) + tril(K_bar P_bar^T, -1),  R = L^-1 (V - K_bar S),
        O = Q_bar S + tril(Q_bar P_bar^T) R,  S <- gamma_C (.) (S + P_bar^T R),
    where, for the diagonal variant, G = p_hat (the predictive variances) and
    c = r + diag(K_bar P_bar^T) (the innovation variances r + sum_i p_hat_i k_i^2), and for the
    isotropic variant G = beta (one gain per token, broadcast over the channels) and c = 1.
    Row t of R is the innovation of token t divided by c_t.
    gainvec: diagonal -> (phat [T, dk], r [T]); isotropic -> beta [T]."""
    T, dk = k.shape
    S = np.array(S0, dtype=np.float64, copy=True)
    O = np.zeros((T, v.shape[1]))
    for c0 in range(0, T, C):
        sl = slice(c0, min(c0 + C, T))
        gamma = np.cumprod(alpha[sl], axis=0)
        Kb = gamma * k[sl]
        Qb = scale * gamma * q[sl]
        if diag:
            phat, r = gainvec
            Pb = phat[sl] * k[sl] / gamma
            G = Kb @ Pb.T
            c = r[sl] + np.diag(G)
        else:
            Pb = gainvec[sl][:, None] * k[sl] / gamma
            G = Kb @ Pb.T
            c = np.ones(sl.stop - sl.start)
        Lm = np.diag(c) + np.tril(G, -1)
        R = np.linalg.solve(Lm, v[sl] - Kb @ S)
        O[sl] = Qb @ S + np.tril(Qb @ Pb.T) @ R
        S = gamma[-1][:, None] * (S + Pb.T @ R)
    return O, S
