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


# ---------------------------------------------------------------------------------------------
# float32 model of how the kernels form the intra-chunk products
# ---------------------------------------------------------------------------------------------

def intra_chunk_exact(k, q, alpha, G):
    """Exact (float64, per pair) intra-chunk products of one chunk:
    M_ts = sum_i k_ti (prod_{s < j <= t} alpha_ji) G_si k_si and M^q with q in place of k, for
    s <= t (zero above the diagonal). k, q, alpha, G: [C, dk]."""
    C = k.shape[0]
    M, Mq = np.zeros((C, C)), np.zeros((C, C))
    for t in range(C):
        for s in range(t + 1):
            ratio = np.prod(alpha[s + 1:t + 1], axis=0)  # empty product = 1
            w = ratio * G[s] * k[s]
            M[t, s] = np.dot(k[t], w)
            Mq[t, s] = np.dot(q[t], w)
    return M, Mq


def intra_chunk_f32(k, q, alpha, G, scheme):
    """The same products as the GPU forms them, every operand and product in float32.

    scheme "chunk_start": gamma_t = prod_{j <= t} alpha_j from the chunk start, K_bar = gamma k and
    P_bar = G k / gamma (one factorisation for the whole chunk).
    scheme "blocks": 16-token blocks; inside a diagonal block both sides are referenced to its
    midpoint, F_t = prod_{8 <= j <= t} alpha_j or 1 / prod_{t < j <= 7} alpha_j (reciprocals
    saturated at 2^126); for a pair of distinct blocks (b > c) the rows are referenced to the
    start of block b, the columns to the end of block c, and the decay of the blocks between
    them scales the columns."""
    f = np.float32
    k, q, alpha, G = (np.asarray(x, dtype=f) for x in (k, q, alpha, G))
    C, dk = k.shape
    M, Mq = np.zeros((C, C), f), np.zeros((C, C), f)
    with np.errstate(over="ignore", invalid="ignore", divide="ignore", under="ignore"):
        if scheme == "chunk_start":
            gam = np.cumprod(alpha, axis=0, dtype=f)
            Kb, Qb, Pb = gam * k, gam * q, (G * k) / gam
            M, Mq = np.tril(Kb @ Pb.T), np.tril(Qb @ Pb.T)
            return M, Mq
        assert scheme == "blocks" and C % 16 == 0
        sat = lambda x: np.minimum(f(1) / np.maximum(x, f(2.0 ** -126)), f(2.0 ** 126))
        nb = C // 16
        blk = [slice(16 * b, 16 * b + 16) for b in range(nb)]
        for b in range(nb):
            a = alpha[blk[b]]
            F = np.ones((16, dk), f)
            acc = np.ones(dk, f)
            for j in range(7, -1, -1):          # t < 8: 1 / prod_{t < j <= 7} alpha
                F[j] = sat(acc)
                acc = acc * a[j]
            Pm = np.ones((16, dk), f)
            acc = np.ones(dk, f)
            for j in range(7, -1, -1):          # column side, t < 8: prod_{t < j <= 7} alpha
                Pm[j] = acc
                acc = acc * a[j]
            acc = np.ones(dk, f)
            for j in range(8, 16):              # t >= 8: prod_{8 <= j <= t} alpha
                acc = acc * a[j]
                F[j] = acc
                Pm[j] = sat(acc)
            Kt, Qt, Pt = k[blk[b]] * F, q[blk[b]] * F, (G * k)[blk[b]] * Pm
            M[blk[b], blk[b]] = np.tril(Kt @ Pt.T)
            Mq[blk[b], blk[b]] = np.tril(Qt @ Pt.T)
        start = [np.cumprod(alpha[blk[b]], axis=0, dtype=f) for b in range(nb)]   # incl. t
        end = []
        for b in range(nb):                       # prod_{s < j <= end of block}
            a = alpha[blk[b]]
            e = np.ones((16, dk), f)
            acc = np.ones(dk, f)
            for j in range(15, -1, -1):
                e[j] = acc
                acc = acc * a[j]
            end.append(e)
        gblk = [np.prod(alpha[blk[b]], axis=0, dtype=f) for b in range(nb)]
        for ib in range(nb):
            for jb in range(ib):
                rho = np.ones(dk, f)
                for m in range(jb + 1, ib):
                    rho = rho * gblk[m]
                Kr, Qr = k[blk[ib]] * start[ib], q[blk[ib]] * start[ib]
                Pc = (G * k)[blk[jb]] * end[jb] * rho
                M[blk[ib], blk[jb]] = Kr @ Pc.T
                Mq[blk[ib], blk[jb]] = Qr @ Pc.T
    return M, Mq
