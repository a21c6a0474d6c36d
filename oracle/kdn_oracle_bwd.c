/*
 * kdn_oracle_bwd.c -- reverse-mode adjoint of the KDN recurrences (CPU oracle, float64).
 *
 * TEST INFRASTRUCTURE ONLY. Only tests/, __graft_entry__.smoke() and the benchmark's CPU
 * baseline may call this code; the GPU library never links or calls it.
 *
 * Paper: arXiv 2609.07816. The forward recurrences are those of Prop. "Diagonal Kalman Delta
 * Network" (eqs. kla-box-mobius, kla-box-gain, kla-box-memory, with the information scale of
 * eq. diag-cov-update) and Prop. "Isotropic Kalman Delta Network" (eqs.
 * iso-kla-box-cov-update, iso-kla-box-gain, iso-kla-box-memory), exactly as in kdn_oracle.c.
 * The paper trains through them (its kernels are differentiated; App. "Detailed Experimental
 * Setup"); it does not print the adjoint, so the one here is the plain chain rule applied to the
 * forward's steps in reverse order:
 *   - per (sequence, head) the forward runs once and keeps S_{t-1} and p_{t-1} of every token;
 *   - the reverse sweep starts from the caller's adjoints of S_T and P_T, adds the adjoint of
 *     o_t at each token and takes every forward assignment back in turn:
 *       o = scale S^T q;  p = p_hat / (1 + u p_hat);  S = S_hat + kappa delta^T;
 *       delta = v - S_hat^T k;  S_hat = diag(alpha) S_prev;  the gain (kappa or beta k);
 *       u = mu k^2 / r (diagonal) or mu ||k||^2 / (dk r) (isotropic);
 *       p_hat = alpha^2 p_prev + omega (diagonal) or a b_prev + omega with
 *       a = mean_i alpha_i^2 (isotropic).
 * Nothing is blocked or reordered: the sweep is the token recurrence itself, run backwards.
 * Pinned by central finite differences of the forward oracle (tests/test_oracle_backward.py).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <omp.h>

typedef struct {
    int t0, len;
} bspan;

static int bspan_of(const int32_t* cu, int n, int T, bspan* s)
{
    if (!cu) {
        s->t0 = n * T;
        s->len = T;
        return 0;
    }
    s->t0 = cu[n];
    s->len = cu[n + 1] - cu[n];
    return s->len < 0 ? -1 : 0;
}

/*
 * Gradients of a scalar loss through one forward call, given its adjoints dO [B,T,H,dv],
 * dS_T [N,H,dk,dv] and dP_T [N,H,dk] (diagonal) / [N,H] (isotropic); each may be NULL (zero).
 * Inputs are those of the forward (S0 / P0 NULL = 0 / 1; mu_t NULL = mu everywhere). Outputs,
 * every one the shape of its input and overwritten: dq, dk, dv, dalpha, domega, dr, dS0
 * [N,H,dk,dv], dP0 (shape of P_T), and dmu_t [B,T,H] when not NULL. variant 0 = diagonal,
 * 1 = isotropic (alpha per channel when alpha_per_channel, else one gate per head).
 */
int oracle_kdn_backward(int variant, const double* q, const double* k, const double* v,
                        const double* alpha, const double* omega, const double* r,
                        const double* S0, const double* P0, const int32_t* cu_seqlens, int N,
                        int B, int T, int H, int dk, int dv, int alpha_per_channel, double mu,
                        double scale, const double* mu_t, const double* dO, const double* dS_T,
                        const double* dP_T, double* dq, double* dkk, double* dvv, double* dalpha,
                        double* domega, double* dr, double* dS0, double* dP0, double* dmu_t,
                        int nthreads)
{
    if (variant != 0 && variant != 1) return -1;
    if (N <= 0 || B <= 0 || T < 0 || H <= 0 || dk <= 0 || dv <= 0) return -1;
    if (!cu_seqlens && N != B) return -1;
    const int diag = variant == 0;
    const int apc = diag || alpha_per_channel;
    const int pc = diag ? dk : 1;              /* variance entries per head */
    const int64_t rows = (int64_t)B * T * H;
    memset(dq, 0, sizeof(double) * rows * dk);
    memset(dkk, 0, sizeof(double) * rows * dk);
    memset(dvv, 0, sizeof(double) * rows * dv);
    memset(dalpha, 0, sizeof(double) * rows * (apc ? dk : 1));
    memset(domega, 0, sizeof(double) * rows * (diag ? dk : 1));
    memset(dr, 0, sizeof(double) * rows);
    if (dmu_t) memset(dmu_t, 0, sizeof(double) * rows);
    for (int n = 0; n < N; ++n) {
        bspan s;
        if (bspan_of(cu_seqlens, n, T, &s)) return -1;
    }
    if (nthreads > 0) omp_set_num_threads(nthreads);
    int bad = 0;
#pragma omp parallel for schedule(dynamic) reduction(| : bad)
    for (int nh = 0; nh < N * H; ++nh) {
        const int n = nh / H, h = nh % H;
        bspan s;
        bspan_of(cu_seqlens, n, T, &s);
        const int L = s.len;
        const size_t SZ = (size_t)dk * dv;
        double* Sh = malloc(sizeof(double) * SZ * ((size_t)L + 1)); /* S_{t-1}, t = 0..L */
        double* Ph = malloc(sizeof(double) * pc * ((size_t)L + 1));  /* p_{t-1}          */
        double* ph = malloc(sizeof(double) * dk);
        double* kap = malloc(sizeof(double) * dk);
        double* del = malloc(sizeof(double) * dv);
        double* Shat = malloc(sizeof(double) * SZ);
        double* Sbar = malloc(sizeof(double) * SZ);
        double* dSh = malloc(sizeof(double) * SZ);
        double* pbar = malloc(sizeof(double) * pc);
        double* dkap = malloc(sizeof(double) * dk);
        double* ddel = malloc(sizeof(double) * dv);
        double* dph = malloc(sizeof(double) * dk);
        if (!Sh || !Ph || !ph || !kap || !del || !Shat || !Sbar || !dSh || !pbar ||
            !dkap || !ddel || !dph) {
            bad |= 1;
        } else {
            /* ---- forward, keeping the state before every token ---- */
            for (size_t e = 0; e < SZ; ++e) Sh[e] = S0 ? S0[(size_t)nh * SZ + e] : 0.0;
            for (int i = 0; i < pc; ++i) Ph[i] = P0 ? P0[(size_t)nh * pc + i] : 1.0;
            for (int t = 0; t < L; ++t) {
                const int64_t row = ((int64_t)(s.t0 + t)) * H + h;
                const double *qt = q + row * dk, *kt = k + row * dk, *vt = v + row * dv;
                const double* at = alpha + row * (apc ? dk : 1);
                const double rt = r[row], mut = mu_t ? mu_t[row] : mu;
                const double* Sp = Sh + (size_t)t * SZ;
                double* Sn = Sh + (size_t)(t + 1) * SZ;
                const double* pp = Ph + (size_t)t * pc;
                double* pn = Ph + (size_t)(t + 1) * pc;
                (void)qt;
                if (diag) {
                    const double* wt = omega + row * dk;
                    double den = rt;
                    for (int i = 0; i < dk; ++i) {
                        ph[i] = at[i] * at[i] * pp[i] + wt[i];
                        den += ph[i] * kt[i] * kt[i];
                    }
                    for (int i = 0; i < dk; ++i) kap[i] = ph[i] * kt[i] / den;
                    for (int i = 0; i < dk; ++i) {
                        const double u = mut * kt[i] * kt[i] / rt;
                        pn[i] = ph[i] / (1.0 + u * ph[i]);
                    }
                } else {
                    double a = 0.0, nk = 0.0;
                    for (int i = 0; i < dk; ++i) nk += kt[i] * kt[i];
                    if (apc) {
                        for (int i = 0; i < dk; ++i) a += at[i] * at[i];
                        a /= (double)dk;
                    } else {
                        a = at[0] * at[0];
                    }
                    const double bh = a * pp[0] + omega[row];
                    const double beta = bh / (rt + bh * nk);
                    for (int i = 0; i < dk; ++i) kap[i] = beta * kt[i];
                    const double u = mut * nk / ((double)dk * rt);
                    pn[0] = bh / (1.0 + u * bh);
                }
                for (int i = 0; i < dk; ++i) {
                    const double ai = apc ? at[i] : at[0];
                    for (int j = 0; j < dv; ++j) Shat[i * dv + j] = ai * Sp[i * dv + j];
                }
                for (int j = 0; j < dv; ++j) {
                    double acc = 0.0;
                    for (int i = 0; i < dk; ++i) acc += Shat[i * dv + j] * kt[i];
                    del[j] = vt[j] - acc;
                }
                for (int i = 0; i < dk; ++i)
                    for (int j = 0; j < dv; ++j) Sn[i * dv + j] = Shat[i * dv + j] + kap[i] * del[j];
            }

            /* ---- reverse sweep ---- */
            for (size_t e = 0; e < SZ; ++e) Sbar[e] = dS_T ? dS_T[(size_t)nh * SZ + e] : 0.0;
            for (int i = 0; i < pc; ++i) pbar[i] = dP_T ? dP_T[(size_t)nh * pc + i] : 0.0;
            for (int t = L - 1; t >= 0; --t) {
                const int64_t row = ((int64_t)(s.t0 + t)) * H + h;
                const double *qt = q + row * dk, *kt = k + row * dk;
                const double* at = alpha + row * (apc ? dk : 1);
                const double rt = r[row], mut = mu_t ? mu_t[row] : mu;
                const double* Sp = Sh + (size_t)t * SZ;
                const double* Sn = Sh + (size_t)(t + 1) * SZ;
                const double* pp = Ph + (size_t)t * pc;
                double *dqt = dq + row * dk, *dkt = dkk + row * dk, *dvt = dvv + row * dv;
                double* dat = dalpha + row * (apc ? dk : 1);
                double drt = 0.0, dmut = 0.0;

                /* recompute the token's forward quantities from S_{t-1}, p_{t-1} */
                double den = rt, nk = 0.0, a = 0.0, bh = 0.0, beta = 0.0;
                for (int i = 0; i < dk; ++i) nk += kt[i] * kt[i];
                if (diag) {
                    const double* wt = omega + row * dk;
                    for (int i = 0; i < dk; ++i) {
                        ph[i] = at[i] * at[i] * pp[i] + wt[i];
                        den += ph[i] * kt[i] * kt[i];
                    }
                    for (int i = 0; i < dk; ++i) kap[i] = ph[i] * kt[i] / den;
                } else {
                    if (apc) {
                        for (int i = 0; i < dk; ++i) a += at[i] * at[i];
                        a /= (double)dk;
                    } else {
                        a = at[0] * at[0];
                    }
                    bh = a * pp[0] + omega[row];
                    den = rt + bh * nk;
                    beta = bh / den;
                    for (int i = 0; i < dk; ++i) kap[i] = beta * kt[i];
                }
                for (int i = 0; i < dk; ++i) {
                    const double ai = apc ? at[i] : at[0];
                    for (int j = 0; j < dv; ++j) Shat[i * dv + j] = ai * Sp[i * dv + j];
                }
                for (int j = 0; j < dv; ++j) {
                    double acc = 0.0;
                    for (int i = 0; i < dk; ++i) acc += Shat[i * dv + j] * kt[i];
                    del[j] = v[row * dv + j] - acc;
                }

                /* o = scale S_t^T q */
                if (dO) {
                    const double* dot = dO + row * dv;
                    for (int i = 0; i < dk; ++i) {
                        double acc = 0.0;
                        for (int j = 0; j < dv; ++j) {
                            acc += Sn[i * dv + j] * dot[j];
                            Sbar[i * dv + j] += scale * qt[i] * dot[j];
                        }
                        dqt[i] = scale * acc;
                    }
                }
                /* p = p_hat / (1 + u p_hat): adjoints of p_hat and of u */
                double du_iso = 0.0;
                for (int i = 0; i < dk; ++i) dph[i] = 0.0;
                if (diag) {
                    for (int i = 0; i < dk; ++i) {
                        const double u = mut * kt[i] * kt[i] / rt;
                        const double g = 1.0 + u * ph[i];
                        dph[i] = pbar[i] / (g * g);
                        const double du = -pbar[i] * ph[i] * ph[i] / (g * g);
                        /* u = mu k^2 / r */
                        dkt[i] += du * 2.0 * mut * kt[i] / rt;
                        drt -= du * mut * kt[i] * kt[i] / (rt * rt);
                        dmut += du * kt[i] * kt[i] / rt;
                    }
                } else {
                    const double u = mut * nk / ((double)dk * rt);
                    const double g = 1.0 + u * bh;
                    dph[0] = pbar[0] / (g * g);
                    du_iso = -pbar[0] * bh * bh / (g * g);
                }
                /* S_t = S_hat + kappa delta^T */
                for (int i = 0; i < dk; ++i) {
                    double acc = 0.0;
                    for (int j = 0; j < dv; ++j) acc += Sbar[i * dv + j] * del[j];
                    dkap[i] = acc;
                }
                for (int j = 0; j < dv; ++j) {
                    double acc = 0.0;
                    for (int i = 0; i < dk; ++i) acc += Sbar[i * dv + j] * kap[i];
                    ddel[j] = acc;
                }
                /* delta = v - S_hat^T k */
                for (int j = 0; j < dv; ++j) dvt[j] = ddel[j];
                for (int i = 0; i < dk; ++i) {
                    double acc = 0.0;
                    for (int j = 0; j < dv; ++j) {
                        acc += Shat[i * dv + j] * ddel[j];
                        dSh[i * dv + j] = Sbar[i * dv + j] - kt[i] * ddel[j];
                    }
                    dkt[i] -= acc;
                }
                /* S_hat = diag(alpha) S_{t-1} */
                for (int i = 0; i < dk; ++i) {
                    const double ai = apc ? at[i] : at[0];
                    double acc = 0.0;
                    for (int j = 0; j < dv; ++j) {
                        acc += Sp[i * dv + j] * dSh[i * dv + j];
                        Sbar[i * dv + j] = ai * dSh[i * dv + j];
                    }
                    if (apc) dat[i] += acc;
                    else dat[0] += acc;
                }
                if (diag) {
                    /* kappa_i = p_hat_i k_i / den, den = r + sum_l p_hat_l k_l^2 */
                    double dden = 0.0;
                    for (int i = 0; i < dk; ++i) dden -= dkap[i] * kap[i] / den;
                    for (int i = 0; i < dk; ++i) {
                        dph[i] += dkap[i] * kt[i] / den + dden * kt[i] * kt[i];
                        dkt[i] += dkap[i] * ph[i] / den + dden * 2.0 * ph[i] * kt[i];
                    }
                    drt += dden;
                    /* p_hat = alpha^2 p_{t-1} + omega */
                    double* dwt = domega + row * dk;
                    for (int i = 0; i < dk; ++i) {
                        dat[i] += dph[i] * 2.0 * at[i] * pp[i];
                        dwt[i] = dph[i];
                        pbar[i] = dph[i] * at[i] * at[i];
                    }
                } else {
                    /* kappa = beta k */
                    double dbeta = 0.0;
                    for (int i = 0; i < dk; ++i) {
                        dbeta += dkap[i] * kt[i];
                        dkt[i] += beta * dkap[i];
                    }
                    /* beta = b_hat / (r + b_hat ||k||^2) */
                    double dbh = dph[0] + dbeta * rt / (den * den);
                    drt -= dbeta * bh / (den * den);
                    double dnk = -dbeta * bh * bh / (den * den);
                    /* u = mu ||k||^2 / (dk r) */
                    dnk += du_iso * mut / ((double)dk * rt);
                    drt -= du_iso * mut * nk / ((double)dk * rt * rt);
                    dmut += du_iso * nk / ((double)dk * rt);
                    for (int i = 0; i < dk; ++i) dkt[i] += 2.0 * kt[i] * dnk;
                    /* b_hat = a b_{t-1} + omega, a = mean_i alpha_i^2 (or alpha^2) */
                    const double da = dbh * pp[0];
                    domega[row] = dbh;
                    pbar[0] = dbh * a;
                    if (apc)
                        for (int i = 0; i < dk; ++i) dat[i] += da * 2.0 * at[i] / (double)dk;
                    else
                        dat[0] += da * 2.0 * at[0];
                }
                dr[row] = drt;
                if (dmu_t) dmu_t[row] = dmut;
            }
            for (size_t e = 0; e < SZ; ++e) dS0[(size_t)nh * SZ + e] = Sbar[e];
            for (int i = 0; i < pc; ++i) dP0[(size_t)nh * pc + i] = pbar[i];
        }
        free(Sh); free(Ph); free(ph); free(kap); free(del); free(Shat); free(Sbar);
        free(dSh); free(pbar); free(dkap); free(ddel); free(dph);
    }
    return bad ? -2 : 0;
}
