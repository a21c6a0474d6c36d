/*
 * KDN CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, sequential, float64 implementation of the Kalman Delta Network recurrences, written
 * from the paper (Bui, Huang, Ying: "Kalman Delta Networks: Uncertainty-aware Associative
 * Memory", arXiv 2609.07816). It exists to check the HIP path and nothing else: only the tests,
 * the smoke check and the benchmark's CPU-baseline leg may load it. It shares no code, header or
 * table with the GPU library.
 *
 * Citations name the paper's propositions and equations:
 *   Prop. "Diagonal Kalman Delta Network" (Sec. 4.1): eqs. kla-box-parameterization,
 *     kla-box-mobius, kla-box-gain, kla-box-memory; the variance update of eqs.
 *     prefix-diag-uncertainty and diag-cov-update (information scale mu).
 *   Prop. "Isotropic Kalman Delta Network" (App. "Isotropic Kalman Delta Network"): eqs.
 *     iso-kla-box-cov-update, iso-kla-box-mobius, iso-kla-box-gain, iso-kla-box-memory.
 *   App. "Hardware-Efficient Chunkwise Algorithm", Sec. "Chunkwise Gain Computation": the Moebius
 *     form eq. diag-cov-scan and the three-pass chunked scan eqs. chunk-gain-summary,
 *     chunk-gain-carry, chunk-gain-local-prefix, chunk-gain-emission.
 *
 * Layouts (all row-major, contiguous, float64):
 *   q, k [B,T,H,dk]; v [B,T,H,dv]; alpha [B,T,H,dk] (or [B,T,H] for a per-head gate);
 *   omega [B,T,H,dk] (diagonal) or [B,T,H] (isotropic); r [B,T,H];
 *   S [N,H,dk,dv]; P [N,H,dk] (diagonal) or [N,H] (isotropic); o [B,T,H,dv].
 * With cu_seqlens (int32 [N+1]) the batch is packed: B == 1 and sequence n owns tokens
 * [cu[n], cu[n+1]). Without it N == B and every row has length T.
 * S0 == NULL means S0 = 0; P0 == NULL means P0 = 1 (p_0 = 1 in eq. prefix-diag-uncertainty and
 * b_0 = 1 in eq. iso-kla-box-cov-update). S_T / P_T may be NULL.
 *
 * Every function returns 0 on success and -1 on an argument it cannot use.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int64_t t0, len, b; /* first token (within row b), length, batch row */
} seq_span;

static int span_of(const int32_t* cu, int n, int T, seq_span* s)
{
    if (cu) {
        s->b = 0;
        s->t0 = cu[n];
        s->len = (int64_t)cu[n + 1] - cu[n];
        if (s->len < 0) return -1;
    } else {
        s->b = n;
        s->t0 = 0;
        s->len = T;
    }
    return 0;
}

static void set_threads(int nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
}

/* ------------------------------------------------------------------------------------------ */
/* One token of Diagonal KDN for one (sequence, head). Prop. "Diagonal Kalman Delta Network":  */
/*   p_hat = alpha^2 * p + omega                     (eq. diag-covariance-prediction)           */
/*   kappa = p_hat * k / (r + sum_i p_hat_i k_i^2)   (eq. kla-box-gain, pre-write variance)     */
/*   S_hat = diag(alpha) S;  S = S_hat + kappa (v - S_hat^T k)^T     (eq. kla-box-memory,      */
/*        in the residual form of Prop. "Kalman Associative Memory")                          */
/*   o = scale * S^T q                               (read after the write)                    */
/*   u = mu * k^2 / r;  p = p_hat / (1 + u p_hat)    (eqs. prefix-diag-uncertainty,            */
/*                                                    diag-cov-update)                          */
/* S is dk x dv row-major; p has dk entries. phat_out / kappa_out / p_out (dk each) optional.  */
/* ------------------------------------------------------------------------------------------ */
static void diag_step(int dk, int dv, double* S, double* p, const double* q, const double* k,
                      const double* v, const double* alpha, const double* omega, double r,
                      double mu, double scale, double* o, double* phat_out, double* kappa_out,
                      double* p_out, double* beff_out, double* ph, double* kappa, double* delta)
{
    double den = r;
    for (int i = 0; i < dk; ++i) {
        ph[i] = alpha[i] * alpha[i] * p[i] + omega[i];
        den += ph[i] * k[i] * k[i];
    }
    for (int i = 0; i < dk; ++i) kappa[i] = ph[i] * k[i] / den;
    if (beff_out) { /* effective write strength k^T kappa (App. "Overwrite and Protection-Write
                       Decoupling") */
        double b = 0.0;
        for (int i = 0; i < dk; ++i) b += k[i] * kappa[i];
        *beff_out = b;
    }
    /* predicted memory S_hat = diag(alpha) S, stored in place */
    for (int i = 0; i < dk; ++i)
        for (int j = 0; j < dv; ++j) S[(int64_t)i * dv + j] *= alpha[i];
    /* innovation delta = v - S_hat^T k */
    for (int j = 0; j < dv; ++j) {
        double acc = 0.0;
        for (int i = 0; i < dk; ++i) acc += S[(int64_t)i * dv + j] * k[i];
        delta[j] = v[j] - acc;
    }
    for (int i = 0; i < dk; ++i)
        for (int j = 0; j < dv; ++j) S[(int64_t)i * dv + j] += kappa[i] * delta[j];
    if (o) {
        for (int j = 0; j < dv; ++j) {
            double acc = 0.0;
            for (int i = 0; i < dk; ++i) acc += S[(int64_t)i * dv + j] * q[i];
            o[j] = scale * acc;
        }
    }
    for (int i = 0; i < dk; ++i) {
        double u = mu * k[i] * k[i] / r;
        p[i] = ph[i] / (1.0 + u * ph[i]);
    }
    if (phat_out) memcpy(phat_out, ph, sizeof(double) * dk);
    if (kappa_out) memcpy(kappa_out, kappa, sizeof(double) * dk);
    if (p_out) memcpy(p_out, p, sizeof(double) * dk);
}

/* ------------------------------------------------------------------------------------------ */
/* One token of Isotropic KDN for one (sequence, head). Prop. "Isotropic Kalman Delta Network": */
/*   a = mean_i alpha_i^2 (trace projection, eq. iso-kla-predict; = alpha^2 for a scalar gate)  */
/*   b_hat = a b + omega;  beta = b_hat / (r + b_hat ||k||^2)            (eq. iso-kla-box-gain) */
/*   S_hat = diag(alpha) S (the memory keeps the full channel-wise transition)                   */
/*   S = S_hat + beta k (v - S_hat^T k)^T;  o = scale S^T q              (eq. iso-kla-box-memory)*/
/*   u = mu ||k||^2 / (dk r);  b = b_hat / (1 + u b_hat)          (eq. iso-kla-box-cov-update)   */
/* alpha points at dk gates when per_channel, else at one scalar gate.                          */
/* ------------------------------------------------------------------------------------------ */
static void iso_step(int dk, int dv, double* S, double* b, const double* q, const double* k,
                     const double* v, const double* alpha, int per_channel, double omega,
                     double r, double mu, double scale, double* o, double* bhat_out,
                     double* beta_out, double* b_out, double* beff_out, double* delta)
{
    double a = 0.0;
    if (per_channel) {
        for (int i = 0; i < dk; ++i) a += alpha[i] * alpha[i];
        a /= (double)dk;
    } else {
        a = alpha[0] * alpha[0];
    }
    double nk = 0.0;
    for (int i = 0; i < dk; ++i) nk += k[i] * k[i];
    double bh = a * (*b) + omega;
    double beta = bh / (r + bh * nk);
    if (beff_out) *beff_out = beta * nk; /* k^T (beta k) */
    for (int i = 0; i < dk; ++i) {
        double ai = per_channel ? alpha[i] : alpha[0];
        for (int j = 0; j < dv; ++j) S[(int64_t)i * dv + j] *= ai;
    }
    for (int j = 0; j < dv; ++j) {
        double acc = 0.0;
        for (int i = 0; i < dk; ++i) acc += S[(int64_t)i * dv + j] * k[i];
        delta[j] = v[j] - acc;
    }
    for (int i = 0; i < dk; ++i)
        for (int j = 0; j < dv; ++j) S[(int64_t)i * dv + j] += beta * k[i] * delta[j];
    if (o) {
        for (int j = 0; j < dv; ++j) {
            double acc = 0.0;
            for (int i = 0; i < dk; ++i) acc += S[(int64_t)i * dv + j] * q[i];
            o[j] = scale * acc;
        }
    }
    double u = mu * nk / ((double)dk * r);
    *b = bh / (1.0 + u * bh);
    if (bhat_out) *bhat_out = bh;
    if (beta_out) *beta_out = beta;
    if (b_out) *b_out = *b;
}

static int check_dims(int N, int B, int T, int H, int dk, int dv, const int32_t* cu)
{
    if (N <= 0 || B <= 0 || T < 0 || H <= 0 || dk <= 0 || dv <= 0) return -1;
    if (cu && B != 1) return -1;
    if (!cu && N != B) return -1;
    return 0;
}

/* Forward pass of Diagonal KDN over every (sequence, head); optional per-token gain traces.   */
/* mu_t (nullable, [B,T,H]): a per-token information scale in place of mu (App. "Overwrite
   and Protection-Write Decoupling"); beff_out (nullable, [B,T,H]): k_t^T kappa_t per token.   */
int oracle_kdn_forward_diag(const double* q, const double* k, const double* v,
                            const double* alpha, const double* omega, const double* r,
                            const double* S0, const double* P0, double* o, double* S_T,
                            double* P_T, double* phat_out, double* kappa_out, double* p_out,
                            const int32_t* cu_seqlens, int N, int B, int T, int H, int dk,
                            int dv, double mu, double scale, int nthreads, const double* mu_t,
                            double* beff_out)
{
    if (check_dims(N, B, T, H, dk, dv, cu_seqlens)) return -1;
    set_threads(nthreads);
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int64_t chain = 0; chain < (int64_t)N * H; ++chain) {
        int n = (int)(chain / H), h = (int)(chain % H);
        seq_span sp;
        if (span_of(cu_seqlens, n, T, &sp)) { bad |= 1; continue; }
        double* S = (double*)malloc(sizeof(double) * ((size_t)dk * dv + 3 * dk + dv));
        double* p = S + (size_t)dk * dv;
        double* ph = p + dk;
        double* kap = ph + dk;
        double* delta = kap + dk;
        const size_t soff = ((size_t)n * H + h) * dk * dv, poff = ((size_t)n * H + h) * dk;
        for (size_t i = 0; i < (size_t)dk * dv; ++i) S[i] = S0 ? S0[soff + i] : 0.0;
        for (int i = 0; i < dk; ++i) p[i] = P0 ? P0[poff + i] : 1.0;
        for (int64_t t = 0; t < sp.len; ++t) {
            const size_t row = ((size_t)sp.b * T + sp.t0 + t) * H + h; /* (b, t, h) */
            diag_step(dk, dv, S, p, q + row * dk, k + row * dk, v + row * dv,
                      alpha + row * dk, omega + row * dk, r[row], mu_t ? mu_t[row] : mu, scale,
                      o ? o + row * dv : NULL, phat_out ? phat_out + row * dk : NULL,
                      kappa_out ? kappa_out + row * dk : NULL, p_out ? p_out + row * dk : NULL,
                      beff_out ? beff_out + row : NULL, ph, kap, delta);
        }
        if (S_T) memcpy(S_T + soff, S, sizeof(double) * dk * dv);
        if (P_T) memcpy(P_T + poff, p, sizeof(double) * dk);
        free(S);
    }
    return bad ? -1 : 0;
}

/* Forward pass of Isotropic KDN; alpha is [B,T,H,dk] when alpha_per_channel else [B,T,H].    */
int oracle_kdn_forward_iso(const double* q, const double* k, const double* v,
                           const double* alpha, const double* omega, const double* r,
                           const double* S0, const double* P0, double* o, double* S_T,
                           double* P_T, double* bhat_out, double* beta_out, double* b_out,
                           const int32_t* cu_seqlens, int N, int B, int T, int H, int dk, int dv,
                           int alpha_per_channel, double mu, double scale, int nthreads,
                           const double* mu_t, double* beff_out)
{
    if (check_dims(N, B, T, H, dk, dv, cu_seqlens)) return -1;
    set_threads(nthreads);
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int64_t chain = 0; chain < (int64_t)N * H; ++chain) {
        int n = (int)(chain / H), h = (int)(chain % H);
        seq_span sp;
        if (span_of(cu_seqlens, n, T, &sp)) { bad |= 1; continue; }
        double* S = (double*)malloc(sizeof(double) * ((size_t)dk * dv + dv));
        double* delta = S + (size_t)dk * dv;
        const size_t soff = ((size_t)n * H + h) * dk * dv, poff = (size_t)n * H + h;
        for (size_t i = 0; i < (size_t)dk * dv; ++i) S[i] = S0 ? S0[soff + i] : 0.0;
        double b = P0 ? P0[poff] : 1.0;
        for (int64_t t = 0; t < sp.len; ++t) {
            const size_t row = ((size_t)sp.b * T + sp.t0 + t) * H + h;
            iso_step(dk, dv, S, &b, q + row * dk, k + row * dk, v + row * dv,
                     alpha + (alpha_per_channel ? row * dk : row), alpha_per_channel,
                     omega[row], r[row], mu_t ? mu_t[row] : mu, scale, o ? o + row * dv : NULL,
                     bhat_out ? bhat_out + row : NULL, beta_out ? beta_out + row : NULL,
                     b_out ? b_out + row : NULL, beff_out ? beff_out + row : NULL, delta);
        }
        if (S_T) memcpy(S_T + soff, S, sizeof(double) * dk * dv);
        if (P_T) P_T[poff] = b;
        free(S);
    }
    return bad ? -1 : 0;
}

/*
 * One decode step: row i of the batch advances the state held in slot slot_idx[i] (slot_idx
 * NULL: slot i; a negative slot skips the row and leaves o untouched). Exactly one recurrence
 * step of the forward pass (variant 0 = diagonal, 1 = isotropic), S and P updated in place.
 * q, k [R,H,dk]; v, o [R,H,dv]; alpha [R,H,dk] or [R,H]; omega [R,H,dk] (diag) or [R,H];
 * r [R,H]; S [num_slots,H,dk,dv]; P [num_slots,H,dk] (diag) or [num_slots,H] (iso).
 */
int oracle_kdn_decode_step(int variant, const double* q, const double* k, const double* v,
                           const double* alpha, const double* omega, const double* r,
                           double* S, double* P, const int32_t* slot_idx, double* o, int R,
                           int num_slots, int H, int dk, int dv, int alpha_per_channel,
                           double mu, double scale, int nthreads, const double* mu_t,
                           double* beff_out)
{
    if (R < 0 || num_slots <= 0 || H <= 0 || dk <= 0 || dv <= 0) return -1;
    if (variant != 0 && variant != 1) return -1;
    set_threads(nthreads);
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int64_t chain = 0; chain < (int64_t)R * H; ++chain) {
        int i = (int)(chain / H), h = (int)(chain % H);
        int slot = slot_idx ? slot_idx[i] : i;
        if (slot < 0) continue;
        if (slot >= num_slots) { bad |= 1; continue; }
        double* buf = (double*)malloc(sizeof(double) * (3 * dk + dv));
        double* ph = buf;
        double* kap = ph + dk;
        double* delta = kap + dk;
        const size_t row = (size_t)i * H + h;
        double* Sl = S + ((size_t)slot * H + h) * dk * dv;
        if (variant == 0) {
            diag_step(dk, dv, Sl, P + ((size_t)slot * H + h) * dk, q + row * dk, k + row * dk,
                      v + row * dv, alpha + row * dk, omega + row * dk, r[row],
                      mu_t ? mu_t[row] : mu, scale, o + row * dv, NULL, NULL, NULL,
                      beff_out ? beff_out + row : NULL, ph, kap, delta);
        } else {
            iso_step(dk, dv, Sl, P + (size_t)slot * H + h, q + row * dk, k + row * dk,
                     v + row * dv, alpha + (alpha_per_channel ? row * dk : row),
                     alpha_per_channel, omega[row], r[row], mu_t ? mu_t[row] : mu, scale,
                     o + row * dv, NULL, NULL, NULL, beff_out ? beff_out + row : NULL, delta);
        }
        free(buf);
    }
    return bad ? -1 : 0;
}

/* ------------------------------------------------------------------------------------------ */
/* Moebius forms of one scalar variance chain (App. "Hardware-Efficient Chunkwise Algorithm",  */
/* eq. diag-cov-scan): M_t = [[a_t, w_t], [u_t a_t, 1 + u_t w_t]] acting on z = [n; d] with     */
/* p = n / d and z_0 = [p_0; 1]. a_t is the transition factor (alpha^2, or the trace average    */
/* for the isotropic chain), w_t the process noise, u_t the scaled precision increment.        */
/* Every form emits phat_t = a_t n_{t-1}/d_{t-1} + w_t from the state before token t and       */
/* p_t = n_t / d_t after it (eq. chunk-gain-emission). Homogeneous vectors and matrices are     */
/* rescaled by a power of two after each product when `renorm` is set: p = n / d is invariant  */
/* to a common factor, and a power of two keeps the rescaling exact.                           */
/* ------------------------------------------------------------------------------------------ */
typedef struct { double m00, m01, m10, m11; } mat2;

static mat2 mat_mul(mat2 x, mat2 y) /* x @ y */
{
    mat2 z = {x.m00 * y.m00 + x.m01 * y.m10, x.m00 * y.m01 + x.m01 * y.m11,
              x.m10 * y.m00 + x.m11 * y.m10, x.m10 * y.m01 + x.m11 * y.m11};
    return z;
}

static mat2 mat_renorm(mat2 x)
{
    double m = fmax(fmax(fabs(x.m00), fabs(x.m01)), fmax(fabs(x.m10), fabs(x.m11)));
    if (m > 0.0 && isfinite(m)) {
        int e;
        frexp(m, &e);
        x.m00 = ldexp(x.m00, -e); x.m01 = ldexp(x.m01, -e);
        x.m10 = ldexp(x.m10, -e); x.m11 = ldexp(x.m11, -e);
    }
    return x;
}

static void vec_renorm(double* n, double* d)
{
    double m = fmax(fabs(*n), fabs(*d));
    if (m > 0.0 && isfinite(m)) {
        int e;
        frexp(m, &e);
        *n = ldexp(*n, -e);
        *d = ldexp(*d, -e);
    }
}

static mat2 token_mat(double a, double w, double u)
{
    mat2 m = {a, w, u * a, 1.0 + u * w};
    return m;
}

static void emit(double a, double w, double n, double d, double* phat)
{
    *phat = a * n / d + w;
}

/* Left fold z_t = M_t z_{t-1}. */
int oracle_mobius_fold(const double* a, const double* w, const double* u, double p0, int64_t T,
                       int renorm, double* phat, double* p)
{
    double n = p0, d = 1.0;
    for (int64_t t = 0; t < T; ++t) {
        emit(a[t], w[t], n, d, &phat[t]);
        mat2 m = token_mat(a[t], w[t], u[t]);
        double n2 = m.m00 * n + m.m01 * d, d2 = m.m10 * n + m.m11 * d;
        n = n2; d = d2;
        if (renorm) vec_renorm(&n, &d);
        p[t] = n / d;
    }
    return 0;
}

/*
 * Blelloch work-efficient exclusive scan of the token matrices under the composition
 * X (*) Y = Y @ X (later tokens multiply on the left), then emission from each exclusive
 * prefix applied to z_0. The length is padded to a power of two with identity matrices.
 */
int oracle_mobius_tree(const double* a, const double* w, const double* u, double p0, int64_t T,
                       int renorm, double* phat, double* p)
{
    int64_t L = 1;
    while (L < T) L <<= 1;
    mat2* x = (mat2*)malloc(sizeof(mat2) * (size_t)(L > 0 ? L : 1));
    if (!x) return -1;
    const mat2 I = {1.0, 0.0, 0.0, 1.0};
    for (int64_t t = 0; t < L; ++t) x[t] = t < T ? token_mat(a[t], w[t], u[t]) : I;
    /* up-sweep */
    for (int64_t s = 1; s < L; s <<= 1)
        for (int64_t i = 2 * s - 1; i < L; i += 2 * s) {
            x[i] = mat_mul(x[i], x[i - s]);
            if (renorm) x[i] = mat_renorm(x[i]);
        }
    /* down-sweep: exclusive prefixes */
    x[L - 1] = I;
    for (int64_t s = L >> 1; s >= 1; s >>= 1)
        for (int64_t i = 2 * s - 1; i < L; i += 2 * s) {
            mat2 left = x[i - s];
            x[i - s] = x[i];
            x[i] = mat_mul(left, x[i]);
            if (renorm) x[i] = mat_renorm(x[i]);
        }
    for (int64_t t = 0; t < T; ++t) {
        /* state before token t: z_{t-1} = X_t z_0 */
        double n = x[t].m00 * p0 + x[t].m01, d = x[t].m10 * p0 + x[t].m11;
        emit(a[t], w[t], n, d, &phat[t]);
        mat2 m = token_mat(a[t], w[t], u[t]);
        double n2 = m.m00 * n + m.m01 * d, d2 = m.m10 * n + m.m11 * d;
        p[t] = n2 / d2;
    }
    free(x);
    return 0;
}

/*
 * Three-pass chunked scan (eqs. chunk-gain-summary, chunk-gain-carry, chunk-gain-local-prefix,
 * chunk-gain-emission): per-chunk summaries M_bar_m = M_r ... M_l, an exclusive carry
 * z_in_m = M_bar_{m-1} ... M_bar_0 z_0, then a replay of each chunk from its carry.
 */
int oracle_mobius_chunked(const double* a, const double* w, const double* u, double p0,
                          int64_t T, int64_t Cg, int renorm, double* phat, double* p)
{
    if (Cg <= 0) return -1;
    int64_t nch = (T + Cg - 1) / Cg;
    mat2* sum = (mat2*)malloc(sizeof(mat2) * (size_t)(nch > 0 ? nch : 1));
    double* zin = (double*)malloc(sizeof(double) * 2 * (size_t)(nch > 0 ? nch : 1));
    if (!sum || !zin) { free(sum); free(zin); return -1; }
    for (int64_t m = 0; m < nch; ++m) { /* pass 1: summaries */
        mat2 acc = {1.0, 0.0, 0.0, 1.0};
        for (int64_t t = m * Cg; t < (m + 1) * Cg && t < T; ++t) {
            acc = mat_mul(token_mat(a[t], w[t], u[t]), acc);
            if (renorm) acc = mat_renorm(acc);
        }
        sum[m] = acc;
    }
    double n = p0, d = 1.0; /* pass 2: exclusive carries */
    for (int64_t m = 0; m < nch; ++m) {
        zin[2 * m] = n; zin[2 * m + 1] = d;
        double n2 = sum[m].m00 * n + sum[m].m01 * d, d2 = sum[m].m10 * n + sum[m].m11 * d;
        n = n2; d = d2;
        if (renorm) vec_renorm(&n, &d);
    }
    for (int64_t m = 0; m < nch; ++m) { /* pass 3: replay and emission */
        double cn = zin[2 * m], cd = zin[2 * m + 1];
        for (int64_t t = m * Cg; t < (m + 1) * Cg && t < T; ++t) {
            emit(a[t], w[t], cn, cd, &phat[t]);
            mat2 mt = token_mat(a[t], w[t], u[t]);
            double n2 = mt.m00 * cn + mt.m01 * cd, d2 = mt.m10 * cn + mt.m11 * cd;
            cn = n2; cd = d2;
            if (renorm) vec_renorm(&cn, &cd);
            p[t] = cn / cd;
        }
    }
    free(sum);
    free(zin);
    return 0;
}

/* ------------------------------------------------------------------------------------------ */
/* Kalman Associative Memory: the exact filter with a dense dk x dk covariance per (sequence,  */
/* head) (Prop. "Kalman Associative Memory", eq. kalman-optimal-update-box), with the          */
/* transition D = diag(alpha) and process noise Omega = diag(omega) of the KDN inputs:         */
/*   P_hat = D P D^T + Omega;  kappa = P_hat k / (r + k^T P_hat k)                            */
/*   S = D S + kappa (v - (D S)^T k)^T;  P = (I - kappa k^T) P_hat;  o = scale S^T q          */
/* P0 [N,H,dk,dk] (NULL = identity), P_T [N,H,dk,dk]; other arguments as the diagonal forward. */
/* ------------------------------------------------------------------------------------------ */
int oracle_kdn_forward_kam(const double* q, const double* k, const double* v, const double* alpha,
                           const double* omega, const double* r, const double* S0,
                           const double* P0, double* o, double* S_T, double* P_T,
                           const int32_t* cu_seqlens, int N, int B, int T, int H, int dk, int dv,
                           double scale, int nthreads)
{
    if (check_dims(N, B, T, H, dk, dv, cu_seqlens)) return -1;
    for (int n = 0; n < N; ++n) {
        seq_span s;
        if (span_of(cu_seqlens, n, T, &s)) return -1;
    }
    set_threads(nthreads);
    int bad = 0;
#pragma omp parallel for schedule(dynamic) reduction(| : bad)
    for (int nh = 0; nh < N * H; ++nh) {
        const int n = nh / H, h = nh % H;
        seq_span s;
        span_of(cu_seqlens, n, T, &s);
        const size_t SZ = (size_t)dk * dv, PZ = (size_t)dk * dk;
        double* S = malloc(sizeof(double) * SZ);
        double* P = malloc(sizeof(double) * PZ);
        double* Pk = malloc(sizeof(double) * dk);   /* P_hat k            */
        double* kP = malloc(sizeof(double) * dk);   /* k^T P_hat          */
        double* del = malloc(sizeof(double) * dv);  /* v - S_hat^T k      */
        if (!S || !P || !Pk || !kP || !del) {
            bad |= 1;
        } else {
            for (size_t e = 0; e < SZ; ++e) S[e] = S0 ? S0[(size_t)nh * SZ + e] : 0.0;
            for (int i = 0; i < dk; ++i)
                for (int j = 0; j < dk; ++j)
                    P[i * dk + j] = P0 ? P0[(size_t)nh * PZ + (size_t)i * dk + j] : (i == j);
            for (int t = 0; t < s.len; ++t) {
                const int64_t row = ((int64_t)s.b * T + s.t0 + t) * H + h;
                const double *qt = q + row * dk, *kt = k + row * dk, *vt = v + row * dv;
                const double *at = alpha + row * dk, *wt = omega + row * dk;
                /* predict: P_hat = D P D + Omega, S_hat = D S */
                for (int i = 0; i < dk; ++i)
                    for (int j = 0; j < dk; ++j)
                        P[i * dk + j] = at[i] * P[i * dk + j] * at[j] + (i == j ? wt[i] : 0.0);
                for (int i = 0; i < dk; ++i)
                    for (int j = 0; j < dv; ++j) S[i * dv + j] *= at[i];
                /* kappa = P_hat k / c with c = r + k^T P_hat k */
                for (int i = 0; i < dk; ++i) {
                    double acc = 0.0, acc2 = 0.0;
                    for (int j = 0; j < dk; ++j) {
                        acc += P[i * dk + j] * kt[j];
                        acc2 += kt[j] * P[j * dk + i];
                    }
                    Pk[i] = acc;
                    kP[i] = acc2;
                }
                double c = r[row];
                for (int i = 0; i < dk; ++i) c += kt[i] * Pk[i];
                /* S = S_hat + kappa (v - S_hat^T k)^T */
                for (int j = 0; j < dv; ++j) {
                    double acc = 0.0;
                    for (int i = 0; i < dk; ++i) acc += S[i * dv + j] * kt[i];
                    del[j] = vt[j] - acc;
                }
                for (int i = 0; i < dk; ++i)
                    for (int j = 0; j < dv; ++j) S[i * dv + j] += Pk[i] / c * del[j];
                /* P = (I - kappa k^T) P_hat = P_hat - kappa (k^T P_hat) */
                for (int i = 0; i < dk; ++i)
                    for (int j = 0; j < dk; ++j) P[i * dk + j] -= Pk[i] / c * kP[j];
                /* o = scale S^T q (read after the write) */
                if (o) {
                    for (int j = 0; j < dv; ++j) {
                        double acc = 0.0;
                        for (int i = 0; i < dk; ++i) acc += S[i * dv + j] * qt[i];
                        o[row * dv + j] = scale * acc;
                    }
                }
            }
            for (size_t e = 0; e < SZ; ++e) S_T[(size_t)nh * SZ + e] = S[e];
            if (P_T)
                for (size_t e = 0; e < PZ; ++e) P_T[(size_t)nh * PZ + e] = P[e];
        }
        free(S); free(P); free(Pk); free(kP); free(del);
    }
    return bad ? -2 : 0;
}
