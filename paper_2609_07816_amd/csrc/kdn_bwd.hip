// Backward pass of the chunked KDN forward (both variants) on gfx950.
//
// The forward's loss gradient is taken through its two stages (App. "Hardware-Efficient
// Chunkwise Algorithm": the gain scan, then the memory scan):
//
//  memory scan, given the gains kappa_t. Within a chunk of C tokens with start state S_in,
//  decays gamma_t = prod_{s <= t} alpha_s = exp(lambda_t) (lambda: cumulative log-decay, float64)
//  and the ratios R_ts = gamma_t / gamma_s = exp(lambda_t - lambda_s) <= 1 (s <= t):
//      (I + T) Delta = V - Kbar S_in,      T_ts = sum_i k_ti kappa_si R_ts,i   (s < t)
//      O = scale (Qbar S_in + B Delta),    B_ts = sum_i q_ti kappa_si R_ts,i   (s <= t)
//      S_out = diag(gamma_C) S_in + Ktail^T Delta,  Ktail_s = (gamma_C / gamma_s) kappa_s
//  with Kbar = gamma k, Qbar = gamma q (eqs. chunk-memory-normalization to
//  chunk-memory-output-state, written with kappa itself). Its adjoint runs a reverse walk over
//  the chunks carrying dS (dS_in = scale Qbar^T dO + diag(gamma_C) dS_out - Kbar^T Psi with
//  Psi = A^T (scale B^T dO + Ktail dS_out), A = (I + T)^-1; dV = Psi), then forms every
//  chunk's gradients on q, k, kappa and the log-decays chunk-parallel from S_in (checkpointed
//  by a forward walk), dS_out, Delta and Psi.
//
//  gain scan. kappa_t = p_hat_t k_t / (r_t + sum_i p_hat_ti k_ti^2) (diagonal) or beta_t k_t
//  (isotropic), p_hat_t = alpha_t^2 p_{t-1} + omega_t (or a_t b_{t-1} + omega_t) and
//  p_t = p_hat_t / (1 + u_t p_hat_t) (eqs. kla-box-gain, diag-cov-update; iso-kla-box-gain,
//  iso-kla-box-cov-update). The adjoint of p_t obeys a linear recurrence backwards in time,
//  lambda_p,{t-1} = A_t lambda_p,t + B_t, whose coefficients are token-local; it is run per
//  channel in reverse, and every other gradient of the gain stage is token-local given it.
//
// Kernels, in launch order (summary and carry scan are the forward's):
//   bw_prep   per (chunk, head): variance replay from the carry, kappa, lambda, T, B, A
//   bw_fwalk  per (sequence, head, value tile): S_in of every chunk, Delta
//   bw_rwalk  per (sequence, head, value tile), chunks in reverse: dS_out, dV, dS0
//   bw_grad   per (chunk, head): dq, dk (memory part), dkappa, d(log-decay) -> dalpha part,
//             the coefficients of the variance adjoint
//   bw_scan   per (sequence, head, variance channel): the variance adjoint, dP0
//   bw_final  per (chunk, head): dk, dalpha, domega, dr of the gain stage
// Everything is float32 arithmetic (the log-decays float64); gradients are float32.
#include "kdn_fwd.h"

namespace kdn {
namespace bwd {

using fwd::C;
constexpr int NTH = 256;  // bw_final and the forward's summary kernel
// bw_prep, the walks and bw_grad hold a whole chunk in LDS (one workgroup per CU): 512 threads
// put two waves on every SIMD to hide the LDS and memory latency
constexpr int NTB = 512, NWB = NTB / 64;
// saturation of the decay factors referenced to a block's token 8 (2^100: beyond the inverse of
// any 8-token decay above 2^-100)
constexpr float RSAT = 1.2676506e30f;

using FF = Frag<float, 16>;  // one 16-deep step of a float32 product: four 16 x 16 x 4 MFMAs

// Per (chunk, head) record written by bw_prep.
template <int DK>
struct BwRec {
    static constexpr size_t F = (size_t)C * DK * 4;
    static constexpr size_t OFF_KAP = 0;        // kappa [C][DK]
    static constexpr size_t OFF_PHAT = F;       // p_hat [C][DK] (isotropic: b_hat in [t][0])
    static constexpr size_t OFF_PPRV = 2 * F;   // p_{t-1} [C][DK] (isotropic: [t][0])
    static constexpr size_t OFF_KBAR = 3 * F;   // gamma k
    static constexpr size_t OFF_QBAR = 4 * F;   // gamma q
    static constexpr size_t OFF_KTL = 5 * F;    // (gamma_C / gamma) kappa
    static constexpr size_t OFF_LAM = 6 * F;    // lambda [C][DK] float64
    static constexpr size_t OFF_A = 8 * F;      // (I + T)^-1 [C][C]
    static constexpr size_t OFF_B = OFF_A + (size_t)C * C * 4;  // B [C][C]
    static constexpr size_t OFF_GC = OFF_B + (size_t)C * C * 4; // gamma_C [DK]
    static constexpr size_t OFF_DEN = OFF_GC + (size_t)DK * 4;  // gain denominator [C]
    static constexpr size_t BYTES = al256(OFF_DEN + (size_t)C * 4);
};

// Workspace of one backward call.
struct BwMap {
    size_t choff, summ, carry, rec, ckpt, dlt, dso, dkap, dal, acf, bcf, aux, cmap, lpe, total;
    int maxch;
};

inline BwMap bw_map(int variant, bool packed, int N, int B, int T, int H, int dk, int dv,
                    size_t rec_bytes)
{
    BwMap m;
    m.maxch = packed ? (int)((size_t)B * T / C + (size_t)N) : N * ((T + C - 1) / C);
    const size_t ch = (size_t)m.maxch * H;
    const size_t nchan = variant == 0 ? (size_t)dk : 1;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t o = off;
        off += al256(bytes);
        return o;
    };
    m.choff = take(packed ? (size_t)(N + 1) * 4 : 0);
    m.summ = take(ch * nchan * 16);
    m.carry = take(ch * nchan * 8);
    m.rec = take(ch * rec_bytes);
    m.ckpt = take(ch * dk * dv * 4);
    m.dlt = take(ch * C * dv * 4);
    m.dso = take(ch * dk * dv * 4);
    m.dkap = take(ch * C * dk * 4);
    m.dal = take(ch * C * dk * 4);
    m.acf = take(ch * C * nchan * 4);
    m.bcf = take(ch * C * nchan * 4);
    m.aux = take(ch * C * 4);
    m.cmap = take(ch * nchan * 8);
    m.lpe = take(ch * nchan * 4);
    m.total = off;
    return m;
}

struct Args {
    const void *q, *k, *v, *alpha, *omega, *r, *dO;
    const float *S0, *dS_T, *dP_T;
    float *dq, *dk, *dv, *dalpha, *domega, *dr, *dS0, *dP0;
    ChunkMap cm;
    int H, DV, BV;
    float mu, scale;
    const float2* carry;
    char* rec;
    float *ckpt, *dlt, *dso, *dkap, *dal, *acf, *bcf, *aux;
    float2* cmap;  // per (chunk, head, variance channel): the chunk's reverse map of the adjoint
    float* lpe;    // per (chunk, head, variance channel): the adjoint at the chunk's end
};

template <class TI>
__device__ __forceinline__ float ld(const void* p, size_t i)
{
    return to_f32(((const TI*)p)[i]);
}

// Eight consecutive inputs from element i (a multiple of 8) in float32: one 16-byte load
// (bf16) or two (float32).
template <class TI>
__device__ __forceinline__ void ld8(const void* p, size_t i, float* x)
{
    if constexpr (sizeof(TI) == 2) {
        const uint4 v = *reinterpret_cast<const uint4*>((const TI*)p + i);
        const float2 a = unpack2(v.x), b = unpack2(v.y), c = unpack2(v.z), d = unpack2(v.w);
        x[0] = a.x; x[1] = a.y; x[2] = b.x; x[3] = b.y;
        x[4] = c.x; x[5] = c.y; x[6] = d.x; x[7] = d.y;
    } else {
        const floatx4 a = *reinterpret_cast<const floatx4*>((const float*)p + i);
        const floatx4 b = *reinterpret_cast<const floatx4*>((const float*)p + i + 4);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            x[u] = a[u];
            x[4 + u] = b[u];
        }
    }
}

// ------------------------------------------------------------------------------------------
// bw_prep
// ------------------------------------------------------------------------------------------
template <int DK>
struct PrepLds {
    static constexpr int SLB = DK < 32 ? DK : 32;  // channel slab of the T / B products
    static constexpr int LDK = DK + 1, LDC = C + 1, LDO = SLB + 4;
    static constexpr size_t SZ_CK = (size_t)C * LDK * 4;
    static constexpr size_t OFF_K = 0;                    // k [C][LDK]
    static constexpr size_t OFF_AQ = OFF_K + SZ_CK;       // alpha, then q [C][LDK]
    static constexpr size_t OFF_WP = OFF_AQ + SZ_CK;      // omega, then p_hat, then kappa
    static constexpr size_t OFF_R = OFF_WP + SZ_CK;       // r [C]
    static constexpr size_t OFF_DEN = OFF_R + C * 4;      // gain denominators [C]
    static constexpr size_t OFF_BETA = OFF_DEN + C * 4;   // isotropic beta [C]
    static constexpr size_t OFF_AA = OFF_BETA + C * 4;    // isotropic mean alpha^2 [C]
    static constexpr size_t OFF_NK = OFF_AA + C * 4;      // isotropic ||k||^2 [C]
    static constexpr size_t OFF_W1 = OFF_NK + C * 4;      // isotropic omega [C]
    static constexpr size_t OFF_LC = al16(OFF_W1 + C * 4);             // lambda_C [DK] double
    static constexpr size_t OFF_MID = al16(OFF_LC + (size_t)DK * 8);   // [3][SLB]
    // six operand slabs [C][LDO] of the T / B products; afterwards T, (I + T)^-1 [C][LDC] and
    // the block products [3][16][17] over them
    static constexpr size_t OFF_OP = al16(OFF_MID + (size_t)3 * SLB * 4);
    static constexpr size_t SZ_OP = (size_t)C * LDO * 4;
    static constexpr size_t OFF_T = OFF_OP;
    static constexpr size_t OFF_A = OFF_T + (size_t)C * LDC * 4;
    static constexpr size_t OFF_X = OFF_A + (size_t)C * LDC * 4;
    static constexpr size_t TOTAL =
        al16(cmax(OFF_OP + 6 * SZ_OP, OFF_X + (size_t)3 * 16 * 17 * 4));
};

template <class TI, int DK, int VARIANT, bool APC>
__global__ __launch_bounds__(NTB) void bw_prep(Args a)
{
    using R = BwRec<DK>;
    using LY = PrepLds<DK>;
    constexpr bool DIAG = VARIANT == 0;
    constexpr int SLB = LY::SLB, LDK = LY::LDK, LDC = LY::LDC, LDO = LY::LDO;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    float* s_k = (float*)(smem + LY::OFF_K);
    float* s_aq = (float*)(smem + LY::OFF_AQ);
    float* s_wp = (float*)(smem + LY::OFF_WP);
    float* s_r = (float*)(smem + LY::OFF_R);
    float* s_den = (float*)(smem + LY::OFF_DEN);
    float* s_beta = (float*)(smem + LY::OFF_BETA);
    float* s_aa = (float*)(smem + LY::OFF_AA);
    float* s_nk = (float*)(smem + LY::OFF_NK);
    float* s_w1 = (float*)(smem + LY::OFF_W1);
    double* s_lc = (double*)(smem + LY::OFF_LC);
    float* s_mid = (float*)(smem + LY::OFF_MID);
    float* s_op = (float*)(smem + LY::OFF_OP);
    float* s_T = (float*)(smem + LY::OFF_T);
    float* s_A = (float*)(smem + LY::OFF_A);
    float* s_X = (float*)(smem + LY::OFF_X);

    const int H = a.H;
    const int g = (int)(blockIdx.x / H), h = (int)(blockIdx.x % H);
    int n, c0, c1;
    bool last;
    if (!locate_chunk<C>(a.cm, g, n, c0, c1, last)) return;
    const int L = c1 - c0;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    char* rec = a.rec + ((size_t)g * H + h) * R::BYTES;
    float* __restrict__ kap = (float*)(rec + R::OFF_KAP);
    float* __restrict__ phat = (float*)(rec + R::OFF_PHAT);
    float* __restrict__ pprv = (float*)(rec + R::OFF_PPRV);
    float* __restrict__ kbar = (float*)(rec + R::OFF_KBAR);
    float* __restrict__ qbar = (float*)(rec + R::OFF_QBAR);
    float* __restrict__ ktl = (float*)(rec + R::OFF_KTL);
    double* __restrict__ lam = (double*)(rec + R::OFF_LAM);
    float* __restrict__ Am = (float*)(rec + R::OFF_A);
    float* __restrict__ Bm = (float*)(rec + R::OFF_B);
    float* __restrict__ gC = (float*)(rec + R::OFF_GC);
    float* __restrict__ den = (float*)(rec + R::OFF_DEN);
    auto row = [&](int t) { return (size_t)(c0 + t) * H + h; };

    // ---- the chunk's inputs in LDS (padding tokens: alpha 1, k 0, omega 0, r 1), eight
    // channels per piece -------------------------------------------------------------------
    for (int e = tid; e < C * DK / 8; e += NTB) {
        const int t = e / (DK / 8), i8 = 8 * (e % (DK / 8));
        const bool ok = t < L;
        float kx[8], ax[8], wx[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            kx[u] = 0.f;
            ax[u] = 1.f;
            wx[u] = 0.f;
        }
        if (ok) {
            ld8<TI>(a.k, row(t) * DK + i8, kx);
            if (APC) {
                ld8<TI>(a.alpha, row(t) * DK + i8, ax);
            } else {
                const float a1 = ld<TI>(a.alpha, row(t));
#pragma unroll
                for (int u = 0; u < 8; ++u) ax[u] = a1;
            }
            if (DIAG) ld8<TI>(a.omega, row(t) * DK + i8, wx);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            s_k[t * LDK + i8 + u] = kx[u];
            s_aq[t * LDK + i8 + u] = ax[u];
            if (DIAG) s_wp[t * LDK + i8 + u] = wx[u];
        }
    }
    if (tid < C) {
        const bool ok = tid < L;
        s_r[tid] = ok ? ld<TI>(a.r, row(tid)) : 1.f;
        if (!DIAG) s_w1[tid] = ok ? ld<TI>(a.omega, row(tid)) : 0.f;
    }
    __syncthreads();

    // ---- the variance chain through the chunk from the carry (eq. kla-box-mobius, or
    // iso-kla-box-cov-update) and the cumulative log-decay -------------------------------------
    if constexpr (DIAG) {
        if (tid < DK) {
            const float2 cz = a.carry[((size_t)g * H + h) * DK + tid];
            float p = cz.x / cz.y;
            for (int t = 0; t < C; ++t) {
                const float al = s_aq[t * LDK + tid], kk = s_k[t * LDK + tid];
                pprv[t * DK + tid] = p;
                const float ph = al * al * p + s_wp[t * LDK + tid];
                phat[t * DK + tid] = ph;
                s_wp[t * LDK + tid] = ph;
                const float u = a.mu * kk * kk * __builtin_amdgcn_rcpf(s_r[t]);
                p = ph * __builtin_amdgcn_rcpf(fmaf(u, ph, 1.f));
            }
        }
    } else {
        for (int j = 0; j < C / NWB; ++j) {  // per-token mean alpha^2 and ||k||^2
            const int t = (C / NWB) * w + j;
            float sa = 0.f, sk = 0.f;
            for (int i = lane; i < DK; i += 64) {
                const float kk = s_k[t * LDK + i], al = s_aq[t * LDK + i];
                sk += kk * kk;
                sa += al * al;
            }
            sa = wave_sum(sa);
            sk = wave_sum(sk);
            if (lane == 0) {
                const float a0 = s_aq[t * LDK];
                s_aa[t] = APC ? sa / (float)DK : a0 * a0;
                s_nk[t] = sk;
            }
        }
        __syncthreads();
        if (tid == 0) {
            const float2 cz = a.carry[(size_t)g * H + h];
            float b = cz.x / cz.y;
            for (int t = 0; t < C; ++t) {
                const float rr = s_r[t];
                pprv[t * DK] = b;
                const float bh = s_aa[t] * b + s_w1[t];
                phat[t * DK] = bh;
                const float dn = rr + bh * s_nk[t];
                s_den[t] = dn;
                den[t] = dn;
                s_beta[t] = bh / dn;
                const float u = a.mu * s_nk[t] / ((float)DK * rr);
                b = bh / (1.f + u * bh);
            }
        }
    }
    if (tid < DK) {
        double lm = 0.0;
        for (int t = 0; t < C; ++t) {
            lm += (double)logf(s_aq[t * LDK + tid]);
            lam[t * DK + tid] = lm;
        }
        s_lc[tid] = lm;
        gC[tid] = expf((float)lm);
    }
    __syncthreads();
    if constexpr (DIAG) {  // gain denominators r + sum_i p_hat_i k_i^2
        for (int j = 0; j < C / NWB; ++j) {
            const int t = (C / NWB) * w + j;
            float z = 0.f;
            for (int i = lane; i < DK; i += 64) {
                const float kk = s_k[t * LDK + i];
                z += s_wp[t * LDK + i] * kk * kk;
            }
            z = wave_sum(z);
            if (lane == 0) {
                const float dn = t < L ? s_r[t] + z : 1.f;
                s_den[t] = dn;
                den[t] = dn;
            }
        }
        __syncthreads();
    }

    // ---- kappa, gamma-scaled operands and the tail operand; q into LDS (alpha is dead) ------
    for (int e8 = tid; e8 < C * DK / 8; e8 += NTB) {  // eight channels per piece
        const int t = e8 / (DK / 8), i8 = 8 * (e8 % (DK / 8)), e = t * DK + i8;
        float qx[8], kpx[8], kbx[8], qbx[8], ktx[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) qx[u] = 0.f;
        if (t < L) ld8<TI>(a.q, row(t) * DK + i8, qx);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int i = i8 + u;
            const float kk = s_k[t * LDK + i];
            const float kp = DIAG ? s_wp[t * LDK + i] * kk * __builtin_amdgcn_rcpf(s_den[t])
                                  : s_beta[t] * kk;
            const double lm = lam[e + u];
            const float gm = expf((float)lm);
            kpx[u] = kp;
            kbx[u] = gm * kk;
            qbx[u] = gm * qx[u];
            ktx[u] = expf((float)(s_lc[i] - lm)) * kp;
            s_wp[t * LDK + i] = kp;
            s_aq[t * LDK + i] = qx[u];
        }
#pragma unroll
        for (int h4 = 0; h4 < 8; h4 += 4) {
            *reinterpret_cast<floatx4*>(kap + e + h4) =
                floatx4{kpx[h4], kpx[h4 + 1], kpx[h4 + 2], kpx[h4 + 3]};
            *reinterpret_cast<floatx4*>(kbar + e + h4) =
                floatx4{kbx[h4], kbx[h4 + 1], kbx[h4 + 2], kbx[h4 + 3]};
            *reinterpret_cast<floatx4*>(qbar + e + h4) =
                floatx4{qbx[h4], qbx[h4 + 1], qbx[h4 + 2], qbx[h4 + 3]};
            *reinterpret_cast<floatx4*>(ktl + e + h4) =
                floatx4{ktx[h4], ktx[h4 + 1], ktx[h4 + 2], ktx[h4 + 3]};
        }
    }
    __syncthreads();

    // ---- T (s < t) and B (s <= t) by 16 x 16 blocks on float32 MFMA, contracting over channel
    // slabs. The decay ratio R_ts,i = gamma_t,i / gamma_s,i splits per block pair: for blocks
    // b > c, the decay from the start of block b to t (row side), over the blocks between them
    // (a per-channel factor on the column side) and from s to the end of block c (column side),
    // each <= 1; inside a diagonal block both sides are referenced to its token 8 (a factor
    // saturates at 2^100). Wave w computes T and B of the lower blocks w and w + 8 of the ten.
    const int li = lane & 15, lg = lane >> 4;
    int pbt[2], pbs[2];
    bool pbo[2];
    floatx4 accT[2], accB[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int q = w + 8 * u;
        pbo[u] = q < 10;
        pbt[u] = q < 1 ? 0 : (q < 3 ? 1 : (q < 6 ? 2 : 3));
        pbs[u] = q - pbt[u] * (pbt[u] + 1) / 2;
        accT[u] = accB[u] = zero4();
    }
    for (int s0 = 0; s0 < DK; s0 += SLB) {
        // operands of channels s0 .. s0 + SLB - 1, row-major [t][ii]: k, q scaled from the start
        // of their block and from its token 8; kappa scaled to the end of its block and to its
        // token 8. Thread: token tid / 8, four channels
        for (int e = tid; e < C * SLB / 4; e += NTB) {
            const int t = e / (SLB / 4), i4 = 4 * (e % (SLB / 4)), b = t >> 4;
            float o[6][4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int i = s0 + i4 + u;
                const double lm = lam[t * DK + i];
                const double lst = b > 0 ? lam[(16 * b - 1) * DK + i] : 0.0;
                const double len = lam[(16 * b + 15) * DK + i], lrf = lam[(16 * b + 7) * DK + i];
                const float ast = __expf((float)(lm - lst));
                const float amd = fminf(__expf((float)(lm - lrf)), RSAT);
                const float ben = __expf((float)(len - lm));
                const float bmd = fminf(__expf((float)(lrf - lm)), RSAT);
                const float kk = s_k[t * LDK + i], qq = s_aq[t * LDK + i], kp = s_wp[t * LDK + i];
                o[0][u] = ast * kk;
                o[1][u] = ast * qq;
                o[2][u] = ben * kp;
                o[3][u] = amd * kk;
                o[4][u] = amd * qq;
                o[5][u] = bmd * kp;
            }
#pragma unroll
            for (int m = 0; m < 6; ++m)
                *reinterpret_cast<float4*>(s_op + m * (C * LDO) + t * LDO + i4) =
                    make_float4(o[m][0], o[m][1], o[m][2], o[m][3]);
        }
        // decay over the blocks between two blocks two or three apart: (2, 0), (3, 0), (3, 1)
        if (tid < 3 * SLB) {
            const int pr = tid / SLB, i = s0 + tid % SLB;
            const int bt = pr == 0 ? 2 : 3, bs = pr == 2 ? 1 : 0;
            s_mid[tid] = __expf((float)(lam[(16 * bt - 1) * DK + i] - lam[(16 * bs + 15) * DK + i]));
        }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            if (!pbo[u]) continue;
            const int tb = pbt[u], sb = pbs[u], dg = tb == sb;
            const float* oK = s_op + (dg ? 3 : 0) * (C * LDO) + 16 * tb * LDO;
            const float* oQ = s_op + (dg ? 4 : 1) * (C * LDO) + 16 * tb * LDO;
            const float* oP = s_op + (dg ? 5 : 2) * (C * LDO) + 16 * sb * LDO;
            const int pm = tb - sb < 2 ? -1 : (tb == 2 ? 0 : (sb == 0 ? 1 : 2));
#pragma unroll
            for (int ks = 0; ks < SLB / 16; ++ks) {
                const int kc = 16 * ks + 4 * lg;
                FF::V bp = FF::ld(oP + li * LDO + kc);
                if (pm >= 0) bp = FF::scale(bp, s_mid + pm * SLB + kc);
                accT[u] = FF::mma(accT[u], FF::ld(oK + li * LDO + kc), bp);
                accB[u] = FF::mma(accB[u], FF::ld(oQ + li * LDO + kc), bp);
            }
        }
        __syncthreads();
    }
    // T and B out (the operand slabs are dead): lower blocks from the products, masked inside
    // the diagonal blocks; zeros above
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        if (!pbo[u]) continue;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int t = 16 * pbt[u] + 4 * lg + r, s2 = 16 * pbs[u] + li;
            Bm[t * C + s2] = s2 <= t ? accB[u][r] : 0.f;
            s_T[t * LDC + s2] = s2 < t ? accT[u][r] : 0.f;
        }
    }
    for (int e = tid; e < 6 * 256; e += NTB) {  // the six blocks above the diagonal
        const int q = e >> 8, tb = q < 3 ? 0 : (q < 5 ? 1 : 2);
        const int sb = tb + 1 + (q - (tb == 0 ? 0 : (tb == 1 ? 3 : 5)));
        const int t = 16 * tb + ((e >> 4) & 15), s2 = 16 * sb + (e & 15);
        Bm[t * C + s2] = 0.f;
        s_T[t * LDC + s2] = 0.f;
    }
    for (int e = tid; e < C * C; e += NTB) s_A[(e / C) * LDC + e % C] = 0.f;
    __syncthreads();

    // ---- A = (I + T)^-1 by 16 x 16 blocks: the diagonal blocks by forward substitution
    // (thread: one column of one block), then the blocks below the diagonal by distance,
    // A_bc = -A_bb sum_{c <= m < b} T_bm A_mc ---------------------------------------------------
    if (tid < C) {
        const int b = tid >> 4, j = tid & 15, o = 16 * b;
        float y[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float acc = r == j ? 1.f : 0.f;
#pragma unroll
            for (int s = 0; s < r; ++s) acc = fmaf(-s_T[(o + r) * LDC + o + s], y[s], acc);
            y[r] = r < j ? 0.f : acc;
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) s_A[(o + r) * LDC + o + j] = y[r];
    }
    __syncthreads();
    for (int d = 1; d < 4; ++d) {
        const int nb = 4 - d;
        for (int e = tid; e < nb * 256; e += NTB) {  // X = sum_m T_bm A_mc
            const int c = e >> 8, b = c + d, r = (e >> 4) & 15, j = e & 15;
            float acc = 0.f;
            for (int m = 16 * c; m < 16 * b; ++m)
                acc = fmaf(s_T[(16 * b + r) * LDC + m], s_A[m * LDC + 16 * c + j], acc);
            s_X[(c * 16 + r) * 17 + j] = acc;
        }
        __syncthreads();
        for (int e = tid; e < nb * 256; e += NTB) {  // A_bc = -A_bb X
            const int c = e >> 8, b = c + d, r = (e >> 4) & 15, j = e & 15;
            float acc = 0.f;
            for (int s = 0; s <= r; ++s)
                acc = fmaf(s_A[(16 * b + r) * LDC + 16 * b + s], s_X[(c * 16 + s) * 17 + j], acc);
            s_A[(16 * b + r) * LDC + 16 * c + j] = -acc;
        }
        __syncthreads();
    }
    for (int e = tid; e < C * C; e += NTB) Am[e] = s_A[(e / C) * LDC + (e % C)];
}

// ------------------------------------------------------------------------------------------
// walks over the chunks of one (sequence, head, value tile of up to 32 columns): every product
// on float32 MFMA (16 x 16 x 4) from LDS operands laid out so that both sides are contiguous
// in the contraction index (the state and the chunk's value-side tiles are kept transposed).
// Wave w of 8 takes 16 x 16 output tiles w, w + 8, ...
// ------------------------------------------------------------------------------------------
template <int DK>
struct WalkLds {
    static constexpr int LDK = DK + 4, LDC = C + 4, BVM = 32;
    // forward walk
    static constexpr size_t F_ST = 0;                                      // S^T [BVM][LDK]
    static constexpr size_t F_KB = F_ST + (size_t)BVM * LDK * 4;           // Kbar [C][LDK]
    static constexpr size_t F_KT = F_KB + (size_t)C * LDK * 4;             // Ktail^T [DK][LDC]
    static constexpr size_t F_A = F_KT + (size_t)DK * LDC * 4;             // A [C][LDC]
    static constexpr size_t F_XT = F_A + (size_t)C * LDC * 4;              // X^T [BVM][LDC]
    static constexpr size_t F_DT = F_XT + (size_t)BVM * LDC * 4;           // Delta^T
    static constexpr size_t F_GC = F_DT + (size_t)BVM * LDC * 4;           // gamma_C [DK]
    static constexpr size_t F_V = al16(F_GC + (size_t)DK * 4);             // V [C][BVM + 1]
    static constexpr size_t F_TOTAL = al16(F_V + (size_t)C * (BVM + 1) * 4);
    // reverse walk
    static constexpr size_t R_ST = 0;                                      // dS^T [BVM][LDK]
    static constexpr size_t R_BT = R_ST + (size_t)BVM * LDK * 4;           // B^T [C][LDC]
    static constexpr size_t R_AT = R_BT + (size_t)C * LDC * 4;             // A^T [C][LDC]
    static constexpr size_t R_OT = R_AT + (size_t)C * LDC * 4;             // scale dO^T [BVM][LDC]
    static constexpr size_t R_DT = R_OT + (size_t)BVM * LDC * 4;           // dDelta^T
    static constexpr size_t R_PT = R_DT + (size_t)BVM * LDC * 4;           // Psi^T
    static constexpr size_t R_GC = R_PT + (size_t)BVM * LDC * 4;           // gamma_C [DK]
    static constexpr size_t R_R = al16(R_GC + (size_t)DK * 4);             // Ktail [C][LDK], or
    static constexpr size_t R_R2 = R_R + (size_t)DK * LDC * 4;             // Qbar^T, Kbar^T [DK][LDC]
    static constexpr size_t R_TOTAL = al16(R_R + cmax((size_t)C * LDK * 4,
                                                      (size_t)2 * DK * LDC * 4));
    static constexpr size_t TOTAL = cmax(F_TOTAL, R_TOTAL);
};


// acc += A[ar0 + 16 rows][k0 .. k0 + 16 * nk) * B[k][br0 + 16 columns], A row-major (lda), B
// stored transposed (row = output column, ldb), k-steps ks0 .. ks1 - 1 of 16
__device__ __forceinline__ floatx4 mfma_rows(floatx4 acc, const float* A, int lda,
                                             const float* Bt, int ldb, int ks0, int ks1,
                                             int lane, bool negA = false)
{
    const int li = lane & 15, lg = lane >> 4;
    for (int ks = ks0; ks < ks1; ++ks) {
        FF::V av = FF::ld(A + li * lda + 16 * ks + 4 * lg);
        const FF::V bv = FF::ld(Bt + li * ldb + 16 * ks + 4 * lg);
        if (negA) av ^= make_uint4(0x80000000u, 0x80000000u, 0x80000000u, 0x80000000u);
        acc = FF::mma(acc, av, bv);
    }
    return acc;
}

// Block -> (sequence-head slot, value tile): the NV tiles of one head get block indices
// congruent modulo 8, so round-robin dispatch puts them on one XCD, where they share the L2 copy
// of the head's chunk records. The grid is padded to a multiple of 8 slots.
__device__ __forceinline__ bool walk_slot(const Args& a, int NV, int& slot, int& vt)
{
    const int xcd = (int)(blockIdx.x % 8), rest = (int)(blockIdx.x / 8);
    vt = rest % NV;
    slot = (rest / NV) * 8 + xcd;
    return slot < a.cm.N * a.H;
}

// Pieces of a chunk's operands each thread moves: float4 pieces of a [C][DK] and a [C][C]
// matrix, values of a [C][32] value tile.
template <int DK>
struct WalkPieces {
    static constexpr int NK4 = C * DK / 4, PK = (NK4 + NTB - 1) / NTB;
    static constexpr int NC4 = C * C / 4, PC = NC4 / NTB;
    static constexpr int PV = C * WalkLds<DK>::BVM / NTB;
    // operands stored transposed move in 4 x 4 blocks (four row pieces in, four column pieces
    // out): one block of a [C][DK] matrix per thread at most, a [C][C] matrix in half the threads
    static constexpr int NKB = (C / 4) * (DK / 4), NCB = (C / 4) * (C / 4);
    static_assert(NKB <= NTB && 2 * NCB == NTB, "one block per thread");
    static_assert(NC4 % NTB == 0 && (C * WalkLds<DK>::BVM) % NTB == 0, "whole pieces");
};

// Block b of an R x K row-major matrix (K / 4 blocks per row band): rows 4 (b / (K / 4)) .. + 3,
// columns 4 (b % (K / 4)) .. + 3. Load: four row pieces; store transposed: four column pieces.
template <int K>
__device__ __forceinline__ void blk_load(const float* src, int b, floatx4* x)
{
    const int r4 = 4 * (b / (K / 4)), c4 = 4 * (b % (K / 4));
#pragma unroll
    for (int r = 0; r < 4; ++r) x[r] = *reinterpret_cast<const floatx4*>(src + (r4 + r) * K + c4);
}
template <int K>
__device__ __forceinline__ void blk_store_t(float* dst, int ld, int b, const floatx4* x)
{
    const int r4 = 4 * (b / (K / 4)), c4 = 4 * (b % (K / 4));
#pragma unroll
    for (int u = 0; u < 4; ++u)
        *reinterpret_cast<floatx4*>(dst + (c4 + u) * ld + r4) =
            floatx4{x[0][u], x[1][u], x[2][u], x[3][u]};
}

// The operands of chunk ci + 1 (fwalk) or ci - 1 (rwalk) are loaded into registers while chunk
// ci is computed, and stored to LDS after the barrier that ends it.
template <class TI, int DK>
__global__ __launch_bounds__(NTB) void bw_fwalk(Args a)
{
    using R = BwRec<DK>;
    using LY = WalkLds<DK>;
    using WP = WalkPieces<DK>;
    constexpr int LDK = LY::LDK, LDC = LY::LDC, NKT = DK / 16, BVM = LY::BVM, LDV = BVM + 1;
    constexpr int PK = WP::PK, PC = WP::PC, PV = WP::PV, NK4 = WP::NK4, NKB = WP::NKB;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    float* s_St = (float*)(smem + LY::F_ST);
    float* s_kb = (float*)(smem + LY::F_KB);
    float* s_ktT = (float*)(smem + LY::F_KT);
    float* s_A = (float*)(smem + LY::F_A);
    float* s_XT = (float*)(smem + LY::F_XT);
    float* s_DT = (float*)(smem + LY::F_DT);
    float* s_gc = (float*)(smem + LY::F_GC);
    float* s_V = (float*)(smem + LY::F_V);

    const int H = a.H, DV = a.DV, BV = a.BV, NV = DV / BV, NJT = BV / 16;
    int slot, vt;
    if (!walk_slot(a, NV, slot, vt)) return;
    const int n = slot / H, h = slot % H, j0 = vt * BV;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, li = lane & 15, lg = lane >> 4;
    float* __restrict__ ckpt = a.ckpt;
    float* __restrict__ dlt = a.dlt;
    int t0, t1, g0, nch;
    seq_span(a.cm, n, t0, t1);
    seq_chunks<C>(a.cm, n, t0, t1, g0, nch);
    for (int e = tid; e < DK * BV; e += NTB) {
        const int i = e / BV, j = e % BV;
        s_St[j * LDK + i] = a.S0 ? a.S0[((size_t)slot * DK + i) * DV + j0 + j] : 0.f;
    }
    floatx4 kb4[PK], ktb[4], am4[PC];
    float vv[PV], gcv = 0.f;
    auto load = [&](int ci) __attribute__((always_inline)) {
        const int c0 = t0 + ci * C, L = min(C, t1 - c0);
        const char* rec = a.rec + ((size_t)(g0 + ci) * H + h) * R::BYTES;
        const floatx4* kbar = (const floatx4*)(rec + R::OFF_KBAR);
        const floatx4* Am = (const floatx4*)(rec + R::OFF_A);
#pragma unroll
        for (int u = 0; u < PK; ++u) kb4[u] = kbar[min(tid + NTB * u, NK4 - 1)];
        blk_load<DK>((const float*)(rec + R::OFF_KTL), min(tid, NKB - 1), ktb);
#pragma unroll
        for (int u = 0; u < PC; ++u) am4[u] = Am[tid + NTB * u];
        if (tid < DK) gcv = ((const float*)(rec + R::OFF_GC))[tid];
#pragma unroll
        for (int u = 0; u < PV; ++u) {  // rows past the end of the sequence read as zeros
            const int e = tid + NTB * u, t = e / BVM, j = e % BVM;
            vv[u] = (t < L && j < BV) ? ld<TI>(a.v, ((size_t)(c0 + t) * H + h) * DV + j0 + j)
                                      : 0.f;
        }
    };
    auto store = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < PK; ++u) {
            const int e = tid + NTB * u;
            if (e < NK4) {
                const int t = e / (DK / 4), i4 = 4 * (e % (DK / 4));
                *reinterpret_cast<floatx4*>(s_kb + t * LDK + i4) = kb4[u];
            }
        }
        if (tid < NKB) blk_store_t<DK>(s_ktT, LDC, tid, ktb);  // Ktail^T
#pragma unroll
        for (int u = 0; u < PC; ++u) {
            const int e = tid + NTB * u, t = e / (C / 4), s4 = 4 * (e % (C / 4));
            *reinterpret_cast<floatx4*>(s_A + t * LDC + s4) = am4[u];
        }
        if (tid < DK) s_gc[tid] = gcv;
#pragma unroll
        for (int u = 0; u < PV; ++u) {
            const int e = tid + NTB * u;
            s_V[(e / BVM) * LDV + e % BVM] = vv[u];
        }
    };
    for (int ci = -1; ci < nch; ++ci) {  // ci = -1: only the first chunk's loads
        const size_t gh = (size_t)(g0 + ci) * H + h;
        if (ci >= 0) {
            __syncthreads();
            for (int e = tid; e < DK * BV; e += NTB) {  // checkpoint: S_in of this chunk
                const int i = e / BV, j = e % BV;
                ckpt[(gh * DK + i) * DV + j0 + j] = s_St[j * LDK + i];
            }
            store();
        }
        if (ci + 1 < nch) load(ci + 1);
        if (ci < 0) continue;
        __syncthreads();
        // X = V - Kbar S_in (tile: rows 16 tb, columns 16 jb); stored as X^T
        for (int tile = w; tile < 4 * NJT; tile += NWB) {
            const int tb = tile / NJT, jb = tile % NJT;
            floatx4 acc = zero4();
            acc = mfma_rows(acc, s_kb + 16 * tb * LDK, LDK, s_St + 16 * jb * LDK, LDK, 0, NKT,
                            lane);
            float x[4];
#pragma unroll
            for (int r = 0; r < 4; ++r)
                x[r] = s_V[(16 * tb + 4 * lg + r) * LDV + 16 * jb + li] - acc[r];
            *reinterpret_cast<float4*>(s_XT + (16 * jb + li) * LDC + 16 * tb + 4 * lg) =
                make_float4(x[0], x[1], x[2], x[3]);
        }
        __syncthreads();
        // Delta = A X (A lower triangular: k-steps up to the row tile); stored as Delta^T and
        // to the workspace
        for (int tile = w; tile < 4 * NJT; tile += NWB) {
            const int tb = tile / NJT, jb = tile % NJT;
            floatx4 acc = zero4();
            acc = mfma_rows(acc, s_A + 16 * tb * LDC, LDC, s_XT + 16 * jb * LDC, LDC, 0, tb + 1,
                            lane);
            *reinterpret_cast<float4*>(s_DT + (16 * jb + li) * LDC + 16 * tb + 4 * lg) =
                make_float4(acc[0], acc[1], acc[2], acc[3]);
#pragma unroll
            for (int r = 0; r < 4; ++r)
                dlt[(gh * C + 16 * tb + 4 * lg + r) * DV + j0 + 16 * jb + li] = acc[r];
        }
        __syncthreads();
        // S_out^T = S_in^T diag(gamma_C) + Delta^T Ktail (tile: rows 16 jb of S^T, columns 16 ib)
        for (int tile = w; tile < NJT * NKT; tile += NWB) {
            const int jb = tile % NJT, ib = tile / NJT;
            const float gc = s_gc[16 * ib + li];
            floatx4 acc;
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[r] = s_St[(16 * jb + 4 * lg + r) * LDK + 16 * ib + li] * gc;
            acc = mfma_rows(acc, s_DT + 16 * jb * LDC, LDC, s_ktT + 16 * ib * LDC, LDC, 0, 4,
                            lane);
#pragma unroll
            for (int r = 0; r < 4; ++r) s_St[(16 * jb + 4 * lg + r) * LDK + 16 * ib + li] = acc[r];
        }
    }
}

template <class TI, int DK>
__global__ __launch_bounds__(NTB) void bw_rwalk(Args a)
{
    using R = BwRec<DK>;
    using LY = WalkLds<DK>;
    using WP = WalkPieces<DK>;
    constexpr int LDK = LY::LDK, LDC = LY::LDC, NKT = DK / 16, BVM = LY::BVM;
    constexpr int PK = WP::PK, PV = WP::PV, NK4 = WP::NK4, NKB = WP::NKB, NCB = WP::NCB;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    float* s_dST = (float*)(smem + LY::R_ST);
    float* s_BT = (float*)(smem + LY::R_BT);
    float* s_AT = (float*)(smem + LY::R_AT);
    float* s_OT = (float*)(smem + LY::R_OT);
    float* s_dDT = (float*)(smem + LY::R_DT);
    float* s_PT = (float*)(smem + LY::R_PT);
    float* s_gc = (float*)(smem + LY::R_GC);
    float* s_kt = (float*)(smem + LY::R_R);    // Ktail [C][LDK] (first half of the chunk)
    float* s_qT = (float*)(smem + LY::R_R);    // Qbar^T [DK][LDC] (second half)
    float* s_kT = (float*)(smem + LY::R_R2);   // Kbar^T [DK][LDC]

    const int H = a.H, DV = a.DV, BV = a.BV, NV = DV / BV, NJT = BV / 16;
    int slot, vt;
    if (!walk_slot(a, NV, slot, vt)) return;
    const int n = slot / H, h = slot % H, j0 = vt * BV;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, li = lane & 15, lg = lane >> 4;
    float* __restrict__ dso = a.dso;
    float* __restrict__ gv = a.dv;
    int t0, t1, g0, nch;
    seq_span(a.cm, n, t0, t1);
    seq_chunks<C>(a.cm, n, t0, t1, g0, nch);
    for (int e = tid; e < DK * BV; e += NTB) {
        const int i = e / BV, j = e % BV;
        s_dST[j * LDK + i] = a.dS_T ? a.dS_T[((size_t)slot * DK + i) * DV + j0 + j] : 0.f;
    }
    // first group: Ktail, B, A, gamma_C, scale dO (stored at the chunk's start); second group:
    // Qbar, Kbar (stored over Ktail once it is read)
    // B or A (half the threads each) and Qbar, Kbar move in 4 x 4 blocks (stored transposed)
    floatx4 kt4[PK], cb[4], qbb[4], kbb[4];
    const bool isb = tid < NCB;
    float ov[PV], gcv = 0.f;
    auto rec_of = [&](int ci) { return a.rec + ((size_t)(g0 + ci) * H + h) * R::BYTES; };
    auto load1 = [&](int ci) __attribute__((always_inline)) {
        const int c0 = t0 + ci * C, L = min(C, t1 - c0);
        const char* rec = rec_of(ci);
        const floatx4* ktl = (const floatx4*)(rec + R::OFF_KTL);
#pragma unroll
        for (int u = 0; u < PK; ++u) kt4[u] = ktl[min(tid + NTB * u, NK4 - 1)];
        blk_load<C>((const float*)(rec + (isb ? R::OFF_B : R::OFF_A)), isb ? tid : tid - NCB, cb);
        if (tid < DK) gcv = ((const float*)(rec + R::OFF_GC))[tid];
#pragma unroll
        for (int u = 0; u < PV; ++u) {
            const int e = tid + NTB * u, t = e / BVM, j = e % BVM;
            ov[u] = (t < L && j < BV && a.dO)
                        ? a.scale * ld<TI>(a.dO, ((size_t)(c0 + t) * H + h) * DV + j0 + j)
                        : 0.f;
        }
    };
    auto store1 = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < PK; ++u) {
            const int e = tid + NTB * u;
            if (e < NK4) {
                const int t = e / (DK / 4), i4 = 4 * (e % (DK / 4));
                *reinterpret_cast<floatx4*>(s_kt + t * LDK + i4) = kt4[u];
            }
        }
        blk_store_t<C>(isb ? s_BT : s_AT, LDC, isb ? tid : tid - NCB, cb);  // B^T or A^T
        if (tid < DK) s_gc[tid] = gcv;
#pragma unroll
        for (int u = 0; u < PV; ++u) {  // scale dO, transposed
            const int e = tid + NTB * u;
            s_OT[(e % BVM) * LDC + e / BVM] = ov[u];
        }
    };
    auto load2 = [&](int ci) __attribute__((always_inline)) {
        const char* rec = rec_of(ci);
        blk_load<DK>((const float*)(rec + R::OFF_QBAR), min(tid, NKB - 1), qbb);
        blk_load<DK>((const float*)(rec + R::OFF_KBAR), min(tid, NKB - 1), kbb);
    };
    auto store2 = [&]() __attribute__((always_inline)) {  // Qbar^T and Kbar^T
        if (tid < NKB) {
            blk_store_t<DK>(s_qT, LDC, tid, qbb);
            blk_store_t<DK>(s_kT, LDC, tid, kbb);
        }
    };
    if (nch > 0) {
        load1(nch - 1);
        load2(nch - 1);
    }
    for (int ci = nch - 1; ci >= 0; --ci) {
        const int c0 = t0 + ci * C, L = min(C, t1 - c0);
        const size_t gh = (size_t)(g0 + ci) * H + h;
        __syncthreads();
        for (int e = tid; e < DK * BV; e += NTB) {  // dS_out of this chunk
            const int i = e / BV, j = e % BV;
            dso[(gh * DK + i) * DV + j0 + j] = s_dST[j * LDK + i];
        }
        store1();
        if (ci > 0) load1(ci - 1);
        __syncthreads();
        // dDelta = B^T (scale dO) + Ktail dS_out (tile: rows 16 sb, columns 16 jb), stored
        // transposed; B^T is upper triangular: k-steps from the row tile on
        for (int tile = w; tile < 4 * NJT; tile += NWB) {
            const int sb = tile / NJT, jb = tile % NJT;
            floatx4 acc = zero4();
            acc = mfma_rows(acc, s_BT + 16 * sb * LDC, LDC, s_OT + 16 * jb * LDC, LDC, sb, 4,
                            lane);
            acc = mfma_rows(acc, s_kt + 16 * sb * LDK, LDK, s_dST + 16 * jb * LDK, LDK, 0, NKT,
                            lane);
            *reinterpret_cast<float4*>(s_dDT + (16 * jb + li) * LDC + 16 * sb + 4 * lg) =
                make_float4(acc[0], acc[1], acc[2], acc[3]);
        }
        __syncthreads();
        // Psi = A^T dDelta = dV (A^T upper triangular), stored transposed and to dv
        for (int tile = w; tile < 4 * NJT; tile += NWB) {
            const int sb = tile / NJT, jb = tile % NJT;
            floatx4 acc = zero4();
            acc = mfma_rows(acc, s_AT + 16 * sb * LDC, LDC, s_dDT + 16 * jb * LDC, LDC, sb, 4,
                            lane);
            *reinterpret_cast<float4*>(s_PT + (16 * jb + li) * LDC + 16 * sb + 4 * lg) =
                make_float4(acc[0], acc[1], acc[2], acc[3]);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int t = 16 * sb + 4 * lg + r;
                if (t < L) gv[((size_t)(c0 + t) * H + h) * DV + j0 + 16 * jb + li] = acc[r];
            }
        }
        __syncthreads();
        store2();
        if (ci > 0) load2(ci - 1);
        __syncthreads();
        // dS_in^T = dS_out^T diag(gamma_C) + (scale dO)^T Qbar - Psi^T Kbar
        for (int tile = w; tile < NJT * NKT; tile += NWB) {
            const int jb = tile % NJT, ib = tile / NJT;
            const float gc = s_gc[16 * ib + li];
            floatx4 acc;
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[r] = s_dST[(16 * jb + 4 * lg + r) * LDK + 16 * ib + li] * gc;
            acc = mfma_rows(acc, s_OT + 16 * jb * LDC, LDC, s_qT + 16 * ib * LDC, LDC, 0, 4, lane);
            acc = mfma_rows(acc, s_PT + 16 * jb * LDC, LDC, s_kT + 16 * ib * LDC, LDC, 0, 4, lane,
                            true);
#pragma unroll
            for (int r = 0; r < 4; ++r) s_dST[(16 * jb + 4 * lg + r) * LDK + 16 * ib + li] = acc[r];
        }
    }
    __syncthreads();
    if (a.dS0)
        for (int e = tid; e < DK * BV; e += NTB) {
            const int i = e / BV, j = e % BV;
            a.dS0[((size_t)slot * DK + i) * DV + j0 + j] = s_dST[j * LDK + i];
        }
}

// ------------------------------------------------------------------------------------------
// bw_grad: chunk-parallel gradients of the memory scan and the variance-adjoint coefficients
// ------------------------------------------------------------------------------------------
// Wave w owns row block rb = w % 4 of the chunk and the channel tiles ct = w / 4 + 2 k: it keeps
// dq, dk and dkappa of those 16 x 16 tiles in registers through both phases (float32 MFMA).
//  1. products over the value columns, by slabs of 32 columns: Psi S_in^T, dO S_in^T and
//     Delta dS_out^T on the owned tiles; dO Delta^T and Psi Delta^T (the adjoints of B and T)
//     on the ten lower 16 x 16 blocks, wave w taking blocks w and w + 8; the diagonal terms
//     sum_j S_in,ij dS_out,ij of the chunk-end decay.
//  2. the terms through T and B, whose entries carry the decay ratios R_ts = gamma_t / gamma_s
//     per channel, by slabs of 32 channels. For 16-token blocks b > c the ratio splits into the
//     decay from the start of block b to t, the decay of the blocks between (a per-channel
//     factor on the block product) and the decay from s to the end of block c, each <= 1;
//     inside a diagonal block both sides are referenced to its token 8 (a factor saturates at
//     2^100, beyond the inverse of any 8-token decay above 2^-100). The scaled operands are
//     staged transposed; each block pair is one 16-deep MFMA step. Wave w forms the rows of
//     block rb as the later token (dq, dk) and as the earlier token (dkappa).
// The log-decay adjoint of an entry is then q dq + k dk - kappa dkappa; its chunk-end part
// enters through column sums.
template <int DK>
struct GradLds {
    static constexpr int SW = 32, LDW = SW + 4;     // value slab, rows padded to 16 bytes
    static constexpr int SLB = DK < 32 ? DK : 32;   // channel slab of phase 2
    static constexpr int LDC = C + 4;
    // phase 1: Delta, Psi, dO [C][LDW]; S_in, dS_out [DK][LDW]
    static constexpr size_t P_D = 0, P_P = (size_t)C * LDW * 4, P_O = 2 * P_P;
    static constexpr size_t P_S = 3 * P_P, P_G = P_S + (size_t)DK * LDW * 4;
    static constexpr size_t P_END = P_G + (size_t)DK * LDW * 4;
    // phase 2: dB, dT, dB^T, dT^T [C][LDC]; six operand slabs [SLB][LDC] (over phase 1)
    static constexpr size_t CC = (size_t)C * LDC * 4, OPS = (size_t)SLB * LDC;
    static constexpr size_t Q_DB = 0, Q_DT = CC, Q_DBT = 2 * CC, Q_DTT = 3 * CC, Q_OP = 4 * CC;
    static constexpr size_t Q_END = Q_OP + 6 * OPS * 4;
    static constexpr size_t MAIN = cmax(P_END, Q_END);
    static constexpr size_t OFF_CP = al16(MAIN);                   // column sums [4][DK]
    static constexpr size_t OFF_P6 = OFF_CP + (size_t)4 * DK * 4;  // [DK]
    static constexpr size_t OFF_BT = OFF_P6 + (size_t)DK * 4;      // block totals [4][DK]
    static constexpr size_t OFF_RP = OFF_BT + (size_t)4 * DK * 4;  // row sums [2][3][C]
    static constexpr size_t OFF_BM = al16(OFF_RP + (size_t)6 * C * 4);  // block maps [4][DK]
    static constexpr size_t TOTAL = al16(OFF_BM + (size_t)4 * DK * 8);
};

template <class TI, int DK, int VARIANT, bool APC>
__global__ __launch_bounds__(NTB) void bw_grad(Args a)
{
    using R = BwRec<DK>;
    using LY = GradLds<DK>;
    constexpr bool DIAG = VARIANT == 0;
    constexpr int SW = LY::SW, LDW = LY::LDW, SLB = LY::SLB, LDC = LY::LDC;
    constexpr int NKT = DK / 16, NCW = (NKT + 1) / 2;  // channel tiles; owned per wave
    constexpr size_t OPS = LY::OPS;
    constexpr int NCHAN = DIAG ? DK : 1;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    float* s_D = (float*)(smem + LY::P_D);
    float* s_P = (float*)(smem + LY::P_P);
    float* s_O = (float*)(smem + LY::P_O);
    float* s_S = (float*)(smem + LY::P_S);
    float* s_G = (float*)(smem + LY::P_G);
    float* s_dB = (float*)(smem + LY::Q_DB);
    float* s_dT = (float*)(smem + LY::Q_DT);
    float* s_dBT = (float*)(smem + LY::Q_DBT);
    float* s_dTT = (float*)(smem + LY::Q_DTT);
    float* s_op = (float*)(smem + LY::Q_OP);  // [6][SLB][LDC]
    float* s_cp = (float*)(smem + LY::OFF_CP);
    float* s_p6 = (float*)(smem + LY::OFF_P6);
    float* s_bt = (float*)(smem + LY::OFF_BT);
    float* s_rp = (float*)(smem + LY::OFF_RP);
    float2* s_bm = (float2*)(smem + LY::OFF_BM);

    const int H = a.H, DV = a.DV;
    const int g = (int)(blockIdx.x / H), h = (int)(blockIdx.x % H);
    int n, c0, c1;
    bool last;
    if (!locate_chunk<C>(a.cm, g, n, c0, c1, last)) return;
    const int L = c1 - c0;
    const int tid = threadIdx.x, lane = tid & 63, li = lane & 15, lg = lane >> 4;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int rb = w & 3, cw = w >> 2;
    const size_t gh = (size_t)g * H + h;
    const char* rec = a.rec + gh * R::BYTES;
    const float* __restrict__ kap = (const float*)(rec + R::OFF_KAP);
    const float* __restrict__ phat = (const float*)(rec + R::OFF_PHAT);
    const double* __restrict__ lam = (const double*)(rec + R::OFF_LAM);
    const float* __restrict__ gC = (const float*)(rec + R::OFF_GC);
    const float* __restrict__ den = (const float*)(rec + R::OFF_DEN);
    float* __restrict__ dkap = a.dkap + gh * C * DK;
    float* __restrict__ dal = a.dal + gh * C * DK;
    float* __restrict__ gq = a.dq;
    float* __restrict__ gk = a.dk;
    auto row = [&](int t) { return (size_t)(c0 + t) * H + h; };

    // ---- 1. products over the value columns -------------------------------------------------
    floatx4 p3[NCW], p4[NCW], p5[NCW], p1[2], p2[2];
#pragma unroll
    for (int k = 0; k < NCW; ++k) p3[k] = p4[k] = p5[k] = zero4();
    // lower blocks numbered row by row: 0 (0,0), 1 (1,0), 2 (1,1), 3 (2,0), ..., 9 (3,3)
    int pbt[2], pbs[2];
    bool pbo[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int q = w + 8 * u;
        pbo[u] = q < 10;
        pbt[u] = q < 1 ? 0 : (q < 3 ? 1 : (q < 6 ? 2 : 3));
        pbs[u] = q - pbt[u] * (pbt[u] + 1) / 2;
        p1[u] = p2[u] = zero4();
    }
    float p6 = 0.f;  // thread: channel tid / 4, columns 8 (tid % 4) .. + 7 of each slab
    // slab pieces of 4 columns, loaded into registers one slab ahead: Delta, Psi, dO (one piece
    // of each per thread), S_in and dS_out (NP2 pieces)
    constexpr int NP2 = DK * SW / 4, PP2 = (NP2 + NTB - 1) / NTB;
    static_assert(C * SW / 4 == NTB, "one row piece per thread");
    floatx4 vd, vp, vo, vs[PP2], vg[PP2];
    auto load1 = [&](int j0) {
        const int SWc = min(SW, DV - j0);
        const floatx4 z = {0.f, 0.f, 0.f, 0.f};
        {
            const int t = tid / (SW / 4), j4 = 4 * (tid % (SW / 4));
            const bool in = j4 < SWc, ok = in && t < L;
            const size_t o = row(t) * DV + j0 + j4;
            vd = in ? *reinterpret_cast<const floatx4*>(a.dlt + (gh * C + t) * DV + j0 + j4) : z;
            vp = ok ? *reinterpret_cast<const floatx4*>(a.dv + o) : z;
            floatx4 ov = z;
            if (ok && a.dO) {
                ov[0] = ld<TI>(a.dO, o);
                ov[1] = ld<TI>(a.dO, o + 1);
                ov[2] = ld<TI>(a.dO, o + 2);
                ov[3] = ld<TI>(a.dO, o + 3);
            }
            vo = ov;
        }
#pragma unroll
        for (int u = 0; u < PP2; ++u) {
            const int e = min(tid + NTB * u, NP2 - 1), i = e / (SW / 4), j4 = 4 * (e % (SW / 4));
            const size_t o = (gh * DK + i) * DV + j0 + j4;
            vs[u] = j4 < SWc ? *reinterpret_cast<const floatx4*>(a.ckpt + o) : z;
            vg[u] = j4 < SWc ? *reinterpret_cast<const floatx4*>(a.dso + o) : z;
        }
    };
    auto store1 = [&]() {
        {
            const int t = tid / (SW / 4), j4 = 4 * (tid % (SW / 4));
            *reinterpret_cast<floatx4*>(s_D + t * LDW + j4) = vd;
            *reinterpret_cast<floatx4*>(s_P + t * LDW + j4) = vp;
            *reinterpret_cast<floatx4*>(s_O + t * LDW + j4) = vo;
        }
#pragma unroll
        for (int u = 0; u < PP2; ++u) {
            const int e = tid + NTB * u, i = e / (SW / 4), j4 = 4 * (e % (SW / 4));
            if (e < NP2) {
                *reinterpret_cast<floatx4*>(s_S + i * LDW + j4) = vs[u];
                *reinterpret_cast<floatx4*>(s_G + i * LDW + j4) = vg[u];
            }
        }
    };
    load1(0);
    for (int j0 = 0; j0 < DV; j0 += SW) {
        const int SWc = min(SW, DV - j0);  // 16 or 32
        __syncthreads();
        store1();
        if (j0 + SW < DV) load1(j0 + SW);
        __syncthreads();
        for (int ks = 0; ks < SWc / 16; ++ks) {
            const int kc = 16 * ks + 4 * lg;
            const FF::V aP = FF::ld(s_P + (16 * rb + li) * LDW + kc);
            const FF::V aO = FF::ld(s_O + (16 * rb + li) * LDW + kc);
            const FF::V aD = FF::ld(s_D + (16 * rb + li) * LDW + kc);
#pragma unroll
            for (int k = 0; k < NCW; ++k) {
                const int ct = cw + 2 * k;
                if (ct < NKT) {
                    const FF::V bS = FF::ld(s_S + (16 * ct + li) * LDW + kc);
                    const FF::V bG = FF::ld(s_G + (16 * ct + li) * LDW + kc);
                    p3[k] = FF::mma(p3[k], aP, bS);
                    p4[k] = FF::mma(p4[k], aO, bS);
                    p5[k] = FF::mma(p5[k], aD, bG);
                }
            }
#pragma unroll
            for (int u = 0; u < 2; ++u)
                if (pbo[u]) {
                    const FF::V bD = FF::ld(s_D + (16 * pbs[u] + li) * LDW + kc);
                    p1[u] = FF::mma(p1[u], FF::ld(s_O + (16 * pbt[u] + li) * LDW + kc), bD);
                    p2[u] = FF::mma(p2[u], FF::ld(s_P + (16 * pbt[u] + li) * LDW + kc), bD);
                }
        }
        if (tid < 4 * DK) {
            const int i = tid >> 2, jq = 8 * (tid & 3);
            if (jq < SWc)
#pragma unroll
                for (int jj = 0; jj < 8; ++jj)
                    p6 = fmaf(s_S[i * LDW + jq + jj], s_G[i * LDW + jq + jj], p6);
        }
    }
    p6 += __shfl_xor(p6, 1, 64);
    p6 += __shfl_xor(p6, 2, 64);
    if (tid < 4 * DK && (tid & 3) == 0) s_p6[tid >> 2] = p6;
    __syncthreads();  // the slabs are dead: the adjoints of B and T over them
#pragma unroll
    for (int u = 0; u < 2; ++u)
        if (pbo[u])
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int t = 16 * pbt[u] + 4 * lg + r, s2 = 16 * pbs[u] + li;
                const float b = s2 <= t ? a.scale * p1[u][r] : 0.f;  // dB = scale dO Delta^T
                const float tt = s2 < t ? -p2[u][r] : 0.f;            // dT = -Psi Delta^T
                s_dB[t * LDC + s2] = b;
                s_dBT[s2 * LDC + t] = b;
                s_dT[t * LDC + s2] = tt;
                s_dTT[s2 * LDC + t] = tt;
            }
    // terms through S_in (O = scale Qbar S_in, X = V - Kbar S_in) and the tail operand
    // (S_out = ... + Ktail^T Delta); the chunk-end decay's column sums of kappa dkappa_tail
    floatx4 gqa[NCW], gka[NCW], gpa[NCW];
#pragma unroll
    for (int k = 0; k < NCW; ++k) {
        gqa[k] = gka[k] = gpa[k] = zero4();
        const int ct = cw + 2 * k;
        if (ct >= NKT) continue;
        const int i = 16 * ct + li;
        const double lmC = lam[(C - 1) * DK + i];
        float cs = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int t = 16 * rb + 4 * lg + r;
            const double lm = lam[t * DK + i];
            const float gm = expf((float)lm), et = expf((float)(lmC - lm));
            gqa[k][r] = a.scale * gm * p4[k][r];
            gka[k][r] = -gm * p3[k][r];
            gpa[k][r] = et * p5[k][r];
            cs = fmaf(kap[t * DK + i], gpa[k][r], cs);
        }
        cs += __shfl_xor(cs, 16, 64);
        cs += __shfl_xor(cs, 32, 64);
        if (lg == 0) s_cp[rb * DK + i] = cs;
    }

    // ---- 2. terms through T and B, by channel slabs ------------------------------------------
    // formation inputs of a slab, loaded into registers one slab ahead. Thread: channel
    // s0 + tid % SLB, tokens 4 (tid / SLB) .. + 3 (one block)
    const bool fth = tid < SLB * 16;
    const int fii = tid % SLB, ftg = min(tid / SLB, 15), fb = ftg >> 2, ft0 = 4 * ftg;
    double flm[4], fst = 0.0, fen = 0.0, frf = 0.0;
    float fkp[4], fq[4], fk[4];
    auto load2 = [&](int s0) {
        const int i = s0 + fii;
        fst = fb > 0 ? lam[(16 * fb - 1) * DK + i] : 0.0;
        fen = lam[(16 * fb + 15) * DK + i];
        frf = lam[(16 * fb + 7) * DK + i];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int t = ft0 + u;
            const bool ok = t < L;
            flm[u] = lam[t * DK + i];
            fkp[u] = kap[t * DK + i];
            fq[u] = ok ? ld<TI>(a.q, row(t) * DK + i) : 0.f;
            fk[u] = ok ? ld<TI>(a.k, row(t) * DK + i) : 0.f;
        }
    };
    if (fth) load2(0);
    for (int s0 = 0, kk = 0; s0 < DK; s0 += SLB, ++kk) {
        __syncthreads();  // dB and dT written; the previous slab's operands read
        // operands, transposed [ii][t]: kappa scaled to the end of its block and to the block's
        // token 8 (the column side of dq, dk); q and k scaled from the start of their block and
        // from its token 8 (the column side of dkappa)
        if (fth) {
            float o[6][4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const float ast = __expf((float)(flm[u] - fst));
                const float amd = fminf(__expf((float)(flm[u] - frf)), RSAT);
                const float ben = __expf((float)(fen - flm[u]));
                const float bmd = fminf(__expf((float)(frf - flm[u])), RSAT);
                o[0][u] = ben * fkp[u];
                o[1][u] = bmd * fkp[u];
                o[2][u] = ast * fq[u];
                o[3][u] = amd * fq[u];
                o[4][u] = ast * fk[u];
                o[5][u] = amd * fk[u];
            }
#pragma unroll
            for (int m = 0; m < 6; ++m)
                *reinterpret_cast<floatx4*>(s_op + m * OPS + fii * LDC + ft0) =
                    floatx4{o[m][0], o[m][1], o[m][2], o[m][3]};
            if (s0 + SLB < DK) load2(s0 + SLB);
        }
        __syncthreads();
        if (16 * cw >= SLB) continue;
        const int i = s0 + 16 * cw + li;
        const float* oKen = s_op + 0 * OPS + 16 * cw * LDC;
        const float* oKmd = s_op + 1 * OPS + 16 * cw * LDC;
        const float* oQst = s_op + 2 * OPS + 16 * cw * LDC;
        const float* oQmd = s_op + 3 * OPS + 16 * cw * LDC;
        const float* oKst = s_op + 4 * OPS + 16 * cw * LDC;
        const float* oKm2 = s_op + 5 * OPS + 16 * cw * LDC;
        // log-decays of channel i: before, at the end of and at token 8 of every block; rows
        double lst[4], len[4], lrf[4], lrow[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            lst[b] = b > 0 ? lam[(16 * b - 1) * DK + i] : 0.0;
            len[b] = lam[(16 * b + 15) * DK + i];
            lrf[b] = lam[(16 * b + 7) * DK + i];
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) lrow[r] = lam[(16 * rb + 4 * lg + r) * DK + i];
        const int ar = (16 * rb + li) * LDC, kc = 4 * lg;
        // rows of block rb as the later token: dq += sum_s dB_ts kappa_s R_ts,
        // dk += sum_s dT_ts kappa_s R_ts
        {
            floatx4 oB = zero4(), oT = zero4();
            for (int jb = 0; jb < rb; ++jb) {
                const FF::V bk = FF::ld(oKen + li * LDC + 16 * jb + kc);
                const floatx4 tB = FF::mma(zero4(), FF::ld(s_dB + ar + 16 * jb + kc), bk);
                const floatx4 tT = FF::mma(zero4(), FF::ld(s_dT + ar + 16 * jb + kc), bk);
                const float m = __expf((float)(lst[rb] - len[jb]));
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    oB[r] = fmaf(m, tB[r], oB[r]);
                    oT[r] = fmaf(m, tT[r], oT[r]);
                }
            }
            const FF::V bk = FF::ld(oKmd + li * LDC + 16 * rb + kc);
            const floatx4 dB = FF::mma(zero4(), FF::ld(s_dB + ar + 16 * rb + kc), bk);
            const floatx4 dT = FF::mma(zero4(), FF::ld(s_dT + ar + 16 * rb + kc), bk);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float ast = __expf((float)(lrow[r] - lst[rb]));
                const float amd = fminf(__expf((float)(lrow[r] - lrf[rb])), RSAT);
                gqa[kk][r] += ast * oB[r] + amd * dB[r];
                gka[kk][r] += ast * oT[r] + amd * dT[r];
            }
        }
        // rows of block rb as the earlier token: dkappa += sum_t (dB_ts q_t + dT_ts k_t) R_ts
        {
            floatx4 oB = zero4(), oT = zero4();
            for (int ib = rb + 1; ib < 4; ++ib) {
                const floatx4 tB = FF::mma(zero4(), FF::ld(s_dBT + ar + 16 * ib + kc),
                                           FF::ld(oQst + li * LDC + 16 * ib + kc));
                const floatx4 tT = FF::mma(zero4(), FF::ld(s_dTT + ar + 16 * ib + kc),
                                           FF::ld(oKst + li * LDC + 16 * ib + kc));
                const float m = __expf((float)(lst[ib] - len[rb]));
#pragma unroll
                for (int r = 0; r < 4; ++r) oB[r] = fmaf(m, tB[r] + tT[r], oB[r]);
            }
            const floatx4 dB = FF::mma(zero4(), FF::ld(s_dBT + ar + 16 * rb + kc),
                                       FF::ld(oQmd + li * LDC + 16 * rb + kc));
            const floatx4 dT = FF::mma(zero4(), FF::ld(s_dTT + ar + 16 * rb + kc),
                                       FF::ld(oKm2 + li * LDC + 16 * rb + kc));
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float ben = __expf((float)(len[rb] - lrow[r]));
                const float bmd = fminf(__expf((float)(lrf[rb] - lrow[r])), RSAT);
                gpa[kk][r] += ben * oB[r] + bmd * (dB[r] + dT[r]);
            }
            (void)oT;
        }
    }

    // ---- the gradients out; the log-decay adjoint q dq + k dk - kappa dkappa, its suffix sums
    // over the chunk (alpha dalpha = sum over t >= s; the chunk-end terms enter at the last
    // token) and the coefficients of the variance adjoint lambda_{t-1} = A_t lambda_t + B_t, all
    // on the owned tiles. Row sums over the channels (the gain denominator's adjoint; isotropic:
    // dbeta, ||k||^2, sum alpha^2) reduce within a tile row, then over the two waves of a row
    // block; the suffix sums run within a tile, then over the row blocks --------------------------
    float kvv[NCW][4], alv[NCW][4], suf[NCW][4], phv[NCW][4];
    float rrv[4], dnv[4];  // r and the gain denominator of the lane's rows
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int t = 16 * rb + 4 * lg + r;
        rrv[r] = t < L ? ld<TI>(a.r, row(t)) : 1.f;
        dnv[r] = den[t];
    }
    float rp0[4] = {0.f, 0.f, 0.f, 0.f}, rp1[4] = {0.f, 0.f, 0.f, 0.f};
    float rp2[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < NCW; ++k) {
        const int ct = cw + 2 * k;
#pragma unroll
        for (int r = 0; r < 4; ++r) kvv[k][r] = alv[k][r] = suf[k][r] = phv[k][r] = 0.f;
        if (ct >= NKT) continue;
        const int i = 16 * ct + li;
        if (DIAG)
#pragma unroll
            for (int r = 0; r < 4; ++r) phv[k][r] = phat[(16 * rb + 4 * lg + r) * DK + i];
        float x0[4], x1[4], x2[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int t = 16 * rb + 4 * lg + r;
            const bool ok = t < L;
            const float qq = ok ? ld<TI>(a.q, row(t) * DK + i) : 0.f;
            const float kv = ok ? ld<TI>(a.k, row(t) * DK + i) : 0.f;
            const float al =
                ok ? (APC ? ld<TI>(a.alpha, row(t) * DK + i) : ld<TI>(a.alpha, row(t))) : 1.f;
            const float kp = kap[t * DK + i];
            if (ok) {
                gq[row(t) * DK + i] = gqa[k][r];
                gk[row(t) * DK + i] = gka[k][r];
            }
            dkap[t * DK + i] = gpa[k][r];
            suf[k][r] = qq * gqa[k][r] + kv * gka[k][r] - kp * gpa[k][r];
            kvv[k][r] = kv;
            alv[k][r] = al;
            x0[r] = DIAG ? gpa[k][r] * kp : gpa[k][r] * kv;
            x1[r] = kv * kv;
            x2[r] = al * al;
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {  // over the tile's 16 channels (the lanes of a row)
            x0[r] = row16_sum(x0[r]);
            if (!DIAG) {
                x1[r] = row16_sum(x1[r]);
                if (APC) x2[r] = row16_sum(x2[r]);
            }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            rp0[r] += x0[r];
            rp1[r] += x1[r];
            rp2[r] += x2[r];
        }
        // suffix within the tile: the lane's rows, then the lanes of the later rows
#pragma unroll
        for (int r = 2; r >= 0; --r) suf[k][r] += suf[k][r + 1];
        const float tot = suf[k][0];
        const float g1 = __shfl(tot, li + 16, 64), g2 = __shfl(tot, li + 32, 64);
        const float g3 = __shfl(tot, li + 48, 64);
        const float later = (lg < 1 ? g1 : 0.f) + (lg < 2 ? g2 : 0.f) + (lg < 3 ? g3 : 0.f);
#pragma unroll
        for (int r = 0; r < 4; ++r) suf[k][r] += later;
        if (lg == 0) s_bt[rb * DK + i] = suf[k][0];
    }
    if (li == 0)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int t = 16 * rb + 4 * lg + r;
            s_rp[(cw * 3 + 0) * C + t] = rp0[r];
            s_rp[(cw * 3 + 1) * C + t] = rp1[r];
            s_rp[(cw * 3 + 2) * C + t] = rp2[r];
        }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < NCW; ++k) {
        const int ct = cw + 2 * k;
        if (ct >= NKT) continue;
        const int i = 16 * ct + li;
        float off = gC[i] * s_p6[i];
#pragma unroll
        for (int b = 0; b < 4; ++b) off += s_cp[b * DK + i] + (b > rb ? s_bt[b * DK + i] : 0.f);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int t = 16 * rb + 4 * lg + r;
            dal[t * DK + i] = t < L ? (suf[k][r] + off) * __builtin_amdgcn_rcpf(alv[k][r]) : 0.f;
        }
        if constexpr (DIAG) {
            float av[4], bv[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int t = 16 * rb + 4 * lg + r;
                const bool ok = t < L;
                // 1 / r_t, 1 / den_t and 1 / (1 + u p_hat): hardware reciprocals (1 ulp)
                const float irr = __builtin_amdgcn_rcpf(rrv[r]);
                const float idn = __builtin_amdgcn_rcpf(dnv[r]);
                const float dden = -(s_rp[0 * C + t] + s_rp[3 * C + t]) * idn;
                const float kv = kvv[k][r], al = alv[k][r];
                const float u = a.mu * kv * kv * irr;
                const float ig = __builtin_amdgcn_rcpf(fmaf(u, phv[k][r], 1.f));
                const float c = gpa[k][r] * kv * idn + dden * kv * kv;
                av[r] = ok ? al * al * ig * ig : 1.f;
                bv[r] = ok ? al * al * c : 0.f;
                a.acf[(gh * C + t) * NCHAN + i] = av[r];
                a.bcf[(gh * C + t) * NCHAN + i] = bv[r];
                if (k == 0 && cw == 0 && li == 0) a.aux[gh * C + t] = dden;
            }
            // the block's map of the variance adjoint (lambda_start = mx lambda_end + my): the
            // lane's rows composed from the last down, then the lane groups in time order
            // (f o g: x -> f.x (g.x x + g.y) + f.y)
            float mx = 1.f, my = 0.f;
#pragma unroll
            for (int r = 3; r >= 0; --r) {
                mx *= av[r];
                my = fmaf(av[r], my, bv[r]);
            }
            float px = __shfl(mx, lane + 16, 64), py = __shfl(my, lane + 16, 64);
            my = fmaf(mx, py, my);  // groups 0, 2: own rows after the next group's
            mx *= px;
            px = __shfl(mx, lane + 32, 64);
            py = __shfl(my, lane + 32, 64);
            my = fmaf(mx, py, my);  // group 0: rows 0-7 after rows 8-15
            mx *= px;
            if (lg == 0) s_bm[rb * DK + i] = make_float2(mx, my);
        }
    }
    if constexpr (!DIAG) {  // one value per token: the row sums of both waves of the row block
        if (cw == 0 && li == 0)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int t = 16 * rb + 4 * lg + r;
                const bool ok = t < L;
                const float rr = rrv[r], dn = dnv[r];
                const float dbeta = s_rp[0 * C + t] + s_rp[3 * C + t];
                const float nk = s_rp[1 * C + t] + s_rp[4 * C + t];
                float aa;
                if (APC) aa = (s_rp[2 * C + t] + s_rp[5 * C + t]) / (float)DK;
                else {
                    const float al = ok ? ld<TI>(a.alpha, row(t)) : 1.f;
                    aa = al * al;
                }
                const float bh = phat[t * DK];
                const float u = a.mu * nk / ((float)DK * rr), gg = 1.f + u * bh;
                a.acf[gh * C + t] = ok ? aa / (gg * gg) : 1.f;
                a.bcf[gh * C + t] = ok ? aa * dbeta * rr / (dn * dn) : 0.f;
                a.aux[gh * C + t] = dbeta;
            }
    }
    // the chunk's map of the variance adjoint from its end to its start, per channel:
    // lambda_start = m.x lambda_end + m.y, the steps lambda_{t-1} = A_t lambda_t + B_t composed
    // from the last token down: diagonal, the four row blocks' maps in time order; isotropic,
    // the one chain's coefficients (this workgroup's own writes above)
    __syncthreads();
    if constexpr (DIAG) {
        if (tid < DK) {
            float2 m = s_bm[3 * DK + tid];
#pragma unroll
            for (int b = 2; b >= 0; --b) {
                const float2 f = s_bm[b * DK + tid];
                m = make_float2(f.x * m.x, fmaf(f.x, m.y, f.y));
            }
            a.cmap[gh * NCHAN + tid] = m;
        }
    } else if (tid < NCHAN) {
        float mx = 1.f, my = 0.f;
        for (int tb = C - 16; tb >= 0; tb -= 16) {
            float av[16], bv[16];
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                av[e] = a.acf[(gh * C + tb + e) * NCHAN + tid];
                bv[e] = a.bcf[(gh * C + tb + e) * NCHAN + tid];
            }
#pragma unroll
            for (int e = 15; e >= 0; --e) {
                mx *= av[e];
                my = fmaf(av[e], my, bv[e]);
            }
        }
        a.cmap[gh * NCHAN + tid] = make_float2(mx, my);
    }
}

// ------------------------------------------------------------------------------------------
// bw_scan: the variance adjoint backwards over the chunks, one thread per (sequence, head,
// channel): each chunk's composed map (from bw_grad) applied in reverse; the adjoint at every
// chunk's end is kept for bw_final, which replays the chunk's tokens from it
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(64) void bw_scan(Args a, int nchan)
{
    const int gid = (int)(blockIdx.x * 64 + threadIdx.x);
    const int H = a.H;
    if (gid >= a.cm.N * H * nchan) return;
    const int slot = gid / nchan, c = gid % nchan, n = slot / H, h = slot % H;
    int t0, t1, g0, nch;
    seq_span(a.cm, n, t0, t1);
    seq_chunks<C>(a.cm, n, t0, t1, g0, nch);
    float lp = a.dP_T ? a.dP_T[(size_t)slot * nchan + c] : 0.f;
    for (int cb = nch; cb > 0; cb -= 16) {  // chunks cb - 1 down to max(cb - 16, 0)
        float2 mv[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int ci = max(cb - 1 - e, 0);
            mv[e] = a.cmap[((size_t)(g0 + ci) * H + h) * nchan + c];
        }
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int ci = cb - 1 - e;
            if (ci >= 0) {
                a.lpe[((size_t)(g0 + ci) * H + h) * nchan + c] = lp;
                lp = fmaf(mv[e].x, lp, mv[e].y);
            }
        }
    }
    if (a.dP0) a.dP0[(size_t)slot * nchan + c] = lp;
}

// ------------------------------------------------------------------------------------------
// bw_final: token-local gradients of the gain stage
// ------------------------------------------------------------------------------------------
template <class TI, int DK, int VARIANT, bool APC>
__global__ __launch_bounds__(NTH) void bw_final(Args a)
{
    using R = BwRec<DK>;
    constexpr bool DIAG = VARIANT == 0;
    constexpr int NCHAN = DIAG ? DK : 1;
    const int H = a.H;
    const int g = (int)(blockIdx.x / H), h = (int)(blockIdx.x % H);
    int n, c0, c1;
    bool last;
    if (!locate_chunk<C>(a.cm, g, n, c0, c1, last)) return;
    const int L = c1 - c0;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const size_t gh = (size_t)g * H + h;
    const char* rec = a.rec + gh * R::BYTES;
    const float* phat = (const float*)(rec + R::OFF_PHAT);
    const float* pprv = (const float*)(rec + R::OFF_PPRV);
    const float* den = (const float*)(rec + R::OFF_DEN);
    const float* dkap = a.dkap + gh * C * DK;
    const float* dal = a.dal + gh * C * DK;
    const float mu = a.mu;
    // the variance adjoint at every token of the chunk, replayed from its value at the chunk's
    // end: lambda_{t-1} = A_t lambda_t + B_t
    __shared__ float s_lp[C * NCHAN];
    if (tid < NCHAN) {
        float lp = a.lpe[gh * NCHAN + tid];
        for (int tb = C - 16; tb >= 0; tb -= 16) {
            float av[16], bv[16];
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                av[e] = a.acf[(gh * C + tb + e) * NCHAN + tid];
                bv[e] = a.bcf[(gh * C + tb + e) * NCHAN + tid];
            }
#pragma unroll
            for (int e = 15; e >= 0; --e) {
                s_lp[(tb + e) * NCHAN + tid] = lp;
                lp = fmaf(av[e], lp, bv[e]);
            }
        }
    }
    __syncthreads();
    constexpr int NI = (DK + 63) / 64;  // channels per lane: i = lane + 64 ii
#pragma unroll 4
    for (int j = 0; j < C / 4; ++j) {
        const int t = (C / 4) * w + j;
        if (t >= L) continue;  // uniform per wave
        const size_t row = (size_t)(c0 + t) * H + h;
        const float rr = ld<TI>(a.r, row), dn = den[t], aux = a.aux[gh * C + t];
        if constexpr (DIAG) {
            // 1 / r_t and 1 / den_t once per token, 1 / (1 + u p_hat) per channel: hardware
            // reciprocals (1 ulp)
            const float irr = __builtin_amdgcn_rcpf(rr), idn = __builtin_amdgcn_rcpf(dn);
            const float dden = aux;
            float s2 = 0.f;
#pragma unroll
            for (int ii = 0; ii < NI; ++ii) {
                const int i = lane + 64 * ii;
                if (i >= DK) break;
                const float kk = ld<TI>(a.k, row * DK + i), al = ld<TI>(a.alpha, row * DK + i);
                const float ph = phat[t * DK + i], pp = pprv[t * DK + i];
                const float dkp = dkap[t * DK + i];
                const float lp = s_lp[t * NCHAN + i];
                const float u = mu * kk * kk * irr;
                const float ig = __builtin_amdgcn_rcpf(fmaf(u, ph, 1.f)), ig2 = ig * ig;
                const float dph = dkp * kk * idn + dden * kk * kk + lp * ig2;
                const float du = -lp * ph * ph * ig2;
                a.dk[row * DK + i] +=
                    dkp * ph * idn + 2.f * dden * ph * kk + du * 2.f * mu * kk * irr;
                s2 += du * mu * kk * kk;
                a.dalpha[row * DK + i] = dal[t * DK + i] + dph * 2.f * al * pp;
                a.domega[row * DK + i] = dph;
            }
            s2 = wave_sum(s2);
            if (lane == 0) a.dr[row] = dden - s2 * irr * irr;
        } else {
            const float dbeta = aux, bh = phat[t * DK], pp = pprv[t * DK];
            const float lp = s_lp[t];
            float sk = 0.f, sa = 0.f, sd = 0.f;
            for (int i = lane; i < DK; i += 64) {
                const float kk = ld<TI>(a.k, row * DK + i);
                sk += kk * kk;
                sd += dal[t * DK + i];
            }
            const float nk = wave_sum(sk);
            sd = wave_sum(sd);
            const float a0 = APC ? 0.f : ld<TI>(a.alpha, row);
            (void)sa;
            const float beta = bh / dn;
            const float u = mu * nk / ((float)DK * rr), gg = 1.f + u * bh, ig2 = 1.f / (gg * gg);
            const float dbh = lp * ig2 + dbeta * rr / (dn * dn);
            const float du = -lp * bh * bh * ig2;
            const float dr = -dbeta * bh / (dn * dn) - du * mu * nk / ((float)DK * rr * rr);
            const float dnk = -dbeta * bh * bh / (dn * dn) + du * mu / ((float)DK * rr);
            const float da = dbh * pp;
            for (int i = lane; i < DK; i += 64) {
                const float kk = ld<TI>(a.k, row * DK + i);
                a.dk[row * DK + i] += beta * dkap[t * DK + i] + 2.f * kk * dnk;
                if (APC) {
                    const float al = ld<TI>(a.alpha, row * DK + i);
                    a.dalpha[row * DK + i] = dal[t * DK + i] + da * 2.f * al / (float)DK;
                }
            }
            if (lane == 0) {
                a.dr[row] = dr;
                a.domega[row] = dbh;
                if (!APC) a.dalpha[row] = sd + da * 2.f * a0;
            }
        }
    }
}

// ------------------------------------------------------------------------------------------
// host side
// ------------------------------------------------------------------------------------------
template <class K>
hipError_t lds_attr(K* kernel, size_t bytes)
{
    if (bytes <= 64 * 1024) return hipSuccess;
    return hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)bytes);
}

size_t rec_bytes(int dk)
{
    switch (dk) {
    case 16: return BwRec<16>::BYTES;
    case 32: return BwRec<32>::BYTES;
    case 64: return BwRec<64>::BYTES;
    default: return BwRec<128>::BYTES;
    }
}

template <class TI, int DK, int VARIANT, bool APC>
hipError_t run(const BwdCall& bc, hipStream_t st)
{
    using VC = fwd::VarCfg<TI, DK, VARIANT, APC>;
    const SeqArgs& sa = bc.sa;
    const bool packed = sa.cu_seqlens != nullptr;
    const BwMap m = bw_map(VARIANT, packed, sa.N, sa.B, sa.T, sa.H, DK, bc.dv, BwRec<DK>::BYTES);
    char* ws = (char*)bc.workspace;
    hipError_t e;
    ChunkMap cm;
    cm.cu = sa.cu_seqlens;
    cm.choff = packed ? (const int32_t*)(ws + m.choff) : nullptr;
    cm.N = sa.N;
    cm.T = sa.T;
    cm.ntok = sa.B * sa.T;
    cm.maxch = m.maxch;
    if (packed &&
        (e = launch_chunk_table(sa.cu_seqlens, sa.N, cm.ntok, C, m.maxch,
                                (int32_t*)(ws + m.choff), st)) != hipSuccess)
        return e;
    const size_t ntok = (size_t)sa.B * sa.T * sa.H;
    fwd::InArgs in = {};
    in.q = bc.q; in.k = bc.k; in.alpha = bc.alpha; in.omega = bc.omega; in.r = bc.r;
    in.bytes_k = (uint32_t)(ntok * DK * sizeof(TI));
    in.bytes_h = (uint32_t)(ntok * sizeof(TI));
    in.H = sa.H;
    in.mu = bc.mu;
    float4* summ = (float4*)(ws + m.summ);
    float2* carry = (float2*)(ws + m.carry);
    const dim3 cgrid((unsigned)((size_t)m.maxch * sa.H));
    if (m.maxch > 0) {
        hipLaunchKernelGGL((fwd::summary_kernel<TI, VC>), cgrid, dim3(NTH), 0, st, in, cm, summ);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = launch_carry_scan(summ, bc.P0, cm, C, sa.H, VC::NCHAN, carry, nullptr, st)) !=
            hipSuccess)
            return e;
    }
    Args a = {};
    a.q = bc.q; a.k = bc.k; a.v = bc.v; a.alpha = bc.alpha; a.omega = bc.omega; a.r = bc.r;
    a.dO = bc.dO; a.S0 = bc.S0; a.dS_T = bc.dS_T; a.dP_T = bc.dP_T;
    a.dq = bc.gq; a.dk = bc.gk; a.dv = bc.gv; a.dalpha = bc.galpha; a.domega = bc.gomega;
    a.dr = bc.gr; a.dS0 = bc.gS0; a.dP0 = bc.gP0;
    a.cm = cm;
    a.H = sa.H;
    a.DV = bc.dv;
    a.BV = bc.dv < 32 ? bc.dv : 32;
    a.mu = bc.mu;
    a.scale = bc.scale;
    a.carry = carry;
    a.rec = ws + m.rec;
    a.ckpt = (float*)(ws + m.ckpt);
    a.dlt = (float*)(ws + m.dlt);
    a.dso = (float*)(ws + m.dso);
    a.dkap = (float*)(ws + m.dkap);
    a.dal = (float*)(ws + m.dal);
    a.acf = (float*)(ws + m.acf);
    a.bcf = (float*)(ws + m.bcf);
    a.aux = (float*)(ws + m.aux);
    a.cmap = (float2*)(ws + m.cmap);
    a.lpe = (float*)(ws + m.lpe);
    static bool attr = false;
    if (!attr) {
        if ((e = lds_attr(bw_prep<TI, DK, VARIANT, APC>, PrepLds<DK>::TOTAL)) != hipSuccess ||
            (e = lds_attr(bw_fwalk<TI, DK>, WalkLds<DK>::F_TOTAL)) != hipSuccess ||
            (e = lds_attr(bw_rwalk<TI, DK>, WalkLds<DK>::R_TOTAL)) != hipSuccess ||
            (e = lds_attr(bw_grad<TI, DK, VARIANT, APC>, GradLds<DK>::TOTAL)) != hipSuccess)
            return e;
        attr = true;
    }
    if (m.maxch > 0) {
        hipLaunchKernelGGL((bw_prep<TI, DK, VARIANT, APC>), cgrid, dim3(NTB), PrepLds<DK>::TOTAL,
                           st, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const int NV = bc.dv / a.BV;
    const dim3 wgrid((unsigned)(((size_t)sa.N * sa.H + 7) / 8 * 8 * NV));
    hipLaunchKernelGGL((bw_fwalk<TI, DK>), wgrid, dim3(NTB), WalkLds<DK>::F_TOTAL, st, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((bw_rwalk<TI, DK>), wgrid, dim3(NTB), WalkLds<DK>::R_TOTAL, st, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (m.maxch > 0) {
        hipLaunchKernelGGL((bw_grad<TI, DK, VARIANT, APC>), cgrid, dim3(NTB), GradLds<DK>::TOTAL,
                           st, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const int nthr = sa.N * sa.H * VC::NCHAN;
    hipLaunchKernelGGL(bw_scan, dim3((unsigned)((nthr + 63) / 64)), dim3(64), 0, st, a,
                       (int)VC::NCHAN);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (m.maxch > 0) {
        hipLaunchKernelGGL((bw_final<TI, DK, VARIANT, APC>), cgrid, dim3(NTH), 0, st, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

template <class TI, int DK>
hipError_t run_v(const BwdCall& bc, hipStream_t st)
{
    if (bc.variant == 0) return run<TI, DK, 0, true>(bc, st);
    if (bc.apc) return run<TI, DK, 1, true>(bc, st);
    return run<TI, DK, 1, false>(bc, st);
}

template <class TI>
hipError_t run_dk(const BwdCall& bc, hipStream_t st)
{
    switch (bc.dk) {
    case 16: return run_v<TI, 16>(bc, st);
    case 32: return run_v<TI, 32>(bc, st);
    case 64: return run_v<TI, 64>(bc, st);
    case 128: return run_v<TI, 128>(bc, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace bwd

size_t backward_workspace_bytes(int variant, bool packed, int N, int B, int T, int H, int dk,
                                int dv)
{
    return bwd::bw_map(variant, packed, N, B, T, H, dk, dv, bwd::rec_bytes(dk)).total;
}

hipError_t launch_backward(const BwdCall& bc, hipStream_t stream)
{
    if (bc.dtype == KDN_F32) return bwd::run_dk<float>(bc, stream);
    return bwd::run_dk<bf16>(bc, stream);
}

}  // namespace kdn
