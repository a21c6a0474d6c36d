// Single-token recurrent decode for Diagonal and Isotropic KDN on gfx950.
//
// One step of Prop. "Diagonal Kalman Delta Network" / Prop. "Isotropic Kalman Delta Network"
// (arXiv 2609.07816) per row, with the float32 state resident in a slot pool and updated in
// place. The step is bound by HBM: each (row, head) streams its dk x dv state once in and once
// out. One workgroup owns one (row, head): every thread keeps RPT rows x 4 columns of S in
// registers between the innovation reduction (delta = v - (diag(alpha) S)^T k) and the read
// (o = scale S^T q), so S crosses HBM exactly twice.
#include "kdn_internal.h"

namespace kdn {
namespace {

template <int DK, int DV>
struct DecodeShape {
    static constexpr int NCG = DV / 4;                                   // float4 column groups
    static constexpr int NT = (DK * DV / 4) < 256 ? (DK * DV / 4) : 256; // threads
    static constexpr int NRG = NT / NCG;                                 // row groups
    static constexpr int RPT = DK / NRG;                                 // rows per thread
    static constexpr int NW = (NT + 63) / 64;                            // waves
};

// Block-wide sum of one value per thread (NT threads, NW waves).
template <int NW>
__device__ __forceinline__ float block_sum(float x, float* scratch)
{
    x = wave_sum(x);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    if (NW == 1) return x;
    __syncthreads();
    if (lane == 0) scratch[w] = x;
    __syncthreads();
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NW; ++i) s += scratch[i];
    return s;
}

// The layer options of one decode call on the device (all off for kdn_decode_step).
template <class T>
struct DecLayer {
    int preact, qknorm;
    float r_min;
    const T* mu_t;    // [R,H] or nullptr
    float* beta_eff;  // [R,H] float32 or nullptr
};

template <class T, int DK, int DV, int VARIANT, bool APC>
__global__ __launch_bounds__((DecodeShape<DK, DV>::NT)) void decode_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const T* __restrict__ alpha, const T* __restrict__ omega, const T* __restrict__ r,
    float* __restrict__ S, float* __restrict__ P, const int32_t* __restrict__ slot_idx,
    T* __restrict__ o, int R, int num_slots, int H, float mu, float scale, DecLayer<T> ly)
{
    using Sh = DecodeShape<DK, DV>;
    const int h = blockIdx.x % H;
    const int row = blockIdx.x / H;
    if (row >= R) return;
    const int slot = slot_idx ? slot_idx[row] : row;
    if (slot < 0 || slot >= num_slots) return;  // uniform across the workgroup

    __shared__ float s_alpha[DK], s_k[DK], s_q[DK], s_kappa[DK], s_delta[DV];
    __shared__ float s_red[Sh::NRG][DV];
    __shared__ float s_scr[16];
    __shared__ float s_beta;

    const int tid = threadIdx.x;
    const size_t rh = (size_t)row * H + h;       // (row, head)
    const size_t sh = (size_t)slot * H + h;      // (slot, head)
    float rr = ldf(r, rh);
    if (ly.preact) rr = ly.r_min + gate_softplus(rr);  // r = r_min + softplus(.)
    if (ly.mu_t) mu = ldf(ly.mu_t, rh);

    // the token's inputs (thread i < DK: channel i), with the layer's maps
    float ki = 0.f, qi = 0.f, ai = 0.f, wi = 0.f;
    if (tid < DK) {
        ki = ldf(k, rh * DK + tid);
        qi = ldf(q, rh * DK + tid);
        ai = (VARIANT == 0 || APC) ? ldf(alpha, rh * DK + tid) : ldf(alpha, rh);
        wi = VARIANT == 0 ? ldf(omega, rh * DK + tid) : ldf(omega, rh);
        if (ly.preact) {
            ai = gate_sigmoid(ai);
            wi = gate_softplus(wi);
        }
    }
    if (ly.qknorm) {  // q and k divided by their L2 norms (a zero row stays zero)
        const float nk2 = block_sum<Sh::NW>(ki * ki, s_scr);
        const float nq2 = block_sum<Sh::NW>(qi * qi, s_scr + 4);
        ki *= nk2 > 0.f ? __builtin_amdgcn_rsqf(nk2) : 0.f;
        qi *= nq2 > 0.f ? __builtin_amdgcn_rsqf(nq2) : 0.f;
    }

    float part = 0.f, part2 = 0.f, ph = 0.f;
    if (tid < DK) {
        s_alpha[tid] = ai;
        s_k[tid] = ki;
        s_q[tid] = qi;
        if (VARIANT == 0) {
            // predictive variance and its share of the innovation variance (eq. kla-box-gain)
            ph = ai * ai * P[sh * DK + tid] + wi;
            part = ph * ki * ki;
        } else {
            part = APC ? ai * ai : 0.f;  // trace of D^2 (eq. iso-kla-predict)
            part2 = ki * ki;             // ||k||^2
        }
    }
    const float den_or_a = block_sum<Sh::NW>(part, s_scr + 8);
    float nk = 0.f;
    if (VARIANT == 1) nk = block_sum<Sh::NW>(part2, s_scr + 12);
    if (VARIANT == 0) {
        if (tid < DK) {
            const float den = rr + den_or_a;
            s_kappa[tid] = ph * ki / den;
            const float u = mu * ki * ki / rr;  // scaled precision increment (eq. diag-cov-update)
            P[sh * DK + tid] = ph / (1.f + u * ph);
        }
        if (ly.beta_eff && tid == 0) ly.beta_eff[rh] = den_or_a / (rr + den_or_a);  // k^T kappa
    } else {
        if (tid == 0) {
            // thread 0 holds channel 0's gate, which is the head's gate when it is per head
            const float a = APC ? den_or_a / (float)DK : ai * ai;
            const float bh = a * P[sh] + wi;
            s_beta = bh / (rr + bh * nk);
            const float u = mu * nk / ((float)DK * rr);
            P[sh] = bh / (1.f + u * bh);
            if (ly.beta_eff) ly.beta_eff[rh] = s_beta * nk;  // k^T (beta k)
        }
        __syncthreads();
        if (tid < DK) s_kappa[tid] = s_beta * s_k[tid];
    }
    __syncthreads();

    // ---- stream S: innovation delta = v - (diag(alpha) S)^T k --------------------------
    const int cg = tid % Sh::NCG, rg = tid / Sh::NCG;
    float* Sb = S + sh * DK * DV;
    float4 s[Sh::RPT];
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int j = 0; j < Sh::RPT; ++j) {
        const int i = rg + j * Sh::NRG;
        s[j] = *reinterpret_cast<const float4*>(Sb + (size_t)i * DV + 4 * cg);
    }
#pragma unroll
    for (int j = 0; j < Sh::RPT; ++j) {
        const int i = rg + j * Sh::NRG;
        const float a = s_alpha[i];
        s[j].x *= a; s[j].y *= a; s[j].z *= a; s[j].w *= a;   // S_hat = diag(alpha) S
        const float kk = s_k[i];
        acc.x += kk * s[j].x; acc.y += kk * s[j].y; acc.z += kk * s[j].z; acc.w += kk * s[j].w;
    }
    *reinterpret_cast<float4*>(&s_red[rg][4 * cg]) = acc;
    __syncthreads();
    if (tid < DV) {
        float sum = 0.f;
#pragma unroll 8
        for (int g = 0; g < Sh::NRG; ++g) sum += s_red[g][tid];
        s_delta[tid] = ldf(v, rh * DV + tid) - sum;
    }
    __syncthreads();

    // ---- residual write S = S_hat + kappa delta^T, then read o = scale S^T q ------------
    const float4 dl = *reinterpret_cast<const float4*>(&s_delta[4 * cg]);
    acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int j = 0; j < Sh::RPT; ++j) {
        const int i = rg + j * Sh::NRG;
        const float kp = s_kappa[i];
        s[j].x += kp * dl.x; s[j].y += kp * dl.y; s[j].z += kp * dl.z; s[j].w += kp * dl.w;
        *reinterpret_cast<float4*>(Sb + (size_t)i * DV + 4 * cg) = s[j];
        const float qq = s_q[i];
        acc.x += qq * s[j].x; acc.y += qq * s[j].y; acc.z += qq * s[j].z; acc.w += qq * s[j].w;
    }
    __syncthreads();  // everyone finished reading s_red from the first reduction
    *reinterpret_cast<float4*>(&s_red[rg][4 * cg]) = acc;
    __syncthreads();
    if (tid < DV) {
        float sum = 0.f;
#pragma unroll 8
        for (int g = 0; g < Sh::NRG; ++g) sum += s_red[g][tid];
        o[rh * DV + tid] = from_f32<T>(scale * sum);
    }
}

template <class T, int DK, int DV>
hipError_t launch_dk_dv(int variant, int apc, const void* q, const void* k, const void* v,
                        const void* alpha, const void* omega, const void* r, float* S, float* P,
                        const int32_t* slot_idx, void* o, int R, int num_slots, int H, float mu,
                        float scale, const LayerOpts& lo, hipStream_t stream)
{
    const DecLayer<T> ly = {lo.preact, lo.qknorm, lo.r_min, (const T*)lo.mu_t, lo.beta_eff};
    const dim3 grid((unsigned)((size_t)R * H)), block(DecodeShape<DK, DV>::NT);
    const T *q_ = (const T*)q, *k_ = (const T*)k, *v_ = (const T*)v, *a_ = (const T*)alpha,
            *w_ = (const T*)omega, *r_ = (const T*)r;
    T* o_ = (T*)o;
    if (variant == 0)
        hipLaunchKernelGGL((decode_kernel<T, DK, DV, 0, true>), grid, block, 0, stream, q_, k_,
                           v_, a_, w_, r_, S, P, slot_idx, o_, R, num_slots, H, mu, scale, ly);
    else if (apc)
        hipLaunchKernelGGL((decode_kernel<T, DK, DV, 1, true>), grid, block, 0, stream, q_, k_,
                           v_, a_, w_, r_, S, P, slot_idx, o_, R, num_slots, H, mu, scale, ly);
    else
        hipLaunchKernelGGL((decode_kernel<T, DK, DV, 1, false>), grid, block, 0, stream, q_, k_,
                           v_, a_, w_, r_, S, P, slot_idx, o_, R, num_slots, H, mu, scale, ly);
    return hipGetLastError();
}

template <class T, int DK>
hipError_t launch_dk(int dv, int variant, int apc, const void* q, const void* k, const void* v,
                     const void* alpha, const void* omega, const void* r, float* S, float* P,
                     const int32_t* slot_idx, void* o, int R, int num_slots, int H, float mu,
                     float scale, const LayerOpts& lo, hipStream_t stream)
{
    switch (dv) {
    case 16: return launch_dk_dv<T, DK, 16>(variant, apc, q, k, v, alpha, omega, r, S, P,
                                             slot_idx, o, R, num_slots, H, mu, scale, lo, stream);
    case 32: return launch_dk_dv<T, DK, 32>(variant, apc, q, k, v, alpha, omega, r, S, P,
                                             slot_idx, o, R, num_slots, H, mu, scale, lo, stream);
    case 64: return launch_dk_dv<T, DK, 64>(variant, apc, q, k, v, alpha, omega, r, S, P,
                                             slot_idx, o, R, num_slots, H, mu, scale, lo, stream);
    case 128: return launch_dk_dv<T, DK, 128>(variant, apc, q, k, v, alpha, omega, r, S, P,
                                               slot_idx, o, R, num_slots, H, mu, scale, lo, stream);
    }
    return hipErrorInvalidValue;
}

template <class T>
hipError_t launch_t(int dk, int dv, int variant, int apc, const void* q, const void* k,
                    const void* v, const void* alpha, const void* omega, const void* r, float* S,
                    float* P, const int32_t* slot_idx, void* o, int R, int num_slots, int H,
                    float mu, float scale, const LayerOpts& lo, hipStream_t stream)
{
    switch (dk) {
    case 16: return launch_dk<T, 16>(dv, variant, apc, q, k, v, alpha, omega, r, S, P, slot_idx,
                                      o, R, num_slots, H, mu, scale, lo, stream);
    case 32: return launch_dk<T, 32>(dv, variant, apc, q, k, v, alpha, omega, r, S, P, slot_idx,
                                      o, R, num_slots, H, mu, scale, lo, stream);
    case 64: return launch_dk<T, 64>(dv, variant, apc, q, k, v, alpha, omega, r, S, P, slot_idx,
                                      o, R, num_slots, H, mu, scale, lo, stream);
    case 128: return launch_dk<T, 128>(dv, variant, apc, q, k, v, alpha, omega, r, S, P,
                                        slot_idx, o, R, num_slots, H, mu, scale, lo, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_decode(int variant, const void* q, const void* k, const void* v,
                         const void* alpha, const void* omega, const void* r, float* S, float* P,
                         const int32_t* slot_idx, void* o, int R, int num_slots, int H, int dk,
                         int dv, kdn_dtype_t dtype, int alpha_per_channel, float mu, float scale,
                         const LayerOpts& lo, hipStream_t stream)
{
    if (R == 0) return hipSuccess;
    if (dtype == KDN_F32)
        return launch_t<float>(dk, dv, variant, alpha_per_channel, q, k, v, alpha, omega, r, S,
                               P, slot_idx, o, R, num_slots, H, mu, scale, lo, stream);
    return launch_t<bf16>(dk, dv, variant, alpha_per_channel, q, k, v, alpha, omega, r, S, P,
                          slot_idx, o, R, num_slots, H, mu, scale, lo, stream);
}

}  // namespace kdn
