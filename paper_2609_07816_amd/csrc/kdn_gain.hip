// Gain scan of Diagonal / Isotropic KDN on gfx950: the variance recurrence as an associative
// scan of 2x2 Moebius matrices (arXiv 2609.07816, App. "Hardware-Efficient Chunkwise
// Algorithm", Sec. "Chunkwise Gain Computation").
//
// Each token acts on the homogeneous state z = [n; d] (p = n / d) through
//   M_t = [[a_t, w_t], [u_t a_t, 1 + u_t w_t]],
// with a = alpha^2, w = omega, u = mu k^2 / r for a diagonal channel, and a = mean_i alpha_i^2,
// w = omega, u = mu ||k||^2 / (dk r) for the isotropic head (eqs. diag-cov-scan,
// iso-kla-box-mobius). Three passes:
//   1. chunk summaries  M_bar_m = M_r ... M_l                      (eq. chunk-gain-summary)
//   2. exclusive carries z_in_m = M_bar_{m-1} ... M_bar_0 z_0, as a Kogge-Stone scan across
//      the chunks of a sequence (log depth; eq. chunk-gain-carry)
//   3. replay of every chunk from its carry, emitting p_hat and the gain before each token's
//      matrix is applied (eqs. chunk-gain-local-prefix, chunk-gain-emission).
// Every product is rescaled by an exact power of two, which leaves n / d unchanged.
// The diagonal chain gives every channel its own thread (channels are independent); the
// isotropic chain gives every token a lane and scans inside the wavefront.
#include "kdn_device.h"

namespace kdn {
namespace {

constexpr int CG = 64;  // gain-chunk length (tokens)

struct Mat2 {
    float a, b, c, d;  // [[a, b], [c, d]]
};

__device__ __forceinline__ Mat2 mul(const Mat2& x, const Mat2& y)  // x @ y
{
    Mat2 z;
    z.a = x.a * y.a + x.b * y.c;
    z.b = x.a * y.b + x.b * y.d;
    z.c = x.c * y.a + x.d * y.c;
    z.d = x.c * y.b + x.d * y.d;
    renorm4(z.a, z.b, z.c, z.d);
    return z;
}

__device__ __forceinline__ Mat2 token_mat(float a, float w, float u)
{
    Mat2 m = {a, w, u * a, fmaf(u, w, 1.f)};
    return m;
}

__device__ __forceinline__ Mat2 shfl_up_mat(const Mat2& x, int off)
{
    Mat2 y;
    y.a = __shfl_up(x.a, off, 64);
    y.b = __shfl_up(x.b, off, 64);
    y.c = __shfl_up(x.c, off, 64);
    y.d = __shfl_up(x.d, off, 64);
    return y;
}

// ------------------------------------------------------------------------------------------
// Diagonal chain
// ------------------------------------------------------------------------------------------

// Pass 1: one thread per channel composes the chunk's token matrices (later on the left).
template <class E, int DK>
__global__ __launch_bounds__(DK) void diag_summary_kernel(
    const E* __restrict__ k, const E* __restrict__ alpha, const E* __restrict__ omega,
    const E* __restrict__ r, ChunkMap cm, int H, float mu, float4* __restrict__ summ)
{
    const int g = blockIdx.x, h = blockIdx.y, c = threadIdx.x;
    int n, c0, c1;
    bool last;
    if (!locate_chunk<CG>(cm, g, n, c0, c1, last)) return;
    Mat2 acc = {1.f, 0.f, 0.f, 1.f};
    for (int t = c0; t < c1; ++t) {
        const size_t row = (size_t)t * H + h;
        const float al = ldf(alpha, row * DK + c), kk = ldf(k, row * DK + c);
        const float a = al * al, u = mu * kk * kk / ldf(r, row);
        acc = mul(token_mat(a, ldf(omega, row * DK + c), u), acc);
    }
    summ[((size_t)g * H + h) * DK + c] = make_float4(acc.a, acc.b, acc.c, acc.d);
}

// Pass 3: replay each chunk from its carry; p_hat_t = a_t n/d + w_t before M_t is applied;
// kappa_t = p_hat_t k_t / (r_t + sum_i p_hat_ti k_ti^2) (eq. chunk-gain-emission).
template <class E, int DK>
__global__ __launch_bounds__(DK) void diag_emit_kernel(
    const E* __restrict__ k, const E* __restrict__ alpha, const E* __restrict__ omega,
    const E* __restrict__ r, const float2* __restrict__ carry, ChunkMap cm, int H, float mu,
    float* __restrict__ kappa_out, float* __restrict__ phat_out, float* __restrict__ P_T)
{
    __shared__ float s_part[CG][DK + 1];
    __shared__ float s_rden[CG];
    const int g = blockIdx.x, h = blockIdx.y, c = threadIdx.x;
    int n, c0, c1;
    bool last;
    if (!locate_chunk<CG>(cm, g, n, c0, c1, last)) return;
    const float2 z = carry[((size_t)g * H + h) * DK + c];
    float zn = z.x, zd = z.y;
    float pk[CG];
    const int L = c1 - c0;
#pragma unroll
    for (int j = 0; j < CG; ++j) {
        if (j < L) {
            const size_t row = (size_t)(c0 + j) * H + h;
            const float al = ldf(alpha, row * DK + c), kk = ldf(k, row * DK + c);
            const float a = al * al, w = ldf(omega, row * DK + c);
            const float u = mu * kk * kk / ldf(r, row);
            const float n2 = fmaf(a, zn, w * zd);     // n_t
            const float ph = n2 / zd;                  // p_hat_t = a n_{t-1}/d_{t-1} + w
            zd = fmaf(u, n2, zd);                      // d_t = u a n + (1 + u w) d = u n_t + d
            zn = n2;
            renorm2(zn, zd);
            pk[j] = ph * kk;
            s_part[j][c] = ph * kk * kk;
            if (phat_out) phat_out[row * DK + c] = ph;
        }
    }
    if (last && P_T) P_T[((size_t)n * H + h) * DK + c] = zn / zd;
    __syncthreads();
    // den_t = r_t + sum_c p_hat k^2 : DK threads reduce CG rows
    for (int j = c; j < L; j += DK) {
        float s = 0.f;
        for (int i = 0; i < DK; ++i) s += s_part[j][i];
        s_rden[j] = 1.f / (ldf(r, (size_t)(c0 + j) * H + h) + s);
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < CG; ++j)
        if (j < L) kappa_out[((size_t)(c0 + j) * H + h) * DK + c] = pk[j] * s_rden[j];
}

// ------------------------------------------------------------------------------------------
// Isotropic chain: one lane per token of the chunk
// ------------------------------------------------------------------------------------------

// Token coefficients of the isotropic chain: a = mean_i alpha_i^2 (or alpha^2), w = omega,
// u = mu ||k||^2 / (dk r); also returns ||k||^2.
template <class E, int DK, bool APC>
__device__ __forceinline__ void iso_coeffs(const E* k, const E* alpha, const E* omega,
                                           const E* r, size_t row, float mu, float& a, float& w,
                                           float& u, float& nk)
{
    float sa = 0.f, sk = 0.f;
#pragma unroll 8
    for (int i = 0; i < DK; ++i) {
        const float kk = ldf(k, row * DK + i);
        sk += kk * kk;
        if (APC) {
            const float al = ldf(alpha, row * DK + i);
            sa += al * al;
        }
    }
    if (APC) {
        a = sa / (float)DK;
    } else {
        const float al = ldf(alpha, row);
        a = al * al;
    }
    w = ldf(omega, row);
    nk = sk;
    u = mu * sk / ((float)DK * ldf(r, row));
}

template <class E, int DK, bool APC>
__global__ __launch_bounds__(64) void iso_summary_kernel(
    const E* __restrict__ k, const E* __restrict__ alpha, const E* __restrict__ omega,
    const E* __restrict__ r, ChunkMap cm, int H, float mu, float4* __restrict__ summ)
{
    const int g = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
    int n, c0, c1;
    bool last;
    if (!locate_chunk<CG>(cm, g, n, c0, c1, last)) return;
    Mat2 x = {1.f, 0.f, 0.f, 1.f};
    if (c0 + lane < c1) {
        float a, w, u, nk;
        iso_coeffs<E, DK, APC>(k, alpha, omega, r, (size_t)(c0 + lane) * H + h, mu, a, w, u, nk);
        x = token_mat(a, w, u);
    }
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {  // tree product over the lanes, later on the left
        Mat2 y;
        y.a = __shfl_down(x.a, off, 64);
        y.b = __shfl_down(x.b, off, 64);
        y.c = __shfl_down(x.c, off, 64);
        y.d = __shfl_down(x.d, off, 64);
        if ((lane & (2 * off - 1)) == 0) x = mul(y, x);
    }
    if (lane == 0) summ[(size_t)g * H + h] = make_float4(x.a, x.b, x.c, x.d);
}

template <class E, int DK, bool APC>
__global__ __launch_bounds__(64) void iso_emit_kernel(
    const E* __restrict__ k, const E* __restrict__ alpha, const E* __restrict__ omega,
    const E* __restrict__ r, const float2* __restrict__ carry, ChunkMap cm, int H, float mu,
    float* __restrict__ beta_out, float* __restrict__ bhat_out, float* __restrict__ P_T)
{
    const int g = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
    int n, c0, c1;
    bool last;
    if (!locate_chunk<CG>(cm, g, n, c0, c1, last)) return;
    const bool valid = c0 + lane < c1;
    const size_t row = (size_t)(c0 + lane) * H + h;
    float a = 1.f, w = 0.f, u = 0.f, nk = 0.f;
    if (valid) iso_coeffs<E, DK, APC>(k, alpha, omega, r, row, mu, a, w, u, nk);
    Mat2 x = token_mat(a, w, u);
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {  // inclusive prefix within the chunk
        const Mat2 y = shfl_up_mat(x, off);
        if (lane >= off) x = mul(x, y);
    }
    const float2 z = carry[(size_t)g * H + h];
    float zn = x.a * z.x + x.b * z.y, zd = x.c * z.x + x.d * z.y;  // state after this token
    renorm2(zn, zd);
    float en = __shfl_up(zn, 1, 64), ed = __shfl_up(zd, 1, 64);    // state before it
    if (lane == 0) { en = z.x; ed = z.y; }
    if (valid) {
        const float bh = a * en / ed + w;
        beta_out[row] = bh / (ldf(r, row) + bh * nk);
        if (bhat_out) bhat_out[row] = bh;
        if (last && P_T && c0 + lane == c1 - 1) P_T[(size_t)n * H + h] = zn / zd;
    }
}

template <class E, int DK>
hipError_t launch_gain_t(int variant, const void* k, const void* alpha, const void* omega,
                         const void* r, const float* P0, float* gain_out, float* phat_out,
                         float* P_T, const SeqArgs& sa, int apc, float mu, char* ws,
                         hipStream_t st)
{
    const E *k_ = (const E*)k, *a_ = (const E*)alpha, *w_ = (const E*)omega, *r_ = (const E*)r;
    const int nchan = variant == 0 ? DK : 1;
    const int maxch = sa.cu_seqlens ? sa.B * sa.T / CG + sa.N : sa.N * ((sa.T + CG - 1) / CG);
    int32_t* choff = (int32_t*)ws;
    size_t off = ((size_t)(sa.N + 1) * sizeof(int32_t) + 255) & ~(size_t)255;
    float4* summ = (float4*)(ws + off);
    off += (size_t)maxch * sa.H * nchan * sizeof(float4);
    float2* carry = (float2*)(ws + off);
    if (maxch == 0) return hipSuccess;
    ChunkMap cm;
    cm.cu = sa.cu_seqlens;
    cm.choff = sa.cu_seqlens ? choff : nullptr;
    cm.N = sa.N;
    cm.T = sa.T;
    cm.ntok = sa.B * sa.T;
    cm.maxch = maxch;
    hipError_t e;
    if (sa.cu_seqlens &&
        (e = launch_chunk_table(sa.cu_seqlens, sa.N, cm.ntok, CG, maxch, choff, st)) != hipSuccess)
        return e;
    const dim3 grid(maxch, sa.H);
    if (variant == 0) {
        hipLaunchKernelGGL((diag_summary_kernel<E, DK>), grid, dim3(DK), 0, st, k_, a_, w_, r_,
                           cm, sa.H, mu, summ);
    } else if (apc) {
        hipLaunchKernelGGL((iso_summary_kernel<E, DK, true>), grid, dim3(64), 0, st, k_, a_, w_,
                           r_, cm, sa.H, mu, summ);
    } else {
        hipLaunchKernelGGL((iso_summary_kernel<E, DK, false>), grid, dim3(64), 0, st, k_, a_,
                           w_, r_, cm, sa.H, mu, summ);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_carry_scan(summ, P0, cm, CG, sa.H, nchan, carry, P_T, st)) != hipSuccess)
        return e;
    if (variant == 0) {
        hipLaunchKernelGGL((diag_emit_kernel<E, DK>), grid, dim3(DK), 0, st, k_, a_, w_, r_,
                           carry, cm, sa.H, mu, gain_out, phat_out, P_T);
    } else if (apc) {
        hipLaunchKernelGGL((iso_emit_kernel<E, DK, true>), grid, dim3(64), 0, st, k_, a_, w_,
                           r_, carry, cm, sa.H, mu, gain_out, phat_out, P_T);
    } else {
        hipLaunchKernelGGL((iso_emit_kernel<E, DK, false>), grid, dim3(64), 0, st, k_, a_, w_,
                           r_, carry, cm, sa.H, mu, gain_out, phat_out, P_T);
    }
    return hipGetLastError();
}

template <class E>
hipError_t launch_gain_dk(int dk, int variant, const void* k, const void* alpha,
                          const void* omega, const void* r, const float* P0, float* gain_out,
                          float* phat_out, float* P_T, const SeqArgs& sa, int apc, float mu,
                          char* ws, hipStream_t st)
{
    switch (dk) {
    case 16: return launch_gain_t<E, 16>(variant, k, alpha, omega, r, P0, gain_out, phat_out,
                                          P_T, sa, apc, mu, ws, st);
    case 32: return launch_gain_t<E, 32>(variant, k, alpha, omega, r, P0, gain_out, phat_out,
                                          P_T, sa, apc, mu, ws, st);
    case 64: return launch_gain_t<E, 64>(variant, k, alpha, omega, r, P0, gain_out, phat_out,
                                          P_T, sa, apc, mu, ws, st);
    case 128: return launch_gain_t<E, 128>(variant, k, alpha, omega, r, P0, gain_out,
                                            phat_out, P_T, sa, apc, mu, ws, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace

size_t gain_workspace_bytes(int variant, int N, int B, int T, int H, int dk)
{
    // chunks: fixed length has N * ceil(T / CG) <= B*T/CG + N; a packed batch (B = 1) has at
    // most T/CG + N because every sequence adds at most one partial chunk
    const size_t maxch = (size_t)B * T / CG + (size_t)N;
    const size_t nchan = variant == 0 ? (size_t)dk : 1;
    size_t off = (((size_t)N + 1) * sizeof(int32_t) + 255) & ~(size_t)255;
    off += maxch * H * nchan * sizeof(float4);
    off += maxch * H * nchan * sizeof(float2);
    return off;
}

hipError_t launch_gain(int variant, const void* k, const void* alpha, const void* omega,
                       const void* r, const float* P0, float* gain_out, float* phat_out,
                       float* P_T, const SeqArgs& sa, int dk, kdn_dtype_t dtype,
                       int alpha_per_channel, float mu, void* workspace, hipStream_t stream)
{
    if (dtype == KDN_F32)
        return launch_gain_dk<float>(dk, variant, k, alpha, omega, r, P0, gain_out, phat_out,
                                     P_T, sa, alpha_per_channel, mu, (char*)workspace, stream);
    return launch_gain_dk<bf16>(dk, variant, k, alpha, omega, r, P0, gain_out, phat_out, P_T, sa,
                                alpha_per_channel, mu, (char*)workspace, stream);
}

}  // namespace kdn
