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
#include "kdn_internal.h"

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

// Token range [t0, t1) (flat token index over B*T) of sequence n.
__device__ __forceinline__ void seq_bounds(const int32_t* cu, int n, int T, int& t0, int& t1)
{
    if (cu) {
        t0 = cu[n];
        t1 = cu[n + 1];
        if (t1 < t0) t1 = t0;
    } else {
        t0 = n * T;
        t1 = t0 + T;
    }
}

// Locate global chunk g: sequence n, chunk start token t (flat), chunk end, last-of-sequence.
// Chunk offsets: fixed length -> n * ceil(T / CG); packed -> the table built on the device.
__device__ __forceinline__ bool locate_chunk(const int32_t* cu, const int32_t* choff, int N,
                                             int T, int g, int& n, int& c0, int& c1,
                                             int& mloc, bool& last, int cg = CG)
{
    if (!cu) {
        const int ncs = (T + cg - 1) / cg;
        n = g / ncs;
        if (n >= N) return false;
        mloc = g - n * ncs;
    } else {
        if (g >= choff[N]) return false;
        int lo = 0, hi = N - 1;  // largest n with choff[n] <= g
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (choff[mid] <= g) lo = mid; else hi = mid - 1;
        }
        n = lo;
        mloc = g - choff[n];
    }
    int t0, t1;
    seq_bounds(cu, n, T, t0, t1);
    c0 = t0 + mloc * cg;
    c1 = min(c0 + cg, t1);
    last = (c1 == t1);
    return c0 < c1;
}

// Chunk-offset table for packed batches: choff[n] = sum_{m < n} ceil(len_m / cg).
__global__ void chunk_table_kernel(const int32_t* __restrict__ cu, int N, int cg,
                                   int32_t* __restrict__ choff)
{
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    int acc = 0;
    for (int n = 0; n < N; ++n) {
        choff[n] = acc;
        int len = cu[n + 1] - cu[n];
        if (len < 0) len = 0;
        acc += (len + cg - 1) / cg;
    }
    choff[N] = acc;
}

// ------------------------------------------------------------------------------------------
// Diagonal chain
// ------------------------------------------------------------------------------------------

// Pass 1: one thread per channel composes the chunk's token matrices (later on the left).
template <class E, int DK>
__global__ __launch_bounds__(DK) void diag_summary_kernel(
    const E* __restrict__ k, const E* __restrict__ alpha, const E* __restrict__ omega,
    const E* __restrict__ r, const int32_t* __restrict__ cu, const int32_t* __restrict__ choff,
    int N, int T, int H, float mu, float4* __restrict__ summ)
{
    const int g = blockIdx.x, h = blockIdx.y, c = threadIdx.x;
    int n, c0, c1, m;
    bool last;
    if (!locate_chunk(cu, choff, N, T, g, n, c0, c1, m, last)) return;
    Mat2 acc = {1.f, 0.f, 0.f, 1.f};
    for (int t = c0; t < c1; ++t) {
        const size_t row = (size_t)t * H + h;
        const float al = ldf(alpha, row * DK + c), kk = ldf(k, row * DK + c);
        const float a = al * al, u = mu * kk * kk / ldf(r, row);
        acc = mul(token_mat(a, ldf(omega, row * DK + c), u), acc);
    }
    summ[((size_t)g * H + h) * DK + c] = make_float4(acc.a, acc.b, acc.c, acc.d);
}

// Pass 2: per (sequence, head, channel) exclusive scan of the summaries over chunks of cg
// tokens. Grid (sequence x head, channel groups of 4); one wavefront per channel, lanes are
// chunks, blocks of 64 chunks carry into the next.
__global__ __launch_bounds__(256) void carry_scan_kernel(
    const float4* __restrict__ summ, const float* __restrict__ P0,
    const int32_t* __restrict__ cu, const int32_t* __restrict__ choff, int N, int T, int H,
    int nchan, int cg, float2* __restrict__ carry, float* __restrict__ P_T)
{
    const int n = blockIdx.x / H, h = blockIdx.x % H;
    if (n >= N) return;
    int t0, t1;
    seq_bounds(cu, n, T, t0, t1);
    const int nch = (t1 - t0 + cg - 1) / cg;
    const int g0 = cu ? choff[n] : n * ((T + cg - 1) / cg);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int c = 4 * blockIdx.y + w;  // one channel per wavefront
    if (c >= nchan) return;
    if (nch == 0) {  // an empty sequence keeps its initial variances
        if (P_T && lane == 0) {
            const size_t pidx = ((size_t)n * H + h) * nchan + c;
            P_T[pidx] = P0 ? P0[pidx] : 1.f;
        }
        return;
    }
    {
        const size_t pidx = ((size_t)n * H + h) * nchan + c;
        float cn = P0 ? P0[pidx] : 1.f, cd = 1.f;  // z_0 = [p_0; 1]
        for (int b0 = 0; b0 < nch; b0 += 64) {
            const int m = b0 + lane;
            Mat2 x = {1.f, 0.f, 0.f, 1.f};
            if (m < nch) {
                const float4 s = summ[((size_t)(g0 + m) * H + h) * nchan + c];
                x = {s.x, s.y, s.z, s.w};
            }
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {  // inclusive Kogge-Stone, later on the left
                const Mat2 y = shfl_up_mat(x, off);
                if (lane >= off) x = mul(x, y);
            }
            float zn = x.a * cn + x.b * cd, zd = x.c * cn + x.d * cd;  // state after chunk m
            renorm2(zn, zd);
            float en = __shfl_up(zn, 1, 64), ed = __shfl_up(zd, 1, 64);
            if (lane == 0) { en = cn; ed = cd; }
            if (m < nch) carry[((size_t)(g0 + m) * H + h) * nchan + c] = make_float2(en, ed);
            const int lastl = min(63, nch - 1 - b0);
            cn = __shfl(zn, lastl, 64);
            cd = __shfl(zd, lastl, 64);
        }
    }
}

// Pass 3: replay each chunk from its carry; p_hat_t = a_t n/d + w_t before M_t is applied;
// kappa_t = p_hat_t k_t / (r_t + sum_i p_hat_ti k_ti^2) (eq. chunk-gain-emission).
template <class E, int DK>
__global__ __launch_bounds__(DK) void diag_emit_kernel(
    const E* __restrict__ k, const E* __restrict__ alpha, const E* __restrict__ omega,
    const E* __restrict__ r, const float2* __restrict__ carry, const int32_t* __restrict__ cu,
    const int32_t* __restrict__ choff, int N, int T, int H, float mu,
    float* __restrict__ kappa_out, float* __restrict__ phat_out, float* __restrict__ P_T)
{
    __shared__ float s_part[CG][DK + 1];
    __shared__ float s_rden[CG];
    const int g = blockIdx.x, h = blockIdx.y, c = threadIdx.x;
    int n, c0, c1, m;
    bool last;
    if (!locate_chunk(cu, choff, N, T, g, n, c0, c1, m, last)) return;
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
    const E* __restrict__ r, const int32_t* __restrict__ cu, const int32_t* __restrict__ choff,
    int N, int T, int H, float mu, float4* __restrict__ summ)
{
    const int g = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
    int n, c0, c1, m;
    bool last;
    if (!locate_chunk(cu, choff, N, T, g, n, c0, c1, m, last)) return;
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
    const E* __restrict__ r, const float2* __restrict__ carry, const int32_t* __restrict__ cu,
    const int32_t* __restrict__ choff, int N, int T, int H, float mu,
    float* __restrict__ beta_out, float* __restrict__ bhat_out, float* __restrict__ P_T)
{
    const int g = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
    int n, c0, c1, m;
    bool last;
    if (!locate_chunk(cu, choff, N, T, g, n, c0, c1, m, last)) return;
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
    if (sa.cu_seqlens)
        hipLaunchKernelGGL(chunk_table_kernel, dim3(1), dim3(1), 0, st, sa.cu_seqlens, sa.N,
                           CG, choff);
    const dim3 grid(maxch, sa.H);
    if (variant == 0) {
        hipLaunchKernelGGL((diag_summary_kernel<E, DK>), grid, dim3(DK), 0, st, k_, a_, w_, r_,
                           sa.cu_seqlens, choff, sa.N, sa.T, sa.H, mu, summ);
    } else if (apc) {
        hipLaunchKernelGGL((iso_summary_kernel<E, DK, true>), grid, dim3(64), 0, st, k_, a_, w_,
                           r_, sa.cu_seqlens, choff, sa.N, sa.T, sa.H, mu, summ);
    } else {
        hipLaunchKernelGGL((iso_summary_kernel<E, DK, false>), grid, dim3(64), 0, st, k_, a_,
                           w_, r_, sa.cu_seqlens, choff, sa.N, sa.T, sa.H, mu, summ);
    }
    hipLaunchKernelGGL(carry_scan_kernel, dim3(sa.N * sa.H, (nchan + 3) / 4), dim3(256), 0, st,
                       summ, P0, sa.cu_seqlens, choff, sa.N, sa.T, sa.H, nchan, CG, carry, P_T);
    if (variant == 0) {
        hipLaunchKernelGGL((diag_emit_kernel<E, DK>), grid, dim3(DK), 0, st, k_, a_, w_, r_,
                           carry, sa.cu_seqlens, choff, sa.N, sa.T, sa.H, mu, gain_out,
                           phat_out, P_T);
    } else if (apc) {
        hipLaunchKernelGGL((iso_emit_kernel<E, DK, true>), grid, dim3(64), 0, st, k_, a_, w_,
                           r_, carry, sa.cu_seqlens, choff, sa.N, sa.T, sa.H, mu, gain_out,
                           phat_out, P_T);
    } else {
        hipLaunchKernelGGL((iso_emit_kernel<E, DK, false>), grid, dim3(64), 0, st, k_, a_, w_,
                           r_, carry, sa.cu_seqlens, choff, sa.N, sa.T, sa.H, mu, gain_out,
                           phat_out, P_T);
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
