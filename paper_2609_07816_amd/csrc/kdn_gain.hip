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
// Pass 1 is the forward's summary kernel and pass 2 the shared carry scan. Pass 3 gives every
// (chunk, head) one wavefront whose lanes hold the channels and read the chunk's rows eight
// tokens ahead: the diagonal chain replays each channel on its lane and sums the gain's
// normalisation across the wavefront; the isotropic chain sums ||k||^2 (and alpha^2) across the
// wavefront per token, hands token t's sums to lane t and scans the chunk inside the wavefront.
#include "kdn_device.h"
#include "kdn_fwd.h"

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

// One wavefront per (chunk, head): lane l holds the CPL adjacent channels from l * CPL
// (CPL = 2 for dk = 128, else 1; lanes past dk idle for dk < 64) and reads them with one load
// per array and token. The chunk's tokens are fetched G at a time into registers, the next
// group while the current one is computed; rows past the chunk's end are clamped to its last
// token, so every load is in bounds and unconditional.
template <class E, int N> struct Lanes;
template <> struct Lanes<float, 1> { typedef float T; };
template <> struct Lanes<float, 2> { typedef float T __attribute__((ext_vector_type(2))); };
template <> struct Lanes<bf16, 1> { typedef bf16 T; };
template <> struct Lanes<bf16, 2> { typedef bf16 T __attribute__((ext_vector_type(2))); };

__device__ __forceinline__ float lane_el(float v, int) { return v; }
__device__ __forceinline__ float lane_el(bf16 v, int) { return (float)v; }
template <class V> __device__ __forceinline__ float lane_el(const V& v, int i)
{
    return (float)v[i];
}

// Row access through a buffer descriptor of one wavefront-uniform row (built on the scalar
// unit per row): the lane's byte offset stays in one vector register and no per-row address
// arithmetic runs on the vector unit; rows are addressed with 64-bit pointers, so tensors of any
// size are reachable.
__device__ __forceinline__ rsrc_t row_rsrc(const void* p, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes,
                                             0x00020000);
}
template <int B> struct RowIO;
template <> struct RowIO<2> {
    template <class V> static __device__ __forceinline__ V load(rsrc_t r, uint32_t off)
    {
        const short x = (short)__builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0);
        return __builtin_bit_cast(V, x);
    }
};
template <> struct RowIO<4> {
    template <class V> static __device__ __forceinline__ V load(rsrc_t r, uint32_t off)
    {
        return __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0));
    }
    static __device__ __forceinline__ void store(float x, float, rsrc_t r, uint32_t off)
    {
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x), r, (int)off, 0, 0);
    }
};
template <> struct RowIO<8> {
    template <class V> static __device__ __forceinline__ V load(rsrc_t r, uint32_t off)
    {
        return __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0));
    }
    static __device__ __forceinline__ void store(float x, float y, rsrc_t r, uint32_t off)
    {
        typedef unsigned u2 __attribute__((ext_vector_type(2)));
        const u2 v = {__float_as_uint(x), __float_as_uint(y)};
        __builtin_amdgcn_raw_buffer_store_b64(v, r, (int)off, 0, 0);
    }
};

template <class E, int DK, int CPL_>
struct DiagLanes {
    static constexpr int CPL = CPL_;
    static constexpr int G = 8;  // tokens per prefetch group
    typedef typename Lanes<E, CPL>::T VT;
    struct Group {
        VT k[G], al[G], w[G];
        float r[G];
    };
    // loads tokens j0 .. j0 + G - 1 of the chunk starting at c0 (length L); every row pointer
    // is wavefront-uniform and the lane adds its byte offset lo
    static __device__ __forceinline__ void load(Group& b, const E* k, const E* alpha,
                                                const E* omega, const E* r, int c0, int L,
                                                int j0, int H, int h, uint32_t lo)
    {
#pragma unroll
        for (int jj = 0; jj < G; ++jj) {
            const size_t row = (size_t)(c0 + min(j0 + jj, L - 1)) * H + h;
            typedef RowIO<sizeof(VT)> IO;
            b.k[jj] = IO::template load<VT>(row_rsrc(k + row * DK, DK * sizeof(E)), lo);
            b.al[jj] = IO::template load<VT>(row_rsrc(alpha + row * DK, DK * sizeof(E)), lo);
            b.w[jj] = IO::template load<VT>(row_rsrc(omega + row * DK, DK * sizeof(E)), lo);
            b.r[jj] = ldf(r, row);
        }
    }
};

// Pass 3 (pass 1 is the forward's summary kernel): replay each chunk from its carry; p_hat_t = a_t n/d + w_t before M_t is applied;
// kappa_t = p_hat_t k_t / (r_t + sum_i p_hat_ti k_ti^2) (eq. chunk-gain-emission), the sum over
// the head's channels taken across the wavefront with DPP.
template <class E, int DK>
__global__ __launch_bounds__(64) void diag_emit_kernel(
    const E* __restrict__ k, const E* __restrict__ alpha, const E* __restrict__ omega,
    const E* __restrict__ r, const float2* __restrict__ carry, ChunkMap cm, int H, float mu,
    float* __restrict__ kappa_out, float* __restrict__ phat_out, float* __restrict__ P_T)
{
    typedef DiagLanes<E, DK, (DK >= 64 ? DK / 64 : 1)> DL;
    constexpr int CPL = DL::CPL, G = DL::G;
    const int g = (int)(blockIdx.x % (unsigned)cm.maxch);
    const int h = (int)(blockIdx.x / (unsigned)cm.maxch), lane = threadIdx.x;
    int n, c0, c1;
    bool last;
    if (!locate_chunk<CG>(cm, g, n, c0, c1, last)) return;
    const bool act = lane * CPL < DK;
    const int c = act ? lane * CPL : 0, L = c1 - c0;
    const uint32_t lo = c * sizeof(E), lo4 = c * 4;
    float zn[CPL], zd[CPL];
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
        const float2 z = carry[((size_t)g * H + h) * DK + c + i];
        zn[i] = z.x;
        zd[i] = z.y;
    }
    typename DL::Group ga, gb;
    auto step = [&](const typename DL::Group& b, int j0) __attribute__((always_inline)) {
#pragma unroll
        for (int jj = 0; jj < G; ++jj) {
            if (j0 + jj >= L) break;
            const size_t row = (size_t)(c0 + j0 + jj) * H + h;
            const float rr = b.r[jj], mur = mu * __builtin_amdgcn_rcpf(rr);
            float ph[CPL], pk[CPL], part = 0.f;
#pragma unroll
            for (int i = 0; i < CPL; ++i) {
                const float al = lane_el(b.al[jj], i), kk = lane_el(b.k[jj], i);
                const float n2 = fmaf(al * al, zn[i], lane_el(b.w[jj], i) * zd[i]);  // n_t
                ph[i] = n2 * __builtin_amdgcn_rcpf(zd[i]);          // a n_{t-1}/d_{t-1} + w
                zd[i] = fmaf(mur * kk * kk, n2, zd[i]);             // d_t = u n_t + d_{t-1}
                zn[i] = n2;
                rescale2(zn[i], zd[i]);
                pk[i] = ph[i] * kk;
                part = fmaf(pk[i], kk, part);
            }
            const float rden = __builtin_amdgcn_rcpf(rr + wave_sum(act ? part : 0.f));
            if (act) {
                typedef RowIO<4 * CPL> IO;
                IO::store(pk[0] * rden, pk[CPL - 1] * rden,
                          row_rsrc(kappa_out + row * DK, DK * 4), lo4);
                if (phat_out)
                    IO::store(ph[0], ph[CPL - 1], row_rsrc(phat_out + row * DK, DK * 4), lo4);
            }
        }
    };
    DL::load(ga, k, alpha, omega, r, c0, L, 0, H, h, lo);
    for (int j0 = 0; j0 < L; j0 += 2 * G) {
        if (j0 + G < L) DL::load(gb, k, alpha, omega, r, c0, L, j0 + G, H, h, lo);
        step(ga, j0);
        if (j0 + G >= L) break;
        if (j0 + 2 * G < L) DL::load(ga, k, alpha, omega, r, c0, L, j0 + 2 * G, H, h, lo);
        step(gb, j0 + G);
    }
    if (last && P_T && act) {
#pragma unroll
        for (int i = 0; i < CPL; ++i) P_T[((size_t)n * H + h) * DK + c + i] = zn[i] / zd[i];
    }
}

// ------------------------------------------------------------------------------------------
// Isotropic chain: one lane per token of the chunk
// ------------------------------------------------------------------------------------------

// ||k_t||^2 and sum_i alpha_ti^2 (per-channel gates) of the chunk's tokens, token t's sums
// returned to lane t: the wavefront reads each row once with its lanes over the channels (CPL
// adjacent channels per lane, as in the diagonal emission), G rows ahead, and sums across the
// lanes by DPP. All 64 lanes must be active.
template <class E, int DK, bool APC>
__device__ __forceinline__ void iso_row_sums(const E* k, const E* alpha, int c0, int L, int H,
                                             int h, int lane, float& nk, float& sa)
{
    constexpr int CPL = DK >= 64 ? DK / 64 : 1, G = 8;
    typedef typename Lanes<E, CPL>::T VT;
    typedef RowIO<sizeof(VT)> IO;
    const bool act = lane * CPL < DK;
    const uint32_t lo = (act ? lane * CPL : 0) * sizeof(E);
    struct Buf {
        VT k[G], a[APC ? G : 1];
    };
    auto load = [&](Buf& b, int j0) __attribute__((always_inline)) {
#pragma unroll
        for (int jj = 0; jj < G; ++jj) {
            const size_t row = (size_t)(c0 + min(j0 + jj, L - 1)) * H + h;
            b.k[jj] = IO::template load<VT>(row_rsrc(k + row * DK, DK * sizeof(E)), lo);
            if constexpr (APC)
                b.a[jj] = IO::template load<VT>(row_rsrc(alpha + row * DK, DK * sizeof(E)), lo);
        }
    };
    auto sums = [&](const Buf& b, int j0) __attribute__((always_inline)) {
#pragma unroll
        for (int jj = 0; jj < G; ++jj) {
            if (j0 + jj >= L) break;
            float s = 0.f, t = 0.f;
#pragma unroll
            for (int i = 0; i < CPL; ++i) {
                const float kk = lane_el(b.k[jj], i);
                s = fmaf(kk, kk, s);
                if constexpr (APC) {
                    const float al = lane_el(b.a[jj], i);
                    t = fmaf(al, al, t);
                }
            }
            s = wave_sum(act ? s : 0.f);
            if (lane == j0 + jj) nk = s;
            if constexpr (APC) {
                t = wave_sum(act ? t : 0.f);
                if (lane == j0 + jj) sa = t;
            }
        }
    };
    nk = 0.f;
    sa = 0.f;
    Buf ba, bb;
    load(ba, 0);
    for (int j0 = 0; j0 < L; j0 += 2 * G) {
        if (j0 + G < L) load(bb, j0 + G);
        sums(ba, j0);
        if (j0 + G >= L) break;
        if (j0 + 2 * G < L) load(ba, j0 + 2 * G);
        sums(bb, j0 + G);
    }
}

// Pass 3 of the isotropic chain (pass 1 is the forward's summary kernel): lane t holds token t
// of the chunk; its coefficients a = mean_i alpha_i^2 (or alpha^2), w = omega,
// u = mu ||k||^2 / (dk r) (eq. iso-kla-box-mobius), the inclusive prefix of the token matrices
// across the lanes, the state before the token from the carry, and
// beta_t = b_hat_t / (r_t + b_hat_t ||k_t||^2) (eq. chunk-gain-emission).
template <class E, int DK, bool APC>
__global__ __launch_bounds__(64) void iso_emit_kernel(
    const E* __restrict__ k, const E* __restrict__ alpha, const E* __restrict__ omega,
    const E* __restrict__ r, const float2* __restrict__ carry, ChunkMap cm, int H, float mu,
    float* __restrict__ beta_out, float* __restrict__ bhat_out, float* __restrict__ P_T)
{
    const int g = (int)(blockIdx.x % (unsigned)cm.maxch);
    const int h = (int)(blockIdx.x / (unsigned)cm.maxch), lane = threadIdx.x;
    int n, c0, c1;
    bool last;
    if (!locate_chunk<CG>(cm, g, n, c0, c1, last)) return;
    const bool valid = c0 + lane < c1;
    const size_t row = (size_t)(c0 + lane) * H + h;
    float nks, sas;
    iso_row_sums<E, DK, APC>(k, alpha, c0, c1 - c0, H, h, lane, nks, sas);
    float a = 1.f, w = 0.f, u = 0.f, nk = 0.f;
    if (valid) {
        if (APC) {
            a = sas / (float)DK;
        } else {
            const float al = ldf(alpha, row);
            a = al * al;
        }
        w = ldf(omega, row);
        nk = nks;
        u = mu * nks / ((float)DK * ldf(r, row));
    }
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
    // one workgroup per (chunk, head), h * maxch + g in a 1-D grid (chunks of a head adjacent)
    const dim3 grid((unsigned)((size_t)maxch * sa.H));
    // pass 1: the forward's summary kernel, four waves per (chunk, head), each with its 16
    // tokens' loads in flight at once, the four block products composed in LDS
    fwd::InArgs in = {};
    in.q = k; in.k = k; in.alpha = alpha; in.omega = omega; in.r = r;
    const size_t ntok = (size_t)sa.B * sa.T * sa.H;
    in.bytes_k = (uint32_t)(ntok * DK * sizeof(E));
    in.bytes_h = (uint32_t)(ntok * sizeof(E));
    in.H = sa.H;
    in.mu = mu;
    const dim3 cgrid((unsigned)((size_t)maxch * sa.H));
    if (variant == 0)
        hipLaunchKernelGGL((fwd::summary_kernel<E, fwd::VarCfg<E, DK, 0, true>>), cgrid,
                           dim3(fwd::NTH), 0, st, in, cm, summ);
    else if (apc)
        hipLaunchKernelGGL((fwd::summary_kernel<E, fwd::VarCfg<E, DK, 1, true>>), cgrid,
                           dim3(fwd::NTH), 0, st, in, cm, summ);
    else
        hipLaunchKernelGGL((fwd::summary_kernel<E, fwd::VarCfg<E, DK, 1, false>>), cgrid,
                           dim3(fwd::NTH), 0, st, in, cm, summ);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_carry_scan(summ, P0, cm, CG, sa.H, nchan, carry, P_T, st)) != hipSuccess)
        return e;
    if (variant == 0) {
        hipLaunchKernelGGL((diag_emit_kernel<E, DK>), grid, dim3(64), 0, st, k_, a_, w_, r_,
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
