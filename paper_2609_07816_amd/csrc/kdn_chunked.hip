// Chunked forward of Diagonal / Isotropic KDN on gfx950: four launches.
//
// arXiv 2609.07816, App. "Hardware-Efficient Chunkwise Algorithm". Tokens are cut into chunks
// of C (chunks restart at every sequence start). With chunk-local index r and cumulative decay
// gamma_r = prod_{j<=r} alpha_j (per channel), Sec. "Chunkwise Memory Scan" writes one chunk as
//   K_bar = Gamma (.) K,  Q_bar = scale Gamma (.) Q,  P_bar_r = p_hat_r (.) k_r / gamma_r
//   den_r = r_r + sum_i p_hat_ri k_ri^2  (= K_bar_r . P_bar_r: gamma cancels)
//   T = tril(K_bar P_bar^T diag(1/den), -1),  A = (I + T)^-1
//   W = A K_bar,  U = A V,  A_qk = tril(Q_bar P_bar^T diag(1/den))
//   K_tail_r = (gamma_C / gamma_r) (.) kappa_r = gamma_C (.) P_bar_r / den_r
// and then only S crosses chunk boundaries:
//   R = U - W S_in,  O = Q_bar S_in + A_qk R,  S_out = diag(gamma_C) S_in + K_tail^T R.
// For the isotropic variant P_bar_r = beta_r k_r / gamma_r and den = 1.
//
// Launches:
//   1. summaries: per (chunk, head) the product of the chunk's 2x2 Moebius token matrices
//      (eq. chunk-gain-summary), per channel for the diagonal variant, and the products of its
//      16-token segments;
//   2. carries: exclusive log-depth scan of the summaries over the chunks of each sequence
//      (eq. chunk-gain-carry; kdn_gain.hip), which also yields P_T;
//   3. prep: per (chunk, head), all chunks in parallel: replay the variance chain from the
//      carry (eqs. chunk-gain-local-prefix, chunk-gain-emission), form the operands, solve
//      the unit-lower triangular system and write W, Q_bar, K_tail^T, A_qk, U, gamma_C;
//   4. state: per (sequence, head, dv tile) the serial walk over chunks, S in registers and
//      LDS (Sec. "Chunkwise Memory Scan", inter-chunk recurrence).
// Dense products run on MFMA (bf16 operands with fp32 accumulation for bf16 inputs, fp32
// MFMA for fp32 inputs); S, the variance chain and the triangular solve stay in fp32.
#include <algorithm>
#include <mutex>

#include "kdn_device.h"

namespace kdn {
namespace {

constexpr int NT = 256;  // threads per workgroup (4 waves)

constexpr size_t al16(size_t x) { return (x + 15) & ~(size_t)15; }
constexpr size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

template <class TI> struct OpOf { using type = bf16; };
template <> struct OpOf<float> { using type = float; };

// ------------------------------------------------------------------------------------------
// Per (chunk, head) record written by the prep kernel and read by the state kernel, in
// operand precision MT (bf16 for bf16 inputs, fp32 for fp32 inputs):
//   W [C][DK], Q_bar [C][DK] (scale folded in), K_tail^T [DK][C], A_qk [C][C] (upper part 0),
//   U packed as MFMA result tiles [DV/16][C/16][64 lanes][4], then gamma_C [DK] float32.
// ------------------------------------------------------------------------------------------
template <class MT, int DK, int DV, int C>
struct Rec {
    static constexpr size_t W = 0;
    static constexpr size_t Q = (size_t)C * DK;
    static constexpr size_t KT = 2 * (size_t)C * DK;
    static constexpr size_t AQ = 3 * (size_t)C * DK;
    static constexpr size_t U = AQ + (size_t)C * C;
    static constexpr size_t NMT = U + (size_t)C * DV;
    static constexpr size_t GC_BYTES = al16(NMT * sizeof(MT));
    static constexpr size_t BYTES = al256(GC_BYTES + (size_t)DK * 4);
};

// Chunk g of the flat chunk list: sequence n, first token c0 (flat over B*T), length L, and
// whether it is the sequence's last. Fixed length: sequence n owns chunks [n*ncs, (n+1)*ncs);
// packed: choff[n] from the device chunk table.
__device__ __forceinline__ bool chunk_at(const int32_t* cu, const int32_t* choff, int N, int T,
                                         int C, int g, int& n, int& c0, int& L, bool* last = nullptr)
{
    int m;
    if (!cu) {
        const int ncs = (T + C - 1) / C;
        n = g / ncs;
        if (n >= N) return false;
        m = g - n * ncs;
    } else {
        if (g >= choff[N]) return false;
        int lo = 0, hi = N - 1;  // largest n with choff[n] <= g
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (choff[mid] <= g) lo = mid; else hi = mid - 1;
        }
        n = lo;
        m = g - choff[n];
    }
    int t0, t1;
    seq_range(cu, n, T, t0, t1);
    c0 = t0 + m * C;
    L = min(C, t1 - c0);
    if (last) *last = c0 + L == t1;
    return L > 0;
}

// The chunks of every sequence are cut into nseg consecutive parts (segments) of near-equal
// count: segment k of a sequence with nch chunks holds its chunks [k nch / nseg, (k+1) nch / nseg).
// The state pass of segment k only needs the prep records of segment k, so it can run while
// the prep pass works on segment k + 1.
__device__ __forceinline__ void seg_range(int nch, int seg, int nseg, int& lo, int& hi)
{
    lo = (int)((long long)seg * nch / nseg);
    hi = (int)((long long)(seg + 1) * nch / nseg);
}

// segoff[k * (N + 1) + n] = number of chunks of segment k in the sequences before n (packed
// batches; fixed-length batches compute it directly).
__global__ void seg_table_kernel(const int32_t* __restrict__ cu, int N, int C, int nseg,
                                 int32_t* __restrict__ segoff)
{
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    for (int k = 0; k < nseg; ++k) {
        int acc = 0;
        for (int n = 0; n < N; ++n) {
            segoff[k * (N + 1) + n] = acc;
            int len = cu[n + 1] - cu[n];
            if (len < 0) len = 0;
            int lo, hi;
            seg_range((len + C - 1) / C, k, nseg, lo, hi);
            acc += hi - lo;
        }
        segoff[k * (N + 1) + N] = acc;
    }
}

// ------------------------------------------------------------------------------------------
// MFMA fragments read straight from memory: a lane (g, i) holds KF/4 consecutive k values of
// row i (A side) or column i (B side); one fragment feeds one bf16 MFMA (KF = 32 or 16) or four
// fp32 MFMAs (KF = 16). Both sides use the same k assignment, so the contraction is exact.
// ------------------------------------------------------------------------------------------
template <class MT, int K> struct Frag;

template <int K> struct Frag<bf16, K> {
    static constexpr int KF = (K % 32 == 0) ? 32 : 16;
    static constexpr int NS = K / KF;
    using V = typename std::conditional<KF == 32, uint4, uint2>::type;
    __device__ static V ld(const bf16* p) { return *reinterpret_cast<const V*>(p); }
    __device__ static floatx4 mma(floatx4 acc, V a, V b)
    {
        if constexpr (KF == 32)
            return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                           __builtin_bit_cast(bf16x8, b), acc, 0,
                                                           0, 0);
        else
            return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(bf16x4, a),
                                                              __builtin_bit_cast(bf16x4, b), acc,
                                                              0, 0, 0);
    }
};

template <int K> struct Frag<float, K> {
    static constexpr int KF = 16;
    static constexpr int NS = K / KF;
    using V = uint4;
    __device__ static V ld(const float* p) { return *reinterpret_cast<const V*>(p); }
    __device__ static floatx4 mma(floatx4 acc, V a, V b)
    {
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x),
                                                    acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y),
                                                    acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z),
                                                    acc, 0, 0, 0);
        return __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w),
                                                     acc, 0, 0, 0);
    }
};

// Four result values of one lane (rows 4g..4g+3 of a tile column) as one vector in MT.
template <class MT>
__device__ __forceinline__ void store4(MT* dst, float x0, float x1, float x2, float x3)
{
    if constexpr (std::is_same<MT, float>::value) {
        *reinterpret_cast<float4*>(dst) = make_float4(x0, x1, x2, x3);
    } else {
        bf16x4 v;
        v[0] = (bf16)x0; v[1] = (bf16)x1; v[2] = (bf16)x2; v[3] = (bf16)x3;
        *reinterpret_cast<bf16x4*>(dst) = v;
    }
}

// 16-byte copy of a [rows][cols] tile from LDS (row stride lds) to contiguous global memory.
template <class MT>
__device__ __forceinline__ void copy_out(MT* dst, const MT* src, int rows, int cols, int lds,
                                         int tid)
{
    constexpr int VE = 16 / (int)sizeof(MT);
    const int vpr = cols / VE;
    for (int idx = tid; idx < rows * vpr; idx += NT) {
        const int r = idx / vpr, e = (idx % vpr) * VE;
        *reinterpret_cast<uint4*>(dst + (size_t)r * cols + e) =
            *reinterpret_cast<const uint4*>(src + r * lds + e);
    }
}

// ------------------------------------------------------------------------------------------
// 1. chunk summaries
// ------------------------------------------------------------------------------------------
__device__ __forceinline__ void mat_mul_left(float* m, const float4& x)  // m <- x @ m
{
    const float a = x.x * m[0] + x.y * m[2], b = x.x * m[1] + x.y * m[3];
    const float c = x.z * m[0] + x.w * m[2], d = x.z * m[1] + x.w * m[3];
    m[0] = a; m[1] = b; m[2] = c; m[3] = d;
    renorm4(m[0], m[1], m[2], m[3]);
}

// Two adjacent inputs from one raw word (bf16 pair) or a float pair.
__device__ __forceinline__ float2 unpack2(unsigned u)
{
    return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xFFFF0000u));
}
__device__ __forceinline__ float2 unpack2(float2 v) { return v; }

// Diagonal: wave s composes the token matrices of segment s (tokens [16 s, 16 s + 16)) for the
// channel pair (2 l, 2 l + 1) of lane l (later tokens on the left), with the segment's decay
// product; wave 0 then composes the segments into the chunk summary.
template <class TI, int DK, int C>
__global__ __launch_bounds__(NT) void summary_diag_kernel(
    const TI* __restrict__ k, const TI* __restrict__ alpha, const TI* __restrict__ omega,
    const TI* __restrict__ r, const int32_t* __restrict__ cu, const int32_t* __restrict__ choff,
    int N, int T, int H, float mu, float4* __restrict__ chunksum, float4* __restrict__ segsum,
    float* __restrict__ seggam)
{
    constexpr int NSEG = C / 16, NP = DK / 2;
    __shared__ float4 s_m[NSEG][DK];
    const int g = blockIdx.x, h = blockIdx.y;
    int n, c0, L;
    if (!chunk_at(cu, choff, N, T, C, g, n, c0, L)) return;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int ch = 2 * lane;
    if (wave < NSEG && lane < NP) {
        float m0[4] = {1.f, 0.f, 0.f, 1.f}, m1[4] = {1.f, 0.f, 0.f, 1.f};
        float g0 = 1.f, g1 = 1.f;
        // every load is issued up front from a valid row (tokens past the end re-read the last
        // one) and its value replaced afterwards: loads under a branch would be waited for one
        // token at a time
        // (raw words: a conversion next to its load would make it wait for the load)
        using P2 = typename std::conditional<sizeof(TI) == 2, unsigned, float2>::type;
        P2 al[16], kk[16], ww[16];
        TI rr[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const size_t row = (size_t)(c0 + min(16 * wave + j, L - 1)) * H + h;
            al[j] = *reinterpret_cast<const P2*>(alpha + row * DK + ch);
            kk[j] = *reinterpret_cast<const P2*>(k + row * DK + ch);
            ww[j] = *reinterpret_cast<const P2*>(omega + row * DK + ch);
            rr[j] = r[row];
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            if (16 * wave + j < L) {  // past the end: identity matrix, no decay
                const float2 alv = unpack2(al[j]), kv = unpack2(kk[j]), wv = unpack2(ww[j]);
                const float mr = mu / to_f32(rr[j]);
                g0 *= alv.x;
                g1 *= alv.y;
                mob_left(m0, alv.x * alv.x, wv.x, kv.x * kv.x * mr);
                mob_left(m1, alv.y * alv.y, wv.y, kv.y * kv.y * mr);
                if (j & 1) {
                    renorm4(m0[0], m0[1], m0[2], m0[3]);
                    renorm4(m1[0], m1[1], m1[2], m1[3]);
                }
            }
        }
        renorm4(m0[0], m0[1], m0[2], m0[3]);
        renorm4(m1[0], m1[1], m1[2], m1[3]);
        const float4 M0 = make_float4(m0[0], m0[1], m0[2], m0[3]);
        const float4 M1 = make_float4(m1[0], m1[1], m1[2], m1[3]);
        s_m[wave][ch] = M0;
        s_m[wave][ch + 1] = M1;
        if (wave < NSEG - 1) {
            const size_t base = (((size_t)g * H + h) * (NSEG - 1) + wave) * DK + ch;
            segsum[base] = M0;
            segsum[base + 1] = M1;
            *reinterpret_cast<float2*>(seggam + base) = make_float2(g0, g1);
        }
    }
    __syncthreads();
    if (threadIdx.x < DK) {
        const int c = threadIdx.x;
        float m[4] = {1.f, 0.f, 0.f, 1.f};
#pragma unroll
        for (int s = 0; s < NSEG; ++s) mat_mul_left(m, s_m[s][c]);
        chunksum[((size_t)g * H + h) * DK + c] = make_float4(m[0], m[1], m[2], m[3]);
    }
}

// Sum of squares of n consecutive values (vector loads when the span is 16-byte aligned).
template <class TI, int NE>
__device__ __forceinline__ float sumsq(const TI* p)
{
    float s = 0.f;
    if constexpr ((NE * sizeof(TI)) % 16 == 0) {
        constexpr int VE = 16 / (int)sizeof(TI);
#pragma unroll
        for (int v = 0; v < NE / VE; ++v) {
            const uint4 u = reinterpret_cast<const uint4*>(p)[v];
            if constexpr (sizeof(TI) == 2) {
                const unsigned w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float lo = __uint_as_float(w[e] << 16), hi = __uint_as_float(w[e] & 0xFFFF0000u);
                    s = fmaf(lo, lo, s);
                    s = fmaf(hi, hi, s);
                }
            } else {
                const float w[4] = {__uint_as_float(u.x), __uint_as_float(u.y),
                                    __uint_as_float(u.z), __uint_as_float(u.w)};
#pragma unroll
                for (int e = 0; e < 4; ++e) s = fmaf(w[e], w[e], s);
            }
        }
    } else {
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            const float x = to_f32(p[e]);
            s = fmaf(x, x, s);
        }
    }
    return s;
}

// Isotropic: per token a = mean_i alpha_i^2 (or alpha^2), w = omega, u = mu ||k||^2 / (dk r);
// thread (token, quarter) reduces a quarter of the channels, one wave composes the tokens.
template <class TI, int DK, int C, bool APC>
__device__ __forceinline__ void iso_token_coeffs(const TI* k, const TI* alpha, const TI* omega,
                                                 const TI* r, int c0, int L, int H, int h,
                                                 float mu, float* s_a, float* s_w, float* s_u,
                                                 float* s_nk, int tid)
{
    constexpr int QW = DK / 4;
    const int t = tid >> 2, qq = tid & 3;
    const size_t row = (size_t)(c0 + min(t, L - 1)) * H + h;  // valid row; masked below
    float sk = sumsq<TI, QW>(k + row * DK + qq * QW);
    float sa = APC ? sumsq<TI, QW>(alpha + row * DK + qq * QW) : 0.f;
    sk += __shfl_xor(sk, 1, 64);
    sk += __shfl_xor(sk, 2, 64);
    if (APC) {
        sa += __shfl_xor(sa, 1, 64);
        sa += __shfl_xor(sa, 2, 64);
    }
    if (t < C && qq == 0) {
        const float al = APC ? 0.f : to_f32(alpha[row]);
        const float wv = to_f32(omega[row]), rv = to_f32(r[row]);
        float a = 1.f, w = 0.f, u = 0.f;
        if (t < L) {
            a = APC ? sa / (float)DK : al * al;
            w = wv;
            u = mu * sk / ((float)DK * rv);
        } else {
            sk = 0.f;
        }
        s_a[t] = a;
        s_w[t] = w;
        s_u[t] = u;
        if (s_nk) s_nk[t] = sk;
    }
}

template <class TI, int DK, int C, bool APC>
__global__ __launch_bounds__(NT) void summary_iso_kernel(
    const TI* __restrict__ k, const TI* __restrict__ alpha, const TI* __restrict__ omega,
    const TI* __restrict__ r, const int32_t* __restrict__ cu, const int32_t* __restrict__ choff,
    int N, int T, int H, float mu, float4* __restrict__ chunksum)
{
    __shared__ float s_a[C], s_w[C], s_u[C];
    const int g = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
    int n, c0, L;
    if (!chunk_at(cu, choff, N, T, C, g, n, c0, L)) return;
    iso_token_coeffs<TI, DK, C, APC>(k, alpha, omega, r, c0, L, H, h, mu, s_a, s_w, s_u, nullptr,
                                     tid);
    __syncthreads();
    if (tid < 64) {
        const int lane = tid;
        float x[4] = {1.f, 0.f, 0.f, 1.f};
        if (lane < C) {
            const float a = s_a[lane], w = s_w[lane], u = s_u[lane];
            x[0] = a; x[1] = w; x[2] = u * a; x[3] = fmaf(u, w, 1.f);
        }
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {  // tree product, later tokens on the left
            const float4 y = make_float4(__shfl_down(x[0], off, 64), __shfl_down(x[1], off, 64),
                                         __shfl_down(x[2], off, 64), __shfl_down(x[3], off, 64));
            if ((lane & (2 * off - 1)) == 0) mat_mul_left(x, y);
        }
        if (lane == 0) chunksum[(size_t)g * H + h] = make_float4(x[0], x[1], x[2], x[3]);
    }
}

// ------------------------------------------------------------------------------------------
// 3. prep: one workgroup per (chunk, head)
// ------------------------------------------------------------------------------------------
template <class TI, int DK_, int DV_, int C_, int VARIANT_, bool APC_>
struct PrepCfg {
    using MT = typename OpOf<TI>::type;
    static constexpr int DK = DK_, DV = DV_, C = C_, VARIANT = VARIANT_;
    static constexpr bool APC = APC_ || VARIANT_ == 0;
    static constexpr int PAD = 16 / (int)sizeof(MT);  // one 16-byte pad per row
    static constexpr int LDK = DK + PAD, LDC = C + PAD, LDT = C + 4, LDI = 16 + PAD;
    static constexpr int NB = C / 16, NSEG = C / 16;
    static constexpr int NSG = NSEG > 1 ? NSEG - 1 : 1;  // segment summaries read per lane
    static constexpr int NWC = (DK / 16 + 3) / 4;       // W column blocks per wave
    static constexpr int NUC = (DV / 16 + 3) / 4;       // U column blocks per wave
    // LDS map (bytes)
    static constexpr size_t OFF_TM = 0;                                    // float [C][LDT]
    static constexpr size_t OFF_AI = OFF_TM + al16((size_t)C * LDT * 4);   // MT [C][LDC]
    static constexpr size_t OFF_AIT = OFF_AI + al16((size_t)C * LDC * sizeof(MT));
    static constexpr size_t OFF_AQ = OFF_AIT + al16((size_t)C * LDC * sizeof(MT));
    static constexpr size_t OFF_INV = OFF_AQ + al16((size_t)C * LDC * sizeof(MT));
    static constexpr size_t OFF_KB = OFF_INV + al16((size_t)4 * 16 * LDI * sizeof(MT));
    static constexpr size_t OFF_QB = OFF_KB + al16((size_t)C * LDK * sizeof(MT));  // then W
    static constexpr size_t OFF_PB = OFF_QB + al16((size_t)C * LDK * sizeof(MT));
    static constexpr size_t OFF_KBT = OFF_PB + al16((size_t)C * LDK * sizeof(MT));  // [DK][LDC]
    static constexpr size_t OFF_PBT = OFF_KBT + al16((size_t)DK * LDC * sizeof(MT));
    static constexpr size_t OFF_SC = OFF_PBT + al16((size_t)DK * LDC * sizeof(MT));
    // scalars: r, mu/r, 1/den, beta (or u), gamma_tok (or ||k||^2), a_tok, w_tok, alpha_tok [C];
    // gamma_C [DK]
    static constexpr size_t SZ_SC = (size_t)(8 * C + DK) * 4;
    static constexpr size_t TOTAL = al16(OFF_SC + SZ_SC);
};

struct PrepArgs {
    const void *q, *k, *v, *alpha, *omega, *r;
    const int32_t *cu, *choff;
    const float2* carry;
    const float4* segsum;
    const float* seggam;
    float* P_T;
    char* rec;
    const int32_t* segoff;  // packed batches: this segment's row of the segment table
    int N, T, H;
    int seg, nseg;
    float mu, scale;
};

// Position of prep slot x of segment a.seg (slots are chunk slot * H + head): head h,
// sequence n, global chunk g, first token c0, length L, and whether the chunk is the
// sequence's last. False past the segment's last slot (and for every later slot).
struct PrepPos {
    int h, n, g, c0, L;
    bool last;
};

__device__ __forceinline__ bool prep_pos(const PrepArgs& a, int C, int x, PrepPos& p)
{
    const int cs = x / a.H;
    p.h = x % a.H;
    int m;
    if (!a.cu) {
        const int ncs = (a.T + C - 1) / C;
        int lo, hi;
        seg_range(ncs, a.seg, a.nseg, lo, hi);
        const int per = hi - lo;
        if (per <= 0) return false;
        p.n = cs / per;
        if (p.n >= a.N) return false;
        m = lo + cs % per;
        p.g = p.n * ncs + m;
    } else {
        if (cs >= a.segoff[a.N]) return false;
        int lo = 0, hi = a.N - 1;  // largest n with segoff[n] <= cs
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (a.segoff[mid] <= cs) lo = mid; else hi = mid - 1;
        }
        p.n = lo;
        const int len = max(0, a.cu[p.n + 1] - a.cu[p.n]);
        int slo, shi;
        seg_range((len + C - 1) / C, a.seg, a.nseg, slo, shi);
        m = slo + (cs - a.segoff[p.n]);
        p.g = a.choff[p.n] + m;
    }
    int t0, t1;
    seq_range(a.cu, p.n, a.T, t0, t1);
    p.c0 = t0 + m * C;
    p.L = min(C, t1 - p.c0);
    p.last = p.c0 + p.L == t1;
    return p.L > 0;
}

// B fragment of U = A V for value columns 16 nt .. 16 nt + 15, contraction slice s over the
// chunk's tokens, read straight from v: lane (g, i) takes column 16 nt + i at KF/4 consecutive
// tokens. Raw values; tokens past the end are zeroed by vfrag_mask.
template <class TI, class MT, int C>
struct VFrag {
    using FC = Frag<MT, C>;
    static constexpr int NE = FC::KF / 4;  // elements per lane
    TI e[NE];
};

template <class TI, class MT, int C>
__device__ __forceinline__ typename Frag<MT, C>::V vfrag_pack(const VFrag<TI, MT, C>& f, int k0,
                                                              int L)
{
    using FC = Frag<MT, C>;
    typename FC::V out;
    MT* o = reinterpret_cast<MT*>(&out);
#pragma unroll
    for (int j = 0; j < VFrag<TI, MT, C>::NE; ++j)
        o[j] = k0 + j < L ? from_f32<MT>(to_f32(f.e[j])) : from_f32<MT>(0.f);
    return out;
}

// Raw global inputs of one (chunk, head) for one thread of the prep kernel. They are loaded
// unconditionally (rows past the end of the sequence re-read its last row and are masked when
// used) and kept raw, so that a persistent workgroup can have the next chunk's loads in flight
// while it computes the current one.
template <class TI, class CF>
struct PrepIn {
    using MT = typename CF::MT;
    using FC = Frag<MT, CF::C>;
    using P2 = typename std::conditional<sizeof(TI) == 2, unsigned, float2>::type;
    TI rraw;                               // r of token tid
    VFrag<TI, MT, CF::C> vf[CF::NUC][FC::NS];  // B fragments of U = A V
    // diagonal variant: carry and earlier-segment summaries of the lane's channel pair, and
    // alpha, k, omega, q of its 16 tokens (bf16 pairs or float pairs)
    float2 z0, z1;
    float4 sgA0[CF::NSG], sgA1[CF::NSG];
    float2 sgG[CF::NSG];
    P2 al[16], kk[16], ww[16], qq[16];
};

template <class TI, class CF>
__device__ __forceinline__ void prep_load_main(PrepIn<TI, CF>& in, const PrepArgs& a,
                                               const PrepPos& p, int ch, int t0s, int tid)
{
    using P2 = typename PrepIn<TI, CF>::P2;
    constexpr int DK = CF::DK, C = CF::C, NSEG = CF::NSEG;
    const int H = a.H;
    const size_t row0 = (size_t)p.c0 * H + p.h;
    in.rraw = ((const TI*)a.r)[row0 + (size_t)min(min(tid, C - 1), p.L - 1) * H];
    if constexpr (CF::VARIANT == 0) {
        const size_t cbase = ((size_t)p.g * H + p.h) * DK + ch;
        in.z0 = a.carry[cbase];
        in.z1 = a.carry[cbase + 1];
        if constexpr (NSEG > 1) {
#pragma unroll
            for (int ps = 0; ps < NSEG - 1; ++ps) {
                const size_t sb = (((size_t)p.g * H + p.h) * (NSEG - 1) + ps) * DK + ch;
                in.sgA0[ps] = a.segsum[sb];
                in.sgA1[ps] = a.segsum[sb + 1];
                in.sgG[ps] = *reinterpret_cast<const float2*>(a.seggam + sb);
            }
        }
        const TI *ga = (const TI*)a.alpha, *gk = (const TI*)a.k, *gw = (const TI*)a.omega,
                 *gq = (const TI*)a.q;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const size_t e = (row0 + (size_t)min(t0s + j, p.L - 1) * H) * DK + ch;
            in.al[j] = *reinterpret_cast<const P2*>(ga + e);
            in.kk[j] = *reinterpret_cast<const P2*>(gk + e);
            in.ww[j] = *reinterpret_cast<const P2*>(gw + e);
            in.qq[j] = *reinterpret_cast<const P2*>(gq + e);
        }
    }
}

template <class TI, class CF>
__device__ __forceinline__ void prep_load_v(PrepIn<TI, CF>& in, const PrepArgs& a,
                                            const PrepPos& p, int wave, int lane)
{
    using FC = Frag<typename CF::MT, CF::C>;
    constexpr int DV = CF::DV;
    const int H = a.H, li = lane & 15, lg = lane >> 4;
    const size_t row0 = (size_t)p.c0 * H + p.h;
    const TI* gv = (const TI*)a.v;
#pragma unroll
    for (int u = 0; u < CF::NUC; ++u) {
        const int nt = min(wave + 4 * u, DV / 16 - 1);
#pragma unroll
        for (int s = 0; s < FC::NS; ++s) {
            const int k0 = FC::KF * s + (FC::KF / 4) * lg;
#pragma unroll
            for (int j = 0; j < VFrag<TI, typename CF::MT, CF::C>::NE; ++j)
                in.vf[u][s].e[j] = gv[(row0 + (size_t)min(k0 + j, p.L - 1) * H) * DV + 16 * nt + li];
        }
    }
}

// Persistent: workgroup b takes the slots b, b + gridDim.x, ... of the segment (one (chunk,
// head) each) and loads the next slot's inputs while it computes the current one.
template <class TI, class CF>
__global__ __launch_bounds__(NT) void prep_kernel(PrepArgs a)
{
    using MT = typename CF::MT;
    using RC = Rec<MT, CF::DK, CF::DV, CF::C>;
    using FC = Frag<MT, CF::C>;
    constexpr int DK = CF::DK, DV = CF::DV, C = CF::C, LDK = CF::LDK, LDC = CF::LDC,
                  LDT = CF::LDT, NB = CF::NB;
    constexpr bool DIAG = CF::VARIANT == 0;
    constexpr bool APC = CF::APC;
    extern __shared__ __attribute__((aligned(16))) char smem[];

    const int H = a.H;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, lg = lane >> 4;
    const TI* gq = (const TI*)a.q;
    const TI* gk = (const TI*)a.k;
    const TI* ga = (const TI*)a.alpha;
    const TI* gw = (const TI*)a.omega;
    const TI* gr = (const TI*)a.r;

    float* Tm = (float*)(smem + CF::OFF_TM);
    MT* Ai = (MT*)(smem + CF::OFF_AI);
    MT* AiT = (MT*)(smem + CF::OFF_AIT);
    MT* Aq = (MT*)(smem + CF::OFF_AQ);
    MT* Inv = (MT*)(smem + CF::OFF_INV);
    MT* Kb = (MT*)(smem + CF::OFF_KB);
    MT* Qb = (MT*)(smem + CF::OFF_QB);
    MT* Wst = Qb;  // W staging once Q_bar has been copied out
    MT* Pb = (MT*)(smem + CF::OFF_PB);
    MT* KbT = (MT*)(smem + CF::OFF_KBT);
    MT* PbT = (MT*)(smem + CF::OFF_PBT);
    float* s_r = (float*)(smem + CF::OFF_SC);
    float* s_mr = s_r + C;
    float* s_rden = s_mr + C;
    float* s_beta = s_rden + C;
    float* s_gtok = s_beta + C;
    float* s_atok = s_gtok + C;
    float* s_wtok = s_atok + C;
    float* s_alph = s_wtok + C;
    float* s_gC = s_alph + C;

    // diagonal variant: wave s replays tokens [16 s, 16 s + 16) for the channel pair
    // (2 l, 2 l + 1) of lane l, from the chunk carry and the summaries of earlier segments
    constexpr int NSEG = CF::NSEG, NP = DK / 2;
    const int seg = wave, pc = lane;
    const bool dact = DIAG && seg < NSEG && pc < NP;
    const int ch = 2 * min(pc, NP - 1), t0s = 16 * min(seg, NSEG - 1);

    PrepPos cur;
    if (!prep_pos(a, C, blockIdx.x, cur)) return;
    PrepIn<TI, CF> in;
    prep_load_main<TI, CF>(in, a, cur, ch, t0s, tid);
    for (int x = blockIdx.x;; x += gridDim.x) {
    PrepPos nxt;
    const bool more = prep_pos(a, C, x + gridDim.x, nxt);
    if (!more) nxt = cur;  // the prefetch below then re-reads valid rows, unused
    const int h = cur.h, n = cur.n, g = cur.g, c0 = cur.c0, L = cur.L;
    const bool last = cur.last;
    const size_t row0 = (size_t)c0 * H + h;  // (token c0, head h)
    char* recb = a.rec + ((size_t)g * H + h) * RC::BYTES;
    MT* rec = (MT*)recb;
    float* rec_gc = (float*)(recb + RC::GC_BYTES);

    if (tid < C) {
        const float rr = tid < L ? to_f32(in.rraw) : 1.f;
        s_r[tid] = rr;
        s_mr[tid] = a.mu / rr;
        s_rden[tid] = 1.f;
    }
    __syncthreads();

    // ---- phase 1: variance replay and operands ------------------------------------------
    // Tokens past the end of the sequence act as alpha = 1, k = q = v = omega = 0: they leave
    // every state unchanged and give zero operand rows (and identity rows of A).
    if (DIAG) {
        if (dact) {
            float zn0 = in.z0.x, zd0 = in.z0.y, zn1 = in.z1.x, zd1 = in.z1.y;
            float g0 = 1.f, g1 = 1.f;
            if constexpr (NSEG > 1) {
#pragma unroll
                for (int ps = 0; ps < NSEG - 1; ++ps) {
                    if (ps < seg) {
                        const float4 A0 = in.sgA0[ps], A1 = in.sgA1[ps];
                        float nn = A0.x * zn0 + A0.y * zd0, dd = A0.z * zn0 + A0.w * zd0;
                        zn0 = nn; zd0 = dd; renorm2(zn0, zd0);
                        nn = A1.x * zn1 + A1.y * zd1; dd = A1.z * zn1 + A1.w * zd1;
                        zn1 = nn; zd1 = dd; renorm2(zn1, zd1);
                        g0 *= in.sgG[ps].x;
                        g1 *= in.sgG[ps].y;
                    }
                }
            }
            float kb0[16], kb1[16], pb0[16], pb1[16];
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int t = t0s + j;
                float2 alv = unpack2(in.al[j]), kv = unpack2(in.kk[j]);
                float2 wv = unpack2(in.ww[j]), qv = unpack2(in.qq[j]);
                if (t >= L) {
                    alv = make_float2(1.f, 1.f);
                    kv = wv = qv = make_float2(0.f, 0.f);
                }
                g0 *= alv.x;
                g1 *= alv.y;
                const float n0 = fmaf(alv.x * alv.x, zn0, wv.x * zd0);  // n_t
                const float n1 = fmaf(alv.y * alv.y, zn1, wv.y * zd1);
                pb0[j] = n0 * kv.x * __builtin_amdgcn_rcpf(zd0 * g0);  // p_hat k / gamma
                pb1[j] = n1 * kv.y * __builtin_amdgcn_rcpf(zd1 * g1);
                const float mr = s_mr[t];
                zd0 = fmaf(kv.x * kv.x * mr, n0, zd0);                 // d_t
                zd1 = fmaf(kv.y * kv.y * mr, n1, zd1);
                zn0 = n0;
                zn1 = n1;
                if (j & 1) {
                    renorm2(zn0, zd0);
                    renorm2(zn1, zd1);
                }
                kb0[j] = g0 * kv.x;
                kb1[j] = g1 * kv.y;
                st2<MT>(Kb + t * LDK + ch, kb0[j], kb1[j]);
                st2<MT>(Qb + t * LDK + ch, a.scale * g0 * qv.x, a.scale * g1 * qv.y);
                st2<MT>(Pb + t * LDK + ch, pb0[j], pb1[j]);
            }
            store8<MT>(PbT + ch * LDC + t0s, pb0);
            store8<MT>(PbT + ch * LDC + t0s + 8, pb0 + 8);
            store8<MT>(PbT + (ch + 1) * LDC + t0s, pb1);
            store8<MT>(PbT + (ch + 1) * LDC + t0s + 8, pb1 + 8);
            store8<MT>(KbT + ch * LDC + t0s, kb0);
            store8<MT>(KbT + ch * LDC + t0s + 8, kb0 + 8);
            store8<MT>(KbT + (ch + 1) * LDC + t0s, kb1);
            store8<MT>(KbT + (ch + 1) * LDC + t0s + 8, kb1 + 8);
            if (seg == NSEG - 1) {
                *reinterpret_cast<float2*>(s_gC + ch) = make_float2(g0, g1);
                if (last && a.P_T)  // the sequence's final variances p_T = n_T / d_T
                    *reinterpret_cast<float2*>(a.P_T + ((size_t)n * H + h) * DK + ch) =
                        make_float2(zn0 / zd0, zn1 / zd1);
            }
        }
    } else {
        // isotropic: per-token coefficients, then the scalar Moebius chain of the head as a
        // Kogge-Stone scan over the chunk's tokens (lane = token) from the chunk carry
        iso_token_coeffs<TI, DK, C, APC>(gk, ga, gw, gr, c0, L, H, h, a.mu, s_atok, s_wtok,
                                         s_beta, s_gtok, tid);
        // (s_beta holds u_t and s_gtok ||k_t||^2 until the scan below)
        if (!APC && tid < C) {
            const float av = to_f32(ga[row0 + (size_t)min(tid, L - 1) * H]);
            s_alph[tid] = tid < L ? av : 1.f;
        }
        __syncthreads();
        if (wave == 0) {
            const int t = lane;
            const bool ok = t < C;
            float ma = 1.f, mb = 0.f, mc = 0.f, md = 1.f, at = 1.f, wt = 0.f, nk = 0.f;
            if (ok) {
                at = s_atok[t];
                wt = s_wtok[t];
                const float u = s_beta[t];
                nk = s_gtok[t];
                ma = at; mb = wt; mc = u * at; md = fmaf(u, wt, 1.f);
            }
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const float ya = __shfl_up(ma, off, 64), yb = __shfl_up(mb, off, 64);
                const float yc = __shfl_up(mc, off, 64), yd = __shfl_up(md, off, 64);
                if (lane >= off) {
                    const float na = ma * ya + mb * yc, nb = ma * yb + mb * yd;
                    const float nc = mc * ya + md * yc, nd = mc * yb + md * yd;
                    ma = na; mb = nb; mc = nc; md = nd;
                    renorm4(ma, mb, mc, md);
                }
            }
            const float2 z = a.carry[(size_t)g * H + h];
            float zn = ma * z.x + mb * z.y, zd = mc * z.x + md * z.y;  // after token t
            renorm2(zn, zd);
            float en = __shfl_up(zn, 1, 64), ed = __shfl_up(zd, 1, 64);  // before token t
            if (lane == 0) { en = z.x; ed = z.y; }
            if (last && a.P_T && lane == 63) a.P_T[(size_t)n * H + h] = zn / zd;  // b_T
            const float bh = at * en / ed + wt;                          // b_hat_t
            float gt = (!APC && ok) ? s_alph[t] : 1.f;
            if (!APC) {
#pragma unroll
                for (int off = 1; off < 64; off <<= 1) {  // gamma_t: prefix product of alpha
                    const float y = __shfl_up(gt, off, 64);
                    if (lane >= off) gt *= y;
                }
            }
            if (ok) {
                s_beta[t] = t < L ? bh / (s_r[t] + bh * nk) : 0.f;
                if (!APC) s_gtok[t] = gt;
            }
        }
        __syncthreads();
        if (APC) {
            // channel-wise gates: thread c (and c + DK for the query side) runs the decay
            // product of channel c over the chunk
            if (tid < 2 * DK) {
                const int c = tid % DK;
                const bool kside = tid < DK;
                float gm = 1.f;
                for (int t8 = 0; t8 < C; t8 += 8) {
                    float pb8[8], kb8[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const int t = t8 + j;
                        const bool ok = t < L;
                        const size_t e = (row0 + (size_t)min(t, L - 1) * H) * DK + c;
                        const float av = to_f32(ga[e]);
                        gm *= ok ? av : 1.f;
                        if (kside) {
                            const float kraw = to_f32(gk[e]);
                            const float kv = ok ? kraw : 0.f;
                            pb8[j] = s_beta[t] * kv * __builtin_amdgcn_rcpf(gm);
                            kb8[j] = gm * kv;
                            Kb[t * LDK + c] = from_f32<MT>(kb8[j]);
                            Pb[t * LDK + c] = from_f32<MT>(pb8[j]);
                        } else {
                            const float qraw = to_f32(gq[e]);
                            const float qv = ok ? qraw : 0.f;
                            Qb[t * LDK + c] = from_f32<MT>(a.scale * gm * qv);
                        }
                    }
                    if (kside) {
                        store8<MT>(PbT + c * LDC + t8, pb8);
                        store8<MT>(KbT + c * LDC + t8, kb8);
                    }
                }
                if (kside) s_gC[c] = gm;
            }
        } else {
            for (int idx = tid; idx < C * DK; idx += NT) {
                const int t = idx / DK, c = idx % DK;
                const bool ok = t < L;
                const size_t e = (row0 + (size_t)min(t, L - 1) * H) * DK + c;
                const float gm = s_gtok[t];
                const float kraw = to_f32(gk[e]), qraw = to_f32(gq[e]);
                const float kv = ok ? kraw : 0.f, qv = ok ? qraw : 0.f;
                const float pb = s_beta[t] * kv / gm, kb = gm * kv;
                Kb[t * LDK + c] = from_f32<MT>(kb);
                Qb[t * LDK + c] = from_f32<MT>(a.scale * gm * qv);
                Pb[t * LDK + c] = from_f32<MT>(pb);
                PbT[c * LDC + t] = from_f32<MT>(pb);
                KbT[c * LDC + t] = from_f32<MT>(kb);
            }
            if (tid < DK) s_gC[tid] = s_gtok[C - 1];
        }
    }
    // the next slot's inputs (this thread is done with the current ones)
    prep_load_main<TI, CF>(in, a, nxt, ch, t0s, tid);
    __syncthreads();

    // ---- phase 2: T = tril(K_bar P_bar^T, -1) / den and A_qk = tril(Q_bar P_bar^T) / den ---
    // 2a: wave b owns diagonal block b: its K_bar P_bar^T diagonal is sum_i p_hat k^2, which
    // gives den; the wave scales the block and inverts I + T_bb by forward substitution.
    if (wave < NB) {
        const int b = wave;
        const floatx4 tdiag =
            mm_kc<MT, DK>(Kb + 16 * b * LDK, LDK, Pb + 16 * b * LDK, LDK, zero4(), lane);
        if (DIAG && lg == (li >> 2)) {
            const int t = 16 * b + li;
            s_rden[t] = 1.f / (s_r[t] + tdiag[li & 3]);
        }
        wave_lds_sync();
        const float rd = s_rden[16 * b + li];
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
            const int row = 4 * lg + rr;
            Tm[(16 * b + row) * LDT + 16 * b + li] = row > li ? tdiag[rr] * rd : 0.f;
        }
        wave_lds_sync();
        if (lg == 0) {
            const int j = li;
            float x[16];
            const float* Tb = Tm + (16 * b) * LDT + 16 * b;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                float trow[16];
#pragma unroll
                for (int v4 = 0; v4 < (i + 3) / 4; ++v4) {
                    const float4 q4 = *reinterpret_cast<const float4*>(Tb + i * LDT + 4 * v4);
                    trow[4 * v4] = q4.x; trow[4 * v4 + 1] = q4.y;
                    trow[4 * v4 + 2] = q4.z; trow[4 * v4 + 3] = q4.w;
                }
                float sum = 0.f;
#pragma unroll
                for (int kq = 0; kq < i; ++kq) sum = fmaf(trow[kq], x[kq], sum);
                x[i] = i < j ? 0.f : (i == j ? 1.f : -sum);
            }
#pragma unroll
            for (int i = 0; i < 16; ++i) Ai[(16 * b + i) * LDC + 16 * b + j] = from_f32<MT>(x[i]);
            store8<MT>(AiT + (16 * b + j) * LDC + 16 * b, x);
            store8<MT>(AiT + (16 * b + j) * LDC + 16 * b + 8, x + 8);
        }
    }
    __syncthreads();
    // 2b: off-diagonal T blocks and every A_qk block, columns scaled by 1/den; T(ib, jb) and
    // A_qk(ib, jb) share the P_bar fragment of block column jb
    {
        constexpr int NPAIR = NB * (NB - 1) / 2, NUNIT = NPAIR + NB;
#pragma unroll
        for (int u0 = 0; u0 < NUNIT; u0 += 4) {
            const int unit = u0 + wave;
            if (unit < NUNIT) {
                int ib, jb;
                if (unit < NPAIR) {  // enumerate (ib > jb) in row order
                    int x = unit;
                    ib = 1;
                    while (x >= ib) { x -= ib; ++ib; }
                    jb = x;
                } else {
                    ib = jb = unit - NPAIR;
                }
                const float rd = s_rden[16 * jb + li];
                if (ib > jb) {
                    floatx4 tacc = zero4(), qacc = zero4();
                    mm_kc2<MT, DK>(Kb + 16 * ib * LDK, Qb + 16 * ib * LDK, LDK,
                                   Pb + 16 * jb * LDK, LDK, tacc, qacc, lane);
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr) {
                        const int row = 16 * ib + 4 * lg + rr, col = 16 * jb + li;
                        Tm[row * LDT + col] = tacc[rr] * rd;
                        Aq[row * LDC + col] = from_f32<MT>(qacc[rr] * rd);
                    }
                } else {
                    const floatx4 qacc = mm_kc<MT, DK>(Qb + 16 * ib * LDK, LDK,
                                                       Pb + 16 * jb * LDK, LDK, zero4(), lane);
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr) {
                        const int row = 16 * ib + 4 * lg + rr, col = 16 * jb + li;
                        Aq[row * LDC + col] =
                            from_f32<MT>((4 * lg + rr) >= li ? qacc[rr] * rd : 0.f);
                    }
                }
            }
        }
        // zero the blocks above the diagonal of A_qk and A: 16-byte stores
        constexpr int VPB = 16 * (int)sizeof(MT) / 16;  // 16-byte vectors per block row
        constexpr int NUP = NB * (NB - 1) / 2;          // blocks above the diagonal
        if constexpr (NUP > 0)
            for (int idx = tid; idx < 2 * NUP * 16 * VPB; idx += NT) {
                const int which = idx / (NUP * 16 * VPB), rem = idx % (NUP * 16 * VPB);
                int blk = rem / (16 * VPB);
                const int row16 = (rem / VPB) % 16, vec = rem % VPB;
                int ib = 0;  // blk -> (ib < jb)
                while (blk >= NB - 1 - ib) { blk -= NB - 1 - ib; ++ib; }
                const int jb = ib + 1 + blk;
                MT* base = which ? Ai : Aq;
                *reinterpret_cast<uint4*>(base + (16 * ib + row16) * LDC + 16 * jb +
                                          vec * (16 / (int)sizeof(MT))) = make_uint4(0, 0, 0, 0);
            }
    }
    __syncthreads();

    // V fragments of this slot for phase 4 (loaded here so that they do not occupy registers
    // during the replay; they land while the record is written and phase 3 runs)
    prep_load_v<TI, CF>(in, a, cur, wave, lane);

    // ---- record: Q_bar, A_qk, K_tail^T = gamma_C (.) P_bar^T / den, gamma_C ---------------
    copy_out<MT>(rec + RC::Q, Qb, C, DK, LDK, tid);
    copy_out<MT>(rec + RC::AQ, Aq, C, C, LDC, tid);
    {
        constexpr int VE = 16 / (int)sizeof(MT);
        constexpr int VPR = C / VE;
        for (int idx = tid; idx < DK * VPR; idx += NT) {
            const int c = idx / VPR, t = (idx % VPR) * VE;
            const float gc = s_gC[c];
            uint4 u = *reinterpret_cast<const uint4*>(PbT + c * LDC + t);
            MT* x = reinterpret_cast<MT*>(&u);
#pragma unroll
            for (int e = 0; e < VE; ++e) x[e] = from_f32<MT>(gc * to_f32(x[e]) * s_rden[t + e]);
            *reinterpret_cast<uint4*>(rec + RC::KT + (size_t)c * C + t) = u;
        }
    }
    if (tid < DK) rec_gc[tid] = s_gC[tid];
    __syncthreads();  // Q_bar has been read out before its region takes W below

    // ---- phase 3: A = (I + T)^-1 off the diagonal (diagonal blocks done in 2a) ----------
    // A_ij = -A_ii sum_{j<=k<i} T_ik A_kj, one block diagonal d = i - j at a time.
#pragma unroll
    for (int d = 1; d < NB; ++d) {
        const int nblk = NB - d;
        if (wave < nblk) {
            const int jb = wave, ib = jb + d;
            floatx4 acc = zero4();
            for (int kb = jb; kb < ib; ++kb)
                acc = mm16_tv<MT>(Tm + (16 * ib) * LDT + 16 * kb, LDT,
                                  AiT + (16 * jb) * LDC + 16 * kb, LDC, acc, lane);
            MT* tmpT = Inv + wave * 16 * CF::LDI;  // tmp stored transposed as the next B operand
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) tmpT[li * CF::LDI + 4 * lg + rr] = from_f32<MT>(acc[rr]);
            wave_lds_sync();
            const floatx4 res = mm_kc<MT, 16>(Ai + (16 * ib) * LDC + 16 * ib, LDC, tmpT, CF::LDI,
                                              zero4(), lane);
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
                const int row = 16 * ib + 4 * lg + rr, col = 16 * jb + li;
                Ai[row * LDC + col] = from_f32<MT>(-res[rr]);
                AiT[col * LDC + row] = from_f32<MT>(-res[rr]);
            }
        }
        __syncthreads();
    }

    // ---- phase 4: W = A K_bar (staged, then copied out) and U = A V (packed tiles) --------
    // Wave w takes column blocks w, w + 4, ... of both; the A fragments of every row block are
    // read once, and A's upper triangle is skipped (row block mt needs k < 16 (mt + 1)).
    {
        typename FC::V afr[NB][FC::NS];
#pragma unroll
        for (int mt = 0; mt < NB; ++mt)
#pragma unroll
            for (int s = 0; s < FC::NS; ++s)
                afr[mt][s] = FC::ld(Ai + (16 * mt + li) * LDC + FC::KF * s + (FC::KF / 4) * lg);
#pragma unroll
        for (int u = 0; u < CF::NWC; ++u) {
            const int nt = wave + 4 * u;
            if (nt < DK / 16) {
                typename FC::V bfr[FC::NS];
#pragma unroll
                for (int s = 0; s < FC::NS; ++s)
                    bfr[s] = FC::ld(KbT + (16 * nt + li) * LDC + FC::KF * s + (FC::KF / 4) * lg);
#pragma unroll
                for (int mt = 0; mt < NB; ++mt) {
                    floatx4 acc = zero4();
#pragma unroll
                    for (int s = 0; s < FC::NS; ++s)
                        if (FC::KF * s < 16 * (mt + 1)) acc = FC::mma(acc, afr[mt][s], bfr[s]);
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr)
                        Wst[(16 * mt + 4 * lg + rr) * LDK + 16 * nt + li] = from_f32<MT>(acc[rr]);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < CF::NUC; ++u) {
            const int nt = wave + 4 * u;
            if (nt < DV / 16) {
                typename FC::V bfr[FC::NS];
#pragma unroll
                for (int s = 0; s < FC::NS; ++s)
                    bfr[s] = vfrag_pack<TI, MT, C>(in.vf[u][s], FC::KF * s + (FC::KF / 4) * lg, L);
#pragma unroll
                for (int mt = 0; mt < NB; ++mt) {
                    floatx4 acc = zero4();
#pragma unroll
                    for (int s = 0; s < FC::NS; ++s)
                        if (FC::KF * s < 16 * (mt + 1)) acc = FC::mma(acc, afr[mt][s], bfr[s]);
                    store4<MT>(rec + RC::U + ((size_t)(nt * NB + mt) * 64 + lane) * 4, acc[0],
                               acc[1], acc[2], acc[3]);
                }
            }
        }
    }
    __syncthreads();
    copy_out<MT>(rec + RC::W, Wst, C, DK, LDK, tid);
    if (!more) break;
    __syncthreads();  // every LDS region is reused by the next slot
    cur = nxt;
    }
}

// ------------------------------------------------------------------------------------------
// 4. state passing: one workgroup per (sequence, head, dv tile), chunks in order
// ------------------------------------------------------------------------------------------
template <class TI, int DK_, int DV_, int BV_, int C_>
struct StateCfg {
    using MT = typename OpOf<TI>::type;
    static constexpr int DK = DK_, DV = DV_, BV = BV_, C = C_;
    static constexpr int PAD = 16 / (int)sizeof(MT);
    static constexpr int LDK = DK + PAD, LDC = C + PAD;
    static constexpr int NB = C / 16, NNT = BV / 16, NKT = DK / 16;
    static constexpr int MB = (NB + 3) / 4;   // output row blocks per wave
    static constexpr int KB = (NKT + 3) / 4;  // state row blocks per wave
    static constexpr int LDO = BV + 16 / (int)sizeof(TI);  // rows of the O staging tile
    static constexpr size_t OFF_SMT = 0;                                        // [BV][LDK]
    static constexpr size_t OFF_RT = al16((size_t)BV * LDK * sizeof(MT));      // [BV][LDC]
    static constexpr size_t OFF_O = OFF_RT + al16((size_t)BV * LDC * sizeof(MT));  // TI [C][LDO]
    static constexpr size_t TOTAL = OFF_O + al16((size_t)C * LDO * sizeof(TI));
};

struct StateArgs {
    const char* rec;
    const int32_t *cu, *choff;
    const float* S0;  // state entering the segment (NULL = 0)
    float* S_T;       // state leaving it (NULL = not stored)
    void* o;
    int N, T, H, DV;
    int seg, nseg;
};

// Record fragments of one chunk for one wave, kept in storage precision until used (a
// conversion at load time would make the load wait for every load issued before it).
template <class MT> struct Raw4 { using type = uint2; };   // four bf16
template <> struct Raw4<float> { using type = uint4; };    // four floats

template <class MT>
__device__ __forceinline__ float4 unpack4(const typename Raw4<MT>::type& v)
{
    if constexpr (std::is_same<MT, float>::value) {
        return make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z),
                           __uint_as_float(v.w));
    } else {
        return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xFFFF0000u),
                           __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xFFFF0000u));
    }
}

template <class CF>
struct ChunkFrags {
    using MT = typename CF::MT;
    using FK = Frag<MT, CF::DK>;
    using FC = Frag<MT, CF::C>;
    typename FK::V w[CF::MB][FK::NS], q[CF::MB][FK::NS];
    typename FC::V aq[CF::MB][FC::NS], kt[CF::KB][FC::NS];
    typename Raw4<MT>::type u[CF::MB][CF::NNT];
    float4 gc[CF::KB];
};

template <class CF>
__device__ __forceinline__ void load_frags_early(ChunkFrags<CF>& F, const char* recb, int wave,
                                                 int lane)
{
    using MT = typename CF::MT;
    using RC = Rec<MT, CF::DK, CF::DV, CF::C>;
    using FK = Frag<MT, CF::DK>;
    constexpr int DK = CF::DK;
    const int li = lane & 15, lg = lane >> 4;
    const MT* rec = (const MT*)recb;
#pragma unroll
    for (int mb = 0; mb < CF::MB; ++mb) {
        const int row = 16 * min(wave + 4 * mb, CF::NB - 1) + li;
#pragma unroll
        for (int s = 0; s < FK::NS; ++s) {
            const int k0 = FK::KF * s + (FK::KF / 4) * lg;
            F.w[mb][s] = FK::ld(rec + RC::W + (size_t)row * DK + k0);
            F.q[mb][s] = FK::ld(rec + RC::Q + (size_t)row * DK + k0);
        }
    }
}

template <class CF>
__device__ __forceinline__ void load_frags_late(ChunkFrags<CF>& F, const char* recb, int wave,
                                                int lane, int col0)
{
    using MT = typename CF::MT;
    using RC = Rec<MT, CF::DK, CF::DV, CF::C>;
    using FC = Frag<MT, CF::C>;
    constexpr int C = CF::C;
    const int li = lane & 15, lg = lane >> 4;
    const MT* rec = (const MT*)recb;
    const float* gcp = (const float*)(recb + RC::GC_BYTES);
#pragma unroll
    for (int mb = 0; mb < CF::MB; ++mb) {
        const int mt = min(wave + 4 * mb, CF::NB - 1);
        const int row = 16 * mt + li;
#pragma unroll
        for (int s = 0; s < FC::NS; ++s)
            F.aq[mb][s] = FC::ld(rec + RC::AQ + (size_t)row * C + FC::KF * s + (FC::KF / 4) * lg);
#pragma unroll
        for (int nt = 0; nt < CF::NNT; ++nt)
            F.u[mb][nt] = *reinterpret_cast<const typename Raw4<MT>::type*>(
                rec + RC::U + ((size_t)((col0 / 16 + nt) * CF::NB + mt) * 64 + lane) * 4);
    }
#pragma unroll
    for (int kb = 0; kb < CF::KB; ++kb) {
        const int it = min(wave + 4 * kb, CF::NKT - 1);
        const int row = 16 * it + li;
#pragma unroll
        for (int s = 0; s < FC::NS; ++s)
            F.kt[kb][s] = FC::ld(rec + RC::KT + (size_t)row * C + FC::KF * s + (FC::KF / 4) * lg);
        F.gc[kb] = *reinterpret_cast<const float4*>(gcp + 16 * it + 4 * lg);
    }
}

// Every load is unconditional (row blocks past the end re-read the last valid one, whose
// values go unused), so the compiler can count them and let them fly across the compute of
// the chunks in between instead of waiting at the first use.
template <class CF>
__device__ __forceinline__ void load_frags(ChunkFrags<CF>& F, const char* recb, int wave,
                                           int lane, int col0)
{
    load_frags_early<CF>(F, recb, wave, lane);
    load_frags_late<CF>(F, recb, wave, lane, col0);
}

// O rows of a finished chunk, staged in LDS by state_step, go out as 16-byte stores (rows past
// the sequence end are not written).
template <class TI, class CF>
__device__ __forceinline__ void store_o(const TI* Ost, TI* go, size_t row0, int L, int H, int DV,
                                        int col0, int tid)
{
    constexpr int VE = 16 / (int)sizeof(TI), VPR = CF::BV / VE;
    for (int idx = tid; idx < CF::C * VPR; idx += NT) {
        const int t = idx / VPR, e = (idx % VPR) * VE;
        if (t < L)
            *reinterpret_cast<uint4*>(go + (row0 + (size_t)t * H) * DV + col0 + e) =
                *reinterpret_cast<const uint4*>(Ost + t * CF::LDO + e);
    }
}

// One chunk of the state recurrence with the chunk's fragments F:
//   R = U - W S_in (to RT), O = Q_bar S_in + A_qk R (staged in Ost), S = gamma_C (.) S +
//   K_tail^T R, and S written back as the next chunk's B operand. The O tile of the previous
//   chunk (row0p, Lp; Lp = 0 for none) is stored first.
template <class TI, class CF>
__device__ __forceinline__ void state_step(ChunkFrags<CF>& F, floatx4 (&Sacc)[CF::KB][CF::NNT],
                                           typename CF::MT* SmT, typename CF::MT* RT, TI* Ost,
                                           TI* go, size_t row0p, int Lp, int H, int DV, int col0,
                                           int wave, int lane, const char* rec_next2)
{
    using MT = typename CF::MT;
    using FK = Frag<MT, CF::DK>;
    using FC = Frag<MT, CF::C>;
    constexpr int LDK = CF::LDK, LDC = CF::LDC;
    const int li = lane & 15, lg = lane >> 4;

    if (Lp > 0) store_o<TI, CF>(Ost, go, row0p, Lp, H, DV, col0, wave * 64 + lane);

    // B fragments of S_in, all issued before the products
    typename FK::V bs[FK::NS][CF::NNT];
#pragma unroll
    for (int s = 0; s < FK::NS; ++s)
#pragma unroll
        for (int nt = 0; nt < CF::NNT; ++nt)
            bs[s][nt] = FK::ld(SmT + (16 * nt + li) * LDK + FK::KF * s + (FK::KF / 4) * lg);

    floatx4 Oacc[CF::MB][CF::NNT];
#pragma unroll
    for (int mb = 0; mb < CF::MB; ++mb) {
        const int mt = wave + 4 * mb;
        floatx4 Racc[CF::NNT];
#pragma unroll
        for (int nt = 0; nt < CF::NNT; ++nt) Racc[nt] = Oacc[mb][nt] = zero4();
        if (mt < CF::NB) {
#pragma unroll
            for (int s = 0; s < FK::NS; ++s) {
#pragma unroll
                for (int nt = 0; nt < CF::NNT; ++nt) {
                    Racc[nt] = FK::mma(Racc[nt], F.w[mb][s], bs[s][nt]);
                    Oacc[mb][nt] = FK::mma(Oacc[mb][nt], F.q[mb][s], bs[s][nt]);
                }
            }
#pragma unroll
            for (int nt = 0; nt < CF::NNT; ++nt) {
                const float4 u = unpack4<MT>(F.u[mb][nt]);
                store4<MT>(RT + (16 * nt + li) * LDC + 16 * mt + 4 * lg, u.x - Racc[nt][0],
                           u.y - Racc[nt][1], u.z - Racc[nt][2], u.w - Racc[nt][3]);
            }
        }
    }
    // W and Q_bar of this set are consumed: the chunk two steps ahead reuses their registers
    load_frags_early<CF>(F, rec_next2, wave, lane);
    __syncthreads();

    // B fragments of R, shared by the O and S products
    typename FC::V br[FC::NS][CF::NNT];
#pragma unroll
    for (int s = 0; s < FC::NS; ++s)
#pragma unroll
        for (int nt = 0; nt < CF::NNT; ++nt)
            br[s][nt] = FC::ld(RT + (16 * nt + li) * LDC + FC::KF * s + (FC::KF / 4) * lg);
#pragma unroll
    for (int mb = 0; mb < CF::MB; ++mb) {
        const int mt = wave + 4 * mb;
        if (mt < CF::NB) {
#pragma unroll
            for (int s = 0; s < FC::NS; ++s) {
                if (FC::KF * s < 16 * (mt + 1)) {  // A_qk is lower triangular
#pragma unroll
                    for (int nt = 0; nt < CF::NNT; ++nt)
                        Oacc[mb][nt] = FC::mma(Oacc[mb][nt], F.aq[mb][s], br[s][nt]);
                }
            }
#pragma unroll
            for (int nt = 0; nt < CF::NNT; ++nt)
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    Ost[(16 * mt + 4 * lg + rr) * CF::LDO + 16 * nt + li] =
                        from_f32<TI>(Oacc[mb][nt][rr]);
        }
    }
#pragma unroll
    for (int kb = 0; kb < CF::KB; ++kb) {
        const int it = wave + 4 * kb;
        if (it < CF::NKT) {
            const float4 gc = F.gc[kb];
#pragma unroll
            for (int nt = 0; nt < CF::NNT; ++nt) {
                Sacc[kb][nt][0] *= gc.x;
                Sacc[kb][nt][1] *= gc.y;
                Sacc[kb][nt][2] *= gc.z;
                Sacc[kb][nt][3] *= gc.w;
            }
#pragma unroll
            for (int s = 0; s < FC::NS; ++s)
#pragma unroll
                for (int nt = 0; nt < CF::NNT; ++nt)
                    Sacc[kb][nt] = FC::mma(Sacc[kb][nt], F.kt[kb][s], br[s][nt]);
            // S_in of the next chunk (every wave finished reading SmT before the barrier above)
#pragma unroll
            for (int nt = 0; nt < CF::NNT; ++nt)
                store4<MT>(SmT + (16 * nt + li) * LDK + 16 * it + 4 * lg, Sacc[kb][nt][0],
                           Sacc[kb][nt][1], Sacc[kb][nt][2], Sacc[kb][nt][3]);
        }
    }
    load_frags_late<CF>(F, rec_next2, wave, lane, col0);
    __syncthreads();
}

// One wave per SIMD: the workgroups of this kernel are few (one per sequence, head and dv
// tile), so the compiler may spend the whole register file on keeping two chunks' fragments in
// flight instead of sharing it with a second wave.
template <class TI, class CF>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(1, 1))) void state_kernel(
    StateArgs a)
{
    using MT = typename CF::MT;
    using RC = Rec<MT, CF::DK, CF::DV, CF::C>;
    constexpr int DK = CF::DK, BV = CF::BV, C = CF::C, LDK = CF::LDK;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    MT* SmT = (MT*)(smem + CF::OFF_SMT);  // S_in, transposed: SmT[col][key]
    MT* RT = (MT*)(smem + CF::OFF_RT);    // R, transposed: RT[col][token]
    TI* Ost = (TI*)(smem + CF::OFF_O);    // O of the last chunk, [token][col]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, lg = lane >> 4;
    const int NH = a.N * a.H;
    const int nh = blockIdx.x % NH, tile = blockIdx.x / NH;  // the tiles of one head share an XCD
    const int n = nh / a.H, h = nh % a.H;
    const int col0 = tile * BV;
    const int H = a.H, DV = a.DV;
    TI* go = (TI*)a.o;

    // S tiles (it, nt), it = wave + 4 kb, in MFMA result layout
    floatx4 Sacc[CF::KB][CF::NNT];
#pragma unroll
    for (int kb = 0; kb < CF::KB; ++kb) {
        const int it = wave + 4 * kb;
#pragma unroll
        for (int nt = 0; nt < CF::NNT; ++nt) {
            Sacc[kb][nt] = zero4();
            if (it < CF::NKT && a.S0) {
                const float* src = a.S0 + (size_t)nh * DK * DV;
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    Sacc[kb][nt][rr] =
                        src[(size_t)(16 * it + 4 * lg + rr) * DV + col0 + 16 * nt + li];
            }
            if (it < CF::NKT)
                store4<MT>(SmT + (16 * nt + li) * LDK + 16 * it + 4 * lg, Sacc[kb][nt][0],
                           Sacc[kb][nt][1], Sacc[kb][nt][2], Sacc[kb][nt][3]);
        }
    }

    int t0, t1;
    seq_range(a.cu, n, a.T, t0, t1);
    int mlo, mhi;  // this segment's chunks of the sequence
    seg_range((t1 - t0 + C - 1) / C, a.seg, a.nseg, mlo, mhi);
    const int gbase = a.cu ? a.choff[n] : n * ((a.T + C - 1) / C);
    auto recp = [&](int m) { return a.rec + ((size_t)(gbase + m) * H + h) * RC::BYTES; };

    // two fragment sets used alternately; while chunk m computes with one, the other holds
    // chunk m + 1, and each half of the first is reloaded with chunk m + 2 as soon as chunk m
    // has consumed it (loads past the segment's last chunk re-read it)
    ChunkFrags<CF> F0, F1;
    if (mhi > mlo) {
        load_frags<CF>(F0, recp(mlo), wave, lane, col0);
        load_frags<CF>(F1, recp(min(mlo + 1, mhi - 1)), wave, lane, col0);
    }
    // the first chunk's fragments are needed at once; waiting for them here, outside the loop,
    // also tells the compiler that nothing is in flight when the loop is entered, so the loop
    // head does not wait for the previous prefetch before issuing the next one
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    // chunk m's O goes out during chunk m + 1 (and after the loop for the last one)
    auto row_of = [&](int m) { return (size_t)(t0 + m * C) * H + h; };
    auto len_of = [&](int m) { return min(C, t1 - (t0 + m * C)); };
    for (int m = mlo; m < mhi; m += 2) {
        state_step<TI, CF>(F0, Sacc, SmT, RT, Ost, go, row_of(m - 1), m > mlo ? len_of(m - 1) : 0,
                           H, DV, col0, wave, lane, recp(min(m + 2, mhi - 1)));
        if (m + 1 >= mhi) break;
        state_step<TI, CF>(F1, Sacc, SmT, RT, Ost, go, row_of(m), len_of(m), H, DV, col0, wave,
                           lane, recp(min(m + 3, mhi - 1)));
    }
    if (mhi > mlo) store_o<TI, CF>(Ost, go, row_of(mhi - 1), len_of(mhi - 1), H, DV, col0, tid);

    if (a.S_T) {
        float* dst = a.S_T + (size_t)nh * DK * DV;
#pragma unroll
        for (int kb = 0; kb < CF::KB; ++kb) {
            const int it = wave + 4 * kb;
            if (it < CF::NKT) {
#pragma unroll
                for (int nt = 0; nt < CF::NNT; ++nt)
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr)
                        dst[(size_t)(16 * it + 4 * lg + rr) * DV + col0 + 16 * nt + li] =
                            Sacc[kb][nt][rr];
            }
        }
    }
}

// ------------------------------------------------------------------------------------------
// host side
// ------------------------------------------------------------------------------------------
template <class TI, int DK, int DV, int C>
constexpr bool prep_fits()
{
    return PrepCfg<TI, DK, DV, C, 0, true>::TOTAL <= 160 * 1024 &&
           PrepCfg<TI, DK, DV, C, 1, false>::TOTAL <= 160 * 1024;
}

// Number of segments the chunks of every sequence are cut into (see seg_range): one for short
// sequences, up to four when the longest possible sequence has 64 chunks or more.
inline int pick_nseg(int T, int C)
{
    const int maxm = (T + C - 1) / C;  // chunks of the longest possible sequence
    return std::max(1, std::min(4, maxm / 16));
}

// Workspace map of one call.
struct WsMap {
    size_t choff, segoff, chunksum, segsum, seggam, carry, S, rec, total;
};

inline WsMap ws_map(int variant, bool packed, size_t maxch, int N, int H, int dk, int dv,
                    int nseg, size_t nseg16_m1, size_t rec_bytes)
{
    const size_t nchan = variant == 0 ? (size_t)dk : 1;
    WsMap m;
    m.choff = 0;
    m.segoff = al256(((size_t)N + 1) * 4);
    m.chunksum = m.segoff + (packed ? al256((size_t)nseg * (N + 1) * 4) : 0);
    m.segsum = m.chunksum + al256(maxch * H * nchan * 16);
    const size_t nsg = variant == 0 ? maxch * H * nseg16_m1 * dk : 0;
    m.seggam = m.segsum + al256(nsg * 16);
    m.carry = m.seggam + al256(nsg * 4);
    m.S = m.carry + al256(maxch * H * nchan * 8);
    m.rec = m.S + (nseg > 1 ? al256((size_t)N * H * dk * dv * 4) : 0);
    m.total = m.rec + maxch * H * rec_bytes;
    return m;
}

inline size_t max_chunks(bool packed, int N, int T, int C)
{
    // fixed length: N * ceil(T / C); packed (B = 1): every sequence adds at most one partial
    // chunk to T / C
    return packed ? (size_t)T / C + N : (size_t)N * ((T + C - 1) / C);
}

template <class TI, int DK, int DV, int C>
size_t ws_bytes_t(int variant, bool packed, int N, int T, int H)
{
    using MT = typename OpOf<TI>::type;
    return ws_map(variant, packed, max_chunks(packed, N, T, C), N, H, DK, DV, pick_nseg(T, C),
                  C / 16 - 1, Rec<MT, DK, DV, C>::BYTES).total;
}

// A second stream per device for the state pass, so that it overlaps the prep pass of the next
// segment; created once, default priority, never destroyed.
hipError_t side_stream(hipStream_t main, hipStream_t& side)
{
    int dev = 0;
    hipError_t e = main ? hipStreamGetDevice(main, &dev) : hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    static std::mutex mu;
    static hipStream_t streams[64] = {};
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!streams[dev]) {
        int cur = 0;
        if ((e = hipGetDevice(&cur)) != hipSuccess) return e;
        if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
        e = hipStreamCreateWithFlags(&streams[dev], hipStreamNonBlocking);
        if (cur != dev) (void)hipSetDevice(cur);
        if (e != hipSuccess) {
            streams[dev] = nullptr;
            return e;
        }
    }
    side = streams[dev];
    return hipSuccess;
}

template <class TI, int DK, int DV, int C, int VARIANT, bool APC>
hipError_t run_t(const FwdCall& fc, hipStream_t st)
{
    using PC = PrepCfg<TI, DK, DV, C, VARIANT, APC>;
    using MT = typename PC::MT;
    using RC = Rec<MT, DK, DV, C>;
    constexpr int BV = DV >= 32 ? 32 : DV;
    using SC = StateCfg<TI, DK, DV, BV, C>;
    const SeqArgs& sa = fc.sa;
    const bool packed = sa.cu_seqlens != nullptr;
    const size_t maxch = max_chunks(packed, sa.N, sa.T, C);
    if (maxch == 0) return hipSuccess;
    const int nseg = pick_nseg(sa.T, C);
    const WsMap wm = ws_map(VARIANT, packed, maxch, sa.N, sa.H, DK, DV, nseg, C / 16 - 1,
                            RC::BYTES);
    char* ws = (char*)fc.workspace;
    int32_t* choff = (int32_t*)(ws + wm.choff);
    int32_t* segoff = (int32_t*)(ws + wm.segoff);
    float4* chunksum = (float4*)(ws + wm.chunksum);
    float4* segsum = (float4*)(ws + wm.segsum);
    float* seggam = (float*)(ws + wm.seggam);
    float2* carry = (float2*)(ws + wm.carry);
    float* Sws = (float*)(ws + wm.S);
    char* rec = ws + wm.rec;
    const TI *k = (const TI*)fc.k, *al = (const TI*)fc.alpha, *om = (const TI*)fc.omega,
             *r = (const TI*)fc.r;
    hipError_t e;

    // 1-2: chunk summaries and carries (every chunk of every sequence)
    if (packed) {
        if ((e = launch_chunk_table(sa.cu_seqlens, sa.N, C, choff, st)) != hipSuccess) return e;
        hipLaunchKernelGGL(seg_table_kernel, dim3(1), dim3(1), 0, st, sa.cu_seqlens, sa.N, C,
                           nseg, segoff);
    }
    const dim3 grid((unsigned)maxch, sa.H);
    if (VARIANT == 0)
        hipLaunchKernelGGL((summary_diag_kernel<TI, DK, C>), grid, dim3(NT), 0, st, k, al, om, r,
                           sa.cu_seqlens, choff, sa.N, sa.T, sa.H, fc.mu, chunksum, segsum,
                           seggam);
    else
        hipLaunchKernelGGL((summary_iso_kernel<TI, DK, C, APC>), grid, dim3(NT), 0, st, k, al,
                           om, r, sa.cu_seqlens, choff, sa.N, sa.T, sa.H, fc.mu, chunksum);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_carry_scan(chunksum, fc.P0, sa, VARIANT == 0 ? DK : 1, C, choff, carry,
                               fc.P_T, st)) != hipSuccess)
        return e;

    // persistent prep: as many workgroups as fit on the device at once (queried once per
    // instantiation and device; the LDS map usually allows one per CU)
    static int prep_slots[64] = {};
    int dev = 0;
    if ((e = st ? hipStreamGetDevice(st, &dev) : hipGetDevice(&dev)) != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    if (!prep_slots[dev]) {
        if ((e = hipFuncSetAttribute((const void*)prep_kernel<TI, PC>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)PC::TOTAL)) != hipSuccess)
            return e;
        int per_cu = 0, ncu = 0;
        if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
                 &per_cu, prep_kernel<TI, PC>, NT, PC::TOTAL)) != hipSuccess)
            return e;
        if ((e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev)) !=
            hipSuccess)
            return e;
        prep_slots[dev] = std::max(1, per_cu) * std::max(1, ncu);
    }
    PrepArgs pa;
    pa.q = fc.q; pa.k = fc.k; pa.v = fc.v; pa.alpha = fc.alpha; pa.omega = fc.omega; pa.r = fc.r;
    pa.cu = sa.cu_seqlens; pa.choff = choff; pa.carry = carry; pa.segsum = segsum;
    pa.seggam = seggam; pa.P_T = fc.P_T; pa.rec = rec; pa.N = sa.N; pa.T = sa.T; pa.H = sa.H;
    pa.nseg = nseg; pa.mu = fc.mu; pa.scale = fc.scale;
    StateArgs sta;
    sta.rec = rec; sta.cu = sa.cu_seqlens; sta.choff = choff; sta.o = fc.o; sta.N = sa.N;
    sta.T = sa.T; sta.H = sa.H; sta.DV = DV; sta.nseg = nseg;
    const unsigned nblk = (unsigned)((size_t)sa.N * sa.H * (DV / BV));

    // 3-4: per segment, prep on the caller's stream, then the state pass on the side stream
    // (ordered after that prep and after the previous segment's state pass)
    hipStream_t side = st;
    if (nseg > 1 && (e = side_stream(st, side)) != hipSuccess) return e;
    hipEvent_t ev[5] = {};
    if (nseg > 1)
        for (int i = 0; i <= nseg; ++i)
            if ((e = hipEventCreateWithFlags(&ev[i], hipEventDisableTiming)) != hipSuccess) {
                for (int j = 0; j < i; ++j) (void)hipEventDestroy(ev[j]);
                return e;
            }
    for (int sg = 0; sg < nseg && e == hipSuccess; ++sg) {
        pa.seg = sg;
        pa.segoff = segoff + (size_t)sg * (sa.N + 1);
        unsigned npg;
        if (packed) {
            npg = (unsigned)(maxch / nseg + sa.N);
        } else {
            const int ncs = (sa.T + C - 1) / C;
            npg = (unsigned)((size_t)sa.N * (((size_t)(sg + 1) * ncs) / nseg - ((size_t)sg * ncs) / nseg));
        }
        const size_t nslot = (size_t)npg * sa.H;
        if (nslot > 0)
            hipLaunchKernelGGL((prep_kernel<TI, PC>),
                               dim3((unsigned)std::min<size_t>(nslot, prep_slots[dev])), dim3(NT),
                               PC::TOTAL, st, pa);
        if ((e = hipGetLastError()) != hipSuccess) break;
        if (nseg > 1) {
            if ((e = hipEventRecord(ev[sg], st)) != hipSuccess) break;
            if ((e = hipStreamWaitEvent(side, ev[sg], 0)) != hipSuccess) break;
        }
        sta.seg = sg;
        sta.S0 = sg == 0 ? fc.S0 : Sws;
        sta.S_T = sg == nseg - 1 ? fc.S_T : Sws;
        hipLaunchKernelGGL((state_kernel<TI, SC>), dim3(nblk), dim3(NT), SC::TOTAL, side, sta);
        e = hipGetLastError();
    }
    if (nseg > 1) {
        // the caller's stream resumes after the last state pass
        if (e == hipSuccess) e = hipEventRecord(ev[nseg], side);
        if (e == hipSuccess) e = hipStreamWaitEvent(st, ev[nseg], 0);
        for (int i = 0; i <= nseg; ++i) (void)hipEventDestroy(ev[i]);
    }
    return e;
}

template <class TI, int DK, int DV, int C>
hipError_t run_variant(const FwdCall& fc, hipStream_t st)
{
    if constexpr (!prep_fits<TI, DK, DV, C>()) {
        return hipErrorInvalidConfiguration;
    } else {
        if (fc.variant == 0) return run_t<TI, DK, DV, C, 0, true>(fc, st);
        if (fc.apc) return run_t<TI, DK, DV, C, 1, true>(fc, st);
        return run_t<TI, DK, DV, C, 1, false>(fc, st);
    }
}

// Compile-time dispatch over (dtype, dk, dv, chunk) calling F::template go<TI, DK, DV, C>().
template <class F>
auto dispatch(kdn_dtype_t dtype, int dk, int dv, int chunk, F f) -> decltype(f.template go<float, 16, 16, 16>())
{
#define KDN_C(TI, DK, DV)                                                   \
    switch (chunk) {                                                        \
    case 16: return f.template go<TI, DK, DV, 16>();                        \
    case 32: return f.template go<TI, DK, DV, 32>();                        \
    default: return f.template go<TI, DK, DV, 64>();                        \
    }
#define KDN_V(TI, DK)                                                       \
    switch (dv) {                                                           \
    case 16: KDN_C(TI, DK, 16)                                              \
    case 32: KDN_C(TI, DK, 32)                                              \
    case 64: KDN_C(TI, DK, 64)                                              \
    default: KDN_C(TI, DK, 128)                                             \
    }
#define KDN_K(TI)                                                           \
    switch (dk) {                                                           \
    case 16: KDN_V(TI, 16)                                                  \
    case 32: KDN_V(TI, 32)                                                  \
    case 64: KDN_V(TI, 64)                                                  \
    default: KDN_V(TI, 128)                                                 \
    }
    if (dtype == KDN_F32) {
        KDN_K(float)
    } else {
        KDN_K(bf16)
    }
#undef KDN_K
#undef KDN_V
#undef KDN_C
    return f.template go<float, 16, 16, 16>();  // not reached
}

struct FitsF {
    template <class TI, int DK, int DV, int C> bool go() const { return prep_fits<TI, DK, DV, C>(); }
};
struct WsF {
    int variant;
    bool packed;
    int N, T, H;
    template <class TI, int DK, int DV, int C> size_t go() const
    {
        if constexpr (!prep_fits<TI, DK, DV, C>()) return 0;
        else return ws_bytes_t<TI, DK, DV, C>(variant, packed, N, T, H);
    }
};
struct RunF {
    const FwdCall* fc;
    hipStream_t st;
    template <class TI, int DK, int DV, int C> hipError_t go() const
    {
        return run_variant<TI, DK, DV, C>(*fc, st);
    }
};

}  // namespace

bool chunked_supported(kdn_dtype_t dtype, int dk, int dv, int chunk)
{
    if (chunk != 16 && chunk != 32 && chunk != 64) return false;
    return dispatch(dtype, dk, dv, chunk, FitsF{});
}

int chunked_default_chunk(kdn_dtype_t dtype, int dk, int dv)
{
    for (int c = 64; c >= 16; c >>= 1)
        if (chunked_supported(dtype, dk, dv, c)) return c;
    return 16;
}

size_t chunked_workspace_bytes(int variant, bool packed, int N, int B, int T, int H, int dk,
                               int dv, kdn_dtype_t dtype, int chunk)
{
    if (chunk == 0) chunk = chunked_default_chunk(dtype, dk, dv);
    (void)B;  // fixed length has N == B; a packed batch has B == 1 and T tokens in total
    return dispatch(dtype, dk, dv, chunk, WsF{variant, packed, N, T, H});
}

hipError_t launch_chunked(const FwdCall& fc, hipStream_t stream)
{
    FwdCall c = fc;
    if (c.chunk == 0) c.chunk = chunked_default_chunk(c.dtype, c.dk, c.dv);
    return dispatch(c.dtype, c.dk, c.dv, c.chunk, RunF{&c, stream});
}

}  // namespace kdn
