// Fused chunkwise forward of Diagonal / Isotropic KDN on gfx950.
//
// arXiv 2609.07816, App. "Hardware-Efficient Chunkwise Algorithm". Tokens are cut into chunks of
// C (chunks restart at every sequence start; the last one may be partial). One workgroup walks
// one (sequence, head, tile of BV value columns) through its chunks in order and carries both
// recurrent states with it:
//   - the variance chain as homogeneous Moebius pairs z = (n, d), p = n / d, one per key channel
//     (diagonal) or one per head (isotropic): eqs. kla-box-mobius / iso-kla-box-mobius, with the
//     carry between chunks of eq. chunk-gain-carry;
//   - the memory S: float32 MFMA accumulators, plus a copy in operand precision in LDS that is
//     the next chunk's MFMA operand.
// Only the inputs, o and the final states cross HBM.
//
// Per chunk, with chunk-local token t and gamma_t = prod_{j<=t} alpha_j (per channel):
//   1. variance (VALU): the chunk is cut into NW segments of C / NW tokens (one per wave); each
//      wave composes its segment's token matrices (eq. chunk-gain-summary), the segment carries
//      follow from the chunk carry (eq. chunk-gain-local-prefix), and each wave replays its
//      tokens (eq. chunk-gain-emission) to get p_hat_t (diagonal) or b_hat_t and
//      beta_t = b_hat_t / (r_t + b_hat_t ||k_t||^2) (isotropic);
//   2. operands: K_bar = Gamma (.) K, Q_bar = Gamma (.) Q, P_bar = G (.) K (/) Gamma with
//      G = p_hat (diagonal) or beta (isotropic);
//   3. L = diag(c) + tril(K_bar P_bar^T, -1) with c_t = r_t + (K_bar P_bar^T)_tt
//      = r_t + sum_i p_hat_ti k_ti^2 (diagonal, the innovation variance of eq. kla-box-gain) or
//      c_t = 1 (isotropic); A = L^-1; A_qk = tril(Q_bar P_bar^T) (diagonal included: the read
//      follows the write);
//   4. R = A (V - K_bar S)   (row t: token t's innovation divided by c_t),
//      O = scale (Q_bar S + A_qk R),  S <- gamma_C (.) (S + P_bar^T R).
// This is Sec. "Chunkwise Memory Scan" (R = U - W S with W = A K_bar and U = A V, K_tail =
// (gamma_C / gamma) (.) kappa) with the gain's normalisation kappa_t = p_hat_t (.) k_t / c_t
// moved into the triangular solve: the unit-lower I + T of the section becomes L, and W, U are
// never formed.
//
// Dense products run on MFMA (bf16 operands with float32 accumulation for bf16 inputs, float32
// MFMA for float32 inputs); S, the variance chain and the triangular solve stay in float32.
#include <algorithm>
#include <atomic>
#include <type_traits>

#include "kdn_device.h"

namespace kdn {
namespace {

constexpr int NW = 8;         // waves per workgroup
constexpr int NTH = 64 * NW;  // threads per workgroup

constexpr size_t al16(size_t x) { return (x + 15) & ~(size_t)15; }
constexpr size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }
constexpr size_t cmax(size_t a, size_t b) { return a > b ? a : b; }

template <class TI> struct OpOf { using type = bf16; };
template <> struct OpOf<float> { using type = float; };

// ------------------------------------------------------------------------------------------
// MFMA fragments read from LDS: lane (g, i) holds KF/4 consecutive k values of row i (A side)
// or of column i (B side, stored transposed); one fragment feeds one bf16 MFMA (KF = 32 or 16)
// or four float32 MFMAs (KF = 16). Both sides use the same k assignment, so the contraction is
// exact whatever order the unit applies internally. Result: acc[r] = D[4 g + r][i].
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

// 16 x 16 x 16 products from register fragments: lane (g, i) holds A[i][4g..4g+3] (A side) or
// B[4g..4g+3][i] (B side). A result tile (lane (g, i): rows 4g..4g+3 of column i) is therefore
// already a B fragment of the next product.
template <class MT> struct F16;
template <> struct F16<bf16> {
    using V = uint2;
    __device__ static V pack(float x0, float x1, float x2, float x3)
    {
        bf16x4 v;
        v[0] = (bf16)x0; v[1] = (bf16)x1; v[2] = (bf16)x2; v[3] = (bf16)x3;
        return __builtin_bit_cast(V, v);
    }
    __device__ static V ld(const bf16* p) { return *reinterpret_cast<const V*>(p); }
    __device__ static floatx4 mma(floatx4 acc, V a, V b)
    {
        return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(bf16x4, a),
                                                          __builtin_bit_cast(bf16x4, b), acc, 0,
                                                          0, 0);
    }
};
template <> struct F16<float> {
    using V = float4;
    __device__ static V pack(float x0, float x1, float x2, float x3)
    {
        return make_float4(x0, x1, x2, x3);
    }
    __device__ static V ld(const float* p) { return *reinterpret_cast<const V*>(p); }
    __device__ static floatx4 mma(floatx4 acc, V a, V b)
    {
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b.x, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b.y, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b.z, acc, 0, 0, 0);
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b.w, acc, 0, 0, 0);
    }
};

// Four values (rows 4g..4g+3 of a result column, or four consecutive elements) in MT.
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

// Four consecutive values in MT as floats (8- or 16-byte aligned source).
template <class MT>
__device__ __forceinline__ float4 ld4f(const MT* src)
{
    if constexpr (std::is_same<MT, float>::value) {
        return *reinterpret_cast<const float4*>(src);
    } else {
        const uint2 u = *reinterpret_cast<const uint2*>(src);
        return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                           __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u));
    }
}

// N consecutive values (N = 2, 4 or 8; the destination is aligned to N elements).
template <class MT, int N>
__device__ __forceinline__ void storeN(MT* dst, const float* x)
{
    if constexpr (N == 8) store8<MT>(dst, x);
    else if constexpr (N == 4) store4<MT>(dst, x[0], x[1], x[2], x[3]);
    else st2<MT>(dst, x[0], x[1]);
}

// Two adjacent inputs from one raw word (bf16 pair) or a float pair.
__device__ __forceinline__ float2 unpack2(unsigned u)
{
    return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xFFFF0000u));
}
__device__ __forceinline__ float2 unpack2(float2 v) { return v; }

// Power-of-two rescale of non-negative homogeneous values (the variance pairs and the Moebius
// products of non-negative token matrices): exact, keeps every ratio, and brings the largest
// entry into [0.5, 1). The exponent instruction gives 0 for 0, Inf and NaN, which leaves such
// values unchanged.
__device__ __forceinline__ void rescale2(float& n, float& d)
{
    const int e = -__builtin_amdgcn_frexp_expf(fmaxf(n, d));
    n = ldexpf(n, e);
    d = ldexpf(d, e);
}

__device__ __forceinline__ void rescale4(float* m)
{
    const int e = -__builtin_amdgcn_frexp_expf(fmaxf(fmaxf(m[0], m[1]), fmaxf(m[2], m[3])));
    m[0] = ldexpf(m[0], e);
    m[1] = ldexpf(m[1], e);
    m[2] = ldexpf(m[2], e);
    m[3] = ldexpf(m[3], e);
}

// z <- M z for a 2x2 matrix M = [x y; z w] (float4) acting on a homogeneous pair.
__device__ __forceinline__ float2 mat_vec(const float4& m, float2 v)
{
    float n = fmaf(m.x, v.x, m.y * v.y), d = fmaf(m.z, v.x, m.w * v.y);
    rescale2(n, d);
    return make_float2(n, d);
}

// ------------------------------------------------------------------------------------------
// Configuration and LDS map of one workgroup. Waves 0..3 (the variance waves) run the variance
// chain and form the operands of chunk m + 1 while waves 4..7 (the matrix waves) run the
// triangular solve and the state update of chunk m; the two groups meet at four barriers per
// chunk, and every SIMD hosts one wave of each, so VALU and MFMA work overlap.
// ------------------------------------------------------------------------------------------
constexpr int NVW = 4;  // variance waves: one segment of C / 4 tokens each
constexpr int NMW = 4;  // matrix waves

template <class TI, int DK_, int DV_, int BV_, int C_, int VARIANT_, bool APC_>
struct WalkCfg {
    using MT = typename OpOf<TI>::type;
    using P2 = typename std::conditional<sizeof(TI) == 2, unsigned, float2>::type;
    static constexpr int DK = DK_, DV = DV_, BV = BV_, C = C_, VARIANT = VARIANT_;
    static constexpr bool DIAG = VARIANT_ == 0;
    static constexpr bool APC = APC_ || DIAG;   // gates per key channel
    static constexpr int NV = DV / BV;          // value tiles (workgroups) per head
    static constexpr int SL = C / NVW;          // tokens per variance segment
    static constexpr int NP = DK / 2;           // key-channel pairs (one per lane)
    static constexpr int NB = C / 16, NNT = BV / 16, NKT = DK / 16;
    static constexpr int NXT = NB * NNT;                                // X / O tiles
    static constexpr int RPW = (NB + NMW - 1) / NMW;  // row blocks per matrix wave
    static constexpr int XPW = RPW * NNT;             // X / O tiles per matrix wave
    static constexpr int JT1 = (SL * 3 + 7) / 8, JT2 = (SL * 6 + 7) / 8;  // replay thirds
    static constexpr int NST = NKT * NNT, SPW = (NST + NMW - 1) / NMW;  // S tiles
    static constexpr int NLU = NB * (NB + 1) / 2;                       // lower block pairs
    static constexpr int NOFF = NB > 1 ? NB * (NB - 1) / 2 : 1;         // below the diagonal
    static constexpr int PAD = 16 / (int)sizeof(MT);  // one 16-byte pad per row
    static constexpr int LDK = DK + PAD, LDC = C + PAD, LDE = 16 + PAD, LDD = 20;
    static constexpr int LDO = BV + 16 / (int)sizeof(TI);
    static constexpr size_t SZ_OP = al16((size_t)C * LDK * sizeof(MT));
    static constexpr size_t SZ_PT = al16((size_t)DK * LDC * sizeof(MT));
    static constexpr size_t SZ_BL = al16((size_t)16 * LDE * sizeof(MT));
    // operands of a chunk: K_bar, Q_bar, P_bar [C][LDK]; P_bar^T [DK][LDC] in two buffers
    // (chunk parity: the variance waves write chunk m + 1's while the matrix waves read m's)
    static constexpr size_t OFF_KB = 0;
    static constexpr size_t OFF_QB = OFF_KB + SZ_OP;
    static constexpr size_t OFF_PB = OFF_QB + SZ_OP;
    static constexpr size_t OFF_PBT = OFF_PB + SZ_OP;
    // L's diagonal blocks (float32 [NB][16][LDD]) and the blocks below them (MT, MFMA
    // operands), the diagonal blocks of L^-1 and A_qk [C][LDC]
    static constexpr size_t OFF_LD = OFF_PBT + 2 * SZ_PT;
    static constexpr size_t OFF_LO = OFF_LD + al16((size_t)NB * 16 * LDD * 4);
    static constexpr size_t OFF_AI = OFF_LO + NOFF * SZ_BL;
    static constexpr size_t OFF_AQ = OFF_AI + NB * SZ_BL;
    // the variance waves' segment summaries and their decay products
    static constexpr size_t OFF_SGA = OFF_AQ + al16((size_t)C * LDC * sizeof(MT));
    static constexpr size_t OFF_SGG = OFF_SGA + (size_t)NVW * DK * 16;
    // S^T [BV][LDK], X^T and R^T [BV][LDC] in MT, O staging [C][LDO] in TI
    static constexpr size_t OFF_SMT = OFF_SGG + (size_t)NVW * DK * 4;
    static constexpr size_t OFF_XT = OFF_SMT + al16((size_t)BV * LDK * sizeof(MT));
    static constexpr size_t OFF_RT = OFF_XT + al16((size_t)BV * LDC * sizeof(MT));
    static constexpr size_t OFF_O = OFF_RT + al16((size_t)BV * LDC * sizeof(MT));
    // by chunk parity: variance carry into the chunk, gamma_C, r and mu / r
    static constexpr size_t OFF_CAR = OFF_O + al16((size_t)C * LDO * sizeof(TI));
    static constexpr size_t OFF_GC = OFF_CAR + (size_t)2 * DK * 8;
    static constexpr size_t OFF_R = OFF_GC + (size_t)2 * DK * 4;
    static constexpr size_t OFF_MR = OFF_R + (size_t)2 * C * 4;
    static constexpr size_t TOTAL = al16(OFF_MR + (size_t)2 * C * 4);
};

struct WalkArgs {
    const void *q, *k, *v, *alpha, *omega, *r;
    const float *S0, *P0;
    void* o;
    float *S_T, *P_T;
    const int32_t* cu;     // packed batches: sequence offsets, else nullptr
    const int32_t* order;  // packed batches: sequences, longest first (nullptr: in order)
    int N, T, H;
    float mu, scale;
    uint32_t bytes_k, bytes_v, bytes_h;  // bytes of q / k / per-channel gates, of v, of r
};

// ------------------------------------------------------------------------------------------
// Buffer loads: 32-bit byte offsets against a descriptor of the whole tensor; the unit checks
// the range and returns 0 past the end, so rows past the end of a sequence need no clamping
// (they belong to the next sequence or read 0, and are masked where they are used).
// ------------------------------------------------------------------------------------------
typedef __amdgpu_buffer_rsrc_t rsrc_t;

__device__ __forceinline__ rsrc_t make_rsrc(const void* p, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes,
                                             0x00020000);
}

template <class T> __device__ __forceinline__ T bload(rsrc_t r, uint32_t off);
template <> __device__ __forceinline__ unsigned bload<unsigned>(rsrc_t r, uint32_t off)
{
    return __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0);
}
template <> __device__ __forceinline__ float bload<float>(rsrc_t r, uint32_t off)
{
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0));
}
template <> __device__ __forceinline__ float2 bload<float2>(rsrc_t r, uint32_t off)
{
    const auto u = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0);
    return make_float2(__uint_as_float(u[0]), __uint_as_float(u[1]));
}
template <> __device__ __forceinline__ bf16 bload<bf16>(rsrc_t r, uint32_t off)
{
    return __builtin_bit_cast(bf16, __builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0));
}

// One stored value held in a register of its own: a bf16 is kept zero-extended in 32 bits, so
// values loaded ahead are never packed two to a register (packing would wait for the load).
template <class TI> struct Raw1;
template <> struct Raw1<bf16> {
    using type = unsigned;
    static __device__ __forceinline__ unsigned load(rsrc_t r, uint32_t off)
    {
        return (unsigned)__builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0);
    }
    static __device__ __forceinline__ float f32(unsigned u) { return __uint_as_float(u << 16); }
};
template <> struct Raw1<float> {
    using type = float;
    static __device__ __forceinline__ float load(rsrc_t r, uint32_t off)
    {
        return bload<float>(r, off);
    }
    static __device__ __forceinline__ float f32(float x) { return x; }
};

// Descriptors and byte strides of one workgroup's inputs.
struct WalkSrc {
    rsrc_t q, k, v, al, om, r;
    uint32_t rowk, rowv, rowh;  // bytes per token row: channel tensors, v, per-head scalars
    uint32_t lane_k, lane_h;    // this lane's byte offset within a row (channel pair; head)
    uint32_t col_v;             // byte offset of the workgroup's first value column in a row
};

// Raw inputs of one chunk held by a variance lane (lane l of wave w: tokens [SL w, SL w + SL)
// of the key-channel pair (2 l, 2 l + 1)), loaded ahead and kept in storage precision (a
// conversion next to its load would make the load wait for everything issued before it).
template <class TI, class CF>
struct WalkIn {
    using P2 = typename CF::P2;
    P2 kk[CF::SL], qq[CF::SL];
    P2 al[CF::APC ? CF::SL : 1];    // per-channel gates
    P2 ww[CF::DIAG ? CF::SL : 1];   // per-channel process noise (diagonal)
    using R1 = typename Raw1<TI>::type;
    R1 als[CF::APC ? 1 : CF::SL];   // one gate per head (isotropic, scalar gates)
    R1 ws[CF::DIAG ? 1 : CF::SL];   // one process noise per head (isotropic)
    R1 rr;                          // r of token tid of the next chunk (tid < C)
};

// Tokens [J0, J1) of a variance lane's segment of the chunk starting at token c0.
template <int J0, int J1, class TI, class CF>
__device__ __forceinline__ void load_part(WalkIn<TI, CF>& in, const WalkSrc& sr, uint32_t c0,
                                          int vw)
{
    using P2 = typename CF::P2;
#pragma unroll
    for (int j = J0; j < J1; ++j) {
        const uint32_t tok = c0 + (uint32_t)(CF::SL * vw + j);
        const uint32_t e = tok * sr.rowk + sr.lane_k, eh = tok * sr.rowh + sr.lane_h;
        in.kk[j] = bload<P2>(sr.k, e);
        in.qq[j] = bload<P2>(sr.q, e);
        if constexpr (CF::APC) in.al[j] = bload<P2>(sr.al, e);
        else in.als[j] = Raw1<TI>::load(sr.al, eh);
        if constexpr (CF::DIAG) in.ww[j] = bload<P2>(sr.om, e);
        else in.ws[j] = Raw1<TI>::load(sr.om, eh);
    }
}

// Token j of a variance lane's segment in float32. In a chunk that may end early (MK), a
// token past the end of the sequence (j >= Lw) reads as no decay, no noise and zero key and
// query, so it leaves the variance and the memory unchanged and gives zero operand rows. The
// registers loaded ahead are only read here, never overwritten.
struct TokIn {
    float2 K, Q, A, W;
};
template <bool MK, class TI, class CF>
__device__ __forceinline__ TokIn tok_in(const WalkIn<TI, CF>& in, int j, int Lw)
{
    const bool pad = MK && j >= Lw;
    const float2 z = make_float2(0.f, 0.f);
    TokIn r;
    r.K = pad ? z : unpack2(in.kk[j]);
    r.Q = pad ? z : unpack2(in.qq[j]);
    if constexpr (CF::APC) {
        r.A = pad ? make_float2(1.f, 1.f) : unpack2(in.al[j]);
    } else {
        const float as = pad ? 1.f : Raw1<TI>::f32(in.als[CF::APC ? 0 : j]);
        r.A = make_float2(as, as);
    }
    if constexpr (CF::DIAG) {
        r.W = pad ? z : unpack2(in.ww[j]);
    } else {
        const float w = pad ? 0.f : Raw1<TI>::f32(in.ws[CF::DIAG ? 0 : j]);
        r.W = make_float2(w, w);
    }
    return r;
}

// V at the rows and column of a matrix lane's X tiles: tile j of matrix wave mw is row block
// mw + 4 (j / NNT), column tile j % NNT.
template <class TI, class CF>
__device__ __forceinline__ void load_v(typename Raw1<TI>::type (&vv)[CF::XPW][4], const WalkSrc& sr,
                                       uint32_t c0,
                                       int mw, int lane)
{
    const int li = lane & 15, lg = lane >> 4;
#pragma unroll
    for (int j = 0; j < CF::XPW; ++j) {
        const int ib = min(mw + NMW * (j / CF::NNT), CF::NB - 1), nt = j % CF::NNT;
        const uint32_t col = sr.col_v + (uint32_t)(16 * nt + li) * (uint32_t)sizeof(TI);
#pragma unroll
        for (int rr = 0; rr < 4; ++rr)
            vv[j][rr] =
                Raw1<TI>::load(sr.v, (c0 + (uint32_t)(16 * ib + 4 * lg + rr)) * sr.rowv + col);
    }
}

// ------------------------------------------------------------------------------------------
// The walk: one workgroup per (sequence, head, value tile). Iteration it runs the variance
// waves on chunk it and the matrix waves on chunk it - 1.
// ------------------------------------------------------------------------------------------
template <class TI, class CF>
__global__ __launch_bounds__(NTH) void walk_kernel(WalkArgs a)
{
    using MT = typename CF::MT;
    using FK = Frag<MT, CF::DK>;
    using FC = Frag<MT, CF::C>;
    using G = F16<MT>;
    constexpr int DK = CF::DK, DV = CF::DV, BV = CF::BV, C = CF::C, SL = CF::SL;
    constexpr int NP = CF::NP, NB = CF::NB, LDK = CF::LDK, LDC = CF::LDC, LDE = CF::LDE;
    constexpr int LDD = CF::LDD, LDO = CF::LDO;
    constexpr bool DIAG = CF::DIAG, APC = CF::APC;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    MT* Kb = (MT*)(smem + CF::OFF_KB);
    MT* Qb = (MT*)(smem + CF::OFF_QB);
    MT* Pb = (MT*)(smem + CF::OFF_PB);
    MT* PbT0 = (MT*)(smem + CF::OFF_PBT);  // [2][DK][LDC]
    float* Ld = (float*)(smem + CF::OFF_LD);
    MT* Lo = (MT*)(smem + CF::OFF_LO);
    MT* Ai = (MT*)(smem + CF::OFF_AI);
    MT* Aq = (MT*)(smem + CF::OFF_AQ);
    float4* segA = (float4*)(smem + CF::OFF_SGA);
    float* segG = (float*)(smem + CF::OFF_SGG);
    MT* SmT = (MT*)(smem + CF::OFF_SMT);
    MT* XT = (MT*)(smem + CF::OFF_XT);
    MT* RT = (MT*)(smem + CF::OFF_RT);
    TI* Ost = (TI*)(smem + CF::OFF_O);
    float2* carry = (float2*)(smem + CF::OFF_CAR);  // [2][DK]
    float* gC = (float*)(smem + CF::OFF_GC);        // [2][DK]
    float* s_r = (float*)(smem + CF::OFF_R);        // [2][C]
    float* s_mr = (float*)(smem + CF::OFF_MR);      // [2][C]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, lg = lane >> 4;
    // the wave index in a scalar register: the variance / matrix split is a uniform branch,
    // so each wave runs exactly one of the two loops below (with four barriers per chunk each)
    const int wu = __builtin_amdgcn_readfirstlane(wave);
    const bool vgrp = wu < NVW;   // variance wave (else matrix wave)
    const int vw = wu, mw = wu - NVW;
    const int mtid = tid - 64 * NVW;  // thread index within the matrix waves

    // block -> (sequence-head slot, value tile): the NV tiles of one head get block indices
    // congruent modulo 8, so round-robin dispatch puts them on one XCD, where they share the
    // L2 copy of the head's inputs
    const int NH = a.N * a.H;
    const int xcd = (int)(blockIdx.x % 8), rest = (int)(blockIdx.x / 8);
    const int vt = rest % CF::NV, slot = (rest / CF::NV) * 8 + xcd;
    if (slot >= NH) return;
    const int H = a.H;
    const int n = a.order ? a.order[slot / H] : slot / H;
    const int h = slot % H;
    if (n < 0 || n >= a.N) return;
    const int nh = n * H + h;
    const int col0 = vt * BV;
    int t0, t1;
    seq_range(a.cu, n, a.T, t0, t1);
    const int nch = (t1 - t0 + C - 1) / C;
    TI* go = (TI*)a.o;

    const int pc = min(lane, NP - 1), ch = 2 * pc;  // a variance lane's key-channel pair
    const bool vact = lane < NP;                    // the lane owns a pair

    WalkSrc sr;
    {
        constexpr uint32_t es = sizeof(TI);
        sr.q = make_rsrc(a.q, a.bytes_k);
        sr.k = make_rsrc(a.k, a.bytes_k);
        sr.v = make_rsrc(a.v, a.bytes_v);
        sr.al = make_rsrc(a.alpha, APC ? a.bytes_k : a.bytes_h);
        sr.om = make_rsrc(a.omega, DIAG ? a.bytes_k : a.bytes_h);
        sr.r = make_rsrc(a.r, a.bytes_h);
        sr.rowk = (uint32_t)H * DK * es;
        sr.rowv = (uint32_t)H * DV * es;
        sr.rowh = (uint32_t)H * es;
        sr.lane_k = ((uint32_t)h * DK + ch) * es;
        sr.lane_h = (uint32_t)h * es;
        sr.col_v = ((uint32_t)h * DV + col0) * es;
    }

    // ---- initial states ----------------------------------------------------------------
    floatx4 Sacc[CF::SPW];  // matrix waves: S tiles (it, nt) = (x % NKT, x / NKT), x = mw + 4 j
    if (!vgrp) {
#pragma unroll
        for (int j = 0; j < CF::SPW; ++j) {
            const int x = mw + NMW * j;
            Sacc[j] = zero4();
            if (x < CF::NST) {
                const int it = x % CF::NKT, nt = x / CF::NKT;
                if (a.S0) {
                    const float* src = a.S0 + (size_t)nh * DK * DV;
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr)
                        Sacc[j][rr] =
                            src[(size_t)(16 * it + 4 * lg + rr) * DV + col0 + 16 * nt + li];
                }
                store4<MT>(SmT + (16 * nt + li) * LDK + 16 * it + 4 * lg, Sacc[j][0],
                           Sacc[j][1], Sacc[j][2], Sacc[j][3]);
            }
        }
    }
    if (!vgrp) {  // the blocks of A_qk right of the diagonal stay zero
        constexpr int NVEC = C * LDC * (int)sizeof(MT) / 16;
        for (int idx = mtid; idx < NVEC; idx += 64 * NMW)
            reinterpret_cast<uint4*>(Aq)[idx] = make_uint4(0, 0, 0, 0);
    }
    if (DIAG ? tid < DK : tid == 0)
        carry[tid] = make_float2(a.P0 ? a.P0[(size_t)nh * (DIAG ? DK : 1) + tid] : 1.f, 1.f);
    if (nch == 0 && a.P_T && vt == 0 && (DIAG ? tid < DK : tid == 0))  // empty sequence
        a.P_T[(size_t)nh * (DIAG ? DK : 1) + tid] =
            a.P0 ? a.P0[(size_t)nh * (DIAG ? DK : 1) + tid] : 1.f;

    WalkIn<TI, CF> in;
    typename Raw1<TI>::type vv[CF::XPW][4];
    floatx4 Oacc[CF::XPW];
    if (nch > 0) {
        if (vgrp) {
            load_part<0, SL, TI, CF>(in, sr, t0, vw);
            if (tid < C) {
                const float rv =
                    to_f32(bload<TI>(sr.r, (uint32_t)(t0 + tid) * sr.rowh + sr.lane_h));
                const bool ok = tid < t1 - t0;
                s_r[tid] = ok ? rv : 1.f;
                s_mr[tid] = ok ? a.mu / rv : 0.f;
            }
        } else {
            load_v<TI, CF>(vv, sr, t0, mw, lane);
        }
    }
    __syncthreads();

    if (vgrp) {
        // ===== variance waves: chunk it; wave w takes tokens [SL w, SL w + SL) ===============
        float kn[DIAG ? 1 : SL], ka[DIAG ? 1 : SL];  // isotropic: ||k_t||^2 and mean alpha^2
        for (int it = 0; it <= nch; ++it) {
            const int mv = it;
            const bool vwork = mv < nch, vlast = mv == nch - 1;
            const int pv = mv & 1;
            const int c0v = t0 + mv * C, Lv = min(C, t1 - c0v);
            const int Lw = Lv - SL * vw;  // tokens of this wave's segment in the chunk
            const float* s_rv = s_r + pv * C;
            const float* s_mrv = s_mr + pv * C;
            MT* PbTv = PbT0 + (size_t)pv * DK * LDC;
            const uint32_t c0n = (uint32_t)(c0v + C);  // the next chunk

            // ---- phase A: the segment's Moebius product and decay product ------------------
            auto summary = [&](auto mk_c) {
                constexpr bool MK = decltype(mk_c)::value;
                if constexpr (DIAG) {
                    if (vact) {
                        float m0[4] = {1.f, 0.f, 0.f, 1.f}, m1[4] = {1.f, 0.f, 0.f, 1.f};
                        float g0 = 1.f, g1 = 1.f;
#pragma unroll
                        for (int j = 0; j < SL; ++j) {
                            const TokIn x = tok_in<MK>(in, j, Lw);
                            const float mr = s_mrv[SL * vw + j];
                            mob_left(m0, x.A.x * x.A.x, x.W.x, x.K.x * x.K.x * mr);
                            mob_left(m1, x.A.y * x.A.y, x.W.y, x.K.y * x.K.y * mr);
                            g0 *= x.A.x;
                            g1 *= x.A.y;
                            if ((j & 3) == 3 || j == SL - 1) {
                                rescale4(m0);
                                rescale4(m1);
                            }
                        }
                        segA[vw * DK + ch] = make_float4(m0[0], m0[1], m0[2], m0[3]);
                        segA[vw * DK + ch + 1] = make_float4(m1[0], m1[1], m1[2], m1[3]);
                        *reinterpret_cast<float2*>(segG + vw * DK + ch) = make_float2(g0, g1);
                    }
                } else {
                    // per-token ||k||^2 and mean_i alpha_i^2 by wave reductions, kept for the
                    // replay; one scalar chain per head, which every lane runs alike
                    float mm[4] = {1.f, 0.f, 0.f, 1.f};
                    float g0 = 1.f, g1 = 1.f;
#pragma unroll
                    for (int j = 0; j < SL; ++j) {
                        const TokIn x = tok_in<MK>(in, j, Lw);
                        kn[j] = wave_sum(vact ? fmaf(x.K.x, x.K.x, x.K.y * x.K.y) : 0.f);
                        if constexpr (APC)
                            ka[j] = wave_sum(vact ? fmaf(x.A.x, x.A.x, x.A.y * x.A.y) : 0.f) *
                                    (1.f / (float)DK);
                        else
                            ka[j] = x.A.x * x.A.x;
                        g0 *= x.A.x;
                        g1 *= x.A.y;
                        const float ut = kn[j] * s_mrv[SL * vw + j] * (1.f / (float)DK);
                        mob_left(mm, ka[j], x.W.x, ut);
                        if ((j & 3) == 3 || j == SL - 1) rescale4(mm);
                    }
                    if (lane == 0) segA[vw * DK] = make_float4(mm[0], mm[1], mm[2], mm[3]);
                    if (vact) *reinterpret_cast<float2*>(segG + vw * DK + ch) = make_float2(g0, g1);
                }
            };
            if (vwork) {
                if (Lw < SL) summary(std::true_type());  // a partial last chunk only
                else summary(std::false_type());
                // r of the next chunk, written to LDS at the end of the iteration (past the end
                // of the sequence the value is never used)
                if (tid < C) in.rr = Raw1<TI>::load(sr.r, (c0n + (uint32_t)tid) * sr.rowh + sr.lane_h);
            }
            __syncthreads();

            // ---- phases B, C, D: the carry into the segment, then the replay in thirds -----
            // variance chain state (n, d) per channel (one per head for the isotropic variant)
            // and the decay since the chunk start, carried from third to third
            float n0 = 0.f, d0 = 1.f, n1 = 0.f, d1 = 1.f, g0 = 1.f, g1 = 1.f;
            float pb0[SL], pb1[SL];
            auto replay_mk = [&](auto ja_c, auto jb_c, auto mk_c) {
                constexpr int JA = decltype(ja_c)::value, JB = decltype(jb_c)::value;
                constexpr bool MK = decltype(mk_c)::value;
#pragma unroll
                for (int j = JA; j < JB; ++j) {
                    const int t = SL * vw + j;
                    const TokIn x = tok_in<MK>(in, j, Lw);
                    const float2 K = x.K, Q = x.Q, A = x.A;
                    g0 *= A.x;
                    g1 *= A.y;
                    if constexpr (DIAG) {
                        const float mr = s_mrv[t];
                        const float nn0 = fmaf(A.x * A.x, n0, x.W.x * d0);  // p_hat d
                        const float nn1 = fmaf(A.y * A.y, n1, x.W.y * d1);
                        pb0[j] = nn0 * K.x * __builtin_amdgcn_rcpf(d0 * g0);  // p_hat k / gamma
                        pb1[j] = nn1 * K.y * __builtin_amdgcn_rcpf(d1 * g1);
                        d0 = fmaf(K.x * K.x * mr, nn0, d0);
                        d1 = fmaf(K.y * K.y * mr, nn1, d1);
                        n0 = nn0;
                        n1 = nn1;
                        if ((j & 3) == 3 || j == SL - 1) {
                            rescale2(n0, d0);
                            rescale2(n1, d1);
                        }
                    } else {
                        const float nn = fmaf(ka[j], n0, x.W.x * d0);  // b_hat d
                        const float beta = nn / fmaf(d0, s_rv[t], nn * kn[j]);
                        pb0[j] = beta * K.x * __builtin_amdgcn_rcpf(g0);
                        pb1[j] = beta * K.y * __builtin_amdgcn_rcpf(g1);
                        d0 = fmaf(kn[j] * s_mrv[t] * (1.f / (float)DK), nn, d0);
                        n0 = nn;
                        if ((j & 3) == 3 || j == SL - 1) rescale2(n0, d0);
                    }
                    if (vact) {
                        st2<MT>(Kb + t * LDK + ch, g0 * K.x, g1 * K.y);
                        st2<MT>(Qb + t * LDK + ch, g0 * Q.x, g1 * Q.y);  // scale: applied to O
                        st2<MT>(Pb + t * LDK + ch, pb0[j], pb1[j]);
                    }
                }
            };
            // tokens [JA, JB) of the segment; the masked form only in a partial last chunk
            auto replay = [&](auto ja_c, auto jb_c) {
                if (Lw < SL) replay_mk(ja_c, jb_c, std::true_type());
                else replay_mk(ja_c, jb_c, std::false_type());
            };
            using J0 = std::integral_constant<int, 0>;
            using J1 = std::integral_constant<int, CF::JT1>;
            using J2 = std::integral_constant<int, CF::JT2>;
            using J3 = std::integral_constant<int, SL>;

            // ---- phase B: the carry into the segment, the first third of the replay --------
            if (vwork) {
                // the chunk carry through the earlier segments' summaries
                // (eq. chunk-gain-local-prefix)
                if constexpr (DIAG) {
                    float2 z0 = carry[pv * DK + ch], z1 = carry[pv * DK + ch + 1];
#pragma unroll
                    for (int ps = 0; ps < NVW - 1; ++ps) {
                        if (ps < vw) {
                            z0 = mat_vec(segA[ps * DK + ch], z0);
                            z1 = mat_vec(segA[ps * DK + ch + 1], z1);
                            const float2 gg = *reinterpret_cast<const float2*>(segG + ps * DK + ch);
                            g0 *= gg.x;
                            g1 *= gg.y;
                        }
                    }
                    n0 = z0.x; d0 = z0.y; n1 = z1.x; d1 = z1.y;
                } else {
                    float2 z = carry[pv * DK];
#pragma unroll
                    for (int ps = 0; ps < NVW - 1; ++ps) {
                        if (ps < vw) {
                            z = mat_vec(segA[ps * DK], z);
                            const float2 gg = *reinterpret_cast<const float2*>(segG + ps * DK + ch);
                            g0 *= gg.x;
                            g1 *= gg.y;
                        }
                    }
                    n0 = z.x; d0 = z.y;
                }
                replay(J0(), J1());
                load_part<0, CF::JT1, TI, CF>(in, sr, c0n, vw);
            }
            __syncthreads();

            // ---- phase C: the second third ---------------------------------------------------
            if (vwork) {
                replay(J1(), J2());
                load_part<CF::JT1, CF::JT2, TI, CF>(in, sr, c0n, vw);
            }
            __syncthreads();

            // ---- phase D: the last third; P_bar^T; the chunk's carry and decay --------------
            if (vwork) {
                replay(J2(), J3());
                if (vact) {
                    storeN<MT, (SL < 8 ? SL : 8)>(PbTv + ch * LDC + SL * vw, pb0);
                    storeN<MT, (SL < 8 ? SL : 8)>(PbTv + (ch + 1) * LDC + SL * vw, pb1);
                    if constexpr (SL > 8) {
                        storeN<MT, 8>(PbTv + ch * LDC + SL * vw + 8, pb0 + 8);
                        storeN<MT, 8>(PbTv + (ch + 1) * LDC + SL * vw + 8, pb1 + 8);
                    }
                }
                if (vw == NVW - 1) {  // the last segment closes the chunk
                    rescale2(n0, d0);
                    if constexpr (DIAG) {
                        rescale2(n1, d1);
                        if (vact) {
                            carry[(pv ^ 1) * DK + ch] = make_float2(n0, d0);
                            carry[(pv ^ 1) * DK + ch + 1] = make_float2(n1, d1);
                            if (vlast && a.P_T && vt == 0)  // the final variances n / d
                                *reinterpret_cast<float2*>(a.P_T + (size_t)nh * DK + ch) =
                                    make_float2(n0 / d0, n1 / d1);
                        }
                    } else if (lane == 0) {
                        carry[(pv ^ 1) * DK] = make_float2(n0, d0);
                        if (vlast && a.P_T && vt == 0) a.P_T[nh] = n0 / d0;
                    }
                    if (vact) *reinterpret_cast<float2*>(gC + pv * DK + ch) = make_float2(g0, g1);
                }
                load_part<CF::JT2, SL, TI, CF>(in, sr, c0n, vw);
                if (!vlast) {
                    if (tid < C) {  // r and mu / r of the next chunk
                        const float rv = Raw1<TI>::f32(in.rr);
                        const bool ok = tid < t1 - (int)c0n;
                        s_r[(pv ^ 1) * C + tid] = ok ? rv : 1.f;
                        s_mr[(pv ^ 1) * C + tid] = ok ? a.mu / rv : 0.f;
                    }
                }
            }
            __syncthreads();
        }
    } else {
        // ===== matrix waves: chunk it - 1; wave mw owns row blocks mw, mw + 4, ... ===========
        for (int it = 0; it <= nch; ++it) {
            const int m = it - 1;
            const bool mwork = m >= 0;
            const int pm = m & 1;
            const int c0m = t0 + m * C, Lm = min(C, t1 - c0m);
            const float* s_rm = s_r + pm * C;
            MT* PbTm = PbT0 + (size_t)pm * DK * LDC;

            // ---- phase A: the previous chunk's O rows; per owned row block: L and A_qk, and
            // X = V - K_bar S (to LDS, transposed) with Q_bar S kept for the output -----------
            if (mwork) {
                // one block pair (ib, jb) of L and A_qk from the row block's K_bar and Q_bar
                // fragments
                auto lq_unit = [&](int ib, int jb, const typename FK::V* kf,
                                   const typename FK::V* qf) {
                    // all fragments are read before the products (fixed by a scheduling barrier),
                    // so their LDS latency overlaps instead of being paid step by step
                    typename FK::V pf[FK::NS];
#pragma unroll
                    for (int s = 0; s < FK::NS; ++s)
                        pf[s] = FK::ld(Pb + (16 * jb + li) * LDK + FK::KF * s + (FK::KF / 4) * lg);
                    __builtin_amdgcn_sched_barrier(0);
                    floatx4 tacc = zero4(), qacc = zero4();
#pragma unroll
                    for (int s = 0; s < FK::NS; ++s) {
                        tacc = FK::mma(tacc, kf[s], pf[s]);
                        qacc = FK::mma(qacc, qf[s], pf[s]);
                    }
                    if (ib > jb) {
                        MT* lo = Lo + (ib * (ib - 1) / 2 + jb) * 16 * LDE;
#pragma unroll
                        for (int rr = 0; rr < 4; ++rr) {
                            const int row = 4 * lg + rr;
                            lo[row * LDE + li] = from_f32<MT>(tacc[rr]);
                            Aq[(16 * ib + row) * LDC + 16 * jb + li] = from_f32<MT>(qacc[rr]);
                        }
                    } else {
                        float* ld = Ld + ib * 16 * LDD;
#pragma unroll
                        for (int rr = 0; rr < 4; ++rr) {
                            const int row = 4 * lg + rr;
                            const float cdiag = DIAG ? s_rm[16 * ib + row] + tacc[rr] : 1.f;
                            ld[row * LDD + li] = row > li ? tacc[rr] : (row == li ? cdiag : 0.f);
                            Aq[(16 * ib + row) * LDC + 16 * jb + li] =
                                from_f32<MT>(row >= li ? qacc[rr] : 0.f);
                        }
                    }
                };
                // with four row blocks, wave 0 also takes the first two pairs of row block 3,
                // so no wave has more than three
                constexpr bool SHIFT = NB == 4 && NMW == 4;
                if (SHIFT && mw == 0) {
                    typename FK::V kf[FK::NS], qf[FK::NS];
#pragma unroll
                    for (int s = 0; s < FK::NS; ++s) {
                        const int k0 = FK::KF * s + (FK::KF / 4) * lg;
                        kf[s] = FK::ld(Kb + (16 * 3 + li) * LDK + k0);
                        qf[s] = FK::ld(Qb + (16 * 3 + li) * LDK + k0);
                    }
                    lq_unit(3, 0, kf, qf);
                    lq_unit(3, 1, kf, qf);
                }
#pragma unroll
                for (int rw = 0; rw < CF::RPW; ++rw) {
                    const int ib = mw + NMW * rw;
                    if (ib < NB) {
                        typename FK::V kf[FK::NS], qf[FK::NS];
#pragma unroll
                        for (int s = 0; s < FK::NS; ++s) {
                            const int k0 = FK::KF * s + (FK::KF / 4) * lg;
                            kf[s] = FK::ld(Kb + (16 * ib + li) * LDK + k0);
                            qf[s] = FK::ld(Qb + (16 * ib + li) * LDK + k0);
                        }
                        for (int jb = SHIFT && ib == 3 ? 2 : 0; jb <= ib; ++jb)
                            lq_unit(ib, jb, kf, qf);
                        // the S fragments of every column tile are read before the products
                        typename FK::V sf[CF::NNT][FK::NS];
#pragma unroll
                        for (int nt = 0; nt < CF::NNT; ++nt)
#pragma unroll
                            for (int s = 0; s < FK::NS; ++s)
                                sf[nt][s] = FK::ld(SmT + (16 * nt + li) * LDK + FK::KF * s +
                                                   (FK::KF / 4) * lg);
                        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                        for (int nt = 0; nt < CF::NNT; ++nt) {
                            const int j = rw * CF::NNT + nt;
                            floatx4 xacc = zero4();
                            Oacc[j] = zero4();
#pragma unroll
                            for (int s = 0; s < FK::NS; ++s) {
                                xacc = FK::mma(xacc, kf[s], sf[nt][s]);
                                Oacc[j] = FK::mma(Oacc[j], qf[s], sf[nt][s]);
                            }
                            float xv[4];
#pragma unroll
                            for (int rr = 0; rr < 4; ++rr) {
                                const int t = 16 * ib + 4 * lg + rr;
                                xv[rr] = (t < Lm ? Raw1<TI>::f32(vv[j][rr]) : 0.f) - xacc[rr];
                            }
                            store4<MT>(XT + (16 * nt + li) * LDC + 16 * ib + 4 * lg, xv[0],
                                       xv[1], xv[2], xv[3]);
                        }
                    }
                }
                load_v<TI, CF>(vv, sr, (uint32_t)(c0m + C), mw, lane);  // unused past the end
            }
            __syncthreads();

            // ---- phase B: the diagonal blocks of L^-1 (wave 0); the previous chunk's O rows
            // (the other matrix waves) ------------------------------------------------------
            if (mwork && mw >= 1 && m >= 1) {  // a full chunk: only the last one can be partial
                constexpr int VE = 16 / (int)sizeof(TI), VPR = BV / VE;
                const int c0p = c0m - C;
#pragma unroll 1
                for (int idx = mtid - 64; idx < C * VPR; idx += 64 * (NMW - 1)) {
                    const int t = idx / VPR, e = (idx % VPR) * VE;
                    *reinterpret_cast<uint4*>(go + ((size_t)(c0p + t) * H + h) * DV + col0 + e) =
                        *reinterpret_cast<const uint4*>(Ost + t * LDO + e);
                }
            }
            // Row i of A_bb = L_bb^-1 solves a^T L_bb = e_i^T: a_i = 1 / L_ii, and going down
            // the rows m = i, i-1, ..., 0 every finished a_m adds a_m L_m,k to the sums of the
            // k < m (right-looking backward substitution; the next row of L is read while the
            // current one is used). Lane (b, i) takes row i of block b.
            if (mwork && mw == 0 && (lane >> 4) < NB) {
                const int b = lane >> 4, i = li;
                const float* Lb = Ld + b * 16 * LDD;
                float sacc[16], y[16], row[2][16];
#pragma unroll
                for (int kq = 0; kq < 16; ++kq) sacc[kq] = 0.f;
#pragma unroll
                for (int v4 = 0; v4 < 4; ++v4) {
                    const float4 q4 = *reinterpret_cast<const float4*>(Lb + 15 * LDD + 4 * v4);
                    row[1][4 * v4] = q4.x; row[1][4 * v4 + 1] = q4.y;
                    row[1][4 * v4 + 2] = q4.z; row[1][4 * v4 + 3] = q4.w;
                }
#pragma unroll
                for (int mq = 15; mq >= 0; --mq) {
                    float* cur = row[mq & 1];
                    if (mq > 0) {
                        float* nx = row[(mq - 1) & 1];
#pragma unroll
                        for (int v4 = 0; v4 < (mq + 3) / 4; ++v4) {
                            const float4 q4 =
                                *reinterpret_cast<const float4*>(Lb + (mq - 1) * LDD + 4 * v4);
                            nx[4 * v4] = q4.x; nx[4 * v4 + 1] = q4.y;
                            nx[4 * v4 + 2] = q4.z; nx[4 * v4 + 3] = q4.w;
                        }
                    }
                    const float ym =
                        ((mq == i ? 1.f : 0.f) - sacc[mq]) * __builtin_amdgcn_rcpf(cur[mq]);
                    y[mq] = mq > i ? 0.f : ym;
#pragma unroll
                    for (int kq = 0; kq < mq; ++kq) sacc[kq] = fmaf(y[mq], cur[kq], sacc[kq]);
                }
                store8<MT>(Ai + (b * 16 + i) * LDE, y);
                store8<MT>(Ai + (b * 16 + i) * LDE + 8, y + 8);
            }
            __syncthreads();

            // ---- phase C: R = L^-1 X by block forward substitution ------------------------
            // One wave per 16-column tile of the value block: R_b = A_bb (X_b - sum_{c<b} L_bc
            // R_c). The chain stays in registers (a result tile is the B fragment of the next
            // product); R^T goes to LDS.
            if (mwork && mw < CF::NNT) {
                const int nt = mw;
                typename G::V ad[NB], lo[CF::NOFF];
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    ad[b] = G::ld(Ai + (b * 16 + li) * LDE + 4 * lg);
#pragma unroll
                    for (int c = 0; c < b; ++c) {
                        const int idx = b * (b - 1) / 2 + c;
                        lo[idx] = G::ld(Lo + (idx * 16 + li) * LDE + 4 * lg);
                    }
                }
                floatx4 Rr[NB];
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    floatx4 acc = zero4();
#pragma unroll
                    for (int c = 0; c < b; ++c)
                        acc = G::mma(acc, lo[b * (b - 1) / 2 + c],
                                     G::pack(Rr[c][0], Rr[c][1], Rr[c][2], Rr[c][3]));
                    const float4 xb = ld4f<MT>(XT + (16 * nt + li) * LDC + 16 * b + 4 * lg);
                    Rr[b] = G::mma(zero4(), ad[b],
                                   G::pack(xb.x - acc[0], xb.y - acc[1], xb.z - acc[2],
                                           xb.w - acc[3]));
                    store4<MT>(RT + (16 * nt + li) * LDC + 16 * b + 4 * lg, Rr[b][0], Rr[b][1],
                               Rr[b][2], Rr[b][3]);
                }
            }
            __syncthreads();

            // ---- phase D: O = Q_bar S + A_qk R (staged for the next iteration's stores) and
            // S <- gamma_C (.) (S + P_bar^T R) ------------------------------------------------
            if (mwork) {
                // every fragment of the phase is read before the products (fixed by a
                // scheduling barrier); the blocks of A_qk right of the diagonal are zero, so the
                // O tiles run the whole contraction
                typename FC::V rf[CF::NNT][FC::NS], af[CF::XPW][FC::NS], pf[CF::SPW][FC::NS];
#pragma unroll
                for (int nt = 0; nt < CF::NNT; ++nt)
#pragma unroll
                    for (int s = 0; s < FC::NS; ++s)
                        rf[nt][s] = FC::ld(RT + (16 * nt + li) * LDC + FC::KF * s + (FC::KF / 4) * lg);
#pragma unroll
                for (int j = 0; j < CF::XPW; ++j) {
                    const int ib = min(mw + NMW * (j / CF::NNT), NB - 1);
#pragma unroll
                    for (int s = 0; s < FC::NS; ++s)
                        af[j][s] = FC::ld(Aq + (16 * ib + li) * LDC + FC::KF * s + (FC::KF / 4) * lg);
                }
#pragma unroll
                for (int j = 0; j < CF::SPW; ++j) {
                    const int ik = min(mw + NMW * j, CF::NST - 1) % CF::NKT;
#pragma unroll
                    for (int s = 0; s < FC::NS; ++s)
                        pf[j][s] =
                            FC::ld(PbTm + (16 * ik + li) * LDC + FC::KF * s + (FC::KF / 4) * lg);
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int j = 0; j < CF::XPW; ++j) {
                    const int ib = mw + NMW * (j / CF::NNT), nt = j % CF::NNT;
                    if (ib < NB) {
#pragma unroll
                        for (int s = 0; s < FC::NS; ++s)
                            Oacc[j] = FC::mma(Oacc[j], af[j][s], rf[nt][s]);
#pragma unroll
                        for (int rr = 0; rr < 4; ++rr)
                            Ost[(16 * ib + 4 * lg + rr) * LDO + 16 * nt + li] =
                                from_f32<TI>(a.scale * Oacc[j][rr]);
                    }
                }
#pragma unroll
                for (int j = 0; j < CF::SPW; ++j) {
                    const int x = mw + NMW * j;
                    if (x < CF::NST) {
                        const int ik = x % CF::NKT, nt = x / CF::NKT;
                        // with NKT a multiple of NMW the column tile depends on j alone
                        constexpr bool NTS = CF::NKT % NMW == 0;
                        const int ntr = NTS ? NMW * j / CF::NKT : nt;
#pragma unroll
                        for (int s = 0; s < FC::NS; ++s)
                            Sacc[j] = FC::mma(Sacc[j], pf[j][s],
                                              ntr == 0 ? rf[0][s] : rf[CF::NNT - 1][s]);
                        const float4 gc =
                            *reinterpret_cast<const float4*>(gC + pm * DK + 16 * ik + 4 * lg);
                        Sacc[j][0] *= gc.x;
                        Sacc[j][1] *= gc.y;
                        Sacc[j][2] *= gc.z;
                        Sacc[j][3] *= gc.w;
                        store4<MT>(SmT + (16 * nt + li) * LDK + 16 * ik + 4 * lg, Sacc[j][0],
                                   Sacc[j][1], Sacc[j][2], Sacc[j][3]);
                    }
                }
            }
            __syncthreads();
        }

        if (nch > 0) {  // the last chunk's O rows
            constexpr int VE = 16 / (int)sizeof(TI), VPR = BV / VE;
            const int c0p = t0 + (nch - 1) * C, Lp = t1 - c0p;
#pragma unroll 1
            for (int idx = mtid; idx < C * VPR; idx += 64 * NMW) {
                const int t = idx / VPR, e = (idx % VPR) * VE;
                if (t < Lp)
                    *reinterpret_cast<uint4*>(go + ((size_t)(c0p + t) * H + h) * DV + col0 + e) =
                        *reinterpret_cast<const uint4*>(Ost + t * LDO + e);
            }
        }
        if (a.S_T) {
            float* dst = a.S_T + (size_t)nh * DK * DV;
#pragma unroll
            for (int j = 0; j < CF::SPW; ++j) {
                const int x = mw + NMW * j;
                if (x < CF::NST) {
                    const int ik = x % CF::NKT, nt = x / CF::NKT;
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr)
                        dst[(size_t)(16 * ik + 4 * lg + rr) * DV + col0 + 16 * nt + li] =
                            Sacc[j][rr];
                }
            }
        }
    }
}

// ------------------------------------------------------------------------------------------
// Packed batches: the sequences in the order they are walked, longest first (a rank sort in
// one workgroup; larger batches keep their own order).
// ------------------------------------------------------------------------------------------
constexpr int ORDER_MAX = 4096;

__global__ __launch_bounds__(1024) void order_kernel(const int32_t* __restrict__ cu, int N,
                                                     int32_t* __restrict__ order)
{
    __shared__ int32_t len[ORDER_MAX];
    for (int i = threadIdx.x; i < N; i += blockDim.x) len[i] = max(0, cu[i + 1] - cu[i]);
    __syncthreads();
    for (int i = threadIdx.x; i < N; i += blockDim.x) {
        const int li = len[i];
        int rank = 0;
        for (int j = 0; j < N; ++j) {
            const int lj = len[j];
            rank += (lj > li) || (lj == li && j < i);
        }
        order[rank] = i;
    }
}

__global__ void copy_floats_kernel(const float* __restrict__ src, float* __restrict__ dst,
                                   size_t n)
{
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x)
        dst[i] = src[i];
}

// ------------------------------------------------------------------------------------------
// host side
// ------------------------------------------------------------------------------------------
template <class TI, int DK, int DV, int C>
constexpr bool walk_fits()
{
    constexpr int BV = DV >= 32 ? 32 : DV;
    return WalkCfg<TI, DK, DV, BV, C, 0, true>::TOTAL <= 160 * 1024 &&
           WalkCfg<TI, DK, DV, BV, C, 1, false>::TOTAL <= 160 * 1024;
}

// Workspace: the walk order of a packed batch (int32 [N]) and, when the caller updates P in
// place (P_T == P0), a copy of P0 that every value tile of a head reads at its start while the
// first tile to finish may already have written P_T.
struct WsMap {
    size_t order, p0, total;
};

inline WsMap ws_map(int variant, bool packed, int N, int H, int dk)
{
    WsMap m;
    m.order = 0;
    m.p0 = packed ? al256((size_t)N * 4) : 0;
    m.total = m.p0 + al256((size_t)N * H * (variant == 0 ? dk : 1) * 4);
    return m;
}

template <class TI, int DK, int DV, int C, int VARIANT, bool APC>
hipError_t run_t(const FwdCall& fc, hipStream_t st)
{
    constexpr int BV = DV >= 32 ? 32 : DV;
    using CF = WalkCfg<TI, DK, DV, BV, C, VARIANT, APC>;
    static std::atomic<bool> attr_done{false};
    hipError_t e;
    if (!attr_done.load()) {
        if ((e = hipFuncSetAttribute((const void*)walk_kernel<TI, CF>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)CF::TOTAL)) != hipSuccess)
            return e;
        attr_done.store(true);
    }
    const SeqArgs& sa = fc.sa;
    const bool packed = sa.cu_seqlens != nullptr;
    const WsMap wm = ws_map(VARIANT, packed, sa.N, sa.H, DK);
    char* ws = (char*)fc.workspace;
    WalkArgs a;
    a.q = fc.q; a.k = fc.k; a.v = fc.v; a.alpha = fc.alpha; a.omega = fc.omega; a.r = fc.r;
    a.S0 = fc.S0; a.P0 = fc.P0; a.o = fc.o; a.S_T = fc.S_T; a.P_T = fc.P_T;
    a.cu = sa.cu_seqlens; a.order = nullptr;
    a.N = sa.N; a.T = sa.T; a.H = sa.H; a.mu = fc.mu; a.scale = fc.scale;
    const size_t ntok = (size_t)sa.B * sa.T * sa.H;
    a.bytes_k = (uint32_t)(ntok * DK * sizeof(TI));
    a.bytes_v = (uint32_t)(ntok * DV * sizeof(TI));
    a.bytes_h = (uint32_t)(ntok * sizeof(TI));
    if (packed && sa.N <= ORDER_MAX) {
        int32_t* order = (int32_t*)(ws + wm.order);
        hipLaunchKernelGGL(order_kernel, dim3(1), dim3(1024), 0, st, sa.cu_seqlens, sa.N, order);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        a.order = order;
    }
    if (fc.P0 && fc.P_T == fc.P0) {
        float* p0 = (float*)(ws + wm.p0);
        const size_t np = (size_t)sa.N * sa.H * (VARIANT == 0 ? DK : 1);
        hipLaunchKernelGGL(copy_floats_kernel, dim3((unsigned)std::min<size_t>((np + 255) / 256, 1024)),
                           dim3(256), 0, st, fc.P0, p0, np);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        a.P0 = p0;
    }
    const size_t nh8 = ((size_t)sa.N * sa.H + 7) / 8 * 8;
    const size_t nblk = nh8 * CF::NV;
    if (nblk == 0) return hipSuccess;
    hipLaunchKernelGGL((walk_kernel<TI, CF>), dim3((unsigned)nblk), dim3(NTH), CF::TOTAL, st, a);
    return hipGetLastError();
}

template <class TI, int DK, int DV, int C>
hipError_t run_variant(const FwdCall& fc, hipStream_t st)
{
    if constexpr (!walk_fits<TI, DK, DV, C>()) {
        return hipErrorInvalidConfiguration;
    } else {
        if (fc.variant == 0) return run_t<TI, DK, DV, C, 0, true>(fc, st);
        if (fc.apc) return run_t<TI, DK, DV, C, 1, true>(fc, st);
        return run_t<TI, DK, DV, C, 1, false>(fc, st);
    }
}

// Compile-time dispatch over (dtype, dk, dv, chunk) calling F::template go<TI, DK, DV, C>().
template <class F>
auto dispatch(kdn_dtype_t dtype, int dk, int dv, int chunk, F f)
    -> decltype(f.template go<float, 16, 16, 16>())
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
    template <class TI, int DK, int DV, int C> bool go() const { return walk_fits<TI, DK, DV, C>(); }
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
    (void)B; (void)T; (void)dv; (void)dtype; (void)chunk;
    return ws_map(variant, packed, N, H, dk).total;
}

hipError_t launch_chunked(const FwdCall& fc, hipStream_t stream)
{
    FwdCall c = fc;
    if (c.chunk == 0) c.chunk = chunked_default_chunk(c.dtype, c.dk, c.dv);
    return dispatch(c.dtype, c.dk, c.dv, c.chunk, RunF{&c, stream});
}

}  // namespace kdn
