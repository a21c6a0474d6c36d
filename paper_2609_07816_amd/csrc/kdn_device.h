// Device helpers shared by the chunked forward kernels of libkdn (summary, prep and walk):
// MFMA fragments over LDS tiles, small vector loads and stores in operand precision, buffer
// loads with whole-tensor descriptors, power-of-two rescaling of the variance chain, and the
// chunk geometry of fixed-length and packed batches.
#pragma once

#include <type_traits>

#include "kdn_internal.h"

namespace kdn {

constexpr size_t al16(size_t x) { return (x + 15) & ~(size_t)15; }
constexpr size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }
constexpr size_t cmax(size_t a, size_t b) { return a > b ? a : b; }

// Operand precision of the dense products: bf16 for bf16 inputs, float32 for float32 inputs.
template <class TI> struct OpOf { using type = bf16; };
template <> struct OpOf<float> { using type = float; };

__device__ __forceinline__ floatx4 zero4()
{
    floatx4 z = {0.f, 0.f, 0.f, 0.f};
    return z;
}

// ------------------------------------------------------------------------------------------
// MFMA fragments read from memory: lane (g, i) = (lane / 16, lane % 16) holds KF/4 consecutive
// k values of row i (A side) or of column i (B side, stored transposed). One fragment feeds one
// bf16 MFMA (KF = 32 or 16) or four float32 MFMAs (KF = 16). Both sides use the same k
// assignment, so the contraction is exact whatever order the unit applies internally.
// Result tile: acc[r] = D[4 g + r][i].
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
    // x <- x (.) s elementwise for the KF/4 k values of a fragment (s: KF/4 floats)
    __device__ static V scale(V x, const float* s)
    {
        constexpr int E = KF / 4;
        bf16 v[E];
        __builtin_memcpy(v, &x, sizeof(V));
#pragma unroll
        for (int e = 0; e < E; ++e) v[e] = (bf16)((float)v[e] * s[e]);
        V y;
        __builtin_memcpy(&y, v, sizeof(V));
        return y;
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
    __device__ static V scale(V x, const float* s)
    {
        return make_uint4(__float_as_uint(__uint_as_float(x.x) * s[0]),
                          __float_as_uint(__uint_as_float(x.y) * s[1]),
                          __float_as_uint(__uint_as_float(x.z) * s[2]),
                          __float_as_uint(__uint_as_float(x.w) * s[3]));
    }
};

// 16 x 16 x 16 float32 products from register fragments: lane (g, i) holds A[i][4g..4g+3]
// (A side) or B[4g..4g+3][i] (B side). A result tile (lane (g, i): rows 4g..4g+3 of column i)
// is therefore already a B fragment of the next product.
__device__ __forceinline__ floatx4 mma16_f32(floatx4 acc, float4 a, floatx4 b)
{
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b[0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b[1], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b[2], acc, 0, 0, 0);
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b[3], acc, 0, 0, 0);
}

// ------------------------------------------------------------------------------------------
// small vector stores and loads in operand precision
// ------------------------------------------------------------------------------------------
template <class MT>
__device__ __forceinline__ void st2(MT* p, float x, float y)
{
    if constexpr (std::is_same<MT, float>::value) {
        *reinterpret_cast<float2*>(p) = make_float2(x, y);
    } else {
        bf16x4 v;  // only the first two lanes are stored
        v[0] = (bf16)x;
        v[1] = (bf16)y;
        *reinterpret_cast<unsigned*>(p) = *reinterpret_cast<const unsigned*>(&v);
    }
}

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

template <class MT>
__device__ __forceinline__ void store8(MT* dst, const float* x)
{
    if constexpr (std::is_same<MT, float>::value) {
        *reinterpret_cast<float4*>(dst) = make_float4(x[0], x[1], x[2], x[3]);
        *reinterpret_cast<float4*>(dst + 4) = make_float4(x[4], x[5], x[6], x[7]);
    } else {
        bf16x8 v;
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = (bf16)x[j];
        *reinterpret_cast<bf16x8*>(dst) = v;
    }
}

// Two adjacent inputs from one raw word (bf16 pair) or a float pair.
__device__ __forceinline__ float2 unpack2(unsigned u)
{
    return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xFFFF0000u));
}
__device__ __forceinline__ float2 unpack2(float2 v) { return v; }

// ------------------------------------------------------------------------------------------
// variance chain: homogeneous pairs z = (n, d), p = n / d, and 2x2 Moebius matrices
// ------------------------------------------------------------------------------------------

// Power-of-two rescale of non-negative homogeneous values: exact, keeps every ratio, brings the
// largest entry into [0.5, 1). The exponent instruction gives 0 for 0, Inf and NaN, which
// leaves such values unchanged.
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

// z <- M z for M = [x y; z w] (float4) acting on a homogeneous pair, rescaled.
__device__ __forceinline__ float2 mat_vec(const float4& m, float2 v)
{
    float n = fmaf(m.x, v.x, m.y * v.y), d = fmaf(m.z, v.x, m.w * v.y);
    rescale2(n, d);
    return make_float2(n, d);
}

// m <- M_t m for the token matrix M_t = [[a, w], [u a, 1 + u w]] (m row-major [m00 m01 m10 m11]);
// the second row uses M_t's structure: row1 = u * row0' + row1.
__device__ __forceinline__ void mob_left(float* m, float a, float w, float u)
{
    const float r00 = fmaf(a, m[0], w * m[2]), r01 = fmaf(a, m[1], w * m[3]);
    m[2] = fmaf(u, r00, m[2]);
    m[3] = fmaf(u, r01, m[3]);
    m[0] = r00;
    m[1] = r01;
}

// x * y for 2x2 matrices (row-major float4), rescaled.
__device__ __forceinline__ float4 mat_mul(const float4& x, const float4& y)
{
    float m[4] = {fmaf(x.x, y.x, x.y * y.z), fmaf(x.x, y.y, x.y * y.w),
                  fmaf(x.z, y.x, x.w * y.z), fmaf(x.z, y.y, x.w * y.w)};
    rescale4(m);
    return make_float4(m[0], m[1], m[2], m[3]);
}

// 1 / x for a non-negative decay product, saturated to 2^126 (x = 0 after an underflow gives
// 2^126, not Inf).
__device__ __forceinline__ float sat_rcp(float x)
{
    return __builtin_amdgcn_rcpf(fmaxf(x, 0x1p-126f));
}

// ------------------------------------------------------------------------------------------
// Buffer loads: 32-bit byte offsets against a descriptor of the whole tensor. The unit checks
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

// ------------------------------------------------------------------------------------------
// Chunk geometry. Tokens are flat indices over B*T. Sequence n owns [t0, t1): n*T.. for a
// fixed-length batch, [cu[n], cu[n+1]) for a packed one, clamped to [0, ntok] so that a broken
// cu_seqlens can never send a kernel outside the caller's buffers. Chunks of CH tokens restart
// at every sequence start; global chunk g of a packed batch is found through the chunk-offset
// table choff (choff[n] = chunks of the sequences before n, capped at maxch).
// ------------------------------------------------------------------------------------------
struct ChunkMap {
    const int32_t* cu;     // device, or nullptr (fixed length)
    const int32_t* choff;  // device [N + 1] (packed), or nullptr
    int N, T, ntok, maxch;
};

__device__ __forceinline__ void seq_span(const ChunkMap& cm, int n, int& t0, int& t1)
{
    if (cm.cu) {
        t0 = min(max(cm.cu[n], 0), cm.ntok);
        t1 = min(max(cm.cu[n + 1], t0), cm.ntok);
    } else {
        t0 = n * cm.T;
        t1 = t0 + cm.T;
    }
}

// First global chunk of sequence n and its chunk count (capped so g0 + count <= maxch).
template <int CH>
__device__ __forceinline__ void seq_chunks(const ChunkMap& cm, int n, int t0, int t1, int& g0,
                                           int& nch)
{
    nch = (t1 - t0 + CH - 1) / CH;
    g0 = cm.cu ? cm.choff[n] : n * ((cm.T + CH - 1) / CH);
    nch = max(0, min(nch, cm.maxch - g0));
}

// Global chunk g -> sequence n, token range [c0, c1) and whether it ends its sequence.
template <int CH>
__device__ __forceinline__ bool locate_chunk(const ChunkMap& cm, int g, int& n, int& c0, int& c1,
                                             bool& last)
{
    if (g >= cm.maxch) return false;
    int m;
    if (!cm.cu) {
        const int ncs = (cm.T + CH - 1) / CH;
        n = g / ncs;
        if (n >= cm.N) return false;
        m = g - n * ncs;
    } else {
        if (g >= cm.choff[cm.N]) return false;
        int lo = 0, hi = cm.N - 1;  // largest n with choff[n] <= g
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (cm.choff[mid] <= g) lo = mid; else hi = mid - 1;
        }
        n = lo;
        m = g - cm.choff[n];
    }
    int t0, t1;
    seq_span(cm, n, t0, t1);
    c0 = t0 + m * CH;
    c1 = min(c0 + CH, t1);
    last = (c1 == t1);
    return c0 < c1;
}

// Host launchers shared by the forward and the gain scan (kdn_scan.hip).
// Chunk-offset table of a packed batch: choff[n] = sum_{m < n} ceil(len_m / ch), capped at maxch
// (the workspace is sized for maxch chunks; a valid cu_seqlens never reaches the cap).
hipError_t launch_chunk_table(const int32_t* cu, int N, int ntok, int ch, int maxch,
                              int32_t* choff, hipStream_t st);
// Exclusive carries of the variance chain across the chunks of every (sequence, head, channel)
// as a log-depth (Kogge-Stone) scan of the chunk summaries summ [maxch][H][nchan]; carry has the
// same layout. Empty sequences get P_T = P0 (P_T may be NULL).
hipError_t launch_carry_scan(const float4* summ, const float* P0, const ChunkMap& cm, int ch,
                             int H, int nchan, float2* carry, float* P_T, hipStream_t st);
// Sequences of a packed batch in walking order, longest first (N <= 4096; else in order).
hipError_t launch_order(const int32_t* cu, int N, int ntok, int32_t* order, hipStream_t st);
constexpr int ORDER_MAX = 4096;

}  // namespace kdn
