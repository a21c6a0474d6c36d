// Device helpers shared by the HIP sources of libkdn: MFMA fragment products over LDS tiles,
// small vector loads and stores in operand precision, and sequence ranges.
#pragma once

#include <type_traits>

#include "kdn_internal.h"

namespace kdn {

// ------------------------------------------------------------------------------------------
// MFMA helpers. Lane l = 16 g + i (i = l % 16, g = l / 16). A 16 x 16 result tile is held as
// acc[r] = D[4 g + r][i]. A operand rows and B operand columns are indexed by i; every lane of
// group g contracts the same k indices on both sides, so the sum over k is exact whatever order
// the unit applies internally.
// ------------------------------------------------------------------------------------------

// acc += A[16 x K] * B[K x 16]; A row-major (k contiguous, lda), B given transposed as
// BT[16][K] (k contiguous, ldb).
template <class MT, int K>
__device__ __forceinline__ floatx4 mm_kc(const MT* A, int lda, const MT* BT, int ldb,
                                         floatx4 acc, int lane)
{
    const int i = lane & 15, g = lane >> 4;
    if constexpr (std::is_same<MT, float>::value) {
#pragma unroll
        for (int ks = 0; ks < K / 4; ++ks)
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A[i * lda + 4 * ks + g],
                                                        BT[i * ldb + 4 * ks + g], acc, 0, 0, 0);
    } else if constexpr (K % 32 == 0) {
#pragma unroll
        for (int ks = 0; ks < K / 32; ++ks) {
            const bf16x8 a = *reinterpret_cast<const bf16x8*>(A + i * lda + 32 * ks + 8 * g);
            const bf16x8 b = *reinterpret_cast<const bf16x8*>(BT + i * ldb + 32 * ks + 8 * g);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
        }
    } else {
        static_assert(K == 16, "bf16 tiles contract over multiples of 16");
        const bf16x4 a = *reinterpret_cast<const bf16x4*>(A + i * lda + 4 * g);
        const bf16x4 b = *reinterpret_cast<const bf16x4*>(BT + i * ldb + 4 * g);
        acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, acc, 0, 0, 0);
    }
    return acc;
}

// acc1 += A1 * B and acc2 += A2 * B over K, sharing each B fragment (layouts as mm_kc).
template <class MT, int K>
__device__ __forceinline__ void mm_kc2(const MT* A1, const MT* A2, int lda, const MT* BT, int ldb,
                                       floatx4& acc1, floatx4& acc2, int lane)
{
    const int i = lane & 15, g = lane >> 4;
    if constexpr (std::is_same<MT, float>::value) {
#pragma unroll
        for (int ks = 0; ks < K / 4; ++ks) {
            const float b = BT[i * ldb + 4 * ks + g];
            acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(A1[i * lda + 4 * ks + g], b, acc1, 0, 0, 0);
            acc2 = __builtin_amdgcn_mfma_f32_16x16x4f32(A2[i * lda + 4 * ks + g], b, acc2, 0, 0, 0);
        }
    } else if constexpr (K % 32 == 0) {
#pragma unroll
        for (int ks = 0; ks < K / 32; ++ks) {
            const bf16x8 b = *reinterpret_cast<const bf16x8*>(BT + i * ldb + 32 * ks + 8 * g);
            const bf16x8 a1 = *reinterpret_cast<const bf16x8*>(A1 + i * lda + 32 * ks + 8 * g);
            const bf16x8 a2 = *reinterpret_cast<const bf16x8*>(A2 + i * lda + 32 * ks + 8 * g);
            acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b, acc1, 0, 0, 0);
            acc2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a2, b, acc2, 0, 0, 0);
        }
    } else {
        static_assert(K == 16, "bf16 tiles contract over multiples of 16");
        const bf16x4 b = *reinterpret_cast<const bf16x4*>(BT + i * ldb + 4 * g);
        const bf16x4 a1 = *reinterpret_cast<const bf16x4*>(A1 + i * lda + 4 * g);
        const bf16x4 a2 = *reinterpret_cast<const bf16x4*>(A2 + i * lda + 4 * g);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a1, b, acc1, 0, 0, 0);
        acc2 = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a2, b, acc2, 0, 0, 0);
    }
}

// acc += A[16 x 16] * B[16 x 16]; A float32 row-major (k contiguous), B given transposed as
// BT[16][16] in operand precision (k contiguous). Vector reads on both sides.
template <class MT>
__device__ __forceinline__ floatx4 mm16_tv(const float* A, int lda, const MT* BT, int ldb,
                                           floatx4 acc, int lane)
{
    const int i = lane & 15, g = lane >> 4;
    const float4 a4 = *reinterpret_cast<const float4*>(A + i * lda + 4 * g);
    if constexpr (std::is_same<MT, float>::value) {
        // fp32 MFMA contracts k = 4 ks + g per step; gather the matching elements
        const float av[4] = {A[i * lda + g], A[i * lda + 4 + g], A[i * lda + 8 + g],
                             A[i * lda + 12 + g]};
        (void)a4;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[ks], BT[i * ldb + 4 * ks + g], acc, 0,
                                                        0, 0);
    } else {
        bf16x4 a;
        a[0] = (bf16)a4.x; a[1] = (bf16)a4.y; a[2] = (bf16)a4.z; a[3] = (bf16)a4.w;
        const bf16x4 b = *reinterpret_cast<const bf16x4*>(BT + i * ldb + 4 * g);
        acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, acc, 0, 0, 0);
    }
    return acc;
}

// acc += A[16 x 16] * B[16 x 16] with A and B both row-major (A of type TA, converted).
template <class MT, class TA>
__device__ __forceinline__ floatx4 mm16_rr(const TA* A, int lda, const MT* B, int ldb,
                                           floatx4 acc, int lane)
{
    const int i = lane & 15, g = lane >> 4;
    if constexpr (std::is_same<MT, float>::value) {
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32((float)A[i * lda + 4 * ks + g],
                                                        B[(4 * ks + g) * ldb + i], acc, 0, 0, 0);
    } else {
        bf16x4 a, b;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            a[s] = (bf16)(float)A[i * lda + 4 * g + s];
            b[s] = B[(4 * g + s) * ldb + i];
        }
        acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, acc, 0, 0, 0);
    }
    return acc;
}

// Make this wave's LDS writes visible to its other lanes (LDS ops of one wave run in order).
__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

__device__ __forceinline__ floatx4 zero4()
{
    floatx4 z = {0.f, 0.f, 0.f, 0.f};
    return z;
}

// Token range [t0, t1) (flat index over B*T) of sequence n.
__device__ __forceinline__ void seq_range(const int32_t* cu, int n, int T, int& t0, int& t1)
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

// Two adjacent elements as floats (bf16 pair in one 32-bit word, or two floats).
__device__ __forceinline__ float2 ld2(const bf16* p)
{
    const unsigned u = *reinterpret_cast<const unsigned*>(p);
    return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xFFFF0000u));
}
__device__ __forceinline__ float2 ld2(const float* p) { return *reinterpret_cast<const float2*>(p); }

// Store two adjacent values in operand precision.
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

// Store 8 consecutive values (16-byte aligned destination).
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

}  // namespace kdn
