// Fused chunkwise forward of Diagonal / Isotropic KDN on gfx950.
//
// arXiv 2609.07816, App. "Hardware-Efficient Chunkwise Algorithm". With the gains kappa_t fixed,
// the memory recurrence S_t = (I - kappa_t k_t^T) diag(alpha_t) S_{t-1} + kappa_t v_t^T is
// evaluated chunk by chunk in compact-WY form (Sec. "Chunkwise Memory Scan"); only S^in crosses
// chunk boundaries. Inside a chunk of C tokens (local index r, cumulative decay
// gamma_r = prod_{j<=r} alpha_j):
//   K_bar = Gamma (.) K,   Q_bar = Gamma (.) Q,   P_bar = (p_hat (.) K) (/) Gamma
//   kappa_r / gamma_r = P_bar_r / den_r           with den_r = r_r + sum_i p_hat_ri k_ri^2
//   T   = tril(K_bar P_bar^T diag(1/den), -1),    A = (I + T)^-1
//   R   = A (V - K_bar S^in)
//   O   = scale (Q_bar S^in + tril(Q_bar P_bar^T diag(1/den)) R)
//   S^out = diag(gamma_C) (S^in + P_bar^T diag(1/den) R)
// This is the paper's W / U / K_tail form with the gain normalisation moved onto the small
// C x C and C x dv factors, so the per-channel operands need no extra pass. den_r itself is the
// diagonal of K_bar P_bar^T (gamma cancels), which the MFMA product already produces.
// For the isotropic variant P_bar = beta_r k_r / gamma_r and den = 1.
//
// The gains come from the variance chain, replayed inside the kernel one chunk at a time from
// the carried homogeneous state z = [n; d] (Moebius form, eq. diag-cov-scan): per token
//   n <- alpha^2 n + omega d,   p_hat = n / d_prev,   d <- u n + d   (u = mu k^2 / r),
// with an exact power-of-two rescale every second token.
//
// One workgroup (256 threads) owns one (sequence, head, dv tile of BV columns) and walks the
// sequence's chunks in order; the S tile stays in MFMA accumulator registers for the whole
// sequence. Dense products run on MFMA: bf16 operands with fp32 accumulation for bf16 inputs,
// fp32 MFMA for fp32 inputs. The workgroups of one head are spaced N*H apart in the grid so that
// the round-robin dispatch puts them on the same XCD, where they share the L2 copy of q, k,
// alpha and omega.
#include <type_traits>

#include "kdn_internal.h"

namespace kdn {
namespace {

constexpr int NT = 256;  // threads per workgroup (4 waves)

constexpr size_t al16(size_t x) { return (x + 15) & ~(size_t)15; }

template <class TI> struct OperandOf { using type = bf16; };
template <> struct OperandOf<float> { using type = float; };

template <class TI, int DK_, int BV_, int C_, int VARIANT_, bool APC_>
struct Cfg {
    using MT = typename OperandOf<TI>::type;  // MFMA operand type
    static constexpr int DK = DK_, BV = BV_, C = C_, VARIANT = VARIANT_;
    static constexpr bool APC = APC_ || VARIANT_ == 0;  // diagonal gates are per channel
    static constexpr int PAD = 16 / (int)sizeof(MT);    // one 16-byte pad per row
    static constexpr int LDK = DK + PAD;                // rows of [*][DK] operand tiles
    static constexpr int LDC = C + PAD;                 // rows of [*][C] operand tiles
    static constexpr int LDT = C + 4;                   // rows of the fp32 T matrix
    static constexpr int NB = C / 16;                   // 16x16 blocks per chunk side
    static constexpr int NMT = C / 16, NNT = BV / 16, NKT = DK / 16;
    static constexpr int NOUT = NMT * NNT;              // [C x BV] output tiles
    static constexpr int NST = NKT * NNT;               // [DK x BV] state tiles
    static constexpr int OUT_PER_WAVE = (NOUT + 3) / 4;
    static constexpr int ST_PER_WAVE = (NST + 3) / 4;
    static constexpr int LDI = 16 + PAD;                // inversion scratch rows

    // ---- LDS map (bytes). The first region holds the chunk's raw inputs while the operands
    // are formed and is then reused for the chunk's C x C and C x BV factors.
    static constexpr size_t RAWN = (size_t)C * DK;
    static constexpr size_t SZ_RAW = 4 * RAWN * sizeof(TI);  // alpha, k, omega, q
    static constexpr size_t OFF_TM = 0;                                   // float [C][LDT]
    static constexpr size_t OFF_AI = OFF_TM + al16((size_t)C * LDT * 4);  // MT [C][LDC]
    static constexpr size_t OFF_AQ = OFF_AI + al16((size_t)C * LDC * sizeof(MT));
    static constexpr size_t OFF_XT = OFF_AQ + al16((size_t)C * LDC * sizeof(MT));  // [BV][LDC]
    static constexpr size_t OFF_RT = OFF_XT + al16((size_t)BV * LDC * sizeof(MT));
    static constexpr size_t OFF_R2T = OFF_RT + al16((size_t)BV * LDC * sizeof(MT));
    static constexpr size_t OFF_INV = OFF_R2T + al16((size_t)BV * LDC * sizeof(MT));
    static constexpr size_t OFF_AIT = OFF_INV + al16((size_t)4 * 16 * LDI * sizeof(MT));  // [C][LDC]
    static constexpr size_t END_ALIAS = OFF_AIT + al16((size_t)C * LDC * sizeof(MT));
    static constexpr size_t SZ_R1 = al16(SZ_RAW > END_ALIAS ? SZ_RAW : END_ALIAS);
    static constexpr size_t OFF_V = SZ_R1;                                         // TI [C][BV]
    static constexpr size_t OFF_KB = OFF_V + al16((size_t)C * BV * sizeof(TI));    // MT [C][LDK]
    static constexpr size_t OFF_QB = OFF_KB + al16((size_t)C * LDK * sizeof(MT));
    static constexpr size_t OFF_PB = OFF_QB + al16((size_t)C * LDK * sizeof(MT));
    static constexpr size_t OFF_PBT = OFF_PB + al16((size_t)C * LDK * sizeof(MT)); // [DK][LDC]
    static constexpr size_t OFF_SMT = OFF_PBT + al16((size_t)DK * LDC * sizeof(MT)); // [BV][LDK]
    static constexpr size_t OFF_SC = OFF_SMT + al16((size_t)BV * LDK * sizeof(MT));
    // scalars: r[C], mr[C], rden[C], beta[C], gtok[C], gC[DK], wtok[C], atok[C]; then the
    // carried variance state z[DK][2] and the segment summaries M[NSEG-1][DK][4], G[NSEG-1][DK]
    static constexpr int NSEG = C / 16;                 // 16-token segments of the variance scan
    static constexpr size_t SZ_SC = (size_t)(7 * C + DK + 4 + 2 * DK + (NSEG - 1) * DK * 5) * 4;
    static constexpr size_t TOTAL = al16(OFF_SC + SZ_SC);  // checked by the launcher
};

struct FwdArgs {
    const void *q, *k, *v, *alpha, *omega, *r;
    const float *S0, *P0;
    void* o;
    float *S_T, *P_T;
    const int32_t* cu;
    int N, T, H, DV;
    float mu, scale;
};

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

// Register staging of one chunk's raw inputs. Every thread issues all of its 16-byte loads for
// the next chunk at once (so they are in flight together while the current chunk computes) and
// writes them to LDS at the top of the next iteration.
template <class TI, class CF>
struct ChunkRegs {
    static constexpr int VE = 16 / (int)sizeof(TI);       // elements per 16 bytes
    static constexpr int VPR = CF::DK / VE;               // vectors per [DK] row
    static constexpr int NVEC = CF::C * VPR;              // vectors per [C][DK] array
    static constexpr int PER = (NVEC + NT - 1) / NT;      // per thread and array
    static constexpr int VPRV = CF::BV / VE;              // vectors per v row
    static constexpr int NVECV = CF::C * VPRV;
    static constexpr int PERV = (NVECV + NT - 1) / NT;
    static constexpr int NARR = 4;                        // alpha, k, omega, q
    uint4 raw[NARR][PER];
    uint4 vv[PERV];
    TI r, w, a;  // per-token scalars (tid < C), kept raw: converting them at load time would
                 // make the load wait for every earlier load of the prefetch
};

template <class TI, class CF>
__device__ __forceinline__ void load_chunk(ChunkRegs<TI, CF>& R, const TI* const* src,
                                           const bool* use, const TI* gv, const TI* gr,
                                           const TI* gw, const TI* ga, size_t row0, int H,
                                           int DV, int col0, int L, int tid)
{
    using CR = ChunkRegs<TI, CF>;
    constexpr int DK = CF::DK;
    const size_t rs = (size_t)H * DK;
    // rows past the sequence end: alpha = 1 (no decay), everything else 0
    const unsigned one = sizeof(TI) == 2 ? 0x3F803F80u : 0x3F800000u;
    if (L == CF::C) {  // full chunk: every row is valid, no predicates
#pragma unroll
        for (int a = 0; a < CR::NARR; ++a) {
            if (!use[a]) continue;
            const TI* base = src[a] + row0 * DK;
#pragma unroll
            for (int j = 0; j < CR::PER; ++j) {
                const int idx = tid + j * NT;
                const int t = idx / CR::VPR, e = (idx % CR::VPR) * CR::VE;
                if (CR::NVEC % NT == 0 || idx < CR::NVEC)
                    R.raw[a][j] = *reinterpret_cast<const uint4*>(base + t * rs + e);
            }
        }
#pragma unroll
        for (int j = 0; j < CR::PERV; ++j) {
            const int idx = tid + j * NT;
            const int t = idx / CR::VPRV, e = (idx % CR::VPRV) * CR::VE;
            if (CR::NVECV % NT == 0 || idx < CR::NVECV)
                R.vv[j] = *reinterpret_cast<const uint4*>(gv + (row0 + (size_t)t * H) * DV + col0 + e);
        }
    } else {
#pragma unroll
        for (int a = 0; a < CR::NARR; ++a) {
#pragma unroll
            for (int j = 0; j < CR::PER; ++j) {
                const int idx = tid + j * NT;
                const int t = idx / CR::VPR, e = (idx % CR::VPR) * CR::VE;
                uint4 val = a == 0 ? make_uint4(one, one, one, one) : make_uint4(0, 0, 0, 0);
                if (use[a] && idx < CR::NVEC && t < L)
                    val = *reinterpret_cast<const uint4*>(src[a] + row0 * DK + t * rs + e);
                R.raw[a][j] = val;
            }
        }
#pragma unroll
        for (int j = 0; j < CR::PERV; ++j) {
            const int idx = tid + j * NT;
            const int t = idx / CR::VPRV, e = (idx % CR::VPRV) * CR::VE;
            uint4 val = make_uint4(0, 0, 0, 0);
            if (idx < CR::NVECV && t < L)
                val = *reinterpret_cast<const uint4*>(gv + (row0 + (size_t)t * H) * DV + col0 + e);
            R.vv[j] = val;
        }
    }
    R.r = from_f32<TI>(1.f); R.w = from_f32<TI>(0.f); R.a = from_f32<TI>(1.f);
    if (tid < L) {
        const size_t row = row0 + (size_t)tid * H;
        R.r = gr[row];
        if (CF::VARIANT == 1) {
            R.w = gw[row];
            if (!CF::APC) R.a = ga[row];
        }
    }
}

template <class TI, class CF>
__device__ __forceinline__ void store_chunk(const ChunkRegs<TI, CF>& R, TI* const* dst,
                                            const bool* use, TI* sV, int tid)
{
    using CR = ChunkRegs<TI, CF>;
#pragma unroll
    for (int a = 0; a < CR::NARR; ++a) {
        if (!use[a]) continue;
#pragma unroll
        for (int j = 0; j < CR::PER; ++j) {
            const int idx = tid + j * NT;
            if (idx < CR::NVEC)
                *reinterpret_cast<uint4*>(dst[a] + (idx / CR::VPR) * CF::DK +
                                          (idx % CR::VPR) * CR::VE) = R.raw[a][j];
        }
    }
#pragma unroll
    for (int j = 0; j < CR::PERV; ++j) {
        const int idx = tid + j * NT;
        if (idx < CR::NVECV)
            *reinterpret_cast<uint4*>(sV + (idx / CR::VPRV) * CF::BV + (idx % CR::VPRV) * CR::VE) =
                R.vv[j];
    }
}

// ------------------------------------------------------------------------------------------
// the kernel
// ------------------------------------------------------------------------------------------
template <class TI, class CF>
__global__ __launch_bounds__(NT, 1) void kdn_fwd_kernel(FwdArgs a)
{
    using MT = typename CF::MT;
    constexpr int DK = CF::DK, BV = CF::BV, C = CF::C, LDK = CF::LDK, LDC = CF::LDC,
                  LDT = CF::LDT, NB = CF::NB;
    constexpr bool DIAG = CF::VARIANT == 0;
    constexpr bool APC = CF::APC;
    extern __shared__ __attribute__((aligned(16))) char smem[];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, lg = lane >> 4;
    const int NH = a.N * a.H;
    const int nh = blockIdx.x % NH, tile = blockIdx.x / NH;
    const int n = nh / a.H, h = nh % a.H;
    const int col0 = tile * BV;
    const int H = a.H, DV = a.DV;

    const TI* gq = (const TI*)a.q;
    const TI* gk = (const TI*)a.k;
    const TI* gv = (const TI*)a.v;
    const TI* ga = (const TI*)a.alpha;
    const TI* gw = (const TI*)a.omega;
    const TI* gr = (const TI*)a.r;
    TI* go = (TI*)a.o;

    TI* sA = (TI*)smem;  // alpha [C][DK]
    TI* sK = sA + CF::RAWN;
    TI* sW = sK + CF::RAWN;
    TI* sQ = sW + CF::RAWN;
    float* Tm = (float*)(smem + CF::OFF_TM);
    MT* Ai = (MT*)(smem + CF::OFF_AI);
    MT* Aq = (MT*)(smem + CF::OFF_AQ);
    MT* XT = (MT*)(smem + CF::OFF_XT);
    MT* RT = (MT*)(smem + CF::OFF_RT);
    MT* R2T = (MT*)(smem + CF::OFF_R2T);
    MT* Inv = (MT*)(smem + CF::OFF_INV);
    MT* AiT = (MT*)(smem + CF::OFF_AIT);  // A transposed: AiT[col][row]
    TI* sV = (TI*)(smem + CF::OFF_V);
    MT* Kb = (MT*)(smem + CF::OFF_KB);
    MT* Qb = (MT*)(smem + CF::OFF_QB);
    MT* Pb = (MT*)(smem + CF::OFF_PB);
    MT* PbT = (MT*)(smem + CF::OFF_PBT);
    MT* SmT = (MT*)(smem + CF::OFF_SMT);
    float* s_r = (float*)(smem + CF::OFF_SC);
    float* s_mr = s_r + C;
    float* s_rden = s_mr + C;
    float* s_beta = s_rden + C;
    float* s_gtok = s_beta + C;
    float* s_gC = s_gtok + C;
    float* s_wtok = s_gC + DK;
    float* s_atok = s_wtok + C;
    float* s_zin = s_atok + C + 4;                 // [DK][2] carried (n, d) per channel
    float* s_segM = s_zin + 2 * DK;                // [NSEG-1][DK][4] segment Moebius products
    float* s_segG = s_segM + (CF::NSEG - 1) * DK * 4;  // [NSEG-1][DK] segment decay products

    int t0, t1;
    seq_range(a.cu, n, a.T, t0, t1);

    // ---- state tile: wave w owns tiles st = w + 4 j of the [DK x BV] tile grid ----------
    floatx4 Sacc[CF::ST_PER_WAVE];
#pragma unroll
    for (int j = 0; j < CF::ST_PER_WAVE; ++j) {
        const int st = wave + 4 * j;
        Sacc[j] = zero4();
        if (st < CF::NST && a.S0) {
            const int it = st / CF::NNT, jt = st % CF::NNT;
            const float* src = a.S0 + (size_t)nh * DK * DV;
#pragma unroll
            for (int rr = 0; rr < 4; ++rr)
                Sacc[j][rr] = src[(size_t)(16 * it + 4 * lg + rr) * DV + col0 + 16 * jt + li];
        }
    }

    // ---- variance state (diagonal: per channel, owned by threads [0, DK)) ------------------
    if (DIAG && tid < DK) {
        s_zin[2 * tid] = a.P0 ? a.P0[(size_t)nh * DK + tid] : 1.f;  // z_0 = [p_0; 1]
        s_zin[2 * tid + 1] = 1.f;
    }
    // isotropic: one chain per head, carried by every lane of wave 0
    float izn = 1.f, izd = 1.f;
    if (!DIAG && a.P0) izn = a.P0[nh];

    // S^in operand of the first chunk (transposed, operand precision)
#pragma unroll
    for (int j = 0; j < CF::ST_PER_WAVE; ++j) {
        const int st = wave + 4 * j;
        if (st < CF::NST) {
            const int it = st / CF::NNT, nt = st % CF::NNT;
#pragma unroll
            for (int rr = 0; rr < 4; ++rr)
                SmT[(16 * nt + li) * LDK + 16 * it + 4 * lg + rr] = from_f32<MT>(Sacc[j][rr]);
        }
    }

    const TI* srcs[4] = {ga, gk, gw, gq};
    TI* dsts[4] = {sA, sK, sW, sQ};
    const bool use[4] = {APC, true, DIAG, true};
    ChunkRegs<TI, CF> pre;
    if (t0 < t1)
        load_chunk<TI, CF>(pre, srcs, use, gv, gr, gw, ga, (size_t)t0 * H + h, H, DV, col0,
                           min(C, t1 - t0), tid);

    for (int c0 = t0; c0 < t1; c0 += C) {
        const int L = min(C, t1 - c0);
        const size_t row0 = (size_t)c0 * H + h;  // (token c0, head h)

        // ---- stage the chunk's raw inputs (prefetched into registers) ------------------
        __syncthreads();  // previous chunk finished with every LDS region
        store_chunk<TI, CF>(pre, dsts, use, sV, tid);
        if (tid < C) {
            const float rr = to_f32(pre.r);
            s_r[tid] = rr;
            s_mr[tid] = a.mu / rr;
            if (!DIAG) {
                s_wtok[tid] = to_f32(pre.w);
                if (!APC) s_atok[tid] = to_f32(pre.a);
            }
        }
        __syncthreads();

        // ---- phase 1: gains and decayed operands ---------------------------------------
        // Tokens past the end of the sequence were staged as alpha = 1, k = q = v = omega = 0,
        // r = 1: they leave every state unchanged and produce zero operand rows, so the token
        // loops below run over the whole chunk without branches (fully unrolled: the LDS loads
        // of later tokens are issued ahead of the serial variance chain).
        if (DIAG) {
            // Segmented scan of the variance chain. Wave s owns tokens [16 s, 16 s + 16) and
            // every lane an adjacent channel pair (2 p, 2 p + 1), so each lane carries two
            // independent chains. Pass 1: each segment's Moebius product (later tokens on the
            // left) and decay product. Pass 2: each wave composes the earlier segments onto the
            // carried state, then replays its tokens emitting P_bar = p_hat k / gamma,
            // K_bar = gamma k and Q_bar = gamma q. The last segment leaves the next carry.
            constexpr int NSEG = CF::NSEG, NP = DK / 2;
            const int seg = wave, pc = lane;
            const bool active = seg < NSEG && pc < NP;
            const int c0 = 2 * pc, t0s = 16 * seg;
            if (active && seg < NSEG - 1) {
                float m0[4] = {1.f, 0.f, 0.f, 1.f}, m1[4] = {1.f, 0.f, 0.f, 1.f};
                float g0 = 1.f, g1 = 1.f;
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const int t = t0s + j;
                    const float2 al = ld2(sA + t * DK + c0), kk = ld2(sK + t * DK + c0);
                    const float2 w = ld2(sW + t * DK + c0);
                    const float mr = s_mr[t];
                    g0 *= al.x;
                    g1 *= al.y;
                    mob_left(m0, al.x * al.x, w.x, kk.x * kk.x * mr);
                    mob_left(m1, al.y * al.y, w.y, kk.y * kk.y * mr);
                    if (j & 1) {
                        renorm4(m0[0], m0[1], m0[2], m0[3]);
                        renorm4(m1[0], m1[1], m1[2], m1[3]);
                    }
                }
                float* M = s_segM + (size_t)(seg * DK + c0) * 4;
                *reinterpret_cast<float4*>(M) = make_float4(m0[0], m0[1], m0[2], m0[3]);
                *reinterpret_cast<float4*>(M + 4) = make_float4(m1[0], m1[1], m1[2], m1[3]);
                *reinterpret_cast<float2*>(s_segG + seg * DK + c0) = make_float2(g0, g1);
            }
            __syncthreads();
            float zn0 = 0.f, zd0 = 1.f, zn1 = 0.f, zd1 = 1.f;
            if (active) {
                zn0 = s_zin[2 * c0]; zd0 = s_zin[2 * c0 + 1];
                zn1 = s_zin[2 * c0 + 2]; zd1 = s_zin[2 * c0 + 3];
                float g0 = 1.f, g1 = 1.f;
                for (int ps = 0; ps < seg; ++ps) {  // state entering this segment
                    const float4 A0 = *reinterpret_cast<const float4*>(s_segM + (ps * DK + c0) * 4);
                    const float4 A1 =
                        *reinterpret_cast<const float4*>(s_segM + (ps * DK + c0) * 4 + 4);
                    float n = A0.x * zn0 + A0.y * zd0, d = A0.z * zn0 + A0.w * zd0;
                    zn0 = n; zd0 = d; renorm2(zn0, zd0);
                    n = A1.x * zn1 + A1.y * zd1; d = A1.z * zn1 + A1.w * zd1;
                    zn1 = n; zd1 = d; renorm2(zn1, zd1);
                    const float2 gg = *reinterpret_cast<const float2*>(s_segG + ps * DK + c0);
                    g0 *= gg.x;
                    g1 *= gg.y;
                }
                float pb0[16], pb1[16];
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const int t = t0s + j;
                    const float2 al = ld2(sA + t * DK + c0), kk = ld2(sK + t * DK + c0);
                    const float2 w = ld2(sW + t * DK + c0), qq = ld2(sQ + t * DK + c0);
                    const float mr = s_mr[t];
                    g0 *= al.x;
                    g1 *= al.y;
                    const float n0 = fmaf(al.x * al.x, zn0, w.x * zd0);  // n_t
                    const float n1 = fmaf(al.y * al.y, zn1, w.y * zd1);
                    pb0[j] = n0 * kk.x * __builtin_amdgcn_rcpf(zd0 * g0);  // p_hat k / gamma
                    pb1[j] = n1 * kk.y * __builtin_amdgcn_rcpf(zd1 * g1);
                    zd0 = fmaf(kk.x * kk.x * mr, n0, zd0);               // d_t
                    zd1 = fmaf(kk.y * kk.y * mr, n1, zd1);
                    zn0 = n0;
                    zn1 = n1;
                    if (j & 1) {
                        renorm2(zn0, zd0);
                        renorm2(zn1, zd1);
                    }
                    st2<MT>(Kb + t * LDK + c0, g0 * kk.x, g1 * kk.y);
                    st2<MT>(Qb + t * LDK + c0, g0 * qq.x, g1 * qq.y);
                    st2<MT>(Pb + t * LDK + c0, pb0[j], pb1[j]);
                }
                store8<MT>(PbT + c0 * LDC + t0s, pb0);
                store8<MT>(PbT + c0 * LDC + t0s + 8, pb0 + 8);
                store8<MT>(PbT + (c0 + 1) * LDC + t0s, pb1);
                store8<MT>(PbT + (c0 + 1) * LDC + t0s + 8, pb1 + 8);
                if (seg == NSEG - 1) {
                    *reinterpret_cast<float2*>(s_gC + c0) = make_float2(g0, g1);
                }
            }
            __syncthreads();  // every wave has read the carried state before it is replaced
            if (active && seg == NSEG - 1)
                *reinterpret_cast<float4*>(s_zin + 2 * c0) = make_float4(zn0, zd0, zn1, zd1);
        } else {
            // isotropic: per-token trace average of alpha^2 and ||k||^2; thread (token, quarter)
            // sums a quarter of the channels, two lane exchanges finish the sum
            {
                constexpr int QW = DK / 4;
                const int t = tid >> 2, qq = tid & 3;
                float sa = 0.f, sk = 0.f;
                if (t < C) {
#pragma unroll
                    for (int e = 0; e < QW; ++e) {
                        const float kk = to_f32(sK[t * DK + qq * QW + e]);
                        sk += kk * kk;
                        if (APC) {
                            const float al = to_f32(sA[t * DK + qq * QW + e]);
                            sa += al * al;
                        }
                    }
                }
                sk += __shfl_xor(sk, 1, 64);
                sk += __shfl_xor(sk, 2, 64);
                if (APC) {
                    sa += __shfl_xor(sa, 1, 64);
                    sa += __shfl_xor(sa, 2, 64);
                }
                if (t < C && qq == 0) {
                    float at;
                    if (APC) {
                        at = sa / (float)DK;
                    } else {
                        const float al = s_atok[t];
                        at = al * al;
                    }
                    s_beta[t] = sk;      // ||k_t||^2 (overwritten by beta below)
                    s_rden[t] = at;      // a_t (temporarily)
                }
            }
            __syncthreads();
            if (wave == 0) {
                // scalar Moebius chain of the head: Kogge-Stone scan over the chunk's tokens
                const int t = lane;
                const bool ok = t < L && t < C;
                float ma = 1.f, mb = 0.f, mc = 0.f, md = 1.f, at = 1.f, wt = 0.f, nk = 0.f;
                if (ok) {
                    at = s_rden[t];
                    wt = s_wtok[t];
                    nk = s_beta[t];
                    const float u = s_mr[t] * nk / (float)DK;   // mu ||k||^2 / (dk r)
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
                float zn2 = ma * izn + mb * izd, zd2 = mc * izn + md * izd;  // after token t
                renorm2(zn2, zd2);
                float en = __shfl_up(zn2, 1, 64), ed = __shfl_up(zd2, 1, 64);  // before token t
                if (lane == 0) { en = izn; ed = izd; }
                if (t < C) s_beta[t] = ok ? (at * en / ed + wt) / (s_r[t] + (at * en / ed + wt) * nk)
                                          : 0.f;
                // decay of a per-head gate: gamma_t as a prefix product over the lanes
                if (!APC) {
                    float gt = ok ? s_atok[t] : 1.f;
#pragma unroll
                    for (int off = 1; off < 64; off <<= 1) {
                        const float y = __shfl_up(gt, off, 64);
                        if (lane >= off) gt *= y;
                    }
                    if (t < C) s_gtok[t] = gt;
                }
                const int lastl = L - 1;
                izn = __shfl(zn2, lastl, 64);
                izd = __shfl(zd2, lastl, 64);
            }
            __syncthreads();
            if (tid < C) s_rden[tid] = 1.f;
            if (APC) {
                if (tid < 2 * DK) {
                    const int c = tid % DK;
                    const bool kside = tid < DK;
                    float g = 1.f;
#pragma unroll
                    for (int t8 = 0; t8 < C; t8 += 8) {
                        float pb8[8];
#pragma unroll
                        for (int j = 0; j < 8; ++j) {
                            const int t = t8 + j;
                            g *= to_f32(sA[t * DK + c]);
                            if (kside) {
                                const float kk = to_f32(sK[t * DK + c]);
                                pb8[j] = s_beta[t] * kk * __builtin_amdgcn_rcpf(g);  // P_bar
                                Kb[t * LDK + c] = from_f32<MT>(g * kk);               // K_bar
                                Pb[t * LDK + c] = from_f32<MT>(pb8[j]);
                            } else {
                                Qb[t * LDK + c] = from_f32<MT>(g * to_f32(sQ[t * DK + c]));
                            }
                        }
                        if (kside) store8<MT>(PbT + c * LDC + t8, pb8);
                    }
                    if (kside) s_gC[c] = g;
                }
            } else {
                for (int idx = tid; idx < C * DK; idx += NT) {
                    const int t = idx / DK, c = idx % DK;
                    const float g = s_gtok[t], kk = to_f32(sK[idx]);
                    const float pb = s_beta[t] * kk / g;
                    Kb[t * LDK + c] = from_f32<MT>(g * kk);
                    Qb[t * LDK + c] = from_f32<MT>(g * to_f32(sQ[idx]));
                    Pb[t * LDK + c] = from_f32<MT>(pb);
                    PbT[c * LDC + t] = from_f32<MT>(pb);
                }
                if (tid < DK) s_gC[tid] = s_gtok[L - 1];
            }
            __syncthreads();
        }

        // issue the next chunk's loads now (after the register-heavy token loops); they land
        // while phases 2-6 of this chunk compute
        // (unconditional: past the last chunk every load is predicated off; a branch on the
        // loop condition here would let the compiler merge the loads into the loop latch)
        load_chunk<TI, CF>(pre, srcs, use, gv, gr, gw, ga, row0 + (size_t)C * H, H, DV, col0,
                           max(0, min(C, t1 - c0 - C)), tid);
        __builtin_amdgcn_sched_barrier(0);  // keep the loads here, ahead of phases 2-6

        // ---- phase 2: T = tril(K_bar P_bar^T, -1) / den and A_qk = tril(Q_bar P_bar^T) / den
        // 2a: wave b owns diagonal block b. Its K_bar P_bar^T diagonal is sum_i p_hat k^2, which
        // gives den; the wave scales the block, stores it and inverts I + T_bb by forward
        // substitution (lanes 0..15, one column each) without waiting for the other waves.
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
                    float trow[16];  // row i of the block, 16-byte broadcast reads
#pragma unroll
                    for (int v4 = 0; v4 < (i + 3) / 4; ++v4) {
                        const float4 q4 = *reinterpret_cast<const float4*>(Tb + i * LDT + 4 * v4);
                        trow[4 * v4] = q4.x; trow[4 * v4 + 1] = q4.y;
                        trow[4 * v4 + 2] = q4.z; trow[4 * v4 + 3] = q4.w;
                    }
                    float sum = 0.f;
#pragma unroll
                    for (int kk = 0; kk < i; ++kk) sum = fmaf(trow[kk], x[kk], sum);
                    x[i] = i < j ? 0.f : (i == j ? 1.f : -sum);
                }
#pragma unroll
                for (int i = 0; i < 16; ++i) Ai[(16 * b + i) * LDC + 16 * b + j] = from_f32<MT>(x[i]);
                // column j of the block is row j of the transposed copy: 16 consecutive values
                store8<MT>(AiT + (16 * b + j) * LDC + 16 * b, x);
                store8<MT>(AiT + (16 * b + j) * LDC + 16 * b + 8, x + 8);
            }
        }
        __syncthreads();
        // 2b: off-diagonal T blocks and every A_qk block, columns scaled by 1/den. T(ib, jb) and
        // A_qk(ib, jb) share the P_bar fragment of block column jb; wave w takes the units
        // w, w + 4, ... of [pairs (ib > jb) ..., diagonal A_qk blocks ...].
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
                            Aq[row * LDC + col] = from_f32<MT>((4 * lg + rr) >= li ? qacc[rr] * rd
                                                                                  : 0.f);
                        }
                    }
                }
            }
            // zero the blocks above the diagonal of A_qk and A: 16-byte stores
            constexpr int VPB = 16 * (int)sizeof(MT) / 16;         // 16-byte vectors per block row
            constexpr int NUP = NB * (NB - 1) / 2;                  // blocks above the diagonal
            if constexpr (NUP > 0)
            for (int idx = tid; idx < 2 * NUP * 16 * VPB; idx += NT) {
                const int which = idx / (NUP * 16 * VPB), rem = idx % (NUP * 16 * VPB);
                int blk = rem / (16 * VPB);
                const int row16 = (rem / VPB) % 16, vec = rem % VPB;
                int ib = 0;                                          // blk -> (ib < jb)
                while (blk >= NB - 1 - ib) { blk -= NB - 1 - ib; ++ib; }
                const int jb = ib + 1 + blk;
                MT* base = which ? Ai : Aq;
                *reinterpret_cast<uint4*>(base + (16 * ib + row16) * LDC + 16 * jb +
                                          vec * (16 / (int)sizeof(MT))) = make_uint4(0, 0, 0, 0);
            }
        }
        __syncthreads();

        // ---- phase 3: A = (I + T)^-1 off the diagonal (diagonal blocks done in 2a) -----
        // A_ij = -A_ii sum_{j<=k<i} T_ik A_kj, one block diagonal d = i - j at a time (blocks
        // further from the diagonal depend on the nearer ones). Operands are read as vectors:
        // T rows (fp32), A columns from the transposed copy.
#pragma unroll
        for (int d = 1; d < NB; ++d) {
            const int nblk = NB - d;
            if (wave < nblk) {
                const int jb = wave, ib = jb + d;
                floatx4 acc = zero4();
                for (int kb = jb; kb < ib; ++kb)
                    acc = mm16_tv<MT>(Tm + (16 * ib) * LDT + 16 * kb, LDT,
                                      AiT + (16 * jb) * LDC + 16 * kb, LDC, acc, lane);
                // tmp = acc, stored transposed (tmpT[col][row]) as the next B operand
                MT* tmpT = Inv + wave * 16 * CF::LDI;
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    tmpT[li * CF::LDI + 4 * lg + rr] = from_f32<MT>(acc[rr]);
                wave_lds_sync();
                const floatx4 res = mm_kc<MT, 16>(Ai + (16 * ib) * LDC + 16 * ib, LDC, tmpT,
                                                  CF::LDI, zero4(), lane);
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) {
                    const int row = 16 * ib + 4 * lg + rr, col = 16 * jb + li;
                    Ai[row * LDC + col] = from_f32<MT>(-res[rr]);
                    AiT[col * LDC + row] = from_f32<MT>(-res[rr]);
                }
            }
            __syncthreads();
        }

        // ---- phase 4: X = V - K_bar S^in (to XT), Q_bar S^in kept in registers ----------
        floatx4 Oacc[CF::OUT_PER_WAVE];
#pragma unroll
        for (int j = 0; j < CF::OUT_PER_WAVE; ++j) {
            const int ot = wave + 4 * j;
            Oacc[j] = zero4();
            if (ot < CF::NOUT) {
                const int mt = ot / CF::NNT, nt = ot % CF::NNT;
                floatx4 x = zero4();
                mm_kc2<MT, DK>(Kb + 16 * mt * LDK, Qb + 16 * mt * LDK, LDK, SmT + 16 * nt * LDK,
                               LDK, x, Oacc[j], lane);
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) {
                    const int t = 16 * mt + 4 * lg + rr, cc = 16 * nt + li;
                    const float vv = to_f32(sV[t * BV + cc]);
                    XT[cc * LDC + t] = from_f32<MT>(vv - x[rr]);
                }
            }
        }
        __syncthreads();

        // ---- phase 5: R = A X (to RT, and R / den to R2T) ------------------------------
#pragma unroll
        for (int j = 0; j < CF::OUT_PER_WAVE; ++j) {
            const int ot = wave + 4 * j;
            if (ot < CF::NOUT) {
                const int mt = ot / CF::NNT, nt = ot % CF::NNT;
                floatx4 rr4 = mm_kc<MT, C>(Ai + 16 * mt * LDC, LDC, XT + 16 * nt * LDC, LDC,
                                           zero4(), lane);
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) {
                    const int t = 16 * mt + 4 * lg + rr, cc = 16 * nt + li;
                    RT[cc * LDC + t] = from_f32<MT>(rr4[rr]);
                    R2T[cc * LDC + t] = from_f32<MT>(rr4[rr] * s_rden[t]);
                }
            }
        }
        __syncthreads();

        // ---- phase 6: O = scale (Q_bar S^in + A_qk R); S = gamma_C (S + P_bar^T R / den) --
#pragma unroll
        for (int j = 0; j < CF::OUT_PER_WAVE; ++j) {
            const int ot = wave + 4 * j;
            if (ot < CF::NOUT) {
                const int mt = ot / CF::NNT, nt = ot % CF::NNT;
                floatx4 acc = mm_kc<MT, C>(Aq + 16 * mt * LDC, LDC, RT + 16 * nt * LDC, LDC,
                                           Oacc[j], lane);
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) {
                    const int t = 16 * mt + 4 * lg + rr;
                    if (t < L)
                        go[(row0 + (size_t)t * H) * DV + col0 + 16 * nt + li] =
                            from_f32<TI>(a.scale * acc[rr]);
                }
            }
        }
#pragma unroll
        for (int j = 0; j < CF::ST_PER_WAVE; ++j) {
            const int st = wave + 4 * j;
            if (st < CF::NST) {
                const int it = st / CF::NNT, nt = st % CF::NNT;
                floatx4 y = mm_kc<MT, C>(PbT + 16 * it * LDC, LDC, R2T + 16 * nt * LDC, LDC,
                                         zero4(), lane);
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) {
                    const int ch = 16 * it + 4 * lg + rr;
                    Sacc[j][rr] = s_gC[ch] * (Sacc[j][rr] + y[rr]);
                }
            }
        }
        // next chunk's S^in operand (written after everyone is done with SmT: phase 4 ended
        // behind two barriers)
#pragma unroll
        for (int j = 0; j < CF::ST_PER_WAVE; ++j) {
            const int st = wave + 4 * j;
            if (st < CF::NST) {
                const int it = st / CF::NNT, nt = st % CF::NNT;
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    SmT[(16 * nt + li) * LDK + 16 * it + 4 * lg + rr] = from_f32<MT>(Sacc[j][rr]);
            }
        }
    }

    // ---- final state ---------------------------------------------------------------------
    if (a.S_T) {
#pragma unroll
        for (int j = 0; j < CF::ST_PER_WAVE; ++j) {
            const int st = wave + 4 * j;
            if (st < CF::NST) {
                const int it = st / CF::NNT, jt = st % CF::NNT;
                float* dst = a.S_T + (size_t)nh * DK * DV;
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    dst[(size_t)(16 * it + 4 * lg + rr) * DV + col0 + 16 * jt + li] = Sacc[j][rr];
            }
        }
    }
    if (a.P_T && tile == 0) {
        if (DIAG) {
            if (tid < DK) a.P_T[(size_t)nh * DK + tid] = s_zin[2 * tid] / s_zin[2 * tid + 1];
        } else if (tid == 0) {
            a.P_T[nh] = izn / izd;
        }
    }
}


template <class TI, int DK, int BV, int C, int VARIANT, bool APC>
hipError_t launch_cfg(const FwdArgs& fa, hipStream_t st)
{
    using CF = Cfg<TI, DK, BV, C, VARIANT, APC>;
    auto kern = kdn_fwd_kernel<TI, CF>;
    static bool attr_done = false;  // one attribute call per instantiation and process
    if (!attr_done) {
        hipError_t e = hipFuncSetAttribute((const void*)kern,
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)CF::TOTAL);
        if (e != hipSuccess) return e;
        attr_done = true;
    }
    const unsigned nblk = (unsigned)((size_t)fa.N * fa.H * (fa.DV / BV));
    hipLaunchKernelGGL(kern, dim3(nblk), dim3(NT), CF::TOTAL, st, fa);
    return hipGetLastError();
}

template <class TI, int DK, int BV, int C>
constexpr bool fits()
{
    return Cfg<TI, DK, BV, C, 0, true>::TOTAL <= 160 * 1024;
}

template <class TI, int DK, int BV, int C>
hipError_t launch_variant(int variant, int apc, const FwdArgs& fa, hipStream_t st)
{
    if constexpr (!fits<TI, DK, BV, C>()) {
        return hipErrorInvalidConfiguration;
    } else {
        if (variant == 0) return launch_cfg<TI, DK, BV, C, 0, true>(fa, st);
        if (apc) return launch_cfg<TI, DK, BV, C, 1, true>(fa, st);
        return launch_cfg<TI, DK, BV, C, 1, false>(fa, st);
    }
}

template <class TI, int DK, int BV>
hipError_t launch_chunk(int chunk, int variant, int apc, const FwdArgs& fa, hipStream_t st)
{
    switch (chunk) {
    case 16: return launch_variant<TI, DK, BV, 16>(variant, apc, fa, st);
    case 32: return launch_variant<TI, DK, BV, 32>(variant, apc, fa, st);
    case 64: return launch_variant<TI, DK, BV, 64>(variant, apc, fa, st);
    }
    return hipErrorInvalidValue;
}

template <class TI, int DK>
hipError_t launch_bv(int dv, int chunk, int variant, int apc, const FwdArgs& fa, hipStream_t st)
{
    if (dv == 16) return launch_chunk<TI, DK, 16>(chunk, variant, apc, fa, st);
    return launch_chunk<TI, DK, 32>(chunk, variant, apc, fa, st);
}

template <class TI>
hipError_t launch_dk(int dk, int dv, int chunk, int variant, int apc, const FwdArgs& fa,
                     hipStream_t st)
{
    switch (dk) {
    case 16: return launch_bv<TI, 16>(dv, chunk, variant, apc, fa, st);
    case 32: return launch_bv<TI, 32>(dv, chunk, variant, apc, fa, st);
    case 64: return launch_bv<TI, 64>(dv, chunk, variant, apc, fa, st);
    case 128: return launch_bv<TI, 128>(dv, chunk, variant, apc, fa, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace

namespace {

template <class TI, int DK>
bool fits_dk(int dv, int chunk)
{
    const bool bv16 = dv == 16;
    switch (chunk) {
    case 16: return bv16 ? fits<TI, DK, 16, 16>() : fits<TI, DK, 32, 16>();
    case 32: return bv16 ? fits<TI, DK, 16, 32>() : fits<TI, DK, 32, 32>();
    case 64: return bv16 ? fits<TI, DK, 16, 64>() : fits<TI, DK, 32, 64>();
    }
    return false;
}

template <class TI>
bool fits_rt(int dk, int dv, int chunk)
{
    switch (dk) {
    case 16: return fits_dk<TI, 16>(dv, chunk);
    case 32: return fits_dk<TI, 32>(dv, chunk);
    case 64: return fits_dk<TI, 64>(dv, chunk);
    case 128: return fits_dk<TI, 128>(dv, chunk);
    }
    return false;
}

}  // namespace

bool forward_chunk_supported(kdn_dtype_t dtype, int dk, int dv, int chunk)
{
    // a chunk is usable when one workgroup's LDS map fits the 160 KiB of a CU
    return dtype == KDN_F32 ? fits_rt<float>(dk, dv, chunk) : fits_rt<bf16>(dk, dv, chunk);
}

int forward_default_chunk(kdn_dtype_t dtype, int dk, int dv)
{
    for (int c = 64; c >= 16; c >>= 1)
        if (forward_chunk_supported(dtype, dk, dv, c)) return c;
    return 16;
}

size_t forward_workspace_bytes(int, int, int, int, int, int, int) { return 0; }

hipError_t launch_forward(int variant, const void* q, const void* k, const void* v,
                          const void* alpha, const void* omega, const void* r, const float* S0,
                          const float* P0, void* o, float* S_T, float* P_T, const SeqArgs& sa,
                          int dk, int dv, kdn_dtype_t dtype, int alpha_per_channel, float mu,
                          float scale, int chunk, void* workspace, hipStream_t stream)
{
    (void)workspace;
    FwdArgs fa;
    fa.q = q; fa.k = k; fa.v = v; fa.alpha = alpha; fa.omega = omega; fa.r = r;
    fa.S0 = S0; fa.P0 = P0; fa.o = o; fa.S_T = S_T; fa.P_T = P_T; fa.cu = sa.cu_seqlens;
    fa.N = sa.N; fa.T = sa.T; fa.H = sa.H; fa.DV = dv; fa.mu = mu; fa.scale = scale;
    if (chunk == 0) chunk = forward_default_chunk(dtype, dk, dv);
    if (dtype == KDN_F32)
        return launch_dk<float>(dk, dv, chunk, variant, alpha_per_channel, fa, stream);
    return launch_dk<bf16>(dk, dv, chunk, variant, alpha_per_channel, fa, stream);
}

}  // namespace kdn
