// Chunked forward of Diagonal / Isotropic KDN on gfx950 (arXiv 2609.07816, App.
// "Hardware-Efficient Chunkwise Algorithm"): the gain computation as a chunk-parallel scan,
// then the chunkwise memory scan.
//
// Tokens are cut into chunks of C = 64 (restarting at every sequence start; the last chunk of a
// sequence may be partial). Four kernels per call:
//   1. summary_kernel (chunk, head): the product of each chunk's 2x2 Moebius token matrices per
//      key channel (diagonal) or per head (isotropic)               eq. chunk-gain-summary
//   2. carry_scan_kernel (sequence, head, channel): the variance state entering every chunk, a
//      log-depth scan of the summaries                               eq. chunk-gain-carry
//   3. prep_kernel (chunk, head): replays the chunk from its carry (eqs. chunk-gain-local-prefix,
//      chunk-gain-emission) and builds everything of the memory scan that does not depend on the
//      memory state S: the decayed keys and queries, the tail-decayed write directions, the
//      inverse of the triangular factor and the intra-chunk read matrix. One record per
//      (chunk, head) in the workspace.
//   4. walk_kernel (sequence, head, 32 value columns): carries S through the chunks in order:
//        X = V - K_bar S,  R = L^-1 X,  O = scale (Q_bar S + A_qk R),  S <- gamma_C (.) S + P_tail^T R
//      (eqs. chunk-memory-wy, chunk-memory-tail-output, chunk-memory-output-state).
//
// Chunk algebra. With gamma_t = prod_{j <= t} alpha_j inside the chunk (per channel), the gain's
// normalisation kappa_t = G_t (.) k_t / c_t (G = p_hat and c = r + sum_i p_hat_i k_i^2 for the
// diagonal variant; G = beta and c = 1 for the isotropic one) is moved into the triangular
// factor:  L = diag(c) + tril(M, -1),  M_ts = sum_i k_ti (gamma_t / gamma_s)_i G_si k_si,
// A_qk = tril(M^q) with q in place of k (diagonal included: the read follows the write), and
// row t of R is token t's innovation divided by c_t. The decay ratios gamma_t / gamma_s <= 1 are
// formed without any factor larger than one where possible (the paper forms them from
// cumulative log-decay differences for the same reason):
//   - products with S use K_bar = gamma (.) k and Q_bar = gamma (.) q (<= 1 per channel), and the
//     state update uses P_tail_s = (gamma_C / gamma_s) G_s (.) k_s (<= G k);
//   - for a pair of distinct 16-token blocks (b > c), the row side is referenced to the start of
//     block b, the column side to the end of block c, and the decay of the blocks between them
//     scales one operand: every factor is <= 1, so underflow only drops terms below 2^-126;
//   - inside a 16-token diagonal block, both sides are referenced to its midpoint: a factor is
//     at most the inverse of the decay over 8 tokens, exact while that decay stays above
//     2^-126 (every alpha >= 2^-15 suffices); past it the factor saturates at 2^126 and the
//     results stay finite.
#pragma once

#include "kdn_device.h"

namespace kdn {
namespace fwd {

constexpr int C = 64;       // memory chunk (tokens)
constexpr int SL = 16;      // tokens per block; one wave per block in the variance phases
constexpr int NB = C / SL;  // blocks per chunk
constexpr int NW = 4;       // waves per workgroup
constexpr int NTH = 64 * NW;

// Record the prep writes for the walk, per (chunk, head), in operand precision MT:
//   Kb [C][DK]   K_bar = gamma (.) k            Qb [C][DK]  Q_bar = gamma (.) q
//   Pt [DK][C]   P_tail^T                       Li [C][C]   L^-1 (zeros above the diagonal)
//   Aq [C][C]    A_qk (zeros above)             gC [DK]     gamma_C (float32)
// The five matrices are stored in MFMA-fragment order (frag_off), so that the walk reads
// every operand fragment as one contiguous block.
template <class MT, int DK>
struct OpRec {
    static constexpr size_t OFF_KB = 0;
    static constexpr size_t OFF_QB = OFF_KB + (size_t)C * DK * sizeof(MT);
    static constexpr size_t OFF_PT = OFF_QB + (size_t)C * DK * sizeof(MT);
    static constexpr size_t OFF_LI = OFF_PT + (size_t)DK * C * sizeof(MT);
    static constexpr size_t OFF_AQ = OFF_LI + (size_t)C * C * sizeof(MT);
    static constexpr size_t OFF_GC = OFF_AQ + (size_t)C * C * sizeof(MT);
    static constexpr size_t BYTES = al256(OFF_GC + (size_t)DK * 4);
};

// Fragment order of an R x K matrix (R and K multiples of 16) used as an MFMA A operand with
// contraction over K: fragment (rb, s) holds rows 16 rb .. 16 rb + 15 and k in [KF s, KF s + KF)
// as 64 consecutive pieces of E = KF / 4 elements, piece 16 g + i = row 16 rb + i,
// k = KF s + E g .. + E - 1. Lane 16 g + i of a wave then loads piece 16 g + i: one fragment is
// one contiguous read of 64 E elements.
template <class MT, int K>
__device__ __forceinline__ size_t frag_off(int row, int k)
{
    using F = Frag<MT, K>;
    constexpr int E = F::KF / 4;
    const int rb = row >> 4, i = row & 15, sk = k / F::KF, g = (k % F::KF) / E, e = k % E;
    return ((size_t)(rb * F::NS + sk) * 64 + 16 * g + i) * E + e;
}

// Lane `lane`'s piece of fragment (rb, s).
template <class MT, int K>
__device__ __forceinline__ const MT* frag_piece(const MT* base, int rb, int sk, int lane)
{
    using F = Frag<MT, K>;
    return base + ((size_t)(rb * F::NS + sk) * 64 + lane) * (F::KF / 4);
}

// Copy an R x K row-major LDS tile (leading dimension ld) to global memory in fragment order,
// one piece of E elements per thread and step.
template <class MT, int R, int K, int NTHR>
__device__ __forceinline__ void copy_frag_order(MT* dst, const MT* src, int ld, int tid)
{
    using F = Frag<MT, K>;
    constexpr int E = F::KF / 4, NPC = R * K / E;
    static_assert(E * sizeof(MT) == 16 || E * sizeof(MT) == 8, "pieces of 8 or 16 bytes");
    for (int p = tid; p < NPC; p += NTHR) {
        const int lane = p & 63, fr = p >> 6;
        const int rb = fr / F::NS, sk = fr % F::NS;
        const int row = 16 * rb + (lane & 15), k = F::KF * sk + E * (lane >> 4);
        if constexpr (E * sizeof(MT) == 16)
            *reinterpret_cast<uint4*>(dst + (size_t)p * E) =
                *reinterpret_cast<const uint4*>(src + row * ld + k);
        else
            *reinterpret_cast<uint2*>(dst + (size_t)p * E) =
                *reinterpret_cast<const uint2*>(src + row * ld + k);
    }
}

template <class MT, int N>
__device__ __forceinline__ void storeN(MT* dst, const float* x)
{
    if constexpr (N == 8) store8<MT>(dst, x);
    else store4<MT>(dst, x[0], x[1], x[2], x[3]);
}

// ------------------------------------------------------------------------------------------
// variance side (summary and prep): wave w takes block w of the chunk; lane l the key-channel
// pair (2l, 2l + 1)
// ------------------------------------------------------------------------------------------
template <class TI, int DK_, int VARIANT_, bool APC_>
struct VarCfg {
    using MT = typename OpOf<TI>::type;
    using P2 = typename std::conditional<sizeof(TI) == 2, unsigned, float2>::type;
    static constexpr int DK = DK_;
    static constexpr bool DIAG = VARIANT_ == 0;
    static constexpr bool APC = APC_ || DIAG;  // gates per key channel
    static constexpr int NP = DK / 2;          // key-channel pairs (one per lane)
    static constexpr int NCHAN = DIAG ? DK : 1;
};

struct InArgs {
    const void *q, *k, *alpha, *omega, *r;
    uint32_t bytes_k, bytes_h;  // bytes of a channel tensor [.., H, DK], of a per-head [.., H]
    int H;
    float mu;
    // read by the layer kernels only (LAYER = true)
    const void* mu_t;  // per-token information scale [.., H], or nullptr (mu)
    float* beta_eff;   // k^T kappa per token [.., H] float32, or nullptr
    float r_min;
    int preact, qknorm;
};

// Descriptors and byte strides of one workgroup's inputs.
struct Src {
    rsrc_t q, k, al, om, r;
    uint32_t rowk, rowh;      // bytes per token row: channel tensors, per-head scalars
    uint32_t lane_k, lane_h;  // this lane's byte offset within a row (channel pair; head)
};

template <class TI, class CF>
__device__ __forceinline__ Src make_src(const InArgs& a, int h, int ch)
{
    constexpr uint32_t es = sizeof(TI);
    Src s;
    s.q = make_rsrc(a.q, a.bytes_k);
    s.k = make_rsrc(a.k, a.bytes_k);
    s.al = make_rsrc(a.alpha, CF::APC ? a.bytes_k : a.bytes_h);
    s.om = make_rsrc(a.omega, CF::DIAG ? a.bytes_k : a.bytes_h);
    s.r = make_rsrc(a.r, a.bytes_h);
    s.rowk = (uint32_t)a.H * CF::DK * es;
    s.rowh = (uint32_t)a.H * es;
    s.lane_k = ((uint32_t)h * CF::DK + ch) * es;
    s.lane_h = (uint32_t)h * es;
    return s;
}

// Raw inputs of one block held by a variance lane, kept in storage precision.
template <class TI, class CF, bool WQ>
struct SegIn {
    using P2 = typename CF::P2;
    using R1 = typename Raw1<TI>::type;
    P2 kk[SL];
    P2 qq[WQ ? SL : 1];
    P2 al[CF::APC ? SL : 1];   // per-channel gates
    P2 ww[CF::DIAG ? SL : 1];  // per-channel process noise (diagonal)
    R1 als[CF::APC ? 1 : SL];  // one gate per head (isotropic, scalar gates)
    R1 ws[CF::DIAG ? 1 : SL];  // one process noise per head (isotropic)
};

template <class TI, class CF, bool WQ>
__device__ __forceinline__ void load_seg(SegIn<TI, CF, WQ>& in, const Src& sr, uint32_t t0)
{
    using P2 = typename CF::P2;
#pragma unroll
    for (int j = 0; j < SL; ++j) {
        const uint32_t tok = t0 + (uint32_t)j;
        const uint32_t e = tok * sr.rowk + sr.lane_k, eh = tok * sr.rowh + sr.lane_h;
        in.kk[j] = bload<P2>(sr.k, e);
        if constexpr (WQ) in.qq[j] = bload<P2>(sr.q, e);
        if constexpr (CF::APC) in.al[j] = bload<P2>(sr.al, e);
        else in.als[j] = Raw1<TI>::load(sr.al, eh);
        if constexpr (CF::DIAG) in.ww[j] = bload<P2>(sr.om, e);
        else in.ws[j] = Raw1<TI>::load(sr.om, eh);
    }
}

// Token j of a block in float32. A token past the end of the sequence (j >= Lw) reads as no
// decay, no noise and zero key and query: it leaves the variance and the memory unchanged and
// gives zero operand rows.
struct TokIn {
    float2 K, Q, A, W;
};
template <class P2> __device__ __forceinline__ P2 pair_of_ones();
template <> __device__ __forceinline__ unsigned pair_of_ones<unsigned>() { return 0x3F803F80u; }
template <> __device__ __forceinline__ float2 pair_of_ones<float2>()
{
    return make_float2(1.f, 1.f);
}

template <bool MK, class TI, class CF, bool WQ>
__device__ __forceinline__ TokIn tok_in(const SegIn<TI, CF, WQ>& in, int j, int Lw)
{
    using P2 = typename CF::P2;
    const bool pad = MK && j >= Lw;
    const float2 z = make_float2(0.f, 0.f);
    // the selects act on the stored pair (one register for two bf16 channels); a pair of zeros
    // or ones unpacks exactly
    const P2 zero2 = P2{}, one2 = pair_of_ones<P2>();
    TokIn r;
    r.K = unpack2(pad ? zero2 : in.kk[j]);
    if constexpr (WQ) r.Q = unpack2(pad ? zero2 : in.qq[j]);
    else r.Q = z;
    if constexpr (CF::APC) {
        r.A = unpack2(pad ? one2 : in.al[j]);
    } else {
        const float as = pad ? 1.f : Raw1<TI>::f32(in.als[CF::APC ? 0 : j]);
        r.A = make_float2(as, as);
    }
    if constexpr (CF::DIAG) {
        r.W = unpack2(pad ? zero2 : in.ww[j]);
    } else {
        const float w = pad ? 0.f : Raw1<TI>::f32(in.ws[CF::DIAG ? 0 : j]);
        r.W = make_float2(w, w);
    }
    return r;
}

// The layer's maps on one token held by a variance lane (layer kernels): gates and noise from
// pre-activations, q and k divided by their L2 norms over the head (wave sums over the active
// lanes; a zero row stays zero). Padding tokens keep their neutral values.
template <class CF, bool WQ>
__device__ __forceinline__ void layer_tok(TokIn& x, const InArgs& a, bool vact, bool pad)
{
    if (a.preact && !pad) {
        if constexpr (CF::APC) {
            x.A = make_float2(gate_sigmoid(x.A.x), gate_sigmoid(x.A.y));
        } else {
            const float g = gate_sigmoid(x.A.x);
            x.A = make_float2(g, g);
        }
        if constexpr (CF::DIAG) {
            x.W = make_float2(gate_softplus(x.W.x), gate_softplus(x.W.y));
        } else {
            const float g = gate_softplus(x.W.x);
            x.W = make_float2(g, g);
        }
    }
    if (a.qknorm) {
        const float nk = wave_sum(vact ? fmaf(x.K.x, x.K.x, x.K.y * x.K.y) : 0.f);
        const float ik = nk > 0.f ? __builtin_amdgcn_rsqf(nk) : 0.f;
        x.K = make_float2(x.K.x * ik, x.K.y * ik);
        if constexpr (WQ) {
            const float nq = wave_sum(vact ? fmaf(x.Q.x, x.Q.x, x.Q.y * x.Q.y) : 0.f);
            const float iq = nq > 0.f ? __builtin_amdgcn_rsqf(nq) : 0.f;
            x.Q = make_float2(x.Q.x * iq, x.Q.y * iq);
        }
    }
}

// r and mu / r of the chunk's tokens (tid < C), with the layer's map of r and the per-token
// information scale in the layer kernels. Tokens past the chunk read r = 1 and mu / r = 0.
template <class TI, bool LAYER>
__device__ __forceinline__ void load_r(const InArgs& a, const Src& sr, int c0, int c1, int tid,
                                       float* s_r, float* s_mr)
{
    const int tok = c0 + tid;
    const uint32_t off = (uint32_t)tok * sr.rowh + sr.lane_h;
    float rv = Raw1<TI>::f32(Raw1<TI>::load(sr.r, off));
    float mu = a.mu;
    if constexpr (LAYER) {
        if (a.preact) rv = a.r_min + gate_softplus(rv);
        if (a.mu_t) mu = Raw1<TI>::f32(Raw1<TI>::load(make_rsrc(a.mu_t, a.bytes_h), off));
    }
    const bool ok = tok < c1;
    if (s_r) s_r[tid] = ok ? rv : 1.f;
    s_mr[tid] = ok ? mu / rv : 0.f;
}

// The block's Moebius product (later tokens on the left) and decay product. Diagonal: per
// channel of the lane's pair (m0, m1). Isotropic: one chain per head, every lane alike, with
// the per-token ||k||^2 and mean alpha^2 (wave reductions) returned in kn, ka.
template <bool MK, bool LAYER, class TI, class CF, bool WQ>
__device__ __forceinline__ void block_summary(const SegIn<TI, CF, WQ>& in, int Lw,
                                              const float* s_mr, bool vact, float* m0, float* m1,
                                              float2& gseg, float* kn, float* ka,
                                              const InArgs& a)
{
    m0[0] = 1.f; m0[1] = 0.f; m0[2] = 0.f; m0[3] = 1.f;
    m1[0] = 1.f; m1[1] = 0.f; m1[2] = 0.f; m1[3] = 1.f;
    float g0 = 1.f, g1 = 1.f;
#pragma unroll
    for (int j = 0; j < SL; ++j) {
        TokIn x = tok_in<MK>(in, j, Lw);
        if constexpr (LAYER) layer_tok<CF, WQ>(x, a, vact, MK && j >= Lw);
        const float mr = s_mr[j];
        if constexpr (CF::DIAG) {
            mob_left(m0, x.A.x * x.A.x, x.W.x, x.K.x * x.K.x * mr);
            mob_left(m1, x.A.y * x.A.y, x.W.y, x.K.y * x.K.y * mr);
        } else {
            kn[j] = wave_sum(vact ? fmaf(x.K.x, x.K.x, x.K.y * x.K.y) : 0.f);
            if constexpr (CF::APC)
                ka[j] = wave_sum(vact ? fmaf(x.A.x, x.A.x, x.A.y * x.A.y) : 0.f) *
                        (1.f / (float)CF::DK);
            else
                ka[j] = x.A.x * x.A.x;
            mob_left(m0, ka[j], x.W.x, kn[j] * mr * (1.f / (float)CF::DK));
        }
        g0 *= x.A.x;
        g1 *= x.A.y;
        if ((j & 3) == 3) {
            rescale4(m0);
            if constexpr (CF::DIAG) rescale4(m1);
        }
    }
    gseg = make_float2(g0, g1);
}

// ------------------------------------------------------------------------------------------
// 1. chunk summaries
// ------------------------------------------------------------------------------------------
template <class TI, class CF, bool LAYER>
__device__ __forceinline__ void summary_body(const InArgs& a, const ChunkMap& cm,
                                             float4* __restrict__ summ)
{
    constexpr int DK = CF::DK, NP = CF::NP;
    __shared__ float4 segA[NB][CF::NCHAN];
    __shared__ float s_mr[C];
    const int g = (int)(blockIdx.x / a.H), h = (int)(blockIdx.x % a.H);
    int n, c0, c1;
    bool last;
    if (!locate_chunk<C>(cm, g, n, c0, c1, last)) return;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int pc = min(lane, NP - 1), ch = 2 * pc;
    const bool vact = lane < NP;
    const Src sr = make_src<TI, CF>(a, h, ch);
    if (tid < C) load_r<TI, LAYER>(a, sr, c0, c1, tid, nullptr, s_mr);
    SegIn<TI, CF, false> in;
    load_seg(in, sr, (uint32_t)(c0 + SL * w));
    __syncthreads();
    const int Lw = c1 - (c0 + SL * w);
    float m0[4], m1[4], kn[CF::DIAG ? 1 : SL], ka[CF::DIAG ? 1 : SL];
    float2 gs;
    if (Lw < SL) block_summary<true, LAYER>(in, Lw, s_mr + SL * w, vact, m0, m1, gs, kn, ka, a);
    else block_summary<false, LAYER>(in, Lw, s_mr + SL * w, vact, m0, m1, gs, kn, ka, a);
    if constexpr (CF::DIAG) {
        if (vact) {
            segA[w][ch] = make_float4(m0[0], m0[1], m0[2], m0[3]);
            segA[w][ch + 1] = make_float4(m1[0], m1[1], m1[2], m1[3]);
        }
    } else if (lane == 0) {
        segA[w][0] = make_float4(m0[0], m0[1], m0[2], m0[3]);
    }
    __syncthreads();
    if (tid < CF::NCHAN) {
        float4 m = segA[0][tid];
#pragma unroll
        for (int b = 1; b < NB; ++b) m = mat_mul(segA[b][tid], m);
        summ[((size_t)g * a.H + h) * CF::NCHAN + tid] = m;
    }
    (void)DK;
}

// The plain bf16 summary asks for six waves per SIMD: 16 workgroups per CU at the
// 4 x 4096 x 16 shape then run in three rounds.
template <class TI, class CF>
__global__ __launch_bounds__(NTH) __attribute__((amdgpu_waves_per_eu(sizeof(TI) == 2 ? 6 : 4)))
void summary_kernel(InArgs a, ChunkMap cm, float4* __restrict__ summ)
{
    summary_body<TI, CF, false>(a, cm, summ);
}

template <class TI, class CF>
__global__ __launch_bounds__(NTH) void summary_layer_kernel(InArgs a, ChunkMap cm,
                                                            float4* __restrict__ summ)
{
    summary_body<TI, CF, true>(a, cm, summ);
}

// ------------------------------------------------------------------------------------------
// 3. prep: the chunk's S-independent operands
// ------------------------------------------------------------------------------------------
template <class TI, int DK_, int VARIANT_, bool APC_>
struct PrepCfg : VarCfg<TI, DK_, VARIANT_, APC_> {
    using B = VarCfg<TI, DK_, VARIANT_, APC_>;
    using MT = typename B::MT;
    static constexpr int DK = DK_;
    static constexpr int PAD = 16 / (int)sizeof(MT);
    static constexpr int LDK = DK + PAD, LDC = C + PAD, LDL = 20;
    static constexpr int NLB = NB * (NB + 1) / 2;  // lower 16 x 16 blocks of a C x C matrix
    static constexpr size_t SZ_OP = al16((size_t)C * LDK * sizeof(MT));
    static constexpr size_t SZ_CC = al16((size_t)C * LDC * sizeof(MT));
    static constexpr size_t SZ_R = cmax(SZ_OP, SZ_CC);
    // operand tiles [C][LDK] (mid-referenced, then start/end-referenced); reused at the end
    // as the staging of A_qk and L^-1 [C][LDC]
    static constexpr size_t OFF_KA = 0, OFF_QA = SZ_R, OFF_PA = 2 * SZ_R;
    // L's lower blocks in float32 [NLB][16][LDL]; the blocks' Moebius products alias them
    static constexpr size_t SZ_LF = al16(cmax((size_t)NLB * 16 * LDL * 4, (size_t)NB * DK * 16));
    static constexpr size_t OFF_LF = 3 * SZ_R;
    static constexpr size_t OFF_AI = OFF_LF + SZ_LF;  // diagonal blocks of L^-1, float32
    static constexpr size_t OFF_SG = OFF_AI + al16((size_t)NB * 16 * LDL * 4);  // [NB][DK]
    static constexpr size_t OFF_RHO = OFF_SG + (size_t)NB * DK * 4;              // [DK]
    static constexpr size_t OFF_R = OFF_RHO + (size_t)DK * 4;                    // r [C]
    static constexpr size_t OFF_MR = OFF_R + (size_t)C * 4;                      // mu / r [C]
    static constexpr size_t TOTAL = al16(OFF_MR + (size_t)C * 4);
};

struct PrepArgs {
    InArgs in;
    ChunkMap cm;
    const float2* carry;  // [maxch][H][nchan]
    char* ops;            // [maxch][H] records
    float* P_T;
};

// One block pair (ib, jb) of M and M^q from LDS operand tiles; the column side optionally
// scaled per channel by rho.
template <class MT, int DK, int LDK>
__device__ __forceinline__ void pair_prod(const MT* Ka, const MT* Qa, const MT* Pa, int ib,
                                          int jb, const float* rho, int lane, floatx4& tacc,
                                          floatx4& qacc)
{
    using FK = Frag<MT, DK>;
    const int li = lane & 15, lg = lane >> 4;
    typename FK::V kf[FK::NS], qf[FK::NS], pf[FK::NS];
#pragma unroll
    for (int s = 0; s < FK::NS; ++s) {
        const int k0 = FK::KF * s + (FK::KF / 4) * lg;
        kf[s] = FK::ld(Ka + (16 * ib + li) * LDK + k0);
        qf[s] = FK::ld(Qa + (16 * ib + li) * LDK + k0);
        pf[s] = FK::ld(Pa + (16 * jb + li) * LDK + k0);
        if (rho) pf[s] = FK::scale(pf[s], rho + k0);
    }
    tacc = zero4();
    qacc = zero4();
#pragma unroll
    for (int s = 0; s < FK::NS; ++s) {
        tacc = FK::mma(tacc, kf[s], pf[s]);
        qacc = FK::mma(qacc, qf[s], pf[s]);
    }
}

template <class TI, class CF, bool LAYER>
__device__ __forceinline__ void prep_body(const PrepArgs& a)
{
    using MT = typename CF::MT;
    using Rec = OpRec<MT, CF::DK>;
    constexpr int DK = CF::DK, NP = CF::NP, LDK = CF::LDK, LDC = CF::LDC, LDL = CF::LDL;
    constexpr bool DIAG = CF::DIAG;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    MT* Ka = (MT*)(smem + CF::OFF_KA);
    MT* Qa = (MT*)(smem + CF::OFF_QA);
    MT* Pa = (MT*)(smem + CF::OFF_PA);
    float* Lf = (float*)(smem + CF::OFF_LF);
    float4* segA = (float4*)(smem + CF::OFF_LF);  // [NB][DK] (dead before Lf is written)
    float* Ai = (float*)(smem + CF::OFF_AI);
    float* segG = (float*)(smem + CF::OFF_SG);
    float* rho = (float*)(smem + CF::OFF_RHO);
    float* s_r = (float*)(smem + CF::OFF_R);
    float* s_mr = (float*)(smem + CF::OFF_MR);

    const int H = a.in.H;
    const int g = (int)(blockIdx.x / H), h = (int)(blockIdx.x % H);
    int n, c0, c1;
    bool last;
    if (!locate_chunk<C>(a.cm, g, n, c0, c1, last)) return;
    const int nh = n * H + h;
    const int tid = threadIdx.x, lane = tid & 63, li = lane & 15, lg = lane >> 4;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int pc = min(lane, NP - 1), ch = 2 * pc;
    const bool vact = lane < NP;

    char* rec = a.ops + ((size_t)g * H + h) * Rec::BYTES;
    MT* gKb = (MT*)(rec + Rec::OFF_KB);
    MT* gQb = (MT*)(rec + Rec::OFF_QB);
    MT* gPt = (MT*)(rec + Rec::OFF_PT);
    MT* gLi = (MT*)(rec + Rec::OFF_LI);
    MT* gAq = (MT*)(rec + Rec::OFF_AQ);
    float* gC = (float*)(rec + Rec::OFF_GC);

    const Src sr = make_src<TI, CF>(a.in, h, ch);
    if (tid < C) load_r<TI, LAYER>(a.in, sr, c0, c1, tid, s_r, s_mr);
    const int Lw = c1 - (c0 + SL * w);  // tokens of this block in the sequence (may be <= 0)
    // the block's tokens in float32, unpacked once
    float2 Kf[SL], Qf[SL], Af[SL], Wf[SL];
    {
        SegIn<TI, CF, true> in;
        load_seg(in, sr, (uint32_t)(c0 + SL * w));
#pragma unroll
        for (int j = 0; j < SL; ++j) {
            TokIn x = tok_in<true>(in, j, Lw);
            if constexpr (LAYER) layer_tok<CF, true>(x, a.in, vact, j >= Lw);
            Kf[j] = x.K;
            Qf[j] = x.Q;
            Af[j] = x.A;
            Wf[j] = x.W;
        }
    }
    __syncthreads();

    // ---- the block's Moebius and decay products (eq. chunk-gain-summary) ----------------------
    float kn[DIAG ? 1 : SL], ka[DIAG ? 1 : SL];  // isotropic: ||k||^2 and mean alpha^2
    {
        float m0[4] = {1.f, 0.f, 0.f, 1.f}, m1[4] = {1.f, 0.f, 0.f, 1.f};
        float2 gs = make_float2(1.f, 1.f);
#pragma unroll
        for (int j = 0; j < SL; ++j) {
            const float mr = s_mr[SL * w + j];
            if constexpr (DIAG) {
                mob_left(m0, Af[j].x * Af[j].x, Wf[j].x, Kf[j].x * Kf[j].x * mr);
                mob_left(m1, Af[j].y * Af[j].y, Wf[j].y, Kf[j].y * Kf[j].y * mr);
            } else {
                kn[j] = wave_sum(vact ? fmaf(Kf[j].x, Kf[j].x, Kf[j].y * Kf[j].y) : 0.f);
                if constexpr (CF::APC)
                    ka[j] = wave_sum(vact ? fmaf(Af[j].x, Af[j].x, Af[j].y * Af[j].y) : 0.f) *
                            (1.f / (float)DK);
                else
                    ka[j] = Af[j].x * Af[j].x;
                mob_left(m0, ka[j], Wf[j].x, kn[j] * mr * (1.f / (float)DK));
            }
            gs.x *= Af[j].x;
            gs.y *= Af[j].y;
            if ((j & 3) == 3) {
                rescale4(m0);
                if constexpr (DIAG) rescale4(m1);
            }
        }
        if (vact) {
            if constexpr (DIAG) {
                segA[w * DK + ch] = make_float4(m0[0], m0[1], m0[2], m0[3]);
                segA[w * DK + ch + 1] = make_float4(m1[0], m1[1], m1[2], m1[3]);
            } else if (lane == 0) {
                segA[w * DK] = make_float4(m0[0], m0[1], m0[2], m0[3]);
            }
            *reinterpret_cast<float2*>(segG + w * DK + ch) = gs;
        }
    }
    __syncthreads();

    // ---- carry into the block; decay before it (Gs) and after it (Gt) within the chunk -------
    float n0, d0, n1 = 0.f, d1 = 1.f;
    float2 Gs = make_float2(1.f, 1.f), Gt = make_float2(1.f, 1.f);
    {
        const size_t cidx = ((size_t)g * H + h) * CF::NCHAN;
        if constexpr (DIAG) {
            float2 z0 = a.carry[cidx + ch], z1 = a.carry[cidx + ch + 1];
#pragma unroll
            for (int b = 0; b < NB - 1; ++b)
                if (b < w) {
                    z0 = mat_vec(segA[b * DK + ch], z0);
                    z1 = mat_vec(segA[b * DK + ch + 1], z1);
                }
            n0 = z0.x; d0 = z0.y; n1 = z1.x; d1 = z1.y;
        } else {
            float2 z = a.carry[cidx];
#pragma unroll
            for (int b = 0; b < NB - 1; ++b)
                if (b < w) z = mat_vec(segA[b * DK], z);
            n0 = z.x; d0 = z.y;
        }
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const float2 gg = *reinterpret_cast<const float2*>(segG + b * DK + ch);
            if (b < w) { Gs.x *= gg.x; Gs.y *= gg.y; }
            if (b > w) { Gt.x *= gg.x; Gt.y *= gg.y; }
        }
    }

    // ---- replay (eqs. chunk-gain-local-prefix, chunk-gain-emission): G_t k_t per channel of the
    // pair, G = p_hat (diagonal) or beta (isotropic) ------------------------------------------
    float2 pk[SL];
#pragma unroll
    for (int j = 0; j < SL; ++j) {
        const int t = SL * w + j;
        if constexpr (DIAG) {
            const float mr = s_mr[t];
            const float nn0 = fmaf(Af[j].x * Af[j].x, n0, Wf[j].x * d0);  // p_hat d
            const float nn1 = fmaf(Af[j].y * Af[j].y, n1, Wf[j].y * d1);
            pk[j] = make_float2(nn0 * Kf[j].x * __builtin_amdgcn_rcpf(d0),
                                nn1 * Kf[j].y * __builtin_amdgcn_rcpf(d1));
            if constexpr (LAYER) {
                if (a.in.beta_eff) {  // k^T kappa = z / (r + z), z = sum_i p_hat_i k_i^2
                    const float z = wave_sum(vact ? fmaf(pk[j].x, Kf[j].x, pk[j].y * Kf[j].y)
                                                  : 0.f);
                    if (lane == 0 && j < Lw)
                        a.in.beta_eff[(size_t)(c0 + t) * H + h] = z / (s_r[t] + z);
                }
            }
            d0 = fmaf(Kf[j].x * Kf[j].x * mr, nn0, d0);
            d1 = fmaf(Kf[j].y * Kf[j].y * mr, nn1, d1);
            n0 = nn0;
            n1 = nn1;
            if ((j & 3) == 3) {
                rescale2(n0, d0);
                rescale2(n1, d1);
            }
        } else {
            const float nn = fmaf(ka[j], n0, Wf[j].x * d0);  // b_hat d
            const float beta = nn * __builtin_amdgcn_rcpf(fmaf(d0, s_r[t], nn * kn[j]));
            pk[j] = make_float2(beta * Kf[j].x, beta * Kf[j].y);
            if constexpr (LAYER) {
                if (a.in.beta_eff && lane == 0 && j < Lw)  // k^T (beta k)
                    a.in.beta_eff[(size_t)(c0 + t) * H + h] = beta * kn[j];
            }
            d0 = fmaf(kn[j] * s_mr[t] * (1.f / (float)DK), nn, d0);
            n0 = nn;
            if ((j & 3) == 3) rescale2(n0, d0);
        }
    }
    if (w == NW - 1 && last && a.P_T) {  // the final variances n / d
        if constexpr (DIAG) {
            if (vact)
                *reinterpret_cast<float2*>(a.P_T + (size_t)nh * DK + ch) =
                    make_float2(n0 / d0, n1 / d1);
        } else if (lane == 0) {
            a.P_T[nh] = n0 / d0;
        }
    }

    // ---- P_tail^T = (gamma_C / gamma_s) G_s k_s (record, fragment order); gamma_C -----------
    {
        float px[SL], py[SL];
        float2 Q = Gt;
#pragma unroll
        for (int j = SL - 1; j >= 0; --j) {
            px[j] = pk[j].x * Q.x;
            py[j] = pk[j].y * Q.y;
            Q.x *= Af[j].x;
            Q.y *= Af[j].y;
        }
        if (vact) {
            constexpr int E = Frag<MT, C>::KF / 4;
#pragma unroll
            for (int e = 0; e < SL; e += E) {
                storeN<MT, E>(gPt + frag_off<MT, C>(ch, SL * w + e), px + e);
                storeN<MT, E>(gPt + frag_off<MT, C>(ch + 1, SL * w + e), py + e);
            }
            if (w == 0) {
                float2 gc = make_float2(1.f, 1.f);
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    const float2 gg = *reinterpret_cast<const float2*>(segG + b * DK + ch);
                    gc.x *= gg.x;
                    gc.y *= gg.y;
                }
                *reinterpret_cast<float2*>(gC + ch) = gc;
            }
        }
    }

    // ---- diagonal blocks: operands referenced to the block midpoint ---------------------------
    // F_t = prod_{8 <= j <= t} alpha_j (t >= 8), 1 / prod_{t < j <= 7} alpha_j (t < 8);
    // K_t F_t and G_s k_s / F_s give F_t / F_s = prod_{s < j <= t} alpha_j.
    if (vact) {
        float2 b = make_float2(1.f, 1.f);
#pragma unroll
        for (int j = SL / 2 - 1; j >= 0; --j) {
            const int t = SL * w + j;
            const float fx = sat_rcp(b.x), fy = sat_rcp(b.y);
            st2<MT>(Ka + t * LDK + ch, Kf[j].x * fx, Kf[j].y * fy);
            st2<MT>(Qa + t * LDK + ch, Qf[j].x * fx, Qf[j].y * fy);
            st2<MT>(Pa + t * LDK + ch, pk[j].x * b.x, pk[j].y * b.y);
            b.x *= Af[j].x;
            b.y *= Af[j].y;
        }
        float2 f = make_float2(1.f, 1.f);
#pragma unroll
        for (int j = SL / 2; j < SL; ++j) {
            const int t = SL * w + j;
            f.x *= Af[j].x;
            f.y *= Af[j].y;
            st2<MT>(Ka + t * LDK + ch, Kf[j].x * f.x, Kf[j].y * f.y);
            st2<MT>(Qa + t * LDK + ch, Qf[j].x * f.x, Qf[j].y * f.y);
            st2<MT>(Pa + t * LDK + ch, pk[j].x * sat_rcp(f.x), pk[j].y * sat_rcp(f.y));
        }
    }
    __syncthreads();

    auto lblk = [&](int b, int c) { return Lf + (b * (b + 1) / 2 + c) * 16 * LDL; };

    // ---- diagonal blocks of M (-> L, float32) and of A_qk (kept in registers) ----------------
    floatx4 aqd;
    {
        floatx4 tacc, qacc;
        pair_prod<MT, DK, LDK>(Ka, Qa, Pa, w, w, nullptr, lane, tacc, qacc);
        float* lb = lblk(w, w);
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
            const int row = 4 * lg + rr;
            const float cdiag = DIAG ? s_r[SL * w + row] + tacc[rr] : 1.f;
            lb[row * LDL + li] = row > li ? tacc[rr] : (row == li ? cdiag : 0.f);
            aqd[rr] = row >= li ? qacc[rr] : 0.f;
        }
    }
    __syncthreads();

    // ---- blocks off the diagonal: rows referenced to their block's start, columns to their
    // block's end, the decay of the blocks between applied to the column side -----------------
    if (vact) {
        float2 P = make_float2(1.f, 1.f);
#pragma unroll
        for (int j = 0; j < SL; ++j) {
            const int t = SL * w + j;
            P.x *= Af[j].x;
            P.y *= Af[j].y;
            st2<MT>(Ka + t * LDK + ch, Kf[j].x * P.x, Kf[j].y * P.y);
            st2<MT>(Qa + t * LDK + ch, Qf[j].x * P.x, Qf[j].y * P.y);
        }
        float2 Q = make_float2(1.f, 1.f);
#pragma unroll
        for (int j = SL - 1; j >= 0; --j) {
            st2<MT>(Pa + (SL * w + j) * LDK + ch, pk[j].x * Q.x, pk[j].y * Q.y);
            Q.x *= Af[j].x;
            Q.y *= Af[j].y;
        }
        if (NB == 4 && w == 0)  // decay of blocks 1 and 2 (pair (3, 0))
            *reinterpret_cast<float2*>(rho + ch) =
                make_float2(segG[DK + ch] * segG[2 * DK + ch],
                            segG[DK + ch + 1] * segG[2 * DK + ch + 1]);
    }
    __syncthreads();

    // pairs (ib, jb) per wave: 0: (1,0) (3,0); 1: (2,1) (3,1); 2: (3,2) (2,0); 3: the diagonal
    // blocks of L^-1
    static_assert(NB == 4 && NW == 4, "block schedule written for four 16-token blocks");
    floatx4 aqo[2];
    int oib[2] = {0, 0}, ojb[2] = {0, 0};
    if (w < 3) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int ib = u == 0 ? w + 1 : (w == 2 ? 2 : 3);
            const int jb = u == 0 ? w : (w == 0 ? 0 : (w == 1 ? 1 : 0));
            const float* rs = (ib - jb == 1) ? nullptr
                              : (ib - jb == 3 ? rho : segG + (jb + 1) * DK);
            floatx4 tacc, qacc;
            pair_prod<MT, DK, LDK>(Ka, Qa, Pa, ib, jb, rs, lane, tacc, qacc);
            float* lb = lblk(ib, jb);
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) lb[(4 * lg + rr) * LDL + li] = tacc[rr];
            aqo[u] = qacc;
            oib[u] = ib;
            ojb[u] = jb;
        }
    } else {
        // Row i of A_bb = L_bb^-1 solves a^T L_bb = e_i^T: a_i = 1 / L_ii, and going down the
        // rows m = i, i-1, ..., 0 every finished a_m adds a_m L_m,k to the sums of the k < m
        // (right-looking backward substitution). Lane (b, i) takes row i of block b.
        const int b = lane >> 4, i = li;
        const float* Lb = lblk(b, b);
        float sacc[16], y[16];
#pragma unroll
        for (int kq = 0; kq < 16; ++kq) sacc[kq] = 0.f;
#pragma unroll
        for (int mq = 15; mq >= 0; --mq) {
            float cur[16];
#pragma unroll
            for (int v4 = 0; v4 < (mq + 4) / 4; ++v4) {
                const float4 q4 = *reinterpret_cast<const float4*>(Lb + mq * LDL + 4 * v4);
                cur[4 * v4] = q4.x; cur[4 * v4 + 1] = q4.y;
                cur[4 * v4 + 2] = q4.z; cur[4 * v4 + 3] = q4.w;
            }
            const float ym = ((mq == i ? 1.f : 0.f) - sacc[mq]) * __builtin_amdgcn_rcpf(cur[mq]);
            y[mq] = mq > i ? 0.f : ym;
#pragma unroll
            for (int kq = 0; kq < mq; ++kq) sacc[kq] = fmaf(y[mq], cur[kq], sacc[kq]);
        }
        float* ab = Ai + b * 16 * LDL + i * LDL;
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4)
            *reinterpret_cast<float4*>(ab + 4 * v4) =
                make_float4(y[4 * v4], y[4 * v4 + 1], y[4 * v4 + 2], y[4 * v4 + 3]);
    }
    __syncthreads();

    // ---- L^-1 by columns of blocks (float32 MFMA): wave c takes block column c,
    // Li_bc = -A_bb sum_{c <= j < b} L_bj Li_jc, Li_cc = A_cc. A_qk and L^-1 are staged in the
    // operand area (now free) and written out in fragment order -------------------------------
    MT* Aqs = Ka;  // [C][LDC]
    MT* Lis = Qa;  // [C][LDC]
    {
        // A_qk: row block w (diagonal tile here, the off-diagonal tiles of this wave below,
        // zeros right of the diagonal)
        auto put = [&](MT* dst, int ib, int jb, floatx4 v) {
#pragma unroll
            for (int rr = 0; rr < 4; ++rr)
                dst[(16 * ib + 4 * lg + rr) * LDC + 16 * jb + li] = from_f32<MT>(v[rr]);
        };
        put(Aqs, w, w, aqd);
        for (int jb = w + 1; jb < NB; ++jb) put(Aqs, w, jb, zero4());
        if (w < 3) {
            put(Aqs, oib[0], ojb[0], aqo[0]);
            put(Aqs, oib[1], ojb[1], aqo[1]);
        }
        const int c = w;
        floatx4 lt[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            if (b < c) {
                lt[b] = zero4();
            } else if (b == c) {
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) lt[b][rr] = Ai[(c * 16 + 4 * lg + rr) * LDL + li];
            } else {
                floatx4 acc = zero4();
#pragma unroll
                for (int j = 0; j < NB; ++j)
                    if (j >= c && j < b)
                        acc = mma16_f32(acc,
                                        *reinterpret_cast<const float4*>(lblk(b, j) + li * LDL +
                                                                         4 * lg),
                                        lt[j]);
                const floatx4 t = mma16_f32(
                    zero4(), *reinterpret_cast<const float4*>(Ai + (b * 16 + li) * LDL + 4 * lg),
                    acc);
                lt[b][0] = -t[0]; lt[b][1] = -t[1]; lt[b][2] = -t[2]; lt[b][3] = -t[3];
            }
            put(Lis, b, c, lt[b]);
        }
    }
    __syncthreads();
    copy_frag_order<MT, C, C, NTH>(gAq, Aqs, LDC, tid);
    copy_frag_order<MT, C, C, NTH>(gLi, Lis, LDC, tid);
    __syncthreads();

    // ---- K_bar = gamma (.) k and Q_bar = gamma (.) q (decay since the chunk start), staged in
    // the operand area and written out in fragment order --------------------------------------
    if (vact) {
        float2 P = Gs;
#pragma unroll
        for (int j = 0; j < SL; ++j) {
            const int t = SL * w + j;
            P.x *= Af[j].x;
            P.y *= Af[j].y;
            st2<MT>(Ka + t * LDK + ch, Kf[j].x * P.x, Kf[j].y * P.y);
            st2<MT>(Qa + t * LDK + ch, Qf[j].x * P.x, Qf[j].y * P.y);
        }
    }
    __syncthreads();
    copy_frag_order<MT, C, DK, NTH>(gKb, Ka, LDK, tid);
    copy_frag_order<MT, C, DK, NTH>(gQb, Qa, LDK, tid);
}

template <class TI, class CF>
__global__ __launch_bounds__(NTH) void prep_kernel(PrepArgs a)
{
    prep_body<TI, CF, false>(a);
}

// bf16: two workgroups per CU, as the plain prep (the LDS allows two; the layer maps must not
// push the registers past that)
template <class TI, class CF>
__global__ __launch_bounds__(NTH) __attribute__((amdgpu_waves_per_eu(sizeof(TI) == 2 ? 2 : 1)))
void prep_layer_kernel(PrepArgs a)
{
    prep_body<TI, CF, true>(a);
}

// ------------------------------------------------------------------------------------------
// 4. walk: the memory state through the chunks of one (sequence, head, value tile)
// ------------------------------------------------------------------------------------------
template <class TI, int DK_, int DV_>
struct WalkCfg {
    using MT = typename OpOf<TI>::type;
    static constexpr int DK = DK_, DV = DV_;
    static constexpr int BV = DV >= 32 ? 32 : DV;  // value columns per workgroup
    static constexpr int NV = DV / BV;
    static constexpr int NNT = BV / 16, NKT = DK / 16, NST = NKT * NNT;
    static constexpr int SPW = (NST + NW - 1) / NW;  // S tiles per wave: x = SPW w + j
    // tiles of a wave share their P_tail rows when the key tile is constant over NNT tiles
    static constexpr bool SHARE = SPW % NNT == 0;
    static constexpr int PPW = SHARE ? SPW / NNT : SPW;
    static constexpr int PAD = 16 / (int)sizeof(MT);
    static constexpr int LDK = DK + PAD, LDC = C + PAD;
    static constexpr int LDO = BV + 16 / (int)sizeof(TI);
    static constexpr size_t OFF_SMT = 0;                                       // S^T [BV][LDK]
    static constexpr size_t OFF_XT = al16((size_t)BV * LDK * sizeof(MT));      // X^T [BV][LDC]
    static constexpr size_t OFF_RT = OFF_XT + al16((size_t)BV * LDC * sizeof(MT));  // R^T
    static constexpr size_t OFF_O = OFF_RT + al16((size_t)BV * LDC * sizeof(MT));   // O [C][LDO]
    static constexpr size_t OFF_V = OFF_O + al16((size_t)C * LDO * sizeof(TI));     // V [C][LDO]
    static constexpr size_t TOTAL = al16(OFF_V + (size_t)C * LDO * sizeof(TI));
    // V tile of a chunk in 16-byte pieces: VPC per row; wave w moves the 16 rows of its own row
    // block (16 VPC pieces), VPW per lane
    static constexpr int VPC = BV * (int)sizeof(TI) / 16;
    static constexpr int VPW = (16 * VPC + 63) / 64;
};

struct WalkArgs {
    const void* v;
    const float* S0;
    void* o;
    float* S_T;
    const char* ops;
    const int32_t* order;  // packed batches: sequences, longest first (nullptr: in order)
    ChunkMap cm;
    int H;
    float scale;
    uint32_t bytes_v;
};

template <class TI, class CF>
__global__ __launch_bounds__(NTH) void walk_kernel(WalkArgs a)
{
    using MT = typename CF::MT;
    using Rec = OpRec<MT, CF::DK>;
    using FK = Frag<MT, CF::DK>;
    using FC = Frag<MT, C>;
    constexpr int DK = CF::DK, DV = CF::DV, BV = CF::BV, NNT = CF::NNT, NST = CF::NST;
    constexpr int SPW = CF::SPW, PPW = CF::PPW, LDK = CF::LDK, LDC = CF::LDC, LDO = CF::LDO;
    constexpr int NSK = FK::NS, NSC = FC::NS;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    MT* SmT = (MT*)(smem + CF::OFF_SMT);
    MT* XT = (MT*)(smem + CF::OFF_XT);
    MT* RT = (MT*)(smem + CF::OFF_RT);
    TI* Ost = (TI*)(smem + CF::OFF_O);
    TI* Vt = (TI*)(smem + CF::OFF_V);

    // block -> (sequence-head slot, value tile): the NV tiles of one head get block indices
    // congruent modulo 8, so round-robin dispatch puts them on one XCD, where they share the L2
    // copy of the head's chunk records
    const int H = a.H, NH = a.cm.N * H;
    const int xcd = (int)(blockIdx.x % 8), rest = (int)(blockIdx.x / 8);
    const int vt = rest % CF::NV, slot = (rest / CF::NV) * 8 + xcd;
    if (slot >= NH) return;
    const int n = a.order ? a.order[slot / H] : slot / H;
    const int h = slot % H;
    if (n < 0 || n >= a.cm.N) return;
    const int nh = n * H + h, col0 = vt * BV;
    int t0, t1, g0, nch;
    seq_span(a.cm, n, t0, t1);
    seq_chunks<C>(a.cm, n, t0, t1, g0, nch);
    TI* go = (TI*)a.o;

    const int tid = threadIdx.x, lane = tid & 63, li = lane & 15, lg = lane >> 4;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);

    // S tiles of this wave: x = SPW w + j -> key tile x / NNT, value tile x % NNT
    floatx4 Sacc[SPW];
#pragma unroll
    for (int j = 0; j < SPW; ++j) {
        const int x = SPW * w + j;
        Sacc[j] = zero4();
        if (x < NST) {
            const int ik = x / NNT, nt = x % NNT;
            if (a.S0) {
                const float* src = a.S0 + (size_t)nh * DK * DV;
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    Sacc[j][rr] = src[(size_t)(16 * ik + 4 * lg + rr) * DV + col0 + 16 * nt + li];
            }
            store4<MT>(SmT + (16 * nt + li) * LDK + 16 * ik + 4 * lg, Sacc[j][0], Sacc[j][1],
                       Sacc[j][2], Sacc[j][3]);
        }
    }

    const rsrc_t rv = make_rsrc(a.v, a.bytes_v);
    constexpr uint32_t es = sizeof(TI);
    const uint32_t rowv = (uint32_t)H * DV * es;
    const uint32_t colv = ((uint32_t)h * DV + col0) * es;
    auto recp = [&](int m) -> const char* {
        const int mm = min(m, max(nch - 1, 0));
        return a.ops + ((size_t)(g0 + mm) * H + h) * Rec::BYTES;
    };
    auto key_tile = [&](int p) { return min(CF::SHARE ? SPW * w / NNT + p : (SPW * w + p) / NNT,
                                            CF::NKT - 1); };

    // operands of the next chunk, loaded one step ahead of their use (fragment order: one
    // contiguous piece per lane)
    typename FK::V kf[NSK], qf[NSK];
    typename FC::V lf[NSC], af[NSC], pf[PPW][NSC];
    float4 gc[PPW];
    uint4 vraw[CF::VPW];  // the wave's rows of the chunk's V tile, 16 bytes per piece
    auto load1 = [&](int m) {
        const char* rec = recp(m);
        const MT* Kb = (const MT*)(rec + Rec::OFF_KB);
        const MT* Qb = (const MT*)(rec + Rec::OFF_QB);
#pragma unroll
        for (int s = 0; s < NSK; ++s) {
            kf[s] = FK::ld(frag_piece<MT, DK>(Kb, w, s, lane));
            qf[s] = FK::ld(frag_piece<MT, DK>(Qb, w, s, lane));
        }
        const uint32_t c0 = (uint32_t)(t0 + min(m, max(nch - 1, 0)) * C);
#pragma unroll
        for (int u = 0; u < CF::VPW; ++u) {
            const int q = min(lane + 64 * u, 16 * CF::VPC - 1);
            const uint32_t r = (uint32_t)(16 * w + q / CF::VPC);
            const uint32_t cb = (uint32_t)(q % CF::VPC) * 16;
            vraw[u] = __builtin_bit_cast(
                uint4, __builtin_amdgcn_raw_buffer_load_b128(rv, (int)((c0 + r) * rowv + colv + cb),
                                                             0, 0));
        }
    };
    // the wave's V rows to LDS: every wave reads only the rows it writes, and LDS operations of
    // one wave run in order, so no barrier is needed between this and their use
    auto store_v = [&]() {
#pragma unroll
        for (int u = 0; u < CF::VPW; ++u) {
            const int q = lane + 64 * u;
            if (q < 16 * CF::VPC)
                *reinterpret_cast<uint4*>(Vt + (16 * w + q / CF::VPC) * LDO +
                                          (q % CF::VPC) * (16 / es)) = vraw[u];
        }
    };
    auto load2 = [&](int m) {
        const MT* Li = (const MT*)(recp(m) + Rec::OFF_LI);
#pragma unroll
        for (int s = 0; s < NSC; ++s) lf[s] = FC::ld(frag_piece<MT, C>(Li, w, s, lane));
    };
    auto load3 = [&](int m) {
        const char* rec = recp(m);
        const MT* Aq = (const MT*)(rec + Rec::OFF_AQ);
#pragma unroll
        for (int s = 0; s < NSC; ++s) af[s] = FC::ld(frag_piece<MT, C>(Aq, w, s, lane));
#pragma unroll
        for (int p = 0; p < PPW; ++p) {
            const int ik = key_tile(p);
            const MT* Pt = (const MT*)(rec + Rec::OFF_PT);
#pragma unroll
            for (int s = 0; s < NSC; ++s) pf[p][s] = FC::ld(frag_piece<MT, C>(Pt, ik, s, lane));
            gc[p] = *reinterpret_cast<const float4*>((const float*)(rec + Rec::OFF_GC) +
                                                     16 * ik + 4 * lg);
        }
    };
    if (nch > 0) {
        load1(0);
        load2(0);
        load3(0);
    }
    __syncthreads();

    constexpr int VE = 16 / (int)sizeof(TI), VPR = BV / VE;
    for (int m = 0; m < nch; ++m) {
        const int c0 = t0 + m * C, L = min(C, t1 - c0);
        // the previous chunk's O rows (a full chunk: only the last one can be partial)
        if (m > 0) {
            const int cp = c0 - C;
            for (int idx = tid; idx < C * VPR; idx += NTH) {
                const int t = idx / VPR, e = (idx % VPR) * VE;
                *reinterpret_cast<uint4*>(go + ((size_t)(cp + t) * H + h) * DV + col0 + e) =
                    *reinterpret_cast<const uint4*>(Ost + t * LDO + e);
            }
        }
        store_v();
        // ---- X = V - K_bar S (to LDS, transposed); Q_bar S kept for the output --------------
        floatx4 Oacc[NNT];
        {
            typename FK::V sf[NNT][NSK];
#pragma unroll
            for (int nt = 0; nt < NNT; ++nt)
#pragma unroll
                for (int s = 0; s < NSK; ++s)
                    sf[nt][s] = FK::ld(SmT + (16 * nt + li) * LDK + FK::KF * s + (FK::KF / 4) * lg);
#pragma unroll
            for (int nt = 0; nt < NNT; ++nt) {
                floatx4 xacc = zero4();
                Oacc[nt] = zero4();
#pragma unroll
                for (int s = 0; s < NSK; ++s) {
                    xacc = FK::mma(xacc, kf[s], sf[nt][s]);
                    Oacc[nt] = FK::mma(Oacc[nt], qf[s], sf[nt][s]);
                }
                // rows past the end of the sequence hold another sequence's V or stale data:
                // every row is read (no divergent reads), then masked
                float vr[4], xv[4];
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    vr[rr] = to_f32(Vt[(16 * w + 4 * lg + rr) * LDO + 16 * nt + li]);
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    xv[rr] = (16 * w + 4 * lg + rr < L ? vr[rr] : 0.f) - xacc[rr];
                store4<MT>(XT + (16 * nt + li) * LDC + 16 * w + 4 * lg, xv[0], xv[1], xv[2],
                           xv[3]);
            }
        }
        load1(m + 1);
        __syncthreads();
        // ---- R = L^-1 X ---------------------------------------------------------------------
        {
            typename FC::V xf[NNT][NSC];
#pragma unroll
            for (int nt = 0; nt < NNT; ++nt)
#pragma unroll
                for (int s = 0; s < NSC; ++s)
                    xf[nt][s] = FC::ld(XT + (16 * nt + li) * LDC + FC::KF * s + (FC::KF / 4) * lg);
#pragma unroll
            for (int nt = 0; nt < NNT; ++nt) {
                floatx4 racc = zero4();
#pragma unroll
                for (int s = 0; s < NSC; ++s) racc = FC::mma(racc, lf[s], xf[nt][s]);
                store4<MT>(RT + (16 * nt + li) * LDC + 16 * w + 4 * lg, racc[0], racc[1],
                           racc[2], racc[3]);
            }
        }
        load2(m + 1);
        __syncthreads();
        // ---- O = scale (Q_bar S + A_qk R); S <- gamma_C (.) S + P_tail^T R --------------------
        {
            typename FC::V rf[NNT][NSC];
#pragma unroll
            for (int nt = 0; nt < NNT; ++nt)
#pragma unroll
                for (int s = 0; s < NSC; ++s)
                    rf[nt][s] = FC::ld(RT + (16 * nt + li) * LDC + FC::KF * s + (FC::KF / 4) * lg);
#pragma unroll
            for (int nt = 0; nt < NNT; ++nt) {
#pragma unroll
                for (int s = 0; s < NSC; ++s) Oacc[nt] = FC::mma(Oacc[nt], af[s], rf[nt][s]);
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    Ost[(16 * w + 4 * lg + rr) * LDO + 16 * nt + li] =
                        from_f32<TI>(a.scale * Oacc[nt][rr]);
            }
#pragma unroll
            for (int j = 0; j < SPW; ++j) {
                const int x = SPW * w + j;
                if (x < NST) {
                    // with SHARE, x % NNT = j % NNT is known at compile time
                    const int ik = x / NNT, nt = CF::SHARE ? j % NNT : x % NNT;
                    const int p = CF::SHARE ? j / NNT : j;
                    Sacc[j][0] *= gc[p].x;
                    Sacc[j][1] *= gc[p].y;
                    Sacc[j][2] *= gc[p].z;
                    Sacc[j][3] *= gc[p].w;
                    static_assert(NNT <= 2, "value tiles of at most 32 columns");
                    // with SHARE the value tile is a compile-time index into rf; otherwise the
                    // fragment is read again from LDS (a runtime index would put rf in scratch)
#pragma unroll
                    for (int s = 0; s < NSC; ++s) {
                        typename FC::V rv;
                        if constexpr (CF::SHARE)
                            rv = rf[j % NNT][s];
                        else
                            rv = FC::ld(RT + (16 * nt + li) * LDC + FC::KF * s + (FC::KF / 4) * lg);
                        Sacc[j] = FC::mma(Sacc[j], pf[p][s], rv);
                    }
                    store4<MT>(SmT + (16 * nt + li) * LDK + 16 * ik + 4 * lg, Sacc[j][0],
                               Sacc[j][1], Sacc[j][2], Sacc[j][3]);
                }
            }
        }
        load3(m + 1);
        __syncthreads();
    }

    if (nch > 0) {  // the last chunk's O rows
        const int cp = t0 + (nch - 1) * C, Lp = t1 - cp;
        for (int idx = tid; idx < C * VPR; idx += NTH) {
            const int t = idx / VPR, e = (idx % VPR) * VE;
            if (t < Lp)
                *reinterpret_cast<uint4*>(go + ((size_t)(cp + t) * H + h) * DV + col0 + e) =
                    *reinterpret_cast<const uint4*>(Ost + t * LDO + e);
        }
    }
    if (a.S_T) {
        float* dst = a.S_T + (size_t)nh * DK * DV;
#pragma unroll
        for (int j = 0; j < SPW; ++j) {
            const int x = SPW * w + j;
            if (x < NST) {
                const int ik = x / NNT, nt = x % NNT;
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    dst[(size_t)(16 * ik + 4 * lg + rr) * DV + col0 + 16 * nt + li] = Sacc[j][rr];
            }
        }
    }
}

// ------------------------------------------------------------------------------------------
// host side
// ------------------------------------------------------------------------------------------

// Workspace of one forward call.
struct WsMap {
    size_t choff, order, summ, carry, ops, total;
    int maxch;
};

inline WsMap ws_map(int variant, bool packed, int N, int B, int T, int H, int dk,
                    size_t rec_bytes)
{
    WsMap m;
    m.maxch = packed ? (int)((size_t)B * T / C + (size_t)N) : N * ((T + C - 1) / C);
    const size_t nchan = variant == 0 ? (size_t)dk : 1;
    size_t off = 0;
    m.choff = off;
    off += packed ? al256((size_t)(N + 1) * 4) : 0;
    m.order = off;
    off += packed ? al256((size_t)N * 4) : 0;
    m.summ = off;
    off += al256((size_t)m.maxch * H * nchan * 16);
    m.carry = off;
    off += al256((size_t)m.maxch * H * nchan * 8);
    m.ops = off;
    off += (size_t)m.maxch * H * rec_bytes;
    m.total = off;
    return m;
}

size_t rec_bytes(kdn_dtype_t dtype, int dk);

template <class K>
hipError_t set_lds(K* kernel, size_t bytes)
{
    if (bytes <= 64 * 1024) return hipSuccess;
    return hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)bytes);
}

template <class TI, bool LAYER, int DK, int DV, int VARIANT, bool APC>
hipError_t run_t(const FwdCall& fc, hipStream_t st)
{
    using VC = VarCfg<TI, DK, VARIANT, APC>;
    using PC = PrepCfg<TI, DK, VARIANT, APC>;
    using WC = WalkCfg<TI, DK, DV>;
    using MT = typename OpOf<TI>::type;
    const SeqArgs& sa = fc.sa;
    const bool packed = sa.cu_seqlens != nullptr;
    const WsMap wm = ws_map(VARIANT, packed, sa.N, sa.B, sa.T, sa.H, DK, OpRec<MT, DK>::BYTES);
    if (wm.maxch == 0) return hipSuccess;
    char* ws = (char*)fc.workspace;
    hipError_t e;
    ChunkMap cm;
    cm.cu = sa.cu_seqlens;
    cm.choff = packed ? (const int32_t*)(ws + wm.choff) : nullptr;
    cm.N = sa.N;
    cm.T = sa.T;
    cm.ntok = sa.B * sa.T;
    cm.maxch = wm.maxch;
    const int32_t* order = nullptr;
    if (packed) {
        if ((e = launch_chunk_table(sa.cu_seqlens, sa.N, cm.ntok, C, wm.maxch,
                                    (int32_t*)(ws + wm.choff), st)) != hipSuccess)
            return e;
        if (sa.N <= ORDER_MAX) {
            if ((e = launch_order(sa.cu_seqlens, sa.N, cm.ntok, (int32_t*)(ws + wm.order), st)) !=
                hipSuccess)
                return e;
            order = (const int32_t*)(ws + wm.order);
        }
    }
    InArgs in;
    in.q = fc.q; in.k = fc.k; in.alpha = fc.alpha; in.omega = fc.omega; in.r = fc.r;
    const size_t ntok = (size_t)sa.B * sa.T * sa.H;
    in.bytes_k = (uint32_t)(ntok * DK * sizeof(TI));
    in.bytes_h = (uint32_t)(ntok * sizeof(TI));
    in.H = sa.H;
    in.mu = fc.mu;
    in.mu_t = fc.ly.mu_t;
    in.beta_eff = fc.ly.beta_eff;
    in.r_min = fc.ly.r_min;
    in.preact = fc.ly.preact;
    in.qknorm = fc.ly.qknorm;
    float4* summ = (float4*)(ws + wm.summ);
    float2* carry = (float2*)(ws + wm.carry);
    const dim3 cgrid((unsigned)((size_t)wm.maxch * sa.H));
    if constexpr (LAYER)
        hipLaunchKernelGGL((summary_layer_kernel<TI, VC>), cgrid, dim3(NTH), 0, st, in, cm, summ);
    else
        hipLaunchKernelGGL((summary_kernel<TI, VC>), cgrid, dim3(NTH), 0, st, in, cm, summ);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_carry_scan(summ, fc.P0, cm, C, sa.H, VC::NCHAN, carry, fc.P_T, st)) !=
        hipSuccess)
        return e;
    void (*prep)(PrepArgs) = [] {
        if constexpr (LAYER) return &prep_layer_kernel<TI, PC>;
        else return &prep_kernel<TI, PC>;
    }();
    static bool attr_done = false;
    if (!attr_done) {
        if ((e = set_lds(prep, PC::TOTAL)) != hipSuccess) return e;
        if ((e = set_lds(walk_kernel<TI, WC>, WC::TOTAL)) != hipSuccess) return e;
        attr_done = true;
    }
    PrepArgs pa;
    pa.in = in;
    pa.cm = cm;
    pa.carry = carry;
    pa.ops = ws + wm.ops;
    pa.P_T = fc.P_T;
    hipLaunchKernelGGL(prep, cgrid, dim3(NTH), PC::TOTAL, st, pa);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    WalkArgs wa;
    wa.v = fc.v;
    wa.S0 = fc.S0;
    wa.o = fc.o;
    wa.S_T = fc.S_T;
    wa.ops = ws + wm.ops;
    wa.order = order;
    wa.cm = cm;
    wa.H = sa.H;
    wa.scale = fc.scale;
    wa.bytes_v = (uint32_t)(ntok * DV * sizeof(TI));
    const size_t nh8 = ((size_t)sa.N * sa.H + 7) / 8 * 8;
    hipLaunchKernelGGL((walk_kernel<TI, WC>), dim3((unsigned)(nh8 * WC::NV)), dim3(NTH),
                       WC::TOTAL, st, wa);
    return hipGetLastError();
}

template <class TI, bool LAYER, int DK, int DV>
hipError_t run_variant(const FwdCall& fc, hipStream_t st)
{
    if (fc.variant == 0) return run_t<TI, LAYER, DK, DV, 0, true>(fc, st);
    if (fc.apc) return run_t<TI, LAYER, DK, DV, 1, true>(fc, st);
    return run_t<TI, LAYER, DK, DV, 1, false>(fc, st);
}

template <class TI, bool LAYER, int DK>
hipError_t run_dv(const FwdCall& fc, hipStream_t st)
{
    switch (fc.dv) {
    case 16: return run_variant<TI, LAYER, DK, 16>(fc, st);
    case 32: return run_variant<TI, LAYER, DK, 32>(fc, st);
    case 64: return run_variant<TI, LAYER, DK, 64>(fc, st);
    case 128: return run_variant<TI, LAYER, DK, 128>(fc, st);
    }
    return hipErrorInvalidValue;
}

template <class TI, bool LAYER>
hipError_t run_forward(const FwdCall& fc, hipStream_t st)
{
    switch (fc.dk) {
    case 16: return run_dv<TI, LAYER, 16>(fc, st);
    case 32: return run_dv<TI, LAYER, 32>(fc, st);
    case 64: return run_dv<TI, LAYER, 64>(fc, st);
    case 128: return run_dv<TI, LAYER, 128>(fc, st);
    }
    return hipErrorInvalidValue;
}

// instantiated once per dtype and mode, in kdn_fwd_{bf16,f32}.hip (the plain forward) and
// kdn_fwd_layer_{bf16,f32}.hip (the layer forward)
extern template hipError_t run_forward<float, false>(const FwdCall& fc, hipStream_t st);
extern template hipError_t run_forward<bf16, false>(const FwdCall& fc, hipStream_t st);
extern template hipError_t run_forward<float, true>(const FwdCall& fc, hipStream_t st);
extern template hipError_t run_forward<bf16, true>(const FwdCall& fc, hipStream_t st);

}  // namespace fwd
}  // namespace kdn
