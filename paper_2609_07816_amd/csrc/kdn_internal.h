// Internal declarations shared by the HIP sources of libkdn (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "kdn.h"

namespace kdn {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------------------------------
// element access: inputs are float32 or bf16, computed in float32
// ------------------------------------------------------------------------------------------
__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }

template <class T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }

template <class T>
__device__ __forceinline__ float ldf(const T* p, size_t i) { return to_f32(p[i]); }

// ------------------------------------------------------------------------------------------
// wavefront reductions (64 lanes)
// ------------------------------------------------------------------------------------------
// Sum over the 64 lanes of a wave, returned to every lane (wave-uniform). All lanes must be
// active. DPP: inclusive scans inside each row of 16 lanes (row_shr 1, 2, 4, 8), then each row
// takes the running total of the rows before it (row_bcast 15 into rows 1 and 3, row_bcast 31
// into rows 2 and 3), so lane 63 holds the total; lanes whose DPP source falls outside their row
// read 0.
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_add(float x)
{
    return x + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
                                             0, __builtin_bit_cast(int, x), CTRL, ROWS, 0xf, false));
}
// Sum over each row of 16 lanes, returned to every lane of the row: DPP quad permutations
// [1,0,3,2] and [2,3,0,1] (quads), then the half-row mirror (lane i with 7 - i: quad pairs) and
// the row mirror (lane i with 15 - i: the two halves). Every source lane is inside the row.
__device__ __forceinline__ float row16_sum(float x)
{
    x = dpp_add<0xb1, 0xf>(x);   // quad_perm [1,0,3,2]
    x = dpp_add<0x4e, 0xf>(x);   // quad_perm [2,3,0,1]
    x = dpp_add<0x141, 0xf>(x);  // row_half_mirror
    x = dpp_add<0x140, 0xf>(x);  // row_mirror
    return x;
}
__device__ __forceinline__ float wave_sum(float x)
{
    x = dpp_add<0x111, 0xf>(x);  // row_shr:1
    x = dpp_add<0x112, 0xf>(x);  // row_shr:2
    x = dpp_add<0x114, 0xf>(x);  // row_shr:4
    x = dpp_add<0x118, 0xf>(x);  // row_shr:8
    x = dpp_add<0x142, 0xa>(x);  // row_bcast:15
    x = dpp_add<0x143, 0xc>(x);  // row_bcast:31
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 63));
}

// Power-of-two rescale of a homogeneous pair (n, d): exact, keeps n/d, keeps max(|n|,|d|) in
// [0.5, 1). The Moebius states and summaries are only defined up to a positive factor.
__device__ __forceinline__ void renorm2(float& n, float& d)
{
    float m = fmaxf(fabsf(n), fabsf(d));
    int e;
    (void)frexpf(m, &e);
    if (m > 0.f && m < INFINITY) {
        n = ldexpf(n, -e);
        d = ldexpf(d, -e);
    }
}

__device__ __forceinline__ void renorm4(float& a, float& b, float& c, float& d)
{
    float m = fmaxf(fmaxf(fabsf(a), fabsf(b)), fmaxf(fabsf(c), fabsf(d)));
    int e;
    (void)frexpf(m, &e);
    if (m > 0.f && m < INFINITY) {
        a = ldexpf(a, -e);
        b = ldexpf(b, -e);
        c = ldexpf(c, -e);
        d = ldexpf(d, -e);
    }
}

// ------------------------------------------------------------------------------------------
// the mixer layer's input maps (eqs. kla-box-parameterization and iso-kla-box-parameterization):
// alpha = sigmoid(.), omega = softplus(.), r = r_min + softplus(.) of pre-activations
// ------------------------------------------------------------------------------------------
__device__ __forceinline__ float gate_sigmoid(float x)
{
    // 1 / (1 + e^-x): e^-x overflows to +inf for x < -88 and the result is then 0
    return __builtin_amdgcn_rcpf(1.f + __expf(-x));
}

__device__ __forceinline__ float gate_softplus(float x)
{
    // max(x, 0) + log1p(e^-|x|). log1p(e) for e in (0, 1] as log(u) e / (u - 1) with u = 1 + e
    // rounded (Goldberg's correction: it cancels the rounding of 1 + e), and e itself when u
    // rounds to 1.
    const float e = __expf(-fabsf(x));
    const float u = 1.f + e;
    const float l = u == 1.f ? e : __logf(u) * (e * __builtin_amdgcn_rcpf(u - 1.f));
    return fmaxf(x, 0.f) + l;
}

// Options of the layer-mode calls (kdn_forward_layer, kdn_decode_step_layer).
struct LayerOpts {
    bool on;             // any of the below (the forward then runs its layer kernels)
    int preact, qknorm;  // gates from pre-activations; q and k divided by their L2 norms
    float r_min;
    const void* mu_t;    // per-token information scale [.., H] (dtype), or nullptr
    float* beta_eff;     // k^T kappa per token [.., H] float32, or nullptr
};

// ------------------------------------------------------------------------------------------
// host-side launchers implemented in the kernel sources
// ------------------------------------------------------------------------------------------
struct SeqArgs {
    const int32_t* cu_seqlens;  // device, or nullptr
    int N, B, T, H;
};

hipError_t launch_decode(int variant, const void* q, const void* k, const void* v,
                         const void* alpha, const void* omega, const void* r, float* S, float* P,
                         const int32_t* slot_idx, void* o, int R, int num_slots, int H, int dk,
                         int dv, kdn_dtype_t dtype, int alpha_per_channel, float mu, float scale,
                         const LayerOpts& ly, hipStream_t stream);

size_t gain_workspace_bytes(int variant, int N, int B, int T, int H, int dk);
hipError_t launch_gain(int variant, const void* k, const void* alpha, const void* omega,
                       const void* r, const float* P0, float* gain_out, float* phat_out,
                       float* P_T, const SeqArgs& sa, int dk, kdn_dtype_t dtype,
                       int alpha_per_channel, float mu, void* workspace, hipStream_t stream);

// Chunked forward (kdn_fwd.hip): chunk summaries, the log-depth carry scan, the per-chunk prep
// and the walk over the chunks.
struct FwdCall {
    int variant, apc;  // 0 = diagonal, 1 = isotropic; per-channel gate (isotropic)
    const void *q, *k, *v, *alpha, *omega, *r;
    const float *S0, *P0;
    void* o;
    float *S_T, *P_T;
    SeqArgs sa;
    int dk, dv;
    kdn_dtype_t dtype;
    float mu, scale;
    void* workspace;  // chunked_workspace_bytes(...) bytes
    LayerOpts ly;
};
// Backward of the chunked forward (kdn_bwd.hip). Gradients are float32.
struct BwdCall {
    int variant, apc;
    const void *q, *k, *v, *alpha, *omega, *r, *dO;  // dO in the input dtype, or nullptr
    const float *S0, *P0, *dS_T, *dP_T;
    float *gq, *gk, *gv, *galpha, *gomega, *gr, *gS0, *gP0;
    SeqArgs sa;
    int dk, dv;
    kdn_dtype_t dtype;
    float mu, scale;
    void* workspace;  // backward_workspace_bytes(...) bytes
};
size_t backward_workspace_bytes(int variant, bool packed, int N, int B, int T, int H, int dk,
                                int dv);
hipError_t launch_backward(const BwdCall& bc, hipStream_t stream);

// Kalman Associative Memory, dense covariance (kdn_kam.hip).
hipError_t launch_kam(const void* q, const void* k, const void* v, const void* alpha,
                      const void* omega, const void* r, const float* S0, const float* P0,
                      void* o, float* S_T, float* P_T, const SeqArgs& sa, int dk, int dv,
                      kdn_dtype_t dtype, float scale, hipStream_t stream);

bool chunked_supported(int chunk);
size_t chunked_workspace_bytes(int variant, bool packed, int N, int B, int T, int H, int dk,
                               kdn_dtype_t dtype);
hipError_t launch_chunked(const FwdCall& fc, hipStream_t stream);

}  // namespace kdn
