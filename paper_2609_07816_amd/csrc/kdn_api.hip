// C ABI of libkdn: host-side argument checks and dispatch to the HIP launchers.
// Nothing here reads device memory or synchronizes; every check uses host-visible sizes only.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "kdn_internal.h"

#include <cstdint>
#include <initializer_list>
#include <utility>

namespace {

// Scratch of kdn_forward_diag_noalloc: one copy per GPU, held until the process ends. Host code
// never uses the array's name as an address: the device address of each GPU's copy comes from
// hipGetSymbolAddress (scratch_on_current_device).
constexpr size_t SCRATCH_BYTES = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[SCRATCH_BYTES];
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};

thread_local char g_err[512] = "";

kdn_status_t fail(kdn_status_t st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

kdn_status_t fail(kdn_status_t st, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return st;
}

kdn_status_t ok()
{
    g_err[0] = '\0';
    return KDN_OK;
}

bool head_ok(int d) { return d == 16 || d == 32 || d == 64 || d == 128; }

size_t esize(kdn_dtype_t dt) { return dt == KDN_F32 ? 4 : 2; }

// Byte ranges [p, p + n) and [q, q + m) overlap.
bool overlaps(const void* p, size_t n, const void* q, size_t m)
{
    if (!p || !q || n == 0 || m == 0) return false;
    const char *a = (const char*)p, *b = (const char*)q;
    return a < b + m && b < a + n;
}

kdn_status_t hip_status(hipError_t e, const char* what)
{
    if (e == hipSuccess) return ok();
    return fail(KDN_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Device address of the current device's copy of `scratch`, looked up once per device.
kdn_status_t scratch_on_current_device(void** out)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(KDN_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= MAX_DEVICES)
        return fail(KDN_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, MAX_DEVICES);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(KDN_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                        hipGetErrorString(e));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return KDN_OK;
}

// Tensors whose innermost dimension is d_k or d_v are read and written in 16-byte pieces: each
// must start at a 16-byte boundary (null pointers are skipped).
kdn_status_t check_aligned(std::initializer_list<std::pair<const void*, const char*>> ptrs)
{
    for (const auto& p : ptrs)
        if (p.first && ((uintptr_t)p.first & 15))
            return fail(KDN_ERR_INVALID_ARG, "%s must be 16-byte aligned", p.second);
    return KDN_OK;
}

// Shared validation of the forward / gain argument sets.
kdn_status_t check_seq(const int32_t* cu, int32_t N, int32_t B, int32_t T, int32_t H)
{
    if (B <= 0 || T <= 0 || H <= 0 || N <= 0)
        return fail(KDN_ERR_INVALID_ARG, "sizes must be positive (N=%d B=%d T=%d H=%d)", N, B,
                    T, H);
    if (cu && B != 1)
        return fail(KDN_ERR_INVALID_ARG, "packed batches (cu_seqlens) need B == 1, got %d", B);
    if (!cu && N != B)
        return fail(KDN_ERR_INVALID_ARG, "without cu_seqlens N must equal B (N=%d B=%d)", N, B);
    if ((int64_t)B * T * H > ((int64_t)1 << 31) / 128)
        return fail(KDN_ERR_INVALID_ARG, "B*T*H too large for 32-bit token indexing");
    return KDN_OK;
}

kdn_status_t check_forward(int variant, const void* q, const void* k, const void* v,
                           const void* alpha, const void* omega, const void* r, const float* S0,
                           const float* P0, const void* o, const float* S_T, const float* P_T,
                           const int32_t* cu, int32_t N, int32_t B, int32_t T, int32_t H,
                           int32_t dk, int32_t dv, kdn_dtype_t dtype, int apc, float mu,
                           float scale, int32_t chunk, void* ws, size_t ws_bytes)
{
    if (!q || !k || !v || !alpha || !omega || !r || !o)
        return fail(KDN_ERR_INVALID_ARG, "null required pointer (q, k, v, alpha, omega, r, o)");
    if (dtype != KDN_F32 && dtype != KDN_BF16)
        return fail(KDN_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
    kdn_status_t st = check_seq(cu, N, B, T, H);
    if (st != KDN_OK) return st;
    if (!head_ok(dk) || !head_ok(dv))
        return fail(KDN_ERR_UNSUPPORTED, "dk=%d dv=%d: head sizes must be 16, 32, 64 or 128", dk,
                    dv);
    if (!(mu > 0.f) || !(scale > 0.f))
        return fail(KDN_ERR_INVALID_ARG, "mu and scale must be positive (mu=%g scale=%g)", mu,
                    scale);
    st = check_aligned({{q, "q"}, {k, "k"}, {v, "v"}, {(variant == 0 || apc) ? alpha : nullptr,
                        "alpha"}, {variant == 0 ? omega : nullptr, "omega"}, {o, "o"},
                        {S0, "S0"}, {S_T, "S_T"}, {variant == 0 ? P0 : nullptr, "P0"},
                        {variant == 0 ? P_T : nullptr, "P_T"}});
    if (st != KDN_OK) return st;
    if (!kdn::chunked_supported(chunk))
        return fail(KDN_ERR_UNSUPPORTED, "chunk=%d: the forward runs chunks of 64 tokens (pass 0 "
                    "or 64)", chunk);
    const size_t ntok = (size_t)B * T * H, es = esize(dtype);
    const size_t nk = ntok * dk * es, nv = ntok * dv * es;
    if (nk >= ((size_t)1 << 31) || nv >= ((size_t)1 << 31))
        return fail(KDN_ERR_UNSUPPORTED, "each input tensor must be smaller than 2 GiB (the "
                    "forward addresses it with 32-bit offsets)");
    const size_t na = (variant == 0 || apc) ? nk : ntok * es;
    const size_t nw = variant == 0 ? nk : ntok * es;
    const void* ins[6] = {q, k, v, alpha, omega, r};
    const size_t insz[6] = {nk, nk, nv, na, nw, ntok * es};
    for (int i = 0; i < 6; ++i)
        if (overlaps(o, nv, ins[i], insz[i]))
            return fail(KDN_ERR_INVALID_ARG, "output o overlaps input %d", i);
    const size_t ns = (size_t)N * H * dk * dv * 4;
    const size_t np = (size_t)N * H * (variant == 0 ? dk : 1) * 4;
    if (S_T && S_T != S0 && overlaps(S_T, ns, S0, ns))
        return fail(KDN_ERR_INVALID_ARG, "S_T partially overlaps S0 (only exact aliasing is "
                                         "allowed)");
    if (P_T && P_T != P0 && overlaps(P_T, np, P0, np))
        return fail(KDN_ERR_INVALID_ARG, "P_T partially overlaps P0");
    if (overlaps(o, nv, S_T, ns) || overlaps(o, nv, P_T, np))
        return fail(KDN_ERR_INVALID_ARG, "o overlaps the state outputs");
    const size_t need = kdn::chunked_workspace_bytes(variant, cu != nullptr, N, B, T, H, dk, dtype);
    if (need > 0 && (!ws || ws_bytes < need))
        return fail(KDN_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                    ws ? ws_bytes : (size_t)0);
    return KDN_OK;
}

kdn::FwdCall fwd_call(int variant, int apc, const void* q, const void* k, const void* v,
                      const void* alpha, const void* omega, const void* r, const float* S0,
                      const float* P0, void* o, float* S_T, float* P_T, const int32_t* cu,
                      int32_t N, int32_t B, int32_t T, int32_t H, int32_t dk, int32_t dv,
                      kdn_dtype_t dtype, float mu, float scale, void* ws)
{
    kdn::FwdCall c;
    c.variant = variant; c.apc = apc;
    c.q = q; c.k = k; c.v = v; c.alpha = alpha; c.omega = omega; c.r = r;
    c.S0 = S0; c.P0 = P0; c.o = o; c.S_T = S_T; c.P_T = P_T;
    c.sa = {cu, N, B, T, H};
    c.dk = dk; c.dv = dv; c.dtype = dtype; c.mu = mu; c.scale = scale;
    c.workspace = ws;
    c.ly = kdn::LayerOpts{false, 0, 0, 0.f, nullptr, nullptr};
    return c;
}

// Layer options from the caller's struct (NULL: all off). Checks the values and that the
// per-token arrays of `rows` entries neither alias nor overlap the call's other buffers.
kdn_status_t layer_opts(const kdn_layer_opts* p, size_t rows, size_t es,
                        const void* const* bufs, const size_t* sizes, int nbufs,
                        kdn::LayerOpts* out)
{
    *out = kdn::LayerOpts{false, 0, 0, 0.f, nullptr, nullptr};
    if (!p) return KDN_OK;
    if (p->gates_preact && !(p->r_min > 0.f))
        return fail(KDN_ERR_INVALID_ARG, "r_min must be positive with gates_preact (r_min=%g)",
                    p->r_min);
    for (int i = 0; i < nbufs; ++i) {
        if (overlaps(p->beta_eff, rows * 4, bufs[i], sizes[i]))
            return fail(KDN_ERR_INVALID_ARG, "beta_eff overlaps argument buffer %d", i);
    }
    if (overlaps(p->beta_eff, rows * 4, p->mu_t, rows * es))
        return fail(KDN_ERR_INVALID_ARG, "beta_eff overlaps mu_t");
    out->preact = p->gates_preact ? 1 : 0;
    out->qknorm = p->qk_l2norm ? 1 : 0;
    out->r_min = p->r_min;
    out->mu_t = p->mu_t;
    out->beta_eff = p->beta_eff;
    out->on = out->preact || out->qknorm || out->mu_t || out->beta_eff;
    return KDN_OK;
}

}  // namespace

extern "C" {

const char* kdn_status_string(kdn_status_t s)
{
    switch (s) {
    case KDN_OK: return "KDN_OK";
    case KDN_ERR_INVALID_ARG: return "KDN_ERR_INVALID_ARG";
    case KDN_ERR_UNSUPPORTED: return "KDN_ERR_UNSUPPORTED";
    case KDN_ERR_WORKSPACE: return "KDN_ERR_WORKSPACE";
    case KDN_ERR_HIP: return "KDN_ERR_HIP";
    }
    return "KDN_ERR_UNKNOWN";
}

const char* kdn_last_error(void) { return g_err; }

const char* kdn_version(void) { return "kdn-mi355x 0.1 (gfx950)"; }

size_t kdn_forward_workspace_bytes(int32_t variant, int32_t N, int32_t B, int32_t T, int32_t H,
                                   int32_t dk, int32_t dv, kdn_dtype_t dtype, int32_t packed,
                                   int32_t chunk)
{
    if (N <= 0 || B <= 0 || T <= 0 || H <= 0 || !head_ok(dk) || !head_ok(dv)) return 0;
    if (dtype != KDN_F32 && dtype != KDN_BF16) return 0;
    if (variant != 0 && variant != 1) return 0;
    if (!kdn::chunked_supported(chunk)) return 0;
    (void)dv;
    return kdn::chunked_workspace_bytes(variant, packed != 0, N, B, T, H, dk, dtype);
}

size_t kdn_gain_workspace_bytes(int32_t variant, int32_t N, int32_t B, int32_t T, int32_t H,
                                int32_t dk)
{
    if (N <= 0 || B <= 0 || T <= 0 || H <= 0) return 0;
    return kdn::gain_workspace_bytes(variant, N, B, T, H, dk);
}

kdn_status_t kdn_forward_diag(const void* q, const void* k, const void* v, const void* alpha,
                              const void* omega, const void* r, const float* S0, const float* P0,
                              void* o, float* S_T, float* P_T, const int32_t* cu_seqlens,
                              int32_t N, int32_t B, int32_t T, int32_t H, int32_t dk, int32_t dv,
                              kdn_dtype_t dtype, float mu, float scale, int32_t chunk,
                              void* workspace, size_t workspace_bytes, void* stream)
{
    kdn_status_t st = check_forward(0, q, k, v, alpha, omega, r, S0, P0, o, S_T, P_T, cu_seqlens,
                                    N, B, T, H, dk, dv, dtype, 1, mu, scale, chunk, workspace,
                                    workspace_bytes);
    if (st != KDN_OK) return st;
    return hip_status(kdn::launch_chunked(fwd_call(0, 1, q, k, v, alpha, omega, r, S0, P0, o, S_T,
                                                   P_T, cu_seqlens, N, B, T, H, dk, dv, dtype,
                                                   mu, scale, workspace),
                                          (hipStream_t)stream),
                      "kdn_forward_diag launch");
}

kdn_status_t kdn_forward_diag_noalloc(const void* q, const void* k, const void* v,
                                      const void* alpha, const void* omega, const void* r,
                                      const float* S0, const float* P0, void* o, float* S_T,
                                      float* P_T, const int32_t* cu_seqlens, int32_t N,
                                      int32_t B, int32_t T, int32_t H, int32_t dk, int32_t dv,
                                      kdn_dtype_t dtype, float mu, float scale, void* stream)
{
    const size_t need = (B > 0 && T > 0 && H > 0 && N > 0 && head_ok(dk) && head_ok(dv) &&
                         (dtype == KDN_F32 || dtype == KDN_BF16))
                            ? kdn::chunked_workspace_bytes(0, cu_seqlens != nullptr, N, B, T, H,
                                                           dk, dtype)
                            : 0;
    if (need > SCRATCH_BYTES)
        return fail(KDN_ERR_UNSUPPORTED, "kdn_forward_diag_noalloc: these sizes need %zu bytes of "
                    "scratch, more than its fixed %zu (use kdn_forward_diag with a workspace)",
                    need, SCRATCH_BYTES);
    void* ws = nullptr;
    kdn_status_t st = scratch_on_current_device(&ws);
    if (st != KDN_OK) return st;
    st = check_forward(0, q, k, v, alpha, omega, r, S0, P0, o, S_T, P_T, cu_seqlens, N, B, T, H,
                       dk, dv, dtype, 1, mu, scale, 0, ws, SCRATCH_BYTES);
    if (st != KDN_OK) return st;
    return hip_status(kdn::launch_chunked(fwd_call(0, 1, q, k, v, alpha, omega, r, S0, P0, o, S_T,
                                                   P_T, cu_seqlens, N, B, T, H, dk, dv, dtype,
                                                   mu, scale, ws),
                                          (hipStream_t)stream),
                      "kdn_forward_diag_noalloc launch");
}

kdn_status_t kdn_forward_iso(const void* q, const void* k, const void* v, const void* alpha,
                             const void* omega, const void* r, const float* S0, const float* P0,
                             void* o, float* S_T, float* P_T, const int32_t* cu_seqlens,
                             int32_t N, int32_t B, int32_t T, int32_t H, int32_t dk, int32_t dv,
                             kdn_dtype_t dtype, int32_t alpha_per_channel, float mu, float scale,
                             int32_t chunk, void* workspace, size_t workspace_bytes,
                             void* stream)
{
    const int apc = alpha_per_channel ? 1 : 0;
    kdn_status_t st = check_forward(1, q, k, v, alpha, omega, r, S0, P0, o, S_T, P_T, cu_seqlens,
                                    N, B, T, H, dk, dv, dtype, apc, mu, scale, chunk, workspace,
                                    workspace_bytes);
    if (st != KDN_OK) return st;
    return hip_status(kdn::launch_chunked(fwd_call(1, apc, q, k, v, alpha, omega, r, S0, P0, o,
                                                   S_T, P_T, cu_seqlens, N, B, T, H, dk, dv,
                                                   dtype, mu, scale, workspace),
                                          (hipStream_t)stream),
                      "kdn_forward_iso launch");
}

kdn_status_t kdn_forward_layer(int32_t variant, const void* q, const void* k, const void* v,
                               const void* alpha, const void* omega, const void* r,
                               const float* S0, const float* P0, void* o, float* S_T, float* P_T,
                               const int32_t* cu_seqlens, int32_t N, int32_t B, int32_t T,
                               int32_t H, int32_t dk, int32_t dv, kdn_dtype_t dtype,
                               int32_t alpha_per_channel, float mu, float scale,
                               const kdn_layer_opts* opts, void* workspace,
                               size_t workspace_bytes, void* stream)
{
    if (variant != 0 && variant != 1)
        return fail(KDN_ERR_INVALID_ARG, "variant must be 0 (diagonal) or 1 (isotropic)");
    const int apc = (variant == 0 || alpha_per_channel) ? 1 : 0;
    kdn_status_t st = check_forward(variant, q, k, v, alpha, omega, r, S0, P0, o, S_T, P_T,
                                    cu_seqlens, N, B, T, H, dk, dv, dtype, apc, mu, scale, 0,
                                    workspace, workspace_bytes);
    if (st != KDN_OK) return st;
    const size_t rows = (size_t)B * T * H, es = esize(dtype);
    const size_t nk = rows * dk * es, nv = rows * dv * es;
    const void* bufs[10] = {q, k, v, alpha, omega, r, o, S_T, P_T, workspace};
    const size_t bsz[10] = {nk, nk, nv, apc ? nk : rows * es, variant == 0 ? nk : rows * es,
                            rows * es, nv, (size_t)N * H * dk * dv * 4,
                            (size_t)N * H * (variant == 0 ? dk : 1) * 4, workspace_bytes};
    kdn::LayerOpts ly;
    st = layer_opts(opts, rows, es, bufs, bsz, 10, &ly);
    if (st != KDN_OK) return st;
    kdn::FwdCall fc = fwd_call(variant, apc, q, k, v, alpha, omega, r, S0, P0, o, S_T, P_T,
                               cu_seqlens, N, B, T, H, dk, dv, dtype, mu, scale, workspace);
    fc.ly = ly;
    return hip_status(kdn::launch_chunked(fc, (hipStream_t)stream), "kdn_forward_layer launch");
}

static kdn_status_t decode_common(int32_t variant, const void* q, const void* k, const void* v,
                                  const void* alpha, const void* omega, const void* r, float* S,
                                  float* P, const int32_t* slot_idx, void* o, int32_t R,
                                  int32_t num_slots, int32_t H, int32_t dk, int32_t dv,
                                  kdn_dtype_t dtype, int32_t alpha_per_channel, float mu,
                                  float scale, const kdn_layer_opts* opts, void* stream)
{
    if (variant != 0 && variant != 1)
        return fail(KDN_ERR_INVALID_ARG, "variant must be 0 (diagonal) or 1 (isotropic)");
    if (!q || !k || !v || !alpha || !omega || !r || !S || !P || !o)
        return fail(KDN_ERR_INVALID_ARG, "null required pointer");
    if (dtype != KDN_F32 && dtype != KDN_BF16)
        return fail(KDN_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
    if (R < 0 || num_slots <= 0 || H <= 0)
        return fail(KDN_ERR_INVALID_ARG, "bad sizes (R=%d num_slots=%d H=%d)", R, num_slots, H);
    if (!slot_idx && R > num_slots)
        return fail(KDN_ERR_INVALID_ARG, "without slot_idx R (%d) must not exceed num_slots (%d)",
                    R, num_slots);
    if (!head_ok(dk) || !head_ok(dv))
        return fail(KDN_ERR_UNSUPPORTED, "dk=%d dv=%d: head sizes must be 16, 32, 64 or 128", dk,
                    dv);
    if (!(mu > 0.f) || !(scale > 0.f))
        return fail(KDN_ERR_INVALID_ARG, "mu and scale must be positive");
    kdn_status_t sa = check_aligned(
        {{q, "q"}, {k, "k"}, {v, "v"}, {(variant == 0 || alpha_per_channel) ? alpha : nullptr,
          "alpha"}, {variant == 0 ? omega : nullptr, "omega"}, {o, "o"}, {S, "S"},
         {variant == 0 ? P : nullptr, "P"}});
    if (sa != KDN_OK) return sa;
    const size_t es = esize(dtype), rows = (size_t)R * H;
    const size_t ns = (size_t)num_slots * H * dk * dv * 4;
    const size_t np = (size_t)num_slots * H * (variant == 0 ? dk : 1) * 4;
    const void* ins[6] = {q, k, v, alpha, omega, r};
    const size_t insz[6] = {rows * dk * es, rows * dk * es, rows * dv * es,
                            rows * ((variant == 0 || alpha_per_channel) ? dk : 1) * es,
                            rows * (variant == 0 ? dk : 1) * es, rows * es};
    for (int i = 0; i < 6; ++i)
        if (overlaps(o, rows * dv * es, ins[i], insz[i]))
            return fail(KDN_ERR_INVALID_ARG, "output o overlaps input %d", i);
    if (overlaps(o, rows * dv * es, S, ns) || overlaps(o, rows * dv * es, P, np) ||
        overlaps(S, ns, P, np))
        return fail(KDN_ERR_INVALID_ARG, "o, S and P must not overlap");
    const void* bufs[9] = {q, k, v, alpha, omega, r, o, S, P};
    const size_t bsz[9] = {insz[0], insz[1], insz[2], insz[3], insz[4], insz[5],
                           rows * dv * es, ns, np};
    kdn::LayerOpts ly;
    kdn_status_t st = layer_opts(opts, rows, es, bufs, bsz, 9, &ly);
    if (st != KDN_OK) return st;
    return hip_status(kdn::launch_decode(variant, q, k, v, alpha, omega, r, S, P, slot_idx, o, R,
                                         num_slots, H, dk, dv, dtype,
                                         alpha_per_channel ? 1 : 0, mu, scale, ly,
                                         (hipStream_t)stream),
                      "kdn_decode_step launch");
}

kdn_status_t kdn_decode_step(int32_t variant, const void* q, const void* k, const void* v,
                             const void* alpha, const void* omega, const void* r, float* S,
                             float* P, const int32_t* slot_idx, void* o, int32_t R,
                             int32_t num_slots, int32_t H, int32_t dk, int32_t dv,
                             kdn_dtype_t dtype, int32_t alpha_per_channel, float mu, float scale,
                             void* stream)
{
    return decode_common(variant, q, k, v, alpha, omega, r, S, P, slot_idx, o, R, num_slots, H,
                         dk, dv, dtype, alpha_per_channel, mu, scale, nullptr, stream);
}

kdn_status_t kdn_decode_step_layer(int32_t variant, const void* q, const void* k, const void* v,
                                   const void* alpha, const void* omega, const void* r, float* S,
                                   float* P, const int32_t* slot_idx, void* o, int32_t R,
                                   int32_t num_slots, int32_t H, int32_t dk, int32_t dv,
                                   kdn_dtype_t dtype, int32_t alpha_per_channel, float mu,
                                   float scale, const kdn_layer_opts* opts, void* stream)
{
    return decode_common(variant, q, k, v, alpha, omega, r, S, P, slot_idx, o, R, num_slots, H,
                         dk, dv, dtype, alpha_per_channel, mu, scale, opts, stream);
}

kdn_status_t kdn_forward_kam(const void* q, const void* k, const void* v, const void* alpha,
                             const void* omega, const void* r, const float* S0, const float* P0,
                             void* o, float* S_T, float* P_T, const int32_t* cu_seqlens,
                             int32_t N, int32_t B, int32_t T, int32_t H, int32_t dk, int32_t dv,
                             kdn_dtype_t dtype, float scale, void* stream)
{
    if (!q || !k || !v || !alpha || !omega || !r || !o)
        return fail(KDN_ERR_INVALID_ARG, "null required pointer (q, k, v, alpha, omega, r, o)");
    if (dtype != KDN_F32 && dtype != KDN_BF16)
        return fail(KDN_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
    kdn_status_t st = check_seq(cu_seqlens, N, B, T, H);
    if (st != KDN_OK) return st;
    if (!head_ok(dk) || !head_ok(dv))
        return fail(KDN_ERR_UNSUPPORTED, "dk=%d dv=%d: head sizes must be 16, 32, 64 or 128", dk,
                    dv);
    if (!(scale > 0.f)) return fail(KDN_ERR_INVALID_ARG, "scale must be positive (%g)", scale);
    st = check_aligned({{q, "q"}, {k, "k"}, {v, "v"}, {alpha, "alpha"}, {omega, "omega"},
                        {o, "o"}, {S0, "S0"}, {P0, "P0"}, {S_T, "S_T"}, {P_T, "P_T"}});
    if (st != KDN_OK) return st;
    const size_t rows = (size_t)B * T * H, es = esize(dtype);
    const size_t nk = rows * dk * es, nv = rows * dv * es;
    const void* ins[6] = {q, k, v, alpha, omega, r};
    const size_t insz[6] = {nk, nk, nv, nk, nk, rows * es};
    for (int i = 0; i < 6; ++i)
        if (overlaps(o, nv, ins[i], insz[i]))
            return fail(KDN_ERR_INVALID_ARG, "output o overlaps input %d", i);
    const size_t ns = (size_t)N * H * dk * dv * 4, np = (size_t)N * H * dk * dk * 4;
    if (S_T && S_T != S0 && overlaps(S_T, ns, S0, ns))
        return fail(KDN_ERR_INVALID_ARG, "S_T partially overlaps S0");
    if (P_T && P_T != P0 && overlaps(P_T, np, P0, np))
        return fail(KDN_ERR_INVALID_ARG, "P_T partially overlaps P0");
    if (overlaps(o, nv, S_T, ns) || overlaps(o, nv, P_T, np) || overlaps(S_T, ns, P_T, np))
        return fail(KDN_ERR_INVALID_ARG, "o, S_T and P_T must not overlap");
    kdn::SeqArgs sa = {cu_seqlens, N, B, T, H};
    return hip_status(kdn::launch_kam(q, k, v, alpha, omega, r, S0, P0, o, S_T, P_T, sa, dk, dv,
                                      dtype, scale, (hipStream_t)stream),
                      "kdn_forward_kam launch");
}

size_t kdn_backward_workspace_bytes(int32_t variant, int32_t N, int32_t B, int32_t T, int32_t H,
                                    int32_t dk, int32_t dv, int32_t packed)
{
    if (N <= 0 || B <= 0 || T <= 0 || H <= 0 || !head_ok(dk) || !head_ok(dv)) return 0;
    if (variant != 0 && variant != 1) return 0;
    return kdn::backward_workspace_bytes(variant, packed != 0, N, B, T, H, dk, dv);
}

kdn_status_t kdn_backward(int32_t variant, const void* q, const void* k, const void* v,
                          const void* alpha, const void* omega, const void* r, const float* S0,
                          const float* P0, const int32_t* cu_seqlens, int32_t N, int32_t B,
                          int32_t T, int32_t H, int32_t dk, int32_t dv, kdn_dtype_t dtype,
                          int32_t alpha_per_channel, float mu, float scale, const void* dO,
                          const float* dS_T, const float* dP_T, float* dq, float* dk_out,
                          float* dv_out, float* dalpha, float* domega, float* dr, float* dS0,
                          float* dP0, void* workspace, size_t workspace_bytes, void* stream)
{
    if (variant != 0 && variant != 1)
        return fail(KDN_ERR_INVALID_ARG, "variant must be 0 (diagonal) or 1 (isotropic)");
    if (!q || !k || !v || !alpha || !omega || !r)
        return fail(KDN_ERR_INVALID_ARG, "null required input (q, k, v, alpha, omega, r)");
    if (!dq || !dk_out || !dv_out || !dalpha || !domega || !dr)
        return fail(KDN_ERR_INVALID_ARG, "null required gradient (dq, dk, dv, dalpha, domega, dr)");
    if (dtype != KDN_F32 && dtype != KDN_BF16)
        return fail(KDN_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
    kdn_status_t st = check_seq(cu_seqlens, N, B, T, H);
    if (st != KDN_OK) return st;
    if (!head_ok(dk) || !head_ok(dv))
        return fail(KDN_ERR_UNSUPPORTED, "dk=%d dv=%d: head sizes must be 16, 32, 64 or 128", dk,
                    dv);
    if (!(mu > 0.f) || !(scale > 0.f))
        return fail(KDN_ERR_INVALID_ARG, "mu and scale must be positive (mu=%g scale=%g)", mu,
                    scale);
    const int apc = (variant == 0 || alpha_per_channel) ? 1 : 0;
    st = check_aligned({{q, "q"}, {k, "k"}, {v, "v"}, {apc ? alpha : nullptr, "alpha"},
                        {variant == 0 ? omega : nullptr, "omega"}, {dO, "dO"}, {S0, "S0"},
                        {variant == 0 ? P0 : nullptr, "P0"}, {dS_T, "dS_T"},
                        {variant == 0 ? dP_T : nullptr, "dP_T"}, {dq, "dq"}, {dk_out, "dk"},
                        {dv_out, "dv"}, {apc ? dalpha : nullptr, "dalpha"},
                        {variant == 0 ? domega : nullptr, "domega"}, {dS0, "dS0"},
                        {variant == 0 ? dP0 : nullptr, "dP0"}});
    if (st != KDN_OK) return st;
    const size_t rows = (size_t)B * T * H, es = esize(dtype);
    const size_t pc = variant == 0 ? (size_t)dk : 1;
    // every buffer the call reads or writes, with its extent; the gradients may overlap none
    const void* bufs[14] = {q, k, v, alpha, omega, r, dO, S0, P0, dS_T, dP_T, cu_seqlens,
                            workspace, nullptr};
    const size_t bsz[14] = {rows * dk * es, rows * dk * es, rows * dv * es,
                            rows * (apc ? dk : 1) * es, rows * pc * es, rows * es, rows * dv * es,
                            (size_t)N * H * dk * dv * 4, (size_t)N * H * pc * 4,
                            (size_t)N * H * dk * dv * 4, (size_t)N * H * pc * 4,
                            cu_seqlens ? (size_t)(N + 1) * 4 : 0, workspace_bytes, 0};
    float* outs[8] = {dq, dk_out, dv_out, dalpha, domega, dr, dS0, dP0};
    const size_t osz[8] = {rows * dk * 4, rows * dk * 4, rows * dv * 4, rows * (apc ? dk : 1) * 4,
                           rows * pc * 4, rows * 4, (size_t)N * H * dk * dv * 4,
                           (size_t)N * H * pc * 4};
    for (int o = 0; o < 8; ++o) {
        for (int i = 0; i < 13; ++i)
            if (overlaps(outs[o], osz[o], bufs[i], bsz[i]))
                return fail(KDN_ERR_INVALID_ARG, "gradient %d overlaps argument buffer %d", o, i);
        for (int o2 = 0; o2 < o; ++o2)
            if (overlaps(outs[o], osz[o], outs[o2], osz[o2]))
                return fail(KDN_ERR_INVALID_ARG, "gradients %d and %d overlap", o2, o);
    }
    const size_t nk = rows * dk * es, nv = rows * dv * es;
    if (nk >= ((size_t)1 << 31) || nv >= ((size_t)1 << 31))
        return fail(KDN_ERR_UNSUPPORTED, "each input tensor must be smaller than 2 GiB");
    const size_t need = kdn::backward_workspace_bytes(variant, cu_seqlens != nullptr, N, B, T, H,
                                                      dk, dv);
    if (!workspace || workspace_bytes < need)
        return fail(KDN_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                    workspace ? workspace_bytes : (size_t)0);
    kdn::BwdCall bc;
    bc.variant = variant; bc.apc = apc;
    bc.q = q; bc.k = k; bc.v = v; bc.alpha = alpha; bc.omega = omega; bc.r = r; bc.dO = dO;
    bc.S0 = S0; bc.P0 = P0; bc.dS_T = dS_T; bc.dP_T = dP_T;
    bc.gq = dq; bc.gk = dk_out; bc.gv = dv_out; bc.galpha = dalpha; bc.gomega = domega;
    bc.gr = dr; bc.gS0 = dS0; bc.gP0 = dP0;
    bc.sa = {cu_seqlens, N, B, T, H};
    bc.dk = dk; bc.dv = dv; bc.dtype = dtype; bc.mu = mu; bc.scale = scale;
    bc.workspace = workspace;
    return hip_status(kdn::launch_backward(bc, (hipStream_t)stream), "kdn_backward launch");
}

static kdn_status_t gain_common(int variant, const void* k, const void* alpha, const void* omega,
                                const void* r, const float* P0, float* gain_out, float* phat_out,
                                float* P_T, const int32_t* cu, int32_t N, int32_t B, int32_t T,
                                int32_t H, int32_t dk, kdn_dtype_t dtype, int apc, float mu,
                                void* ws, size_t ws_bytes, void* stream)
{
    if (!k || !alpha || !omega || !r || !gain_out)
        return fail(KDN_ERR_INVALID_ARG, "null required pointer (k, alpha, omega, r, gain)");
    if (dtype != KDN_F32 && dtype != KDN_BF16)
        return fail(KDN_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
    kdn_status_t st = check_seq(cu, N, B, T, H);
    if (st != KDN_OK) return st;
    if (!head_ok(dk)) return fail(KDN_ERR_UNSUPPORTED, "dk=%d: must be 16, 32, 64 or 128", dk);
    if (!(mu > 0.f)) return fail(KDN_ERR_INVALID_ARG, "mu must be positive (mu=%g)", mu);
    st = check_aligned({{k, "k"}, {(variant == 0 || apc) ? alpha : nullptr, "alpha"},
                        {variant == 0 ? omega : nullptr, "omega"},
                        {variant == 0 ? gain_out : nullptr, "gain"},
                        {variant == 0 ? phat_out : nullptr, "phat"},
                        {variant == 0 ? P0 : nullptr, "P0"},
                        {variant == 0 ? P_T : nullptr, "P_T"}});
    if (st != KDN_OK) return st;
    if ((size_t)B * T * H * dk * esize(dtype) >= ((size_t)1 << 31))
        return fail(KDN_ERR_UNSUPPORTED, "each input tensor must be smaller than 2 GiB (the "
                    "chunk summaries address it with 32-bit offsets)");
    const size_t need = kdn::gain_workspace_bytes(variant, N, B, T, H, dk);
    if (!ws || ws_bytes < need)
        return fail(KDN_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                    ws ? ws_bytes : (size_t)0);
    kdn::SeqArgs sa = {cu, N, B, T, H};
    return hip_status(kdn::launch_gain(variant, k, alpha, omega, r, P0, gain_out, phat_out, P_T,
                                       sa, dk, dtype, apc, mu, ws, (hipStream_t)stream),
                      "kdn_gain launch");
}

kdn_status_t kdn_gain_diag(const void* k, const void* alpha, const void* omega, const void* r,
                           const float* P0, float* kappa_out, float* phat_out, float* P_T,
                           const int32_t* cu_seqlens, int32_t N, int32_t B, int32_t T,
                           int32_t H, int32_t dk, kdn_dtype_t dtype, float mu, void* workspace,
                           size_t workspace_bytes, void* stream)
{
    return gain_common(0, k, alpha, omega, r, P0, kappa_out, phat_out, P_T, cu_seqlens, N, B, T,
                       H, dk, dtype, 1, mu, workspace, workspace_bytes, stream);
}

kdn_status_t kdn_gain_iso(const void* k, const void* alpha, const void* omega, const void* r,
                          const float* P0, float* beta_out, float* bhat_out, float* P_T,
                          const int32_t* cu_seqlens, int32_t N, int32_t B, int32_t T, int32_t H,
                          int32_t dk, kdn_dtype_t dtype, int32_t alpha_per_channel, float mu,
                          void* workspace, size_t workspace_bytes, void* stream)
{
    return gain_common(1, k, alpha, omega, r, P0, beta_out, bhat_out, P_T, cu_seqlens, N, B, T,
                       H, dk, dtype, alpha_per_channel ? 1 : 0, mu, workspace, workspace_bytes,
                       stream);
}

}  // extern "C"
