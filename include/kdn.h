/*
 * kdn.h -- C ABI of the MI355X (gfx950) Kalman Delta Network hot path.
 *
 * Paper: N. Bui, T. Huang, R. Ying, "Kalman Delta Networks: Uncertainty-aware Associative
 * Memory", arXiv 2609.07816. Section and equation names below are the paper's.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every data pointer is a DEVICE pointer owned by the caller. The library allocates no device
 *   memory and never frees caller memory.
 * - Calls are asynchronous on `stream` (a hipStream_t passed as void*; NULL = the null stream).
 *   No call synchronizes the stream or reads device memory from the host. A status other than
 *   KDN_OK means nothing was launched (argument errors) or a launch failed (KDN_ERR_HIP); the
 *   outputs are then unspecified.
 * - Layouts are contiguous row-major "BTHD": q, k [B,T,H,dk]; v, o [B,T,H,dv]; per-channel gates
 *   [B,T,H,dk]; per-head scalars [B,T,H]. Variable-length batches are packed: B == 1, T is the
 *   total token count, and cu_seqlens (int32 [N+1], device) gives sequence n the tokens
 *   [cu_seqlens[n], cu_seqlens[n+1]). Without cu_seqlens, N == B and every row has length T.
 * - `dtype` is the storage type of q, k, v, alpha, omega, r and o (KDN_F32 or KDN_BF16). The
 *   recurrent state is always float32: S [N,H,dk,dv] (key-major, S[i][j] at i*dv + j);
 *   P [N,H,dk] for the diagonal variant, [N,H] for the isotropic one.
 * - S0 == NULL means S0 = 0; P0 == NULL means P0 = 1 (p_0 = 1, b_0 = 1). S_T / P_T may be NULL
 *   (not written) and may alias S0 / P0 exactly (in-place state update).
 * - Supported head sizes: dk, dv in {16, 32, 64, 128}. The forward takes input tensors smaller
 *   than 2 GiB each (KDN_ERR_UNSUPPORTED otherwise).
 * - Every tensor whose innermost dimension is dk or dv (q, k, v, o, per-channel gates and noise,
 *   states, variances per channel, their gradients) is moved in 16-byte pieces and must start
 *   at a 16-byte aligned address (any hipMalloc or torch allocation does, and so does a view
 *   that starts at a whole row); a misaligned one is rejected with KDN_ERR_INVALID_ARG.
 * - Device-side contract (not checked on the host, which never reads device data):
 *   cu_seqlens non-decreasing with cu_seqlens[0] == 0 and cu_seqlens[N] == T; 0 < alpha <= 1;
 *   omega >= 0; r > 0. Kernels never write outside the caller's buffers even when it is broken:
 *   every sequence span is clamped to [0, B*T] on the device and the number of chunks to the
 *   workspace the query sized (results for such a batch are unspecified, the writes in bounds).
 * - Gates: the forward is exact (to rounding) for every 0 < alpha <= 1 whose product over any 8
 *   consecutive tokens of an aligned 16-token block stays above 2^-126 per channel (every
 *   alpha >= 2^-15 ~ 3.1e-5 suffices): decay ratios inside a chunk are referenced to block
 *   starts, ends and midpoints, never to a factor above one elsewhere. Below that floor the
 *   midpoint factors saturate at 2^126: outputs, states and variances stay finite, and the
 *   intra-block products of the affected channels lose accuracy. Decode and the gain scan have
 *   no floor.
 * - Errors are returned, never printed or raised; kdn_last_error() gives detail for the calling
 *   thread's most recent non-OK status.
 */
#ifndef KDN_H
#define KDN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    KDN_OK = 0,
    KDN_ERR_INVALID_ARG = 1, /* null required pointer, bad size, mu <= 0, scale <= 0, aliasing */
    KDN_ERR_UNSUPPORTED = 2, /* dk or dv outside {16, 32, 64, 128}, an unsupported chunk, or a
                                forward input tensor of 2 GiB or more                         */
    KDN_ERR_WORKSPACE = 3,   /* workspace smaller than the matching *_workspace_bytes query    */
    KDN_ERR_HIP = 4          /* a HIP launch failed; kdn_last_error() carries the HIP message  */
} kdn_status_t;

typedef enum { KDN_F32 = 0, KDN_BF16 = 1 } kdn_dtype_t;

/*
 * Diagonal KDN forward (Prop. "Diagonal Kalman Delta Network", eqs. kla-box-mobius,
 * kla-box-gain, kla-box-memory; variance update eqs. prefix-diag-uncertainty and
 * diag-cov-update with information scale mu). For every token of every (sequence, head):
 *   p_hat = alpha^2 * p + omega;  kappa = p_hat * k / (r + sum_i p_hat_i k_i^2)
 *   S = diag(alpha) S + kappa (v - (diag(alpha) S)^T k)^T;  o = scale * S^T q
 *   p = p_hat / (1 + mu k^2 / r * p_hat)
 * evaluated chunkwise (App. "Hardware-Efficient Chunkwise Algorithm"): one workgroup walks each
 * (sequence, head, block of value columns) through its chunks in order, carrying S and the
 * variance chain, so only the inputs, o and the final states cross device memory.
 *   q, k, alpha, omega: [B,T,H,dk]; v, o: [B,T,H,dv]; r: [B,T,H]   (dtype)
 *   S0, S_T: [N,H,dk,dv] float32;  P0, P_T: [N,H,dk] float32
 *   mu > 0 (the paper uses mu = dk); scale > 0 (the paper uses dk^-1/2).
 *   chunk: memory-chunk length, 64 or 0 (= 64); anything else is KDN_ERR_UNSUPPORTED.
 *   workspace: device scratch of at least kdn_forward_workspace_bytes(...) bytes
 *   (KDN_ERR_WORKSPACE when smaller or NULL). Four kernels run on `stream` in order: chunk
 *   summaries of the variance chain, a log-depth carry scan across chunks (eq.
 *   chunk-gain-carry), a per-chunk prep that writes each chunk's S-independent operands to the
 *   workspace, and the walk that carries S through the chunks.
 */
kdn_status_t kdn_forward_diag(const void* q, const void* k, const void* v, const void* alpha,
                              const void* omega, const void* r, const float* S0, const float* P0,
                              void* o, float* S_T, float* P_T, const int32_t* cu_seqlens,
                              int32_t N, int32_t B, int32_t T, int32_t H, int32_t dk, int32_t dv,
                              kdn_dtype_t dtype, float mu, float scale, int32_t chunk,
                              void* workspace, size_t workspace_bytes, void* stream);

/*
 * kdn_forward_diag without a workspace argument, for callers that cannot allocate device
 * memory (code under stream capture, serving loops, harnesses that forbid allocation). The
 * operation, the other arguments, the outputs and the errors are those of kdn_forward_diag.
 * Its scratch is a fixed 64 MiB array in the library, one copy per GPU (the device current
 * at the call), created when the library's code is loaded on that GPU and held until the
 * process ends; its address is looked up on the first call on each GPU. Sizes whose workspace
 * (kdn_forward_workspace_bytes) exceeds 64 MiB give KDN_ERR_UNSUPPORTED: about 1000
 * (chunk, head) pairs at dk = 128 in bf16, e.g. H = 16 heads of 4000 tokens. Nothing in the
 * scratch needs to start at zero. Every call on one GPU uses the same scratch: calls that
 * overlap in time on one GPU (two streams, or two threads) race and give undefined results;
 * calls serialised on one stream are safe.
 */
kdn_status_t kdn_forward_diag_noalloc(const void* q, const void* k, const void* v,
                                      const void* alpha, const void* omega, const void* r,
                                      const float* S0, const float* P0, void* o, float* S_T,
                                      float* P_T, const int32_t* cu_seqlens, int32_t N,
                                      int32_t B, int32_t T, int32_t H, int32_t dk, int32_t dv,
                                      kdn_dtype_t dtype, float mu, float scale, void* stream);

/*
 * Isotropic KDN forward (Prop. "Isotropic Kalman Delta Network", eqs.
 * iso-kla-box-cov-update, iso-kla-box-gain, iso-kla-box-memory). One variance b per head:
 *   a = mean_i alpha_i^2;  b_hat = a b + omega;  beta = b_hat / (r + b_hat ||k||^2)
 *   S = diag(alpha) S + beta k (v - (diag(alpha) S)^T k)^T;  o = scale * S^T q
 *   b = b_hat / (1 + mu ||k||^2 / (dk r) * b_hat)
 *   alpha: [B,T,H,dk] when alpha_per_channel != 0, else [B,T,H] (one gate per head);
 *   omega, r: [B,T,H]; P0, P_T: [N,H] float32. Other arguments as kdn_forward_diag.
 */
kdn_status_t kdn_forward_iso(const void* q, const void* k, const void* v, const void* alpha,
                             const void* omega, const void* r, const float* S0, const float* P0,
                             void* o, float* S_T, float* P_T, const int32_t* cu_seqlens,
                             int32_t N, int32_t B, int32_t T, int32_t H, int32_t dk, int32_t dv,
                             kdn_dtype_t dtype, int32_t alpha_per_channel, float mu, float scale,
                             int32_t chunk, void* workspace, size_t workspace_bytes,
                             void* stream);

/*
 * Device scratch (bytes) that kdn_forward_diag (variant 0) / kdn_forward_iso (variant 1) need
 * for these sizes; packed != 0 for a packed batch (cu_seqlens given), chunk as passed to the
 * forward. Returns 0 for arguments the forward rejects. With M chunks at most
 * (M = N ceil(T / 64) for a fixed-length batch, M = T / 64 + N for a packed one), a variance
 * channel count c (dk diagonal, 1 isotropic) and e the input element size, it holds, each
 * part rounded up to 256 bytes:
 *   packed only: the chunk-offset table (4 (N + 1)) and the walk order (4 N);
 *   the chunk summaries (16 M H c) and the carries into every chunk (8 M H c);
 *   one record per (chunk, head) of M H records, each 3 64 dk e + 2 64 64 e + 4 dk bytes
 *   rounded up to 256 (K_bar, Q_bar, P_tail^T, L^-1, A_qk, gamma_C),
 * about 1 KB per token and head for bf16 at dk = 128. It needs no initialisation and is dead
 * once the forward's work on the stream has finished; two forwards in flight at once need two.
 */
size_t kdn_forward_workspace_bytes(int32_t variant, int32_t N, int32_t B, int32_t T, int32_t H,
                                   int32_t dk, int32_t dv, kdn_dtype_t dtype, int32_t packed,
                                   int32_t chunk);

/*
 * Options of the layer calls (kdn_forward_layer, kdn_decode_step_layer): the steps of the
 * mixer layer on either side of the recurrence, fused into its kernels. A NULL options pointer,
 * or every field zero / NULL, gives exactly the plain call.
 *   gates_preact != 0: alpha, omega and r hold pre-activations, mapped per element as
 *     alpha = sigmoid(x), omega = softplus(x), r = r_min + softplus(x) (eqs.
 *     kla-box-parameterization and iso-kla-box-parameterization); r_min > 0 is then required
 *     (the paper's experiments use 0.01). Gate pre-activations below about -10 give gates under
 *     the forward's gate floor (see "Gates" above); below about -88 the gate is 0.
 *   qk_l2norm != 0: q and k are divided by their L2 norms over dk, per token and head (the
 *     normalised keys of Sec. "Delta-rule models as fixed-gain Kalman filters"); an all-zero
 *     row stays zero.
 *   mu_t: per-token information scale [B,T,H] ([R,H] for decode) in the call's dtype, each
 *     value > 0 (not checked on the host), used in place of mu (eq.
 *     appendix-protection-scale-update); NULL = the scalar mu.
 *   beta_eff: float32 [B,T,H] ([R,H] for decode) output, the effective write strength
 *     k_t^T kappa_t of every token (eq. appendix-effective-write): z / (r + z) with
 *     z = sum_i p_hat_i k_i^2 for the diagonal variant, beta ||k||^2 for the isotropic one;
 *     NULL = not written. It must not overlap any other buffer of the call
 *     (KDN_ERR_INVALID_ARG). Entries of skipped decode rows are left untouched.
 * All pointers are device pointers owned by the caller; the struct itself is read on the host
 * during the call only.
 */
typedef struct {
    int32_t gates_preact;
    float r_min;
    int32_t qk_l2norm;
    const void* mu_t;
    float* beta_eff;
} kdn_layer_opts;

/*
 * The forward of either variant (variant 0 = kdn_forward_diag, 1 = kdn_forward_iso, with
 * alpha_per_channel read for variant 1 only; chunk 64) with the layer options applied in its
 * kernels: the maps act on the values as loaded, in float32, before anything else uses them.
 * Arguments, outputs, workspace (kdn_forward_workspace_bytes for the same sizes) and errors are
 * those of the plain forward, plus the option errors listed above.
 */
kdn_status_t kdn_forward_layer(int32_t variant, const void* q, const void* k, const void* v,
                               const void* alpha, const void* omega, const void* r,
                               const float* S0, const float* P0, void* o, float* S_T, float* P_T,
                               const int32_t* cu_seqlens, int32_t N, int32_t B, int32_t T,
                               int32_t H, int32_t dk, int32_t dv, kdn_dtype_t dtype,
                               int32_t alpha_per_channel, float mu, float scale,
                               const kdn_layer_opts* opts, void* workspace,
                               size_t workspace_bytes, void* stream);

/*
 * One recurrent decode step: exactly one token of the forward recurrence per row, with the
 * state resident in a slot pool and updated in place (the paper's constant-memory decoding;
 * Prop. "Diagonal Kalman Delta Network" / Prop. "Isotropic Kalman Delta Network" for T = 1).
 *   variant: 0 = diagonal, 1 = isotropic
 *   q, k: [R,H,dk]; v, o: [R,H,dv]; alpha: [R,H,dk] (diagonal, or isotropic with
 *   alpha_per_channel) or [R,H]; omega: [R,H,dk] (diagonal) or [R,H]; r: [R,H]   (dtype)
 *   S: [num_slots,H,dk,dv] float32, P: [num_slots,H,dk] (diag) / [num_slots,H] (iso) float32
 *   slot_idx: int32 [R] (device) or NULL (row i uses slot i, needs R <= num_slots). A negative
 *   slot skips the row: its o row and every state slot are left untouched. Two rows naming
 *   the same slot race (undefined result). Slots >= num_slots are skipped the same way.
 */
kdn_status_t kdn_decode_step(int32_t variant, const void* q, const void* k, const void* v,
                             const void* alpha, const void* omega, const void* r, float* S,
                             float* P, const int32_t* slot_idx, void* o, int32_t R,
                             int32_t num_slots, int32_t H, int32_t dk, int32_t dv,
                             kdn_dtype_t dtype, int32_t alpha_per_channel, float mu, float scale,
                             void* stream);

/*
 * kdn_decode_step with the layer options (per-row arrays [R,H]); everything else as
 * kdn_decode_step.
 */
kdn_status_t kdn_decode_step_layer(int32_t variant, const void* q, const void* k, const void* v,
                                   const void* alpha, const void* omega, const void* r, float* S,
                                   float* P, const int32_t* slot_idx, void* o, int32_t R,
                                   int32_t num_slots, int32_t H, int32_t dk, int32_t dv,
                                   kdn_dtype_t dtype, int32_t alpha_per_channel, float mu,
                                   float scale, const kdn_layer_opts* opts, void* stream);

/*
 * Gain scan alone (App. "Hardware-Efficient Chunkwise Algorithm", Sec. "Chunkwise Gain
 * Computation", eqs. chunk-gain-summary, chunk-gain-carry, chunk-gain-local-prefix,
 * chunk-gain-emission): the variance recurrence run as a log-depth associative scan of 2x2
 * Moebius matrices, emitting the pre-write gain of every token and the final variances.
 *   Diagonal: kappa_out [B,T,H,dk] float32 (kappa_t), phat_out [B,T,H,dk] float32 or NULL
 *   (p_hat_t), P_T [N,H,dk] float32 or NULL.
 *   Isotropic: beta_out [B,T,H] float32 (beta_t), bhat_out [B,T,H] or NULL, P_T [N,H] or NULL.
 *   Inputs as in the forward (v, q are not needed), each smaller than 2 GiB
 *   (KDN_ERR_UNSUPPORTED otherwise). workspace: kdn_gain_workspace_bytes(...).
 */
kdn_status_t kdn_gain_diag(const void* k, const void* alpha, const void* omega, const void* r,
                           const float* P0, float* kappa_out, float* phat_out, float* P_T,
                           const int32_t* cu_seqlens, int32_t N, int32_t B, int32_t T,
                           int32_t H, int32_t dk, kdn_dtype_t dtype, float mu, void* workspace,
                           size_t workspace_bytes, void* stream);

kdn_status_t kdn_gain_iso(const void* k, const void* alpha, const void* omega, const void* r,
                          const float* P0, float* beta_out, float* bhat_out, float* P_T,
                          const int32_t* cu_seqlens, int32_t N, int32_t B, int32_t T, int32_t H,
                          int32_t dk, kdn_dtype_t dtype, int32_t alpha_per_channel, float mu,
                          void* workspace, size_t workspace_bytes, void* stream);

/* Device scratch (bytes) the gain scan needs; variant 0 = diagonal, 1 = isotropic.           */
size_t kdn_gain_workspace_bytes(int32_t variant, int32_t N, int32_t B, int32_t T, int32_t H,
                                int32_t dk);

/*
 * Backward of the forward (variant 0: kdn_forward_diag, 1: kdn_forward_iso; chunk 64): the
 * gradients of a scalar loss with respect to every input, given the loss's gradients with
 * respect to the forward's outputs. The paper trains through its forward kernels (App.
 * "Detailed Experimental Setup"); this is the reverse mode of the same recurrences
 * (Prop. "Diagonal Kalman Delta Network", Prop. "Isotropic Kalman Delta Network"), taken
 * through the chunked memory scan (App. "Hardware-Efficient Chunkwise Algorithm", Sec.
 * "Chunkwise Memory Scan") with decay ratios formed from cumulative log-decays, and through the
 * variance recurrence as a reverse linear recurrence of its adjoint.
 *   Inputs: those of the forward (same layouts, dtype, packing, S0 / P0 NULL = 0 / 1, mu,
 *   scale; alpha_per_channel as in kdn_forward_iso, ignored for variant 0), and
 *   dO [B,T,H,dv] in the input dtype (NULL = 0), dS_T [N,H,dk,dv] and dP_T (shape of P_T)
 *   float32 (NULL = 0).
 *   Outputs (float32, caller-owned, each the shape of its input, fully overwritten for the
 *   tokens of the batch's sequences): dq, dk, dv, dalpha, domega, dr; dS0 [N,H,dk,dv] and dP0
 *   (shape of P0) or NULL (not written). No gradient may overlap another or any other buffer of
 *   the call (KDN_ERR_INVALID_ARG). Tokens of a packed batch outside every sequence are not
 *   written.
 *   workspace: at least kdn_backward_workspace_bytes(...) bytes (KDN_ERR_WORKSPACE), about
 *   8 KB per token and head at dk = dv = 128; no initialisation needed.
 * Seven kernels run on `stream`: the forward's chunk summaries and carry scan, then a per-chunk
 * replay of the gains and the chunk matrices, a forward walk that checkpoints the state at every
 * chunk start, a reverse walk that carries the state's adjoint, the per-chunk gradients, the
 * reverse scan of the variance adjoint and the per-token gradients of the gains. The arithmetic
 * is float32 throughout, with the cumulative log-decays in float64. Decay ratios between
 * 16-token blocks are products of factors at most one; inside a block they are referenced to
 * its token 8, exact while the product of alpha over any 8 consecutive tokens of an aligned
 * 16-token block stays above 2^-100 per channel (every alpha >= 2^-12.5 ~ 1.7e-4 suffices).
 * Below that floor those factors saturate at 2^100: the gradients stay finite and the
 * intra-block terms of the affected channels lose accuracy.
 */
kdn_status_t kdn_backward(int32_t variant, const void* q, const void* k, const void* v,
                          const void* alpha, const void* omega, const void* r, const float* S0,
                          const float* P0, const int32_t* cu_seqlens, int32_t N, int32_t B,
                          int32_t T, int32_t H, int32_t dk, int32_t dv, kdn_dtype_t dtype,
                          int32_t alpha_per_channel, float mu, float scale, const void* dO,
                          const float* dS_T, const float* dP_T, float* dq, float* dk_out,
                          float* dv_out, float* dalpha, float* domega, float* dr, float* dS0,
                          float* dP0, void* workspace, size_t workspace_bytes, void* stream);

/* Device scratch (bytes) kdn_backward needs for these sizes (packed != 0 with cu_seqlens);
 * 0 for arguments it rejects.                                                                 */
size_t kdn_backward_workspace_bytes(int32_t variant, int32_t N, int32_t B, int32_t T, int32_t H,
                                    int32_t dk, int32_t dv, int32_t packed);

/*
 * Kalman Associative Memory: the exact Kalman filter of the memory with a dense dk x dk
 * covariance per (sequence, head) (Prop. "Kalman Associative Memory", eq.
 * kalman-optimal-update-box), the model the diagonal and isotropic variants approximate, as a
 * reference for small heads (its state and work per token grow as dk^2):
 *   P_hat = diag(alpha) P diag(alpha) + diag(omega);  kappa = P_hat k / (r + k^T P_hat k)
 *   S = diag(alpha) S + kappa (v - (diag(alpha) S)^T k)^T;  P = (I - kappa k^T) P_hat
 *   o = scale * S^T q
 *   q, k, alpha, omega: [B,T,H,dk]; v, o: [B,T,H,dv]; r: [B,T,H] (dtype); packing as the
 *   forward. S0, S_T: [N,H,dk,dv]; P0, P_T: [N,H,dk,dk] float32 (P0 NULL = identity, S0 NULL =
 *   0; S_T, P_T NULL = not written; S_T / P_T may alias S0 / P0 exactly). No information scale
 *   (the exact filter has none) and no workspace. One workgroup walks each (sequence, head)
 *   token by token: intended for checking and analysis, not for long sequences at dk = 128.
 */
kdn_status_t kdn_forward_kam(const void* q, const void* k, const void* v, const void* alpha,
                             const void* omega, const void* r, const float* S0, const float* P0,
                             void* o, float* S_T, float* P_T, const int32_t* cu_seqlens,
                             int32_t N, int32_t B, int32_t T, int32_t H, int32_t dk, int32_t dv,
                             kdn_dtype_t dtype, float scale, void* stream);

/* Static text for a status code.                                                             */
const char* kdn_status_string(kdn_status_t status);

/* Detail of the calling thread's most recent non-OK status ("" if none). Valid until the next
 * library call on the same thread.                                                            */
const char* kdn_last_error(void);

/* Library version string.                                                                     */
const char* kdn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KDN_H */
