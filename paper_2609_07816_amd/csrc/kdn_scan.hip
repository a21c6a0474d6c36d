// Chunk bookkeeping and the log-depth carry of the variance chain (arXiv 2609.07816, App.
// "Hardware-Efficient Chunkwise Algorithm", Sec. "Chunkwise Gain Computation", eq.
// chunk-gain-carry), shared by the forward and the gain scan.
//
// The variance recurrence of every (sequence, head, channel) is a product of 2x2 Moebius
// matrices acting on z = [n; d] (p = n / d). Given each chunk's summary M_bar_m (the product of
// its token matrices, later on the left), the state entering chunk m is
//   z_in_m = M_bar_{m-1} ... M_bar_0 z_0,   z_0 = [p_0; 1],
// an exclusive scan with an associative operator, run here as a Kogge-Stone scan inside one
// wavefront (64 chunks per step, log2(64) = 6 rounds; longer sequences carry block to block).
#include "kdn_device.h"

namespace kdn {
namespace {

__global__ void chunk_table_kernel(const int32_t* __restrict__ cu, int N, int ntok, int ch,
                                   int maxch, int32_t* __restrict__ choff)
{
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    int acc = 0;
    for (int n = 0; n < N; ++n) {
        choff[n] = acc;
        const int t0 = min(max(cu[n], 0), ntok), t1 = min(max(cu[n + 1], t0), ntok);
        acc = min(acc + (t1 - t0 + ch - 1) / ch, maxch);
    }
    choff[N] = acc;
}

__device__ __forceinline__ float4 shfl_up4(float4 x, int off)
{
    return make_float4(__shfl_up(x.x, off, 64), __shfl_up(x.y, off, 64),
                       __shfl_up(x.z, off, 64), __shfl_up(x.w, off, 64));
}

// Grid (N * H, ceil(nchan / 4)), 256 threads: one wavefront per (sequence, head, channel), its
// lanes are chunks.
__global__ __launch_bounds__(256) void carry_scan_kernel(const float4* __restrict__ summ,
                                                         const float* __restrict__ P0,
                                                         ChunkMap cm, int ch, int H, int nchan,
                                                         float2* __restrict__ carry,
                                                         float* __restrict__ P_T)
{
    const int n = blockIdx.x / H, h = blockIdx.x % H;
    if (n >= cm.N) return;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int c = 4 * blockIdx.y + w;  // one channel per wavefront
    if (c >= nchan) return;
    int t0, t1;
    seq_span(cm, n, t0, t1);
    const int nchs = (t1 - t0 + ch - 1) / ch;
    const int g0 = cm.cu ? cm.choff[n] : n * ((cm.T + ch - 1) / ch);
    const int nch = max(0, min(nchs, cm.maxch - g0));
    const size_t pidx = ((size_t)n * H + h) * nchan + c;
    if (nch == 0) {  // an empty sequence keeps its initial variances
        if (P_T && lane == 0) P_T[pidx] = P0 ? P0[pidx] : 1.f;
        return;
    }
    float cn = P0 ? P0[pidx] : 1.f, cd = 1.f;  // z_0 = [p_0; 1]
    for (int b0 = 0; b0 < nch; b0 += 64) {
        const int m = b0 + lane;
        float4 x = make_float4(1.f, 0.f, 0.f, 1.f);
        if (m < nch) x = summ[((size_t)(g0 + m) * H + h) * nchan + c];
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {  // inclusive prefix, later chunks on the left
            const float4 y = shfl_up4(x, off);
            if (lane >= off) x = mat_mul(x, y);
        }
        float zn = fmaf(x.x, cn, x.y * cd), zd = fmaf(x.z, cn, x.w * cd);  // after chunk m
        rescale2(zn, zd);
        float en = __shfl_up(zn, 1, 64), ed = __shfl_up(zd, 1, 64);       // before chunk m
        if (lane == 0) {
            en = cn;
            ed = cd;
        }
        if (m < nch) carry[((size_t)(g0 + m) * H + h) * nchan + c] = make_float2(en, ed);
        const int lastl = min(63, nch - 1 - b0);
        cn = __shfl(zn, lastl, 64);
        cd = __shfl(zd, lastl, 64);
    }
}

__global__ __launch_bounds__(1024) void order_kernel(const int32_t* __restrict__ cu, int N,
                                                     int ntok, int32_t* __restrict__ order)
{
    __shared__ int32_t len[ORDER_MAX];
    for (int i = threadIdx.x; i < N; i += blockDim.x) {
        const int t0 = min(max(cu[i], 0), ntok), t1 = min(max(cu[i + 1], t0), ntok);
        len[i] = t1 - t0;
    }
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

}  // namespace

hipError_t launch_chunk_table(const int32_t* cu, int N, int ntok, int ch, int maxch,
                              int32_t* choff, hipStream_t st)
{
    hipLaunchKernelGGL(chunk_table_kernel, dim3(1), dim3(1), 0, st, cu, N, ntok, ch, maxch,
                       choff);
    return hipGetLastError();
}

hipError_t launch_carry_scan(const float4* summ, const float* P0, const ChunkMap& cm, int ch,
                             int H, int nchan, float2* carry, float* P_T, hipStream_t st)
{
    const dim3 grid((unsigned)(cm.N * H), (unsigned)((nchan + 3) / 4));
    hipLaunchKernelGGL(carry_scan_kernel, grid, dim3(256), 0, st, summ, P0, cm, ch, H, nchan,
                       carry, P_T);
    return hipGetLastError();
}

hipError_t launch_order(const int32_t* cu, int N, int ntok, int32_t* order, hipStream_t st)
{
    if (N > ORDER_MAX) return hipErrorInvalidValue;
    hipLaunchKernelGGL(order_kernel, dim3(1), dim3(1024), 0, st, cu, N, ntok, order);
    return hipGetLastError();
}

}  // namespace kdn
