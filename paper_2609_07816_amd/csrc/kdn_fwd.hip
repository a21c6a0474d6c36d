// Host entry of the chunked forward: chunk support, workspace size and the dispatch to the
// instantiations per dtype and mode in kdn_fwd_{bf16,f32}.hip and kdn_fwd_layer_{bf16,f32}.hip
// (kernels in kdn_fwd.h).
#include "kdn_fwd.h"

namespace kdn {
namespace fwd {

size_t rec_bytes(kdn_dtype_t dtype, int dk)
{
    if (dtype == KDN_F32) {
        switch (dk) {
        case 16: return OpRec<float, 16>::BYTES;
        case 32: return OpRec<float, 32>::BYTES;
        case 64: return OpRec<float, 64>::BYTES;
        default: return OpRec<float, 128>::BYTES;
        }
    }
    switch (dk) {
    case 16: return OpRec<bf16, 16>::BYTES;
    case 32: return OpRec<bf16, 32>::BYTES;
    case 64: return OpRec<bf16, 64>::BYTES;
    default: return OpRec<bf16, 128>::BYTES;
    }
}

}  // namespace fwd

bool chunked_supported(int chunk) { return chunk == 0 || chunk == fwd::C; }

size_t chunked_workspace_bytes(int variant, bool packed, int N, int B, int T, int H, int dk,
                               kdn_dtype_t dtype)
{
    return fwd::ws_map(variant, packed, N, B, T, H, dk, fwd::rec_bytes(dtype, dk)).total;
}

hipError_t launch_chunked(const FwdCall& fc, hipStream_t stream)
{
    if (fc.ly.on) {
        if (fc.dtype == KDN_F32) return fwd::run_forward<float, true>(fc, stream);
        return fwd::run_forward<bf16, true>(fc, stream);
    }
    if (fc.dtype == KDN_F32) return fwd::run_forward<float, false>(fc, stream);
    return fwd::run_forward<bf16, false>(fc, stream);
}

}  // namespace kdn
