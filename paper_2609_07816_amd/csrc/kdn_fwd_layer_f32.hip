// f32 instantiation of the layer forward: the chunked forward with the layer's input maps,
// per-token information scale and effective-write output (kernels in kdn_fwd.h).
#include "kdn_fwd.h"

namespace kdn {
namespace fwd {
template hipError_t run_forward<float, true>(const FwdCall& fc, hipStream_t st);
}  // namespace fwd
}  // namespace kdn
