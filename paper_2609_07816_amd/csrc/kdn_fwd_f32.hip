// f32 instantiation of the chunked forward (kernels in kdn_fwd.h).
#include "kdn_fwd.h"

namespace kdn {
namespace fwd {
template hipError_t run_forward<float, false>(const FwdCall& fc, hipStream_t st);
}  // namespace fwd
}  // namespace kdn
