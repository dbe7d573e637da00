// Persistent 128 x 128 backward with Eq. 6 logits, bf16 storage (fp32 arithmetic).
#include "gspn_widebwd_impl.hpp"

namespace gspn {
template hipError_t launch_wide_bwd<bf16, true>(const WideBwdParams& p, hipStream_t st);
}  // namespace gspn
