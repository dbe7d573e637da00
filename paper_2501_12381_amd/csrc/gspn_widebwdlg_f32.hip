// Persistent 128 x 128 backward with Eq. 6 logits, fp32.
#include "gspn_widebwd_impl.hpp"

namespace gspn {
template hipError_t launch_wide_bwd<float, true>(const WideBwdParams& p, hipStream_t st);
}  // namespace gspn
