// Persistent 128 x 128 forward, bf16 storage (fp32 arithmetic).
#include "gspn_wide_impl.hpp"

namespace gspn {
template hipError_t launch_wide<bf16>(const ResFwdParams& p, hipStream_t st);
}  // namespace gspn
