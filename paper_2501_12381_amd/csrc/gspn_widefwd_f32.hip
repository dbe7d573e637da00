// Persistent 128 x 128 forward, fp32.
#include "gspn_wide_impl.hpp"

namespace gspn {
template hipError_t launch_wide<float>(const ResFwdParams& p, hipStream_t st);
}  // namespace gspn
