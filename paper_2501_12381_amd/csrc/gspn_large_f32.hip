// Two-pass forward kernels, fp32.
#include "gspn_large_impl.hpp"

namespace gspn {
hipError_t large_fwd_f32(const LargeFwdArgs& a) { return large_fwd_t<float>(a); }
bool large_fwd_fits(int H, int W, int dtype) {
  return dtype == 0 ? large_fwd_supported<float>(H, W) : large_fwd_supported<bf16>(H, W);
}
}  // namespace gspn
