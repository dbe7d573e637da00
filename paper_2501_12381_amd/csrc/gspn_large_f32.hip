// Two-pass forward kernels, fp32.
#include "gspn_large_impl.hpp"

namespace gspn {
hipError_t large_fwd_f32(const LargeFwdArgs& a) { return large_fwd_t<float>(a); }
bool large_fwd_fits(int H, int W, int dtype) {
  return dtype == 0 ? large_fwd_supported<float>(H, W) : large_fwd_supported<bf16>(H, W);
}
// the pass kernels are also the backward's recompute: instantiated here once
template hipError_t launch_large_h<float>(const LargeHParams& p, int nw, int64_t grid, size_t lds, bool lg,
                                        hipStream_t st);
template hipError_t launch_large_v<float, 1>(const LargeVParams& p, bool both, hipStream_t st, bool rec, bool lg);
template hipError_t launch_large_v<float, 2>(const LargeVParams& p, bool both, hipStream_t st, bool rec, bool lg);
template hipError_t launch_large_v<float, 4>(const LargeVParams& p, bool both, hipStream_t st, bool rec, bool lg);
}  // namespace gspn
