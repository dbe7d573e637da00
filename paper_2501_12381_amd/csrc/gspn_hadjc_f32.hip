// Two-pass backward: horizontal adjoint kernels (8 waves), fp32.
#include "gspn_large_bwd_impl.hpp"

namespace gspn {
template hipError_t launch_large_hadj_nw<float, 8>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds, bool lg,
                                                  hipStream_t st);
template hipError_t launch_large_hadj2_nw<float, 8>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                   int64_t grid, size_t lds, bool lg, hipStream_t st);
}  // namespace gspn
