// Two-pass backward: horizontal adjoint kernels (5 6 7 waves), fp32.
#include "gspn_large_bwd_impl.hpp"

namespace gspn {
template hipError_t launch_large_hadj_nw<float, 5>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds, bool lg,
                                                  hipStream_t st);
template hipError_t launch_large_hadj_nw<float, 6>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds, bool lg,
                                                  hipStream_t st);
template hipError_t launch_large_hadj_nw<float, 7>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds, bool lg,
                                                  hipStream_t st);
template hipError_t launch_large_hadj2_nw<float, 5>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                   int64_t grid, size_t lds, bool lg, hipStream_t st);
template hipError_t launch_large_hadj2_nw<float, 6>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                   int64_t grid, size_t lds, bool lg, hipStream_t st);
template hipError_t launch_large_hadj2_nw<float, 7>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                   int64_t grid, size_t lds, bool lg, hipStream_t st);
}  // namespace gspn
