// Two-pass backward: horizontal adjoint kernels (5 6 7 waves), bf16 storage (fp32 arithmetic).
#include "gspn_large_bwd_impl.hpp"

namespace gspn {
template hipError_t launch_large_hadj_nw<bf16, 5>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds, bool lg,
                                                  hipStream_t st);
template hipError_t launch_large_hadj_nw<bf16, 6>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds, bool lg,
                                                  hipStream_t st);
template hipError_t launch_large_hadj_nw<bf16, 7>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds, bool lg,
                                                  hipStream_t st);
template hipError_t launch_large_hadj2_nw<bf16, 5>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                   int64_t grid, size_t lds, bool lg, hipStream_t st);
template hipError_t launch_large_hadj2_nw<bf16, 6>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                   int64_t grid, size_t lds, bool lg, hipStream_t st);
template hipError_t launch_large_hadj2_nw<bf16, 7>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                   int64_t grid, size_t lds, bool lg, hipStream_t st);
}  // namespace gspn
