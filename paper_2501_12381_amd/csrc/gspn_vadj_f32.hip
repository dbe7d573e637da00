// Two-pass backward: vertical adjoint kernels, fp32.
#include "gspn_large_bwd_impl.hpp"

namespace gspn {
template hipError_t launch_large_vadj_mode<float, 1, true>(const LargeVAdjParams& p, bool lg, hipStream_t st);
template hipError_t launch_large_vadj_mode<float, 1, false>(const LargeVAdjParams& p, bool lg, hipStream_t st);
template hipError_t launch_large_vadj_mode<float, 2, true>(const LargeVAdjParams& p, bool lg, hipStream_t st);
template hipError_t launch_large_vadj_mode<float, 2, false>(const LargeVAdjParams& p, bool lg, hipStream_t st);
template hipError_t launch_large_vadj_mode<float, 4, true>(const LargeVAdjParams& p, bool lg, hipStream_t st);
template hipError_t launch_large_vadj_mode<float, 4, false>(const LargeVAdjParams& p, bool lg, hipStream_t st);
}  // namespace gspn
