// Two-pass backward: vertical adjoint kernels, bf16 storage (fp32 arithmetic).
#include "gspn_large_bwd_impl.hpp"

namespace gspn {
template hipError_t launch_large_vadj_mode<bf16, 1, true>(const LargeVAdjParams& p, bool lg, hipStream_t st);
template hipError_t launch_large_vadj_mode<bf16, 1, false>(const LargeVAdjParams& p, bool lg, hipStream_t st);
template hipError_t launch_large_vadj_mode<bf16, 2, true>(const LargeVAdjParams& p, bool lg, hipStream_t st);
template hipError_t launch_large_vadj_mode<bf16, 2, false>(const LargeVAdjParams& p, bool lg, hipStream_t st);
template hipError_t launch_large_vadj_mode<bf16, 4, true>(const LargeVAdjParams& p, bool lg, hipStream_t st);
template hipError_t launch_large_vadj_mode<bf16, 4, false>(const LargeVAdjParams& p, bool lg, hipStream_t st);
}  // namespace gspn
