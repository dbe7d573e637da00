// LDS-staged backward kernels (16, 28, 32), fp32.
#include "gspn_staged_bwd_impl.hpp"

namespace gspn {
template hipError_t launch_staged_bwd_size<float>(const ResBwdParams& p, int S, hipStream_t st);
}  // namespace gspn
