// LDS-staged backward kernels (16, 28, 32), bf16 storage (fp32 arithmetic).
#include "gspn_staged_bwd_impl.hpp"

namespace gspn {
template hipError_t launch_staged_bwd_size<bf16>(const ResBwdParams& p, int S, hipStream_t st);
}  // namespace gspn
