// Size-specialised resident forward kernels (16, 28, 32, 56, 64), bf16 storage (fp32 arithmetic).
#include "gspn_fixed_impl.hpp"

namespace gspn {
template hipError_t launch_fixed<bf16, 16>(const ResFwdParams& p, hipStream_t st);
template hipError_t launch_fixed<bf16, 28>(const ResFwdParams& p, hipStream_t st);
template hipError_t launch_fixed<bf16, 32>(const ResFwdParams& p, hipStream_t st);
template hipError_t launch_fixed<bf16, 56>(const ResFwdParams& p, hipStream_t st);
template hipError_t launch_fixed<bf16, 64>(const ResFwdParams& p, hipStream_t st);
}  // namespace gspn
