// Size-specialised resident forward kernels (16, 28, 32, 56, 64), fp32.
#include "gspn_fixed_impl.hpp"

namespace gspn {
template hipError_t launch_fixed<float, 16>(const ResFwdParams& p, hipStream_t st);
template hipError_t launch_fixed<float, 28>(const ResFwdParams& p, hipStream_t st);
template hipError_t launch_fixed<float, 32>(const ResFwdParams& p, hipStream_t st);
template hipError_t launch_fixed<float, 56>(const ResFwdParams& p, hipStream_t st);
template hipError_t launch_fixed<float, 64>(const ResFwdParams& p, hipStream_t st);
}  // namespace gspn
