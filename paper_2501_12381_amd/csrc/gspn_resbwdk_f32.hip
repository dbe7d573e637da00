// Per-wave resident backward kernels (16, 28, 32, 56, 64), fp32.
#include "gspn_resident_bwd_impl.hpp"

namespace gspn {
template hipError_t launch_resident_bwd<float, 16>(const ResBwdParams& p, hipStream_t st);
template hipError_t launch_resident_bwd<float, 28>(const ResBwdParams& p, hipStream_t st);
template hipError_t launch_resident_bwd<float, 32>(const ResBwdParams& p, hipStream_t st);
template hipError_t launch_resident_bwd<float, 56>(const ResBwdParams& p, hipStream_t st);
template hipError_t launch_resident_bwd<float, 64>(const ResBwdParams& p, hipStream_t st);
}  // namespace gspn
