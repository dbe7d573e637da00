// Per-wave resident backward kernels (16, 28, 32, 56, 64), bf16 storage (fp32 arithmetic).
#include "gspn_resident_bwd_impl.hpp"

namespace gspn {
template hipError_t launch_resident_bwd<bf16, 16>(const ResBwdParams& p, hipStream_t st);
template hipError_t launch_resident_bwd<bf16, 28>(const ResBwdParams& p, hipStream_t st);
template hipError_t launch_resident_bwd<bf16, 32>(const ResBwdParams& p, hipStream_t st);
template hipError_t launch_resident_bwd<bf16, 56>(const ResBwdParams& p, hipStream_t st);
template hipError_t launch_resident_bwd<bf16, 64>(const ResBwdParams& p, hipStream_t st);
}  // namespace gspn
