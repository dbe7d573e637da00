// Two-pass forward kernels, bf16 storage with fp32 arithmetic.
#include "gspn_large_impl.hpp"

namespace gspn {
hipError_t large_fwd_bf16(const LargeFwdArgs& a) { return large_fwd_t<bf16>(a); }
}  // namespace gspn
