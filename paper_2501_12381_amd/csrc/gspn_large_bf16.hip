// Two-pass forward kernels, bf16 storage with fp32 arithmetic.
#include "gspn_large_impl.hpp"

namespace gspn {
hipError_t large_fwd_bf16(const LargeFwdArgs& a) { return large_fwd_t<bf16>(a); }
// the pass kernels are also the backward's recompute: instantiated here once
template hipError_t launch_large_h<bf16>(const LargeHParams& p, int nw, int64_t grid, size_t lds, bool lg,
                                        hipStream_t st);
template hipError_t launch_large_v<bf16, 1>(const LargeVParams& p, bool both, hipStream_t st, bool rec, bool lg);
template hipError_t launch_large_v<bf16, 2>(const LargeVParams& p, bool both, hipStream_t st, bool rec, bool lg);
template hipError_t launch_large_v<bf16, 4>(const LargeVParams& p, bool both, hipStream_t st, bool rec, bool lg);
}  // namespace gspn
