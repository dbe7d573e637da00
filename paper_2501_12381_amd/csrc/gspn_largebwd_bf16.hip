// Backward of the horizontal directions for large planes, bf16 storage.
#include "gspn_large_bwd_impl.hpp"

namespace gspn {
hipError_t large_bwd_h_bf16(const LargeBwdHArgs& a) { return large_bwd_h_t<bf16>(a); }
hipError_t large_bwd_v_rec_bf16(const LargeBwdVArgs& a) { return large_bwd_v_rec_t<bf16>(a); }
}  // namespace gspn
