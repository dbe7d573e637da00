// Two-pass backward kernels for large planes, fp32.
#include "gspn_large_bwd_impl.hpp"

namespace gspn {
hipError_t large_bwd_h_f32(const LargeBwdHArgs& a) { return large_bwd_h_t<float>(a); }
hipError_t large_bwd_v_rec_f32(const LargeBwdVArgs& a) { return large_bwd_v_rec_t<float>(a); }
hipError_t large_bwd_v_adj_f32(const LargeBwdVAdjArgs& a) { return large_bwd_v_adj_t<float>(a); }
}  // namespace gspn
