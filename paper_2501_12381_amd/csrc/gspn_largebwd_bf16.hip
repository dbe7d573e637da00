// Two-pass backward kernels for large planes, bf16 storage with fp32 arithmetic.
#include "gspn_large_bwd_impl.hpp"

namespace gspn {
hipError_t large_bwd_h_bf16(const LargeBwdHArgs& a) { return large_bwd_h_t<bf16>(a); }
hipError_t large_bwd_v_rec_bf16(const LargeBwdVArgs& a) { return large_bwd_v_rec_t<bf16>(a); }
hipError_t large_bwd_v_adj_bf16(const LargeBwdVAdjArgs& a) { return large_bwd_v_adj_t<bf16>(a); }
}  // namespace gspn
