// Streaming-family kernels instantiated for fp32 storage.
#include "gspn_stream_impl.hpp"

namespace gspn {
hipError_t stream_fwd_pass_f32(const StreamFwdArgs& a) { return stream_fwd_pass_t<float>(a); }
hipError_t stream_adj_pass_f32(const StreamAdjArgs& a) { return stream_adj_pass_t<float>(a); }
hipError_t grad_finish_f32(const GradFinishArgs& a) { return grad_finish_t<float>(a); }
}  // namespace gspn
