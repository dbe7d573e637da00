// Streaming-family kernels instantiated for bf16 storage (fp32 arithmetic).
#include "gspn_stream_impl.hpp"

namespace gspn {
hipError_t stream_fwd_pass_bf16(const StreamFwdArgs& a) { return stream_fwd_pass_t<bf16>(a); }
hipError_t stream_adj_pass_bf16(const StreamAdjArgs& a) { return stream_adj_pass_t<bf16>(a); }
hipError_t grad_finish_bf16(const GradFinishArgs& a) { return grad_finish_t<bf16>(a); }
}  // namespace gspn
