// Persistent 128 x 128 backward instantiated for fp32 storage (fp32 arithmetic).
#include "gspn_widebwd_impl.hpp"

namespace gspn {
hipError_t wide_bwd_launch_f32(const WideBwdParams& p, hipStream_t st) { return launch_wide_bwd<float>(p, st); }
}  // namespace gspn
