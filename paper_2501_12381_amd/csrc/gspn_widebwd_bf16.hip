// Persistent 128 x 128 backward instantiated for bf16 storage (fp32 arithmetic).
#include "gspn_widebwd_impl.hpp"

namespace gspn {
hipError_t wide_bwd_launch_bf16(const WideBwdParams& p, hipStream_t st) { return launch_wide_bwd<bf16>(p, st); }
}  // namespace gspn
