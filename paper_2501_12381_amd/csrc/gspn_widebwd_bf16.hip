// Persistent 128 x 128 backward, bf16 storage (fp32 arithmetic): plain weights, and the dispatch
// (the logits variant is instantiated in gspn_widebwdlg_bf16.hip).
#include "gspn_widebwd_impl.hpp"

namespace gspn {
extern template hipError_t launch_wide_bwd<bf16, true>(const WideBwdParams& p, hipStream_t st);
hipError_t wide_bwd_launch_bf16(const WideBwdParams& p, hipStream_t st) {
  return p.logits ? launch_wide_bwd<bf16, true>(p, st) : launch_wide_bwd<bf16, false>(p, st);
}
}  // namespace gspn
