// Persistent 128 x 128 backward, fp32: plain weights, and the dispatch
// (the logits variant is instantiated in gspn_widebwdlg_f32.hip).
#include "gspn_widebwd_impl.hpp"

namespace gspn {
extern template hipError_t launch_wide_bwd<float, true>(const WideBwdParams& p, hipStream_t st);
hipError_t wide_bwd_launch_f32(const WideBwdParams& p, hipStream_t st) {
  return p.logits ? launch_wide_bwd<float, true>(p, st) : launch_wide_bwd<float, false>(p, st);
}
}  // namespace gspn
