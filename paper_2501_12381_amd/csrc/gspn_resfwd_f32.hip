// Resident-family forward dispatch and the generic resident kernels, fp32.
// The size-specialised and persistent 128 x 128 kernels are instantiated in
// their own translation units (gspn_fixed_*, gspn_widefwd_*).
#include "gspn_resident_impl.hpp"

namespace gspn {
hipError_t resident_fwd_f32(const ResidentFwdArgs& a) { return resident_fwd_t<float>(a); }
}  // namespace gspn

#include "gspn_resident_bwd_impl.hpp"

namespace gspn {
bool resident_fits(int H, int W, int dtype, bool backward, int narr) {
  return backward ? resident_bwd_size_supported(H, W) : resident_fwd_fits(H, W, dtype, narr);
}
}  // namespace gspn
