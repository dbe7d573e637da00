// Resident-family kernels instantiated for fp32 storage.
#include "gspn_resident_impl.hpp"
#include "gspn_fixed_impl.hpp"
#include "gspn_wide_impl.hpp"
#include "gspn_staged_bwd_impl.hpp"

namespace gspn {
hipError_t resident_fwd_f32(const ResidentFwdArgs& a) { return resident_fwd_t<float>(a); }
hipError_t resident_bwd_f32(const ResidentBwdArgs& a) { return resident_bwd_t<float>(a); }
}  // namespace gspn

namespace gspn {
bool resident_fits(int H, int W, int dtype, bool backward) {
  return backward ? resident_bwd_size_supported(H, W) : resident_fwd_fits(H, W, dtype);
}
}  // namespace gspn
