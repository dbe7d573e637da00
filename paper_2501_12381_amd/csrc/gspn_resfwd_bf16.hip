// Resident-family forward dispatch and the generic resident kernels, bf16 storage (fp32 arithmetic).
// The size-specialised and persistent 128 x 128 kernels are instantiated in
// their own translation units (gspn_fixed_*, gspn_widefwd_*).
#include "gspn_resident_impl.hpp"

namespace gspn {
hipError_t resident_fwd_bf16(const ResidentFwdArgs& a) { return resident_fwd_t<bf16>(a); }
}  // namespace gspn
