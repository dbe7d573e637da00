// Resident-family kernels instantiated for bf16 storage (fp32 arithmetic).
#include "gspn_resident_impl.hpp"
#include "gspn_fixed_impl.hpp"
#include "gspn_wide_impl.hpp"
#include "gspn_staged_bwd_impl.hpp"

namespace gspn {
hipError_t resident_fwd_bf16(const ResidentFwdArgs& a) { return resident_fwd_t<bf16>(a); }
hipError_t resident_bwd_bf16(const ResidentBwdArgs& a) { return resident_bwd_t<bf16>(a); }
}  // namespace gspn
