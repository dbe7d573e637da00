// Resident-family backward dispatch, fp32.  The staged and per-wave resident
// kernels are instantiated in their own translation units (gspn_staged_*,
// gspn_resbwdk_*), the persistent 128 x 128 one in gspn_widebwd_*.
#include "gspn_staged_bwd_impl.hpp"

namespace gspn {
extern template hipError_t launch_staged_bwd_size<float>(const ResBwdParams& p, int S, hipStream_t st);
extern template hipError_t launch_resident_bwd<float, 16>(const ResBwdParams& p, hipStream_t st);
extern template hipError_t launch_resident_bwd<float, 28>(const ResBwdParams& p, hipStream_t st);
extern template hipError_t launch_resident_bwd<float, 32>(const ResBwdParams& p, hipStream_t st);
extern template hipError_t launch_resident_bwd<float, 56>(const ResBwdParams& p, hipStream_t st);
extern template hipError_t launch_resident_bwd<float, 64>(const ResBwdParams& p, hipStream_t st);
hipError_t resident_bwd_f32(const ResidentBwdArgs& a) { return resident_bwd_t<float>(a); }
}  // namespace gspn
