// Resident-family backward dispatch, bf16 storage (fp32 arithmetic).  The staged and per-wave resident
// kernels are instantiated in their own translation units (gspn_staged_*,
// gspn_resbwdk_*), the persistent 128 x 128 one in gspn_widebwd_*.
#include "gspn_staged_bwd_impl.hpp"

namespace gspn {
extern template hipError_t launch_staged_bwd_size<bf16>(const ResBwdParams& p, int S, hipStream_t st);
extern template hipError_t launch_resident_bwd<bf16, 16>(const ResBwdParams& p, hipStream_t st);
extern template hipError_t launch_resident_bwd<bf16, 28>(const ResBwdParams& p, hipStream_t st);
extern template hipError_t launch_resident_bwd<bf16, 32>(const ResBwdParams& p, hipStream_t st);
extern template hipError_t launch_resident_bwd<bf16, 56>(const ResBwdParams& p, hipStream_t st);
extern template hipError_t launch_resident_bwd<bf16, 64>(const ResBwdParams& p, hipStream_t st);
hipError_t resident_bwd_bf16(const ResidentBwdArgs& a) { return resident_bwd_t<bf16>(a); }
}  // namespace gspn
