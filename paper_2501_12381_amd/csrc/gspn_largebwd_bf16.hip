// Two-pass backward kernels for large planes, bf16 storage with fp32 arithmetic.
#include "gspn_large_bwd_impl.hpp"

namespace gspn {
extern template hipError_t launch_large_h<bf16>(const LargeHParams& p, int nw, int64_t grid, size_t lds, bool lg,
                                               hipStream_t st);
extern template hipError_t launch_large_v<bf16, 1>(const LargeVParams& p, bool both, hipStream_t st, bool rec, bool lg);
extern template hipError_t launch_large_v<bf16, 2>(const LargeVParams& p, bool both, hipStream_t st, bool rec, bool lg);
extern template hipError_t launch_large_v<bf16, 4>(const LargeVParams& p, bool both, hipStream_t st, bool rec, bool lg);
extern template hipError_t launch_large_hadj_nw<bf16, 1>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds,
                                                           bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj_nw<bf16, 2>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds,
                                                           bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj_nw<bf16, 3>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds,
                                                           bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj_nw<bf16, 4>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds,
                                                           bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj_nw<bf16, 5>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds,
                                                           bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj_nw<bf16, 6>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds,
                                                           bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj_nw<bf16, 7>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds,
                                                           bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj_nw<bf16, 8>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds,
                                                           bool lg, hipStream_t st);
extern template hipError_t launch_large_vadj_mode<bf16, 1, true>(const LargeVAdjParams& p, bool lg, hipStream_t st);
extern template hipError_t launch_large_vadj_mode<bf16, 1, false>(const LargeVAdjParams& p, bool lg, hipStream_t st);
extern template hipError_t launch_large_vadj_mode<bf16, 2, true>(const LargeVAdjParams& p, bool lg, hipStream_t st);
extern template hipError_t launch_large_vadj_mode<bf16, 2, false>(const LargeVAdjParams& p, bool lg, hipStream_t st);
extern template hipError_t launch_large_vadj_mode<bf16, 4, true>(const LargeVAdjParams& p, bool lg, hipStream_t st);
extern template hipError_t launch_large_vadj_mode<bf16, 4, false>(const LargeVAdjParams& p, bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj2_nw<bf16, 1>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                            int64_t grid, size_t lds, bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj2_nw<bf16, 2>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                            int64_t grid, size_t lds, bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj2_nw<bf16, 3>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                            int64_t grid, size_t lds, bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj2_nw<bf16, 4>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                            int64_t grid, size_t lds, bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj2_nw<bf16, 5>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                            int64_t grid, size_t lds, bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj2_nw<bf16, 6>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                            int64_t grid, size_t lds, bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj2_nw<bf16, 7>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                            int64_t grid, size_t lds, bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj2_nw<bf16, 8>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                            int64_t grid, size_t lds, bool lg, hipStream_t st);
hipError_t large_bwd_h_bf16(const LargeBwdHArgs& a) { return large_bwd_h_t<bf16>(a); }
hipError_t large_bwd_h_pair_bf16(const LargeBwdHArgs& l2r, const LargeBwdHArgs& r2l) {
  return large_bwd_h_pair_t<bf16>(l2r, r2l);
}
hipError_t large_bwd_v_rec_bf16(const LargeBwdVArgs& a) { return large_bwd_v_rec_t<bf16>(a); }
hipError_t large_bwd_v_adj_bf16(const LargeBwdVAdjArgs& a) { return large_bwd_v_adj_t<bf16>(a); }
}  // namespace gspn
