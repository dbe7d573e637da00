// Two-pass backward kernels for large planes, fp32.
#include "gspn_large_bwd_impl.hpp"

namespace gspn {
extern template hipError_t launch_large_h<float>(const LargeHParams& p, int nw, int64_t grid, size_t lds, bool lg,
                                               hipStream_t st);
extern template hipError_t launch_large_v<float, 1>(const LargeVParams& p, bool both, hipStream_t st, bool rec, bool lg);
extern template hipError_t launch_large_v<float, 2>(const LargeVParams& p, bool both, hipStream_t st, bool rec, bool lg);
extern template hipError_t launch_large_v<float, 4>(const LargeVParams& p, bool both, hipStream_t st, bool rec, bool lg);
extern template hipError_t launch_large_hadj_nw<float, 1>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds,
                                                           bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj_nw<float, 2>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds,
                                                           bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj_nw<float, 3>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds,
                                                           bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj_nw<float, 4>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds,
                                                           bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj_nw<float, 5>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds,
                                                           bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj_nw<float, 6>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds,
                                                           bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj_nw<float, 7>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds,
                                                           bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj_nw<float, 8>(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds,
                                                           bool lg, hipStream_t st);
extern template hipError_t launch_large_vadj_mode<float, 1, true>(const LargeVAdjParams& p, bool lg, hipStream_t st);
extern template hipError_t launch_large_vadj_mode<float, 1, false>(const LargeVAdjParams& p, bool lg, hipStream_t st);
extern template hipError_t launch_large_vadj_mode<float, 2, true>(const LargeVAdjParams& p, bool lg, hipStream_t st);
extern template hipError_t launch_large_vadj_mode<float, 2, false>(const LargeVAdjParams& p, bool lg, hipStream_t st);
extern template hipError_t launch_large_vadj_mode<float, 4, true>(const LargeVAdjParams& p, bool lg, hipStream_t st);
extern template hipError_t launch_large_vadj_mode<float, 4, false>(const LargeVAdjParams& p, bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj2_nw<float, 1>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                            int64_t grid, size_t lds, bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj2_nw<float, 2>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                            int64_t grid, size_t lds, bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj2_nw<float, 3>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                            int64_t grid, size_t lds, bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj2_nw<float, 4>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                            int64_t grid, size_t lds, bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj2_nw<float, 5>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                            int64_t grid, size_t lds, bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj2_nw<float, 6>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                            int64_t grid, size_t lds, bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj2_nw<float, 7>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                            int64_t grid, size_t lds, bool lg, hipStream_t st);
extern template hipError_t launch_large_hadj2_nw<float, 8>(const LargeHAdjParams& p0, const LargeHAdjParams& p1,
                                                            int64_t grid, size_t lds, bool lg, hipStream_t st);
hipError_t large_bwd_h_f32(const LargeBwdHArgs& a) { return large_bwd_h_t<float>(a); }
hipError_t large_bwd_h_pair_f32(const LargeBwdHArgs& l2r, const LargeBwdHArgs& r2l) {
  return large_bwd_h_pair_t<float>(l2r, r2l);
}
hipError_t large_bwd_v_rec_f32(const LargeBwdVArgs& a) { return large_bwd_v_rec_t<float>(a); }
hipError_t large_bwd_v_adj_f32(const LargeBwdVAdjArgs& a) { return large_bwd_v_adj_t<float>(a); }
}  // namespace gspn
