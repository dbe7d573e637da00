// Internal launch interface between the C ABI (gspn_api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace gspn {

enum { DIR_T2B = 1, DIR_B2T = 2, DIR_L2R = 4, DIR_R2L = 8 };
enum { MODE_STORE = 0, MODE_ADD = 1, MODE_FINAL = 2, MODE_REC = 3 };
constexpr int kMaxWaves = 16;

// ---- streaming family: one pass per direction --------------------------------
struct StreamFwdArgs {
  const void* x;
  const void* lam;
  const void* w;      // this direction's w0 (w1, w2 follow at +wstride, +2*wstride)
  int64_t wstride;    // elements between the three weight maps (B*C*H*W)
  const void* u;      // MODE_FINAL, or every mode with ugate
  float* acc;         // fp32 accumulator (MODE_REC: running sum of h)
  void* y;            // MODE_FINAL only
  float* hprev_out;   // MODE_REC only: h of the previous line, per line
  const void* dy;     // MODE_REC with per-direction gradients: this direction's dy
  void* du;           // MODE_REC: du = dy * h written here (per-direction u), or null
  int first;          // MODE_REC: first direction (store instead of add)
  int mode;
  int64_t planes;
  int H, W, dir, dtype;
  int group;          // lines per local-GSPN group along the scan axis (0: global)
  int logits, renorm; // w holds logits normalised by Eq. 6 (renorm: on-line neighbours only)
  int ugate;          // per-direction u: merge u * h instead of h
  int hdy;            // MODE_REC: hsum accumulates dy * h
  void* stream;
};
hipError_t stream_fwd_pass_f32(const StreamFwdArgs& a);
hipError_t stream_fwd_pass_bf16(const StreamFwdArgs& a);
inline hipError_t stream_fwd_pass(const StreamFwdArgs& a) {
  return a.dtype == 0 ? stream_fwd_pass_f32(a) : stream_fwd_pass_bf16(a);
}

struct StreamAdjArgs {
  const void* dy;     // this direction's dy
  const void* u;      // this direction's u
  const void* w;
  int64_t wstride;
  const float* hprev;
  void* dw;           // this direction's dw0 (dw1, dw2 at +wstride, +2*wstride)
  float* gsum;
  const void* lam;    // lamw: this direction's lam
  const void* x;      // lamw
  void* dlam;         // lamw: this direction's dlam = x * g
  int first;
  int64_t planes;
  int H, W, dir, dtype;
  int group;
  int logits, renorm;
  int lamw;           // per-direction lam: gsum accumulates lam * g, dlam written here
  void* stream;
};
hipError_t stream_adj_pass_f32(const StreamAdjArgs& a);
hipError_t stream_adj_pass_bf16(const StreamAdjArgs& a);
inline hipError_t stream_adj_pass(const StreamAdjArgs& a) {
  return a.dtype == 0 ? stream_adj_pass_f32(a) : stream_adj_pass_bf16(a);
}

struct GradFinishArgs {
  const void* x;
  const void* lam;
  const void* dy;
  const float* gsum;
  const float* hsum;
  const float* hsum2;  // further parts of sum_d h_d (null when absent)
  const float* hsum3;
  const void* dy2;     // du_mode 3: du = hsum + dy2 * hsum2 + dy3 * hsum3 (unmerged outputs)
  const void* dy3;
  void* dx;
  void* dlam;         // null when dlam was written per direction
  void* du;
  int64_t n;
  int dx_mode;        // 0: dx = lam * gsum; 1: dx = gsum
  int du_mode;        // 0: du = dy * hsum; 1: du = hsum; 2: du written per direction;
                      // 3: du = hsum + dy2 * hsum2 + dy3 * hsum3
  int dtype;
  void* stream;
};
hipError_t grad_finish_f32(const GradFinishArgs& a);
hipError_t grad_finish_bf16(const GradFinishArgs& a);
inline hipError_t grad_finish(const GradFinishArgs& a) {
  return a.dtype == 0 ? grad_finish_f32(a) : grad_finish_bf16(a);
}

// ---- resident family: whole planes on chip, all directions in one launch ----
struct ResidentFwdArgs {
  const void* x;
  const void* lam;
  const void* w;   // all n directions, packed [n][3][B][C][H][W]
  const void* u;
  void* y;
  uint32_t mask;
  int64_t planes;
  int H, W, dtype;
  int group_h, group_w;  // local-GSPN group lengths (0: global)
  int logits, renorm;    // w holds Eq. 6 logits (renorm: over on-line neighbours only)
  int lam_pd, u_pd, y_pd;  // per-direction maps (generic kernels; u_pd needs y_pd)
  int use_fixed;   // allow the size-specialised kernel when one exists for H x W
  void* stream;
};
hipError_t resident_fwd_f32(const ResidentFwdArgs& a);
hipError_t resident_fwd_bf16(const ResidentFwdArgs& a);
inline hipError_t resident_fwd(const ResidentFwdArgs& a) {
  return a.dtype == 0 ? resident_fwd_f32(a) : resident_fwd_bf16(a);
}
struct ResidentBwdArgs {
  const void* dy;
  const void* x;
  const void* lam;
  const void* w;
  const void* u;
  void* dx;
  void* dw;
  void* dlam;
  void* du;
  uint32_t mask;
  int64_t planes;
  int H, W, dtype;
  int group_h, group_w;  // local-GSPN group lengths (0: global)
  int logits, renorm;    // w holds Eq. 6 logits; dw is the gradient for the logits
  int lam_pd, u_pd, y_pd;  // per-direction maps (per-wave resident kernel only)
  int use_staged;  // allow the LDS-staged kernel for small planes
  void* stream;
};
hipError_t resident_bwd_f32(const ResidentBwdArgs& a);
hipError_t resident_bwd_bf16(const ResidentBwdArgs& a);
inline hipError_t resident_bwd(const ResidentBwdArgs& a) {
  return a.dtype == 0 ? resident_bwd_f32(a) : resident_bwd_bf16(a);
}
// narr: accumulator arrays per plane of the forward (the directions present
// for unmerged outputs, else 1)
bool resident_fits(int H, int W, int dtype, bool backward, int narr);

// ---- two-pass family: planes too large for LDS -------------------------------
struct LargeFwdArgs {
  const void* x;
  const void* lam;
  const void* w;   // all n directions, packed [n][3][B][C][H][W]
  const void* u;
  void* y;
  float* acc;      // fp32 partial sums, B*C*H*W (needed when n > 1)
  float* acc_b;    // second partial-sum array: bottom-to-top's h when both vertical
                   // directions and a horizontal one are present (else null)
  float* state;    // 2 * 2 * B*C*H floats (needed with a horizontal direction)
  uint32_t mask;
  int64_t planes;
  int H, W, dtype;
  int group_h, group_w;  // local-GSPN group lengths (0: global)
  int logits, renorm;    // w holds Eq. 6 logits (renorm: over on-line neighbours only)
  int y_pd;              // unmerged outputs (y is (n, B, C, H, W)); no partial sums needed
  // state kept for the backward (null when not kept): acc / acc_b then keep
  // the vertical directions' h, `sum` takes the horizontal pass's partial and
  // final sums, hsave[0] / hsave[1] left-to-right's / right-to-left's h
  float* sum;
  float* hsave[2];
  void* stream;
};
hipError_t large_fwd_f32(const LargeFwdArgs& a);
hipError_t large_fwd_bf16(const LargeFwdArgs& a);
inline hipError_t large_fwd(const LargeFwdArgs& a) {
  return a.dtype == 0 ? large_fwd_f32(a) : large_fwd_bf16(a);
}
bool large_fwd_fits(int H, int W, int dtype);

// backward of one horizontal direction for large planes (recompute + adjoint)
struct LargeBwdHArgs {
  const void* x;
  const void* lam;
  const void* dy;
  const void* u;
  const void* w;     // this direction's w0
  void* dw;          // this direction's dw0
  float* hbuf;       // B*C*H*W floats
  float* hsum;
  float* gsum;
  float* state;      // large_bwd_state_floats(planes, H) floats
  int first;         // first direction: hsum and gsum are stored, not added
  int dir;           // 0: left-to-right, 1: right-to-left
  int64_t planes;
  int H, W;
  int group;         // columns per local-GSPN group (0 or >= W: global)
  int logits, renorm;  // w holds Eq. 6 logits; dw is the gradient for the logits
  const void* hdy;   // unmerged outputs: this direction's dy; hsum (+)= dy * h
  int saved;         // hbuf already holds h (kept by the forward): no recompute, hsum untouched
  void* stream;
};

inline int64_t large_bwd_state_floats(int64_t planes, int H) { return 6 * planes * (int64_t)H; }
// recompute of the vertical directions' h for the same backward (the forward's
// vertical pass storing h): top-to-bottom into h_t2b, bottom-to-top into
// h_b2t (both present: one workgroup per direction and plane)
struct LargeBwdVArgs {
  const void* x;
  const void* lam;
  const void* w;     // all n directions, packed
  int slot_t2b, slot_b2t;  // weight slots, -1 when absent
  float* h_t2b;
  float* h_b2t;
  int64_t planes;
  int H, W;
  int group;         // rows per local-GSPN group (0: global)
  int logits, renorm;
  void* stream;
};
hipError_t large_bwd_v_rec_f32(const LargeBwdVArgs& a);
hipError_t large_bwd_v_rec_bf16(const LargeBwdVArgs& a);
inline hipError_t large_bwd_v_rec(const LargeBwdVArgs& a, int dtype) {
  return dtype == 0 ? large_bwd_v_rec_f32(a) : large_bwd_v_rec_bf16(a);
}
// adjoint of the vertical directions for the same backward (after
// large_bwd_v_rec): dw of both, gsum += g (fixed order)
struct LargeBwdVAdjArgs {
  const void* dy;
  const void* u;
  const void* w;     // all n directions, packed
  void* dw;          // all n directions, packed
  int slot_t2b, slot_b2t;
  const float* h_t2b;
  const float* h_b2t;
  float* gsum;
  int64_t planes;
  int H, W;
  int group;
  int logits, renorm;  // w holds Eq. 6 logits; dw is the gradient for the logits
  int y_pd;            // dy is (n, B, C, H, W): each direction's seed from its own map
  void* stream;
};
hipError_t large_bwd_v_adj_f32(const LargeBwdVAdjArgs& a);
hipError_t large_bwd_v_adj_bf16(const LargeBwdVAdjArgs& a);
inline hipError_t large_bwd_v_adj(const LargeBwdVAdjArgs& a, int dtype) {
  return dtype == 0 ? large_bwd_v_adj_f32(a) : large_bwd_v_adj_bf16(a);
}
hipError_t large_bwd_h_f32(const LargeBwdHArgs& a);
hipError_t large_bwd_h_bf16(const LargeBwdHArgs& a);
inline hipError_t large_bwd_h(const LargeBwdHArgs& a, int dtype) {
  return dtype == 0 ? large_bwd_h_f32(a) : large_bwd_h_bf16(a);
}
// both horizontal directions' adjoints at once, on h kept by the forward
// (l2r: dir 0, r2l: dir 1, both with saved set; separate state arrays)
hipError_t large_bwd_h_pair_f32(const LargeBwdHArgs& l2r, const LargeBwdHArgs& r2l);
hipError_t large_bwd_h_pair_bf16(const LargeBwdHArgs& l2r, const LargeBwdHArgs& r2l);
inline hipError_t large_bwd_h_pair(const LargeBwdHArgs& l2r, const LargeBwdHArgs& r2l, int dtype) {
  return dtype == 0 ? large_bwd_h_pair_f32(l2r, r2l) : large_bwd_h_pair_bf16(l2r, r2l);
}

}  // namespace gspn
