// C ABI of the GSPN line scan: argument checking, workspace sizing and dispatch.
// Host code only; the kernels live in the gspn_stream_*, gspn_resident_* and
// gspn_large_* sources.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <mutex>
#include <vector>

#include "../../include/gspn.h"
#include "gspn_launch.hpp"

using namespace gspn;

// Scratch of gspn_scan_fwd_noalloc: a file-scope device array, one copy per
// GPU.  In host code `scratch` names a host-side stand-in, so host code uses
// only the device address hipGetSymbolAddress returns (kept per device below).
static __device__ __align__(256) unsigned char scratch[GSPN_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// device address of the current device's scratch array (looked up once per device)
int scratch_for_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return GSPN_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return GSPN_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return GSPN_ERR_HIP;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return GSPN_OK;
}

constexpr size_t kWsAlign = 256;
// families whose kernels take local-GSPN groups (the streaming family always does)
constexpr bool kResidentGroupsFwd = true;
constexpr bool kResidentGroupsBwd = true;
constexpr bool kTwoPassGroups = true;

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

int popcount4(uint32_t m) { return (int)((m & 1) + ((m >> 1) & 1) + ((m >> 2) & 1) + ((m >> 3) & 1)); }

std::vector<int> dirs_of(uint32_t mask) {
  std::vector<int> d;
  for (int b : {DIR_T2B, DIR_B2T, DIR_L2R, DIR_R2L})
    if (mask & (uint32_t)b) d.push_back(b);
  return d;
}

size_t esize(int dtype) { return dtype == GSPN_F32 ? 4 : 2; }

// checked a*b for non-negative int64
bool mul_ok(int64_t a, int64_t b, int64_t* out) {
  if (a == 0 || b == 0) { *out = 0; return true; }
  if (a > INT64_MAX / b) return false;
  *out = a * b;
  return true;
}

constexpr uint32_t kAllFlags = GSPN_FLAG_W_LOGITS | GSPN_FLAG_EDGE_RENORM | GSPN_FLAG_LAM_PER_DIR |
                               GSPN_FLAG_U_PER_DIR | GSPN_FLAG_Y_PER_DIR | GSPN_FLAG_SAVE_STATE;

struct Problem {
  int64_t B, C, H, W, planes, npc;  // npc = elements per (B,C,H,W) tensor
  int n;
  bool empty;
  int gh, gw;                       // group lengths, 0 when the scan is global on that axis
  uint32_t flags;
  uint32_t mask;
  bool grouped() const { return gh > 0 || gw > 0; }
  bool lam_pd() const { return flags & GSPN_FLAG_LAM_PER_DIR; }
  bool u_pd() const { return flags & GSPN_FLAG_U_PER_DIR; }
  bool y_pd() const { return flags & GSPN_FLAG_Y_PER_DIR; }
  bool logits() const { return flags & GSPN_FLAG_W_LOGITS; }
};

int check_shape(int64_t B, int64_t C, int64_t H, int64_t W, uint32_t mask, int dtype, int64_t group_h,
                int64_t group_w, uint32_t flags, int algo, Problem* p) {
  if (dtype != GSPN_F32 && dtype != GSPN_BF16) return GSPN_ERR_DTYPE;
  if (mask == 0 || mask > 15u) return GSPN_ERR_MASK;
  if (algo < GSPN_ALGO_AUTO || algo > GSPN_ALGO_TWO_PASS) return GSPN_ERR_UNSUPPORTED;
  if (flags & ~kAllFlags) return GSPN_ERR_UNSUPPORTED;
  if ((flags & GSPN_FLAG_EDGE_RENORM) && !(flags & GSPN_FLAG_W_LOGITS)) return GSPN_ERR_UNSUPPORTED;
  if (group_h < 0 || group_w < 0) return GSPN_ERR_UNSUPPORTED;
  p->flags = flags;
  p->mask = mask;
  // a group at least as long as the axis is the global scan
  p->gh = (group_h == 0 || group_h >= H) ? 0 : (int)group_h;
  p->gw = (group_w == 0 || group_w >= W) ? 0 : (int)group_w;
  if (B < 0 || C < 0 || H < 0 || W < 0) return GSPN_ERR_SHAPE;
  p->B = B; p->C = C; p->H = H; p->W = W;
  p->n = popcount4(mask);
  int64_t planes, plane, npc, wtot;
  if (!mul_ok(B, C, &planes) || !mul_ok(H, W, &plane) || !mul_ok(planes, plane, &npc) ||
      !mul_ok(npc, 3 * p->n, &wtot) || !mul_ok(wtot, 4, &wtot))
    return GSPN_ERR_SHAPE;
  p->planes = planes;
  p->npc = npc;
  p->empty = npc == 0;
  if (p->empty) return GSPN_OK;
  if (H > GSPN_MAX_LINE || W > GSPN_MAX_LINE) return GSPN_ERR_UNSUPPORTED;
  if (planes > 0x7fffffffLL) return GSPN_ERR_UNSUPPORTED;
  return GSPN_OK;
}

struct Range {
  uintptr_t lo, hi;
};
bool overlap(Range a, Range b) { return a.lo < b.hi && b.lo < a.hi; }

int check_ptrs(const std::vector<std::pair<const void*, size_t>>& ins,
               const std::vector<std::pair<const void*, size_t>>& outs, size_t align) {
  for (auto& p : ins)
    if (!p.first) return GSPN_ERR_NULL;
  for (auto& p : outs)
    if (!p.first) return GSPN_ERR_NULL;
  for (auto& p : ins)
    if ((uintptr_t)p.first % align) return GSPN_ERR_ALIGN;
  for (auto& p : outs)
    if ((uintptr_t)p.first % align) return GSPN_ERR_ALIGN;
  for (size_t i = 0; i < outs.size(); ++i) {
    Range o{(uintptr_t)outs[i].first, (uintptr_t)outs[i].first + outs[i].second};
    for (auto& p : ins)
      if (overlap(o, Range{(uintptr_t)p.first, (uintptr_t)p.first + p.second})) return GSPN_ERR_ALIAS;
    for (size_t j = i + 1; j < outs.size(); ++j)
      if (overlap(o, Range{(uintptr_t)outs[j].first, (uintptr_t)outs[j].first + outs[j].second}))
        return GSPN_ERR_ALIAS;
  }
  return GSPN_OK;
}

int check_ws(void* ws, size_t ws_bytes, size_t need,
             const std::vector<std::pair<const void*, size_t>>& others) {
  if (need == 0) return GSPN_OK;
  if (!ws || ws_bytes < need) return GSPN_ERR_WORKSPACE;
  if ((uintptr_t)ws % kWsAlign) return GSPN_ERR_ALIGN;
  Range r{(uintptr_t)ws, (uintptr_t)ws + need};
  for (auto& p : others)
    if (p.first && overlap(r, Range{(uintptr_t)p.first, (uintptr_t)p.first + p.second}))
      return GSPN_ERR_ALIAS;
  return GSPN_OK;
}

// Eq. 6 logits and edge renormalisation are taken by every family; the
// per-direction maps by the generic resident kernels (forward: y_d unmerged,
// lam_d; u_d only with unmerged outputs), the per-wave resident backward and
// the streaming family.  Every family takes groups.
constexpr uint32_t kEq6Flags = GSPN_FLAG_W_LOGITS | GSPN_FLAG_EDGE_RENORM;
constexpr uint32_t kPdFlags = GSPN_FLAG_LAM_PER_DIR | GSPN_FLAG_U_PER_DIR | GSPN_FLAG_Y_PER_DIR;

bool resident_fits(const Problem& p, int dtype, bool backward) {
  if (p.flags & kPdFlags) {
    if (!backward && p.u_pd() && !p.y_pd()) return false;
    if (backward && p.H == 128 && p.W == 128) return false;  // the persistent backward merges
  }
  if (p.grouped() && !(backward ? kResidentGroupsBwd : kResidentGroupsFwd)) return false;
  return gspn::resident_fits((int)p.H, (int)p.W, dtype, backward, (!backward && p.y_pd()) ? p.n : 1);
}

// the two-pass family takes unmerged outputs (per-direction y and dy) but not
// per-direction lam or u
bool two_pass_fits(const Problem& p, int dtype, bool backward) {
  if ((p.flags & ~(kEq6Flags | GSPN_FLAG_Y_PER_DIR | GSPN_FLAG_SAVE_STATE)) || (p.grouped() && !kTwoPassGroups))
    return false;
  // the backward runs its horizontal directions on the two-pass kernels
  // (their vertical ones on the streaming kernels)
  if (backward && !(p.mask & (DIR_L2R | DIR_R2L))) return false;
  return gspn::large_fwd_fits((int)p.H, (int)p.W, dtype);
}

int choose_algo(const Problem& p, int dtype, int algo, bool backward) {
  if (algo == GSPN_ALGO_STREAM) return GSPN_ALGO_STREAM;
  if (algo == GSPN_ALGO_RESIDENT || algo == GSPN_ALGO_RESIDENT_GENERIC)
    return resident_fits(p, dtype, backward) ? algo : -1;
  if (algo == GSPN_ALGO_TWO_PASS) return two_pass_fits(p, dtype, backward) ? algo : -1;
  if (resident_fits(p, dtype, backward)) return GSPN_ALGO_RESIDENT;
  return two_pass_fits(p, dtype, backward) ? GSPN_ALGO_TWO_PASS : GSPN_ALGO_STREAM;
}

// two-pass layout: fp32 partial sums (n > 1; a second array when both vertical
// directions and a horizontal one are present: the vertical directions then
// run as independent workgroups, one array each), then the column state of the
// horizontal pass (2 parities x 2 directions x planes x H floats)
bool two_pass_split_v(uint32_t mask) {
  return (mask & DIR_T2B) && (mask & DIR_B2T) && (mask & (DIR_L2R | DIR_R2L));
}
size_t two_pass_acc_bytes(const Problem& p, uint32_t mask) {
  if (p.n <= 1) return 0;
  return round_up((size_t)p.npc * 4, kWsAlign) * (two_pass_split_v(mask) ? 2 : 1);
}
size_t two_pass_state_bytes(const Problem& p, uint32_t mask) {
  return (mask & (DIR_L2R | DIR_R2L)) ? round_up((size_t)4 * p.planes * p.H * 4, kWsAlign) : 0;
}

// GSPN_FLAG_SAVE_STATE: kept by the two-pass forward (merged outputs, a
// horizontal direction) as fp32 B*C*H*W arrays at the start of the workspace:
// the vertical directions' h (top-to-bottom, bottom-to-top), sum_d h_d (the
// horizontal pass's partial, then final sum), the horizontal directions' h
// (left-to-right, right-to-left), then the forward's column state.  The
// backward's own arrays follow.  `fwd_algo` is the family the forward runs.
constexpr size_t kAbsent = SIZE_MAX;
bool saves_state(const Problem& p, int fwd_algo) {
  return fwd_algo == GSPN_ALGO_TWO_PASS && (p.flags & GSPN_FLAG_SAVE_STATE) && !(p.flags & kPdFlags) &&
         (p.mask & (DIR_L2R | DIR_R2L));
}
struct SavedLayout {
  size_t h[4];  // T2B, B2T, L2R, R2L (kAbsent when the direction is not in the mask)
  size_t sum, state, total;
};
SavedLayout saved_layout(const Problem& p) {
  const size_t fb = round_up((size_t)p.npc * 4, kWsAlign);
  SavedLayout l{};
  size_t off = 0;
  const int bit[4] = {DIR_T2B, DIR_B2T, DIR_L2R, DIR_R2L};
  for (int d = 0; d < 2; ++d) l.h[d] = (p.mask & bit[d]) ? (off += fb) - fb : kAbsent;
  l.sum = off;
  off += fb;
  for (int d = 2; d < 4; ++d) l.h[d] = (p.mask & bit[d]) ? (off += fb) - fb : kAbsent;
  l.state = off;
  l.total = off + two_pass_state_bytes(p, p.mask);
  return l;
}
// backward reading the kept state: the forward's bytes, the sum of g, the
// column products of the two horizontal adjoints (they run together)
size_t bwd_state_bytes(const Problem& p) {
  return round_up((size_t)gspn::large_bwd_state_floats(p.planes, (int)p.H) * 4, kWsAlign);
}
size_t saved_bwd_ws_bytes(const Problem& p) {
  return saved_layout(p).total + round_up((size_t)p.npc * 4, kWsAlign) + 2 * bwd_state_bytes(p);
}

size_t fwd_ws_bytes(const Problem& p, int algo, uint32_t mask) {
  if (saves_state(p, algo)) return saved_layout(p).total;
  if (algo == GSPN_ALGO_STREAM && p.n > 1 && !p.y_pd()) return round_up((size_t)p.npc * 4, kWsAlign);
  if (algo == GSPN_ALGO_TWO_PASS)
    return (p.y_pd() ? 0 : two_pass_acc_bytes(p, mask)) + two_pass_state_bytes(p, mask);
  return 0;
}

// streaming backward: the previous line's h of one direction, the running
// sums of h and g (fp32 B*C*H*W arrays).  Two-pass backward: h of one
// direction (a horizontal one, then top-to-bottom), the sums of the
// horizontal directions' h and of every g, bottom-to-top's h when both
// vertical directions are present, then the column state of the horizontal
// launches.
bool both_vertical(uint32_t mask) { return (mask & DIR_T2B) && (mask & DIR_B2T); }
size_t bwd_ws_bytes(const Problem& p, int algo) {
  const size_t fb = round_up((size_t)p.npc * 4, kWsAlign);
  if (algo == GSPN_ALGO_STREAM) return 3 * fb;
  if (algo == GSPN_ALGO_TWO_PASS)
    return (both_vertical(p.mask) ? 4 : 3) * fb +
           round_up((size_t)gspn::large_bwd_state_floats(p.planes, (int)p.H) * 4, kWsAlign);
  return 0;
}

int hip_status(hipError_t e) { return e == hipSuccess ? GSPN_OK : GSPN_ERR_HIP; }

}  // namespace

extern "C" {

size_t gspn_scan_fwd_workspace_bytes(int64_t B, int64_t C, int64_t H, int64_t W, uint32_t mask,
                                     gspn_dtype dtype, int64_t group_h, int64_t group_w, uint32_t flags,
                                     int algo) {
  Problem p;
  if (check_shape(B, C, H, W, mask, dtype, group_h, group_w, flags, algo, &p) != GSPN_OK || p.empty)
    return 0;
  const int a = choose_algo(p, dtype, algo, false);
  return a < 0 ? 0 : fwd_ws_bytes(p, a, mask);
}

size_t gspn_scan_bwd_workspace_bytes(int64_t B, int64_t C, int64_t H, int64_t W, uint32_t mask,
                                     gspn_dtype dtype, int64_t group_h, int64_t group_w, uint32_t flags,
                                     int algo) {
  Problem p;
  if (check_shape(B, C, H, W, mask, dtype, group_h, group_w, flags, algo, &p) != GSPN_OK || p.empty)
    return 0;
  if (saves_state(p, choose_algo(p, dtype, algo, false))) return saved_bwd_ws_bytes(p);
  const int a = choose_algo(p, dtype, algo, true);
  if (a < 0) return 0;
  // AUTO runs the streaming family instead of the resident one when a pointer
  // is not 16-byte aligned, so its size covers that case too
  if (algo == GSPN_ALGO_AUTO && (a == GSPN_ALGO_RESIDENT || a == GSPN_ALGO_RESIDENT_GENERIC))
    return bwd_ws_bytes(p, GSPN_ALGO_STREAM);
  return bwd_ws_bytes(p, a);
}

int gspn_scan_fwd(const void* x, const void* w, const void* lam, const void* u, void* y,
                  int64_t B, int64_t C, int64_t H, int64_t W, uint32_t mask, gspn_dtype dtype,
                  int64_t group_h, int64_t group_w, uint32_t flags, int algo,
                  void* workspace, size_t workspace_bytes, void* stream) {
  Problem p;
  int st = check_shape(B, C, H, W, mask, dtype, group_h, group_w, flags, algo, &p);
  if (st != GSPN_OK || p.empty) return st;
  const size_t es = esize(dtype);
  const size_t tb = (size_t)p.npc * es, wb = tb * 3 * (size_t)p.n;
  const size_t lb = p.lam_pd() ? tb * p.n : tb, ub = p.u_pd() ? tb * p.n : tb, yb = p.y_pd() ? tb * p.n : tb;
  st = check_ptrs({{x, tb}, {w, wb}, {lam, lb}, {u, ub}}, {{y, yb}}, es);
  if (st != GSPN_OK) return st;
  int a = choose_algo(p, dtype, algo, false);
  if (a < 0) return GSPN_ERR_UNSUPPORTED;
  const bool keep = saves_state(p, a);
  if (a == GSPN_ALGO_TWO_PASS) {
    // the two-pass kernels read and write 16-byte vectors
    for (const void* q : {x, w, lam, u, (const void*)y})
      if ((uintptr_t)q % 16) {
        // a kept state must come from the two-pass kernels: no fallback then
        if (algo != GSPN_ALGO_AUTO || keep) return GSPN_ERR_ALIGN;
        a = GSPN_ALGO_STREAM;  // its workspace is never larger than the two-pass one
        break;
      }
  }
  const size_t need = fwd_ws_bytes(p, a, mask);
  st = check_ws(workspace, workspace_bytes, need, {{x, tb}, {w, wb}, {lam, lb}, {u, ub}, {y, yb}});
  if (st != GSPN_OK) return st;

  if (a == GSPN_ALGO_RESIDENT || a == GSPN_ALGO_RESIDENT_GENERIC) {
    ResidentFwdArgs r{};
    r.x = x; r.lam = lam; r.w = w; r.u = u; r.y = y;
    r.mask = mask; r.planes = p.planes; r.H = (int)H; r.W = (int)W; r.dtype = dtype;
    r.group_h = p.gh; r.group_w = p.gw;
    r.logits = p.logits(); r.renorm = (flags & GSPN_FLAG_EDGE_RENORM) ? 1 : 0;
    r.lam_pd = p.lam_pd(); r.u_pd = p.u_pd(); r.y_pd = p.y_pd();
    r.use_fixed = a == GSPN_ALGO_RESIDENT;
    r.stream = stream;
    return hip_status(resident_fwd(r));
  }
  if (a == GSPN_ALGO_TWO_PASS) {
    LargeFwdArgs l{};
    l.x = x; l.lam = lam; l.w = w; l.u = u; l.y = y;
    const size_t accb = p.y_pd() ? 0 : two_pass_acc_bytes(p, mask);
    l.acc = p.y_pd() ? nullptr : (float*)workspace;
    l.acc_b = (!p.y_pd() && two_pass_split_v(mask))
                  ? (float*)((char*)workspace + round_up((size_t)p.npc * 4, kWsAlign)) : nullptr;
    l.state = (float*)((char*)workspace + accb);
    if (keep) {
      // vertical h in acc / acc_b, the sums and horizontal h in their arrays
      const SavedLayout k = saved_layout(p);
      auto at = [&](size_t off) { return off == kAbsent ? nullptr : (float*)((char*)workspace + off); };
      l.acc = at(k.h[0] != kAbsent ? k.h[0] : k.h[1]);
      l.acc_b = (k.h[0] != kAbsent && k.h[1] != kAbsent) ? at(k.h[1]) : nullptr;
      l.sum = at(k.sum);
      l.hsave[0] = at(k.h[2]);
      l.hsave[1] = at(k.h[3]);
      l.state = at(k.state);
    }
    l.y_pd = p.y_pd();
    l.mask = mask; l.planes = p.planes; l.H = (int)H; l.W = (int)W; l.dtype = dtype;
    l.group_h = p.gh; l.group_w = p.gw;
    l.logits = p.logits(); l.renorm = (flags & GSPN_FLAG_EDGE_RENORM) ? 1 : 0;
    l.stream = stream;
    return hip_status(large_fwd(l));
  }
  const std::vector<int> ds = dirs_of(mask);
  const int n = (int)ds.size();
  const bool merge = n > 1 && !p.y_pd();
  for (int i = 0; i < n; ++i) {
    StreamFwdArgs s{};
    s.x = x;
    s.lam = (const char*)lam + (p.lam_pd() ? i * tb : 0);
    s.u = (const char*)u + (p.u_pd() ? i * tb : 0);
    s.y = (char*)y + (p.y_pd() ? i * tb : 0);
    s.w = (const char*)w + (size_t)i * 3 * tb;
    s.wstride = p.npc;
    s.acc = merge ? (float*)workspace : nullptr;
    s.hprev_out = nullptr;
    s.first = i == 0;
    s.mode = (!merge || i == n - 1) ? MODE_FINAL : (i == 0 ? MODE_STORE : MODE_ADD);
    s.planes = p.planes; s.H = (int)H; s.W = (int)W; s.dir = ds[i]; s.dtype = dtype;
    s.group = (ds[i] == DIR_T2B || ds[i] == DIR_B2T) ? p.gh : p.gw;
    s.logits = p.logits(); s.renorm = (flags & GSPN_FLAG_EDGE_RENORM) ? 1 : 0;
    s.ugate = merge && p.u_pd();
    s.stream = stream;
    st = hip_status(stream_fwd_pass(s));
    if (st != GSPN_OK) return st;
  }
  return GSPN_OK;
}

int gspn_scan_fwd_noalloc(const void* x, const void* w, const void* lam, const void* u, void* y,
                          int64_t B, int64_t C, int64_t H, int64_t W, uint32_t mask, gspn_dtype dtype,
                          int64_t group_h, int64_t group_w, uint32_t flags, void* stream) {
  Problem p;
  int st = check_shape(B, C, H, W, mask, dtype, group_h, group_w, flags, GSPN_ALGO_AUTO, &p);
  if (st != GSPN_OK || p.empty) return st;
  if (flags & GSPN_FLAG_SAVE_STATE) return GSPN_ERR_UNSUPPORTED;  // a kept state needs the caller's workspace
  const int a = choose_algo(p, dtype, GSPN_ALGO_AUTO, false);
  if (a < 0) return GSPN_ERR_UNSUPPORTED;
  // the AUTO size also covers the streaming fallback of misaligned two-pass calls
  const size_t need = fwd_ws_bytes(p, a, mask);
  if (need > (size_t)GSPN_NOALLOC_SCRATCH_BYTES) return GSPN_ERR_WORKSPACE;
  void* ws = nullptr;
  if (need > 0) {
    st = scratch_for_current_device(&ws);
    if (st != GSPN_OK) return st;
  }
  return gspn_scan_fwd(x, w, lam, u, y, B, C, H, W, mask, dtype, group_h, group_w, flags, GSPN_ALGO_AUTO,
                       ws, need > 0 ? (size_t)GSPN_NOALLOC_SCRATCH_BYTES : 0, stream);
}

int gspn_scan_bwd(const void* dy, const void* x, const void* w, const void* lam, const void* u,
                  void* dx, void* dw, void* dlam, void* du, int64_t B, int64_t C, int64_t H,
                  int64_t W, uint32_t mask, gspn_dtype dtype, int64_t group_h, int64_t group_w,
                  uint32_t flags, int algo, void* workspace, size_t workspace_bytes, void* stream) {
  Problem p;
  int st = check_shape(B, C, H, W, mask, dtype, group_h, group_w, flags, algo, &p);
  if (st != GSPN_OK || p.empty) return st;
  const size_t es = esize(dtype);
  const size_t tb = (size_t)p.npc * es, wb = tb * 3 * (size_t)p.n;
  const size_t lb = p.lam_pd() ? tb * p.n : tb, ub = p.u_pd() ? tb * p.n : tb, yb = p.y_pd() ? tb * p.n : tb;
  st = check_ptrs({{dy, yb}, {x, tb}, {w, wb}, {lam, lb}, {u, ub}},
                  {{dx, tb}, {dw, wb}, {dlam, lb}, {du, ub}}, es);
  if (st != GSPN_OK) return st;
  // a state kept by the forward (two-pass family) is read by the two-pass backward
  bool keep = saves_state(p, choose_algo(p, dtype, algo, false));
  int a = keep ? GSPN_ALGO_TWO_PASS : choose_algo(p, dtype, algo, true);
  if (a < 0) return GSPN_ERR_UNSUPPORTED;
  if (a == GSPN_ALGO_RESIDENT || a == GSPN_ALGO_RESIDENT_GENERIC || a == GSPN_ALGO_TWO_PASS) {
    // the resident and two-pass backward kernels read and write 16-byte vectors
    for (const void* q : {dy, x, w, lam, u, (const void*)dx, (const void*)dw, (const void*)dlam, (const void*)du})
      if ((uintptr_t)q % 16) {
        if (algo != GSPN_ALGO_AUTO) return GSPN_ERR_ALIGN;
        a = GSPN_ALGO_STREAM;  // the AUTO workspace size includes this case (a kept state is ignored)
        keep = false;
        break;
      }
  }
  const size_t need = keep ? saved_bwd_ws_bytes(p) : bwd_ws_bytes(p, a);
  st = check_ws(workspace, workspace_bytes, need,
                {{dy, yb}, {x, tb}, {w, wb}, {lam, lb}, {u, ub}, {dx, tb}, {dw, wb}, {dlam, lb}, {du, ub}});
  if (st != GSPN_OK) return st;

  if (a == GSPN_ALGO_RESIDENT || a == GSPN_ALGO_RESIDENT_GENERIC) {
    ResidentBwdArgs r{};
    r.dy = dy; r.x = x; r.lam = lam; r.w = w; r.u = u;
    r.dx = dx; r.dw = dw; r.dlam = dlam; r.du = du;
    r.mask = mask; r.planes = p.planes; r.H = (int)H; r.W = (int)W; r.dtype = dtype;
    r.group_h = p.gh; r.group_w = p.gw;
    r.logits = p.logits(); r.renorm = (flags & GSPN_FLAG_EDGE_RENORM) ? 1 : 0;
    r.lam_pd = p.lam_pd(); r.u_pd = p.u_pd(); r.y_pd = p.y_pd();
    r.use_staged = a == GSPN_ALGO_RESIDENT;
    r.stream = stream;
    return hip_status(resident_bwd(r));
  }
  const size_t fb = round_up((size_t)p.npc * 4, kWsAlign);
  float* hprev = (float*)workspace;
  float* hsum = (float*)((char*)workspace + fb);
  float* gsum = (float*)((char*)workspace + 2 * fb);
  const std::vector<int> ds = dirs_of(mask);
  if (a == GSPN_ALGO_TWO_PASS) {
    // horizontal directions first (their h through the first array), then the
    // vertical directions' h at once (first and fourth arrays), then their
    // adjoints; the finish adds the vertical h to the horizontal sum.  With a
    // kept state every h and their sum come from the forward instead.
    float* hb = both_vertical(mask) ? (float*)((char*)workspace + 3 * fb) : nullptr;
    float* state = (float*)((char*)workspace + (both_vertical(mask) ? 4 : 3) * fb);
    const SavedLayout k = saved_layout(p);
    auto kept = [&](size_t off) { return off == kAbsent ? nullptr : (float*)((char*)workspace + off); };
    if (keep) {
      gsum = (float*)((char*)workspace + k.total);
      state = (float*)((char*)workspace + k.total + fb);
    }
    int slot[4] = {-1, -1, -1, -1};
    for (int i = 0; i < (int)ds.size(); ++i) slot[ds[i] == DIR_T2B ? 0 : ds[i] == DIR_B2T ? 1 : ds[i] == DIR_L2R ? 2 : 3] = i;
    bool first = true;
    LargeBwdHArgs hz[2] = {};
    for (int d = 2; d < 4; ++d) {
      if (slot[d] < 0) continue;
      LargeBwdHArgs& l = hz[d - 2];
      l.x = x; l.lam = lam; l.u = u;
      l.dy = (const char*)dy + (p.y_pd() ? (size_t)slot[d] * tb : 0);
      l.hdy = p.y_pd() ? l.dy : nullptr;
      l.w = (const char*)w + (size_t)slot[d] * 3 * tb;
      l.dw = (char*)dw + (size_t)slot[d] * 3 * tb;
      l.hbuf = keep ? kept(k.h[d]) : hprev; l.hsum = keep ? nullptr : hsum; l.gsum = gsum; l.state = state;
      l.saved = keep ? 1 : 0;
      l.first = first ? 1 : 0;
      l.dir = d == 3 ? 1 : 0;
      l.planes = p.planes; l.H = (int)H; l.W = (int)W;
      l.group = p.gw;
      l.logits = p.logits(); l.renorm = (flags & GSPN_FLAG_EDGE_RENORM) ? 1 : 0;
      l.stream = stream;
      if (keep && slot[2] >= 0 && slot[3] >= 0) {
        // both adjoints at once below, each with its own column products
        if (d == 3) l.state = (float*)((char*)state + bwd_state_bytes(p));
        continue;
      }
      st = hip_status(large_bwd_h(l, dtype));
      if (st != GSPN_OK) return st;
      first = false;
    }
    if (keep && slot[2] >= 0 && slot[3] >= 0) {
      st = hip_status(large_bwd_h_pair(hz[0], hz[1], dtype));
      if (st != GSPN_OK) return st;
    }
    float* hv[2] = {nullptr, nullptr};  // h of top-to-bottom, bottom-to-top
    if (keep) {
      hv[0] = kept(k.h[0]);
      hv[1] = kept(k.h[1]);
    } else if (slot[0] >= 0 || slot[1] >= 0) {
      hv[0] = slot[0] >= 0 ? hprev : nullptr;
      hv[1] = slot[1] >= 0 ? (slot[0] >= 0 ? hb : hprev) : nullptr;
      LargeBwdVArgs v{};
      v.x = x; v.lam = lam; v.w = w;
      v.slot_t2b = slot[0]; v.slot_b2t = slot[1];
      v.h_t2b = hv[0]; v.h_b2t = hv[1];
      v.planes = p.planes; v.H = (int)H; v.W = (int)W;
      v.group = p.gh;
      v.logits = p.logits(); v.renorm = (flags & GSPN_FLAG_EDGE_RENORM) ? 1 : 0;
      v.stream = stream;
      st = hip_status(large_bwd_v_rec(v, dtype));
      if (st != GSPN_OK) return st;
    }
    if (slot[0] >= 0 || slot[1] >= 0) {
      LargeBwdVAdjArgs r{};
      r.dy = dy; r.u = u; r.w = w; r.dw = dw;
      r.slot_t2b = slot[0]; r.slot_b2t = slot[1];
      r.h_t2b = hv[0]; r.h_b2t = hv[1];
      r.gsum = gsum;
      r.planes = p.planes; r.H = (int)H; r.W = (int)W;
      r.group = p.gh;
      r.logits = p.logits(); r.renorm = (flags & GSPN_FLAG_EDGE_RENORM) ? 1 : 0;
      r.y_pd = p.y_pd();
      r.stream = stream;
      st = hip_status(large_bwd_v_adj(r, dtype));
      if (st != GSPN_OK) return st;
    }
    GradFinishArgs g{};
    g.x = x; g.lam = lam; g.dy = dy; g.gsum = gsum; g.hsum = hsum; g.hsum2 = hv[0] ? hv[0] : hv[1];
    g.hsum3 = hv[0] ? hv[1] : nullptr;
    if (keep) {
      // du = dy * sum_d h_d, the sum the forward formed
      g.hsum = kept(k.sum);
      g.hsum2 = g.hsum3 = nullptr;
    }
    if (p.y_pd()) {
      // unmerged outputs: du = sum_d dy_d h_d (the horizontal part is in hsum)
      const int s2 = hv[0] ? slot[0] : slot[1], s3 = hv[0] ? slot[1] : -1;
      g.du_mode = 3;
      g.dy2 = s2 >= 0 ? (const char*)dy + (size_t)s2 * tb : nullptr;
      g.dy3 = s3 >= 0 ? (const char*)dy + (size_t)s3 * tb : nullptr;
    }
    g.dx = dx; g.dlam = dlam; g.du = du; g.n = p.npc; g.dtype = dtype;
    g.stream = stream;
    return hip_status(grad_finish(g));
  }
  const bool per_dir = p.lam_pd() || p.u_pd() || p.y_pd();
  for (int i = 0; i < (int)ds.size(); ++i) {
    const void* dy_i = (const char*)dy + (p.y_pd() ? i * tb : 0);
    const void* lam_i = (const char*)lam + (p.lam_pd() ? i * tb : 0);
    const void* u_i = (const char*)u + (p.u_pd() ? i * tb : 0);
    const int group = (ds[i] == DIR_T2B || ds[i] == DIR_B2T) ? p.gh : p.gw;
    StreamFwdArgs f{};
    f.x = x; f.lam = lam_i; f.u = nullptr; f.y = nullptr;
    f.w = (const char*)w + (size_t)i * 3 * tb;
    f.wstride = p.npc;
    f.acc = hsum;
    f.hprev_out = hprev;
    if (per_dir && (p.u_pd() || p.y_pd())) {
      f.dy = dy_i;                                      // hsum (+)= dy_d h, or du_d = dy_d h
      f.du = p.u_pd() ? (char*)du + i * tb : nullptr;
      f.hdy = p.u_pd() ? 0 : 1;
    }
    f.first = i == 0;
    f.mode = MODE_REC;
    f.planes = p.planes; f.H = (int)H; f.W = (int)W; f.dir = ds[i]; f.dtype = dtype;
    f.group = group;
    f.logits = p.logits(); f.renorm = (flags & GSPN_FLAG_EDGE_RENORM) ? 1 : 0;
    f.stream = stream;
    st = hip_status(stream_fwd_pass(f));
    if (st != GSPN_OK) return st;
    StreamAdjArgs r{};
    r.dy = dy_i; r.u = u_i;
    r.w = f.w;
    r.wstride = p.npc;
    r.hprev = hprev;
    r.dw = (char*)dw + (size_t)i * 3 * tb;
    r.gsum = gsum;
    if (p.lam_pd()) {
      r.lamw = 1;
      r.lam = lam_i;
      r.x = x;
      r.dlam = (char*)dlam + i * tb;
    }
    r.first = i == 0;
    r.planes = p.planes; r.H = (int)H; r.W = (int)W; r.dir = ds[i]; r.dtype = dtype;
    r.group = group;
    r.logits = f.logits; r.renorm = f.renorm;
    r.stream = stream;
    st = hip_status(stream_adj_pass(r));
    if (st != GSPN_OK) return st;
  }
  GradFinishArgs g{};
  g.x = x; g.lam = lam; g.dy = dy; g.gsum = gsum; g.hsum = hsum;
  g.dx = dx; g.dlam = p.lam_pd() ? nullptr : dlam; g.du = du; g.n = p.npc; g.dtype = dtype;
  g.dx_mode = p.lam_pd() ? 1 : 0;
  g.du_mode = p.u_pd() ? 2 : (p.y_pd() ? 1 : 0);
  g.stream = stream;
  return hip_status(grad_finish(g));
}

const char* gspn_strerror(int status) {
  switch (status) {
    case GSPN_OK: return "success";
    case GSPN_ERR_NULL: return "a required pointer is NULL";
    case GSPN_ERR_SHAPE: return "invalid shape: negative dimension or element count overflow";
    case GSPN_ERR_MASK: return "invalid direction mask: must be in [1, 15]";
    case GSPN_ERR_DTYPE: return "unknown dtype";
    case GSPN_ERR_ALIGN: return "misaligned pointer";
    case GSPN_ERR_ALIAS: return "an output overlaps an input or another output";
    case GSPN_ERR_UNSUPPORTED: return "unsupported: line longer than GSPN_MAX_LINE, too many planes, unknown flags, "
                                      "edge renormalisation without logits, negative group, or forced algorithm cannot run";
    case GSPN_ERR_WORKSPACE: return "workspace missing or too small (gspn_scan_fwd_noalloc: the problem needs "
                                    "more than GSPN_NOALLOC_SCRATCH_BYTES of scratch)";
    case GSPN_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

int gspn_version(void) { return 200; }

}  // extern "C"
