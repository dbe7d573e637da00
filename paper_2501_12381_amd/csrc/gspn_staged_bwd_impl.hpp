// Staged backward kernel for small square planes (S x S, S <= 32): every input
// of the workgroup's planes is copied into LDS once (direct global -> LDS
// 16-byte copies, consecutive lanes on consecutive addresses), the scans read
// only LDS, and every gradient leaves in coalesced 16-byte stores.  HBM sees
// the algorithmic bytes: 4 + 3n maps read (x, lam, u, dy, the n directions'
// w) and 3 + 3n written (dx, dlam, du, dw) per plane.
//
// Work split (the order of operations of the resident backward):
//   prologue  all threads: the planes' input maps -> LDS (input dtype);
//   phase F   wave d recomputes h_d (Eq. 1) into its fp32 array;
//   du        du = dy * (h_T2B + h_B2T + h_L2R + h_R2L), fixed order;
//   phase A   wave d runs the adjoint scan g = u dy + (transposed stencil of
//             the next line's w and g), writes dw_k = g * h_prev(p+k-1) over
//             the w_k entry it has just consumed, and g over h in its array,
//             then stores its three dw maps LDS -> HBM without waiting for the
//             other waves;
//   dx, dlam  from the fixed-order sum of g.
// One workgroup per group of planes; with at most ~80 KB of LDS each, two
// workgroups share a compute unit, so one's copies overlap the other's scans.
#pragma once

#include "gspn_device.hpp"
#include "gspn_launch.hpp"
#include "gspn_resident_impl.hpp"
#include "gspn_resident_bwd_impl.hpp"
#include "gspn_widebwd_impl.hpp"

namespace gspn {

template <typename T, int S>
struct StagedCfg {
  static constexpr int SEG = S <= 15 ? 16 : (S <= 31 ? 32 : 64);  // lanes per plane (> S, or one plane)
  static constexpr int HW = S * S;
  static constexpr int MAPB = HW * (int)sizeof(T);  // bytes of one map
  static constexpr int P = S + 1;                   // array pitch
  static constexpr int ARR = (S + 1) * P;           // floats per direction array
  static constexpr int VE = 16 / (int)sizeof(T);    // elements per 16-byte vector
  static constexpr int NVM = MAPB / 16;             // 16-byte vectors per map
  // LDS of a group of ppw planes with nd directions: the 4 + 3 nd input maps,
  // then one fp32 array per (plane, direction)
  static constexpr int bytes(int ppw, int nd) { return ppw * (4 + 3 * nd) * MAPB + ppw * nd * ARR * 4; }
  // planes per workgroup: as many as the segments of a wave allow while the
  // workgroup's LDS stays within 80 KiB (two workgroups per compute unit)
  static constexpr int PPW = (64 / SEG >= 4 && bytes(4, 4) <= 80 * 1024) ? 4
                           : (64 / SEG >= 2 && bytes(2, 4) <= 80 * 1024) ? 2 : 1;
  static constexpr int MS = PPW * HW;  // elements between consecutive maps (LDS is [map][plane][HW])
  static constexpr int MV = PPW * NVM;  // 16-byte vectors of one map in LDS
  static_assert(S <= 32 && S % 2 == 0, "staged backward takes even S <= 32");
  static_assert(MAPB % 16 == 0, "a map must be a whole number of 16-byte vectors");
  static_assert(MV <= 256, "the elementwise passes take one vector per thread");
};

// map indices of the staged block: x, lam, u, dy, then w of slot s, k at 4 + 3 s + k.
// LDS holds [map][plane][HW]: the group's planes of one map are contiguous, as
// they are in global memory.
enum { SM_X = 0, SM_LAM = 1, SM_U = 2, SM_DY = 3, SM_W = 4 };

template <typename T>
__device__ __forceinline__ float lds_elem(const T* p) { return to_f(*p); }

// Two consecutive LDS elements (address aligned to two elements) as floats, and back.
__device__ __forceinline__ void lds_get2(const bf16* p, float& a, float& b) {
  const uint32_t v = *reinterpret_cast<const uint32_t*>(p);
  a = bf_lo(v);
  b = bf_hi(v);
}
__device__ __forceinline__ void lds_get2(const float* p, float& a, float& b) {
  const float2 v = *reinterpret_cast<const float2*>(p);
  a = v.x;
  b = v.y;
}
__device__ __forceinline__ void lds_put2(bf16* p, float a, float b) { *reinterpret_cast<uint32_t*>(p) = pack_bf2(a, b); }
__device__ __forceinline__ void lds_put2(float* p, float a, float b) { *reinterpret_cast<float2*>(p) = make_float2(a, b); }

// The scans run in pairs of steps, with the operands of the next pair read
// (in program order before this pair's stores, which never touch them) while
// this pair computes.  In a horizontal scan the two lines of a pair are
// adjacent elements of each row, so one 2-element access serves both steps.

// One direction's forward recompute from LDS into harr.  harr holds lam * x on
// entry; each line's entry is read (one pair ahead) before h overwrites it.
// GRP: local GSPN; bit l of gst is set when line l starts a group.
// LG: w holds Eq. 6 logits, normalised as they are read.
template <typename T, int S, bool HZ, bool REV, bool GRP, bool LG>
__device__ __forceinline__ void staged_forward(const T* __restrict__ w3, float* __restrict__ harr, int sl,
                                               bool lane_ok, uint64_t gst, bool renorm) {
  using C = StagedCfg<T, S>;
  constexpr int NP = S / 2;
  const bool valid = lane_ok && sl < S;
  const int pos = valid ? sl : 0;
  const int aoff = valid ? (HZ ? sl * C::P : sl) : (HZ ? S * C::P : S);
  auto line_of = [](int s) { return REV ? S - 1 - s : s; };
  auto elem = [&](int line) { return HZ ? pos * S + line : line * S + pos; };
  auto aidx = [&](int line) { return aoff + (HZ ? line : line * C::P); };
  // lower line of pair j, and which step of the pair takes it
  auto pair_lo = [](int j) { return REV ? S - 2 - 2 * j : 2 * j; };
  constexpr int SA = REV ? 1 : 0;
  // operands of the pair's two steps: lam * x, w0, w1, w2
  auto fetch = [&](float (&d)[2][4], int j) __attribute__((always_inline)) {
    if constexpr (HZ) {
      const int lo = pair_lo(j), e = elem(lo);
      d[SA][0] = harr[aidx(lo)];
      d[1 - SA][0] = harr[aidx(lo + 1)];
      lds_get2(w3 + e, d[SA][1], d[1 - SA][1]);
      lds_get2(w3 + C::MS + e, d[SA][2], d[1 - SA][2]);
      lds_get2(w3 + 2 * C::MS + e, d[SA][3], d[1 - SA][3]);
    } else {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int line = line_of(2 * j + t), e = elem(line);
        d[t][0] = harr[aidx(line)];
        d[t][1] = lds_elem(w3 + e);
        d[t][2] = lds_elem(w3 + C::MS + e);
        d[t][3] = lds_elem(w3 + 2 * C::MS + e);
      }
    }
  };
  float pre[2][4];
  fetch(pre, 0);
  float hp = 0.f;
#pragma unroll
  for (int j = 0; j < NP; ++j) {
    float cur[2][4];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) cur[t][i] = pre[t][i];
    if (j + 1 < NP) fetch(pre, j + 1);
    if constexpr (LG) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const Norm3 r = normalize3(cur[t][1], cur[t][2], cur[t][3], sl == 0, sl == S - 1, renorm);
        cur[t][1] = r.w[0];
        cur[t][2] = r.w[1];
        cur[t][3] = r.w[2];
      }
    }
    float hv[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      if (GRP && ((gst >> line_of(2 * j + t)) & 1)) hp = 0.f;  // a group starts at this line
      const float hl = from_prev_lane(hp), hr = from_next_lane(hp);
      float h = fmaf(cur[t][2], hp, cur[t][0]);
      h = fmaf(cur[t][1], hl, h);
      h = fmaf(cur[t][3], hr, h);
      hp = valid ? h : 0.f;  // padding lanes stay zero: they are the row's zero boundary
      hv[t] = hp;
      if constexpr (!HZ) harr[aidx(line_of(2 * j + t))] = hp;
    }
    if constexpr (HZ) {
      const int lo = pair_lo(j);
      harr[aidx(lo)] = hv[SA];
      harr[aidx(lo + 1)] = hv[1 - SA];
    }
  }
}

// One direction's adjoint from LDS; dw overwrites the consumed w entries and
// g overwrites h.  Padding lanes (and lanes of absent planes) hold g = 0, so
// their finite weights (absent planes' are zero-filled) send nothing to a
// real lane; their stores are skipped.
// LG: w holds Eq. 6 logits; dw becomes their gradient (the Jacobian of the
// normalisation applied per pixel).
template <typename T, int S, bool HZ, bool REV, bool GRP, bool LG>
__device__ __forceinline__ void staged_adjoint(const float* __restrict__ udy, T* __restrict__ w3,
                                               float* __restrict__ harr, int sl, bool lane_ok,
                                               uint64_t gst, bool renorm) {
  using C = StagedCfg<T, S>;
  constexpr int NP = S / 2;
  const bool valid = lane_ok && sl < S;
  const int pos = valid ? sl : 0;
  const int aoff = valid ? (HZ ? sl * C::P : sl) : (HZ ? S * C::P : S);
  auto line_of = [](int s) { return REV ? s : S - 1 - s; };  // against the scan order
  auto prev_of = [](int line) { return REV ? line + 1 : line - 1; };  // previous line in scan order
  // a line that starts a group read a zero state
  auto has_prev = [&](int line) { return (REV ? line + 1 < S : line > 0) && !(GRP && ((gst >> line) & 1)); };
  auto elem = [&](int line) { return HZ ? pos * S + line : line * S + pos; };
  auto aidx = [&](int line) { return aoff + (HZ ? line : line * C::P); };
  auto pair_lo = [](int j) { return REV ? 2 * j : S - 2 - 2 * j; };
  constexpr int SA = REV ? 0 : 1;  // step of the pair that takes the lower line
  // per step: u*dy, w0, w1, w2 of the line and h of its previous line
  auto fetch = [&](float (&d)[2][5], int j) __attribute__((always_inline)) {
    if constexpr (HZ) {
      const int lo = pair_lo(j), e = elem(lo);
      lds_get2(udy + e, d[SA][0], d[1 - SA][0]);
      lds_get2(w3 + e, d[SA][1], d[1 - SA][1]);
      lds_get2(w3 + C::MS + e, d[SA][2], d[1 - SA][2]);
      lds_get2(w3 + 2 * C::MS + e, d[SA][3], d[1 - SA][3]);
      d[SA][4] = has_prev(lo) ? harr[aidx(prev_of(lo))] : 0.f;
      d[1 - SA][4] = has_prev(lo + 1) ? harr[aidx(prev_of(lo + 1))] : 0.f;
    } else {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int line = line_of(2 * j + t), e = elem(line);
        d[t][0] = udy[e];
        d[t][1] = lds_elem(w3 + e);
        d[t][2] = lds_elem(w3 + C::MS + e);
        d[t][3] = lds_elem(w3 + 2 * C::MS + e);
        d[t][4] = has_prev(line) ? harr[aidx(prev_of(line))] : 0.f;
      }
    }
  };
  float pre[2][5];
  fetch(pre, 0);
  float gn = 0.f, wn0 = 0.f, wn1 = 0.f, wn2 = 0.f;
#pragma unroll
  for (int j = 0; j < NP; ++j) {
    float cur[2][5];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 5; ++i) cur[t][i] = pre[t][i];
    if (j + 1 < NP) fetch(pre, j + 1);
    float gv[2], dv[2][3];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      // u * dy + transposed stencil of the next line (neighbour p+1 sends its
      // k = 0 term, neighbour p-1 its k = 2 term); none when that line starts a group
      if constexpr (GRP) {
        const int succ = REV ? line_of(2 * j + t) - 1 : line_of(2 * j + t) + 1;
        if (succ >= 0 && succ < S && ((gst >> succ) & 1)) gn = 0.f;
      }
      const float a0 = wn0 * gn, a2 = wn2 * gn;
      float g = fmaf(wn1, gn, cur[t][0]);
      g += from_next_lane(a0);
      g += from_prev_lane(a2);
      const float hpv = cur[t][4];
      dv[t][0] = g * from_prev_lane(hpv);
      dv[t][1] = g * hpv;
      dv[t][2] = g * from_next_lane(hpv);
      gv[t] = g;
      gn = valid ? g : 0.f;
      if constexpr (LG) {
        const Norm3 r = normalize3(cur[t][1], cur[t][2], cur[t][3], sl == 0, sl == S - 1, renorm);
        norm3_vjp(r, dv[t][0], dv[t][1], dv[t][2]);
        wn0 = r.w[0];
        wn1 = r.w[1];
        wn2 = r.w[2];
      } else {
        wn0 = cur[t][1];
        wn1 = cur[t][2];
        wn2 = cur[t][3];
      }
      if constexpr (!HZ) {
        if (valid) {
          const int line = line_of(2 * j + t), e = elem(line);
          harr[aidx(line)] = g;
          w3[e] = from_f<T>(dv[t][0]);
          w3[C::MS + e] = from_f<T>(dv[t][1]);
          w3[2 * C::MS + e] = from_f<T>(dv[t][2]);
        }
      }
    }
    if constexpr (HZ) {
      if (valid) {
        const int lo = pair_lo(j), e = elem(lo);
        harr[aidx(lo)] = gv[SA];
        harr[aidx(lo + 1)] = gv[1 - SA];
        lds_put2(w3 + e, dv[SA][0], dv[1 - SA][0]);
        lds_put2(w3 + C::MS + e, dv[SA][1], dv[1 - SA][1]);
        lds_put2(w3 + 2 * C::MS + e, dv[SA][2], dv[1 - SA][2]);
      }
    }
  }
}

// Row-major element e of a plane -> its index in a direction array (row pitch S + 1).
template <int S>
__device__ __forceinline__ int staged_aidx(int e0, int r0, int c0, int q) {
  return e0 + q + r0 + (c0 + q >= S ? 1 : 0);  // a vector (fewer than S elements) breaks a row at most once
}

// ND: directions present (compile time, so every index below divides by
// constants).  Direction arrays are indexed by slot (present directions in
// increasing direction order), [plane][slot][(S + 1) x (S + 1)].
template <typename T, int S, int ND, bool GRP, bool LG>
__global__ void __launch_bounds__(256) staged_bwd_kernel(ResBwdParams p) {
  using C = StagedCfg<T, S>;
  constexpr int PPW = C::PPW, HW = C::HW, NVM = C::NVM, VE = C::VE, MV = C::MV;
  constexpr int nm = 4 + 3 * ND;  // maps per plane (x, lam, u, dy, w of each present direction)
  constexpr int NCH = (MV + 63) / 64;
  constexpr int NA = PPW * ND;    // direction arrays
  extern __shared__ float4 lds4[];
  T* s_flat = reinterpret_cast<T*>(lds4);
  float* s_arr = reinterpret_cast<float*>(lds4 + nm * MV);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;  // wave = direction
  const int64_t g0 = (int64_t)blockIdx.x * PPW;
  const int64_t pmax = p.planes - g0;
  const int np = (int)(pmax < PPW ? pmax : PPW);  // planes of this group
  const int nv = np * NVM;                        // vectors per map present

  // zero the arrays' padding row and column (the zero boundary that padding
  // lanes read and write) before any copy is in flight
  {
    constexpr int NZ = 2 * S + 1;
    for (int i = tid; i < NA * NZ; i += 256) {
      const int a = i / NZ, k = i - a * NZ;
      s_arr[a * C::ARR + (k <= S ? k * C::P + S : S * C::P + (k - S - 1))] = 0.f;
    }
  }

  // the weight maps of planes past the end of the tensor are zero-filled (the
  // copies skip them; their lanes multiply these weights by g = 0)
  if (np < PPW) {
    for (int i = tid; i < 3 * ND * (PPW - np) * HW; i += 256) {
      const int m = i / ((PPW - np) * HW), r = i - m * ((PPW - np) * HW);
      s_flat[(SM_W + m) * C::MS + np * HW + r] = from_f<T>(0.f);
    }
  }

  // the group's maps into LDS, [map][plane][HW]: map m of the group is one
  // contiguous run in global memory and in LDS; wave w copies maps w, w + 4, ...
  // with 16-byte direct copies (consecutive lanes on consecutive vectors), the
  // last block of a run with its lanes past the end switched off
  for (int m = wave; m < nm; m += 4) {
    const char* src = (const char*)(m == SM_X ? p.x : (m == SM_LAM ? p.lam : (m == SM_U ? p.u : (m == SM_DY ? p.dy : p.w))));
    if (m >= SM_W) src += (int64_t)(m - SM_W) * p.npc * (int64_t)sizeof(T);  // w maps: slot-major, packed
    src += g0 * HW * (int64_t)sizeof(T);
    float4* dst = lds4 + m * MV;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      if (c * 64 + lane < nv)
        __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(src + (c * 64 + lane) * 16),
                                         (__attribute__((address_space(3))) void*)(dst + c * 64), 16, 0, 0);
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  const int seg = lane / C::SEG, sl = lane % C::SEG;
  const bool lane_ok = seg < np;
  const int sg = seg < PPW ? seg : 0;  // lanes past the group use plane 0's padding
  const int slot = p.slot[wave];
  const int sl0 = slot < 0 ? 0 : slot;
  const bool rn = LG && p.renorm;
  T* w3 = s_flat + sg * HW + (SM_W + 3 * sl0) * C::MS;
  // u * dy (fp32, written after du) over the u and dy maps: [plane][HW] floats
  float* s_udy = reinterpret_cast<float*>(s_flat + SM_U * C::MS);
  float* harr = s_arr + (sg * ND + sl0) * C::ARR;

  // thread i < MV owns 16-byte vector i of every map: plane pl, elements e0 ...
  const bool own = tid < MV;
  const int iv = own ? tid : 0;
  const int vpl = iv / NVM, ve0 = (iv - vpl * NVM) * VE, vr0 = ve0 / S, vc0 = ve0 - vr0 * S;
  const bool vreal = own && vpl < np;
  const float* varr = s_arr + vpl * ND * C::ARR;

  // lam * x into every direction array (the forward reads it there and
  // overwrites it with h)
  if (own) {
    Pack<T, VE> pl_, px;
    pl_.load(s_flat + SM_LAM * C::MS + iv * VE);
    px.load(s_flat + SM_X * C::MS + iv * VE);
    float* a = s_arr + vpl * ND * C::ARR;
#pragma unroll
    for (int q = 0; q < VE; ++q) {
      const int li = staged_aidx<S>(ve0, vr0, vc0, q);
      const float lx = pl_.get(q) * px.get(q);
#pragma unroll
      for (int k = 0; k < ND; ++k) a[k * C::ARR + li] = lx;
    }
  }
  lds_barrier();

  if (slot >= 0) {
    switch (wave) {
      case 0: staged_forward<T, S, false, false, GRP, LG>(w3, harr, sl, lane_ok, p.gstart[0], rn); break;
      case 1: staged_forward<T, S, false, true, GRP, LG>(w3, harr, sl, lane_ok, p.gstart[1], rn); break;
      case 2: staged_forward<T, S, true, false, GRP, LG>(w3, harr, sl, lane_ok, p.gstart[2], rn); break;
      default: staged_forward<T, S, true, true, GRP, LG>(w3, harr, sl, lane_ok, p.gstart[3], rn); break;
    }
  }
  lds_barrier();

  // du = dy * (sum of h over the present directions, in direction order), and
  // u * dy in fp32 for the adjoint, written over the u and dy maps once every
  // thread has read them (zero for planes past the end of the tensor: their
  // lanes must see finite values)
  {
    float ud[VE];
    if (own) {
      Pack<T, VE> pdy, pu;
      pdy.load(s_flat + SM_DY * C::MS + iv * VE);
      pu.load(s_flat + SM_U * C::MS + iv * VE);
      float dd[VE];
#pragma unroll
      for (int q = 0; q < VE; ++q) {
        const int li = staged_aidx<S>(ve0, vr0, vc0, q);
        float sum = varr[li];
#pragma unroll
        for (int k = 1; k < ND; ++k) sum += varr[k * C::ARR + li];
        dd[q] = pdy.get(q) * sum;
        ud[q] = vreal ? pu.get(q) * pdy.get(q) : 0.f;
      }
      if (vreal) stv<VE>((T*)p.du + (g0 + vpl) * HW + ve0, dd);
    }
    lds_barrier();
    if (own) stv<VE>(s_udy + iv * VE, ud);
  }
  lds_barrier();

  if (slot >= 0) {
    switch (wave) {
      case 0: staged_adjoint<T, S, false, false, GRP, LG>(s_udy + sg * HW, w3, harr, sl, lane_ok, p.gstart[0], rn); break;
      case 1: staged_adjoint<T, S, false, true, GRP, LG>(s_udy + sg * HW, w3, harr, sl, lane_ok, p.gstart[1], rn); break;
      case 2: staged_adjoint<T, S, true, false, GRP, LG>(s_udy + sg * HW, w3, harr, sl, lane_ok, p.gstart[2], rn); break;
      default: staged_adjoint<T, S, true, true, GRP, LG>(s_udy + sg * HW, w3, harr, sl, lane_ok, p.gstart[3], rn); break;
    }
    // this direction's three dw maps (written over its w maps by this wave
    // alone) leave at once, while the other waves may still be scanning; the
    // runs are contiguous in LDS and in global memory
    uint4 r[3][NCH];
#pragma unroll
    for (int k = 0; k < 3; ++k)
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        const int v = c * 64 + lane < nv ? c * 64 + lane : nv - 1;
        r[k][c] = reinterpret_cast<const uint4*>(lds4)[(SM_W + 3 * slot + k) * MV + v];
      }
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      T* dst = (T*)p.dw + (int64_t)(3 * slot + k) * p.npc + g0 * HW;  // dw maps: slot-major, packed like w
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        const int v = c * 64 + lane;
        if (v < nv) *reinterpret_cast<uint4*>(dst + v * VE) = r[k][c];
      }
    }
  }
  lds_barrier();

  // dx = lam * gsum and dlam = x * gsum (fixed-order sum of the directions' g)
  if (vreal) {
    Pack<T, VE> pl_, px;
    pl_.load(s_flat + SM_LAM * C::MS + iv * VE);
    px.load(s_flat + SM_X * C::MS + iv * VE);
    float ra[VE], rb[VE];
#pragma unroll
    for (int q = 0; q < VE; ++q) {
      const int li = staged_aidx<S>(ve0, vr0, vc0, q);
      float sum = varr[li];
#pragma unroll
      for (int k = 1; k < ND; ++k) sum += varr[k * C::ARR + li];
      ra[q] = pl_.get(q) * sum;
      rb[q] = px.get(q) * sum;
    }
    const int64_t o = (g0 + vpl) * HW + ve0;
    stv<VE>((T*)p.dx + o, ra);
    stv<VE>((T*)p.dlam + o, rb);
  }
}

template <typename T>
inline bool staged_bwd_size_supported(int H, int W) {
  if (H != W) return false;
  switch (H) {
    case 16: return (StagedCfg<T, 16>::MAPB % 16) == 0;
    case 28: return (StagedCfg<T, 28>::MAPB % 16) == 0;
    case 32: return (StagedCfg<T, 32>::MAPB % 16) == 0;
    default: return false;
  }
}

template <typename T, int S, int ND>
hipError_t launch_staged_bwd_nd(const ResBwdParams& p, hipStream_t st) {
  using C = StagedCfg<T, S>;
  constexpr int lds = C::bytes(C::PPW, ND);
  auto kern = p.logits ? (p.grouped ? staged_bwd_kernel<T, S, ND, true, true> : staged_bwd_kernel<T, S, ND, false, true>)
                       : (p.grouped ? staged_bwd_kernel<T, S, ND, true, false> : staged_bwd_kernel<T, S, ND, false, false>);
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
  }
  const int64_t groups = (p.planes + C::PPW - 1) / C::PPW;
  hipLaunchKernelGGL(kern, dim3((unsigned)groups), dim3(256), lds, st, p);
  return hipGetLastError();
}

template <typename T, int S>
hipError_t launch_staged_bwd(const ResBwdParams& p, hipStream_t st) {
  switch (p.nd) {
    case 1: return launch_staged_bwd_nd<T, S, 1>(p, st);
    case 2: return launch_staged_bwd_nd<T, S, 2>(p, st);
    case 3: return launch_staged_bwd_nd<T, S, 3>(p, st);
    default: return launch_staged_bwd_nd<T, S, 4>(p, st);
  }
}

template <typename T>
hipError_t launch_staged_bwd_size(const ResBwdParams& p, int S, hipStream_t st) {
  switch (S) {
    case 16: return launch_staged_bwd<T, 16>(p, st);
    case 28: return launch_staged_bwd<T, 28>(p, st);
    default: return launch_staged_bwd<T, 32>(p, st);
  }
}

// Backward dispatch of the resident family: the staged kernel where it applies,
// else the per-wave resident kernel.
template <typename T>
hipError_t resident_bwd_t(const ResidentBwdArgs& a) {
  ResBwdParams p;
  p.dy = a.dy; p.x = a.x; p.lam = a.lam; p.w = a.w; p.u = a.u;
  p.dx = a.dx; p.dw = a.dw; p.dlam = a.dlam; p.du = a.du;
  p.planes = a.planes;
  p.npc = (int64_t)a.planes * a.H * a.W;
  int n = 0;
  for (int d = 0; d < 4; ++d) p.slot[d] = (a.mask >> d) & 1 ? n++ : -1;
  p.nd = n;
  p.logits = a.logits;
  p.renorm = a.renorm;
  p.lam_pd = a.lam_pd; p.u_pd = a.u_pd; p.y_pd = a.y_pd;
  const bool pd = a.lam_pd || a.u_pd || a.y_pd;
  const int gh = (a.group_h > 0 && a.group_h < a.H) ? a.group_h : a.H;
  const int gw = (a.group_w > 0 && a.group_w < a.W) ? a.group_w : a.W;
  p.grouped = gh < a.H || gw < a.W;
  for (int d = 0; d < 4; ++d) {
    const bool hz = d >= 2, rev = d & 1;
    const int L = hz ? a.W : a.H, G = hz ? gw : gh;
    p.gstart[d] = 0;
    for (int l = 0; l < L && l < 64; ++l)
      if (rev ? ((l + 1) % G == 0 || l == L - 1) : (l % G == 0)) p.gstart[d] |= 1ull << l;
  }
  auto al16 = [](const void* q) { return ((uintptr_t)q % 16) == 0; };
  p.vec = al16(a.dy) && al16(a.x) && al16(a.lam) && al16(a.u) && al16(a.dx) && al16(a.dlam) && al16(a.du);
  const bool ok = al16(a.x) && al16(a.lam) && al16(a.w) && al16(a.u) && al16(a.dy) && al16(a.dw);
  if (!ok || !resident_bwd_size_supported(a.H, a.W)) return hipErrorInvalidValue;
  hipStream_t st = (hipStream_t)a.stream;
  if (a.H == 128) {
    // persistent 128 x 128 kernel: every pointer 16-byte aligned, merged maps
    if (!p.vec || pd) return hipErrorInvalidValue;
    WideBwdParams q;
    q.dy = a.dy; q.x = a.x; q.lam = a.lam; q.w = a.w; q.u = a.u;
    q.dx = a.dx; q.dw = a.dw; q.dlam = a.dlam; q.du = a.du;
    q.npc = p.npc; q.planes = a.planes;
    q.logits = a.logits; q.renorm = a.renorm;
    for (int d = 0; d < 4; ++d) q.slot[d] = p.slot[d];
    const int gh = (a.group_h > 0 && a.group_h < 128) ? a.group_h : 128;
    const int gw = (a.group_w > 0 && a.group_w < 128) ? a.group_w : 128;
    for (int d = 0; d < 4; ++d) {
      const bool rev = d & 1;
      const int G = d >= 2 ? gw : gh;
      q.gstart[d][0] = q.gstart[d][1] = 0;
      for (int l = 0; l < 128; ++l)
        if (rev ? ((l + 1) % G == 0 || l == 127) : (l % G == 0)) q.gstart[d][l >> 6] |= 1ull << (l & 63);
    }
    return sizeof(T) == 4 ? wide_bwd_launch_f32(q, st) : wide_bwd_launch_bf16(q, st);
  }
  if (a.use_staged && p.vec && !pd && staged_bwd_size_supported<T>(a.H, a.W))
    return launch_staged_bwd_size<T>(p, a.H, st);
  switch (a.H) {
    case 16: return launch_resident_bwd<T, 16>(p, st);
    case 28: return launch_resident_bwd<T, 28>(p, st);
    case 32: return launch_resident_bwd<T, 32>(p, st);
    case 56: return launch_resident_bwd<T, 56>(p, st);
    default: return launch_resident_bwd<T, 64>(p, st);
  }
}

}  // namespace gspn
