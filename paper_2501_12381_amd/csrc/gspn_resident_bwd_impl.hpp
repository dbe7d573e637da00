// Resident backward kernel for square S x S planes (S <= 64): the whole
// adjoint (Alg. 2, exact adjoint of Eq. 1-2 for the loss <dy, y>) of a group
// of planes in one launch, reading every input once from HBM and writing
// every gradient once.
//
// A workgroup has four waves, one per scan direction (absent directions idle).
//   phase F: each wave recomputes its direction's forward state h_d and keeps
//            it in its own fp32 LDS array (no sharing, no ordering issues);
//   du:      du = dy * (h_T2B + h_B2T + h_L2R + h_R2L), summed in that fixed
//            order by all waves;
//   phase A: each wave runs the reverse (adjoint) scan of its direction:
//              g[line] = u*dy + sum_k w_k[next] * g[next] (transposed stencil),
//            emits dw_k[line][p] = g[line][p] * h[prev][p + k - 1], and stores
//            g[line] over h[line] in its LDS array (h[line] was last needed as
//            the previous-line state of the line processed just before);
//   dx, dlam: gsum = g_T2B + g_B2T + g_L2R + g_R2L (fixed order),
//            dx = lam * gsum, dlam = x * gsum.
// Every sum has a fixed order, so results are bitwise reproducible.
//
// Plane packing, padding lanes, register rings and row-segment access of the
// horizontal directions follow the forward kernel.
#pragma once

#include "gspn_device.hpp"
#include "gspn_launch.hpp"
#include "gspn_resident_impl.hpp"

namespace gspn {

template <typename T, int S>
struct BwdCfg {
  static constexpr int NP = 1;                                    // S <= 64
  static constexpr int SEG = S <= 15 ? 16 : (S <= 31 ? 32 : 64);
  static constexpr int PPW = 64 / SEG;
  static constexpr int P = S + 1;
  static constexpr int ROWS = S + 1;
  static constexpr int ARR = ROWS * P;                            // floats per direction array
  static constexpr int VLH = (S % (16 / (int)sizeof(T)) == 0) ? 16 / (int)sizeof(T)
                           : (S % (8 / (int)sizeof(T)) == 0 ? 8 / (int)sizeof(T) : 4 / (int)sizeof(T));
  static constexpr int RV = S % 8 == 0 ? 8 : 7;
  static constexpr int RH = 6;
  static constexpr bool ALL_VALID = (S == SEG);
  static constexpr int LDS_BYTES = PPW * 4 * ARR * 4;
  // vector width of the elementwise passes (16- or 8-byte vectors, else scalars)
  static constexpr int VE = (S % (16 / (int)sizeof(T)) == 0) ? 16 / (int)sizeof(T)
                          : (S % (8 / (int)sizeof(T)) == 0 ? 8 / (int)sizeof(T) : 1);
  static_assert(S <= 64 && S % 2 == 0, "resident backward takes even S <= 64");
};

struct ResBwdParams {
  const void* dy;
  const void* x;
  const void* lam;
  const void* w;
  const void* u;
  void* dx;
  void* dw;
  void* dlam;
  void* du;
  int64_t npc;
  int64_t planes;
  int slot[4];
  int nd;   // directions present
  int vec;  // 16-byte vectors legal for the elementwise passes
  int grouped;          // local GSPN: some direction restarts inside the plane
  // per direction (T2B, B2T, L2R, R2L): bit l set when line l starts a group
  // in that direction's scan order (lines <= 64)
  uint64_t gstart[4];
  int logits, renorm;  // w holds Eq. 6 logits (dw: their gradient); renorm: on-line neighbours only
  // per-direction maps (per-wave kernel only): lam, u, y (and dlam, du, dy)
  // are (n, B, C, H, W) when set
  int lam_pd, u_pd, y_pd;
};

// Input ring shared by phase F (x, lam, w0, w1, w2) and phase A (u, dy, w0, w1, w2).
template <typename T, int S, bool HZ, bool REV>
struct Ring {
  using C = BwdCfg<T, S>;
  static constexpr int TL = HZ ? C::VLH : 1;
  static constexpr int R = HZ ? C::RH : C::RV;
  static constexpr int NT = S / TL;
  typedef Pack<T, TL> PK;
  PK slot[R][5];
  int eoff;  // element offset of the lane's position (row start for HZ)

  __device__ __forceinline__ static int tile_line(int ti) { return REV ? (NT - 1 - ti) * TL : ti * TL; }
  __device__ __forceinline__ void load(const T* const (&pb)[5], int k, int ti) {
    const int l = tile_line(ti < NT ? ti : NT - 1);
#pragma unroll
    for (int m = 0; m < 5; ++m) slot[k][m].load(pb[m] + eoff + (HZ ? l : l * S));
  }
};

// Forward recompute of one direction into its LDS array: h[line][pos].
// LG: the weight maps hold Eq. 6 logits, normalised as they are unpacked.
template <typename T, int S, bool HZ, bool REV, bool LG>
__device__ __forceinline__ void bwd_forward(const T* const (&pb)[5], float* __restrict__ harr, int sl,
                                            uint64_t gst, bool renorm) {
  using C = BwdCfg<T, S>;
  using RG = Ring<T, S, HZ, REV>;
  constexpr int TL = RG::TL, R = RG::R, NT = RG::NT;
  const bool valid = C::ALL_VALID || sl < S;
  const int pos = valid ? sl : 0;
  RG ring;
  ring.eoff = HZ ? pos * S : pos;
  const int aoff = valid ? (HZ ? sl * C::P : sl) : (HZ ? S * C::P : S);
#pragma unroll
  for (int k = 0; k < R; ++k) ring.load(pb, k, k);
  float hp[1] = {0.f};
  const bool vv[1] = {valid};
#pragma unroll
  for (int ti = 0; ti < NT; ++ti) {
    const int k = ti % R;
    float v[5][TL];
#pragma unroll
    for (int m = 0; m < 5; ++m)
#pragma unroll
      for (int e = 0; e < TL; ++e) v[m][e] = ring.slot[k][m].get(e);
    ring.load(pb, k, ti + R);
#pragma unroll
    for (int ee = 0; ee < TL; ++ee) {
      const int e = REV ? TL - 1 - ee : ee;
      const int line = RG::tile_line(ti) + e;
      float xv[1] = {v[0][e]}, lv[1] = {v[1][e]}, a[1] = {v[2][e]}, b[1] = {v[3][e]}, c[1] = {v[4][e]};
      if ((gst >> line) & 1) hp[0] = 0.f;  // local GSPN: a group starts here
      norm_weights<LG, 1>(a, b, c, sl, S, renorm);
      line_step<1>(xv, lv, a, b, c, vv, hp);
      harr[aoff + (HZ ? line : line * C::P)] = hp[0];
    }
  }
}

// Adjoint scan of one direction: reads h from harr, overwrites it with g,
// writes the direction's three dw maps (LG: the gradients of the logits,
// through Eq. 6's Jacobian).
template <typename T, int S, bool HZ, bool REV, bool LG>
__device__ __forceinline__ void bwd_adjoint(const T* const (&pb)[5], T* const (&dwp)[3],
                                            float* __restrict__ harr, int sl, uint64_t gst, bool renorm) {
  using C = BwdCfg<T, S>;
  // the adjoint visits lines in the opposite order of the forward scan
  using RG = Ring<T, S, HZ, !REV>;
  constexpr int TL = RG::TL, R = RG::R, NT = RG::NT;
  const bool valid = C::ALL_VALID || sl < S;
  const int pos = valid ? sl : 0;
  RG ring;
  ring.eoff = HZ ? pos * S : pos;
  const int aoff = valid ? (HZ ? sl * C::P : sl) : (HZ ? S * C::P : S);
#pragma unroll
  for (int k = 0; k < R; ++k) ring.load(pb, k, k);
  // g and weights of the line after the current one (in forward scan order)
  float gn = 0.f, wn0 = 0.f, wn1 = 0.f, wn2 = 0.f;
  // horizontal directions buffer dw for TL lines and store them as row segments
  float dwb[3][TL];
#pragma unroll
  for (int ti = 0; ti < NT; ++ti) {
    const int k = ti % R;
    float v[5][TL];
#pragma unroll
    for (int m = 0; m < 5; ++m)
#pragma unroll
      for (int e = 0; e < TL; ++e) v[m][e] = ring.slot[k][m].get(e);
    ring.load(pb, k, ti + R);
#pragma unroll
    for (int ee = 0; ee < TL; ++ee) {
      const int e = !REV ? TL - 1 - ee : ee;  // adjoint order inside the tile
      const int line = RG::tile_line(ti) + e;
      // previous line in forward order (its h is the state this line read)
      const int prev = REV ? line + 1 : line - 1;
      // a line that starts a group read a zero state, and the line after it in
      // forward order, if it starts a group, took nothing from this one
      const bool has_prev = (REV ? line + 1 < S : line > 0) && !((gst >> line) & 1);
      const int succ = REV ? line - 1 : line + 1;
      if (succ >= 0 && succ < S && ((gst >> succ) & 1)) gn = 0.f;
      const float a0 = wn0 * gn, a1 = wn1 * gn, a2 = wn2 * gn;
      const float a0n = from_next_lane(a0);  // neighbour p+1 received with k = 0
      const float a2p = from_prev_lane(a2);  // neighbour p-1 received with k = 2
      float g = v[0][e] * v[1][e] + a1 + a0n + a2p;  // u * dy + transposed stencil
      g = valid ? g : 0.f;
      const float hpv = has_prev ? harr[aoff + (HZ ? prev : prev * C::P)] : 0.f;
      const float hl = from_prev_lane(hpv);
      const float hr = from_next_lane(hpv);
      harr[aoff + (HZ ? line : line * C::P)] = g;
      float d0 = g * hl, d1 = g * hpv, d2 = g * hr;
      float c0 = v[2][e], c1 = v[3][e], c2 = v[4][e];
      if constexpr (LG) {
        const Norm3 r = normalize3(c0, c1, c2, sl == 0, sl == S - 1, renorm);
        norm3_vjp(r, d0, d1, d2);
        c0 = r.w[0];
        c1 = r.w[1];
        c2 = r.w[2];
      }
      if constexpr (HZ) {
        dwb[0][e] = d0; dwb[1][e] = d1; dwb[2][e] = d2;
      } else {
        if (valid) {
          const int64_t off = (int64_t)line * S + pos;
          dwp[0][off] = from_f<T>(d0);
          dwp[1][off] = from_f<T>(d1);
          dwp[2][off] = from_f<T>(d2);
        }
      }
      gn = g;
      wn0 = valid ? c0 : 0.f;  // padding lanes hold clamped (foreign) weights
      wn1 = valid ? c1 : 0.f;
      wn2 = valid ? c2 : 0.f;
    }
    if constexpr (HZ) {
      if (valid) {
        const int64_t off = (int64_t)pos * S + RG::tile_line(ti);
        stv<TL>(dwp[0] + off, dwb[0]);
        stv<TL>(dwp[1] + off, dwb[1]);
        stv<TL>(dwp[2] + off, dwb[2]);
      }
    }
  }
}

// out = a * (s0 + s1 + s2 + s3) over one plane, the sums read from the four
// direction arrays (absent directions are zero-filled), in that order.
template <typename T, int S, int VE>
__device__ __forceinline__ void bwd_combine(const T* __restrict__ a0, T* __restrict__ o0,
                                            const T* __restrict__ a1, T* __restrict__ o1,
                                            const float* __restrict__ arr, int tid) {
  using C = BwdCfg<T, S>;
  constexpr int PR = S / VE;
  for (int e = tid; e < S * PR; e += 256) {
    const int r = e / PR, c = (e - r * PR) * VE;
    Pack<T, VE> va, vb;
    va.load(a0 + r * S + c);
    if (a1) vb.load(a1 + r * S + c);
    float oa[VE], ob[VE];
#pragma unroll
    for (int q = 0; q < VE; ++q) {
      const int li = r * C::P + c + q;
      const float sum = ((arr[li] + arr[C::ARR + li]) + arr[2 * C::ARR + li]) + arr[3 * C::ARR + li];
      oa[q] = va.get(q) * sum;
      if (a1) ob[q] = vb.get(q) * sum;
    }
    stv<VE>(o0 + r * S + c, oa);
    if (a1) stv<VE>(o1 + r * S + c, ob);
  }
}

// Per-direction maps: du (or du_d) = sum over the present directions, in
// order, of dy (or dy_d) * h_d, from the direction arrays of one plane.
template <typename T, int S, int VE>
__device__ __forceinline__ void bwd_du_pd(const ResBwdParams& p, int64_t pofs, const float* __restrict__ arr,
                                          int tid) {
  using C = BwdCfg<T, S>;
  constexpr int PR = S / VE;
  for (int e = tid; e < S * PR; e += 256) {
    const int r = e / PR, c = (e - r * PR) * VE;
    const int64_t o = pofs + r * S + c;
    float acc[VE];
#pragma unroll
    for (int q = 0; q < VE; ++q) acc[q] = 0.f;
    for (int d = 0; d < 4; ++d) {
      const int s = p.slot[d];
      if (s < 0) continue;
      Pack<T, VE> vd;
      vd.load((const T*)p.dy + (p.y_pd ? s * p.npc : 0) + o);
      float t[VE];
#pragma unroll
      for (int q = 0; q < VE; ++q) t[q] = vd.get(q) * arr[d * C::ARR + r * C::P + c + q];
      if (p.u_pd) {
        stv<VE>((T*)p.du + s * p.npc + o, t);
      } else {
#pragma unroll
        for (int q = 0; q < VE; ++q) acc[q] += t[q];
      }
    }
    if (!p.u_pd) stv<VE>((T*)p.du + o, acc);
  }
}

// Per-direction lam: dx = sum over the present directions of lam_d g_d, and
// dlam_d = x g_d.
template <typename T, int S, int VE>
__device__ __forceinline__ void bwd_dx_pd(const ResBwdParams& p, int64_t pofs, const float* __restrict__ arr,
                                          int tid) {
  using C = BwdCfg<T, S>;
  constexpr int PR = S / VE;
  for (int e = tid; e < S * PR; e += 256) {
    const int r = e / PR, c = (e - r * PR) * VE;
    const int64_t o = pofs + r * S + c;
    Pack<T, VE> vx;
    vx.load((const T*)p.x + o);
    float acc[VE];
#pragma unroll
    for (int q = 0; q < VE; ++q) acc[q] = 0.f;
    for (int d = 0; d < 4; ++d) {
      const int s = p.slot[d];
      if (s < 0) continue;
      Pack<T, VE> vl;
      vl.load((const T*)p.lam + s * p.npc + o);
      float t[VE];
#pragma unroll
      for (int q = 0; q < VE; ++q) {
        const float g = arr[d * C::ARR + r * C::P + c + q];
        acc[q] += vl.get(q) * g;
        t[q] = vx.get(q) * g;
      }
      stv<VE>((T*)p.dlam + s * p.npc + o, t);
    }
    stv<VE>((T*)p.dx + o, acc);
  }
}

template <typename T, int S, bool LG>
__global__ void __launch_bounds__(256, 2) resident_bwd_kernel(ResBwdParams p) {
  using C = BwdCfg<T, S>;
  constexpr int PPW = C::PPW;
  constexpr int HW = S * S;
  extern __shared__ float lds[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;  // wave = direction
  const int64_t g0 = (int64_t)blockIdx.x * PPW;
  const int seg = lane / C::SEG, sl = lane % C::SEG;
  const int64_t plane = (g0 + seg < p.planes) ? g0 + seg : p.planes - 1;
  // per plane group: four direction arrays per plane, plane-major
  float* arr_of_plane = lds + seg * 4 * C::ARR;
  float* harr = arr_of_plane + wave * C::ARR;

  for (int e = tid; e < PPW * 4 * C::ARR; e += 256) lds[e] = 0.f;
  __syncthreads();

  const int slot = p.slot[wave];
  const T* w0 = slot >= 0 ? (const T*)p.w + (int64_t)slot * 3 * p.npc + plane * HW : nullptr;
  const int64_t pofs = plane * HW;
  const bool rn = LG && p.renorm;
  if (slot >= 0) {
    const T* pb[5] = {(const T*)p.x + pofs, (const T*)p.lam + (p.lam_pd ? slot * p.npc : 0) + pofs, w0,
                      w0 + p.npc, w0 + 2 * p.npc};
    switch (wave) {
      case 0: bwd_forward<T, S, false, false, LG>(pb, harr, sl, p.gstart[0], rn); break;
      case 1: bwd_forward<T, S, false, true, LG>(pb, harr, sl, p.gstart[1], rn); break;
      case 2: bwd_forward<T, S, true, false, LG>(pb, harr, sl, p.gstart[2], rn); break;
      default: bwd_forward<T, S, true, true, LG>(pb, harr, sl, p.gstart[3], rn); break;
    }
  }
  __syncthreads();

  // du = dy * sum_d h_d (per-direction maps: the sum of dy_d h_d, or du_d)
  for (int pl = 0; pl < PPW; ++pl) {
    const int64_t pi = g0 + pl;
    if (pi >= p.planes) break;
    const float* arr = lds + pl * 4 * C::ARR;
    if (p.u_pd || p.y_pd) {
      if (p.vec) bwd_du_pd<T, S, C::VE>(p, pi * HW, arr, tid);
      else bwd_du_pd<T, S, 1>(p, pi * HW, arr, tid);
      continue;
    }
    const T* dyb = (const T*)p.dy + pi * HW;
    T* dub = (T*)p.du + pi * HW;
    if (p.vec) bwd_combine<T, S, C::VE>(dyb, dub, nullptr, nullptr, arr, tid);
    else bwd_combine<T, S, 1>(dyb, dub, nullptr, nullptr, arr, tid);
  }
  __syncthreads();

  if (slot >= 0) {
    const T* pb[5] = {(const T*)p.u + (p.u_pd ? slot * p.npc : 0) + pofs,
                      (const T*)p.dy + (p.y_pd ? slot * p.npc : 0) + pofs, w0, w0 + p.npc, w0 + 2 * p.npc};
    T* dw0 = (T*)p.dw + (int64_t)slot * 3 * p.npc + pofs;
    T* const dwp[3] = {dw0, dw0 + p.npc, dw0 + 2 * p.npc};
    switch (wave) {
      case 0: bwd_adjoint<T, S, false, false, LG>(pb, dwp, harr, sl, p.gstart[0], rn); break;
      case 1: bwd_adjoint<T, S, false, true, LG>(pb, dwp, harr, sl, p.gstart[1], rn); break;
      case 2: bwd_adjoint<T, S, true, false, LG>(pb, dwp, harr, sl, p.gstart[2], rn); break;
      default: bwd_adjoint<T, S, true, true, LG>(pb, dwp, harr, sl, p.gstart[3], rn); break;
    }
  }
  // an absent direction's array stays zero from the initial fill
  __syncthreads();

  // dx = lam * gsum, dlam = x * gsum
  for (int pl = 0; pl < PPW; ++pl) {
    const int64_t pi = g0 + pl;
    if (pi >= p.planes) break;
    const float* arr = lds + pl * 4 * C::ARR;
    const int64_t o = pi * HW;
    if (p.lam_pd) {
      if (p.vec) bwd_dx_pd<T, S, C::VE>(p, o, arr, tid);
      else bwd_dx_pd<T, S, 1>(p, o, arr, tid);
      continue;
    }
    if (p.vec)
      bwd_combine<T, S, C::VE>(
          (const T*)p.lam + o, (T*)p.dx + o, (const T*)p.x + o, (T*)p.dlam + o, arr, tid);
    else
      bwd_combine<T, S, 1>((const T*)p.lam + o, (T*)p.dx + o, (const T*)p.x + o, (T*)p.dlam + o, arr, tid);
  }
}

inline bool resident_bwd_size_supported(int H, int W) {
  return H == W && (H == 16 || H == 28 || H == 32 || H == 56 || H == 64 || H == 128);
}

template <typename T, int S>
hipError_t launch_resident_bwd(const ResBwdParams& p, hipStream_t st) {
  using C = BwdCfg<T, S>;
  auto kern = p.logits ? resident_bwd_kernel<T, S, true> : resident_bwd_kernel<T, S, false>;
  if (C::LDS_BYTES > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       C::LDS_BYTES);
    if (e != hipSuccess) return e;
  }
  const int64_t groups = (p.planes + C::PPW - 1) / C::PPW;
  hipLaunchKernelGGL(kern, dim3((unsigned)groups), dim3(256), C::LDS_BYTES, st, p);
  return hipGetLastError();
}

}  // namespace gspn
