// Size-specialised resident forward kernel for square S x S planes (S <= 64).
//
// Same decomposition as the generic resident kernel (one workgroup of two
// waves per group of planes; phase V = top-to-bottom and bottom-to-top,
// phase H = left-to-right and right-to-left; sum_d h_d accumulated in fp32 in
// LDS with the midpoint barriers that fix the addition order), but with the
// plane size a compile-time constant:
//   * every global and LDS address of a line is a base register plus an
//     immediate offset, so a line step carries no address arithmetic;
//   * the phases are fully unrolled (the middle barrier and the padding masks
//     resolve at compile time);
//   * inputs are prefetched through a register ring of R tiles (a tile is one
//     row for vertical scans, a row segment of THZ columns for horizontal ones);
//   * lam * x is formed once per element and kept in LDS next to the
//     accumulator, so x and lam are read from HBM once, not once per direction;
//   * LDS values are read G lines ahead of their use, never across the middle
//     barrier, so LDS latency stays off the critical path.
#pragma once

#include "gspn_device.hpp"
#include "gspn_launch.hpp"
#include "gspn_resident_impl.hpp"

namespace gspn {

template <typename T, int S>
struct FixedCfg {
  static constexpr int SEG = S <= 15 ? 16 : (S <= 31 ? 32 : 64); // lanes per plane
  static constexpr int PPW = 64 / SEG;                           // planes per wave
  static constexpr int P = S + 1;                                // LDS pitch (odd)
  static constexpr int ROWS = S + 1;                             // + padding row
  static constexpr int ACC = ROWS * P;                           // floats per plane array
  static constexpr int MID = S / 2;
  // horizontal vector: largest of 16/8/4 bytes whose element count divides S
  static constexpr int VLH = (S % (16 / (int)sizeof(T)) == 0) ? 16 / (int)sizeof(T)
                           : (S % (8 / (int)sizeof(T)) == 0 ? 8 / (int)sizeof(T) : 4 / (int)sizeof(T));
  static constexpr int THZ = VLH;                                 // horizontal tile: lines per row segment
  static constexpr int RV = S % 8 == 0 ? 8 : 7;                   // vertical ring (lines)
  static constexpr int RH = 6;                                    // horizontal ring (tiles)
  static constexpr int G = 4;                                     // LDS lookahead
  static constexpr bool ALL_VALID = (S == SEG);
  // epilogue vectors of u and y: the widest of 16/8/4 bytes whose element
  // count divides S, used when u and y are aligned for them (ULVL: the vec_y
  // level this needs); the group's vectors spread over the 128 threads
  static constexpr int VEU = VLH;
  static constexpr int ULVL = VEU * (int)sizeof(T) == 16 ? 2 : (VEU * (int)sizeof(T) == 8 ? 1 : 3);  // 3: never
  static constexpr int NEU = S * (S / VEU);             // vectors per plane
  static constexpr int KU = (PPW * NEU + 127) / 128;    // vectors per thread
  static constexpr int LDS_BYTES = 2 * PPW * ACC * 4;             // accumulators, then lam * x
  static_assert(S % 2 == 0 && S <= 64, "fixed kernel takes even sizes up to 64");
};

// One direction's scan over a phase.  HZ: lines are columns.  REV: lines are
// visited from S-1 down to 0.  pbase[m]: plane base of map m (x, lam, w0..w2).
// PRESENT: the direction is in the mask (a vertical wave whose direction is
// absent still does its first-half duties below).
//
// lam * x is formed once per element: in phase V each wave reads x and lam
// for the lines it reaches first, stores lam * x in LDS next to the
// accumulator, and stores its h there (the first arrival: no zeroing, no
// read).  After the middle barrier, and in phase H, lam * x and the
// accumulator come from LDS, read G lines ahead of their use (never across the
// middle barrier), so each input is read from HBM once.
// GRP: local GSPN; bit l of gst is set when line l starts a group (the state
// restarts from zero there).  LG: the weight maps hold Eq. 6 logits,
// normalised as they are unpacked (renorm: over the on-line neighbours).
template <typename T, int S, bool HZ, bool REV, bool PRESENT, bool GRP, bool LG>
__device__ __forceinline__ void fixed_phase(const T* const (&pbase)[5], float* __restrict__ acc,
                                            float* __restrict__ lxa, int sl, uint64_t gst, bool renorm) {
  using C = FixedCfg<T, S>;
  constexpr int TL = HZ ? C::THZ : 1;   // lines per tile
  constexpr int R = HZ ? C::RH : C::RV; // tiles in flight
  constexpr int NT = S / TL;            // tiles per phase
  constexpr int MID = C::MID, G = C::G;
  static_assert(S % TL == 0, "tile must divide the line count");
  typedef Pack<T, TL> PK;

  const bool valid = C::ALL_VALID || sl < S;
  const int pos = valid ? sl : 0;                  // padding lanes read position 0 (masked below)
  const int eoff = HZ ? pos * S : pos;
  // LDS offset of (line 0, the lane's position); padding lanes use the padding row/column
  const int aoff = valid ? (HZ ? sl * C::P : sl) : (HZ ? S * C::P : S);

  auto tile_line = [](int ti) { return REV ? (NT - 1 - ti) * TL : ti * TL; };
  auto line_of = [](int s) { return REV ? S - 1 - s : s; };
  auto lds_line = [](int line) { return HZ ? line : line * C::P; };

  // ring slots: x, lam (vertical first half only), w0, w1, w2
  PK ring[R][5];
  auto load_tile = [&](PK (&slot)[5], int ti) __attribute__((always_inline)) {
    if (ti >= NT) return;
    const int l = tile_line(ti);
    if (!HZ && ti < MID) {
      slot[0].load(pbase[0] + eoff + l * S);
      slot[1].load(pbase[1] + eoff + l * S);
    }
    if (PRESENT) {
#pragma unroll
      for (int m = 2; m < 5; ++m) slot[m].load(pbase[m] + eoff + (HZ ? l : l * S));
    }
  };
#pragma unroll
  for (int k = 0; k < R; ++k) load_tile(ring[k], k);

  float hp = 0.f;
  float lv[G], av[G];  // lookahead: lam * x and the accumulator, slot s % G
  auto lds_read = [&](int s) __attribute__((always_inline)) {
    const int o = aoff + lds_line(line_of(s));
    lv[s % G] = lxa[o];
    av[s % G] = acc[o];
  };
  if (HZ) {
#pragma unroll
    for (int g = 0; g < G; ++g) lds_read(g);
  }

#pragma unroll
  for (int k = 0; k < NT; ++k) {
    const int slot = k % R;
    // vertical tiles are one line: unpack and refill the slot at once; horizontal
    // tiles are unpacked line by line and the slot is refilled after its last line
    float v1[5];
    if constexpr (!HZ) {
#pragma unroll
      for (int m = 0; m < 5; ++m) v1[m] = ring[slot][m].get(0);
      load_tile(ring[slot], k + R);
    }
#pragma unroll
    for (int ee = 0; ee < TL; ++ee) {
      const int e = REV ? TL - 1 - ee : ee;  // memory order inside the tile
      const int s = k * TL + ee;             // step inside the phase
      if (s == MID) {
        lds_barrier();  // the other wave's first half is done
        if (!HZ && !PRESENT) return;
#pragma unroll
        for (int g = 0; g < G; ++g)
          if (s + g < S) lds_read(s + g);
      }
      const int o = aoff + lds_line(line_of(s));
      float lx, a = 0.f, b = 0.f, c = 0.f;
      if (!HZ && s < MID) {
        lx = v1[1] * v1[0];
        lxa[o] = lx;
      } else {
        lx = lv[s % G];
      }
      if (PRESENT) {
        a = HZ ? ring[slot][2].get(e) : v1[2];
        b = HZ ? ring[slot][3].get(e) : v1[3];
        c = HZ ? ring[slot][4].get(e) : v1[4];
        if constexpr (LG) {
          const Norm3 r = normalize3(a, b, c, sl == 0, sl == S - 1, renorm);
          a = r.w[0];
          b = r.w[1];
          c = r.w[2];
        }
        if (GRP && ((gst >> line_of(s)) & 1)) hp = 0.f;
        const float hl = from_prev_lane(hp), hr = from_next_lane(hp);
        float v = fmaf(a, hl, lx);
        v = fmaf(b, hp, v);
        v = fmaf(c, hr, v);
        hp = valid ? v : 0.f;
      }
      if (!HZ && s < MID) {
        acc[o] = PRESENT ? hp : 0.f;  // first arrival at this line
      } else {
        acc[o] = av[s % G] + hp;
        const int sn = s + G;
        if (sn < S && !(s < MID && sn >= MID)) lds_read(sn);
      }
    }
    if constexpr (HZ) load_tile(ring[slot], k + R);
  }
}

template <typename T, int S, bool GRP, bool LG>
__global__ void __launch_bounds__(128, (FixedCfg<T, S>::SEG < 64 ? 4 : 2))
fixed_fwd_kernel(ResFwdParams p) {
  using C = FixedCfg<T, S>;
  constexpr int PPW = C::PPW;
  constexpr int HW = S * S;
  extern __shared__ float lds[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t g0 = (int64_t)blockIdx.x * PPW;
  const int seg = lane / C::SEG, sl = lane % C::SEG;
  const int64_t plane = (g0 + seg < p.planes) ? g0 + seg : p.planes - 1;
  float* acc = lds + seg * C::ACC;
  float* lxa = lds + (PPW + seg) * C::ACC;
  const bool rn = LG && p.renorm;

  // phase V: wave 0 top-to-bottom, wave 1 bottom-to-top
  {
    const int slot = p.slot[wave];
    const T* w0 = (const T*)p.w + (int64_t)(slot < 0 ? 0 : slot) * 3 * p.npc + plane * HW;
    const T* pb[5] = {(const T*)p.x + plane * HW, (const T*)p.lam + plane * HW, w0, w0 + p.npc, w0 + 2 * p.npc};
    const uint64_t gst = p.gstart[wave][0];
    if (wave == 0) {
      if (slot >= 0) fixed_phase<T, S, false, false, true, GRP, LG>(pb, acc, lxa, sl, gst, rn);
      else fixed_phase<T, S, false, false, false, GRP, LG>(pb, acc, lxa, sl, gst, rn);
    } else {
      if (slot >= 0) fixed_phase<T, S, false, true, true, GRP, LG>(pb, acc, lxa, sl, gst, rn);
      else fixed_phase<T, S, false, true, false, GRP, LG>(pb, acc, lxa, sl, gst, rn);
    }
  }
  __syncthreads();
  // u of every plane of the group for the epilogue, requested now so that its
  // latency passes under phase H (planes past the end repeat the last one)
  constexpr int VEU = C::VEU, NEU = C::NEU, KU = C::KU;
  const bool uvec = p.vec_y >= C::ULVL;
  Pack<T, VEU> uv[KU];
  auto u_elem = [&](int k, int64_t& pi, int& off) __attribute__((always_inline)) {
    int e = tid + k * 128;
    e = e < PPW * NEU ? e : PPW * NEU - 1;
    const int pl = e / NEU, r = (e - pl * NEU) / (S / VEU), c = (e - pl * NEU - r * (S / VEU)) * VEU;
    pi = g0 + pl < p.planes ? g0 + pl : p.planes - 1;
    off = r * S + c;
  };
  if (uvec) {
#pragma unroll
    for (int k = 0; k < KU; ++k) {
      int64_t pi;
      int off;
      u_elem(k, pi, off);
      uv[k].load((const T*)p.u + pi * HW + off);
    }
  }
  // phase H: wave 0 left-to-right, wave 1 right-to-left
  {
    const int slot = p.slot[2 + wave];
    if (slot < 0) {
      lds_barrier();  // keep the middle barrier of the phase in step
    } else {
      const T* w0 = (const T*)p.w + (int64_t)slot * 3 * p.npc + plane * HW;
      const T* pb[5] = {(const T*)p.x + plane * HW, (const T*)p.lam + plane * HW, w0, w0 + p.npc,
                        w0 + 2 * p.npc};
      const uint64_t gst = p.gstart[2 + wave][0];
      if (wave == 0) fixed_phase<T, S, true, false, true, GRP, LG>(pb, acc, lxa, sl, gst, rn);
      else fixed_phase<T, S, true, true, true, GRP, LG>(pb, acc, lxa, sl, gst, rn);
    }
  }
  __syncthreads();

  if (uvec) {
    // y = u * acc: the LDS reads of all the thread's vectors first, then the stores
    float yv[KU][VEU];
#pragma unroll
    for (int k = 0; k < KU; ++k) {
      int64_t pi;
      int off;
      u_elem(k, pi, off);
      const int e = tid + k * 128 < PPW * NEU ? tid + k * 128 : PPW * NEU - 1;
      const int pl = e / NEU;
      const float* ac = lds + pl * C::ACC + (off / S) * C::P + off % S;
#pragma unroll
      for (int q = 0; q < VEU; ++q) yv[k][q] = ac[q];
    }
#pragma unroll
    for (int k = 0; k < KU; ++k) {
      int64_t pi;
      int off;
      u_elem(k, pi, off);
      const int e = tid + k * 128;
      if (e < PPW * NEU && g0 + e / NEU < p.planes) {
#pragma unroll
        for (int q = 0; q < VEU; ++q) yv[k][q] *= uv[k].get(q);
        stv<VEU>((T*)p.y + pi * HW + off, yv[k]);
      }
    }
    return;
  }
  for (int pl = 0; pl < PPW; ++pl) {
    const int64_t pi = g0 + pl;
    if (pi >= p.planes) break;
    const T* ub = (const T*)p.u + pi * HW;
    T* yb = (T*)p.y + pi * HW;
    const float* ac = lds + pl * C::ACC;
    if (p.vec_y == 2) epilogue<T, 16 / sizeof(T)>(ub, yb, ac, S, S, C::P, tid);
    else if (p.vec_y == 1) epilogue<T, 8 / sizeof(T)>(ub, yb, ac, S, S, C::P, tid);
    else epilogue<T, 1>(ub, yb, ac, S, S, C::P, tid);
  }
}

template <typename T, int S>
hipError_t launch_fixed(const ResFwdParams& p, hipStream_t st) {
  using C = FixedCfg<T, S>;
  auto kern = p.logits ? (p.grouped ? fixed_fwd_kernel<T, S, true, true> : fixed_fwd_kernel<T, S, false, true>)
                       : (p.grouped ? fixed_fwd_kernel<T, S, true, false> : fixed_fwd_kernel<T, S, false, false>);
  if (C::LDS_BYTES > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       C::LDS_BYTES);
    if (e != hipSuccess) return e;
  }
  const int64_t groups = (p.planes + C::PPW - 1) / C::PPW;
  hipLaunchKernelGGL(kern, dim3((unsigned)groups), dim3(128), C::LDS_BYTES, st, p);
  return hipGetLastError();
}

}  // namespace gspn
