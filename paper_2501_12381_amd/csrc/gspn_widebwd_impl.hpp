// Persistent backward (Alg. 2, the exact adjoint of Eq. 1-2) for 128 x 128
// planes.
//
// One workgroup of four waves per compute unit walks its share of the planes.
// Wave d owns direction d (T2B, B2T, L2R, R2L); a lane owns two adjacent
// positions of every line (columns for the vertical waves, rows for the
// horizontal ones) and keeps its direction's state for the whole plane in
// registers: 128 lines x 2 positions of fp32, h after the forward recompute,
// overwritten line by line with g during the adjoint (h of a line is last
// needed by the step of the next line).  LDS holds two fp32 arrays of the
// plane (row pitch 129): A = lam * x, later u * dy; B = the direction sums,
// and during the adjoint the horizontal waves' dw staging.
//
// Per plane:
//   P0  all waves: A = lam * x (a quarter of the rows each)
//   F   wave d: forward recompute of h_d (weights streamed from HBM, lam * x
//       from A), kept in registers
//   Sh  B = sum_d h_d in a fixed order (four rounds, two waves each)
//   P2  all waves: du = dy * B, A = u * dy
//   A   wave d: adjoint g(line) = u*dy + transposed stencil of the next line's
//       weights and g; dw_k = g * h(previous line)(p + k - 1).  The vertical
//       waves store dw rows directly; the horizontal waves stage dw in LDS and
//       write it out as row segments every SC columns
//   Sg  B = sum_d g_d in the same fixed order
//   P4  all waves: dx = lam * B, dlam = x * B
// Every sum has a fixed order, so results are reproducible run to run.
//
// HBM traffic: the inputs once, except x and lam (P0 and P4) and the weights
// (F and A), which are read twice: 90 bytes per pixel against 62 algorithmic
// (bf16).
#pragma once

#include <atomic>

#include "gspn_device.hpp"
#include "gspn_launch.hpp"
#include "gspn_resident_impl.hpp"
#include "gspn_resident_bwd_impl.hpp"
#include "gspn_wide_impl.hpp"

namespace gspn {

template <typename T>
struct WideBwdCfg {
  static constexpr int S = 128;
  static constexpr int NP = 2;                     // positions per lane
  static constexpr int P = S + 1;                  // LDS row pitch (odd)
  static constexpr int ARR = S * P;                // floats per array
  static constexpr int RV = 14;                    // vertical ring: rows in flight
  static constexpr int VE = 16 / (int)sizeof(T);   // columns per 16-byte vector
  static constexpr int CG = 3;                     // horizontal ring: column groups of VE columns
  static constexpr int SC = 64 / (int)sizeof(T);   // horizontal dw staging: columns per flush (64 bytes)
  static constexpr int SPW = 17;                   // staging row pitch in 4-byte words (64 bytes + 4)
  static constexpr int SREG = 3 * S * SPW;         // words of one horizontal wave's staging region
  static constexpr int G = 4;                      // LDS lookahead (lines)
  static constexpr int LDS_BYTES = 2 * ARR * 4;
  static_assert(2 * SREG <= ARR, "both staging regions fit in B");
  static_assert(S % SC == 0 && SC % VE == 0, "staging blocks divide the plane");
};

struct WideBwdParams {
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
  // per direction: bit l of word l / 64 set when line l starts a group (the
  // first line of the direction's scan is always set)
  uint64_t gstart[4][2];
  int logits, renorm;  // w holds Eq. 6 logits (dw: their gradient); renorm: on-line neighbours only
};

template <int L>
__device__ __forceinline__ bool wb_gbit(const uint64_t (&g)[2]) {
  return (g[L >> 6] >> (L & 63)) & 1;
}

// One wave's direction: forward recompute, its part of the sums, adjoint.
template <typename T, bool HZ, bool REV>
struct WideBwdRole {
  using C = WideBwdCfg<T>;
  static constexpr int S = C::S, NP = C::NP, P = C::P, G = C::G;
  static constexpr int RB = S * (int)sizeof(T), PB = S * RB;  // bytes of a row, of a plane
  typedef Pack<T, NP> PK2;
  typedef Pack<T, C::VE> PKV;

  // scan order: line of step s
  template <int s> static constexpr int fline() { return REV ? S - 1 - s : s; }

  // --- LDS offset of (line, the lane's first position) in an array
  __device__ __forceinline__ static int aoff(int line, int lane) {
    return HZ ? (2 * lane) * P + line : line * P + 2 * lane;
  }
  // the lane's two values of a line from an LDS array
  __device__ __forceinline__ static void lds_get(const float* __restrict__ a, int line, int lane, float (&v)[NP]) {
    const int o = aoff(line, lane);
    v[0] = a[o];
    v[1] = a[o + (HZ ? P : 1)];
  }
};

// ----------------------------------------------------------------------------
// vertical role: lines are rows, the lane owns columns 2 lane, 2 lane + 1
// ----------------------------------------------------------------------------
// LG: the weight maps hold Eq. 6 logits (normalised as they are unpacked; the
// adjoint's dw go through the Jacobian before they are stored).
template <typename T, bool REV, bool LG>
__device__ __forceinline__ void wb_vertical(const WideBwdParams& p, int64_t plane, int slot, float (&hreg)[128][2],
                                            float* __restrict__ A, const uint64_t (&gst)[2], int lane,
                                            bool forward) {
  using C = WideBwdCfg<T>;
  using RL = WideBwdRole<T, false, REV>;
  constexpr int S = C::S, NP = C::NP, R = C::RV, G = C::G, RB = RL::RB, PB = RL::PB;
  typedef Pack<T, NP> PK;
  const int64_t pof = plane * (S * S);
  const T* w0 = (const T*)p.w + (int64_t)slot * 3 * p.npc + pof;
  wide_rsrc_t rw[3];
#pragma unroll
  for (int m = 0; m < 3; ++m) rw[m] = wide_rsrc(w0 + m * p.npc, PB);
  const int voff = 2 * lane * (int)sizeof(T);
  const bool rn = LG && p.renorm != 0;
  // forward order visits lines fline(0..S-1); the adjoint the reverse
  auto line_at = [&](int s) { return forward ? (REV ? S - 1 - s : s) : (REV ? s : S - 1 - s); };
  PK ring[R][3];
  auto load_row = [&](PK (&sl)[3], int s) __attribute__((always_inline)) {
    const int so = s < S ? line_at(s) * RB : kWideOob;
#pragma unroll
    for (int m = 0; m < 3; ++m) wide_load(sl[m], rw[m], voff, so);
  };
#pragma unroll
  for (int k = 0; k < R; ++k) load_row(ring[k], k);
  float la[G][NP];
#pragma unroll
  for (int g = 0; g < G; ++g) RL::lds_get(A, line_at(g), lane, la[g]);

  if (forward) {
    float hp[NP] = {0.f, 0.f};
    static_for<0, S>([&](auto sc) __attribute__((always_inline)) {
      constexpr int s = decltype(sc)::value, k = s % R, gi = s % G;
      constexpr int line = REV ? S - 1 - s : s;
      float lx[NP], a[NP], b[NP], c[NP];
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        lx[q] = la[gi][q];
        a[q] = ring[k][0].get(q);
        b[q] = ring[k][1].get(q);
        c[q] = ring[k][2].get(q);
      }
      load_row(ring[k], s + R);
      if (s + G < S) RL::lds_get(A, line_at(s + G), lane, la[gi]);
      if (wb_gbit<line>(gst)) hp[0] = hp[1] = 0.f;  // a group starts here
      norm_weights<LG, NP>(a, b, c, 2 * lane, S, rn);
      wide_step<NP>(lx, a, b, c, hp);
      hreg[line][0] = hp[0];
      hreg[line][1] = hp[1];
      __builtin_amdgcn_sched_barrier(0);  // keep steps apart: the state leaves no room for overlap
    });
  } else {
    // adjoint: lines in reverse scan order; (gn, wn) belong to the line after
    // the current one in scan order
    T* dwb = (T*)p.dw + (int64_t)slot * 3 * p.npc + pof;
    const wide_rsrc_t rd[3] = {wide_rsrc(dwb, PB), wide_rsrc(dwb + p.npc, PB), wide_rsrc(dwb + 2 * p.npc, PB)};
    float gn[NP] = {0.f, 0.f}, wn[3][NP] = {{0.f, 0.f}, {0.f, 0.f}, {0.f, 0.f}};
    static_for<0, S>([&](auto sc) __attribute__((always_inline)) {
      constexpr int s = decltype(sc)::value, k = s % R, gi = s % G;
      constexpr int line = REV ? s : S - 1 - s;
      constexpr int succ = REV ? line - 1 : line + 1;   // next line in scan order
      constexpr int prev = REV ? line + 1 : line - 1;   // previous line in scan order
      if constexpr (succ >= 0 && succ < S) {
        if (wb_gbit<succ>(gst)) gn[0] = gn[1] = 0.f;    // that line took nothing from this one
      }
      float udy[NP];
#pragma unroll
      for (int q = 0; q < NP; ++q) udy[q] = la[gi][q];
      if (s + G < S) RL::lds_get(A, line_at(s + G), lane, la[gi]);
      float a0[NP], a1[NP], a2[NP];
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        a0[q] = wn[0][q] * gn[q];
        a1[q] = wn[1][q] * gn[q];
        a2[q] = wn[2][q] * gn[q];
      }
      float g[NP];
      g[0] = udy[0] + a1[0] + a0[1] + from_prev_lane(a2[1]);
      g[1] = udy[1] + a1[1] + from_next_lane(a0[0]) + a2[0];
      float hv[NP] = {0.f, 0.f};
      if constexpr (prev >= 0 && prev < S) {
        if (!wb_gbit<line>(gst)) {
          hv[0] = hreg[prev][0];
          hv[1] = hreg[prev][1];
        }
      }
      const float hl0 = from_prev_lane(hv[1]), hr1 = from_next_lane(hv[0]);
      float d[3][NP];
      d[0][0] = g[0] * hl0;   d[1][0] = g[0] * hv[0]; d[2][0] = g[0] * hv[1];
      d[0][1] = g[1] * hv[0]; d[1][1] = g[1] * hv[1]; d[2][1] = g[1] * hr1;
      if constexpr (LG) {
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          const int col = 2 * lane + q;
          const Norm3 nr = normalize3(ring[k][0].get(q), ring[k][1].get(q), ring[k][2].get(q), col == 0,
                                      col == S - 1, rn);
          norm3_vjp(nr, d[0][q], d[1][q], d[2][q]);
          wn[0][q] = nr.w[0];
          wn[1][q] = nr.w[1];
          wn[2][q] = nr.w[2];
        }
      }
#pragma unroll
      for (int m = 0; m < 3; ++m) wide_store<T, NP>(d[m], rd[m], voff, line * RB);
      if constexpr (!LG) {
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          wn[0][q] = ring[k][0].get(q);
          wn[1][q] = ring[k][1].get(q);
          wn[2][q] = ring[k][2].get(q);
        }
      }
      load_row(ring[k], s + R);
      hreg[line][0] = g[0];
      hreg[line][1] = g[1];
      gn[0] = g[0];
      gn[1] = g[1];
      __builtin_amdgcn_sched_barrier(0);
    });
  }
}

// ----------------------------------------------------------------------------
// horizontal role: lines are columns, the lane owns rows 2 lane, 2 lane + 1.
// Weights arrive as 16-byte row pieces (VE columns) through a ring of CG
// column groups; the adjoint stages dw in LDS (region `stg`, [map][row][SC]
// with a 17-word row pitch) and writes it out as 64-byte row segments.
// ----------------------------------------------------------------------------
template <typename T, bool REV, bool LG>
__device__ __forceinline__ void wb_horizontal(const WideBwdParams& p, int64_t plane, int slot,
                                              float (&hreg)[128][2], float* __restrict__ A,
                                              uint32_t* __restrict__ stg, const uint64_t (&gst)[2], int lane,
                                              bool forward) {
  using C = WideBwdCfg<T>;
  using RL = WideBwdRole<T, true, REV>;
  constexpr int S = C::S, NP = C::NP, G = C::G, VE = C::VE, CG = C::CG, RB = RL::RB, PB = RL::PB;
  constexpr int NGR = S / VE;  // column groups per plane
  typedef Pack<T, VE> PKV;
  const int64_t pof = plane * (S * S);
  const T* w0 = (const T*)p.w + (int64_t)slot * 3 * p.npc + pof;
  wide_rsrc_t rw[3];
#pragma unroll
  for (int m = 0; m < 3; ++m) rw[m] = wide_rsrc(w0 + m * p.npc, PB);
  const int r0 = 2 * lane;
  const int voff[NP] = {r0 * RB, (r0 + 1) * RB};
  const bool rn = LG && p.renorm != 0;
  // column-group order: forward visits groups fgrp(0..), the adjoint the reverse
  auto grp_at = [&](int i) { return forward ? (REV ? NGR - 1 - i : i) : (REV ? i : NGR - 1 - i); };
  auto line_at = [&](int s) { return forward ? (REV ? S - 1 - s : s) : (REV ? s : S - 1 - s); };
  PKV ring[CG][3][NP];
  auto load_grp = [&](PKV (&sl)[3][NP], int i) __attribute__((always_inline)) {
    const int so = i < NGR ? grp_at(i) * VE * (int)sizeof(T) : kWideOob;
#pragma unroll
    for (int m = 0; m < 3; ++m)
#pragma unroll
      for (int q = 0; q < NP; ++q) wide_load(sl[m][q], rw[m], voff[q], so);
  };
#pragma unroll
  for (int i = 0; i < CG; ++i) load_grp(ring[i], i);
  float la[G][NP];
#pragma unroll
  for (int g = 0; g < G; ++g) RL::lds_get(A, line_at(g), lane, la[g]);

  if (forward) {
    float hp[NP] = {0.f, 0.f};
    static_for<0, S>([&](auto sc) __attribute__((always_inline)) {
      constexpr int s = decltype(sc)::value, gi = s % G;
      constexpr int line = REV ? S - 1 - s : s;
      constexpr int i = s / VE, k = i % CG, e = line % VE;  // group step, ring slot, column inside the piece
      float lx[NP], a[NP], b[NP], c[NP];
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        lx[q] = la[gi][q];
        a[q] = ring[k][0][q].get(e);
        b[q] = ring[k][1][q].get(e);
        c[q] = ring[k][2][q].get(e);
      }
      if (s % VE == VE - 1) load_grp(ring[k], i + CG);  // the group's last column is read
      if (s + G < S) RL::lds_get(A, line_at(s + G), lane, la[gi]);
      if (wb_gbit<line>(gst)) hp[0] = hp[1] = 0.f;
      norm_weights<LG, NP>(a, b, c, r0, S, rn);
      wide_step<NP>(lx, a, b, c, hp);
      hreg[line][0] = hp[0];
      hreg[line][1] = hp[1];
      __builtin_amdgcn_sched_barrier(0);  // keep steps apart: the state leaves no room for overlap
    });
  } else {
    constexpr int SC = C::SC, SPW = C::SPW;
    T* dwb = (T*)p.dw + (int64_t)slot * 3 * p.npc + pof;
    float gn[NP] = {0.f, 0.f}, wn[3][NP] = {{0.f, 0.f}, {0.f, 0.f}, {0.f, 0.f}};
    // staging element (map, row, column inside the SC block) as a T in LDS
    T* st = reinterpret_cast<T*>(stg);
    auto st_idx = [&](int m, int row, int cc) { return (m * S + row) * (SPW * 4 / (int)sizeof(T)) + cc; };
    static_for<0, S>([&](auto sc) __attribute__((always_inline)) {
      constexpr int s = decltype(sc)::value, gi = s % G;
      constexpr int line = REV ? s : S - 1 - s;
      constexpr int succ = REV ? line - 1 : line + 1;
      constexpr int prev = REV ? line + 1 : line - 1;
      constexpr int i = s / VE, k = i % CG, e = line % VE;
      if constexpr (succ >= 0 && succ < S) {
        if (wb_gbit<succ>(gst)) gn[0] = gn[1] = 0.f;
      }
      float udy[NP];
#pragma unroll
      for (int q = 0; q < NP; ++q) udy[q] = la[gi][q];
      if (s + G < S) RL::lds_get(A, line_at(s + G), lane, la[gi]);
      float a0[NP], a1[NP], a2[NP];
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        a0[q] = wn[0][q] * gn[q];
        a1[q] = wn[1][q] * gn[q];
        a2[q] = wn[2][q] * gn[q];
      }
      float g[NP];
      g[0] = udy[0] + a1[0] + a0[1] + from_prev_lane(a2[1]);
      g[1] = udy[1] + a1[1] + from_next_lane(a0[0]) + a2[0];
      float hv[NP] = {0.f, 0.f};
      if constexpr (prev >= 0 && prev < S) {
        if (!wb_gbit<line>(gst)) {
          hv[0] = hreg[prev][0];
          hv[1] = hreg[prev][1];
        }
      }
      const float hl0 = from_prev_lane(hv[1]), hr1 = from_next_lane(hv[0]);
      float d[3][NP];
      d[0][0] = g[0] * hl0;   d[1][0] = g[0] * hv[0]; d[2][0] = g[0] * hv[1];
      d[0][1] = g[1] * hv[0]; d[1][1] = g[1] * hv[1]; d[2][1] = g[1] * hr1;
      if constexpr (LG) {
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          const Norm3 nr = normalize3(ring[k][0][q].get(e), ring[k][1][q].get(e), ring[k][2][q].get(e),
                                      r0 + q == 0, r0 + q == S - 1, rn);
          norm3_vjp(nr, d[0][q], d[1][q], d[2][q]);
          wn[0][q] = nr.w[0];
          wn[1][q] = nr.w[1];
          wn[2][q] = nr.w[2];
        }
      }
      constexpr int cc = line % SC;  // column inside the staged block
#pragma unroll
      for (int m = 0; m < 3; ++m)
#pragma unroll
        for (int q = 0; q < NP; ++q) st[st_idx(m, r0 + q, cc)] = from_f<T>(d[m][q]);
      if constexpr (!LG) {
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          wn[0][q] = ring[k][0][q].get(e);
          wn[1][q] = ring[k][1][q].get(e);
          wn[2][q] = ring[k][2][q].get(e);
        }
      }
      if (s % VE == VE - 1) load_grp(ring[k], i + CG);
      hreg[line][0] = g[0];
      hreg[line][1] = g[1];
      gn[0] = g[0];
      gn[1] = g[1];
      if constexpr (s % SC == SC - 1) {
        // the block of SC columns is complete: write it out as 64-byte row
        // segments (the wave's own LDS writes are ordered before its reads)
        constexpr int c0 = REV ? line - (SC - 1) : line;  // first column of the block
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        constexpr int NPC = 3 * S * 4;  // 16-byte pieces: [map][row][4]
        static_for<0, NPC / 64 / 4>([&](auto jb) __attribute__((always_inline)) {
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            const int v = (decltype(jb)::value * 4 + jj) * 64 + lane, m = v / (4 * S), row = (v / 4) % S, pc = v % 4;
            const uint32_t* src = stg + (m * S + row) * SPW + pc * 4;
            uint4 t;
            t.x = src[0]; t.y = src[1]; t.z = src[2]; t.w = src[3];
            T* dst = dwb + (int64_t)m * p.npc + row * S + c0 + pc * (16 / (int)sizeof(T));
            *reinterpret_cast<uint4*>(dst) = t;
          }
          __builtin_amdgcn_sched_barrier(0);  // a batch of 4 pieces at a time
        });
        // the next block's LDS writes come after these reads (in order per wave)
      }
      __builtin_amdgcn_sched_barrier(0);
    });
  }
}

// The sum over directions into B, in direction order: round d adds wave d's
// registers (stores when d is the first present direction).  Absent
// directions keep the rounds' barriers in step.
// The sums over directions go into B (zeroed first) in four rounds with a
// barrier after each; in a round two waves of one kind add disjoint halves of
// their lines (rows for the vertical waves, columns for the horizontal ones):
//   round 0: T2B rows [0, 64), B2T rows [64, 128); round 1: the other halves;
//   round 2: L2R columns [0, 64), R2L columns [64, 128); round 3: the others.
// So every element receives its terms in a fixed order.  Lines go in batches
// of BT, the reads of the next batch issued before the writes of the current.
template <bool HZ, int L0>
__device__ __forceinline__ void wb_sum_half(float* __restrict__ B, const float (&hreg)[128][2], int lane) {
  constexpr int P = 129, BT = 16, NB = 64 / BT;
  auto off = [&](int line) { return HZ ? (2 * lane) * P + line : line * P + 2 * lane; };
  constexpr int O1 = HZ ? P : 1;
  float t[2][BT][2];
  static_for<0, BT>([&](auto jc) __attribute__((always_inline)) {
    constexpr int line = L0 + decltype(jc)::value;
    t[0][line - L0][0] = B[off(line)];
    t[0][line - L0][1] = B[off(line) + O1];
  });
  static_for<0, NB>([&](auto bc) __attribute__((always_inline)) {
    constexpr int b = decltype(bc)::value, cur = b & 1;
    if constexpr (b + 1 < NB) {
      static_for<0, BT>([&](auto jc) __attribute__((always_inline)) {
        constexpr int j = decltype(jc)::value, line = L0 + (b + 1) * BT + j;
        t[cur ^ 1][j][0] = B[off(line)];
        t[cur ^ 1][j][1] = B[off(line) + O1];
      });
    }
    static_for<0, BT>([&](auto jc) __attribute__((always_inline)) {
      constexpr int j = decltype(jc)::value, line = L0 + b * BT + j;
      B[off(line)] = t[cur][j][0] + hreg[line][0];
      B[off(line) + O1] = t[cur][j][1] + hreg[line][1];
    });
    __builtin_amdgcn_sched_barrier(0);
  });
}

// B = sum over the present directions of the waves' registers (B zeroed before).
template <int D>
__device__ __forceinline__ void wb_sum_rounds(float* __restrict__ B, const float (&hreg)[128][2], int lane,
                                              bool present) {
  constexpr bool HZ = D >= 2;
  constexpr int first_half = (D & 1) ? 64 : 0;  // round 2k: the lower-numbered wave takes lines [0, 64)
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if (present && (r >> 1) == (HZ ? 1 : 0)) {
      if ((r & 1) == 0) wb_sum_half<HZ, first_half>(B, hreg, lane);
      else wb_sum_half<HZ, 64 - first_half>(B, hreg, lane);
    }
    lds_barrier();
  }
}

// Zero this wave's quarter of an LDS array.
__device__ __forceinline__ void wb_zero_quarter(float* __restrict__ B, int wave, int lane) {
  constexpr int N = 128 * 129, Q = (N + 3) / 4;
  const int lo = wave * Q, hi = lo + Q < N ? lo + Q : N;
  for (int i = lo + lane; i < hi; i += 64) B[i] = 0.f;
}

// Elementwise passes over the rows [32 wave, 32 wave + 32).  lam * x loads
// and uses its rows in batches; the du and dx passes take their 32 rows of
// operands loaded earlier (issued before the sum rounds, which need no memory,
// so their latency passes under the rounds).
template <typename T>
struct WbRows {
  static constexpr int S = 128, P = 129, RB = S * (int)sizeof(T), PB = S * RB, BT = 8, NR = 32;
  typedef Pack<T, 2> PK;
  // A = lam * x
  __device__ __forceinline__ static void lamx(const WideBwdParams& p, int64_t pof, float* __restrict__ A, int wave,
                                              int lane) {
    const wide_rsrc_t rx = wide_rsrc((const T*)p.x + pof, PB), rl = wide_rsrc((const T*)p.lam + pof, PB);
    const int vo = 2 * lane * (int)sizeof(T);
#pragma unroll
    for (int b0 = 0; b0 < NR; b0 += BT) {
      PK vx[BT], vl[BT];
#pragma unroll
      for (int j = 0; j < BT; ++j) {
        wide_load(vx[j], rx, vo, (NR * wave + b0 + j) * RB);
        wide_load(vl[j], rl, vo, (NR * wave + b0 + j) * RB);
      }
#pragma unroll
      for (int j = 0; j < BT; ++j) {
        const int o = (NR * wave + b0 + j) * P + 2 * lane;
        A[o] = vl[j].get(0) * vx[j].get(0);
        A[o + 1] = vl[j].get(1) * vx[j].get(1);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  // the wave's rows of two maps
  __device__ __forceinline__ static void fetch(const void* ma, const void* mb, int64_t pof, PK (&va)[NR],
                                               PK (&vb)[NR], int wave, int lane) {
    const wide_rsrc_t ra = wide_rsrc((const T*)ma + pof, PB), rb = wide_rsrc((const T*)mb + pof, PB);
    const int vo = 2 * lane * (int)sizeof(T);
#pragma unroll
    for (int j = 0; j < NR; ++j) {
      wide_load(va[j], ra, vo, (NR * wave + j) * RB);
      wide_load(vb[j], rb, vo, (NR * wave + j) * RB);
    }
  }
  // du = dy * B, A = u * dy   (vd = dy, vu = u)
  __device__ __forceinline__ static void dudy(const WideBwdParams& p, int64_t pof, float* __restrict__ A,
                                              const float* __restrict__ B, const PK (&vd)[NR], const PK (&vu)[NR],
                                              int wave, int lane) {
    const wide_rsrc_t rdu = wide_rsrc((T*)p.du + pof, PB);
    const int vo = 2 * lane * (int)sizeof(T);
#pragma unroll
    for (int j = 0; j < NR; ++j) {
      const int r = NR * wave + j, o = r * P + 2 * lane;
      const float du[2] = {vd[j].get(0) * B[o], vd[j].get(1) * B[o + 1]};
      wide_store<T, 2>(du, rdu, vo, r * RB);
      A[o] = vu[j].get(0) * vd[j].get(0);
      A[o + 1] = vu[j].get(1) * vd[j].get(1);
    }
  }
  // dx = lam * B, dlam = x * B   (vl = lam, vx = x)
  __device__ __forceinline__ static void dxdl(const WideBwdParams& p, int64_t pof, const float* __restrict__ B,
                                              const PK (&vl)[NR], const PK (&vx)[NR], int wave, int lane) {
    const wide_rsrc_t rdx = wide_rsrc((T*)p.dx + pof, PB), rdl = wide_rsrc((T*)p.dlam + pof, PB);
    const int vo = 2 * lane * (int)sizeof(T);
#pragma unroll
    for (int j = 0; j < NR; ++j) {
      const int r = NR * wave + j, o = r * P + 2 * lane;
      const float dx[2] = {vl[j].get(0) * B[o], vl[j].get(1) * B[o + 1]};
      const float dl[2] = {vx[j].get(0) * B[o], vx[j].get(1) * B[o + 1]};
      wide_store<T, 2>(dx, rdx, vo, r * RB);
      wide_store<T, 2>(dl, rdl, vo, r * RB);
    }
  }
};

// The whole per-plane sequence for the wave of direction D (so the state in
// registers never meets another direction's code at a branch merge).  Every
// wave executes the same barriers in the same order.
template <typename T, int D, bool LG>
__device__ __forceinline__ void wide_bwd_wave(const WideBwdParams& p, float* __restrict__ A, float* __restrict__ B,
                                              int lane0) {
  using C = WideBwdCfg<T>;
  using RW = WbRows<T>;
  constexpr int S = C::S;
  constexpr bool HZ = D >= 2, REV = D & 1;
  const int slot = p.slot[D];
  const bool present = slot >= 0;
  uint32_t* stg = reinterpret_cast<uint32_t*>(B) + (HZ ? (D - 2) * C::SREG : 0);
  float hreg[128][2];
  typename RW::PK va[RW::NR], vb[RW::NR];
  for (int64_t plane = blockIdx.x; plane < p.planes; plane += gridDim.x) {
    // the lane index is made opaque per plane, so the compiler cannot hoist
    // the (many) per-line addresses out of the plane loop and keep them live
    int lane = lane0;
    asm volatile("" : "+v"(lane));
    const int64_t pof = plane * (S * S);
    // STAMP(0)
    RW::lamx(p, pof, A, D, lane);
    // STAMP(1)
    lds_barrier();
    // STAMP(2)
    wb_zero_quarter(B, D, lane);  // the sums' array (free until the sum rounds)
    if (present) {
      if constexpr (HZ) wb_horizontal<T, REV, LG>(p, plane, slot, hreg, A, stg, p.gstart[D], lane, true);
      else wb_vertical<T, REV, LG>(p, plane, slot, hreg, A, p.gstart[D], lane, true);
    }
    int lf = lane;
    asm volatile("" : "+v"(lf));  // keeps the loads below after the scan
    RW::fetch(p.dy, p.u, pof, va, vb, D, lf);  // operands of the du pass
    // STAMP(3)
    lds_barrier();
    // STAMP(4)
    wb_sum_rounds<D>(B, hreg, lane, present);  // B = sum_d h_d
    // STAMP(5)
    RW::dudy(p, pof, A, B, va, vb, D, lane);
    // STAMP(6)
    lds_barrier();
    // STAMP(7)
    if (present) {
      if constexpr (HZ) wb_horizontal<T, REV, LG>(p, plane, slot, hreg, A, stg, p.gstart[D], lane, false);
      else wb_vertical<T, REV, LG>(p, plane, slot, hreg, A, p.gstart[D], lane, false);
    }
    lf = lane;
    asm volatile("" : "+v"(lf));
    RW::fetch(p.lam, p.x, pof, va, vb, D, lf);  // operands of the dx pass
    // STAMP(8)
    lds_barrier();  // the horizontal waves' staging in B is written out
    wb_zero_quarter(B, D, lane);
    lds_barrier();
    // STAMP(9)
    wb_sum_rounds<D>(B, hreg, lane, present);  // B = sum_d g_d
    // STAMP(10)
    RW::dxdl(p, pof, B, va, vb, D, lane);
    // STAMP(11)
    // the next plane's first pass writes only A (last read before the adjoint's
    // barrier); B is written again only after its forward barrier
  }
}

template <typename T, bool LG>
__global__ void __launch_bounds__(256, 1) wide_bwd_kernel(WideBwdParams p) {
  using C = WideBwdCfg<T>;
  extern __shared__ float lds[];
  float* A = lds;
  float* B = lds + C::ARR;
  const int lane = threadIdx.x & 63;
  switch (__builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6)) {
    case 0: wide_bwd_wave<T, 0, LG>(p, A, B, lane); break;
    case 1: wide_bwd_wave<T, 1, LG>(p, A, B, lane); break;
    case 2: wide_bwd_wave<T, 2, LG>(p, A, B, lane); break;
    default: wide_bwd_wave<T, 3, LG>(p, A, B, lane); break;
  }
}

// instantiated once per element type and weight kind (gspn_widebwd_*.hip: plain
// weights and the dispatch; gspn_widebwdlg_*.hip: logits)
hipError_t wide_bwd_launch_f32(const WideBwdParams& p, hipStream_t st);
hipError_t wide_bwd_launch_bf16(const WideBwdParams& p, hipStream_t st);

template <typename T, bool LG>
hipError_t launch_wide_bwd(const WideBwdParams& p, hipStream_t st) {
  using C = WideBwdCfg<T>;
  auto kern = wide_bwd_kernel<T, LG>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_BYTES);
  if (e != hipSuccess) return e;
  const int64_t cus = wide_cu_count();
  const int64_t grid = p.planes < cus ? p.planes : cus;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(256), C::LDS_BYTES, st, p);
  return hipGetLastError();
}

}  // namespace gspn
