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
//   Sh  B = sum_d h_d, the waves adding in direction order (one barrier each)
//   P2  all waves: du = dy * B, A = u * dy
//   A   wave d: adjoint g(line) = u*dy + transposed stencil of the next line's
//       weights and g; dw_k = g * h(previous line)(p + k - 1).  The vertical
//       waves store dw rows directly; the horizontal waves stage dw in LDS and
//       write it out as row segments every SC columns
//   Sg  B = sum_d g_d in direction order
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
  static constexpr int RV = 10;                    // vertical ring: rows in flight
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
template <typename T, bool REV>
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
#pragma unroll
      for (int m = 0; m < 3; ++m) wide_store<T, NP>(d[m], rd[m], voff, line * RB);
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        wn[0][q] = ring[k][0].get(q);
        wn[1][q] = ring[k][1].get(q);
        wn[2][q] = ring[k][2].get(q);
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
template <typename T, bool REV>
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
      constexpr int cc = line % SC;  // column inside the staged block
#pragma unroll
      for (int m = 0; m < 3; ++m)
#pragma unroll
        for (int q = 0; q < NP; ++q) st[st_idx(m, r0 + q, cc)] = from_f<T>(d[m][q]);
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        wn[0][q] = ring[k][0][q].get(e);
        wn[1][q] = ring[k][1][q].get(e);
        wn[2][q] = ring[k][2][q].get(e);
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
// Lines go in batches of 8 (reads, then writes) with scheduling barriers
// between batches, so no more than a batch of reads is in flight in registers
// beside the 256 of state.
template <bool HZ>
__device__ __forceinline__ void wb_sum_round(float* __restrict__ B, const float (&hreg)[128][2], int lane,
                                             bool first) {
  constexpr int P = 129, BT = 8;
  static_for<0, 128 / BT>([&](auto bc) __attribute__((always_inline)) {
    constexpr int l0 = decltype(bc)::value * BT;
    float t[BT][2];
    if (!first) {
      static_for<0, BT>([&](auto jc) __attribute__((always_inline)) {
        constexpr int line = l0 + decltype(jc)::value;
        const int o0 = HZ ? (2 * lane) * P + line : line * P + 2 * lane;
        t[line - l0][0] = B[o0];
        t[line - l0][1] = B[o0 + (HZ ? P : 1)];
      });
    }
    static_for<0, BT>([&](auto jc) __attribute__((always_inline)) {
      constexpr int line = l0 + decltype(jc)::value;
      const int o0 = HZ ? (2 * lane) * P + line : line * P + 2 * lane;
      B[o0] = first ? hreg[line][0] : t[line - l0][0] + hreg[line][0];
      B[o0 + (HZ ? P : 1)] = first ? hreg[line][1] : t[line - l0][1] + hreg[line][1];
    });
    __builtin_amdgcn_sched_barrier(0);
  });
}

// Elementwise passes over the rows [32 wave, 32 wave + 32), in batches of 8
// rows whose loads are issued before their use.
template <typename T>
struct WbRows {
  static constexpr int S = 128, P = 129, RB = S * (int)sizeof(T), PB = S * RB, BT = 8;
  // A = lam * x
  __device__ __forceinline__ static void lamx(const WideBwdParams& p, int64_t pof, float* __restrict__ A, int wave,
                                              int lane) {
    const wide_rsrc_t rx = wide_rsrc((const T*)p.x + pof, PB), rl = wide_rsrc((const T*)p.lam + pof, PB);
    const int vo = 2 * lane * (int)sizeof(T);
#pragma unroll
    for (int b0 = 0; b0 < 32; b0 += BT) {
      Pack<T, 2> vx[BT], vl[BT];
#pragma unroll
      for (int j = 0; j < BT; ++j) {
        wide_load(vx[j], rx, vo, (32 * wave + b0 + j) * RB);
        wide_load(vl[j], rl, vo, (32 * wave + b0 + j) * RB);
      }
#pragma unroll
      for (int j = 0; j < BT; ++j) {
        const int o = (32 * wave + b0 + j) * P + 2 * lane;
        A[o] = vl[j].get(0) * vx[j].get(0);
        A[o + 1] = vl[j].get(1) * vx[j].get(1);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  // du = dy * B, A = u * dy
  __device__ __forceinline__ static void dudy(const WideBwdParams& p, int64_t pof, float* __restrict__ A,
                                              const float* __restrict__ B, int wave, int lane) {
    const wide_rsrc_t rdy = wide_rsrc((const T*)p.dy + pof, PB), ru = wide_rsrc((const T*)p.u + pof, PB);
    const wide_rsrc_t rdu = wide_rsrc((T*)p.du + pof, PB);
    const int vo = 2 * lane * (int)sizeof(T);
#pragma unroll
    for (int b0 = 0; b0 < 32; b0 += BT) {
      Pack<T, 2> vd[BT], vu[BT];
#pragma unroll
      for (int j = 0; j < BT; ++j) {
        wide_load(vd[j], rdy, vo, (32 * wave + b0 + j) * RB);
        wide_load(vu[j], ru, vo, (32 * wave + b0 + j) * RB);
      }
#pragma unroll
      for (int j = 0; j < BT; ++j) {
        const int r = 32 * wave + b0 + j, o = r * P + 2 * lane;
        const float du[2] = {vd[j].get(0) * B[o], vd[j].get(1) * B[o + 1]};
        wide_store<T, 2>(du, rdu, vo, r * RB);
        A[o] = vu[j].get(0) * vd[j].get(0);
        A[o + 1] = vu[j].get(1) * vd[j].get(1);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  // dx = lam * B, dlam = x * B
  __device__ __forceinline__ static void dxdl(const WideBwdParams& p, int64_t pof, const float* __restrict__ B,
                                              int wave, int lane) {
    const wide_rsrc_t rl = wide_rsrc((const T*)p.lam + pof, PB), rx = wide_rsrc((const T*)p.x + pof, PB);
    const wide_rsrc_t rdx = wide_rsrc((T*)p.dx + pof, PB), rdl = wide_rsrc((T*)p.dlam + pof, PB);
    const int vo = 2 * lane * (int)sizeof(T);
#pragma unroll
    for (int b0 = 0; b0 < 32; b0 += BT) {
      Pack<T, 2> vl[BT], vx[BT];
#pragma unroll
      for (int j = 0; j < BT; ++j) {
        wide_load(vl[j], rl, vo, (32 * wave + b0 + j) * RB);
        wide_load(vx[j], rx, vo, (32 * wave + b0 + j) * RB);
      }
#pragma unroll
      for (int j = 0; j < BT; ++j) {
        const int r = 32 * wave + b0 + j, o = r * P + 2 * lane;
        const float dx[2] = {vl[j].get(0) * B[o], vl[j].get(1) * B[o + 1]};
        const float dl[2] = {vx[j].get(0) * B[o], vx[j].get(1) * B[o + 1]};
        wide_store<T, 2>(dx, rdx, vo, r * RB);
        wide_store<T, 2>(dl, rdl, vo, r * RB);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
};

// The whole per-plane sequence for the wave of direction D (so the state in
// registers never meets another direction's code at a branch merge).  Every
// wave executes the same barriers in the same order.
template <typename T, int D>
__device__ __forceinline__ void wide_bwd_wave(const WideBwdParams& p, float* __restrict__ A, float* __restrict__ B,
                                              int lane0) {
  using C = WideBwdCfg<T>;
  constexpr int S = C::S;
  constexpr bool HZ = D >= 2, REV = D & 1;
  const int slot = p.slot[D];
  int first_dir = 0;
  while (first_dir < 4 && p.slot[first_dir] < 0) ++first_dir;
  uint32_t* stg = reinterpret_cast<uint32_t*>(B) + (HZ ? (D - 2) * C::SREG : 0);
  float hreg[128][2];
  for (int64_t plane = blockIdx.x; plane < p.planes; plane += gridDim.x) {
    // the lane index is made opaque per plane, so the compiler cannot hoist
    // the (many) per-line addresses out of the plane loop and keep them live
    int lane = lane0;
    asm volatile("" : "+v"(lane));
    const int64_t pof = plane * (S * S);
    WbRows<T>::lamx(p, pof, A, D, lane);
    lds_barrier();
    if (slot >= 0) {
      if constexpr (HZ) wb_horizontal<T, REV>(p, plane, slot, hreg, A, stg, p.gstart[D], lane, true);
      else wb_vertical<T, REV>(p, plane, slot, hreg, A, p.gstart[D], lane, true);
    }
    lds_barrier();
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      if (d == D && slot >= 0) wb_sum_round<HZ>(B, hreg, lane, D == first_dir);
      lds_barrier();
    }
    WbRows<T>::dudy(p, pof, A, B, D, lane);
    lds_barrier();
    if (slot >= 0) {
      if constexpr (HZ) wb_horizontal<T, REV>(p, plane, slot, hreg, A, stg, p.gstart[D], lane, false);
      else wb_vertical<T, REV>(p, plane, slot, hreg, A, p.gstart[D], lane, false);
    }
    lds_barrier();
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      if (d == D && slot >= 0) wb_sum_round<HZ>(B, hreg, lane, D == first_dir);
      lds_barrier();
    }
    WbRows<T>::dxdl(p, pof, B, D, lane);
    // the next plane's first pass writes only A (last read before the adjoint's
    // barrier); B is written again only after its forward barrier
  }
}

template <typename T>
__global__ void __launch_bounds__(256, 1) wide_bwd_kernel(WideBwdParams p) {
  using C = WideBwdCfg<T>;
  extern __shared__ float lds[];
  float* A = lds;
  float* B = lds + C::ARR;
  const int lane = threadIdx.x & 63;
  switch (__builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6)) {
    case 0: wide_bwd_wave<T, 0>(p, A, B, lane); break;
    case 1: wide_bwd_wave<T, 1>(p, A, B, lane); break;
    case 2: wide_bwd_wave<T, 2>(p, A, B, lane); break;
    default: wide_bwd_wave<T, 3>(p, A, B, lane); break;
  }
}

// instantiated once per element type (gspn_widebwd_{f32,bf16}.hip)
hipError_t wide_bwd_launch_f32(const WideBwdParams& p, hipStream_t st);
hipError_t wide_bwd_launch_bf16(const WideBwdParams& p, hipStream_t st);

template <typename T>
hipError_t launch_wide_bwd(const WideBwdParams& p, hipStream_t st) {
  using C = WideBwdCfg<T>;
  auto kern = wide_bwd_kernel<T>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_BYTES);
  if (e != hipSuccess) return e;
  const int64_t cus = wide_cu_count();
  const int64_t grid = p.planes < cus ? p.planes : cus;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(256), C::LDS_BYTES, st, p);
  return hipGetLastError();
}

}  // namespace gspn
