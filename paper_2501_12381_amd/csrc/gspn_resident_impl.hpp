// Resident kernels: one workgroup owns whole planes and runs every direction of
// the mask in one launch, so each input is read from HBM once and y is written
// once (the algorithmic minimum of traffic).
//
// Layout of the work:
//   * a workgroup has two waves; a line (row or column) of a plane is held by
//     one wave, each lane owning NP consecutive positions, so the neighbour
//     exchange of Sec. 3.3's three-way connection is two DPP wave shifts per
//     line, with no barrier;
//   * small planes (lines of at most 31 positions) are packed several to a
//     wave in SEG-lane segments, the padding lanes between them holding zeros;
//   * phase V: wave 0 runs top-to-bottom while wave 1 runs bottom-to-top;
//     phase H: wave 0 runs left-to-right while wave 1 runs right-to-left;
//   * sum_d h_d accumulates in fp32 in LDS.  Within a phase the two waves touch
//     disjoint lines until the middle line; a barrier there (and one more for
//     the shared middle line of an odd count) fixes the order of every
//     addition, so results are bitwise reproducible;
//   * inputs stream from global memory in tiles of PD lines, double-buffered in
//     registers: the next tile's loads are in flight while the current one is
//     computed.  Vertical tiles load NP contiguous positions per line,
//     horizontal tiles load PD contiguous lines per position (row segments);
//   * loads are branch-free: indices past the end of a line, of the plane or of
//     the batch are clamped to valid memory and the corresponding h is forced
//     to 0 (LDS writes of such lanes land in a padding row/column), so no load
//     result has to be merged across divergent paths and the prefetched tiles
//     really stay in flight;
//   * the epilogue writes y = u * acc with coalesced vector stores.
#pragma once

#include "gspn_device.hpp"
#include "gspn_launch.hpp"

namespace gspn {

// ---------------------------------------------------------------------------
// packed element groups: N consecutive elements of T kept as raw 32-bit words
// until the step that uses them (the convert of bf16 is one shift or mask)
// ---------------------------------------------------------------------------
template <typename T, int N>
struct Pack;

template <int N>
struct Pack<float, N> {
  static constexpr int kWords = N;
  uint32_t w[N];
  __device__ __forceinline__ void load(const float* __restrict__ p) {
    if constexpr (N == 1) {
      w[0] = __float_as_uint(p[0]);
    } else if constexpr (N == 2) {
      const uint2 t = *reinterpret_cast<const uint2*>(p);
      w[0] = t.x; w[1] = t.y;
    } else {
#pragma unroll
      for (int i = 0; i < N; i += 4) {
        const uint4 t = *reinterpret_cast<const uint4*>(p + i);
        w[i] = t.x; w[i + 1] = t.y; w[i + 2] = t.z; w[i + 3] = t.w;
      }
    }
  }
  __device__ __forceinline__ float get(int i) const { return __uint_as_float(w[i]); }
};

template <int N>
struct Pack<bf16, N> {
  static constexpr int kWords = (N + 1) / 2;
  uint32_t w[kWords];
  __device__ __forceinline__ void load(const bf16* __restrict__ p) {
    if constexpr (N == 1) {
      w[0] = *reinterpret_cast<const uint16_t*>(p);
    } else if constexpr (N == 2) {
      w[0] = *reinterpret_cast<const uint32_t*>(p);
    } else if constexpr (N == 4) {
      const uint2 t = *reinterpret_cast<const uint2*>(p);
      w[0] = t.x; w[1] = t.y;
    } else {
#pragma unroll
      for (int i = 0; i < N; i += 8) {
        const uint4 t = *reinterpret_cast<const uint4*>(p + i);
        w[i / 2] = t.x; w[i / 2 + 1] = t.y; w[i / 2 + 2] = t.z; w[i / 2 + 3] = t.w;
      }
    }
  }
  __device__ __forceinline__ float get(int i) const { return (i & 1) ? bf_hi(w[i >> 1]) : bf_lo(w[i >> 1]); }
};

// Geometry of one phase for one wave.
struct Phase {
  int L;   // lines in the phase (H for vertical, W for horizontal)
  int Pn;  // positions per line
  int W;   // row pitch of the global tensors
  int P;   // row pitch of the LDS accumulator
  int G;   // lines per local-GSPN group (L: the global scan)
  bool renorm;  // Eq. 6 logits: normalise over the on-line neighbours only
};

// The five inputs of a line step: x, lam, w0, w1, w2 (pointers at the plane base).
template <typename T>
struct Maps {
  const T* m[5];
};

// One step of the recurrence for the lane's NP positions (Eq. 1):
//   h[q] = w0 * hprev[q-1] + w1 * hprev[q] + w2 * hprev[q+1] + lam * x
// with the neighbours outside the lane taken from the adjacent lanes.
template <int NP>
__device__ __forceinline__ void line_step(const float (&xv)[NP], const float (&lv)[NP],
                                          const float (&a)[NP], const float (&b)[NP],
                                          const float (&c)[NP], const bool (&valid)[NP],
                                          float (&hp)[NP]) {
  const float left = from_prev_lane(hp[NP - 1]);
  const float right = from_next_lane(hp[0]);
  float h[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    const float hl = q == 0 ? left : hp[q - 1];
    const float hr = q == NP - 1 ? right : hp[q + 1];
    float v = lv[q] * xv[q];
    v = fmaf(a[q], hl, v);
    v = fmaf(b[q], hp[q], v);
    v = fmaf(c[q], hr, v);
    h[q] = valid[q] ? v : 0.f;
  }
#pragma unroll
  for (int q = 0; q < NP; ++q) hp[q] = h[q];
}

// Eq. 6 on the lane's NP positions (LG: the weight maps hold logits): w0..w2
// of each position in place, renormalised over on-line neighbours when
// renorm is set.  Positions past the line keep whatever they get (their h is
// forced to 0).
template <bool LG, int NP>
__device__ __forceinline__ void norm_weights(float (&a)[NP], float (&b)[NP], float (&c)[NP], int pos0, int Pn,
                                             bool renorm) {
  if constexpr (LG) {
#pragma unroll
    for (int q = 0; q < NP; ++q) {
      const Norm3 r = normalize3(a[q], b[q], c[q], pos0 + q == 0, pos0 + q == Pn - 1, renorm);
      a[q] = r.w[0];
      b[q] = r.w[1];
      c[q] = r.w[2];
    }
  }
}

// Add h into the accumulator at the step's line.  The value to add to was
// read one step earlier (`cur`); the read for the next line is issued here,
// except across the middle barrier, where the other wave may still write.
// At the middle step the two waves of the phase synchronise so that all the
// additions of the first half precede those of the second (and, for an odd
// number of lines, the forward wave's addition to the shared middle line
// precedes the reverse wave's).
template <bool REV, int NP>
__device__ __forceinline__ void acc_step(float* __restrict__ acc, const int (&off)[NP],
                                         const int (&noff)[NP], bool has_next, float (&cur)[NP],
                                         const float (&h)[NP], int s, int mid, bool odd) {
  if (s == mid) {
    lds_barrier();
    if (odd) {
      if (!REV) {
#pragma unroll
        for (int q = 0; q < NP; ++q) acc[off[q]] += h[q];
      }
      lds_barrier();
      if (REV) {
#pragma unroll
        for (int q = 0; q < NP; ++q) acc[off[q]] += h[q];
      }
    } else {
#pragma unroll
      for (int q = 0; q < NP; ++q) acc[off[q]] += h[q];
    }
    if (has_next) {
#pragma unroll
      for (int q = 0; q < NP; ++q) cur[q] = acc[noff[q]];
    }
    return;
  }
  float nxt[NP];
  const bool pre = has_next && s + 1 != mid;
  if (pre) {
#pragma unroll
    for (int q = 0; q < NP; ++q) nxt[q] = acc[noff[q]];
  }
#pragma unroll
  for (int q = 0; q < NP; ++q) acc[off[q]] = cur[q] + h[q];
  if (pre) {
#pragma unroll
    for (int q = 0; q < NP; ++q) cur[q] = nxt[q];
  } else if (has_next && s + 1 == mid) {
    // read after the barrier of the next step
  }
}

// Vertical phase (rows are lines): each lane owns NP contiguous columns.  The
// five inputs of the next D lines are kept in flight in a register ring: the
// step that consumes slot k re-issues it for the line D steps ahead.
template <typename T, bool REV, int NP, int D, bool VV, bool LG>
__device__ __forceinline__ void scan_v(const Maps<T>& mp, const Phase& g, float* __restrict__ acc,
                                       int pos0, int pad_off) {
  bool valid[NP];
  int poff[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    valid[q] = pos0 + q < g.Pn;
    poff[q] = valid[q] ? pos0 + q : pad_off;
  }
  const int pc = pos0 < g.Pn ? pos0 : 0;  // VV: whole vectors are in or out of the row
  auto line_of = [&](int s) { return REV ? g.L - 1 - s : s; };
  auto load_slot = [&](Pack<T, NP> (&slot)[5], int s) {
    int line = line_of(s < g.L ? s : g.L - 1);
    const int64_t base = (int64_t)line * g.W;
#pragma unroll
    for (int m = 0; m < 5; ++m) {
      if constexpr (VV) {
        slot[m].load(mp.m[m] + base + pc);
      } else {
        // element-wise, each column clamped into the row
        Pack<T, NP> t;
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          const int cidx = pos0 + q < g.Pn ? pos0 + q : g.Pn - 1;
          Pack<T, 1> e;
          e.load(mp.m[m] + base + cidx);
          if constexpr (sizeof(T) == 4) t.w[q] = e.w[0];
          else t.w[q >> 1] = (q & 1) ? ((t.w[q >> 1] & 0xffffu) | (e.w[0] << 16)) : e.w[0];
        }
        slot[m] = t;
      }
    }
  };
  Pack<T, NP> ring[D][5];
#pragma unroll
  for (int k = 0; k < D; ++k) load_slot(ring[k], k);
  float hp[NP], cur[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    hp[q] = 0.f;
    cur[q] = acc[poff[q] + line_of(0) * g.P];
  }
  const int mid = g.L / 2;
  const bool odd = g.L & 1;
  for (int s0 = 0; s0 < g.L; s0 += D) {
#pragma unroll
    for (int k = 0; k < D; ++k) {
      const int s = s0 + k;
      if (s < g.L) {  // uniform
        float v[5][NP];
#pragma unroll
        for (int m = 0; m < 5; ++m)
#pragma unroll
          for (int q = 0; q < NP; ++q) v[m][q] = ring[k][m].get(q);
        load_slot(ring[k], s + D);
        const int line = line_of(s);
        if (group_start(line, g.G, REV)) {
#pragma unroll
          for (int q = 0; q < NP; ++q) hp[q] = 0.f;
        }
        norm_weights<LG, NP>(v[2], v[3], v[4], pos0, g.Pn, g.renorm);
        line_step<NP>(v[0], v[1], v[2], v[3], v[4], valid, hp);
        int off[NP], noff[NP];
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          off[q] = poff[q] + line * g.P;
          noff[q] = poff[q] + (REV ? line - 1 : line + 1) * g.P;
        }
        acc_step<REV, NP>(acc, off, noff, s + 1 < g.L, cur, hp, s, mid, odd);
      }
    }
  }
}

// Horizontal phase (columns are lines): each lane owns NP contiguous rows and
// reads, per row and map, PD consecutive columns as back-to-back vectors of VL
// elements (a 32-byte row segment).  Tiles of PD lines are double-buffered.
template <typename T, bool REV, int NP, int PD, int VL, bool LG>
__device__ __forceinline__ void scan_h(const Maps<T>& mp, const Phase& g, float* __restrict__ acc,
                                       int pos0, int pad_off) {
  bool valid[NP];
  int poff[NP];
  int64_t rbase[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    valid[q] = pos0 + q < g.Pn;
    poff[q] = valid[q] ? (pos0 + q) * g.P : pad_off;
    rbase[q] = (int64_t)(valid[q] ? pos0 + q : 0) * g.W;
  }
  typedef Pack<T, VL> Vec;
  constexpr int NV = PD / VL;
  auto load_tile = [&](Vec (&tl)[5][NP][NV], int t) {
    const int l0 = t * PD;
#pragma unroll
    for (int m = 0; m < 5; ++m)
#pragma unroll
      for (int q = 0; q < NP; ++q)
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          const int c = l0 + v * VL < g.L ? l0 + v * VL : 0;  // vectors past the row end re-point at its start
          tl[m][q][v].load(mp.m[m] + rbase[q] + c);
        }
  };
  const int ntiles = (g.L + PD - 1) / PD;
  const int mid = g.L / 2;
  const bool odd = g.L & 1;
  float hp[NP], cur[NP];
  const int first_line = REV ? g.L - 1 : 0;
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    hp[q] = 0.f;
    cur[q] = acc[poff[q] + first_line];
  }
  int s = 0;
  auto run = [&](const Vec (&tl)[5][NP][NV], int t) {
    const int l0 = t * PD;
#pragma unroll
    for (int ll = 0; ll < PD; ++ll) {
      const int l = REV ? PD - 1 - ll : ll;
      const int line = l0 + l;
      if (line < g.L) {  // uniform
        float v[5][NP];
#pragma unroll
        for (int m = 0; m < 5; ++m)
#pragma unroll
          for (int q = 0; q < NP; ++q) v[m][q] = tl[m][q][l / VL].get(l % VL);
        if (group_start(line, g.G, REV)) {
#pragma unroll
          for (int q = 0; q < NP; ++q) hp[q] = 0.f;
        }
        norm_weights<LG, NP>(v[2], v[3], v[4], pos0, g.Pn, g.renorm);
        line_step<NP>(v[0], v[1], v[2], v[3], v[4], valid, hp);
        int off[NP], noff[NP];
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          off[q] = poff[q] + line;
          noff[q] = poff[q] + (REV ? line - 1 : line + 1);
        }
        acc_step<REV, NP>(acc, off, noff, s + 1 < g.L, cur, hp, s, mid, odd);
        ++s;
      }
    }
  };
  Vec A[5][NP][NV], Bt[5][NP][NV];
  constexpr int dt = REV ? -1 : 1;
  int t = REV ? ntiles - 1 : 0;
  load_tile(A, t);
  for (int k = 0; k < ntiles; k += 2) {
    const bool hasB = k + 1 < ntiles;
    if (hasB) load_tile(Bt, t + dt);
    run(A, t);
    if (hasB) {
      if (k + 2 < ntiles) load_tile(A, t + 2 * dt);
      run(Bt, t + dt);
    }
    t += 2 * dt;
  }
}

// ---------------------------------------------------------------------------
// forward kernel
//   blockIdx.x -> a group of PPW = 64/SEG planes; in phase V wave 0 scans
//   top-to-bottom and wave 1 bottom-to-top, in phase H wave 0 scans
//   left-to-right and wave 1 right-to-left.  `slot[d]` is the index of
//   direction d's weights in w (-1 if d is not in the mask).
//   LDS per plane: (H + 1) x P floats, the last row and the columns >= W
//   being padding that absorbs the writes of lanes past the end of a line.
// ---------------------------------------------------------------------------
// y = u * acc over one plane with VE-element vectors (W % VE == 0), in
// batches of U vectors per thread whose loads are issued together.
template <typename T, int VE>
__device__ __forceinline__ void epilogue(const T* __restrict__ ub, T* __restrict__ yb,
                                         const float* __restrict__ ac, int H, int W, int P, int tid) {
  constexpr int U = 16;
  const int per_row = W / VE;
  const int n = H * per_row;
  for (int base = tid; base < n; base += 128 * U) {
    Pack<T, VE> uv[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int e = base + k * 128 < n ? base + k * 128 : base;
      const int r = e / per_row, c = (e - r * per_row) * VE;
      uv[k].load(ub + (int64_t)r * W + c);
    }
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int e = base + k * 128;
      if (e < n) {
        const int r = e / per_row, c = (e - r * per_row) * VE;
        float yv[VE];
#pragma unroll
        for (int q = 0; q < VE; ++q) yv[q] = uv[k].get(q) * ac[r * P + c + q];
        stv<VE>(yb + (int64_t)r * W + c, yv);
      }
    }
  }
}

// Unmerged outputs: y_d = u_d * acc_d for the n directions of one plane in one
// pass (u read once when it is shared), acc_d at ac + d * accsz.
template <typename T, int VE>
__device__ __forceinline__ void epilogue_pd(const T* __restrict__ ub, int64_t ustride, T* __restrict__ yb,
                                            int64_t ystride, const float* __restrict__ ac, int accsz, int n,
                                            int H, int W, int P, int tid) {
  const int per_row = W / VE;
  const int cnt = H * per_row;
  for (int e = tid; e < cnt; e += 128) {
    const int r = e / per_row, c = (e - r * per_row) * VE;
    Pack<T, VE> uv;
    uv.load(ub + (int64_t)r * W + c);
    for (int d = 0; d < n; ++d) {
      if (d > 0 && ustride) uv.load(ub + d * ustride + (int64_t)r * W + c);
      float yv[VE];
#pragma unroll
      for (int q = 0; q < VE; ++q) yv[q] = uv.get(q) * ac[d * accsz + r * P + c + q];
      stv<VE>(yb + d * ystride + (int64_t)r * W + c, yv);
    }
  }
}

struct ResFwdParams {
  const void* x;
  const void* lam;
  const void* w;
  const void* u;
  void* y;
  int64_t npc;  // elements per (B, C, H, W) tensor = stride between weight maps
  int64_t planes;
  int H, W, P;  // P: LDS row pitch (odd, > W)
  int slot[4];  // T2B, B2T, L2R, R2L -> weight slot or -1
  int vec_y;
  int gh, gw;   // local-GSPN group lengths along rows and columns (the line count: global)
  int grouped;  // gh < H or gw < W
  // per direction (T2B, B2T, L2R, R2L): bit l of word l / 64 set when line l
  // (< 128) starts a group in that direction's scan order
  uint64_t gstart[4][2];
  int logits, renorm;  // w holds Eq. 6 logits (renorm: normalised over on-line neighbours)
  // per-direction maps (generic kernel only): lam_pd: lam is (n, B, C, H, W);
  // y_pd: y is (n, B, C, H, W), y_d = u_d h_d, one LDS array per direction;
  // u_pd (with y_pd): u is (n, B, C, H, W)
  int lam_pd, u_pd, y_pd;
  int nd;              // directions present
};

template <typename T, int NP, int SEG, int DV, int PDH, bool VV, int VL, int MINW, bool LG>
__global__ void __launch_bounds__(128, MINW) resident_fwd_kernel(ResFwdParams p) {
  constexpr int PPW = 64 / SEG;
  extern __shared__ float lds[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t g0 = (int64_t)blockIdx.x * PPW;
  const int seg = lane / SEG, sl = lane % SEG;
  const int64_t plane = (g0 + seg < p.planes) ? g0 + seg : p.planes - 1;  // clamp: stores are skipped
  const int64_t HW = (int64_t)p.H * p.W;
  const int accsz = (p.H + 1) * p.P;
  const int narr = p.y_pd ? p.nd : 1;  // accumulator arrays per plane

  for (int e = tid; e < PPW * narr * accsz; e += 128) lds[e] = 0.f;
  __syncthreads();

  const int pos0 = sl * NP;
  const T* xb = (const T*)p.x + plane * HW;

#pragma unroll
  for (int ph = 0; ph < 2; ++ph) {
    const bool hz = ph == 1;
    const int slot = p.slot[hz ? 2 + wave : wave];
    Phase g;
    g.L = hz ? p.W : p.H;
    g.Pn = hz ? p.H : p.W;
    g.W = p.W;
    g.P = p.P;
    g.G = hz ? p.gw : p.gh;
    g.renorm = p.renorm != 0;
    if (slot < 0) {
      // the direction is not in the mask: keep the phase's barriers in step
      const int nbar = (g.L & 1) ? 2 : 1;
      for (int b = 0; b < nbar; ++b) lds_barrier();
    } else {
      const T* w0 = (const T*)p.w + (int64_t)slot * 3 * p.npc + plane * HW;
      const T* lb = (const T*)p.lam + (p.lam_pd ? slot * p.npc : 0) + plane * HW;
      // the direction's own array (unmerged outputs) or the shared accumulator
      float* acc = lds + (seg * narr + (p.y_pd ? slot : 0)) * accsz;
      Maps<T> mp;
      mp.m[0] = xb; mp.m[1] = lb; mp.m[2] = w0; mp.m[3] = w0 + p.npc; mp.m[4] = w0 + 2 * p.npc;
      if (!hz) {
        const int pad = p.W;  // padding column (row offset added per step)
        if (wave == 0) scan_v<T, false, NP, DV, VV, LG>(mp, g, acc, pos0, pad);
        else scan_v<T, true, NP, DV, VV, LG>(mp, g, acc, pos0, pad);
      } else {
        const int pad = p.H * p.P;  // padding row (column added per step)
        if (wave == 0) scan_h<T, false, NP, PDH, VL, LG>(mp, g, acc, pos0, pad);
        else scan_h<T, true, NP, PDH, VL, LG>(mp, g, acc, pos0, pad);
      }
    }
    __syncthreads();
  }

  // y = u * acc for the PPW planes of the group.  The u loads of a batch are
  // all issued before the first is used, so the epilogue pays one memory
  // latency per batch instead of one per element group.
  for (int pl = 0; pl < PPW; ++pl) {
    const int64_t pi = g0 + pl;
    if (pi >= p.planes) break;
    const T* ub = (const T*)p.u + pi * HW;
    T* yb = (T*)p.y + pi * HW;
    const float* ac = lds + pl * narr * accsz;
    if (p.y_pd) {
      const int64_t us = p.u_pd ? p.npc : 0;
      if (p.vec_y == 2) epilogue_pd<T, 16 / sizeof(T)>(ub, us, yb, p.npc, ac, accsz, narr, p.H, p.W, p.P, tid);
      else if (p.vec_y == 1) epilogue_pd<T, 8 / sizeof(T)>(ub, us, yb, p.npc, ac, accsz, narr, p.H, p.W, p.P, tid);
      else epilogue_pd<T, 1>(ub, us, yb, p.npc, ac, accsz, narr, p.H, p.W, p.P, tid);
      continue;
    }
    if (p.vec_y == 2) epilogue<T, 16 / sizeof(T)>(ub, yb, ac, p.H, p.W, p.P, tid);
    else if (p.vec_y == 1) epilogue<T, 8 / sizeof(T)>(ub, yb, ac, p.H, p.W, p.P, tid);
    else epilogue<T, 1>(ub, yb, ac, p.H, p.W, p.P, tid);
  }
}

}  // namespace gspn

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
namespace gspn {
// Sizes with a specialised forward kernel (square planes).
inline bool fixed_size_supported(int H, int W) {
  return H == W && (H == 16 || H == 28 || H == 32 || H == 56 || H == 64);
}
template <typename T, int S> hipError_t launch_fixed(const ResFwdParams& p, hipStream_t st);
template <typename T> hipError_t launch_wide(const ResFwdParams& p, hipStream_t st);
namespace resident_detail {

constexpr int kMaxLds = 160 * 1024;  // LDS per CU on gfx950
constexpr int kMaxLine = 256;        // longest line one wave holds (64 lanes x 4 positions)

struct Config {
  int np, seg, vl, lds, P;
  bool vv;
};

inline bool al(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// narr: accumulator arrays per plane (one per direction for unmerged outputs)
inline bool config_for(int H, int W, size_t es, const void* const* ptrs, int nptr, Config* c, int narr = 1) {
  const int mx = H > W ? H : W;
  if (mx > kMaxLine) return false;
  c->np = mx <= 64 ? 1 : (mx <= 128 ? 2 : 4);
  c->seg = mx <= 15 ? 16 : (mx <= 31 ? 32 : 64);
  c->P = W + 1 + (W & 1);
  const long lds = (long)(64 / c->seg) * narr * (H + 1) * c->P * 4;
  if (lds > kMaxLds) return false;
  c->lds = (int)lds;
  auto ptrs_al = [&](int n_el) {
    const size_t b = (size_t)n_el * es, need = b >= 16 ? 16 : b;
    for (int i = 0; i < nptr; ++i)
      if (ptrs[i] && !al(ptrs[i], need)) return false;
    return true;
  };
  c->vl = 1;
  for (int v : {8, 4, 2})
    if (W % v == 0 && ptrs_al(v)) { c->vl = v; break; }
  c->vv = c->np > 1 && W % c->np == 0 && ptrs_al(c->np);
  return true;
}

template <typename T, int NP, int SEG, bool VV, int VL>
hipError_t launch_fwd(const ResFwdParams& p, const Config& c, hipStream_t st) {
  // DV: lines in flight in the vertical ring (5 loads each, kept under the
  // 63 outstanding loads a wave can track); PDH: columns per horizontal row
  // segment (32 bytes).  Packed small planes run more waves per SIMD.
  constexpr int DV = SEG < 64 ? 6 : (NP > 2 ? 4 : 12);
  constexpr int PDH = (VL == 1 || NP > 2) ? 16 / (int)sizeof(T) / (VL == 1 ? 2 : 1) : 32 / (int)sizeof(T);
  constexpr int MINW = SEG < 64 ? 4 : (NP == 1 ? 2 : 1);
  constexpr int VLc = VL > 16 / (int)sizeof(T) ? 16 / (int)sizeof(T) : VL;
  auto kern = p.logits ? resident_fwd_kernel<T, NP, SEG, DV, PDH, VV, VLc, MINW, true>
                       : resident_fwd_kernel<T, NP, SEG, DV, PDH, VV, VLc, MINW, false>;
  if (c.lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, c.lds);
    if (e != hipSuccess) return e;
  }
  const int64_t groups = (p.planes + (64 / SEG) - 1) / (64 / SEG);
  hipLaunchKernelGGL(kern, dim3((unsigned)groups), dim3(128), c.lds, st, p);
  return hipGetLastError();
}

template <typename T, int NP, int SEG, bool VV>
hipError_t launch_fwd_vl(const ResFwdParams& p, const Config& c, hipStream_t st) {
  switch (c.vl) {
    case 8: return launch_fwd<T, NP, SEG, VV, 8>(p, c, st);
    case 4: return launch_fwd<T, NP, SEG, VV, 4>(p, c, st);
    case 2: return launch_fwd<T, NP, SEG, VV, 2>(p, c, st);
    default: return launch_fwd<T, NP, SEG, VV, 1>(p, c, st);
  }
}

}  // namespace resident_detail

template <typename T>
hipError_t resident_fwd_t(const ResidentFwdArgs& a) {
  using namespace resident_detail;
  const void* ptrs[] = {a.x, a.lam, a.w};
  int n = 0;
  for (int d = 0; d < 4; ++d) n += (a.mask >> d) & 1;
  const bool pd = a.lam_pd || a.u_pd || a.y_pd;
  if (a.u_pd && !a.y_pd) return hipErrorInvalidValue;  // a merged y with per-direction u: streaming family
  Config c;
  if (!config_for(a.H, a.W, sizeof(T), ptrs, 3, &c, a.y_pd ? n : 1)) return hipErrorInvalidValue;
  ResFwdParams p;
  p.x = a.x; p.lam = a.lam; p.w = a.w; p.u = a.u; p.y = a.y;
  p.npc = (int64_t)a.planes * a.H * a.W;
  p.planes = a.planes;
  p.H = a.H; p.W = a.W; p.P = c.P;
  n = 0;
  for (int d = 0; d < 4; ++d) p.slot[d] = (a.mask >> d) & 1 ? n++ : -1;
  p.nd = n;
  p.lam_pd = a.lam_pd; p.u_pd = a.u_pd; p.y_pd = a.y_pd;
  p.gh = (a.group_h > 0 && a.group_h < a.H) ? a.group_h : a.H;
  p.gw = (a.group_w > 0 && a.group_w < a.W) ? a.group_w : a.W;
  p.grouped = p.gh < a.H || p.gw < a.W;
  p.logits = a.logits;
  p.renorm = a.renorm;
  for (int d = 0; d < 4; ++d) {
    const bool hz = d >= 2, rev = d & 1;
    const int L = hz ? a.W : a.H, G = hz ? p.gw : p.gh;
    p.gstart[d][0] = p.gstart[d][1] = 0;
    for (int l = 0; l < L && l < 128; ++l)
      if (rev ? ((l + 1) % G == 0 || l == L - 1) : (l % G == 0)) p.gstart[d][l >> 6] |= 1ull << (l & 63);
  }
  // epilogue vectors: 16 bytes if rows allow, else 8 bytes, else scalars
  const int v16 = 16 / (int)sizeof(T), v8 = 8 / (int)sizeof(T);
  // per-direction maps start npc elements apart: their starts must keep the alignment too
  const size_t mapb = (size_t)p.npc * sizeof(T);
  p.vec_y = (a.W % v16 == 0 && al(a.u, 16) && al(a.y, 16) && (!pd || mapb % 16 == 0)) ? 2
          : (a.W % v8 == 0 && al(a.u, 8) && al(a.y, 8) && (!pd || mapb % 8 == 0)) ? 1 : 0;
  hipStream_t st = (hipStream_t)a.stream;
  // per-direction maps run on the generic kernels only
  if (!pd && a.use_fixed && !p.grouped && a.H == 128 && a.W == 128 && al(a.x, 16) && al(a.lam, 16) &&
      al(a.w, 16) && al(a.u, 16) && al(a.y, 16))
    return launch_wide<T>(p, st);  // persistent, every input read once
  if (!pd && a.use_fixed && fixed_size_supported(a.H, a.W) && al(a.x, 16) && al(a.lam, 16) && al(a.w, 16)) {
    switch (a.H) {
      case 16: return launch_fixed<T, 16>(p, st);
      case 28: return launch_fixed<T, 28>(p, st);
      case 32: return launch_fixed<T, 32>(p, st);
      case 56: return launch_fixed<T, 56>(p, st);
      default: return launch_fixed<T, 64>(p, st);
    }
  }
  if (c.np == 1 && c.seg == 16) return launch_fwd_vl<T, 1, 16, true>(p, c, st);
  if (c.np == 1 && c.seg == 32) return launch_fwd_vl<T, 1, 32, true>(p, c, st);
  if (c.np == 1) return launch_fwd_vl<T, 1, 64, true>(p, c, st);
  if (c.np == 2) return c.vv ? launch_fwd_vl<T, 2, 64, true>(p, c, st) : launch_fwd_vl<T, 2, 64, false>(p, c, st);
  return c.vv ? launch_fwd_vl<T, 4, 64, true>(p, c, st) : launch_fwd_vl<T, 4, 64, false>(p, c, st);
}

// narr: accumulator arrays per plane (the directions present, for unmerged outputs)
inline bool resident_fwd_fits(int H, int W, int dtype, int narr = 1) {
  resident_detail::Config c;
  return resident_detail::config_for(H, W, dtype == 0 ? 4 : 2, nullptr, 0, &c, narr);
}

}  // namespace gspn
