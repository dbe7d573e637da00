// Persistent forward kernel for 128 x 128 planes.
//
// One workgroup of four waves per compute unit walks its share of the planes
// one plane at a time, so a batch of planes costs ceil(planes / CUs) plane
// times with no partly filled last round.  LDS holds two fp32 arrays of the
// plane (row pitch 129): the accumulator of sum_d h_d, and lam * x.  Every
// input element is read from HBM exactly once.  Waves 0 and 1 scan the
// vertical directions (top-to-bottom, bottom-to-top; a lane owns two adjacent
// columns), waves 2 and 3 the horizontal ones (left-to-right, right-to-left;
// a lane owns two adjacent rows), so the two kinds of scan overlap:
//
//   B0..B1   the vertical waves store lam * x and h of the rows each reached
//            first (computed in registers during the previous plane's tail)
//   B1..B2   vertical second halves (lam * x from LDS, h kept in registers)
//            alongside the horizontal first halves (adding h to acc)
//   B2..B3   the vertical waves add their second-half h to acc
//   B3..     horizontal second halves, then y = u * acc by the horizontal
//            waves (each for the columns its second half covers), alongside
//            the vertical first halves of the next plane
//
// Every element of acc receives its terms in a fixed order (first vertical
// half, first horizontal half, second vertical half, second horizontal half),
// so results are reproducible run to run.  A direction absent from the mask
// costs nothing but its barriers (its vertical wave still supplies lam * x
// and zeros for its first-half rows).
#pragma once

#include <atomic>

#include "gspn_device.hpp"
#include "gspn_launch.hpp"
#include "gspn_resident_impl.hpp"

namespace gspn {

template <typename T>
struct WideCfg {
  static constexpr int S = 128;
  static constexpr int NP = 2;                   // positions per lane
  static constexpr int P = S + 1;                // LDS row pitch (odd)
  static constexpr int ARR = S * P;              // floats per array
  static constexpr int MID = S / 2;
  static constexpr int RV = 16;                  // vertical ring: rows in flight per wave
  static constexpr int VE = 16 / (int)sizeof(T); // elements per 16-byte vector
  static constexpr int TH = 128 / (int)sizeof(T);// horizontal tile: columns of a 128-byte row segment
  static constexpr int NV = TH / VE;             // 16-byte vectors per row segment
  static constexpr int NTH = S / TH;             // tiles per horizontal phase
  static constexpr int G = 4;                    // LDS lookahead (steps)
  static constexpr int NT = 256;                 // two vertical and two horizontal waves
  static constexpr int LDS_BYTES = 2 * ARR * 4;
  static_assert(MID % RV == 0 && MID % TH == 0 && NTH % 2 == 0, "ring and tiles must align with the middle line");
};

// Buffer loads: the plane base and size live in a scalar resource, the lane
// offset in one VGPR and the line offset in a scalar, so no 64-bit address
// is kept per unrolled load; reads past the plane return zero.
typedef __amdgpu_buffer_rsrc_t wide_rsrc_t;
__device__ __forceinline__ wide_rsrc_t wide_rsrc(const void* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
}
template <typename T, int N>
__device__ __forceinline__ void wide_load(Pack<T, N>& pk, wide_rsrc_t r, int voff, int soff) {
  constexpr int NW = Pack<T, N>::kWords;
  if constexpr (NW == 1) {
    pk.w[0] = __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0);
  } else if constexpr (NW == 2) {
    const auto t = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
    pk.w[0] = t[0];
    pk.w[1] = t[1];
  } else {
    static_assert(NW == 4, "one 16-byte load per pack");
    const auto t = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
#pragma unroll
    for (int i = 0; i < 4; ++i) pk.w[i] = t[i];
  }
}

template <typename T, int N>
__device__ __forceinline__ void wide_store(const float (&v)[N], wide_rsrc_t r, int voff, int soff) {
  static_assert(N == 2, "two elements per lane");
  if constexpr (sizeof(T) == 2) {
    __builtin_amdgcn_raw_buffer_store_b32(pack_bf2(v[0], v[1]), r, voff, soff, 0);
  } else {
    typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
    const u32x2 t = {__float_as_uint(v[0]), __float_as_uint(v[1])};
    __builtin_amdgcn_raw_buffer_store_b64(t, r, voff, soff, 0);
  }
}

// h[q] = w0 * hprev[q-1] + w1 * hprev[q] + w2 * hprev[q+1] + lam*x over the
// lane's NP positions, neighbours outside the lane from the adjacent lanes.
template <int NP>
__device__ __forceinline__ void wide_step(const float (&lx)[NP], const float (&a)[NP], const float (&b)[NP],
                                          const float (&c)[NP], float (&hp)[NP]) {
  const float left = from_prev_lane(hp[NP - 1]);
  const float right = from_next_lane(hp[0]);
  float h[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    const float hl = q == 0 ? left : hp[q - 1];
    const float hr = q == NP - 1 ? right : hp[q + 1];
    float v = fmaf(b[q], hp[q], lx[q]);
    v = fmaf(a[q], hl, v);
    h[q] = fmaf(c[q], hr, v);
  }
#pragma unroll
  for (int q = 0; q < NP; ++q) hp[q] = h[q];
}

// Offset past every plane: a buffer load there returns zero without touching
// memory, which turns the refills past the end of a phase into no-ops
// without a branch around the loads.
constexpr int kWideOob = 0x40000000;

// Vertical role (waves 0 and 1): the wave's direction for every plane of the
// workgroup.  Per plane, in the wave's row order s = 0 .. S-1:
//   first half  (s < MID): x, lam and the weights from HBM; lam * x and h are
//               kept in registers (lxr, hr) and stored to LDS only at the next
//               plane's start, since this half runs while the horizontal
//               waves still use the previous plane's arrays;
//   second half (s >= MID): the weights from HBM, lam * x from LDS (stored by
//               the other vertical wave); h is kept in registers (hv) and added
//               to acc once the horizontal first halves are done with it.
// A ring of R rows keeps the loads in flight across steps, barriers and
// planes: the last steps of a plane request the next plane's first rows.
// PRESENT: the direction is in the mask (otherwise the wave only supplies
// lam * x and zeros for its first-half rows).
// LG: the weight maps hold Eq. 6 logits, normalised as they are unpacked.
template <typename T, bool REV, bool PRESENT, bool LG>
__device__ __forceinline__ void wide_v_role(const ResFwdParams& p, int slot, float* __restrict__ acc,
                                            float* __restrict__ lxa, int lane) {
  using C = WideCfg<T>;
  constexpr int S = C::S, NP = C::NP, P = C::P, MID = C::MID, R = C::RV, G = C::G;
  constexpr int RB = S * (int)sizeof(T), PB = S * RB;  // bytes of a row, of a plane
  static_assert(R % G == 0 && MID % R == 0, "lookahead and ring slots repeat with the halves");
  typedef Pack<T, NP> PK;
  const int col = lane * NP;
  const int voff = col * (int)sizeof(T);
  const bool rn = LG && p.renorm;
  auto line_of = [](int s) { return REV ? S - 1 - s : s; };
  auto plane_res = [&](int64_t plane, wide_rsrc_t (&rb)[5]) __attribute__((always_inline)) {
    const int64_t pof = plane * (S * S);
    const T* w0 = (const T*)p.w + (int64_t)(slot < 0 ? 0 : slot) * 3 * p.npc + pof;
    rb[0] = wide_rsrc((const T*)p.x + pof, PB);
    rb[1] = wide_rsrc((const T*)p.lam + pof, PB);
    rb[2] = wide_rsrc(w0, PB);
    rb[3] = wide_rsrc(w0 + p.npc, PB);
    rb[4] = wide_rsrc(w0 + 2 * p.npc, PB);
  };

  PK ring[R][5];
  // row s of a plane (wave order): x and lam in the first half, the weights
  // throughout; ok = false turns the loads into no-ops
  auto load_row = [&](PK (&sl)[5], const wide_rsrc_t (&rb)[5], int s, bool ok) __attribute__((always_inline)) {
    const int so = ok ? line_of(s) * RB : kWideOob;
    if (s < MID) {
      wide_load(sl[0], rb[0], voff, so);
      wide_load(sl[1], rb[1], voff, so);
    }
    if (PRESENT) {
#pragma unroll
      for (int m = 2; m < 5; ++m) wide_load(sl[m], rb[m], voff, so);
    }
  };
  auto preload = [&](const wide_rsrc_t (&rb)[5]) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < R; ++k) load_row(ring[k], rb, k, true);
  };

  float lxr[MID][NP], hr[MID][NP], hv[MID][NP], hp[NP];
  auto first_half = [&](const wide_rsrc_t (&rb)[5]) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < NP; ++q) hp[q] = 0.f;
    static_for<0, MID>([&](auto sc) __attribute__((always_inline)) {
      constexpr int s = decltype(sc)::value, k = s % R;
      float lx[NP], a[NP], b[NP], c[NP];
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        lx[q] = ring[k][1].get(q) * ring[k][0].get(q);
        if (PRESENT) {
          a[q] = ring[k][2].get(q);
          b[q] = ring[k][3].get(q);
          c[q] = ring[k][4].get(q);
        }
      }
      if (PRESENT || s + R < MID) load_row(ring[k], rb, s + R, true);
#pragma unroll
      for (int q = 0; q < NP; ++q) lxr[s][q] = lx[q];
      if (PRESENT) {
        norm_weights<LG, NP>(a, b, c, col, S, rn);
        wide_step<NP>(lx, a, b, c, hp);
#pragma unroll
        for (int q = 0; q < NP; ++q) hr[s][q] = hp[q];
      }
    });
  };
  // rbn: the next plane (has_next), whose first rows the last steps request
  auto second_half = [&](const wide_rsrc_t (&rb)[5], const wide_rsrc_t (&rbn)[5], bool has_next)
                         __attribute__((always_inline)) {
    float la[G][NP];
    auto lds_read = [&](float (&l)[NP], int s) __attribute__((always_inline)) {
      const int o = line_of(s) * P + col;
#pragma unroll
      for (int q = 0; q < NP; ++q) l[q] = lxa[o + q];
    };
#pragma unroll
    for (int g = 0; g < G; ++g) lds_read(la[g], MID + g);
    static_for<MID, S>([&](auto sc) __attribute__((always_inline)) {
      constexpr int s = decltype(sc)::value, k = s % R, gi = (s - MID) % G;
      float lx[NP], a[NP], b[NP], c[NP];
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        lx[q] = la[gi][q];
        a[q] = ring[k][2].get(q);
        b[q] = ring[k][3].get(q);
        c[q] = ring[k][4].get(q);
      }
      if (s + R < S) load_row(ring[k], rb, s + R, true);
      else load_row(ring[k], rbn, s + R - S, has_next);
      if (s + G < S) lds_read(la[gi], s + G);
      norm_weights<LG, NP>(a, b, c, col, S, rn);
      wide_step<NP>(lx, a, b, c, hp);
#pragma unroll
      for (int q = 0; q < NP; ++q) hv[s - MID][q] = hp[q];
    });
  };

  int64_t plane = blockIdx.x;
  wide_rsrc_t rb[5];
  plane_res(plane, rb);
  preload(rb);
  for (;;) {
    first_half(rb);
    const int64_t nxt = plane + gridDim.x;
    const bool has_next = nxt < p.planes;
    wide_rsrc_t rbn[5];
    plane_res(has_next ? nxt : plane, rbn);
    lds_barrier();  // B0: the previous plane's epilogue has read acc
    static_for<0, MID>([&](auto sc) __attribute__((always_inline)) {
      constexpr int s = decltype(sc)::value;
      const int o = line_of(s) * P + col;
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        lxa[o + q] = lxr[s][q];
        acc[o + q] = PRESENT ? hr[s][q] : 0.f;
      }
    });
    lds_barrier();  // B1: lam * x and the first halves are stored
    if (PRESENT) second_half(rb, rbn, has_next);
    lds_barrier();  // B2: the horizontal first halves have added to acc
    if (PRESENT) {
      // in batches whose reads are all issued before their writes
      constexpr int AB = 8;
      static_for<0, MID / AB>([&](auto bc) __attribute__((always_inline)) {
        constexpr int b0 = MID + decltype(bc)::value * AB;
        float t[AB][NP];
        static_for<0, AB>([&](auto jc) __attribute__((always_inline)) {
          constexpr int j = decltype(jc)::value;
          const int o = line_of(b0 + j) * P + col;
#pragma unroll
          for (int q = 0; q < NP; ++q) t[j][q] = acc[o + q];
        });
        static_for<0, AB>([&](auto jc) __attribute__((always_inline)) {
          constexpr int j = decltype(jc)::value;
          const int o = line_of(b0 + j) * P + col;
#pragma unroll
          for (int q = 0; q < NP; ++q) acc[o + q] = t[j][q] + hv[b0 + j - MID][q];
        });
      });
    }
    lds_barrier();  // B3: acc holds everything but the horizontal second halves
    if (!has_next) break;
    plane = nxt;
    static_for<0, 5>([&](auto m) __attribute__((always_inline)) { rb[m] = rbn[m]; });
    if (!PRESENT) preload(rb);
  }
}

// Horizontal role (waves 2 and 3): each lane owns two adjacent rows.  The
// first half of the columns (H1) runs after B1, concurrently with the vertical
// second halves, adding h to acc; the second half (H2) after B3; then the
// wave writes y = u * acc for the columns of its second half (final once its
// own H2 has passed them).  Weights arrive as 128-byte row segments (a line's
// eight 16-byte pieces in consecutive instructions, so it is fetched into the
// L1 once) into two register tiles.  The wave's own loads go where the
// vertical waves are busy with LDS only and the memory is otherwise quiet:
// tile 1 whole while they store their first halves (B0-B1), u for the
// epilogue while they add their second halves (B2-B3); tiles after the
// second are staggered over the current tile's columns, and the next plane's
// first tile follows the last one.
template <typename T, bool REV, bool PRESENT, bool LG>
__device__ __forceinline__ void wide_h_role(const ResFwdParams& p, int slot, float* __restrict__ acc,
                                            const float* __restrict__ lxa, int lane) {
  using C = WideCfg<T>;
  constexpr int S = C::S, NP = C::NP, P = C::P, G = C::G;
  constexpr int VE = C::VE, TH = C::TH, NV = C::NV, NTH = C::NTH;
  constexpr int RB = S * (int)sizeof(T), PB = S * RB;
  constexpr int NL = 3 * NP, GAP = TH / NL;   // row segments per tile, steps between their requests
  constexpr int NU = S / 2;                   // epilogue instructions (two half rows each)
  static_assert(TH % G == 0 && GAP >= 1, "lookahead slots repeat with the tile");
  typedef Pack<T, VE> PK;
  typedef Pack<T, NP> UK;
  const int row0 = lane * NP;
  const bool rn = LG && p.renorm;
  auto tile_so = [](int t) { return (REV ? NTH - 1 - t : t) * TH * (int)sizeof(T); };
  auto plane_res = [&](int64_t plane, wide_rsrc_t (&rw)[3]) __attribute__((always_inline)) {
    const T* w0 = (const T*)p.w + (int64_t)slot * 3 * p.npc + plane * (S * S);
#pragma unroll
    for (int m = 0; m < 3; ++m) rw[m] = wide_rsrc(w0 + m * p.npc, PB);
  };
  // epilogue lanes: lanes 0-31 and 32-63 cover two rows, NP columns each, of
  // this wave's half of the columns
  const int ec = (REV ? 0 : S / 2) + (lane & 31) * NP, erow = lane >> 5;
  const int uvoff = (erow * S + ec) * (int)sizeof(T);

  PK tile[2][3][NP][NV];
  int voff[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) voff[q] = (row0 + q) * RB;
  auto load_seg = [&](PK (&tb)[3][NP][NV], const wide_rsrc_t (&rw)[3], int m, int q, int so)
                      __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int v = REV ? NV - 1 - i : i;  // the order the columns are used
      wide_load(tb[m][q][v], rw[m], voff[q], so + v * VE * (int)sizeof(T));
    }
  };
  auto load_tile0 = [&](const wide_rsrc_t (&rw)[3]) __attribute__((always_inline)) {
#pragma unroll
    for (int m = 0; m < 3; ++m)
#pragma unroll
      for (int q = 0; q < NP; ++q) load_seg(tile[0], rw, m, q, tile_so(0));
  };
  UK ur[NU];
  float hp[NP];
  float la[G][NP], aa[G][NP];

  auto run_tile = [&](auto tc, const wide_rsrc_t (&rw)[3]) __attribute__((always_inline)) {
    constexpr int t = decltype(tc)::value, b = t & 1;
    const int c0 = (REV ? NTH - 1 - t : t) * TH;
    auto lds_read = [&](float (&l)[NP], float (&a)[NP], int e) __attribute__((always_inline)) {
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        l[q] = lxa[(row0 + q) * P + c0 + e];
        a[q] = acc[(row0 + q) * P + c0 + e];
      }
    };
    // lookahead inside the tile only, so it never crosses a barrier
#pragma unroll
    for (int g = 0; g < G; ++g) lds_read(la[g], aa[g], REV ? TH - 1 - g : g);
#pragma unroll
    for (int i = 0; i < TH; ++i) {
      const int e = REV ? TH - 1 - i : i;  // column inside the tile
      const int v = e / VE, el = e % VE, gi = i % G;
      float lx[NP], av[NP], a[NP], bb[NP], c[NP];
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        lx[q] = la[gi][q];
        av[q] = aa[gi][q];
        a[q] = tile[b][0][q][v].get(el);
        bb[q] = tile[b][1][q][v].get(el);
        c[q] = tile[b][2][q][v].get(el);
      }
      // tile 1 was requested whole before B1, u before B3
      if (t >= 1 && t + 1 < NTH) {
        if (i % GAP == 0 && i / GAP < NL) load_seg(tile[1 - b], rw, (i / GAP) / NP, (i / GAP) % NP, tile_so(t + 1));
      }
      if (i + G < TH) lds_read(la[gi], aa[gi], REV ? TH - 1 - (i + G) : i + G);
      norm_weights<LG, NP>(a, bb, c, row0, S, rn);
      wide_step<NP>(lx, a, bb, c, hp);
#pragma unroll
      for (int q = 0; q < NP; ++q) acc[(row0 + q) * P + c0 + e] = av[q] + hp[q];
    }
  };

  int64_t plane = blockIdx.x;
  wide_rsrc_t rw[3];
  if (PRESENT) {
    plane_res(plane, rw);
    load_tile0(rw);
  }
  for (;;) {
    const int64_t pof = plane * (S * S);
    const int64_t nxt = plane + gridDim.x;
    const bool has_next = nxt < p.planes;
    const wide_rsrc_t ru = wide_rsrc((const T*)p.u + pof, PB);
    lds_barrier();  // B0
    // the second tile while the vertical waves store their first halves
    if (PRESENT) {
#pragma unroll
      for (int m = 0; m < 3; ++m)
#pragma unroll
        for (int q = 0; q < NP; ++q) load_seg(tile[1], rw, m, q, tile_so(1));
    }
    lds_barrier();  // B1: lam * x and the vertical first halves are in LDS
#pragma unroll
    for (int q = 0; q < NP; ++q) hp[q] = 0.f;
    if (PRESENT) static_for<0, NTH / 2>([&](auto tc) __attribute__((always_inline)) { run_tile(tc, rw); });
    lds_barrier();  // B2
    // u for the epilogue while the vertical waves add their second halves
#pragma unroll
    for (int r = 0; r < NU; ++r) wide_load(ur[r], ru, uvoff, 2 * r * RB);
    lds_barrier();  // B3: the vertical second halves are added
    if (PRESENT) {
      static_for<NTH / 2, NTH>([&](auto tc) __attribute__((always_inline)) { run_tile(tc, rw); });
      if (has_next) {
        plane_res(nxt, rw);
        load_tile0(rw);
      }
    }
    // y = u * acc over this wave's half of the columns
    // (the reads of a batch of rows are issued before its stores)
    const wide_rsrc_t ry = wide_rsrc((T*)p.y + pof, PB);
    constexpr int EB = 8;
    static_for<0, NU / EB>([&](auto bc) __attribute__((always_inline)) {
      constexpr int r0 = decltype(bc)::value * EB;
      float y[EB][NP];
#pragma unroll
      for (int j = 0; j < EB; ++j)
#pragma unroll
        for (int q = 0; q < NP; ++q) y[j][q] = acc[(2 * (r0 + j) + erow) * P + ec + q];
#pragma unroll
      for (int j = 0; j < EB; ++j) {
#pragma unroll
        for (int q = 0; q < NP; ++q) y[j][q] *= ur[r0 + j].get(q);
        wide_store<T, NP>(y[j], ry, uvoff, 2 * (r0 + j) * RB);
      }
    });
    if (!has_next) break;
    plane = nxt;
  }
}

template <typename T, bool LG>
__global__ void __launch_bounds__(256, 1) wide_fwd_kernel(ResFwdParams p) {
  using C = WideCfg<T>;
  extern __shared__ float lds[];
  float* acc = lds;
  float* lxa = lds + C::ARR;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);  // uniform per wave
  const int slot = p.slot[wave];  // T2B, B2T, L2R, R2L
  switch (wave) {
    case 0:
      if (slot >= 0) wide_v_role<T, false, true, LG>(p, slot, acc, lxa, lane);
      else wide_v_role<T, false, false, LG>(p, slot, acc, lxa, lane);
      break;
    case 1:
      if (slot >= 0) wide_v_role<T, true, true, LG>(p, slot, acc, lxa, lane);
      else wide_v_role<T, true, false, LG>(p, slot, acc, lxa, lane);
      break;
    case 2:
      if (slot >= 0) wide_h_role<T, false, true, LG>(p, slot, acc, lxa, lane);
      else wide_h_role<T, false, false, LG>(p, slot, acc, lxa, lane);
      break;
    default:
      if (slot >= 0) wide_h_role<T, true, true, LG>(p, slot, acc, lxa, lane);
      else wide_h_role<T, true, false, LG>(p, slot, acc, lxa, lane);
      break;
  }
}

// Compute units of the current device (cached per device).
inline int wide_cu_count() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = 0;
  const int slot = dev < 64 ? dev : 63;
  int n = cache[slot].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cache[slot].store(n, std::memory_order_relaxed);
  }
  return n;
}

template <typename T>
hipError_t launch_wide(const ResFwdParams& p, hipStream_t st) {
  using C = WideCfg<T>;
  auto kern = p.logits ? wide_fwd_kernel<T, true> : wide_fwd_kernel<T, false>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_BYTES);
  if (e != hipSuccess) return e;
  const int64_t cus = wide_cu_count();
  const int64_t grid = p.planes < cus ? p.planes : cus;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(C::NT), C::LDS_BYTES, st, p);
  return hipGetLastError();
}

}  // namespace gspn
