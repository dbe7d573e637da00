// Persistent forward kernel for 128 x 128 planes.
//
// One workgroup of two waves per compute unit walks its share of the planes
// one plane at a time, so a batch of planes costs ceil(planes / CUs) plane
// times with no partly filled last round.  LDS holds two fp32 arrays of the
// plane (row pitch 129): the accumulator of sum_d h_d, and lam * x.  Every
// input element is read from HBM exactly once:
//
//   phase V  wave 0 scans top-to-bottom, wave 1 bottom-to-top, each lane
//            owning two adjacent columns.  In the first half of the phase a
//            wave reads x, lam and its three weights for the rows it reaches
//            first, stores lam * x and its h (a plain store: nothing was there
//            before); after the middle barrier it reads only its weights and
//            takes lam * x of the other half, and the accumulator, from LDS.
//   phase H  wave 0 scans left-to-right, wave 1 right-to-left, each lane
//            owning two adjacent rows.  Weights arrive as 128-byte row
//            segments (whole cache lines) into two register tiles, the next
//            tile's segments staggered over the current tile's columns;
//            lam * x and the accumulator come from LDS.
//   epilogue y = u * acc, whole rows per store; u is requested during the
//            last horizontal tile.
//
// The order of the additions is the one of the resident kernels: in each
// phase the first half's direction adds before the second half's, and the
// vertical pair before the horizontal pair.  A direction absent from the mask
// costs nothing but its barriers (in phase V its wave still stores lam * x
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
  static constexpr int LDS_BYTES = 2 * ARR * 4;
  static_assert(MID % RV == 0 && MID % TH == 0, "ring and tiles must align with the middle line");
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

// Phase V for one wave.  PRESENT: the direction is in the mask.  rb: plane
// resources of x, lam, w0, w1, w2.  The steps run as a loop over ring turns
// (R rows per iteration): straight-line code for all rows would not fit the
// instruction cache.
template <typename T, bool REV, bool PRESENT>
__device__ __forceinline__ void wide_v(const wide_rsrc_t (&rb)[5], float* __restrict__ acc, float* __restrict__ lxa,
                                       int lane) {
  using C = WideCfg<T>;
  constexpr int S = C::S, NP = C::NP, P = C::P, MID = C::MID, R = C::RV, G = C::G;
  static_assert(R % G == 0 && MID % R == 0, "lookahead slots repeat with the ring");
  typedef Pack<T, NP> PK;
  const int col = lane * NP;
  const int voff = col * (int)sizeof(T);
  auto line_of = [](int s) { return REV ? S - 1 - s : s; };
  auto row_off = [&](int s, int lim) { return s < lim ? line_of(s) * S * (int)sizeof(T) : kWideOob; };

  // ring of R rows: x, lam (first half only) and the three weights
  PK ring[R][5];
  auto load_row = [&](PK (&slot)[5], int s, bool xl) __attribute__((always_inline)) {
    if (xl) {
      const int so = row_off(s, MID);
      wide_load(slot[0], rb[0], voff, so);
      wide_load(slot[1], rb[1], voff, so);
    }
    if (PRESENT) {
      const int so = row_off(s, S);
#pragma unroll
      for (int m = 2; m < 5; ++m) wide_load(slot[m], rb[m], voff, so);
    }
  };
#pragma unroll
  for (int k = 0; k < R; ++k) load_row(ring[k], k, true);

  float hp[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) hp[q] = 0.f;

  // first half: rows this wave reaches first; lam * x and h are stored
  for (int it = 0; it < MID / R; ++it) {
#pragma unroll
    for (int k = 0; k < R; ++k) {
      const int s = it * R + k;
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
      load_row(ring[k], s + R, true);
      float* la = lxa + line_of(s) * P + col;
      float* ac = acc + line_of(s) * P + col;
#pragma unroll
      for (int q = 0; q < NP; ++q) la[q] = lx[q];
      if (PRESENT) {
        wide_step<NP>(lx, a, b, c, hp);
#pragma unroll
        for (int q = 0; q < NP; ++q) ac[q] = hp[q];
      } else {
#pragma unroll
        for (int q = 0; q < NP; ++q) ac[q] = 0.f;
      }
    }
  }
  lds_barrier();  // middle: the other wave's first-half rows are stored
  if (!PRESENT) return;

  // second half: lam * x and the accumulator from LDS, read G rows ahead
  // (clamped to the last row at the end of the phase)
  float la[G][NP], aa[G][NP];
  auto lds_read = [&](float (&l)[NP], float (&a)[NP], int s) __attribute__((always_inline)) {
    const int o = line_of(s < S ? s : S - 1) * P + col;
#pragma unroll
    for (int q = 0; q < NP; ++q) {
      l[q] = lxa[o + q];
      a[q] = acc[o + q];
    }
  };
#pragma unroll
  for (int g = 0; g < G; ++g) lds_read(la[g], aa[g], MID + g);
  for (int it = MID / R; it < S / R; ++it) {
#pragma unroll
    for (int k = 0; k < R; ++k) {
      const int s = it * R + k, gi = k % G;
      float lx[NP], av[NP], a[NP], b[NP], c[NP];
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        lx[q] = la[gi][q];
        av[q] = aa[gi][q];
        a[q] = ring[k][2].get(q);
        b[q] = ring[k][3].get(q);
        c[q] = ring[k][4].get(q);
      }
      load_row(ring[k], s + R, false);
      lds_read(la[gi], aa[gi], s + G);
      wide_step<NP>(lx, a, b, c, hp);
      float* ac = acc + line_of(s) * P + col;
#pragma unroll
      for (int q = 0; q < NP; ++q) ac[q] = av[q] + hp[q];
    }
  }
}

// Phase H for one wave (the direction is present).  rw: plane resources of
// w0..w2.  Two register tiles: tile t is consumed from one while tile t + 1
// arrives in the other, requested as whole 128-byte row segments (a line's
// eight 16-byte pieces in consecutive instructions, so it is fetched into the
// L1 once) and staggered over tile t's columns, which keeps a steady stream
// of loads under the arithmetic.  During the last tile the wave requests its
// epilogue rows of u instead (ru; into ur).
template <typename T, bool REV>
__device__ __forceinline__ void wide_h(const wide_rsrc_t (&rw)[3], float* __restrict__ acc,
                                       const float* __restrict__ lxa, int lane, int wave, wide_rsrc_t ru,
                                       Pack<T, WideCfg<T>::NP> (&ur)[WideCfg<T>::S / 2]) {
  using C = WideCfg<T>;
  constexpr int S = C::S, NP = C::NP, P = C::P, G = C::G;
  constexpr int VE = C::VE, TH = C::TH, NV = C::NV, NTH = C::NTH;
  constexpr int NL = 3 * NP, GAP = TH / NL;  // row segments per tile, steps between their requests
  constexpr int UPS = (S / 2 + TH - 1) / TH;  // u rows requested per step of the last tile
  static_assert(TH % G == 0 && GAP >= 1, "lookahead slots repeat with the tile");
  typedef Pack<T, VE> PK;
  const int row0 = lane * NP;
  auto tile_so = [](int t) { return (REV ? NTH - 1 - t : t) * TH * (int)sizeof(T); };

  PK tile[2][3][NP][NV];
  int voff[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) voff[q] = (row0 + q) * S * (int)sizeof(T);
  auto load_seg = [&](PK (&tb)[3][NP][NV], int m, int q, int so) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int v = REV ? NV - 1 - i : i;  // the order the columns are used
      wide_load(tb[m][q][v], rw[m], voff[q], so + v * VE * (int)sizeof(T));
    }
  };
#pragma unroll
  for (int m = 0; m < 3; ++m)
#pragma unroll
    for (int q = 0; q < NP; ++q) load_seg(tile[0], m, q, tile_so(0));

  const int uvoff = lane * NP * (int)sizeof(T);
  float hp[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) hp[q] = 0.f;
  float la[G][NP], aa[G][NP];

#pragma unroll
  for (int t = 0; t < NTH; ++t) {
    const int b = t & 1;
    if (t == NTH / 2) lds_barrier();  // middle: the other wave's first-half additions are done
    const int c0 = (REV ? NTH - 1 - t : t) * TH;
    auto lds_read = [&](float (&l)[NP], float (&a)[NP], int e) __attribute__((always_inline)) {
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        l[q] = lxa[(row0 + q) * P + c0 + e];
        a[q] = acc[(row0 + q) * P + c0 + e];
      }
    };
    // lookahead inside the tile only, so it never crosses the middle barrier
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
      if (t + 1 < NTH) {
        if (i % GAP == 0 && i / GAP < NL) load_seg(tile[1 - b], (i / GAP) / NP, (i / GAP) % NP, tile_so(t + 1));
      } else {
#pragma unroll
        for (int k = 0; k < UPS; ++k) {
          const int r = i * UPS + k;
          if (r < S / 2) wide_load(ur[r], ru, uvoff, (wave * (S / 2) + r) * S * (int)sizeof(T));
        }
      }
      if (i + G < TH) lds_read(la[gi], aa[gi], REV ? TH - 1 - (i + G) : i + G);
      wide_step<NP>(lx, a, bb, c, hp);
#pragma unroll
      for (int q = 0; q < NP; ++q) acc[(row0 + q) * P + c0 + e] = av[q] + hp[q];
    }
  }
}

// y = u * acc: wave w writes rows [64 w, 64 w + 64), each lane two adjacent
// columns of a row (whole-row stores, LDS reads without conflicts beyond
// two-way); u of those rows is already in registers (ur).
template <typename T>
__device__ __forceinline__ void wide_epilogue(const Pack<T, WideCfg<T>::NP> (&ur)[WideCfg<T>::S / 2], wide_rsrc_t ry,
                                              const float* __restrict__ acc, int lane, int wave) {
  using C = WideCfg<T>;
  constexpr int S = C::S, NP = C::NP, P = C::P;
  const int col = lane * NP, voff = col * (int)sizeof(T);
#pragma unroll
  for (int r = 0; r < S / 2; ++r) {
    const int row = wave * (S / 2) + r;
    float y[NP];
#pragma unroll
    for (int q = 0; q < NP; ++q) y[q] = ur[r].get(q) * acc[row * P + col + q];
    wide_store<T, NP>(y, ry, voff, row * S * (int)sizeof(T));
  }
}

template <typename T>
__global__ void __launch_bounds__(128, 1) wide_fwd_kernel(ResFwdParams p) {
  using C = WideCfg<T>;
  constexpr int S = C::S, HW = S * S, PB = HW * (int)sizeof(T);  // bytes of one plane of a map
  extern __shared__ float lds[];
  float* acc = lds;
  float* lxa = lds + C::ARR;

  for (int64_t plane = blockIdx.x; plane < p.planes; plane += gridDim.x) {
    // lane-dependent offsets are rebuilt in every iteration: hoisting the
    // unrolled loops' addresses out of the plane loop would exhaust the VGPRs
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);  // uniform per wave
    const int64_t pof = plane * HW;
    // phase V: wave 0 top-to-bottom, wave 1 bottom-to-top
    {
      const int slot = p.slot[wave];
      const T* w0 = (const T*)p.w + (int64_t)(slot < 0 ? 0 : slot) * 3 * p.npc + pof;
      const wide_rsrc_t rb[5] = {wide_rsrc((const T*)p.x + pof, PB), wide_rsrc((const T*)p.lam + pof, PB),
                                 wide_rsrc(w0, PB), wide_rsrc(w0 + p.npc, PB), wide_rsrc(w0 + 2 * p.npc, PB)};
      if (wave == 0) {
        if (slot >= 0) wide_v<T, false, true>(rb, acc, lxa, lane);
        else wide_v<T, false, false>(rb, acc, lxa, lane);
      } else {
        if (slot >= 0) wide_v<T, true, true>(rb, acc, lxa, lane);
        else wide_v<T, true, false>(rb, acc, lxa, lane);
      }
    }
    __syncthreads();
    // phase H: wave 0 left-to-right, wave 1 right-to-left; each wave's rows of
    // u for the epilogue arrive during its last tile
    const wide_rsrc_t ru = wide_rsrc((const T*)p.u + pof, PB);
    Pack<T, C::NP> ur[S / 2];
    {
      const int slot = p.slot[2 + wave];
      if (slot < 0) {
        const int uvoff = lane * C::NP * (int)sizeof(T);
#pragma unroll
        for (int r = 0; r < S / 2; ++r) wide_load(ur[r], ru, uvoff, (wave * (S / 2) + r) * S * (int)sizeof(T));
        lds_barrier();  // the middle barrier of the phase
      } else {
        const T* w0 = (const T*)p.w + (int64_t)slot * 3 * p.npc + pof;
        const wide_rsrc_t rw[3] = {wide_rsrc(w0, PB), wide_rsrc(w0 + p.npc, PB), wide_rsrc(w0 + 2 * p.npc, PB)};
        if (wave == 0) wide_h<T, false>(rw, acc, lxa, lane, wave, ru, ur);
        else wide_h<T, true>(rw, acc, lxa, lane, wave, ru, ur);
      }
    }
    __syncthreads();
    wide_epilogue<T>(ur, wide_rsrc((T*)p.y + pof, PB), acc, lane, wave);
    __syncthreads();  // the next plane overwrites both arrays
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
  auto kern = wide_fwd_kernel<T>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_BYTES);
  if (e != hipSuccess) return e;
  const int64_t cus = wide_cu_count();
  const int64_t grid = p.planes < cus ? p.planes : cus;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(128), C::LDS_BYTES, st, p);
  return hipGetLastError();
}

}  // namespace gspn
