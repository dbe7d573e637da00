// Size-specialised resident forward kernel for square S x S planes.
//
// Same decomposition as the generic resident kernel (one workgroup of two
// waves per group of planes; phase V = top-to-bottom and bottom-to-top,
// phase H = left-to-right and right-to-left; sum_d h_d accumulated in fp32 in
// LDS with the midpoint barriers that fix the addition order), but with the
// plane size a compile-time constant:
//   * every global and LDS address of a line is a base register plus an
//     immediate offset, so a line step carries no address arithmetic;
//   * phases of up to 64 lines are fully unrolled (the middle barrier and the
//     padding masks resolve at compile time); 128-line phases run chunks of 64
//     lines whose boundary falls on the middle line;
//   * inputs are prefetched through a register ring of R tiles (a tile is one
//     row for vertical scans, a row segment of THZ columns for horizontal ones);
//   * accumulator values are read G lines ahead of their update, never across
//     the middle barrier, so LDS latency stays off the critical path.
#pragma once

#include "gspn_device.hpp"
#include "gspn_launch.hpp"
#include "gspn_resident_impl.hpp"

namespace gspn {

template <typename T, int S>
struct FixedCfg {
  static constexpr int NP = S <= 64 ? 1 : (S <= 128 ? 2 : 4);  // positions per lane
  static constexpr int SEG = S <= 15 ? 16 : (S <= 31 ? 32 : 64); // lanes per plane
  static constexpr int PPW = 64 / SEG;                           // planes per wave
  static constexpr int P = S + 1;                                // LDS pitch (odd)
  static constexpr int ROWS = S + 1;                             // + padding row
  static constexpr int MID = S / 2;
  static constexpr bool FULL = S <= 64;                          // fully unrolled phases
  static constexpr int CHUNK = FULL ? S : 64;                    // lines per loop iteration
  // horizontal vector: largest of 16/8/4 bytes whose element count divides S
  static constexpr int VLH = (S % (16 / (int)sizeof(T)) == 0) ? 16 / (int)sizeof(T)
                           : (S % (8 / (int)sizeof(T)) == 0 ? 8 / (int)sizeof(T) : 4 / (int)sizeof(T));
  // horizontal tile: lines per row segment.  Long planes read 128-byte row
  // segments (eight 16-byte vectors back to back, one tile in flight) so every
  // cache line fetched for a row is consumed by the same load; shorter segments
  // let the line be evicted before its neighbours are read and fetch it again.
  static constexpr int THZ = FULL ? VLH : 128 / (int)sizeof(T);
  static constexpr int RV = FULL ? (S % 8 == 0 ? 8 : 7) : 8;     // vertical ring (lines)
  static constexpr int RH = FULL ? 6 : 1;                         // horizontal ring (tiles)
  static constexpr int G = 4;                                     // accumulator lookahead
  static constexpr bool ALL_VALID = (S == SEG * NP);
  static constexpr int LDS_BYTES = PPW * ROWS * P * 4;
  static_assert(S % 2 == 0, "fixed kernel takes even sizes");
  static_assert(FULL || (MID % CHUNK == 0), "chunk boundary must fall on the middle line");
};

// One direction's scan over a phase.  HZ: lines are columns.  REV: lines are
// visited from S-1 down to 0.  pbase[m]: plane base of map m (x, lam, w0..w2).
template <typename T, int S, bool HZ, bool REV>
__device__ __forceinline__ void fixed_phase(const T* const (&pbase)[5], float* __restrict__ acc,
                                            int sl) {
  using C = FixedCfg<T, S>;
  constexpr int NP = C::NP;
  constexpr int TL = HZ ? C::THZ : 1;   // lines per tile
  constexpr int R = HZ ? C::RH : C::RV; // tiles in flight
  constexpr int NT = S / TL;            // tiles per phase
  constexpr int CT = C::CHUNK / TL;     // tiles per chunk
  static_assert(S % TL == 0, "tile must divide the line count");
  static_assert(C::FULL || CT % R == 0, "ring slots must repeat per chunk");
  typedef Pack<T, HZ ? TL : NP> PK;

  const int pos0 = sl * NP;
  bool valid[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) valid[q] = C::ALL_VALID || pos0 + q < S;
  // per-lane element offsets inside a plane (clamped into the plane for padding lanes)
  int eoff[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    const int pos = valid[q] ? pos0 + q : 0;
    eoff[q] = HZ ? pos * S : pos;
  }
  // LDS element offset of (line 0, position q); padding lanes use the padding row/column
  int aoff[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) aoff[q] = valid[q] ? (HZ ? (pos0 + q) * C::P : pos0 + q) : (HZ ? S * C::P : S);

  // tile ti (scan order) -> first memory line of the tile
  auto tile_line = [](int ti) { return REV ? (NT - 1 - ti) * TL : ti * TL; };
  // scan step s -> line
  auto line_of = [](int s) { return REV ? S - 1 - s : s; };
  // LDS offset of line `line` relative to aoff
  auto lds_line = [](int line) { return HZ ? line : line * C::P; };

  PK ring[R][5][HZ ? NP : 1];
  auto load_tile = [&](PK (&slot)[5][HZ ? NP : 1], int ti) {
    const int l = tile_line(ti < NT ? ti : NT - 1);
#pragma unroll
    for (int m = 0; m < 5; ++m) {
      if constexpr (HZ) {
#pragma unroll
        for (int q = 0; q < NP; ++q) slot[m][q].load(pbase[m] + eoff[q] + l);
      } else {
        slot[m][0].load(pbase[m] + eoff[0] + l * S);
      }
    }
  };

  float hp[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) hp[q] = 0.f;
  // accumulator lookahead buffer: value of acc at the line G steps ahead
  float av[C::G][NP];

#pragma unroll
  for (int k = 0; k < R; ++k) load_tile(ring[k], k);

  auto acc_read = [&](float (&dst)[NP], int s) {
#pragma unroll
    for (int q = 0; q < NP; ++q) dst[q] = acc[aoff[q] + lds_line(line_of(s))];
  };

  // Process tiles [c*CT, c*CT + CT) of the phase; `c` may be a runtime chunk index.
  auto run_chunk = [&](int c) {
    const int s_base = c * C::CHUNK;
    // acc lookahead: first G lines of the chunk (after any barrier at its start)
#pragma unroll
    for (int g = 0; g < C::G; ++g) acc_read(av[g], s_base + g);
#pragma unroll
    for (int k = 0; k < CT; ++k) {
      const int ti = c * CT + k;
      const int slot = k % R;
      // vertical tiles are one line: unpack and refill the slot at once; horizontal
      // tiles are unpacked line by line and the slot is refilled after its last line
      float v1[5][NP];
      if constexpr (!HZ) {
#pragma unroll
        for (int m = 0; m < 5; ++m)
#pragma unroll
          for (int q = 0; q < NP; ++q) v1[m][q] = ring[slot][m][0].get(q);
        load_tile(ring[slot], ti + R);  // clamped to the last tile past the end
      }
#pragma unroll
      for (int ee = 0; ee < TL; ++ee) {
        const int e = REV ? TL - 1 - ee : ee;  // memory order inside the tile
        const int kk = k * TL + ee;            // step inside the chunk
        const int s = s_base + kk;             // step inside the phase
        float v[5][NP];
#pragma unroll
        for (int m = 0; m < 5; ++m)
#pragma unroll
          for (int q = 0; q < NP; ++q) v[m][q] = HZ ? ring[slot][m][q].get(e) : v1[m][q];
        line_step<NP>(v[0], v[1], v[2], v[3], v[4], valid, hp);
        const int gi = kk % C::G;
        const int line = line_of(s);
        if (C::FULL && s == C::MID) {
          // middle of a fully unrolled phase: the other wave's first half is done
          lds_barrier();
#pragma unroll
          for (int q = 0; q < NP; ++q) acc[aoff[q] + lds_line(line)] += hp[q];
          // lookahead restarts after the barrier
#pragma unroll
          for (int g = 1; g <= C::G; ++g)
            if (s + g < S) {
              float t[NP];
              acc_read(t, s + g);
#pragma unroll
              for (int q = 0; q < NP; ++q) av[(kk + g) % C::G][q] = t[q];
            }
        } else {
#pragma unroll
          for (int q = 0; q < NP; ++q) acc[aoff[q] + lds_line(line)] = av[gi][q] + hp[q];
          // read G lines ahead unless that crosses the middle barrier or the chunk end
          const int sn = s + C::G;
          const bool cross = C::FULL ? (s < C::MID && sn >= C::MID) : false;
          if (kk + C::G < C::CHUNK && sn < S && !cross) acc_read(av[gi], sn);
        }
      }
      if constexpr (HZ) load_tile(ring[slot], ti + R);
    }
  };

  if constexpr (C::FULL) {
    run_chunk(0);
  } else {
    constexpr int NCH = S / C::CHUNK;
    for (int c = 0; c < NCH; ++c) {
      if (c == NCH / 2) lds_barrier();  // middle of the phase
      run_chunk(c);
    }
  }
}

template <typename T, int S>
__global__ void __launch_bounds__(128, (FixedCfg<T, S>::SEG < 64 ? 4 : (FixedCfg<T, S>::NP > 1 ? 1 : 2)))
fixed_fwd_kernel(ResFwdParams p) {
  using C = FixedCfg<T, S>;
  constexpr int PPW = C::PPW;
  constexpr int HW = S * S;
  constexpr int ACC = C::ROWS * C::P;
  extern __shared__ float lds[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t g0 = (int64_t)blockIdx.x * PPW;
  const int seg = lane / C::SEG, sl = lane % C::SEG;
  const int64_t plane = (g0 + seg < p.planes) ? g0 + seg : p.planes - 1;

  for (int e = tid; e < PPW * ACC; e += 128) lds[e] = 0.f;
  __syncthreads();
  float* acc = lds + seg * ACC;

#pragma unroll
  for (int ph = 0; ph < 2; ++ph) {
    const int slot = p.slot[ph * 2 + wave];
    if (slot < 0) {
      lds_barrier();  // keep the middle barrier of the phase in step
    } else {
      const T* w0 = (const T*)p.w + (int64_t)slot * 3 * p.npc + plane * HW;
      const T* pb[5] = {(const T*)p.x + plane * HW, (const T*)p.lam + plane * HW, w0, w0 + p.npc,
                        w0 + 2 * p.npc};
      if (ph == 0) {
        if (wave == 0) fixed_phase<T, S, false, false>(pb, acc, sl);
        else fixed_phase<T, S, false, true>(pb, acc, sl);
      } else {
        if (wave == 0) fixed_phase<T, S, true, false>(pb, acc, sl);
        else fixed_phase<T, S, true, true>(pb, acc, sl);
      }
    }
    __syncthreads();
  }

  for (int pl = 0; pl < PPW; ++pl) {
    const int64_t pi = g0 + pl;
    if (pi >= p.planes) break;
    const T* ub = (const T*)p.u + pi * HW;
    T* yb = (T*)p.y + pi * HW;
    const float* ac = lds + pl * ACC;
    if (p.vec_y == 2) epilogue<T, 16 / sizeof(T)>(ub, yb, ac, S, S, C::P, tid);
    else if (p.vec_y == 1) epilogue<T, 8 / sizeof(T)>(ub, yb, ac, S, S, C::P, tid);
    else epilogue<T, 1>(ub, yb, ac, S, S, C::P, tid);
  }
}

// Sizes with a specialised kernel (square planes).
inline bool fixed_size_supported(int H, int W) {
  return H == W && (H == 16 || H == 28 || H == 32 || H == 56 || H == 64 || H == 128);
}

template <typename T, int S>
hipError_t launch_fixed(const ResFwdParams& p, hipStream_t st) {
  using C = FixedCfg<T, S>;
  auto kern = fixed_fwd_kernel<T, S>;
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
