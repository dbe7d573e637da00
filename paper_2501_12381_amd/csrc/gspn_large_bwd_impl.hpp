// Two-pass backward for planes too large to keep on chip (e.g. 2048 x 2048):
// the exact adjoint of Eq. 1-2 in launch sequences that each stream the plane
// once, with fp32 h and g sums in the workspace.
//
// Horizontal directions, one at a time, over blocks of K columns (K = 128
// bytes of a row, the block of the forward's pass H):
//   recompute  large_hrec_kernel (pass H in its `rec` mode), blocks in scan order: h of
//              the direction into an fp32 plane `hbuf`, and hsum (+)= h.
//   adjoint    large_hadj_kernel, blocks in reverse scan order.  A workgroup
//              owns a band of rows plus a halo of K rows towards each
//              neighbouring band (one row per lane), as in the forward:
//              starting from the exact
//              products of the column after the block (carried between
//              launches in a small workspace), the transposed stencil
//                g[l][p] = u dy[l][p] + w0[n][p+1] g[n][p+1] + w1[n][p] g[n][p]
//                          + w2[n][p-1] g[n][p-1]          (n: the next line)
//              leaves the band exact after K columns.  The band's rows of the
//              block's h (and one row above and below) sit in LDS;
//                dw_k[l][p] = g[l][p] h[prev][p+k-1]
//              is formed per step in registers and stored as 128-byte row
//              segments; g replaces the h column that no later step reads and
//              is added to gsum with coalesced accesses at the end.  The row
//              segments of dy, u and the three weight maps come in as one
//              register tile per launch; the dw words are produced as the tile
//              words die, so the two share the register budget.
// Vertical directions, both at once:
//   recompute  large_vrec_kernel, the forward's vertical pass (one workgroup
//              per direction and plane) storing each direction's h in its own
//              fp32 plane.
//   adjoint    large_vadj_kernel: one workgroup per plane, top-to-bottom's
//              adjoint walking up and bottom-to-top's walking down, meeting at
//              the middle row; rows stream through register rings.
// The gradient finish then forms dx = lam gsum, dlam = x gsum and
// du = dy (hsum + h_t2b + h_b2t).
#pragma once

#include "gspn_large_impl.hpp"

namespace gspn {

struct LargeHAdjParams {
  const void* dy;
  const void* u;
  const void* w;       // this direction's w0 (w1, w2 at +npc, +2 npc)
  void* dw;            // this direction's dw0 (dw1, dw2 at +npc, +2 npc)
  const float* hbuf;   // h of this direction (fp32)
  float* gsum;         // fp32 running sum of g over the directions
  float* state;        // [2 parities][3][planes * H]: w_k * g of the last column done
  int64_t planes, npc;
  int H, W;
  int first;           // store gsum instead of adding
  int step, nblk;
  int band_rows, edge_rows, nbands, halo;  // bands as in the forward's pass H
  // bit i: window column i takes nothing from the next line (that line starts
  // a group); bit i of gmask: window column i starts a group (zero previous state)
  uint64_t zmask, gmask;
  int renorm;          // Eq. 6 logits (LG kernels): normalise over on-line neighbours only
};

// DIR 0: left-to-right (its adjoint walks the blocks and columns right to left);
// DIR 1: right-to-left (adjoint left to right).  LG: the weight maps hold
// Eq. 6 logits; dw becomes their gradient.
// b / G: the workgroup's index among the G workgroups of this direction.
template <typename T, int NW, int DIR, bool LG>
__device__ __forceinline__ void large_hadj_body(const LargeHAdjParams& p, int64_t b, int64_t G) {
  using C = LargeCfg<T>;
  constexpr int K = C::KH, HV = C::HV, VE = C::VE;
  constexpr int HC = K + 4;           // h columns in LDS: the window and 4 on its scan-previous side
  constexpr int HP = HC + 1;          // LDS pitch (odd: column accesses hit distinct banks)
  constexpr int HOFF = DIR ? 0 : 4;   // LDS column of window column 0
  constexpr int PREV = DIR ? 1 : -1;  // window offset of the scan-previous column
  typedef Pack<T, VE> PK;
  // [edge_rows + 2][HP]; edges [2 parities][NW + 2][2] (wave w at slot w + 1,
  // zeros at slots 0 and NW + 1); 64 dummy slots
  extern __shared__ float lds[];
  float* edge = lds + (p.edge_rows + 2) * HP;
  constexpr int ES = (NW + 2) * 2;

  if (p.step < 0 || p.step >= p.nblk) return;  // this direction has no block in the launch
  // workgroup -> (plane, band); the bands of a plane share an XCD
  const int64_t G8 = G / 8 * 8;
  const int64_t id = b < G8 ? (b % 8) * (G8 / 8) + b / 8 : b;
  const int band = (int)(id % p.nbands);
  const int64_t plane = id / p.nbands;
  const int blk = DIR ? p.step : p.nblk - 1 - p.step;
  const int H = p.H, W = p.W;
  const int c0 = blk * K;
  const int ws = c0 + K <= W ? c0 : W - K;
  const int lo = c0 - ws;  // first window column of this block

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // kept rows [bs, be); halo rows only towards a neighbouring band
  const bool last = band == p.nbands - 1;
  const int bs = band == 0 ? 0 : p.edge_rows + (band - 1) * p.band_rows;
  const int be = last ? H : min(H, bs + (band == 0 ? p.edge_rows : p.band_rows));
  const int htop = band == 0 ? 0 : p.halo;
  const int used = be - bs + htop + (last ? 0 : p.halo);
  const int r = bs - htop + (tid < used ? tid : used - 1);
  const bool row_ok = tid < used && r >= 0 && r < H;
  const int rc = r < 0 ? 0 : (r >= H ? H - 1 : r);
  const int br = r - bs;
  const bool in_band = row_ok && br >= 0 && br < be - bs;
  const int rows = be - bs;

  const int64_t HW = (int64_t)H * W;
  const int64_t rb = plane * HW + (int64_t)rc * W + ws;
  const T* wb = (const T*)p.w;
  const T* base[5] = {(const T*)p.dy + rb, (const T*)p.u + rb, wb + rb, wb + p.npc + rb, wb + 2 * p.npc + rb};

  // the register tile: dy, u, w0, w1, w2 of the lane's row over the window,
  // map by map, each row segment's vectors back to back
  PK tile[5][HV];
#pragma unroll
  for (int m = 0; m < 5; ++m) {
#pragma unroll
    for (int i = 0; i < HV; ++i) tile[m][i].load(base[m] + i * VE);
    __builtin_amdgcn_sched_barrier(0);
  }
  // h of the band rows and one row on each side, window columns shifted by
  // HOFF, into LDS (zero outside the plane)
  {
    constexpr int NV = HC / 4;  // float4 vectors per LDS row
    const int nrow = rows + 2;
    const int nvec = nrow * NV;
    const int r0 = bs - 1;
    const int cb = ws - HOFF;
    const float* hp0 = p.hbuf + plane * HW;
    constexpr int TT = 64 * NW, UB = 4;
    for (int e0 = tid; e0 < nvec; e0 += TT * UB) {
      float4 v[UB];
#pragma unroll
      for (int k = 0; k < UB; ++k) {
        const int e = e0 + k * TT;
        const int rr = e / NV, cv = e - rr * NV;
        const int gr = r0 + rr, gc = cb + cv * 4;
        const bool ok = e < nvec && gr >= 0 && gr < H && gc >= 0 && gc < W;
        v[k] = ok ? *reinterpret_cast<const float4*>(hp0 + (int64_t)gr * W + gc) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int k = 0; k < UB; ++k) {
        const int e = e0 + k * TT;
        if (e < nvec) {
          const int rr = e / NV, cv = e - rr * NV;
          float* d = lds + rr * HP + cv * 4;
          d[0] = v[k].x; d[1] = v[k].y; d[2] = v[k].z; d[3] = v[k].w;
        }
      }
    }
  }

  // products of the column after the block (scan order), from the previous launch
  float a0 = 0.f, a1 = 0.f, a2 = 0.f;
  const int64_t sp = plane * H;
  const int64_t sst = p.planes * H;
  if (p.step > 0) {
    const float* sin = p.state + (int64_t)((p.step - 1) & 1) * 3 * sst + sp + rc;
    a0 = sin[0];
    a1 = sin[sst];
    a2 = sin[2 * sst];
  }
  if (!row_ok) a0 = a1 = a2 = 0.f;
  // wave edges: lane 0 publishes its a0 (row above it reads it), lane 63 its a2
  if (lane == 0) edge[ES + (wave + 1) * 2 + 0] = a0;
  if (lane == 63) edge[ES + (wave + 1) * 2 + 1] = a2;
  if (tid < 8) edge[((tid >> 2) & 1) * ES + ((tid >> 1) & 1) * ((NW + 1) * 2) + (tid & 1)] = 0.f;  // zero slots
  auto eslot = [&](int par) {
    return lane == 0 ? par * ES + (wave + 1) * 2 : (lane == 63 ? par * ES + (wave + 1) * 2 + 1 : 2 * ES + lane);
  };
  const int eo0 = eslot(0), eo1 = eslot(1);
  float* hrow = lds + (in_band ? br + 1 : 1) * HP;  // this row's h (then g) in LDS

  // dw words: bf16 pairs (or fp32) per map and column, filled as the steps go
  constexpr int DWW = PK::kWords * HV;
  uint32_t dwv[3][DWW];
  float pend[3] = {0.f, 0.f, 0.f};
  const uint64_t zm = p.zmask, gm = p.gmask;
  lds_barrier();  // h and the initial edges are in LDS

  auto step = [&](auto ic) __attribute__((always_inline)) {
    constexpr int i = decltype(ic)::value;
    constexpr int ti = DIR ? i : K - 1 - i;  // window column of this step
    if (ti < lo) return;                     // columns of the next block (uniform)
    const int par = i & 1;
    const bool zr = (zm >> ti) & 1;
    // products from the adjacent waves (zero slots past the first and last)
    float nd = 0.f, nu = 0.f;
    if constexpr (NW > 1) {
      nd = edge[(par ^ 1) * ES + (wave + 2) * 2 + 0];
      nu = edge[(par ^ 1) * ES + wave * 2 + 1];
    }
    const float an = from_next_lane_or(a0, nd), ap = from_prev_lane_or(a2, nu);
    float gin = a1 + an + ap;
    gin = zr ? 0.f : gin;
    const float dyv = tile[0][ti / VE].get(ti % VE), uv = tile[1][ti / VE].get(ti % VE);
    float g = fmaf(uv, dyv, gin);
    g = row_ok ? g : 0.f;
    float wa = tile[2][ti / VE].get(ti % VE), wb = tile[3][ti / VE].get(ti % VE), wc = tile[4][ti / VE].get(ti % VE);
    Norm3 nr;
    if constexpr (LG) {
      nr = normalize3(wa, wb, wc, r == 0, r == H - 1, p.renorm != 0);
      wa = nr.w[0];
      wb = nr.w[1];
      wc = nr.w[2];
    }
    a0 = wa * g;
    a1 = wb * g;
    a2 = wc * g;
    edge[par ? eo1 : eo0] = lane == 0 ? a0 : a2;
    // dw from the previous column's h on rows p-1, p, p+1 (zero at a group start)
    const bool gr = (gm >> ti) & 1;
    const int hc = ti + HOFF + PREV;
    const float hl = gr ? 0.f : hrow[hc - HP], hm = gr ? 0.f : hrow[hc], hr = gr ? 0.f : hrow[hc + HP];
    float d0 = g * hl, d1 = g * hm, d2 = g * hr;
    if constexpr (LG) norm3_vjp(nr, d0, d1, d2);
    if constexpr (sizeof(T) == 2) {
      // a word holds columns 2j (low half) and 2j + 1; the second one done completes it
      constexpr bool second = DIR ? (ti & 1) : !(ti & 1);
      if constexpr (!second) {
        pend[0] = d0; pend[1] = d1; pend[2] = d2;
      } else {
        constexpr int wi = ti / 2;
        if constexpr (DIR) {
          dwv[0][wi] = pack_bf2(pend[0], d0); dwv[1][wi] = pack_bf2(pend[1], d1); dwv[2][wi] = pack_bf2(pend[2], d2);
        } else {
          dwv[0][wi] = pack_bf2(d0, pend[0]); dwv[1][wi] = pack_bf2(d1, pend[1]); dwv[2][wi] = pack_bf2(d2, pend[2]);
        }
      }
    } else {
      dwv[0][ti] = __float_as_uint(d0); dwv[1][ti] = __float_as_uint(d1); dwv[2][ti] = __float_as_uint(d2);
    }
    if (in_band) hrow[ti + HOFF] = g;  // h of this column is read by no later step
    lds_barrier();
  };
  static_for<0, K>([&](auto ic) __attribute__((always_inline)) { step(ic); });

  // products of the last column for the next launch (band rows cover the plane)
  if (in_band) {
    float* so = p.state + (int64_t)(p.step & 1) * 3 * sst + sp + r;
    so[0] = a0;
    so[sst] = a1;
    so[2 * sst] = a2;
  }
  // dw: the lane's row segments of the block's columns, 16 bytes at a time
  if (in_band) {
    T* d0p = (T*)p.dw + rb;
#pragma unroll
    for (int k = 0; k < 3; ++k)
#pragma unroll
      for (int v = 0; v < HV; ++v) {
        if (v * VE < lo) continue;
        uint4 q;
        q.x = dwv[k][v * 4 + 0]; q.y = dwv[k][v * 4 + 1]; q.z = dwv[k][v * 4 + 2]; q.w = dwv[k][v * 4 + 3];
        *reinterpret_cast<uint4*>(d0p + (int64_t)k * p.npc + v * VE) = q;
      }
  }
  __syncthreads();

  // gsum (+)= g over the band rows and the block's columns, 4 floats a thread
  const int nvr = (K - lo) / 4;
  const int n = rows * nvr;
  const int64_t ob = plane * HW + (int64_t)bs * W + ws;
  constexpr int TT = 64 * NW, U = 8;
  for (int e0 = tid; e0 < n; e0 += TT * U) {
    float av[U][4];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int e = e0 + k * TT < n ? e0 + k * TT : e0;
      const int rr = e / nvr, cc = lo + (e - rr * nvr) * 4;
      if (!p.first) ldv<4>(p.gsum + ob + (int64_t)rr * W + cc, av[k]);
    }
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int e = e0 + k * TT;
      if (e < n) {
        const int rr = e / nvr, cc = lo + (e - rr * nvr) * 4;
        const float* gl = lds + (rr + 1) * HP + cc + HOFF;
        float s[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) s[q] = (p.first ? 0.f : av[k][q]) + gl[q];
        stv<4>(p.gsum + ob + (int64_t)rr * W + cc, s);
      }
    }
  }
}

template <typename T, int NW, int DIR, bool LG>
__global__ void __launch_bounds__(64 * NW) large_hadj_kernel(LargeHAdjParams p) {
  large_hadj_body<T, NW, DIR, LG>(p, blockIdx.x, gridDim.x);
}
// Both horizontal adjoints in one grid (each direction's h kept by the
// forward, so neither waits for the other's recompute): the first half of
// the workgroups runs left-to-right's adjoint, the second half
// right-to-left's, each on its own column block of the launch.
template <typename T, int NW, bool LG>
__global__ void __launch_bounds__(64 * NW) large_hadj2_kernel(LargeHAdjParams p0, LargeHAdjParams p1) {
  const int64_t half = gridDim.x / 2, b = blockIdx.x;
  if (b < half) large_hadj_body<T, NW, 0, LG>(p0, b, half);
  else large_hadj_body<T, NW, 1, LG>(p1, b - half, half);
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------

// grid: workgroups per direction
template <typename T, int NW>
hipError_t launch_large_hadj2_nw(const LargeHAdjParams& p0, const LargeHAdjParams& p1, int64_t grid, size_t lds,
                                 bool lg, hipStream_t st) {
  auto kern = lg ? large_hadj2_kernel<T, NW, true> : large_hadj2_kernel<T, NW, false>;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)(2 * grid)), dim3(64 * NW), lds, st, p0, p1);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_large_hadj2(const LargeHAdjParams& p0, const LargeHAdjParams& p1, int nw, int64_t grid,
                              size_t lds, bool lg, hipStream_t st) {
  switch (nw) {
    case 1: return launch_large_hadj2_nw<T, 1>(p0, p1, grid, lds, lg, st);
    case 2: return launch_large_hadj2_nw<T, 2>(p0, p1, grid, lds, lg, st);
    case 3: return launch_large_hadj2_nw<T, 3>(p0, p1, grid, lds, lg, st);
    case 4: return launch_large_hadj2_nw<T, 4>(p0, p1, grid, lds, lg, st);
    case 5: return launch_large_hadj2_nw<T, 5>(p0, p1, grid, lds, lg, st);
    case 6: return launch_large_hadj2_nw<T, 6>(p0, p1, grid, lds, lg, st);
    case 7: return launch_large_hadj2_nw<T, 7>(p0, p1, grid, lds, lg, st);
    case 8: return launch_large_hadj2_nw<T, 8>(p0, p1, grid, lds, lg, st);
    default: return hipErrorInvalidValue;
  }
}

template <typename T, int NW>
hipError_t launch_large_hadj_nw(const LargeHAdjParams& p, int dir, int64_t grid, size_t lds, bool lg,
                                hipStream_t st) {
  auto kern = lg ? (dir ? large_hadj_kernel<T, NW, 1, true> : large_hadj_kernel<T, NW, 0, true>)
                 : (dir ? large_hadj_kernel<T, NW, 1, false> : large_hadj_kernel<T, NW, 0, false>);
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(64 * NW), lds, st, p);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_large_hadj(const LargeHAdjParams& p, int dir, int nw, int64_t grid, size_t lds, bool lg,
                             hipStream_t st) {
  switch (nw) {
    case 1: return launch_large_hadj_nw<T, 1>(p, dir, grid, lds, lg, st);
    case 2: return launch_large_hadj_nw<T, 2>(p, dir, grid, lds, lg, st);
    case 3: return launch_large_hadj_nw<T, 3>(p, dir, grid, lds, lg, st);
    case 4: return launch_large_hadj_nw<T, 4>(p, dir, grid, lds, lg, st);
    case 5: return launch_large_hadj_nw<T, 5>(p, dir, grid, lds, lg, st);
    case 6: return launch_large_hadj_nw<T, 6>(p, dir, grid, lds, lg, st);
    case 7: return launch_large_hadj_nw<T, 7>(p, dir, grid, lds, lg, st);
    case 8: return launch_large_hadj_nw<T, 8>(p, dir, grid, lds, lg, st);
    default: return hipErrorInvalidValue;
  }
}

// parameters of the banded adjoint of one horizontal direction, and its
// per-launch block (step j of the adjoint's order; outside [0, nblk) the
// direction has nothing to do in the launch) with that block's group masks
template <typename T>
LargeHAdjParams large_hadj_params(const LargeBwdHArgs& a, const LargeGeom<T>& g) {
  LargeHAdjParams p{};
  p.dy = a.dy; p.u = a.u; p.w = a.w; p.dw = a.dw; p.hbuf = a.hbuf; p.gsum = a.gsum; p.state = a.state;
  p.planes = a.planes; p.npc = a.planes * (int64_t)a.H * a.W; p.H = a.H; p.W = a.W;
  p.first = a.first;
  p.renorm = a.renorm;
  p.nblk = g.nblk;
  p.band_rows = g.hb_mid; p.edge_rows = g.hb_edge; p.nbands = g.hb_n; p.halo = g.halo;
  return p;
}
template <typename T>
size_t large_hadj_lds(const LargeGeom<T>& g) {
  return ((size_t)(g.hb_edge + 2) * (LargeCfg<T>::KH + 5) + 4 * (8 + 2) + 64) * sizeof(float);
}
template <typename T>
void large_hadj_step(LargeHAdjParams& p, const LargeBwdHArgs& a, const LargeGeom<T>& g, int j) {
  constexpr int K = LargeCfg<T>::KH;
  p.step = j;
  p.zmask = p.gmask = 0;
  if (j < 0 || j >= g.nblk) return;
  const int GW = (a.group > 0 && a.group < a.W) ? a.group : a.W;
  if (GW >= a.W) return;
  // scan order: left-to-right visits column c after c - 1, right-to-left after c + 1
  auto starts = [&](int c) { return a.dir ? ((c + 1) % GW == 0) : (c % GW == 0); };
  const int blk = a.dir ? j : g.nblk - 1 - j;
  const int c0 = blk * K;
  const int ws = c0 + K <= a.W ? c0 : a.W - K;
  for (int i = 0; i < K; ++i) {
    const int c = ws + i, nxt = a.dir ? c - 1 : c + 1;
    if (starts(c)) p.gmask |= 1ull << i;
    if (nxt >= 0 && nxt < a.W && starts(nxt)) p.zmask |= 1ull << i;
  }
}

template <typename T>
hipError_t large_bwd_h_t(const LargeBwdHArgs& a) {
  using C = LargeCfg<T>;
  constexpr int K = C::KH;
  if (!large_fwd_supported<T>(a.H, a.W)) return hipErrorInvalidValue;
  const LargeGeom<T> g = large_geom<T>(a.H, a.W);
  hipStream_t st = (hipStream_t)a.stream;
  const int64_t npc = a.planes * (int64_t)a.H * a.W;
  const int64_t grid = (int64_t)g.hb_n * a.planes;
  if (grid > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  const int GW = (a.group > 0 && a.group < a.W) ? a.group : a.W;
  // scan order: left-to-right visits column c after c - 1, right-to-left after c + 1
  auto starts = [&](int c) { return a.dir ? ((c + 1) % GW == 0) : (c % GW == 0); };
  auto window = [&](int blk) {
    const int c0 = blk * K;
    return c0 + K <= a.W ? c0 : a.W - K;
  };

  // recompute: h into hbuf, hsum (+)= h; blocks in scan order
  LargeHParams h{};
  h.x = a.x; h.lam = a.lam; h.w = a.w; h.u = nullptr; h.y = nullptr; h.acc = a.hsum; h.state = a.state;
  h.planes = a.planes; h.npc = npc; h.H = a.H; h.W = a.W;
  // the weight slot is 0: w points at this direction's three maps
  h.slot0 = a.dir ? -1 : 0;
  h.slot1 = a.dir ? 0 : -1;
  h.nblk = g.nblk; h.delay = 0; h.half = 0;
  h.band_rows = g.hb_mid; h.edge_rows = g.hb_edge; h.nbands = g.hb_n; h.halo = g.halo;
  h.has_v = a.first ? 0 : 1;
  h.acc_b = nullptr;
  h.rec = 1;
  h.hbuf = a.hbuf;
  h.renorm = a.renorm;
  h.hdy = a.hdy;
  for (int j = 0; j < g.nblk && !a.saved; ++j) {
    const int blk = a.dir ? g.nblk - 1 - j : j;
    const int ws = window(blk);
    uint64_t m = 0;
    if (GW < a.W)
      for (int i = 0; i < K; ++i)
        if (starts(ws + i)) m |= 1ull << i;
    h.step = j;
    h.gmask[0] = a.dir ? 0 : m;
    h.gmask[1] = a.dir ? m : 0;
    hipError_t e = launch_large_h<T>(h, g.hb_nw, grid, g.lds_hb, a.logits != 0, st);
    if (e != hipSuccess) return e;
  }

  // adjoint: blocks in reverse scan order
  LargeHAdjParams p = large_hadj_params<T>(a, g);
  for (int j = 0; j < g.nblk; ++j) {
    large_hadj_step(p, a, g, j);
    hipError_t e = launch_large_hadj<T>(p, a.dir, g.hb_nw, grid, large_hadj_lds<T>(g), a.logits != 0, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Both horizontal adjoints at once on h kept by the forward (l2r.saved and
// r2l.saved): one launch per column block, left-to-right's adjoint on block
// nblk - 1 - j, right-to-left's on block j (one launch later for an odd block
// count, so no block is visited by both in one launch).  The direction that
// reaches a block first stores its g in gsum, the other adds: every element
// gets the same two terms as in the sequential order (addition of two terms
// commutes exactly).  Each direction has its own column-product state.
template <typename T>
hipError_t large_bwd_h_pair_t(const LargeBwdHArgs& l2r, const LargeBwdHArgs& r2l) {
  if (!large_fwd_supported<T>(l2r.H, l2r.W)) return hipErrorInvalidValue;
  if (!l2r.saved || !r2l.saved || l2r.dir != 0 || r2l.dir != 1) return hipErrorInvalidValue;
  const LargeGeom<T> g = large_geom<T>(l2r.H, l2r.W);
  const int64_t grid = (int64_t)g.hb_n * l2r.planes;
  if (2 * grid > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  LargeHAdjParams p0 = large_hadj_params<T>(l2r, g), p1 = large_hadj_params<T>(r2l, g);
  const int delay = g.nblk & 1;
  for (int j = 0; j < g.nblk + delay; ++j) {
    const bool first = 2 * j < g.nblk - 1 + delay;  // both directions reach their blocks first
    large_hadj_step(p0, l2r, g, j);
    large_hadj_step(p1, r2l, g, j - delay);
    p0.first = p1.first = first ? 1 : 0;
    hipError_t e = launch_large_hadj2<T>(p0, p1, g.hb_nw, grid, large_hadj_lds<T>(g), l2r.logits != 0,
                                         (hipStream_t)l2r.stream);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <typename T>
hipError_t large_bwd_v_rec_t(const LargeBwdVArgs& a) {
  if (!large_fwd_supported<T>(a.H, a.W)) return hipErrorInvalidValue;
  const LargeGeom<T> g = large_geom<T>(a.H, a.W);
  const bool both = a.slot_t2b >= 0 && a.slot_b2t >= 0;
  LargeVParams v{};
  v.x = a.x; v.lam = a.lam; v.w = a.w; v.u = nullptr; v.y = nullptr;
  v.acc = a.slot_t2b >= 0 ? a.h_t2b : a.h_b2t;
  v.acc_b = both ? a.h_b2t : nullptr;
  v.planes = a.planes; v.npc = a.planes * (int64_t)a.H * a.W; v.H = a.H; v.W = a.W;
  v.slot0 = a.slot_t2b; v.slot1 = a.slot_b2t;
  v.final_out = 0;
  v.split = both ? 1 : 0;
  v.grp = (a.group > 0 && a.group < a.H) ? a.group : a.H;
  v.renorm = a.renorm;
  if (both && 2 * a.planes > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  hipStream_t st = (hipStream_t)a.stream;
  switch (g.wpd) {
    case 1: return launch_large_v<T, 1>(v, false, st, true, a.logits != 0);
    case 2: return launch_large_v<T, 2>(v, false, st, true, a.logits != 0);
    case 4: return launch_large_v<T, 4>(v, false, st, true, a.logits != 0);
    default: return hipErrorInvalidValue;
  }
}


// ---------------------------------------------------------------------------
// adjoint of the vertical directions (after large_bwd_v_rec): one workgroup per
// plane.  Top-to-bottom's adjoint walks the rows upwards, bottom-to-top's
// downwards; with both present each takes half of the waves and they meet at
// the middle row, as the forward's vertical pass does (every row's g is added
// to gsum by the direction that reaches it first, then, after a barrier, by
// the other).  Lanes hold chunk-interleaved positions (whole cache lines per
// load instruction); rows stream through register rings.  Per row:
//   g = u dy + [a1 + a0(p+1) + a2(p-1)]   (a_k = w_k g of the previous row done)
//   dw_k = g h[prev](p+k-1),   gsum += g
// ---------------------------------------------------------------------------
struct LargeVAdjParams {
  const void* dy;
  const void* u;
  const void* w;        // all directions, packed
  void* dw;             // all directions, packed
  const float* h[2];    // h of top-to-bottom, bottom-to-top
  float* gsum;
  int64_t planes, npc;
  int H, W;
  int slot[2];          // weight slots of top-to-bottom, bottom-to-top (-1 absent)
  int grp;              // rows per local-GSPN group (H: global)
  int renorm;           // Eq. 6 logits (LG kernels): normalise over on-line neighbours only
  int y_pd;             // dy is (n, B, C, H, W): the direction's map at slot * npc
};

// LG: the weight maps hold Eq. 6 logits; dw becomes their gradient.
template <typename T, int WPD, bool BOTH, bool LG>
__global__ void __launch_bounds__((BOTH ? 128 : 64) * WPD, 2) large_vadj_kernel(LargeVAdjParams p) {
  using C = LargeCfg<T>;
  // rings: R rows of the bf16/fp32 input maps, RH rows of h, RA rows of gsum
  constexpr int NP = C::NPV, R = C::RV, RH = 1, RA = 1;
  constexpr int G = 4;            // positions per lane and chunk
  constexpr int NQ = NP / G;      // chunks per wave span
  constexpr int SPAN = 64 * G;    // positions per chunk
  typedef Pack<T, G> PK;
  __shared__ float edge[2][2 * WPD][2];  // [step parity][wave][a0 of the first position, a2 of the last]

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int dir = BOTH ? (wave >= WPD ? 1 : 0) : (p.slot[0] >= 0 ? 0 : 1);
  const int wi = BOTH ? wave - dir * WPD : wave;
  const int64_t plane = blockIdx.x;
  const int H = p.H, W = p.W;
  int po[NQ];
  bool qok[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int pos = wi * NQ * SPAN + q * SPAN + lane * G;
    qok[q] = pos < W;  // W is a multiple of G
    po[q] = qok[q] ? pos : 0;
  }
  const int wlo = wi * NQ * SPAN - 1, whi = (wi + 1) * NQ * SPAN;  // neighbours of the wave's span
  const bool wlo_ok = wlo >= 0, whi_ok = whi < W;
  const int64_t pb = plane * (int64_t)H * W;
  const int slot = p.slot[dir];
  const int odd = BOTH ? (H & 1) : 0;
  const int nsteps = H + odd;
  const int sm = BOTH ? H / 2 + odd : nsteps;  // first step of the second half
  const int delay = dir ? odd : 0;
  const int grp = p.grp;

  for (int i = threadIdx.x; i < 2 * 2 * WPD * 2; i += blockDim.x) (&edge[0][0][0])[i] = 0.f;
  __syncthreads();

  const T* w0 = (const T*)p.w + (int64_t)slot * 3 * p.npc + pb;
  const T* dyb = (const T*)p.dy + (p.y_pd ? (int64_t)slot * p.npc : 0);
  const T* base[5] = {dyb + pb, (const T*)p.u + pb, w0, w0 + p.npc, w0 + 2 * p.npc};
  T* d0 = (T*)p.dw + (int64_t)slot * 3 * p.npc + pb;
  const float* hb = p.h[dir] + pb;
  float* gs = p.gsum + pb;

  auto t_of = [&](int s) { return s - delay; };
  // adjoint order: top-to-bottom's rows upwards, bottom-to-top's downwards
  auto line_of = [&](int t) {
    t = t < 0 ? 0 : (t >= H ? H - 1 : t);
    return dir ? t : H - 1 - t;
  };
  auto prev_of = [&](int line) { return dir ? line + 1 : line - 1; };  // previous row in scan order
  // scan order enters a group at its first line (top-to-bottom: lowest row)
  auto starts = [&](int line) { return dir ? ((line + 1) % grp == 0) : (line % grp == 0); };

  PK ring[R][5][NQ];
  float hring[RH][NQ][G];
  float hedge[RH][2];
  auto load_main = [&](int k, int s) __attribute__((always_inline)) {
    const int64_t off = (int64_t)line_of(t_of(s)) * W;
#pragma unroll
    for (int m = 0; m < 5; ++m)
#pragma unroll
      for (int q = 0; q < NQ; ++q) ring[k][m][q].load(base[m] + off + po[q]);
  };
  auto load_h = [&](int k, int s) __attribute__((always_inline)) {
    int pl = prev_of(line_of(t_of(s)));
    pl = pl < 0 ? 0 : (pl >= H ? H - 1 : pl);
    const int64_t hoff = (int64_t)pl * W;
#pragma unroll
    for (int q = 0; q < NQ; ++q) ldv<G>(hb + hoff + po[q], hring[k][q]);
    hedge[k][0] = hb[hoff + (wlo_ok ? wlo : 0)];
    hedge[k][1] = hb[hoff + (whi_ok ? whi : 0)];
  };
  float gring[RA][NQ][G];
  auto load_aux = [&](int k, int s) __attribute__((always_inline)) {
    const int64_t off = (int64_t)line_of(t_of(s)) * W;
#pragma unroll
    for (int q = 0; q < NQ; ++q) ldv<G>(gs + off + po[q], gring[k][q]);
  };
  auto consume = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < R; ++k) {
#pragma unroll
      for (int m = 0; m < 5; ++m)
#pragma unroll
        for (int q = 0; q < NQ; ++q)
#pragma unroll
          for (int i = 0; i < PK::kWords; ++i) asm volatile("" ::"v"(ring[k][m][q].w[i]));
    }
#pragma unroll
    for (int k = 0; k < RH; ++k) {
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int j = 0; j < G; ++j) asm volatile("" ::"v"(hring[k][q][j]));
      asm volatile("" ::"v"(hedge[k][0]), "v"(hedge[k][1]));
    }
#pragma unroll
    for (int k = 0; k < RA; ++k)
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int j = 0; j < G; ++j) asm volatile("" ::"v"(gring[k][q][j]));
  };

  float a0[NQ][G], a1[NQ][G], a2[NQ][G];  // w_k * g of the previous row done
#pragma unroll
  for (int q = 0; q < NQ; ++q)
#pragma unroll
    for (int j = 0; j < G; ++j) a0[q][j] = a1[q][j] = a2[q][j] = 0.f;

  // one step; the gsum refills stop at s_end (the middle, before the barrier)
  auto step = [&](int k, int s, int s_end) __attribute__((always_inline)) {
    const int t = t_of(s);
    const bool act = t >= 0 && t < H;
    const int par = s & 1;
    const int line = line_of(t);
    const int nx = dir ? line - 1 : line + 1;  // next row in scan order
    const bool zr = !(nx >= 0 && nx < H) || starts(nx);
    const int pl = prev_of(line);
    const bool hzero = !(pl >= 0 && pl < H) || starts(line);  // no previous state
    // a0 from position p+1 and a2 from p-1 (previous row done), across lanes,
    // chunks and waves
    float ar[NQ], al[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      ar[q] = from_next_lane(a0[q][0]);
      al[q] = from_prev_lane(a2[q][G - 1]);
    }
    float er = 0.f, el = 0.f;
    if constexpr (WPD > 1) {
      const float nr = edge[par ^ 1][wi < WPD - 1 ? wave + 1 : wave][0];
      const float nl = edge[par ^ 1][wi > 0 ? wave - 1 : wave][1];
      er = wi < WPD - 1 ? nr : 0.f;
      el = wi > 0 ? nl : 0.f;
    }
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const float cr = q < NQ - 1 ? __builtin_bit_cast(float, __builtin_amdgcn_readlane(
                                                              __builtin_bit_cast(int, a0[q + 1][0]), 0))
                                  : er;
      const float cl = q > 0 ? __builtin_bit_cast(float, __builtin_amdgcn_readlane(
                                                         __builtin_bit_cast(int, a2[q - 1][G - 1]), 63))
                             : el;
      if (lane == 63) ar[q] = cr;
      if (lane == 0) al[q] = cl;
    }
    // h of the previous row and its neighbours (zero past the row end)
    const float(&hv)[NQ][G] = hring[k % RH];
    float hr[NQ], hl[NQ], hf[NQ], hb3[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      hf[q] = qok[q] ? hv[q][0] : 0.f;
      hb3[q] = qok[q] ? hv[q][G - 1] : 0.f;
      hr[q] = from_next_lane(hf[q]);
      hl[q] = from_prev_lane(hb3[q]);
    }
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const float n0 = q < NQ - 1 ? __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, hf[q + 1]), 0))
                                  : (whi_ok ? hedge[k % RH][1] : 0.f);
      const float n3 = q > 0 ? __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, hb3[q - 1]), 63))
                             : (wlo_ok ? hedge[k % RH][0] : 0.f);
      if (lane == 63) hr[q] = n0;
      if (lane == 0) hl[q] = n3;
    }
    // chunk by chunk: g from the old products, then the new products, dw and
    // gsum stored at once (keeps few values live)
    const int64_t off = (int64_t)line * W;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const bool ok = qok[q] && act;
      const PK(&v)[5][NQ] = ring[k];
      float g[G];
#pragma unroll
      for (int j = 0; j < G; ++j) {
        const float an = j == G - 1 ? ar[q] : a0[q][j + 1];
        const float ap = j == 0 ? al[q] : a2[q][j - 1];
        const float in = zr ? 0.f : a1[q][j] + an + ap;
        const float gv = fmaf(v[1][q].get(j), v[0][q].get(j), in);
        g[j] = ok ? gv : 0.f;
      }
      float dv[3][G], go[G];
#pragma unroll
      for (int j = 0; j < G; ++j) {
        float wa = v[2][q].get(j), wb = v[3][q].get(j), wc = v[4][q].get(j);
        Norm3 nr;
        if constexpr (LG) {
          nr = normalize3(wa, wb, wc, po[q] + j == 0, po[q] + j == W - 1, p.renorm != 0);
          wa = nr.w[0];
          wb = nr.w[1];
          wc = nr.w[2];
        }
        a0[q][j] = wa * g[j];
        a1[q][j] = wb * g[j];
        a2[q][j] = wc * g[j];
        const float hm = hzero ? 0.f : hv[q][j];
        const float hlv = hzero ? 0.f : (j == 0 ? hl[q] : hv[q][j - 1]);
        const float hrv = hzero ? 0.f : (j == G - 1 ? hr[q] : hv[q][j + 1]);
        dv[0][j] = g[j] * hlv;
        dv[1][j] = g[j] * hm;
        dv[2][j] = g[j] * hrv;
        if constexpr (LG) norm3_vjp(nr, dv[0][j], dv[1][j], dv[2][j]);
        go[j] = gring[k % RA][q][j] + g[j];
      }
      if (ok) {
#pragma unroll
        for (int m = 0; m < 3; ++m) stv<G>(d0 + (int64_t)m * p.npc + off + po[q], dv[m]);
        stv<G>(gs + off + po[q], go);
      }
    }
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int j = 0; j < G; ++j) {
        asm volatile("" : "+v"(a0[q][j]));
        asm volatile("" : "+v"(a1[q][j]));
        asm volatile("" : "+v"(a2[q][j]));
      }
    if (lane == 0) edge[par][wave][0] = a0[0][0];
    if (lane == 63) edge[par][wave][1] = a2[NQ - 1][G - 1];
    asm volatile("" ::: "memory");
    load_main(k, s + R);
    load_h(k % RH, s + RH);
    if (s + RA < s_end) load_aux(k % RA, s + RA);
    lds_barrier();
  };

  // first half: rows this direction reaches first; second half (after every
  // wave's first-half gsum stores are visible): the rest
  const int o = (R - sm % R) % R;  // idle steps before step 0 align the first loop to the ring
  static_assert(R % RA == 0 && R % RH == 0, "the small rings' slots repeat with the main ring");
#pragma unroll
  for (int k = 0; k < R; ++k) load_main(k, k - o);
#pragma unroll
  for (int k = 0; k < RH; ++k) load_h(k, k - o);
#pragma unroll
  for (int k = 0; k < RA; ++k) load_aux(k, k - o);
  for (int s0 = -o; s0 < sm; s0 += R) {
#pragma unroll
    for (int k = 0; k < R; ++k) step(k, s0 + k, sm);
  }
  if (sm < nsteps) {
    consume();
    __syncthreads();
#pragma unroll
    for (int k = 0; k < RA; ++k) load_aux(k, sm + k);
    for (int s0 = sm; s0 < nsteps; s0 += R) {
#pragma unroll
      for (int k = 0; k < R; ++k) step(k, s0 + k, nsteps + R);
    }
  }
  consume();
}

template <typename T, int WPD, bool BOTH>
hipError_t launch_large_vadj_mode(const LargeVAdjParams& p, bool lg, hipStream_t st) {
  auto kern = lg ? large_vadj_kernel<T, WPD, BOTH, true> : large_vadj_kernel<T, WPD, BOTH, false>;
  hipLaunchKernelGGL(kern, dim3((unsigned)p.planes), dim3((BOTH ? 128 : 64) * WPD), 0, st, p);
  return hipGetLastError();
}

template <typename T>
hipError_t large_bwd_v_adj_t(const LargeBwdVAdjArgs& a) {
  if (!large_fwd_supported<T>(a.H, a.W)) return hipErrorInvalidValue;
  if (a.planes > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  const LargeGeom<T> g = large_geom<T>(a.H, a.W);
  LargeVAdjParams p{};
  p.dy = a.dy; p.u = a.u; p.w = a.w; p.dw = a.dw;
  p.h[0] = a.h_t2b; p.h[1] = a.h_b2t;
  p.gsum = a.gsum;
  p.planes = a.planes; p.npc = a.planes * (int64_t)a.H * a.W; p.H = a.H; p.W = a.W;
  p.slot[0] = a.slot_t2b; p.slot[1] = a.slot_b2t;
  p.grp = (a.group > 0 && a.group < a.H) ? a.group : a.H;
  p.renorm = a.renorm;
  p.y_pd = a.y_pd;
  const bool both = a.slot_t2b >= 0 && a.slot_b2t >= 0, lg = a.logits != 0;
  hipStream_t st = (hipStream_t)a.stream;
  switch (g.wpd) {
    case 1: return both ? launch_large_vadj_mode<T, 1, true>(p, lg, st) : launch_large_vadj_mode<T, 1, false>(p, lg, st);
    case 2: return both ? launch_large_vadj_mode<T, 2, true>(p, lg, st) : launch_large_vadj_mode<T, 2, false>(p, lg, st);
    case 4: return both ? launch_large_vadj_mode<T, 4, true>(p, lg, st) : launch_large_vadj_mode<T, 4, false>(p, lg, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace gspn
