// Streaming kernels: one launch per scan direction, any H, W up to GSPN_MAX_LINE.
//
// A plane is seen as L lines of P positions.  Vertical directions (T2B, B2T)
// have lines = rows, positions = columns; horizontal ones (L2R, R2L) have
// lines = columns, positions = rows.  One workgroup owns one plane and walks
// its lines in scan order (Sec. 3.3: lines are sequential, positions are
// parallel).  Each lane owns NP consecutive positions; a line is spread over
// NW = blockDim/64 waves.  Neighbour values inside a wave move with DPP wave
// shifts; at wave edges they go through LDS with one barrier per line.
//
// Memory is read in tiles of NL lines x NP positions per lane, vectorised along
// whichever axis is contiguous (positions for vertical, lines for horizontal),
// so every global access is a 4- to 16-byte vector access.
//
// Directions are merged through an fp32 accumulator in the workspace: the first
// pass stores its h, later passes add theirs, the last one writes y = u * acc.
#pragma once
#include "gspn_device.hpp"
#include "gspn_launch.hpp"

namespace gspn {

struct Geo {
  int L;          // lines in the plane
  int P;          // positions per line
  int W;          // row pitch (elements)
  int64_t plane;  // elements per plane (H * W)
  int rev;        // lines visited from L-1 down to 0
};

// element (line l, position p):  vertical l*W + p,  horizontal p*W + l
template <bool HZ, int NL, int NP, typename T>
__device__ __forceinline__ void load_tile(const T* __restrict__ base, const Geo& g, int l0, int p0,
                                          bool vec_ok, float (&t)[NL][NP]) {
  if constexpr (!HZ) {
#pragma unroll
    for (int l = 0; l < NL; ++l) {
      const int line = l0 + l;
      if (line >= 0 && line < g.L) {
        const T* row = base + (int64_t)line * g.W;
        if (vec_ok && p0 + NP <= g.P) {
          ldv<NP>(row + p0, t[l]);
        } else {
#pragma unroll
          for (int q = 0; q < NP; ++q) t[l][q] = (p0 + q < g.P) ? to_f(row[p0 + q]) : 0.f;
        }
      } else {
#pragma unroll
        for (int q = 0; q < NP; ++q) t[l][q] = 0.f;
      }
    }
  } else {
#pragma unroll
    for (int q = 0; q < NP; ++q) {
      const int pos = p0 + q;
      float v[NL];
      if (pos < g.P) {
        const T* row = base + (int64_t)pos * g.W;
        if (vec_ok && l0 >= 0 && l0 + NL <= g.L) {
          ldv<NL>(row + l0, v);
        } else {
#pragma unroll
          for (int l = 0; l < NL; ++l) v[l] = (l0 + l >= 0 && l0 + l < g.L) ? to_f(row[l0 + l]) : 0.f;
        }
      } else {
#pragma unroll
        for (int l = 0; l < NL; ++l) v[l] = 0.f;
      }
#pragma unroll
      for (int l = 0; l < NL; ++l) t[l][q] = v[l];
    }
  }
}

template <bool HZ, int NL, int NP, typename T>
__device__ __forceinline__ void store_tile(T* __restrict__ base, const Geo& g, int l0, int p0,
                                           bool vec_ok, const float (&t)[NL][NP]) {
  if constexpr (!HZ) {
#pragma unroll
    for (int l = 0; l < NL; ++l) {
      const int line = l0 + l;
      if (line < g.L) {
        T* row = base + (int64_t)line * g.W;
        if (vec_ok && p0 + NP <= g.P) {
          stv<NP>(row + p0, t[l]);
        } else {
#pragma unroll
          for (int q = 0; q < NP; ++q)
            if (p0 + q < g.P) row[p0 + q] = from_f<T>(t[l][q]);
        }
      }
    }
  } else {
#pragma unroll
    for (int q = 0; q < NP; ++q) {
      const int pos = p0 + q;
      if (pos < g.P) {
        T* row = base + (int64_t)pos * g.W;
        float v[NL];
#pragma unroll
        for (int l = 0; l < NL; ++l) v[l] = t[l][q];
        if (vec_ok && l0 + NL <= g.L) {
          stv<NL>(row + l0, v);
        } else {
#pragma unroll
          for (int l = 0; l < NL; ++l)
            if (l0 + l < g.L) row[l0 + l] = from_f<T>(v[l]);
        }
      }
    }
  }
}

// Neighbour exchange across wave edges: each wave publishes the values of its
// first and last position, the neighbours read them after one barrier.
struct Edges {
  float lo[2][kMaxWaves];  // [parity][wave] value at the wave's first position
  float hi[2][kMaxWaves];  // [parity][wave] value at the wave's last position
};

// ---------------------------------------------------------------------------
// forward pass of one direction
//   MODE_STORE: acc = h            (ugate: acc = u * h)
//   MODE_ADD:   acc += h           (ugate: acc += u * h)
//   MODE_FINAL: y = u * (acc + h)  (ugate: y = acc + u * h; acc may be null)
//   MODE_REC:   hprev_out[line] = h of the previous line (0 for a group's first
//               line), hsum (+)= h, or dy * h with hdy; with du: du = dy * h
//               (recompute step of the backward)
// EXT enables the per-direction and logit options (runtime flags inside).
// ---------------------------------------------------------------------------
struct StreamFwdParams {
  const void* x;
  const void* lam;
  const void* w;
  int64_t wstride;
  const void* u;
  float* acc;
  void* y;
  float* hprev_out;
  const void* dy;
  void* du;
  int first;
  Geo g;
  int vec_ok, vec_ok_f;
  int G;       // lines per group (L for the global scan)
  int logits, renorm, ugate, hdy;
};

template <typename T, bool HZ, bool REV, int NP, int NL, int MODE, bool EXT>
__global__ void __launch_bounds__(1024) stream_fwd_kernel(StreamFwdParams p) {
  const Geo g = p.g;
  const int64_t pbase = (int64_t)blockIdx.x * g.plane;
  const T* x = (const T*)p.x + pbase;
  const T* lam = (const T*)p.lam + pbase;
  const T* w = (const T*)p.w + pbase;
  const int64_t wstride = p.wstride;
  const T* u = p.u ? (const T*)p.u + pbase : nullptr;
  float* acc = p.acc ? p.acc + pbase : nullptr;
  T* y = p.y ? (T*)p.y + pbase : nullptr;
  float* hprev_out = p.hprev_out ? p.hprev_out + pbase : nullptr;
  const T* dyp = (EXT && p.dy) ? (const T*)p.dy + pbase : nullptr;
  T* dup = (EXT && p.du) ? (T*)p.du + pbase : nullptr;
  const bool vec_ok = p.vec_ok, vec_ok_f = p.vec_ok_f, first = p.first;
  const bool ugate = EXT && p.ugate;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = blockDim.x >> 6;
  const int p0 = tid * NP;
  __shared__ Edges ex;

  float hp[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) hp[q] = 0.f;

  const int nchunks = (g.L + NL - 1) / NL;
  int step = 0;
  for (int cc = 0; cc < nchunks; ++cc) {
    const int c = REV ? nchunks - 1 - cc : cc;
    const int l0 = c * NL;
    float tx[NL][NP], tl[NL][NP], t0[NL][NP], t1[NL][NP], t2[NL][NP], to[NL][NP];
    load_tile<HZ, NL, NP>(x, g, l0, p0, vec_ok, tx);
    load_tile<HZ, NL, NP>(lam, g, l0, p0, vec_ok, tl);
    load_tile<HZ, NL, NP>(w, g, l0, p0, vec_ok, t0);
    load_tile<HZ, NL, NP>(w + wstride, g, l0, p0, vec_ok, t1);
    load_tile<HZ, NL, NP>(w + 2 * wstride, g, l0, p0, vec_ok, t2);
    if (EXT && p.logits) {
#pragma unroll
      for (int l = 0; l < NL; ++l)
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          const Norm3 r = normalize3(t0[l][q], t1[l][q], t2[l][q], p0 + q == 0, p0 + q == g.P - 1, p.renorm);
          // positions past the line keep zero weights (their h must stay 0)
          const bool on = p0 + q < g.P;
          t0[l][q] = on ? r.w[0] : 0.f;
          t1[l][q] = on ? r.w[1] : 0.f;
          t2[l][q] = on ? r.w[2] : 0.f;
        }
    }
    if (MODE == MODE_ADD || (MODE == MODE_FINAL && acc) || (MODE == MODE_REC && !first))
      load_tile<HZ, NL, NP>(acc, g, l0, p0, vec_ok_f, to);
    else {
#pragma unroll
      for (int l = 0; l < NL; ++l)
#pragma unroll
        for (int q = 0; q < NP; ++q) to[l][q] = 0.f;
    }
    float tu[NL][NP];
    if (MODE == MODE_FINAL || ugate) load_tile<HZ, NL, NP>(u, g, l0, p0, vec_ok, tu);
    float th[NL][NP];  // MODE_REC: previous-line state per line
    float tdy[NL][NP], tdu[NL][NP];
    if (EXT && MODE == MODE_REC && dyp) load_tile<HZ, NL, NP>(dyp, g, l0, p0, vec_ok, tdy);

#pragma unroll
    for (int ll = 0; ll < NL; ++ll) {
      const int l = REV ? NL - 1 - ll : ll;
      if (l0 + l < g.L) {  // uniform over the workgroup
        if (group_start(l0 + l, p.G, REV)) {
#pragma unroll
          for (int q = 0; q < NP; ++q) hp[q] = 0.f;
        }
        if (MODE == MODE_REC) {
#pragma unroll
          for (int q = 0; q < NP; ++q) th[l][q] = hp[q];
        }
        float left = from_prev_lane(hp[NP - 1]);
        float right = from_next_lane(hp[0]);
        if (nw > 1) {
          const int par = step & 1;
          if (lane == 0) ex.lo[par][wave] = hp[0];
          if (lane == 63) ex.hi[par][wave] = hp[NP - 1];
          __syncthreads();
          if (lane == 0 && wave > 0) left = ex.hi[par][wave - 1];
          if (lane == 63 && wave < nw - 1) right = ex.lo[par][wave + 1];
        }
        float h[NP];
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          const float hl = q == 0 ? left : hp[q - 1];
          const float hr = q == NP - 1 ? right : hp[q + 1];
          float v = tl[l][q] * tx[l][q];
          v = fmaf(t0[l][q], hl, v);
          v = fmaf(t1[l][q], hp[q], v);
          v = fmaf(t2[l][q], hr, v);
          h[q] = v;
        }
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          hp[q] = h[q];
          if (EXT && MODE == MODE_REC && dyp) {
            const float dh = tdy[l][q] * h[q];
            tdu[l][q] = dh;
            to[l][q] += p.hdy ? dh : h[q];
          } else {
            to[l][q] += ugate ? tu[l][q] * h[q] : h[q];
          }
        }
        ++step;
      }
    }
    if (MODE == MODE_FINAL) {
      if (!ugate) {
#pragma unroll
        for (int l = 0; l < NL; ++l)
#pragma unroll
          for (int q = 0; q < NP; ++q) to[l][q] *= tu[l][q];
      }
      store_tile<HZ, NL, NP>(y, g, l0, p0, vec_ok, to);
    } else {
      store_tile<HZ, NL, NP>(acc, g, l0, p0, vec_ok_f, to);
      if (MODE == MODE_REC) store_tile<HZ, NL, NP>(hprev_out, g, l0, p0, vec_ok_f, th);
      if (EXT && MODE == MODE_REC && dup) store_tile<HZ, NL, NP>(dup, g, l0, p0, vec_ok, tdu);
    }
  }
}

// ---------------------------------------------------------------------------
// adjoint pass of one direction (reverse scan order)
//   g[line][p] = u*dy + sum_k wn_k[p - (k-1)] * gn[p - (k-1)]
// where gn, wn_k are g and w of the line after this one in scan order (none
// when that line starts a group).
//   dw_k[line][p] = g[p] * hprev[line][p + k - 1]   (logits: through Eq. 6's Jacobian)
//   gsum (+)= g   (lamw: gsum (+)= lam * g and dlam = x * g)
// ---------------------------------------------------------------------------
struct StreamAdjParams {
  const void* dy;
  const void* u;
  const void* w;
  int64_t wstride;
  const float* hprev;
  void* dw;
  float* gsum;
  const void* lam;  // lamw only
  const void* x;    // lamw only
  void* dlam;       // lamw only
  int first;
  Geo g;
  int vec_ok, vec_ok_f;
  int G;
  int logits, renorm, lamw;
};

template <typename T, bool HZ, bool REV, int NP, int NL, bool EXT>
__global__ void __launch_bounds__(1024) stream_adj_kernel(StreamAdjParams p) {
  const Geo g = p.g;
  const int64_t pbase = (int64_t)blockIdx.x * g.plane;
  const T* dy = (const T*)p.dy + pbase;
  const T* u = (const T*)p.u + pbase;
  const T* w = (const T*)p.w + pbase;
  const int64_t wstride = p.wstride;
  const float* hprev = p.hprev + pbase;
  T* dw = (T*)p.dw + pbase;
  float* gsum = p.gsum + pbase;
  const bool lamw = EXT && p.lamw, logits = EXT && p.logits;
  const T* lamp = lamw ? (const T*)p.lam + pbase : nullptr;
  const T* xp = lamw ? (const T*)p.x + pbase : nullptr;
  T* dlamp = lamw ? (T*)p.dlam + pbase : nullptr;
  const bool vec_ok = p.vec_ok, vec_ok_f = p.vec_ok_f;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = blockDim.x >> 6;
  const int p0 = tid * NP;
  __shared__ Edges ea, eb;  // a: w0*g / w2*g products, b: hprev

  float gn[NP], wn0[NP], wn1[NP], wn2[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) gn[q] = wn0[q] = wn1[q] = wn2[q] = 0.f;

  const int nchunks = (g.L + NL - 1) / NL;
  constexpr bool adj_rev = !REV;  // adjoint visits lines in the opposite order
  int step = 0;
  for (int cc = 0; cc < nchunks; ++cc) {
    const int c = adj_rev ? nchunks - 1 - cc : cc;
    const int l0 = c * NL;
    float tdy[NL][NP], tu[NL][NP], t0[NL][NP], t1[NL][NP], t2[NL][NP], th[NL][NP], tg[NL][NP];
    load_tile<HZ, NL, NP>(dy, g, l0, p0, vec_ok, tdy);
    load_tile<HZ, NL, NP>(u, g, l0, p0, vec_ok, tu);
    load_tile<HZ, NL, NP>(w, g, l0, p0, vec_ok, t0);
    load_tile<HZ, NL, NP>(w + wstride, g, l0, p0, vec_ok, t1);
    load_tile<HZ, NL, NP>(w + 2 * wstride, g, l0, p0, vec_ok, t2);
    load_tile<HZ, NL, NP>(hprev, g, l0, p0, vec_ok_f, th);
    if (!p.first) load_tile<HZ, NL, NP>(gsum, g, l0, p0, vec_ok_f, tg);
    else {
#pragma unroll
      for (int l = 0; l < NL; ++l)
#pragma unroll
        for (int q = 0; q < NP; ++q) tg[l][q] = 0.f;
    }
    float tl[NL][NP], tx[NL][NP], tdl[NL][NP];
    if (lamw) {
      load_tile<HZ, NL, NP>(lamp, g, l0, p0, vec_ok, tl);
      load_tile<HZ, NL, NP>(xp, g, l0, p0, vec_ok, tx);
    }
    float d0[NL][NP], d1[NL][NP], d2[NL][NP];

#pragma unroll
    for (int ll = 0; ll < NL; ++ll) {
      const int l = adj_rev ? NL - 1 - ll : ll;
      const int line = l0 + l;
      if (line < g.L) {
        // the line after this one (in scan order) starts a group: it took nothing from here
        const int nxt = REV ? line - 1 : line + 1;
        if (nxt >= 0 && nxt < g.L && group_start(nxt, p.G, REV)) {
#pragma unroll
          for (int q = 0; q < NP; ++q) gn[q] = 0.f;
        }
        float a0[NP], a1[NP], a2[NP];
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          a0[q] = wn0[q] * gn[q];
          a1[q] = wn1[q] * gn[q];
          a2[q] = wn2[q] * gn[q];
        }
        // a0 comes from position p+1, a2 from p-1; hprev neighbours from p-1 and p+1
        float a0_next = from_next_lane(a0[0]);
        float a2_prev = from_prev_lane(a2[NP - 1]);
        float h_prev = from_prev_lane(th[l][NP - 1]);
        float h_next = from_next_lane(th[l][0]);
        if (nw > 1) {
          const int par = step & 1;
          if (lane == 0) { ea.lo[par][wave] = a0[0]; eb.lo[par][wave] = th[l][0]; }
          if (lane == 63) { ea.hi[par][wave] = a2[NP - 1]; eb.hi[par][wave] = th[l][NP - 1]; }
          __syncthreads();
          if (lane == 0 && wave > 0) { a2_prev = ea.hi[par][wave - 1]; h_prev = eb.hi[par][wave - 1]; }
          if (lane == 63 && wave < nw - 1) { a0_next = ea.lo[par][wave + 1]; h_next = eb.lo[par][wave + 1]; }
        }
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          const float an = q == NP - 1 ? a0_next : a0[q + 1];
          const float ap = q == 0 ? a2_prev : a2[q - 1];
          const float gv = tu[l][q] * tdy[l][q] + a1[q] + an + ap;
          const float hl = q == 0 ? h_prev : th[l][q - 1];
          const float hr = q == NP - 1 ? h_next : th[l][q + 1];
          float e0 = gv * hl, e1 = gv * th[l][q], e2 = gv * hr;
          float c0 = t0[l][q], c1 = t1[l][q], c2 = t2[l][q];
          if (logits) {
            const Norm3 r = normalize3(c0, c1, c2, p0 + q == 0, p0 + q == g.P - 1, p.renorm);
            const float inner = r.w[0] * e0 + r.w[1] * e1 + r.w[2] * e2;
            e0 = r.m[0] * r.sg[0] * (1.f - r.sg[0]) * (e0 - inner) * r.inv;
            e1 = r.m[1] * r.sg[1] * (1.f - r.sg[1]) * (e1 - inner) * r.inv;
            e2 = r.m[2] * r.sg[2] * (1.f - r.sg[2]) * (e2 - inner) * r.inv;
            const bool on = p0 + q < g.P;  // positions past the line keep zero weights
            c0 = on ? r.w[0] : 0.f;
            c1 = on ? r.w[1] : 0.f;
            c2 = on ? r.w[2] : 0.f;
          }
          d0[l][q] = e0;
          d1[l][q] = e1;
          d2[l][q] = e2;
          if (lamw) {
            tg[l][q] += tl[l][q] * gv;
            tdl[l][q] = tx[l][q] * gv;
          } else {
            tg[l][q] += gv;
          }
          gn[q] = gv;
          wn0[q] = c0;
          wn1[q] = c1;
          wn2[q] = c2;
        }
        ++step;
      }
    }
    store_tile<HZ, NL, NP>(dw, g, l0, p0, vec_ok, d0);
    store_tile<HZ, NL, NP>(dw + wstride, g, l0, p0, vec_ok, d1);
    store_tile<HZ, NL, NP>(dw + 2 * wstride, g, l0, p0, vec_ok, d2);
    store_tile<HZ, NL, NP>(gsum, g, l0, p0, vec_ok_f, tg);
    if (lamw) store_tile<HZ, NL, NP>(dlamp, g, l0, p0, vec_ok, tdl);
  }
}

// dx = lam * gsum (or gsum itself when it already holds sum_d lam_d g_d),
// dlam = x * gsum (unless written per direction), du = dy * hsum, hsum, or
// nothing (per-direction du), where hsum may come in up to three fp32 arrays
// (added in a fixed order).  Flat and elementwise; VEC: 8 elements a thread
// with 16-byte accesses (every pointer 16-byte aligned, n a multiple of 8).
template <typename T, int VEC>
__global__ void __launch_bounds__(256)
grad_finish_kernel(const T* __restrict__ x, const T* __restrict__ lam, const T* __restrict__ dy,
                   const float* __restrict__ gsum, const float* __restrict__ hsum,
                   const float* __restrict__ hsum2, const float* __restrict__ hsum3,
                   const T* __restrict__ dy2, const T* __restrict__ dy3,
                   T* __restrict__ dx, T* __restrict__ dlam, T* __restrict__ du, int64_t n,
                   int dx_mode, int du_mode) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x * VEC;
  for (int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * VEC; i < n; i += stride) {
    float gs[VEC], hs[VEC], a[VEC], o[VEC];
    ldv<VEC>(gsum + i, gs);
    if (dx_mode == 0) {
      ldv<VEC>(lam + i, a);
#pragma unroll
      for (int q = 0; q < VEC; ++q) o[q] = a[q] * gs[q];
      stv<VEC>(dx + i, o);
    } else {
      stv<VEC>(dx + i, gs);
    }
    if (dlam) {
      ldv<VEC>(x + i, a);
#pragma unroll
      for (int q = 0; q < VEC; ++q) o[q] = a[q] * gs[q];
      stv<VEC>(dlam + i, o);
    }
    if (du_mode == 2) continue;
    ldv<VEC>(hsum + i, hs);
    if (du_mode == 3) {
      // unmerged outputs: hsum already holds dy_d h_d of its directions; the
      // vertical ones are weighted by their own dy here
      float b[VEC];
      if (hsum2) {
        ldv<VEC>(hsum2 + i, a);
        ldv<VEC>(dy2 + i, b);
#pragma unroll
        for (int q = 0; q < VEC; ++q) hs[q] = fmaf(b[q], a[q], hs[q]);
      }
      if (hsum3) {
        ldv<VEC>(hsum3 + i, a);
        ldv<VEC>(dy3 + i, b);
#pragma unroll
        for (int q = 0; q < VEC; ++q) hs[q] = fmaf(b[q], a[q], hs[q]);
      }
      stv<VEC>(du + i, hs);
      continue;
    }
    if (hsum2) {
      ldv<VEC>(hsum2 + i, a);
#pragma unroll
      for (int q = 0; q < VEC; ++q) hs[q] += a[q];
    }
    if (hsum3) {
      ldv<VEC>(hsum3 + i, a);
#pragma unroll
      for (int q = 0; q < VEC; ++q) hs[q] += a[q];
    }
    if (du_mode == 0) {
      ldv<VEC>(dy + i, a);
#pragma unroll
      for (int q = 0; q < VEC; ++q) hs[q] *= a[q];
    }
    stv<VEC>(du + i, hs);
  }
}

// ---------------------------------------------------------------------------
// host-side launchers, instantiated once per element type
// ---------------------------------------------------------------------------
namespace stream_detail {

struct Shape {
  int np;  // positions per lane
  int nw;  // waves per line
};

inline Shape pick_shape(int P) {
  if (P <= 64) return {1, 1};
  if (P <= 128) return {2, 1};
  return {4, (P + 255) / 256};
}

inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// vector access is legal when every row start and base pointer is aligned to
// the vector (capped at 16 bytes) along the contiguous axis
inline bool vec_ok_for(bool hz, int np, int nl, int W, const void* const* ptrs, int nptr, size_t esz) {
  const int n = hz ? nl : np;
  const size_t bytes = (size_t)n * esz;
  const size_t need = bytes >= 16 ? 16 : bytes;
  if (W % n != 0) return false;
  for (int i = 0; i < nptr; ++i)
    if (ptrs[i] && !aligned(ptrs[i], need)) return false;
  return true;
}

// lines per tile: NL * NP = 8 elements per map keeps the tiles in registers at
// 1024 threads per workgroup (128 VGPRs)
template <int NP> constexpr int nl_for() { return 8 / NP; }

inline Geo make_geo(int H, int W, int dir) {
  Geo g;
  const bool hz = dir == DIR_L2R || dir == DIR_R2L;
  g.L = hz ? W : H;
  g.P = hz ? H : W;
  g.W = W;
  g.plane = (int64_t)H * W;
  g.rev = (dir == DIR_B2T || dir == DIR_R2L) ? 1 : 0;
  return g;
}

template <typename T, bool HZ, bool REV, int NP, int MODE, bool EXT>
hipError_t fwd_np(const StreamFwdParams& p, int64_t planes, int nw, hipStream_t st) {
  hipLaunchKernelGGL((stream_fwd_kernel<T, HZ, REV, NP, nl_for<NP>(), MODE, EXT>), dim3((unsigned)planes),
                     dim3(64 * nw), 0, st, p);
  return hipGetLastError();
}

template <typename T, bool HZ, bool REV, int MODE>
hipError_t fwd_mode(const StreamFwdArgs& a, const Geo& g) {
  const Shape s = pick_shape(g.P);
  const char* w = (const char*)a.w;
  const void* in[] = {a.x, a.lam, w, w + a.wstride * sizeof(T), w + 2 * a.wstride * sizeof(T), a.u, a.y,
                      a.dy, a.du};
  const void* fp[] = {a.acc, a.hprev_out};
  StreamFwdParams p{};
  p.x = a.x; p.lam = a.lam; p.w = a.w; p.wstride = a.wstride; p.u = a.u; p.acc = a.acc; p.y = a.y;
  p.hprev_out = a.hprev_out; p.dy = a.dy; p.du = a.du; p.first = a.first; p.g = g;
  p.vec_ok = vec_ok_for(HZ, s.np, 8 / s.np, g.W, in, 9, sizeof(T));
  p.vec_ok_f = vec_ok_for(HZ, s.np, 8 / s.np, g.W, fp, 2, sizeof(float));
  p.G = (a.group <= 0 || a.group >= g.L) ? g.L : a.group;
  p.logits = a.logits; p.renorm = a.renorm; p.ugate = a.ugate; p.hdy = a.hdy;
  const bool ext = a.logits || a.ugate || a.dy != nullptr;
  hipStream_t st = (hipStream_t)a.stream;
  switch (s.np) {
    case 1: return ext ? fwd_np<T, HZ, REV, 1, MODE, true>(p, a.planes, s.nw, st)
                       : fwd_np<T, HZ, REV, 1, MODE, false>(p, a.planes, s.nw, st);
    case 2: return ext ? fwd_np<T, HZ, REV, 2, MODE, true>(p, a.planes, s.nw, st)
                       : fwd_np<T, HZ, REV, 2, MODE, false>(p, a.planes, s.nw, st);
    default: return ext ? fwd_np<T, HZ, REV, 4, MODE, true>(p, a.planes, s.nw, st)
                        : fwd_np<T, HZ, REV, 4, MODE, false>(p, a.planes, s.nw, st);
  }
}

template <typename T, bool HZ, bool REV>
hipError_t fwd_dir(const StreamFwdArgs& a, const Geo& g) {
  switch (a.mode) {
    case MODE_STORE: return fwd_mode<T, HZ, REV, MODE_STORE>(a, g);
    case MODE_ADD: return fwd_mode<T, HZ, REV, MODE_ADD>(a, g);
    case MODE_FINAL: return fwd_mode<T, HZ, REV, MODE_FINAL>(a, g);
    default: return fwd_mode<T, HZ, REV, MODE_REC>(a, g);
  }
}

template <typename T, bool HZ, bool REV, int NP, bool EXT>
hipError_t adj_np(const StreamAdjParams& p, int64_t planes, int nw, hipStream_t st) {
  hipLaunchKernelGGL((stream_adj_kernel<T, HZ, REV, NP, nl_for<NP>(), EXT>), dim3((unsigned)planes),
                     dim3(64 * nw), 0, st, p);
  return hipGetLastError();
}

template <typename T, bool HZ, bool REV>
hipError_t adj_dir(const StreamAdjArgs& a, const Geo& g) {
  const Shape s = pick_shape(g.P);
  const char* w = (const char*)a.w;
  const char* dw = (const char*)a.dw;
  const void* in[] = {a.dy, a.u, w, w + a.wstride * sizeof(T), w + 2 * a.wstride * sizeof(T), dw,
                      dw + a.wstride * sizeof(T), dw + 2 * a.wstride * sizeof(T), a.lam, a.x, a.dlam};
  const void* fp[] = {a.hprev, a.gsum};
  StreamAdjParams p{};
  p.dy = a.dy; p.u = a.u; p.w = a.w; p.wstride = a.wstride; p.hprev = a.hprev; p.dw = a.dw;
  p.gsum = a.gsum; p.lam = a.lam; p.x = a.x; p.dlam = a.dlam; p.first = a.first; p.g = g;
  p.vec_ok = vec_ok_for(HZ, s.np, 8 / s.np, g.W, in, 11, sizeof(T));
  p.vec_ok_f = vec_ok_for(HZ, s.np, 8 / s.np, g.W, fp, 2, sizeof(float));
  p.G = (a.group <= 0 || a.group >= g.L) ? g.L : a.group;
  p.logits = a.logits; p.renorm = a.renorm; p.lamw = a.lamw;
  const bool ext = a.logits || a.lamw;
  hipStream_t st = (hipStream_t)a.stream;
  switch (s.np) {
    case 1: return ext ? adj_np<T, HZ, REV, 1, true>(p, a.planes, s.nw, st)
                       : adj_np<T, HZ, REV, 1, false>(p, a.planes, s.nw, st);
    case 2: return ext ? adj_np<T, HZ, REV, 2, true>(p, a.planes, s.nw, st)
                       : adj_np<T, HZ, REV, 2, false>(p, a.planes, s.nw, st);
    default: return ext ? adj_np<T, HZ, REV, 4, true>(p, a.planes, s.nw, st)
                        : adj_np<T, HZ, REV, 4, false>(p, a.planes, s.nw, st);
  }
}

}  // namespace stream_detail

template <typename T>
hipError_t stream_fwd_pass_t(const StreamFwdArgs& a) {
  using namespace stream_detail;
  const Geo g = make_geo(a.H, a.W, a.dir);
  switch (a.dir) {
    case DIR_T2B: return fwd_dir<T, false, false>(a, g);
    case DIR_B2T: return fwd_dir<T, false, true>(a, g);
    case DIR_L2R: return fwd_dir<T, true, false>(a, g);
    default: return fwd_dir<T, true, true>(a, g);
  }
}

template <typename T>
hipError_t stream_adj_pass_t(const StreamAdjArgs& a) {
  using namespace stream_detail;
  const Geo g = make_geo(a.H, a.W, a.dir);
  switch (a.dir) {
    case DIR_T2B: return adj_dir<T, false, false>(a, g);
    case DIR_B2T: return adj_dir<T, false, true>(a, g);
    case DIR_L2R: return adj_dir<T, true, false>(a, g);
    default: return adj_dir<T, true, true>(a, g);
  }
}

template <typename T>
hipError_t grad_finish_t(const GradFinishArgs& a) {
  const int64_t n = a.n;
  bool vec = n % 8 == 0;
  for (const void* q : {(const void*)a.x, (const void*)a.lam, (const void*)a.dy, (const void*)a.gsum,
                        (const void*)a.hsum, (const void*)a.hsum2, (const void*)a.hsum3, a.dy2, a.dy3,
                        (const void*)a.dx, (const void*)a.dlam, (const void*)a.du})
    if ((uintptr_t)q % 16) vec = false;
  const int per = vec ? 8 : 1;
  int64_t blocks = (n / per + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  auto kern = vec ? grad_finish_kernel<T, 8> : grad_finish_kernel<T, 1>;
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)a.stream,
                     (const T*)a.x, (const T*)a.lam, (const T*)a.dy, a.gsum, a.hsum, a.hsum2, a.hsum3,
                     (const T*)a.dy2, (const T*)a.dy3, (T*)a.dx, (T*)a.dlam, (T*)a.du, n, a.dx_mode,
                     a.du_mode);
  return hipGetLastError();
}

}  // namespace gspn
