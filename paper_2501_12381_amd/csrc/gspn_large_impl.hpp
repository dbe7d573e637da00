// Two-pass forward for planes too large to keep on chip (e.g. 2048 x 2048).
//
// The four directions cannot share one sweep (their dependency orders
// conflict), so sum_d h_d goes through an fp32 workspace `acc` twice:
//
//   pass V  (one launch): a workgroup per plane; half of its waves run
//           top-to-bottom, the other half bottom-to-top.  A row is spread over
//           the waves of its direction, each lane owning 32 bytes of
//           positions; the three-way neighbours come from the adjacent lanes
//           (DPP) and, at wave edges, from an LDS exchange with one barrier per
//           row.  Each direction stores h for the rows it reaches first; after
//           the middle row it adds its h to what the other direction stored.
//   pass H  (one launch per block of K columns, K = 128 bytes of a row):
//           left-to-right and right-to-left.  A workgroup owns a band of rows
//           plus a halo of K rows on each side that has a neighbouring band
//           (the first and last bands keep K more rows instead), one row per
//           lane, and holds the
//           block's K columns of each input as 128-byte row segments in
//           registers, so every cache line of a row is read by one load.
//           Starting from the exact state of the previous block (a column of
//           h per direction, passed between launches in a small workspace),
//           the halo rows shrink the exact region by one row per column and
//           leave it equal to the band after K columns.  The band's h goes to
//           LDS and is added to acc (first half of the blocks) or combined
//           into y = u * (acc + h) (second half) with coalesced accesses.
//
// Both passes pair opposite directions with the same middle-line rule as the
// resident kernels, so every addition happens in a fixed order and results
// are reproducible run to run.
#pragma once

#include "gspn_device.hpp"
#include "gspn_launch.hpp"
#include "gspn_resident_impl.hpp"

namespace gspn {

template <typename T>
struct LargeCfg {
  static constexpr int VE = 16 / (int)sizeof(T);   // elements per 16-byte vector
  static constexpr int NPV = 2 * VE;               // vertical: positions per lane (32 bytes)
  static constexpr int RV = 2;                     // vertical prefetch depth of the inputs (rows)
  static constexpr int RA = 2;                     // ... of acc and u in the second half
  static constexpr int KH = 128 / (int)sizeof(T);  // horizontal block: columns per launch
  static constexpr int HV = KH / VE;               // 16-byte vectors per row segment
  static constexpr int HROWS = 512;                // rows (lanes) per horizontal workgroup
  static constexpr int MAX_WPD = 4;                // vertical: waves per direction
  static constexpr int MAX_W = MAX_WPD * 64 * NPV; // widest row of the vertical pass
};

// ---------------------------------------------------------------------------
// pass V
// ---------------------------------------------------------------------------
struct LargeVParams {
  const void* x;
  const void* lam;
  const void* w;     // packed [n][3][planes][H][W]
  const void* u;
  void* y;
  float* acc;
  int64_t planes, npc;
  int H, W;
  int slot0, slot1;  // weight slot of top-to-bottom / bottom-to-top, -1 when absent
  int final_out;     // nonzero: write y = u * sum; zero: write the fp32 partial sum
  float* acc_b;      // split: the grid holds both directions as separate workgroups
                     // (blockIdx / planes), bottom-to-top writing its h here
  int split;
  int grp;           // rows per local-GSPN group (H: the global scan)
  int renorm;        // Eq. 6 logits (LG kernels): normalise over on-line neighbours only
  int y_pd;          // unmerged outputs: y is (n, B, C, H, W), this direction's map at slot * npc
};

// Layout of a row over a wave: the wave's span of 64 * NP positions is cut into
// NQ chunks of 64 * G positions; lane l holds positions [l G, l G + G) of every
// chunk.  Each load or store instruction then covers one chunk: consecutive
// lanes, consecutive addresses, whole cache lines (bf16 and fp32 alike).  The
// left neighbour of a chunk's first position is lane 63's last one of the
// previous chunk (a lane read), of the previous wave (LDS) or padding.
//
// BOTH: both vertical directions are present; FIN: write y (no pass H follows).
// LG: the weight maps hold Eq. 6 logits, normalised as they are unpacked.
template <typename T, int WPD, bool BOTH, bool FIN, bool LG>
__device__ __forceinline__ void large_v_body(const LargeVParams& p) {
  using C = LargeCfg<T>;
  constexpr int NP = C::NPV, R = C::RV, RA = C::RA;
  static_assert(R % RA == 0, "acc ring slots must repeat with the input ring");
  constexpr int G = 4;           // positions per lane and chunk
  constexpr int NQ = NP / G;     // chunks per wave span
  constexpr int SPAN = 64 * G;   // positions per chunk
  typedef Pack<T, G> PK;
  __shared__ float edge[2][2 * WPD][2];  // [step parity][wave][first, last position]

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr bool both = BOTH, fin = FIN;
  const int dir = both ? (wave >= WPD ? 1 : 0) : (p.split ? (blockIdx.x >= p.planes ? 1 : 0) : (p.slot0 >= 0 ? 0 : 1));
  const int wi = both ? wave - dir * WPD : wave;
  const int64_t plane = p.split && dir ? blockIdx.x - p.planes : blockIdx.x;
  float* const accw = p.split && dir ? p.acc_b : p.acc;  // where a single direction's h goes
  const int H = p.H, W = p.W;
  // per chunk: position of the lane's first element, whether it is in the row
  int po[NQ];
  bool qok[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int pos = wi * NQ * SPAN + q * SPAN + lane * G;
    qok[q] = pos < W;  // W is a multiple of G
    po[q] = qok[q] ? pos : 0;
  }
  const int64_t pb = plane * (int64_t)H * W;
  const int slot = dir ? p.slot1 : p.slot0;
  const int odd = both ? (H & 1) : 0;
  const int nsteps = H + odd;
  const int sm = both ? H / 2 + odd : nsteps;  // first step of the second half
  const int delay = dir ? odd : 0;             // bottom-to-top starts a step late for odd H

  for (int i = threadIdx.x; i < 2 * 2 * WPD * 2; i += blockDim.x) (&edge[0][0][0])[i] = 0.f;
  __syncthreads();

  const T* w0 = (const T*)p.w + (int64_t)slot * 3 * p.npc;
  const T* base[5] = {(const T*)p.x + pb, (const T*)p.lam + pb, w0 + pb, w0 + p.npc + pb,
                      w0 + 2 * p.npc + pb};
  const T* ubase = (const T*)p.u + pb;
  const float* abase = p.acc + pb;

  auto t_of = [&](int s) { return s - delay; };
  auto line_of = [&](int t) {
    t = t < 0 ? 0 : (t >= H ? H - 1 : t);
    return dir ? H - 1 - t : t;
  };

  PK ring[R][5][NQ];
  // Keeps the last prefetches "used" after a loop: without a use the compiler
  // drains every outstanding load at the top of each iteration.
  auto consume_ring = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < R; ++k)
#pragma unroll
      for (int m = 0; m < 5; ++m)
#pragma unroll
        for (int q = 0; q < NQ; ++q)
#pragma unroll
          for (int i = 0; i < PK::kWords; ++i) asm volatile("" ::"v"(ring[k][m][q].w[i]));
  };
  auto load_main = [&](PK (&sl)[5][NQ], int s) __attribute__((always_inline)) {
    const int64_t off = (int64_t)line_of(t_of(s)) * W;
#pragma unroll
    for (int m = 0; m < 5; ++m)
#pragma unroll
      for (int q = 0; q < NQ; ++q) sl[m][q].load(base[m] + off + po[q]);
  };
  // second-half (or final single-direction) operands: acc and u of the step's row
  PK uring[RA][NQ];
  float aring[RA][NQ][G];
  auto load_aux = [&](int k, int s) __attribute__((always_inline)) {
    const int64_t off = (int64_t)line_of(t_of(s)) * W;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      if constexpr (fin) uring[k][q].load(ubase + off + po[q]);
      if constexpr (both) ldv<G>(abase + off + po[q], aring[k][q]);
    }
  };

  float hp[NQ][G];
#pragma unroll
  for (int q = 0; q < NQ; ++q)
#pragma unroll
    for (int j = 0; j < G; ++j) hp[q][j] = 0.f;

  // one step of the scan; SECOND: combine with the other direction's stored h
  auto step = [&](auto second_tag, int k, int s) __attribute__((always_inline)) {
    constexpr bool SECOND = decltype(second_tag)::value;
    const PK(&v)[5][NQ] = ring[k];  // unpacked at use; the slot is refilled after the step
    const int t = t_of(s);
    const bool act = t >= 0 && t < H;
    const int par = s & 1;
    // local GSPN: the first row of a group starts from a zero state (uniform per direction)
    const bool rst = act && group_start(line_of(t), p.grp, dir != 0);
    if (rst) {
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int j = 0; j < G; ++j) hp[q][j] = 0.f;
    }
    // neighbours of each chunk's first and last position on the previous row
    float el[NQ], er[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      el[q] = from_prev_lane(hp[q][G - 1]);
      er[q] = from_next_lane(hp[q][0]);
    }
    float wl = 0.f, wr = 0.f;  // across waves
    if constexpr (WPD > 1) {
      const float nl = edge[par ^ 1][wi > 0 ? wave - 1 : wave][1];
      const float nr = edge[par ^ 1][wi < WPD - 1 ? wave + 1 : wave][0];
      wl = (wi > 0 && !rst) ? nl : 0.f;
      wr = (wi < WPD - 1 && !rst) ? nr : 0.f;
    }
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const float pl = q > 0 ? __builtin_bit_cast(float, __builtin_amdgcn_readlane(
                                                              __builtin_bit_cast(int, hp[q - 1][G - 1]), 63))
                             : wl;
      const float nr = q < NQ - 1 ? __builtin_bit_cast(float, __builtin_amdgcn_readlane(
                                                                   __builtin_bit_cast(int, hp[q + 1][0]), 0))
                                  : wr;
      if (lane == 0) el[q] = pl;
      if (lane == 63) er[q] = nr;
    }
    float h[NQ][G];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const bool ok = qok[q] && act;
#pragma unroll
      for (int j = 0; j < G; ++j) {
        const float hl = j == 0 ? el[q] : hp[q][j - 1];
        const float hr = j == G - 1 ? er[q] : hp[q][j + 1];
        float wa = v[2][q].get(j), wb = v[3][q].get(j), wc = v[4][q].get(j);
        if constexpr (LG) {
          const Norm3 nr = normalize3(wa, wb, wc, po[q] + j == 0, po[q] + j == W - 1, p.renorm != 0);
          wa = nr.w[0];
          wb = nr.w[1];
          wc = nr.w[2];
        }
        float r = v[1][q].get(j) * v[0][q].get(j);
        r = fmaf(wa, hl, r);
        r = fmaf(wb, hp[q][j], r);
        r = fmaf(wc, hr, r);
        h[q][j] = ok ? r : 0.f;
      }
    }
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int j = 0; j < G; ++j) hp[q][j] = h[q][j];
    // the new h is materialised before anything below, so the refills of the
    // ring slots land in the registers just consumed and no loop-carried copy
    // (which would wait for the loads) is needed
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int j = 0; j < G; ++j) asm volatile("" : "+v"(hp[q][j]));
    if (lane == 0) edge[par][wave][0] = hp[0][0];
    if (lane == 63) edge[par][wave][1] = hp[NQ - 1][G - 1];
    if (act) {
      const int64_t off = (int64_t)line_of(t) * W;
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        if (!qok[q]) continue;
        if constexpr (SECOND) {
          const int ka = k % RA;
          float o[G];
#pragma unroll
          for (int j = 0; j < G; ++j) o[j] = (both ? aring[ka][q][j] : 0.f) + hp[q][j];
          if constexpr (fin) {
#pragma unroll
            for (int j = 0; j < G; ++j) o[j] *= uring[ka][q].get(j);
            stv<G>((T*)p.y + (p.y_pd ? (int64_t)slot * p.npc : 0) + pb + off + po[q], o);
          } else {
            stv<G>(p.acc + pb + off + po[q], o);
          }
        } else {
          stv<G>(accw + pb + off + po[q], hp[q]);
        }
      }
    }
    // refills come after the stores, which they may alias, so they stay here
    asm volatile("" ::: "memory");
    load_main(ring[k], s + R);
    if constexpr (SECOND) load_aux(k % RA, s + RA);
    lds_barrier();
  };

  // Steps [.., s1) store h (the first half of a pair, or a single direction
  // that feeds pass H); steps [s1, nsteps) combine with the stored sum.  Idle
  // steps before step 0 and after the last one align both loops to the ring,
  // so every load is unconditional and stays in flight across steps.
  constexpr bool single_final = !both && fin;
  const int s1 = single_final ? 0 : sm;
  const int o = (R - s1 % R) % R;
#pragma unroll
  for (int k = 0; k < R; ++k) load_main(ring[k], k - o);
  for (int s0 = -o; s0 < s1; s0 += R) {
#pragma unroll
    for (int k = 0; k < R; ++k) step(std::false_type{}, k, s0 + k);
  }
  if (s1 >= nsteps) {
    consume_ring();
    return;
  }
  // the other direction's stores of the first half must be visible
  __syncthreads();
#pragma unroll
  for (int k = 0; k < RA; ++k) load_aux(k, s1 + k);
  // the first turn of the ring is peeled so that the loop is entered with the
  // loads in flight in the same order as in its steady state (otherwise the
  // waits at its top follow the order of the preloads and drain the ring)
#pragma unroll
  for (int k = 0; k < R; ++k) step(std::true_type{}, k, s1 + k);
  for (int s0 = s1 + R; s0 < nsteps; s0 += R) {
#pragma unroll
    for (int k = 0; k < R; ++k) step(std::true_type{}, k, s0 + k);
  }
  consume_ring();
#pragma unroll
  for (int k = 0; k < RA; ++k)
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      if constexpr (both) {
#pragma unroll
        for (int j = 0; j < G; ++j) asm volatile("" ::"v"(aring[k][q][j]));
      }
      if constexpr (fin) {
#pragma unroll
        for (int i = 0; i < PK::kWords; ++i) asm volatile("" ::"v"(uring[k][q].w[i]));
      }
    }
}

template <typename T, int WPD, bool BOTH, bool FIN, bool LG>
__global__ void __launch_bounds__(128 * WPD, 2) large_v_kernel(LargeVParams p) {
  large_v_body<T, WPD, BOTH, FIN, LG>(p);
}
// the same pass as the backward's recompute of the vertical directions' h
// (its own name in kernel traces and counter profiles)
template <typename T, int WPD, bool BOTH, bool FIN, bool LG>
__global__ void __launch_bounds__(128 * WPD, 2) large_vrec_kernel(LargeVParams p) {
  large_v_body<T, WPD, BOTH, FIN, LG>(p);
}

// ---------------------------------------------------------------------------
// pass H
// ---------------------------------------------------------------------------
struct LargeHParams {
  const void* x;
  const void* lam;
  const void* w;
  const void* u;
  void* y;
  float* acc;
  float* state;       // [2 parities][2 directions][planes][H]
  int64_t planes, npc;
  int H, W;
  int slot0, slot1;   // weight slot of left-to-right / right-to-left, -1 when absent
  int step;           // launch index
  int nblk;           // column blocks
  int delay;          // right-to-left starts one launch late (odd block count, both present)
  int half;           // first launch of the second half (pairs)
  // bands: the first and last keep edge_rows rows (one halo each), the others
  // band_rows (halo rows above and below); one band keeps the whole plane
  int band_rows, edge_rows, nbands, halo;
  int has_v;          // acc holds the vertical pass's partial sum
  const float* acc_b; // non-null: the vertical sum is acc + acc_b until the first horizontal direction adds
  // local GSPN, per direction (left-to-right, right-to-left): bit i set when
  // window column i of this launch starts a group (the state restarts from zero)
  uint64_t gmask[2];
  // recompute step of the backward (one direction): acc (+)= h, and h itself
  // to hbuf; nothing is multiplied by u
  int rec;
  float* hbuf;
  int renorm;         // Eq. 6 logits (LG kernels): normalise over on-line neighbours only
  // unmerged outputs: each direction writes y_d = u * h_d to its own map
  // (slot * npc); nothing is combined
  int y_pd;
  // rec mode with unmerged outputs: acc (+)= dy_d * h instead of h (dy_d: this
  // direction's output gradient), the sum du needs
  const void* hdy;
  // forward keeping its state for the backward: the partial and final sums go
  // to `sum` (acc keeps the vertical pass's h), each direction's h to hsave[dir]
  float* sum;
  float* hsave[2];
};

// LG: the weight maps hold Eq. 6 logits, normalised as they are unpacked.
template <typename T, int NW, bool LG>
__device__ __forceinline__ void large_h_body(const LargeHParams& p) {
  using C = LargeCfg<T>;
  constexpr int K = C::KH, HV = C::HV, VE = C::VE, KP = K + 1;
  typedef Pack<T, VE> PK;
  // [edge_rows][KP] h of the band; edges [2 parities][NW + 2][2]: wave w's first
  // and last rows at slot w + 1, zeros at slots 0 and NW + 1 (no neighbour
  // wave); 64 dummy slots
  extern __shared__ float lds[];
  float* edge = lds + p.edge_rows * KP;
  constexpr int ES = (NW + 2) * 2;  // floats per parity

  // workgroup -> (direction, plane, band); consecutive ids (the bands of a plane,
  // which share halo rows) are placed on the same XCD
  const int64_t G = gridDim.x, b = blockIdx.x;
  const int64_t G8 = G / 8 * 8;
  int64_t id = b < G8 ? (b % 8) * (G8 / 8) + b / 8 : b;
  const int band = (int)(id % p.nbands);
  id /= p.nbands;
  const int64_t plane = id % p.planes;
  const int dsel = (int)(id / p.planes);
  const bool both = p.slot0 >= 0 && p.slot1 >= 0;
  const int dir = both ? dsel : (p.slot0 >= 0 ? 0 : 1);  // 0: left-to-right, 1: right-to-left
  const int slot = dir ? p.slot1 : p.slot0;
  const int seq = dir ? p.step - p.delay : p.step;         // position in this direction's order
  if (seq < 0 || seq >= p.nblk) return;
  const int blk = dir ? p.nblk - 1 - seq : seq;
  const int H = p.H, W = p.W;
  // window of K columns: the block itself, or the last K columns for a short last block
  const int c0 = blk * K;
  const int ws = c0 + K <= W ? c0 : W - K;
  const int lo = c0 - ws;  // first valid column of the window

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // kept rows [bs, be) of the band; halo rows only towards a neighbouring band,
  // so every lane in use holds a row of the plane
  const bool last = band == p.nbands - 1;
  const int bs = band == 0 ? 0 : p.edge_rows + (band - 1) * p.band_rows;
  const int be = last ? H : min(H, bs + (band == 0 ? p.edge_rows : p.band_rows));
  const int htop = band == 0 ? 0 : p.halo;
  const int used = be - bs + htop + (last ? 0 : p.halo);
  // lanes past the band and its halos duplicate the last row in use (no traffic)
  const int r = bs - htop + (tid < used ? tid : used - 1);
  const bool row_ok = tid < used && r >= 0 && r < H;
  const int rc = r < 0 ? 0 : (r >= H ? H - 1 : r);
  const int br = r - bs;  // row inside the band
  const bool in_band = row_ok && br >= 0 && br < be - bs;

  const int64_t HW = (int64_t)H * W;
  const int64_t rb = plane * HW + (int64_t)rc * W + ws;
  const T* w0 = (const T*)p.w + (int64_t)slot * 3 * p.npc;
  const T* base[5] = {(const T*)p.x + rb, (const T*)p.lam + rb, w0 + rb, w0 + p.npc + rb,
                      w0 + 2 * p.npc + rb};
  // state of the previous block first: it is needed before any column
  const int64_t sdir = (int64_t)dir * p.planes * H + plane * H;
  float hp = 0.f;
  if (seq > 0) {
    const float* sin = p.state + (int64_t)((p.step - 1) & 1) * 2 * p.planes * H + sdir;
    hp = sin[rc];
  }
  hp = row_ok ? hp : 0.f;
  if (lane == 0) edge[ES + (wave + 1) * 2 + 0] = hp;
  if (lane == 63) edge[ES + (wave + 1) * 2 + 1] = hp;
  if (tid < 4) edge[(tid >> 1) * ES + (tid & 1) * ((NW + 1) * 2)] = 0.f;  // slots 0 and NW + 1, first row
  if (tid >= 4 && tid < 8) edge[((tid - 4) >> 1) * ES + ((tid - 4) & 1) * ((NW + 1) * 2) + 1] = 0.f;  // ... last row

  float* hrow = lds + (in_band ? br : 0) * KP;
  // edge slot of this lane per step parity: lanes 0 and 63 publish their row's
  // h for the neighbouring waves, the other lanes write a private dummy slot
  auto eslot = [&](int par) {
    return lane == 0 ? par * ES + (wave + 1) * 2 : (lane == 63 ? par * ES + (wave + 1) * 2 + 1 : 2 * ES + lane);
  };
  const int eo0 = eslot(0), eo1 = eslot(1);
  // epilogue operands: the first UP vectors of each thread are requested
  // during the scan, one each time a tile vector of every map has been used
  // up (the registers it frees hold them), so the epilogue finds them in
  // registers and the workgroup keeps loads in flight while it scans
  const bool second = both && p.step >= p.half && !p.y_pd;
  const bool fin = !p.rec && (!both || second || p.y_pd);
  const bool read_acc = (second || p.has_v) && !p.y_pd;
  const bool add_b = p.acc_b != nullptr && !second && !p.y_pd;  // the vertical sum still lives in two arrays
  T* const yout = (T*)p.y + (p.y_pd ? (int64_t)slot * p.npc : 0);
  const T* const hdy = (const T*)p.hdy;
  // the partial sum this launch adds to and where its result goes: acc, or
  // with a kept state the separate sum array (acc keeps the vertical h)
  const float* const acc_in = (second && p.sum) ? p.sum : p.acc;
  float* const acc_out = p.sum ? p.sum : p.acc;
  float* const hout = p.rec ? p.hbuf : p.hsave[dir];  // this direction's h, when kept
  const int rows = be - bs;
  const int nvr = (K - lo) / VE;
  const int n = rows * nvr;
  const int64_t ob = plane * HW + (int64_t)bs * W + ws;
  constexpr int TT = 64 * NW, UP = HV - 1;
  float pav[UP][VE], pbv[UP][VE];
  Pack<T, VE> puv[UP];
  auto prefetch = [&](int k) __attribute__((always_inline)) {
    const int e = tid + k * TT < n ? tid + k * TT : 0;
    const int rr = e / nvr, cc = lo + (e - rr * nvr) * VE;
    const int64_t o = ob + (int64_t)rr * W + cc;
    if (read_acc) ldv<VE>(acc_in + o, pav[k]);
    if (add_b) ldv<VE>(p.acc_b + o, pbv[k]);
    if (fin) puv[k].load((const T*)p.u + o);
    if (hdy) puv[k].load(hdy + o);  // rec mode: the direction's dy (u is not needed there)
  };

  const uint64_t gm = p.gmask[dir];
  auto scan = [&](auto rev_tag) __attribute__((always_inline)) {
    constexpr bool REV = decltype(rev_tag)::value;
    // the tile is loaded map by map, each row segment's vectors back to back:
    // a lane's 128-byte line is then requested by consecutive instructions and
    // is still in the L1 for all of them (vector-major order, which would let
    // the first columns start earlier, re-fetches each line from L2 once per
    // vector).  Scheduling barriers keep this issue order.
    PK tile[5][HV];
#pragma unroll
    for (int m = 0; m < 5; ++m) {
#pragma unroll
      for (int i = 0; i < HV; ++i) {
        const int v = REV ? HV - 1 - i : i;
        tile[m][v].load(base[m] + v * VE);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    lds_barrier();  // initial edges published
    auto step = [&](auto ic) __attribute__((always_inline)) {
      constexpr int i = decltype(ic)::value;
      const int ti = REV ? K - 1 - i : i;  // window column of this step
      if (ti < lo) return;                 // short last block (uniform)
      const int par = i & 1;
      // neighbours from the adjacent waves (zero slots past the first and last)
      float nu = 0.f, nd = 0.f;
      if constexpr (NW > 1) {
        nu = edge[(par ^ 1) * ES + wave * 2 + 1];
        nd = edge[(par ^ 1) * ES + (wave + 2) * 2 + 0];
      }
      if ((gm >> ti) & 1) {  // this column starts a group: the state restarts (uniform)
        hp = 0.f;
        nu = 0.f;
        nd = 0.f;
      }
      const float up = from_prev_lane_or(hp, nu), dn = from_next_lane_or(hp, nd);
      const float xv = tile[0][ti / VE].get(ti % VE), lv = tile[1][ti / VE].get(ti % VE);
      float a = tile[2][ti / VE].get(ti % VE), bw = tile[3][ti / VE].get(ti % VE),
            cw = tile[4][ti / VE].get(ti % VE);
      if constexpr (LG) {
        const Norm3 nr = normalize3(a, bw, cw, r == 0, r == H - 1, p.renorm != 0);
        a = nr.w[0];
        bw = nr.w[1];
        cw = nr.w[2];
      }
      float h = lv * xv;
      h = fmaf(a, up, h);
      h = fmaf(bw, hp, h);
      h = fmaf(cw, dn, h);
      hp = row_ok ? h : 0.f;
      edge[par ? eo1 : eo0] = hp;  // one store for every lane (no branch per step)
      if (in_band) hrow[ti] = hp;
      lds_barrier();
    };
    // the steps unrolled; after every VE of them the epilogue's next vector
    static_for<0, K>([&](auto ic) __attribute__((always_inline)) {
      step(ic);
      constexpr int i = decltype(ic)::value;
      if constexpr ((i + 1) % VE == 0 && (i + 1) / VE - 1 < UP) prefetch((i + 1) / VE - 1);
    });
  };
  if (dir) scan(std::true_type{});
  else scan(std::false_type{});
  if (in_band) p.state[(int64_t)(p.step & 1) * 2 * p.planes * H + sdir + r] = hp;
  __syncthreads();

  // combine the band's h with acc: y = u * (acc + h) or acc + h, one 16-byte
  // vector of T (VE columns) a thread: first the prefetched vectors, then any
  // beyond them in batches whose loads are all issued before any is used
  auto combine = [&](int e, const float* av, const float* bv, const Pack<T, VE>& uv) __attribute__((always_inline)) {
    const int rr = e / nvr, cc = lo + (e - rr * nvr) * VE;
    const int64_t o = ob + (int64_t)rr * W + cc;
    float s[VE];
#pragma unroll
    for (int q = 0; q < VE; ++q) {
      const float hv = hdy ? lds[rr * KP + cc + q] * uv.get(q) : lds[rr * KP + cc + q];
      s[q] = (read_acc ? (add_b ? av[q] + bv[q] : av[q]) : 0.f) + hv;
    }
    if (hout) stv<VE>(hout + o, lds + rr * KP + cc);
    if (fin) {
      if (p.sum) stv<VE>(p.sum + o, s);  // sum_d h_d, kept for the backward
#pragma unroll
      for (int q = 0; q < VE; ++q) s[q] *= uv.get(q);
      stv<VE>(yout + o, s);
    } else {
      stv<VE>(acc_out + o, s);
    }
  };
#pragma unroll
  for (int k = 0; k < UP; ++k)
    if (tid + k * TT < n) combine(tid + k * TT, pav[k], pbv[k], puv[k]);
  constexpr int U = 8;
  for (int e0 = tid + UP * TT; e0 < n; e0 += TT * U) {
    float av[U][VE], bv[U][VE];
    Pack<T, VE> uv[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int e = e0 + k * TT < n ? e0 + k * TT : e0;
      const int rr = e / nvr, cc = lo + (e - rr * nvr) * VE;
      const int64_t o = ob + (int64_t)rr * W + cc;
      if (read_acc) ldv<VE>(acc_in + o, av[k]);
      if (add_b) ldv<VE>(p.acc_b + o, bv[k]);
      if (fin) uv[k].load((const T*)p.u + o);
      if (hdy) uv[k].load(hdy + o);
    }
#pragma unroll
    for (int k = 0; k < U; ++k)
      if (e0 + k * TT < n) combine(e0 + k * TT, av[k], bv[k], uv[k]);
  }
}

template <typename T, int NW, bool LG>
__global__ void __launch_bounds__(64 * NW) large_h_kernel(LargeHParams p) {
  large_h_body<T, NW, LG>(p);
}
// the same pass in its `rec` mode: the backward's recompute of a horizontal
// direction's h (its own name in kernel traces and counter profiles)
template <typename T, int NW, bool LG>
__global__ void __launch_bounds__(64 * NW) large_hrec_kernel(LargeHParams p) {
  large_h_body<T, NW, LG>(p);
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
template <typename T>
inline bool large_fwd_supported(int H, int W) {
  using C = LargeCfg<T>;
  return H >= 1 && W >= C::KH && W % C::VE == 0 && W <= C::MAX_W;
}

template <typename T>
struct LargeGeom {
  int wpd;        // vertical: waves per direction (power of two)
  // horizontal bands (forward, recompute and adjoint): the first and last keep
  // hb_edge rows (one halo of `halo` rows), the others hb_mid (two halos)
  int hb_n, hb_mid, hb_edge, hb_nw, halo;
  int nblk;
  size_t lds_hb;  // dynamic LDS of pass H
};

template <typename T>
inline LargeGeom<T> large_geom(int H, int W) {
  using C = LargeCfg<T>;
  LargeGeom<T> g{};
  const int need = (W + 64 * C::NPV - 1) / (64 * C::NPV);
  g.wpd = 1;
  while (g.wpd < need) g.wpd *= 2;
  if (H <= C::HROWS) {
    g.hb_n = 1;
    g.hb_mid = g.hb_edge = H;
    g.halo = 0;
  } else {
    // every band takes HROWS lanes, the kept rows balanced over the bands
    g.hb_n = (H - 2 * C::KH + C::HROWS - 2 * C::KH - 1) / (C::HROWS - 2 * C::KH);
    g.hb_mid = (H - 2 * C::KH + g.hb_n - 1) / g.hb_n;
    g.hb_edge = g.hb_mid + C::KH;
    g.halo = C::KH;
  }
  g.hb_nw = ((g.hb_n == 1 ? H : g.hb_mid + 2 * C::KH) + 63) / 64;  // lanes: kept rows and halos
  g.nblk = (W + C::KH - 1) / C::KH;
  g.lds_hb = ((size_t)g.hb_edge * (C::KH + 1) + 4 * (8 + 2) + 64) * sizeof(float);  // h, edges, dummy slots
  return g;
}

template <typename T, int WPD, bool BOTH, bool FIN>
hipError_t launch_large_v_mode(const LargeVParams& p, bool rec, bool lg, hipStream_t st) {
  auto kern = lg ? (rec ? large_vrec_kernel<T, WPD, BOTH, FIN, true> : large_v_kernel<T, WPD, BOTH, FIN, true>)
                 : (rec ? large_vrec_kernel<T, WPD, BOTH, FIN, false> : large_v_kernel<T, WPD, BOTH, FIN, false>);
  hipLaunchKernelGGL(kern, dim3((unsigned)(p.planes * (p.split ? 2 : 1))), dim3((BOTH ? 128 : 64) * WPD), 0, st,
                     p);
  return hipGetLastError();
}

// rec: the backward's recompute (same kernel under its own name); lg: the
// weight maps hold Eq. 6 logits
template <typename T, int WPD>
hipError_t launch_large_v(const LargeVParams& p, bool both, hipStream_t st, bool rec, bool lg) {
  if (both) return p.final_out ? launch_large_v_mode<T, WPD, true, true>(p, rec, lg, st)
                               : launch_large_v_mode<T, WPD, true, false>(p, rec, lg, st);
  return p.final_out ? launch_large_v_mode<T, WPD, false, true>(p, rec, lg, st)
                     : launch_large_v_mode<T, WPD, false, false>(p, rec, lg, st);
}

template <typename T, int NW>
hipError_t launch_large_h_nw(const LargeHParams& p, int64_t grid, size_t lds, bool lg, hipStream_t st) {
  auto kern = lg ? (p.rec ? large_hrec_kernel<T, NW, true> : large_h_kernel<T, NW, true>)
                 : (p.rec ? large_hrec_kernel<T, NW, false> : large_h_kernel<T, NW, false>);
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(64 * NW), lds, st, p);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_large_h(const LargeHParams& p, int nw, int64_t grid, size_t lds, bool lg, hipStream_t st) {
  switch (nw) {
    case 1: return launch_large_h_nw<T, 1>(p, grid, lds, lg, st);
    case 2: return launch_large_h_nw<T, 2>(p, grid, lds, lg, st);
    case 3: return launch_large_h_nw<T, 3>(p, grid, lds, lg, st);
    case 4: return launch_large_h_nw<T, 4>(p, grid, lds, lg, st);
    case 5: return launch_large_h_nw<T, 5>(p, grid, lds, lg, st);
    case 6: return launch_large_h_nw<T, 6>(p, grid, lds, lg, st);
    case 7: return launch_large_h_nw<T, 7>(p, grid, lds, lg, st);
    case 8: return launch_large_h_nw<T, 8>(p, grid, lds, lg, st);
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t large_fwd_t(const LargeFwdArgs& a) {
  using C = LargeCfg<T>;
  if (!large_fwd_supported<T>(a.H, a.W)) return hipErrorInvalidValue;
  const LargeGeom<T> g = large_geom<T>(a.H, a.W);
  hipStream_t st = (hipStream_t)a.stream;
  const int64_t npc = a.planes * (int64_t)a.H * a.W;
  int slot[4], n = 0;
  for (int d = 0; d < 4; ++d) slot[d] = (a.mask >> d) & 1 ? n++ : -1;
  const bool has_v = slot[0] >= 0 || slot[1] >= 0, has_h = slot[2] >= 0 || slot[3] >= 0;

  if (has_v) {
    LargeVParams v{};
    v.x = a.x; v.lam = a.lam; v.w = a.w; v.u = a.u; v.y = a.y; v.acc = a.acc;
    v.planes = a.planes; v.npc = npc; v.H = a.H; v.W = a.W;
    v.slot0 = slot[0]; v.slot1 = slot[1];
    v.final_out = has_h ? 0 : 1;
    // both vertical directions feeding a horizontal pass: twice the workgroups,
    // one direction each, each with its own partial sum (no midpoint pairing,
    // so the grid has no partly filled last round of whole planes)
    v.grp = (a.group_h > 0 && a.group_h < a.H) ? a.group_h : a.H;
    v.split = slot[0] >= 0 && slot[1] >= 0 && has_h && a.acc_b != nullptr;
    v.renorm = a.renorm;
    if (a.y_pd) {
      // unmerged outputs: every direction writes its own y, nothing is summed
      v.final_out = 1;
      v.split = slot[0] >= 0 && slot[1] >= 0;
      v.y_pd = 1;
    }
    v.acc_b = a.acc_b;
    if (v.split && 2 * a.planes > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const bool both = slot[0] >= 0 && slot[1] >= 0 && !v.split;
    hipError_t e;
    switch (g.wpd) {
      case 1: e = launch_large_v<T, 1>(v, both, st, false, a.logits != 0); break;
      case 2: e = launch_large_v<T, 2>(v, both, st, false, a.logits != 0); break;
      case 4: e = launch_large_v<T, 4>(v, both, st, false, a.logits != 0); break;
      default: e = hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
  }
  if (!has_h) return hipSuccess;
  LargeHParams h{};
  h.x = a.x; h.lam = a.lam; h.w = a.w; h.u = a.u; h.y = a.y; h.acc = a.acc; h.state = a.state;
  h.planes = a.planes; h.npc = npc; h.H = a.H; h.W = a.W;
  h.slot0 = slot[2]; h.slot1 = slot[3];
  const bool both = slot[2] >= 0 && slot[3] >= 0;
  h.nblk = g.nblk;
  h.delay = both ? (g.nblk & 1) : 0;
  h.half = both ? g.nblk / 2 + h.delay : 0;
  h.band_rows = g.hb_mid; h.edge_rows = g.hb_edge; h.nbands = g.hb_n; h.halo = g.halo;
  h.has_v = has_v && !a.y_pd ? 1 : 0;
  h.renorm = a.renorm;
  h.y_pd = a.y_pd;
  h.acc_b = (slot[0] >= 0 && slot[1] >= 0 && a.acc_b != nullptr && !a.y_pd) ? a.acc_b : nullptr;
  h.sum = a.y_pd ? nullptr : a.sum;
  h.hsave[0] = a.y_pd ? nullptr : a.hsave[0];
  h.hsave[1] = a.y_pd ? nullptr : a.hsave[1];
  const int64_t grid = (int64_t)g.hb_n * a.planes * (both ? 2 : 1);
  if (grid > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  const int GW = (a.group_w > 0 && a.group_w < a.W) ? a.group_w : a.W;
  // bit i of the mask: window column i of the launch starts a group
  auto window_mask = [&](int dir, int seq) -> uint64_t {
    if (seq < 0 || seq >= g.nblk || GW >= a.W) return 0;
    const int blk = dir ? g.nblk - 1 - seq : seq;
    const int c0 = blk * C::KH;
    const int ws = c0 + C::KH <= a.W ? c0 : a.W - C::KH;
    uint64_t m = 0;
    for (int i = 0; i < C::KH; ++i) {
      const int c = ws + i;
      if (dir ? ((c + 1) % GW == 0) : (c % GW == 0)) m |= 1ull << i;
    }
    return m;
  };
  static_assert(C::KH <= 64, "one mask bit per window column");
  for (int j = 0; j < g.nblk + h.delay; ++j) {
    h.step = j;
    h.gmask[0] = window_mask(0, j);
    h.gmask[1] = window_mask(1, j - h.delay);
    hipError_t e = launch_large_h<T>(h, g.hb_nw, grid, g.lds_hb, a.logits != 0, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace gspn
