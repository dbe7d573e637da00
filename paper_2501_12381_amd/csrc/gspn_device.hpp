// Device-side helpers shared by the GSPN kernels (gfx950 / CDNA4, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace gspn {

typedef __bf16 bf16;

// ---------------------------------------------------------------------------
// element conversion: inputs are widened to fp32, outputs rounded once
// (bf16 stores use the hardware round-to-nearest-even convert).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
// two floats -> two bf16 in one word (a in the low half), one packed convert
__device__ __forceinline__ uint32_t pack_bf2(float a, float b) {
  const f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ float to_f(float v) { return v; }
__device__ __forceinline__ float to_f(bf16 v) { return (float)v; }
template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f<bf16>(float v) { return (bf16)v; }

// Load N consecutive elements starting at p into fp32 registers.  The address
// must be aligned to min(16, N * sizeof(T)) bytes.
template <int N> __device__ __forceinline__ void ldv(const float* __restrict__ p, float* v) {
  if constexpr (N == 1) {
    v[0] = p[0];
  } else if constexpr (N == 2) {
    float2 t = *reinterpret_cast<const float2*>(p);
    v[0] = t.x; v[1] = t.y;
  } else {
#pragma unroll
    for (int q = 0; q < N; q += 4) {
      float4 t = *reinterpret_cast<const float4*>(p + q);
      v[q] = t.x; v[q + 1] = t.y; v[q + 2] = t.z; v[q + 3] = t.w;
    }
  }
}
template <int N> __device__ __forceinline__ void ldv(const bf16* __restrict__ p, float* v) {
  if constexpr (N == 1) {
    v[0] = (float)p[0];
  } else if constexpr (N == 2) {
    uint32_t t = *reinterpret_cast<const uint32_t*>(p);
    v[0] = bf_lo(t); v[1] = bf_hi(t);
  } else if constexpr (N == 4) {
    uint2 t = *reinterpret_cast<const uint2*>(p);
    v[0] = bf_lo(t.x); v[1] = bf_hi(t.x); v[2] = bf_lo(t.y); v[3] = bf_hi(t.y);
  } else {
#pragma unroll
    for (int q = 0; q < N; q += 8) {
      uint4 t = *reinterpret_cast<const uint4*>(p + q);
      v[q] = bf_lo(t.x); v[q + 1] = bf_hi(t.x); v[q + 2] = bf_lo(t.y); v[q + 3] = bf_hi(t.y);
      v[q + 4] = bf_lo(t.z); v[q + 5] = bf_hi(t.z); v[q + 6] = bf_lo(t.w); v[q + 7] = bf_hi(t.w);
    }
  }
}

// Store N consecutive elements (same alignment rule as ldv).
template <int N> __device__ __forceinline__ void stv(float* __restrict__ p, const float* v) {
  if constexpr (N == 1) {
    p[0] = v[0];
  } else if constexpr (N == 2) {
    *reinterpret_cast<float2*>(p) = make_float2(v[0], v[1]);
  } else {
#pragma unroll
    for (int q = 0; q < N; q += 4)
      *reinterpret_cast<float4*>(p + q) = make_float4(v[q], v[q + 1], v[q + 2], v[q + 3]);
  }
}
template <int N> __device__ __forceinline__ void stv(bf16* __restrict__ p, const float* v) {
  if constexpr (N == 1) {
    p[0] = (bf16)v[0];
  } else if constexpr (N == 2) {
    *reinterpret_cast<uint32_t*>(p) = pack_bf2(v[0], v[1]);
  } else if constexpr (N == 4) {
    *reinterpret_cast<uint2*>(p) = make_uint2(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]));
  } else {
#pragma unroll
    for (int q = 0; q < N; q += 8)
      *reinterpret_cast<uint4*>(p + q) =
          make_uint4(pack_bf2(v[q], v[q + 1]), pack_bf2(v[q + 2], v[q + 3]),
                     pack_bf2(v[q + 4], v[q + 5]), pack_bf2(v[q + 6], v[q + 7]));
  }
}

// ---------------------------------------------------------------------------
// cross-lane moves inside a wave64 (DPP wave shifts with the bound control set,
// so the lane without a source reads zero; all 64 lanes must be active)
// ---------------------------------------------------------------------------
// lane l receives lane l-1's value; lane 0 receives 0
__device__ __forceinline__ float from_prev_lane(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x138 /* wave_shr:1 */,
                                                            0xf, 0xf, true));
}
// lane l receives lane l+1's value; lane 63 receives 0
__device__ __forceinline__ float from_next_lane(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x130 /* wave_shl:1 */,
                                                            0xf, 0xf, true));
}

// the same shifts without the bound control: the lane without a source keeps
// `edge` (its neighbour from outside the wave), so no select is needed
__device__ __forceinline__ float from_prev_lane_or(float v, float edge) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, edge),
                                                               __builtin_bit_cast(int, v), 0x138, 0xf, 0xf, false));
}
__device__ __forceinline__ float from_next_lane_or(float v, float edge) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, edge),
                                                               __builtin_bit_cast(int, v), 0x130, 0xf, 0xf, false));
}

// Workgroup barrier that orders LDS accesses only: waits for this wave's LDS
// operations, then for every wave.  Global loads stay in flight across it
// (a full __syncthreads would drain them), which keeps register prefetches
// useful across the barriers of a scan.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Local GSPN (groups of G lines along the scan axis): true when `line` is the
// first line a scan visits in its group, where the state restarts from zero.
// Forward scans enter a group [kG, (k+1)G) at its lowest line, reverse scans
// at its highest one.  G = the line count (or more) is the global scan.
__device__ __forceinline__ bool group_start(int line, int G, bool rev) {
  return rev ? ((line + 1) % G == 0) : (line % G == 0);
}

// Eq. 6: the three logits of one pixel -> its three weights (sigmoid, then
// normalised over the neighbours that count: all three, or with edge
// renormalisation the ones on the line).  Also returns the sigmoids and the
// normaliser for the Jacobian of the backward.  The reciprocals are the
// hardware's (v_rcp_f32, within 1 ulp): an IEEE division would cost a dozen
// instructions per weight in the kernels' line steps.  A normaliser that
// underflows to zero (every sigmoid zero) is clamped, giving zero weights.
struct Norm3 {
  float w[3], sg[3], m[3], inv;
};
__device__ __forceinline__ Norm3 normalize3(float l0, float l1, float l2, bool first_pos, bool last_pos,
                                            bool renorm) {
  Norm3 r;
  r.sg[0] = __builtin_amdgcn_rcpf(1.f + __expf(-l0));
  r.sg[1] = __builtin_amdgcn_rcpf(1.f + __expf(-l1));
  r.sg[2] = __builtin_amdgcn_rcpf(1.f + __expf(-l2));
  r.m[0] = (renorm && first_pos) ? 0.f : 1.f;
  r.m[1] = 1.f;
  r.m[2] = (renorm && last_pos) ? 0.f : 1.f;
  const float s0 = r.m[0] * r.sg[0], s1 = r.sg[1], s2 = r.m[2] * r.sg[2];
  r.inv = __builtin_amdgcn_rcpf(fmaxf(s0 + s1 + s2, 1e-30f));
  r.w[0] = s0 * r.inv;
  r.w[1] = s1 * r.inv;
  r.w[2] = s2 * r.inv;
  return r;
}

// The Jacobian of the normalisation applied to the gradients e_k of the three
// weights: dl_k = m_k sig_k (1 - sig_k) (e_k - sum_j w_j e_j) / S, where S is
// the normaliser (r.inv = 1 / S).
__device__ __forceinline__ void norm3_vjp(const Norm3& r, float& e0, float& e1, float& e2) {
  const float inner = r.w[0] * e0 + r.w[1] * e1 + r.w[2] * e2;
  e0 = r.m[0] * r.sg[0] * (1.f - r.sg[0]) * (e0 - inner) * r.inv;
  e1 = r.m[1] * r.sg[1] * (1.f - r.sg[1]) * (e1 - inner) * r.inv;
  e2 = r.m[2] * r.sg[2] * (1.f - r.sg[2]) * (e2 - inner) * r.inv;
}

// Calls f(std::integral_constant<int, i>) for i = B .. E-1 (compile-time indices,
// fully unrolled by construction, where a large unrolled loop body may not be).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

}  // namespace gspn
