// Fast Walsh-Hadamard transform of blocks held by one 64-lane wavefront, and
// the cross-lane exchanges it is built from.
//
// Layout: lane l holds E consecutive elements [l*E, (l+1)*E) of a segment of
// 64*E elements. With block size G >= 64 the segment is one block (G = 64*E);
// with G < 64 (then E = 1) the segment holds 64/G independent blocks. The
// butterflies over element bits below log2(E) run inside a lane; the ones
// over lane bits use cross-lane exchanges. Applying the 2x2 butterfly
// (a, b) -> (a + b, a - b) over every bit of the element index gives H x for
// the natural-order (Sylvester) Hadamard matrix H[r][c] = (-1)^popcount(r&c).
//
// The exchanges stay in the vector ALU: lane distances 1 and 2 are DPP quad
// permutes, 4 two bank-masked DPP row rotations, 8 a DPP row rotation, 16 and
// 32 the gfx950 permlane16/permlane32 swaps. No LDS traffic, no waits.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace higgs {

// 32-bit value of lane (lane ^ M), M in {1, 2, 4, 8}.
template <int M>
__device__ inline uint32_t lane_xor_small(uint32_t v) {
  static_assert(M == 1 || M == 2 || M == 4 || M == 8, "DPP distance");
  const int x = int(v);
  if constexpr (M == 1) {
    return uint32_t(__builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, true));  // quad_perm 1,0,3,2
  } else if constexpr (M == 2) {
    return uint32_t(__builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, true));  // quad_perm 2,3,0,1
  } else if constexpr (M == 4) {
    // lanes 0-3 and 8-11 of a row read lane + 4 (row_ror:12), lanes 4-7 and
    // 12-15 read lane - 4 (row_ror:4); the bank mask picks the lanes written
    const int t = __builtin_amdgcn_update_dpp(0, x, 0x12C, 0xF, 0x5, false);
    return uint32_t(__builtin_amdgcn_update_dpp(t, x, 0x124, 0xF, 0xA, false));
  } else {
    return uint32_t(__builtin_amdgcn_mov_dpp(x, 0x128, 0xF, 0xF, true));  // row_ror:8
  }
}

// For M in {16, 32}: lo = value of lane (lane & ~M), hi = value of lane (lane | M).
template <int M>
__device__ inline void lane_pair(uint32_t v, uint32_t& lo, uint32_t& hi) {
  static_assert(M == 16 || M == 32, "permlane distance");
  if constexpr (M == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    lo = r[0];
    hi = r[1];
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    lo = r[0];
    hi = r[1];
  }
}

// Value of lane (lane ^ M) (M a power of two <= 32).
template <int M>
__device__ inline uint32_t lane_xor_u32(uint32_t v, int lane) {
  if constexpr (M < 16) {
    return lane_xor_small<M>(v);
  } else {
    uint32_t lo, hi;
    lane_pair<M>(v, lo, hi);
    return (lane & M) ? lo : hi;
  }
}

// The same for float or double values.
template <int M, typename T>
__device__ inline T lane_xor(T v, int lane) {
  if constexpr (sizeof(T) == 4) {
    return __builtin_bit_cast(T, lane_xor_u32<M>(__builtin_bit_cast(uint32_t, v), lane));
  } else {
    static_assert(sizeof(T) == 8, "float or double");
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint64_t lo = lane_xor_u32<M>(uint32_t(u), lane);
    const uint64_t hi = lane_xor_u32<M>(uint32_t(u >> 32), lane);
    return __builtin_bit_cast(T, lo | (hi << 32));
  }
}

// In-lane stages (element strides 1 .. E/2).
template <int E, typename T>
__device__ inline void fwht_in_lane(T (&v)[E]) {
#pragma unroll
  for (int h = 1; h < E; h <<= 1) {
#pragma unroll
    for (int i = 0; i < E; ++i) {
      if ((i & h) == 0) {
        const T a = v[i], b = v[i + h];
        v[i] = a + b;
        v[i + h] = a - b;
      }
    }
  }
}

// One cross-lane stage over lane bit M: the lower lane of a pair keeps
// a + b, the upper one a - b (a the lower lane's value).
__device__ inline float fma_t(float a, float b, float c) { return __builtin_fmaf(a, b, c); }
__device__ inline double fma_t(double a, double b, double c) { return __builtin_fma(a, b, c); }

// Sum of v over the 64 lanes of the wave, in every lane (partners at
// distances 32, 16, ..., 1, in that order).
template <typename T>
__device__ inline T wave_sum(T v, int lane) {
  v += lane_xor<32>(v, lane);
  v += lane_xor<16>(v, lane);
  v += lane_xor<8>(v, lane);
  v += lane_xor<4>(v, lane);
  v += lane_xor<2>(v, lane);
  v += lane_xor<1>(v, lane);
  return v;
}

// Maximum of v over the 64 lanes of the wave, in every lane.
__device__ inline float wave_max(float v, int lane) {
  v = fmaxf(v, lane_xor<32>(v, lane));
  v = fmaxf(v, lane_xor<16>(v, lane));
  v = fmaxf(v, lane_xor<8>(v, lane));
  v = fmaxf(v, lane_xor<4>(v, lane));
  v = fmaxf(v, lane_xor<2>(v, lane));
  v = fmaxf(v, lane_xor<1>(v, lane));
  return v;
}

__device__ inline double wave_max(double v, int lane) {
  v = fmax(v, lane_xor<32>(v, lane));
  v = fmax(v, lane_xor<16>(v, lane));
  v = fmax(v, lane_xor<8>(v, lane));
  v = fmax(v, lane_xor<4>(v, lane));
  v = fmax(v, lane_xor<2>(v, lane));
  v = fmax(v, lane_xor<1>(v, lane));
  return v;
}

// Cross-lane stages with the signs deferred: each stage leaves the upper lane
// of a pair holding the negation of its true value, (w - w') instead of
// (w' - w), which needs no sign operand and lets the exchange fold into one
// v_fmac (DPP distances) or one fma (permlane distances). Since the two lanes
// of a pair carry the same deferred sign, the stages compose, and the true
// value of every element is sign * v with the returned per-lane sign
// (-1)^popcount(lane & stages). Rounding is unchanged: round(a - b) =
// -round(b - a).
template <int M, int E, typename T>
__device__ inline void fwht_lane_stage_deferred(T (&v)[E], int lane) {
  const T s = (lane & M) ? T(-1) : T(1);
  if constexpr (M < 16 && sizeof(T) == 4) {
    // all exchanges first, then all updates: no DPP read waits on a
    // just-written register
    T p[E];
#pragma unroll
    for (int i = 0; i < E; ++i) p[i] = lane_xor<M>(v[i], lane);
#pragma unroll
    for (int i = 0; i < E; ++i) v[i] = fma_t(p[i], s, v[i]);
  } else if constexpr (sizeof(T) == 4) {
    uint32_t lo[E], hi[E];
#pragma unroll
    for (int i = 0; i < E; ++i) lane_pair<M>(__builtin_bit_cast(uint32_t, v[i]), lo[i], hi[i]);
#pragma unroll
    for (int i = 0; i < E; ++i)
      v[i] = fma_t(s, __builtin_bit_cast(T, lo[i]), __builtin_bit_cast(T, hi[i]));
  } else {
#pragma unroll
    for (int i = 0; i < E; ++i) v[i] = fma_t(lane_xor<M>(v[i], lane), s, v[i]);
  }
}

template <int E, typename T>
__device__ inline T fwht_cross_lane_deferred(T (&v)[E], int lane, int G) {
  // stage over lane bit m runs while m * E < G (uniform across the wave)
  int mask = 0;
  if (E < G) { fwht_lane_stage_deferred<1>(v, lane); mask |= 1; }
  if (2 * E < G) { fwht_lane_stage_deferred<2>(v, lane); mask |= 2; }
  if (4 * E < G) { fwht_lane_stage_deferred<4>(v, lane); mask |= 4; }
  if (8 * E < G) { fwht_lane_stage_deferred<8>(v, lane); mask |= 8; }
  if (16 * E < G) { fwht_lane_stage_deferred<16>(v, lane); mask |= 16; }
  if (32 * E < G) { fwht_lane_stage_deferred<32>(v, lane); mask |= 32; }
  return (__builtin_popcount(lane & mask) & 1) ? T(-1) : T(1);
}

// The same with the block size G known at compile time (every stage that
// runs is unconditional: no branches, no copies to merge their results).
template <int E, int G, typename T>
__device__ inline T fwht_cross_lane_deferred_fixed(T (&v)[E], int lane) {
  int mask = 0;
  if constexpr (E < G) { fwht_lane_stage_deferred<1>(v, lane); mask |= 1; }
  if constexpr (2 * E < G) { fwht_lane_stage_deferred<2>(v, lane); mask |= 2; }
  if constexpr (4 * E < G) { fwht_lane_stage_deferred<4>(v, lane); mask |= 4; }
  if constexpr (8 * E < G) { fwht_lane_stage_deferred<8>(v, lane); mask |= 8; }
  if constexpr (16 * E < G) { fwht_lane_stage_deferred<16>(v, lane); mask |= 16; }
  if constexpr (32 * E < G) { fwht_lane_stage_deferred<32>(v, lane); mask |= 32; }
  return (__builtin_popcount(lane & mask) & 1) ? T(-1) : T(1);
}

template <int E, typename T>
__device__ inline void fwht_cross_lane(T (&v)[E], int lane, int G) {
  const T sign = fwht_cross_lane_deferred<E>(v, lane, G);
#pragma unroll
  for (int i = 0; i < E; ++i) v[i] *= sign;
}

template <int E, typename T>
__device__ inline void fwht_wave(T (&v)[E], int lane, int G) {
  fwht_in_lane<E>(v);
  fwht_cross_lane<E>(v, lane, G);
}

}  // namespace higgs
