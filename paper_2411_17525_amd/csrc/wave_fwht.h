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
// fwht1024_lds (below) is the LDS-transposed form for 1024 values.
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

// Orders this wave's LDS accesses: the ones after it see its earlier writes
// (a wave's LDS instructions complete in order; this keeps the compiler from
// moving them across).
__device__ inline void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// LDS floats of fwht1024_lds's scratch (one per wave).
constexpr int kFwht1024Scratch = 1088;

// Unnormalised FWHT of 1024 fp32 values held 16 per lane (lane l: elements
// 16 l .. 16 l + 15) with every butterfly inside a lane: element bits 0-3 in
// place; then, through the wave's own LDS scratch `w` (kFwht1024Scratch
// floats, 16-byte aligned), each lane takes the 16 elements that differ in
// bits 4-7 (lane bits 0-3 and 4-5 = element bits 0-3 and 8-9); then the 16
// that differ in bits 8-9 and 0-1 (lane bits = element bits 2-7), where bits
// 8 and 9 are done. The stages run in the order of the element bits and each
// is (a + b, a - b), as in fwht_wave, so the result is the same bit for bit;
// the cross-lane moves become LDS accesses (element n at float n + 16 (n /
// 256), so the strided ones hit distinct banks). On return lane l holds
// element 256 h + 4 l + j in v[4 h + j] (h, j = 0..3).
__device__ inline void fwht1024_lds(float (&v)[16], float* w, int lane) {
  typedef float f32x4_v __attribute__((ext_vector_type(4)));
  wave_lds_sync();      // this wave's earlier accesses of w come first
  fwht_in_lane<16>(v);  // element bits 0-3
  {
    f32x4_v* p = reinterpret_cast<f32x4_v*>(w + 16 * lane + 16 * (lane >> 4));
#pragma unroll
    for (int k = 0; k < 4; ++k)
      p[k] = f32x4_v{v[4 * k], v[4 * k + 1], v[4 * k + 2], v[4 * k + 3]};
  }
  wave_lds_sync();
  // lane l: elements 256 (l / 16) + 16 i + l % 16, i = 0..15
  float* t1 = w + 272 * (lane >> 4) + (lane & 15);
#pragma unroll
  for (int i = 0; i < 16; ++i) v[i] = t1[16 * i];
  fwht_in_lane<16>(v);  // element bits 4-7
#pragma unroll
  for (int i = 0; i < 16; ++i) t1[16 * i] = v[i];
  wave_lds_sync();
  // lane l: elements 256 h + 4 l + j at v[4 h + j]
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const f32x4_v u = *reinterpret_cast<const f32x4_v*>(w + 272 * h + 4 * lane);
    v[4 * h] = u.x;
    v[4 * h + 1] = u.y;
    v[4 * h + 2] = u.z;
    v[4 * h + 3] = u.w;
  }
#pragma unroll
  for (int st = 4; st < 16; st <<= 1)  // element bits 8 and 9
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if ((i & st) == 0) {
        const float x0 = v[i], x1 = v[i + st];
        v[i] = x0 + x1;
        v[i + st] = x0 - x1;
      }
}

}  // namespace higgs
