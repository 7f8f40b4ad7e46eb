// Fast Walsh-Hadamard transform of blocks held by one 64-lane wavefront.
//
// Layout: lane l holds E consecutive elements [l*E, (l+1)*E) of a segment of
// 64*E elements. With block size G >= 64 the segment is one block (G = 64*E);
// with G < 64 (then E = 1) the segment holds 64/G independent blocks. The
// butterflies over element bits below log2(E) run inside a lane; the ones
// over lane bits use cross-lane exchanges. Applying the 2x2 butterfly
// (a, b) -> (a + b, a - b) over every bit of the element index gives H x for
// the natural-order (Sylvester) Hadamard matrix H[r][c] = (-1)^popcount(r&c).
#pragma once

#include <hip/hip_runtime.h>

namespace higgs {

template <typename T>
__device__ inline T lane_xor(T v, int mask) {
  return __shfl_xor(v, mask, 64);
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

// Cross-lane stages: lane bit m (element stride m*E) while m*E < G.
template <int E, typename T>
__device__ inline void fwht_cross_lane(T (&v)[E], int lane, int G) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) {
    if (m * E >= G) break;  // uniform across the wave
    const bool upper = (lane & m) != 0;
#pragma unroll
    for (int i = 0; i < E; ++i) {
      const T other = lane_xor(v[i], m);
      v[i] = upper ? (other - v[i]) : (v[i] + other);
    }
  }
}

template <int E, typename T>
__device__ inline void fwht_wave(T (&v)[E], int lane, int G) {
  fwht_in_lane<E>(v);
  fwht_cross_lane<E>(v, lane, G);
}

}  // namespace higgs
