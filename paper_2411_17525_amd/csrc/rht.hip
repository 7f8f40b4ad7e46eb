// Activation rotation for inference in the rotated space (App. G, "rotating
// activations"): x_rot[b, block i] = H (sigma * x[b, block i]) / sqrt(g).
//
// One wavefront transforms one segment of max(g, 64) consecutive elements of
// the flattened [batch][in] activation (one block when g >= 64, 64/g blocks
// otherwise). Each lane loads E = max(g/64, 1) contiguous elements, applies the
// signs, runs the in-register / cross-lane butterflies in fp32 and stores fp32.
// The kernel streams x once and x_rot once: HBM bound.

#include <algorithm>
#include <cmath>

#include "internal.h"
#include "wave_fwht.h"

namespace higgs {
namespace {

constexpr int kWavesPerBlock = 4;

template <typename InT>
__device__ inline float to_f32(InT v);
template <>
__device__ inline float to_f32<float>(float v) { return v; }
template <>
__device__ inline float to_f32<uint16_t>(uint16_t v) {
  return __uint_as_float(uint32_t(v) << 16);
}

template <int E, typename InT>
__device__ inline void load_elems(const InT* __restrict__ src, float (&v)[E]) {
  constexpr int kBytes = E * int(sizeof(InT));
  if constexpr (kBytes % 16 == 0) {
    constexpr int kVec = kBytes / 16;
    constexpr int kPer = 16 / int(sizeof(InT));
    const uint4* p = reinterpret_cast<const uint4*>(src);
#pragma unroll
    for (int q = 0; q < kVec; ++q) {
      const uint4 u = p[q];
      const InT* e = reinterpret_cast<const InT*>(&u);
#pragma unroll
      for (int i = 0; i < kPer; ++i) v[q * kPer + i] = to_f32<InT>(e[i]);
    }
  } else {
#pragma unroll
    for (int i = 0; i < E; ++i) v[i] = to_f32<InT>(src[i]);
  }
}

template <int E>
__device__ inline void store_elems(float* __restrict__ dst, const float (&v)[E]) {
  if constexpr (E % 4 == 0) {
    float4* p = reinterpret_cast<float4*>(dst);
#pragma unroll
    for (int q = 0; q < E / 4; ++q) p[q] = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
  } else {
#pragma unroll
    for (int i = 0; i < E; ++i) dst[i] = v[i];
  }
}

template <int E, typename InT>
__global__ __launch_bounds__(64 * kWavesPerBlock) void rht_kernel(
    const InT* __restrict__ x, int64_t total, int g, uint64_t seed, float scale,
    float* __restrict__ x_rot) {
  const int lane = int(threadIdx.x) & 63;
  const int64_t seg_elems = int64_t(64) * E;
  const int64_t nsegs = (total + seg_elems - 1) / seg_elems;
  const int64_t wave0 = int64_t(blockIdx.x) * kWavesPerBlock + (threadIdx.x >> 6);
  const int64_t nwaves = int64_t(gridDim.x) * kWavesPerBlock;

  // The sign of an element depends only on its position inside its block,
  // which is the same for this lane in every segment.
  uint64_t neg = 0;
#pragma unroll
  for (int i = 0; i < E; ++i) {
    const uint32_t pos = uint32_t((lane * E + i) & (g - 1));
    neg |= uint64_t(rht_sign_negative(seed, pos)) << i;
  }

  for (int64_t seg = wave0; seg < nsegs; seg += nwaves) {
    const int64_t base = seg * seg_elems + int64_t(lane) * E;
    const bool active = base < total;  // can only fail in the last segment when g < 64
    float v[E];
    if (active) {
      load_elems<E, InT>(x + base, v);
    } else {
#pragma unroll
      for (int i = 0; i < E; ++i) v[i] = 0.f;
    }
#pragma unroll
    for (int i = 0; i < E; ++i)
      if ((neg >> i) & 1) v[i] = -v[i];
    fwht_wave<E>(v, lane, g);
#pragma unroll
    for (int i = 0; i < E; ++i) v[i] *= scale;
    if (active) store_elems<E>(x_rot + base, v);
  }
}

template <typename InT>
hipError_t launch_typed(const InT* x, int64_t batch, int64_t in, int g, uint64_t seed,
                        float* x_rot, hipStream_t stream) {
  const int64_t total = batch * in;
  const int E = g >= 64 ? g / 64 : 1;
  const int64_t seg_elems = int64_t(64) * E;
  const int64_t segs = (total + seg_elems - 1) / seg_elems;
  // enough waves to cover the chip a few times; the kernel loops over the rest
  const int64_t blocks = std::min<int64_t>((segs + kWavesPerBlock - 1) / kWavesPerBlock, 4096);
  const dim3 grid{unsigned(blocks)};
  const dim3 block(64 * kWavesPerBlock);
  const float scale = float(1.0 / std::sqrt(double(g)));
  switch (E) {
#define HIGGS_RHT_CASE(EV)                                                                   \
  case EV:                                                                                   \
    hipLaunchKernelGGL((rht_kernel<EV, InT>), grid, block, 0, stream, x, total, g, seed, \
                       scale, x_rot);                                                        \
    break;
    HIGGS_RHT_CASE(1)
    HIGGS_RHT_CASE(2)
    HIGGS_RHT_CASE(4)
    HIGGS_RHT_CASE(8)
    HIGGS_RHT_CASE(16)
    HIGGS_RHT_CASE(32)
    HIGGS_RHT_CASE(64)
#undef HIGGS_RHT_CASE
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_rht_activations(const void* x, higgs_dtype dtype, int64_t batch, int64_t in,
                                  int g, uint64_t seed, float* x_rot, hipStream_t stream) {
  if (dtype == HIGGS_F32)
    return launch_typed(static_cast<const float*>(x), batch, in, g, seed, x_rot, stream);
  return launch_typed(static_cast<const uint16_t*>(x), batch, in, g, seed, x_rot, stream);
}

}  // namespace higgs
