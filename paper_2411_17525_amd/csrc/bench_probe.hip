// Measurement helper for the benchmark (not part of the method): a plain
// streaming read of a device buffer, the memory-system ceiling that a kernel
// reading the same number of bytes in one launch can reach on this GPU.
//
// Each thread reads four 16-byte pieces per iteration (non-temporal: read
// once), grid-stride over the buffer, and folds them into a checksum that is
// stored only if it equals a fixed value (never in practice), so the loads
// cannot be dropped and nothing is written.

#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

__global__ __launch_bounds__(kThreads) void stream_read_kernel(const u32x4* __restrict__ p,
                                                                int64_t n16,
                                                                uint32_t* __restrict__ sink) {
  const int64_t stride = int64_t(gridDim.x) * kThreads;
  uint32_t acc = 0;
  int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  for (; i + (kUnroll - 1) * stride < n16; i += kUnroll * stride) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n16; i += stride) {
    const u32x4 v = __builtin_nontemporal_load(p + i);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if (acc == 0x9E3779B9u) sink[threadIdx.x & 63] = acc;
}

}  // namespace

extern "C" {

// Reads `bytes` (a multiple of 16) from device memory at `buf` (16-byte
// aligned) on `stream`; `sink` is a device buffer of 64 uint32 that is
// written only if the checksum hits a fixed value. Returns a hipError_t.
int higgs_bench_stream_read(const void* buf, int64_t bytes, uint32_t* sink, void* stream) {
  if (buf == nullptr || sink == nullptr || bytes <= 0 || bytes % 16 != 0 ||
      reinterpret_cast<uintptr_t>(buf) % 16 != 0)
    return int(hipErrorInvalidValue);
  const int64_t n16 = bytes / 16;
  int cus = 256;
  int dev = 0;
  if (hipGetDevice(&dev) == hipSuccess) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        v > 0)
      cus = v;
  }
  // four blocks per compute unit, fewer when there is less work than that
  const int64_t want = (n16 + kThreads * kUnroll - 1) / (kThreads * kUnroll);
  const int64_t blocks = want < int64_t(cus) * 4 ? (want > 0 ? want : 1) : int64_t(cus) * 4;
  hipLaunchKernelGGL(stream_read_kernel, dim3(unsigned(blocks)), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const u32x4*>(buf), n16, sink);
  return int(hipGetLastError());
}

}  // extern "C"
