// Lookup-table GEMM for HIGGS layers at batch >= 16 on the matrix cores,
// computed in the rotated space (App. G):
//   y[b][o] = sum_i scale[o][i] * sum_j < G[code(o,i,j)], x_rot[b, ig+jp : ig+(j+1)p] >
// At these batch sizes the layer is a dense contraction, so the dequantised
// weights feed v_mfma_f32_32x32x16_f16 directly:
//   * A block owns 128 rows (4 waves x 32) and a K-range of the layer; the
//     grid's second dimension splits K when the layer has too few rows to
//     fill the chip. Partial sums of a split go to the workspace and are
//     added in a fixed order by qgemm_reduce (deterministic).
//   * A operand: each lane reads 16 bytes of codes of its row (16 codes = 32
//     weights) per 64-weight K-block and turns them into fp16 pairs through
//     an LDS lookup table (32 copies, lane-private within a half wave). The
//     MFMA's reduction index is mapped so that lane half h of step s covers
//     weights 32h + 8s .. 32h + 8s + 7 of the K-block, for A and B alike.
//   * B operand: activations of the K-chunk (the group of g weights, at most
//     256) staged in LDS as fp16 after an exact power-of-two rescale per
//     batch row and chunk (no overflow, full fp16 precision).
//   * Each chunk accumulates in fp32 MFMA registers; at the chunk's end the
//     group scale (fp16 -> fp32) and the activation rescale are applied and
//     the result is added into fp32 totals.
// Code format: 8-bit codes (p = 2, n = 256; p = 1, n = 16 read as byte
// values indexing a table of grid-point pairs).

#include <algorithm>
#include <mutex>

#include "internal.h"
#include "wave_fwht.h"

namespace higgs {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kTileRows = 32 * kWaves;  // rows per block
constexpr int kCopiesLog2 = 5;          // table copies (one per lane of a half wave)
constexpr int kLutWords = 256 << kCopiesLog2;
constexpr int kXPad = 8;                // halves of padding per staged activation row

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f16x_acc __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));

__device__ inline uint32_t pack_h2(float a, float b) {
  const _Float16 ha = static_cast<_Float16>(a), hb = static_cast<_Float16>(b);
  return uint32_t(__builtin_bit_cast(uint16_t, ha)) |
         (uint32_t(__builtin_bit_cast(uint16_t, hb)) << 16);
}

// NB: 32-column batch tiles per launch (1 or 2).
template <int NB>
__global__ __launch_bounds__(kThreads) void qgemm_kernel(
    const float* __restrict__ x_rot, int nb_rows, const uint8_t* __restrict__ codes,
    const uint16_t* __restrict__ scales, const float* __restrict__ grid, int pair_table,
    int log2g, int log2kc, int64_t out, int64_t in, int64_t k_per_split,
    float* __restrict__ dst, int64_t dst_split_stride) {
  constexpr int kBatch = 32 * NB;
  __shared__ uint32_t s_lut[kLutWords];
  __shared__ uint32_t s_compact[256];
  extern __shared__ u32x4v smem4[];
  _Float16* s_x = reinterpret_cast<_Float16*>(smem4);  // [kBatch][kc + kXPad]
  float* s_xs = reinterpret_cast<float*>(smem4) + 0;   // placed after s_x (set below)

  const int lane = int(threadIdx.x) & 63;
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
  const int kc = 1 << log2kc;
  const int xstride = kc + kXPad;  // halves per staged row
  s_xs = reinterpret_cast<float*>(s_x + kBatch * xstride);

  const int64_t row0 = int64_t(blockIdx.x) * kTileRows + wave * 32;
  const int64_t kbeg = int64_t(blockIdx.y) * k_per_split;
  const int64_t kend = min(in, kbeg + k_per_split);
  const int64_t row_bytes = in / 2;          // 8-bit codes: one byte per 2 weights
  const int64_t groups_per_row = in >> log2g;

  // ---- lookup table ----
  {
    const int c = int(threadIdx.x);  // 256 threads, 256 entries
    s_compact[c] = pair_table ? pack_h2(grid[c & 15], grid[c >> 4])
                              : pack_h2(grid[2 * c], grid[2 * c + 1]);
  }
  __syncthreads();
  for (int w4 = int(threadIdx.x) * 4; w4 < kLutWords; w4 += kThreads * 4) {
    const uint32_t e = s_compact[w4 >> kCopiesLog2];
    *reinterpret_cast<u32x4v*>(&s_lut[w4]) = u32x4v{e, e, e, e};
  }

  // this lane's A row and half
  const int arow_l = lane & 31, ahalf = lane >> 5;
  const int64_t arow = min(row0 + arow_l, out - 1);  // rows past `out` are computed, not stored
  const uint8_t* arow_codes = codes + arow * row_bytes;
  const uint32_t copy8 = uint32_t(lane & 31) << 3;  // table copy, pre-shifted for perm + >> 1

  f16x_acc total[NB];
#pragma unroll
  for (int t = 0; t < NB; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) total[t][r] = 0.f;

  // rows of this lane's accumulators: 8 * (r / 4) + 4 * ahalf + (r % 4)
  for (int64_t k0 = kbeg; k0 < kend; k0 += kc) {
    // ---- stage the activations of this chunk: one batch row per wave step ----
    __syncthreads();  // previous chunk fully consumed (and, first time, table built)
    // all loads first (kBatch / kWaves rows per wave), then rescale and store
    constexpr int kRowsPerWave = kBatch / kWaves;
    float v[kRowsPerWave][4];
#pragma unroll
    for (int i = 0; i < kRowsPerWave; ++i) {
      const int b = wave + i * kWaves;
      // a chunk row has kc <= 256 values: lanes 0 .. kc/4 - 1 hold 4 each
      if (b < nb_rows && lane * 4 < kc) {
        const float4 f = *reinterpret_cast<const float4*>(x_rot + int64_t(b) * in + k0 + lane * 4);
        v[i][0] = f.x; v[i][1] = f.y; v[i][2] = f.z; v[i][3] = f.w;
      } else {
        v[i][0] = v[i][1] = v[i][2] = v[i][3] = 0.f;
      }
    }
#pragma unroll
    for (int i = 0; i < kRowsPerWave; ++i) {
      const int b = wave + i * kWaves;
      float m = fmaxf(fmaxf(fabsf(v[i][0]), fabsf(v[i][1])), fmaxf(fabsf(v[i][2]), fabsf(v[i][3])));
      m = wave_max(m, lane);
      int e = m > 0.f ? ilogbf(m) - 14 : 0;
      e = e < -126 ? -126 : e;
      if (lane * 4 < kc) {
        uint32_t* d = reinterpret_cast<uint32_t*>(s_x + b * xstride + lane * 4);
        d[0] = pack_h2(ldexpf(v[i][0], -e), ldexpf(v[i][1], -e));
        d[1] = pack_h2(ldexpf(v[i][2], -e), ldexpf(v[i][3], -e));
      }
      if (lane == 0) s_xs[b] = ldexpf(1.0f, e);
    }
    __syncthreads();

    f16x_acc acc[NB];
#pragma unroll
    for (int t = 0; t < NB; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;

    for (int kb = 0; kb < kc; kb += 64) {
      // 16 codes of this lane's row: weights k0 + kb + 32 * ahalf .. + 31
      const u32x4 cw = load_stream16(arow_codes + ((k0 + kb) >> 1) + 16 * ahalf);
      const uint32_t w4[4] = {cw.x, cw.y, cw.z, cw.w};
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        // A: codes 4s .. 4s+3 -> 8 halves (weights 32h + 8s .. + 7)
        uint32_t a32[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t sel = 0x0c0c0000u | (uint32_t(4 + q) << 8);
          const uint32_t off = __builtin_amdgcn_perm(w4[s], copy8, sel) >> 1;
          a32[q] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(s_lut) + off);
        }
        const half8 a = __builtin_bit_cast(half8, u32x4v{a32[0], a32[1], a32[2], a32[3]});
#pragma unroll
        for (int t = 0; t < NB; ++t) {
          // B: batch row 32t + (lane % 32), the same 8 weights
          const half8 bv = *reinterpret_cast<const half8*>(
              s_x + (32 * t + (lane & 31)) * xstride + kb + 32 * ahalf + 8 * s);
          acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, bv, acc[t], 0, 0, 0);
        }
      }
    }

    // ---- fold the chunk: group scale of each accumulator row, activation
    //      rescale of the column ----
    const int64_t grp = k0 >> log2g;
    float srow[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t row = min(row0 + 8 * (r / 4) + 4 * ahalf + (r % 4), out - 1);
      srow[r] = float(__builtin_bit_cast(_Float16, scales[row * groups_per_row + grp]));
    }
#pragma unroll
    for (int t = 0; t < NB; ++t) {
      const float xs = s_xs[32 * t + (lane & 31)];
#pragma unroll
      for (int r = 0; r < 16; ++r) total[t][r] = fmaf(acc[t][r], srow[r] * xs, total[t][r]);
    }
  }

  // ---- store: column = batch row 32t + lane % 32 ----
#pragma unroll
  for (int t = 0; t < NB; ++t) {
    const int b = 32 * t + (lane & 31);
    if (b >= nb_rows) continue;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t row = row0 + 8 * (r / 4) + 4 * ahalf + (r % 4);
      if (row < out) dst[int64_t(blockIdx.y) * dst_split_stride + int64_t(b) * out + row] = total[t][r];
    }
  }
}

// y = sum over splits of the partial products, in split order.
__global__ __launch_bounds__(256) void qgemm_reduce(const float* __restrict__ part, int splits,
                                                    int64_t n, float* __restrict__ y) {
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) {
    float s = part[i];
    for (int k = 1; k < splits; ++k) s += part[int64_t(k) * n + i];
    y[i] = s;
  }
}

int device_cus() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] == 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
      v = 256;
    cus[dev] = v;
  }
  return cus[dev];
}

template <int NB>
size_t dyn_lds(int kc) {
  return size_t(32 * NB) * size_t(kc + kXPad) * 2 + size_t(32 * NB) * 4;
}

template <int NB>
hipError_t launch_nb(const float* x_rot, int nb_rows, const uint8_t* codes, const uint16_t* scales,
                     const float* grid, int pair_table, int log2g, int64_t out, int64_t in,
                     int splits, float* dst, hipStream_t stream) {
  const int log2kc = std::min(log2g, 8);
  const int64_t kc = int64_t(1) << log2kc;
  const int64_t chunks = in / kc;
  const int64_t chunks_per_split = (chunks + splits - 1) / splits;
  static std::once_flag once;
  static hipError_t attr = hipSuccess;
  std::call_once(once, [] {
    attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&qgemm_kernel<NB>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, int(dyn_lds<NB>(256)));
  });
  if (attr != hipSuccess) return attr;
  const dim3 grid_dim{unsigned((out + kTileRows - 1) / kTileRows), unsigned(splits)};
  hipLaunchKernelGGL((qgemm_kernel<NB>), grid_dim, dim3(kThreads), dyn_lds<NB>(int(kc)), stream,
                     x_rot, nb_rows, codes, scales, grid, pair_table, log2g, log2kc, out, in,
                     chunks_per_split * kc, dst, int64_t(nb_rows) * out);
  return hipGetLastError();
}

}  // namespace

// Splits of K for a launch of `batch` rows: enough blocks for ~2 per compute
// unit, keeping at least 1024 weights of K per split.
int qgemm_splits(int64_t out, int64_t in, int g) {
  const int64_t tiles = (out + kTileRows - 1) / kTileRows;
  const int64_t kc = std::min<int64_t>(g, 256);
  const int64_t chunks = in / kc;
  int64_t s = 1;
  while (tiles * s < 2 * int64_t(device_cus()) && (chunks / (2 * s)) * kc >= 1024) s *= 2;
  return int(s);
}

int64_t qgemm_workspace_bytes(int64_t batch, int64_t out, int64_t in, int g) {
  const int s = qgemm_splits(out, in, g);
  if (s <= 1) return 0;
  return int64_t(s) * std::min<int64_t>(batch, 64) * out * 4;
}

hipError_t launch_qgemm(const float* x_rot, int64_t batch, const uint8_t* codes,
                        const uint16_t* scales, const float* grid, int p, int g, int64_t out,
                        int64_t in, float* y, float* workspace, hipStream_t stream) {
  const int pair_table = p == 1 ? 1 : 0;
  const int log2g = log2_exact(g);
  const int splits = qgemm_splits(out, in, g);
  for (int64_t b0 = 0; b0 < batch; b0 += 64) {
    const int nb = int(std::min<int64_t>(64, batch - b0));
    const float* xb = x_rot + b0 * in;
    float* yb = y + b0 * out;
    float* dst = splits > 1 ? workspace : yb;
    hipError_t err = nb > 32 ? launch_nb<2>(xb, nb, codes, scales, grid, pair_table, log2g, out, in,
                                            splits, dst, stream)
                             : launch_nb<1>(xb, nb, codes, scales, grid, pair_table, log2g, out, in,
                                            splits, dst, stream);
    if (err != hipSuccess) return err;
    if (splits > 1) {
      const int64_t n = int64_t(nb) * out;
      const int64_t blocks = std::min<int64_t>((n + 255) / 256, 4096);
      hipLaunchKernelGGL(qgemm_reduce, dim3(unsigned(blocks)), dim3(256), 0, stream, workspace,
                         splits, n, yb);
      err = hipGetLastError();
      if (err != hipSuccess) return err;
    }
  }
  return hipSuccess;
}

}  // namespace higgs
