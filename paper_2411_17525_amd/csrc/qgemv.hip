// Lookup-table GEMV for HIGGS layers at small batch (1..8 activation rows),
// computed in the rotated space (App. G):
//   y[b][o] = sum_i scale[o][i] * sum_j < G[code(o,i,j)], x_rot[b, ig+jp : ig+(j+1)p] >
// Decoding is memory bound at this batch (Sec. 3.3), so the kernel is built to
// stream the packed codes from HBM once, coalesced:
//   * A lane owns a chunk of 16 codes (32 weights) of a row; a wave covers a
//     K-range of 64 chunks (2048 inputs) and walks its rows, so the lane's
//     activations stay in registers for every row of the K-range.
//   * Grid points are read from a lookup table in LDS, one fp16 pair per
//     entry, replicated per lane so that the 64 random reads of a wave hit
//     distinct banks (the grid-in-fast-memory constraint of Sec. 3.3).
//   * Each entry meets its activation pair in one v_dot2_f32_f16 (fp32
//     accumulation). Activations are rescaled by an exact power of two per
//     K-range and batch row before the fp16 rounding, so any finite fp32
//     input keeps fp16 precision without overflow.
//   * Per-group scales multiply each lane's partial sum; partial sums are
//     reduced across lanes with a fixed butterfly (deterministic).
// Code formats: MODE 0 = 8-bit codes (p = 2, n = 256; also p = 1, n = 16 read
// as 256 byte values indexing a table of grid-point pairs), MODE 1 = 6-bit
// (p = 2, n = 64), MODE 2 = 10-bit (p = 2, n = 1024).

#include <algorithm>

#include "internal.h"

namespace higgs {
namespace {

constexpr int kWaves = 4;
constexpr int kChunkCodes = 16;
constexpr int kChunkWeights = 32;
constexpr int kRangeWeights = 64 * kChunkWeights;

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

template <int MODE>
struct Fmt;
template <>
struct Fmt<0> {
  static constexpr int kBits = 8, kWords = 4, kEntriesLog2 = 8, kReplicasLog2 = 6;
};
template <>
struct Fmt<1> {
  static constexpr int kBits = 6, kWords = 3, kEntriesLog2 = 6, kReplicasLog2 = 6;
};
template <>
struct Fmt<2> {
  static constexpr int kBits = 10, kWords = 5, kEntriesLog2 = 10, kReplicasLog2 = 4;
};

template <int MODE>
constexpr int lut_words() {
  return 1 << (Fmt<MODE>::kEntriesLog2 + Fmt<MODE>::kReplicasLog2);
}

__device__ inline uint32_t pack_half2(float a, float b) {
  const _Float16 ha = static_cast<_Float16>(a), hb = static_cast<_Float16>(b);
  return uint32_t(__builtin_bit_cast(uint16_t, ha)) |
         (uint32_t(__builtin_bit_cast(uint16_t, hb)) << 16);
}

// Code j (0..15) of a chunk held in little-endian dwords.
template <int MODE>
__device__ inline uint32_t chunk_code(const uint32_t (&d)[Fmt<MODE>::kWords], int j) {
  constexpr int kBits = Fmt<MODE>::kBits;
  const int bit = j * kBits, word = bit >> 5, off = bit & 31;
  uint32_t v;
  if (off + kBits <= 32)
    v = d[word] >> off;
  else
    v = __builtin_amdgcn_alignbit(d[word + 1], d[word], off);
  return v & ((1u << kBits) - 1);
}

template <int MODE>
__device__ inline void load_chunk(const uint8_t* __restrict__ p, uint32_t (&d)[Fmt<MODE>::kWords]) {
  const uint32_t* q = reinterpret_cast<const uint32_t*>(p);
  if constexpr (MODE == 0) {
    const u32x4 u = load_stream16(p);
    d[0] = u.x; d[1] = u.y; d[2] = u.z; d[3] = u.w;
  } else if constexpr (MODE == 1) {
#pragma unroll
    for (int i = 0; i < 3; ++i) d[i] = __builtin_nontemporal_load(q + i);
  } else {
    const u32x4 u = load_stream16(p);
    d[0] = u.x; d[1] = u.y; d[2] = u.z; d[3] = u.w;
    d[4] = __builtin_nontemporal_load(q + 4);
  }
}

// B: batch rows (1..8); RW: rows per wave; MODE: code format.
template <int B, int RW, int MODE>
__global__ __launch_bounds__(64 * kWaves) void qgemv_kernel(
    const float* __restrict__ x_rot, const uint8_t* __restrict__ codes,
    const uint16_t* __restrict__ scales, const float* __restrict__ grid, int pair_table,
    int g, int64_t out, int64_t in, float* __restrict__ y) {
  using F = Fmt<MODE>;
  constexpr int kChunkBytes = kChunkCodes * F::kBits / 8;
  extern __shared__ uint32_t s_lut[];

  const int lane = int(threadIdx.x) & 63;
  const int wave = int(threadIdx.x) >> 6;
  const int64_t row_bytes = in / kChunkWeights * kChunkBytes;
  const int64_t groups_per_row = in / g;
  const int nchunks = int(in / kChunkWeights);
  const int nranges = (nchunks + 63) / 64;

  // ---- lookup table: entry c replicated; word (c << R) | replica ----
  {
    constexpr int kWordsTotal = lut_words<MODE>();
    for (int w4 = int(threadIdx.x) * 4; w4 < kWordsTotal; w4 += 64 * kWaves * 4) {
      const int c = w4 >> F::kReplicasLog2;
      uint32_t e;
      if (pair_table)
        e = pack_half2(grid[c & 15], grid[c >> 4]);
      else
        e = pack_half2(grid[2 * c], grid[2 * c + 1]);
      *reinterpret_cast<uint4*>(&s_lut[w4]) = make_uint4(e, e, e, e);
    }
  }
  __syncthreads();

  const int64_t row0 = (int64_t(blockIdx.x) * kWaves + wave) * RW;
  const uint32_t lane_word = F::kReplicasLog2 == 6 ? uint32_t(lane) : uint32_t(lane & 15);

  float acc[RW][B];
#pragma unroll
  for (int i = 0; i < RW; ++i)
#pragma unroll
    for (int b = 0; b < B; ++b) acc[i][b] = 0.f;

  for (int kr = 0; kr < nranges; ++kr) {
    const int chunk = kr * 64 + lane;
    const bool cvalid = chunk < nchunks;

    // codes of this K-range for the wave's rows (issued first: long latency)
    uint32_t d[RW][F::kWords];
#pragma unroll
    for (int i = 0; i < RW; ++i) {
      const int64_t row = row0 + i;
      if (cvalid && row < out) {
        load_chunk<MODE>(codes + row * row_bytes + int64_t(chunk) * kChunkBytes, d[i]);
      } else {
#pragma unroll
        for (int q = 0; q < F::kWords; ++q) d[i][q] = 0;
      }
    }

    // activations of this chunk: fp32 -> exact power-of-two rescale -> fp16 pairs
    half2_t xh[B][kChunkCodes];
    float xscale[B];
#pragma unroll
    for (int b = 0; b < B; ++b) {
      float xv[kChunkWeights];
      if (cvalid) {
        const float4* src =
            reinterpret_cast<const float4*>(x_rot + int64_t(b) * in + int64_t(chunk) * kChunkWeights);
#pragma unroll
        for (int q = 0; q < kChunkWeights / 4; ++q) {
          const float4 f = src[q];
          xv[4 * q] = f.x; xv[4 * q + 1] = f.y; xv[4 * q + 2] = f.z; xv[4 * q + 3] = f.w;
        }
      } else {
#pragma unroll
        for (int q = 0; q < kChunkWeights; ++q) xv[q] = 0.f;
      }
      float m = 0.f;
#pragma unroll
      for (int q = 0; q < kChunkWeights; ++q) m = fmaxf(m, fabsf(xv[q]));
#pragma unroll
      for (int s = 32; s >= 1; s >>= 1) m = fmaxf(m, __shfl_xor(m, s, 64));
      // largest |x| lands in [2^14, 2^15): fp16 keeps 11 bits without overflow
      int e = m > 0.f ? ilogbf(m) - 14 : 0;
      e = e < -126 ? -126 : e;  // keep the power of two a normal float
      xscale[b] = ldexpf(1.0f, e);
#pragma unroll
      for (int j = 0; j < kChunkCodes; ++j) {
        half2_t h;
        h.x = static_cast<_Float16>(ldexpf(xv[2 * j], -e));
        h.y = static_cast<_Float16>(ldexpf(xv[2 * j + 1], -e));
        xh[b][j] = h;
      }
    }

    const int64_t gidx = cvalid ? int64_t(chunk) * kChunkWeights / g : 0;
#pragma unroll
    for (int i = 0; i < RW; ++i) {
      const int64_t row = row0 + i;
      float part[B];
#pragma unroll
      for (int b = 0; b < B; ++b) part[b] = 0.f;
#pragma unroll
      for (int j = 0; j < kChunkCodes; ++j) {
        const uint32_t c = chunk_code<MODE>(d[i], j);
        const uint32_t e = s_lut[(c << F::kReplicasLog2) | lane_word];
        const half2_t gv = __builtin_bit_cast(half2_t, e);
#pragma unroll
        for (int b = 0; b < B; ++b) part[b] = __builtin_amdgcn_fdot2(gv, xh[b][j], part[b], false);
      }
      float sc = 0.f;
      if (cvalid && row < out) {
        const _Float16 h = __builtin_bit_cast(_Float16, scales[row * groups_per_row + gidx]);
        sc = float(h);
      }
#pragma unroll
      for (int b = 0; b < B; ++b) acc[i][b] = fmaf(part[b], sc * xscale[b], acc[i][b]);
    }
  }

#pragma unroll
  for (int i = 0; i < RW; ++i) {
#pragma unroll
    for (int b = 0; b < B; ++b) {
      float v = acc[i][b];
#pragma unroll
      for (int s = 32; s >= 1; s >>= 1) v += __shfl_xor(v, s, 64);
      acc[i][b] = v;
    }
  }
  if (lane == 0) {
#pragma unroll
    for (int i = 0; i < RW; ++i) {
      const int64_t row = row0 + i;
      if (row < out) {
#pragma unroll
        for (int b = 0; b < B; ++b) y[int64_t(b) * out + row] = acc[i][b];
      }
    }
  }
}

template <int B, int MODE>
hipError_t launch_b(int rw, const float* x_rot, const uint8_t* codes, const uint16_t* scales,
                    const float* grid, int pair_table, int g, int64_t out, int64_t in, float* y,
                    hipStream_t stream) {
  const size_t lds = size_t(lut_words<MODE>()) * 4;
  const int64_t rows_per_block = int64_t(kWaves) * rw;
  const dim3 grid_dim{unsigned((out + rows_per_block - 1) / rows_per_block)}, block{64 * kWaves};
  switch (rw) {
    case 1:
      hipLaunchKernelGGL((qgemv_kernel<B, 1, MODE>), grid_dim, block, lds, stream, x_rot, codes,
                         scales, grid, pair_table, g, out, in, y);
      break;
    case 2:
      hipLaunchKernelGGL((qgemv_kernel<B, 2, MODE>), grid_dim, block, lds, stream, x_rot, codes,
                         scales, grid, pair_table, g, out, in, y);
      break;
    default:
      hipLaunchKernelGGL((qgemv_kernel<B, 4, MODE>), grid_dim, block, lds, stream, x_rot, codes,
                         scales, grid, pair_table, g, out, in, y);
      break;
  }
  return hipGetLastError();
}

template <int MODE>
hipError_t launch_mode(int64_t batch, int rw, const float* x_rot, const uint8_t* codes,
                       const uint16_t* scales, const float* grid, int pair_table, int g,
                       int64_t out, int64_t in, float* y, hipStream_t stream) {
  switch (batch) {
    case 1: return launch_b<1, MODE>(rw, x_rot, codes, scales, grid, pair_table, g, out, in, y, stream);
    case 2: return launch_b<2, MODE>(rw, x_rot, codes, scales, grid, pair_table, g, out, in, y, stream);
    case 3: return launch_b<3, MODE>(rw, x_rot, codes, scales, grid, pair_table, g, out, in, y, stream);
    case 4: return launch_b<4, MODE>(rw, x_rot, codes, scales, grid, pair_table, g, out, in, y, stream);
    case 5: return launch_b<5, MODE>(rw, x_rot, codes, scales, grid, pair_table, g, out, in, y, stream);
    case 6: return launch_b<6, MODE>(rw, x_rot, codes, scales, grid, pair_table, g, out, in, y, stream);
    case 7: return launch_b<7, MODE>(rw, x_rot, codes, scales, grid, pair_table, g, out, in, y, stream);
    default: return launch_b<8, MODE>(rw, x_rot, codes, scales, grid, pair_table, g, out, in, y, stream);
  }
}

}  // namespace

hipError_t launch_qgemv(const float* x_rot, int64_t batch, const uint8_t* codes,
                        const uint16_t* scales, const float* grid, int p, int n, int g,
                        int64_t out, int64_t in, float* y, hipStream_t stream) {
  const int bits = code_bits(p, n);
  const int mode = bits == 6 ? 1 : bits == 10 ? 2 : 0;
  const int pair_table = p == 1 ? 1 : 0;
  // rows per wave: aim for at least ~2 blocks per compute unit
  const int rw = out >= 8192 ? 4 : out >= 4096 ? 2 : 1;
  for (int64_t b0 = 0; b0 < batch; b0 += 8) {
    const int64_t nb = std::min<int64_t>(8, batch - b0);
    const float* xb = x_rot + b0 * in;
    float* yb = y + b0 * out;
    hipError_t err;
    if (mode == 0)
      err = launch_mode<0>(nb, rw, xb, codes, scales, grid, pair_table, g, out, in, yb, stream);
    else if (mode == 1)
      err = launch_mode<1>(nb, rw, xb, codes, scales, grid, pair_table, g, out, in, yb, stream);
    else
      err = launch_mode<2>(nb, rw, xb, codes, scales, grid, pair_table, g, out, in, yb, stream);
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

}  // namespace higgs
