// Lookup-table GEMV for HIGGS layers at small batch (1..8 activation rows),
// computed in the rotated space (App. G):
//   y[b][o] = sum_i scale[o][i] * sum_j < G[code(o,i,j)], x_rot[b, ig+jp : ig+(j+1)p] >
// Decoding at this batch is memory bound (Sec. 3.3): the kernel streams the
// packed codes from HBM once, coalesced, and keeps everything else on chip.
//   * A block (8 waves) first stages the activations in LDS as fp16 pairs,
//     rescaled by an exact power of two per batch row and K-range so that any
//     finite fp32 input keeps fp16 precision without overflow, and builds the
//     lookup table of grid points (fp16 pairs) with one copy per lane, so the
//     64 random reads of a wave never share a bank (the grid-in-fast-memory
//     constraint of Sec. 3.3, replicated against bank conflicts).
//   * Each wave then owns tiles of RW rows and walks all of K for them. A
//     K-range is 64 lane chunks; a chunk is 8 (8-bit codes) or 16 (6- and
//     10-bit codes) consecutive codes of a row. Row and K-range offsets are
//     wave-uniform, so loads use a scalar base plus a per-lane offset, and the
//     codes of the next K-range are in flight while the current one decodes.
//   * Per code: one LDS read of the table entry and one v_dot2_f32_f16 per
//     batch row (fp32 accumulation); per row and K-range one group scale.
//   * Lanes are reduced by a fixed butterfly at the end of each tile
//     (deterministic).
// Code formats: MODE 0 = 8-bit codes (p = 2, n = 256; also p = 1, n = 16 read
// as 256 byte values indexing a table of grid-point pairs), MODE 1 = 6-bit
// (p = 2, n = 64), MODE 2 = 10-bit (p = 2, n = 1024).

#include <algorithm>
#include <mutex>
#include <type_traits>

#include "internal.h"
#include "wave_fwht.h"

namespace higgs {
namespace {

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr size_t kLdsLimit = 160 * 1024;

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <int MODE>
struct Fmt;
template <>
struct Fmt<0> {  // 8-bit codes
  static constexpr int kBits = 8, kCodes = 8, kWords = 2, kEntriesLog2 = 8;
};
template <>
struct Fmt<1> {  // 6-bit codes
  static constexpr int kBits = 6, kCodes = 16, kWords = 3, kEntriesLog2 = 6;
};
template <>
struct Fmt<2> {  // 10-bit codes
  static constexpr int kBits = 10, kCodes = 16, kWords = 5, kEntriesLog2 = 10;
};

// Table copies (log2): one per lane where the table is small enough.
template <int MODE, int B>
constexpr int replicas_log2() {
  if constexpr (MODE == 2) return 4;
  else if constexpr (MODE == 0 && B >= 4) return 5;
  else return 6;
}

__device__ inline uint32_t pack_half2(float a, float b) {
  const _Float16 ha = static_cast<_Float16>(a), hb = static_cast<_Float16>(b);
  return uint32_t(__builtin_bit_cast(uint16_t, ha)) |
         (uint32_t(__builtin_bit_cast(uint16_t, hb)) << 16);
}

// Byte offset in the table of the entry of code j of a chunk, for this lane's
// copy (entry-major: code * copies + copy, 4 bytes each).
template <int MODE, int RL>
__device__ inline uint32_t lut_offset(const uint32_t (&d)[Fmt<MODE>::kWords], int j,
                                      uint32_t copy4) {
  constexpr int kBits = Fmt<MODE>::kBits;
  if constexpr (MODE == 0 && RL == 6) {
    // code byte to bits 8..15 next to copy * 4 in bits 0..7: one v_perm_b32
    const uint32_t sel = 0x0c0c0000u | (uint32_t(4 + (j & 3)) << 8);
    return __builtin_amdgcn_perm(d[j >> 2], copy4, sel);
  } else {
    const int bit = j * kBits, word = bit >> 5, off = bit & 31;
    uint32_t v;
    if (off + kBits <= 32)
      v = d[word] >> off;
    else
      v = __builtin_amdgcn_alignbit(d[word + 1], d[word], off);
    return ((v & ((1u << kBits) - 1)) << (RL + 2)) | copy4;
  }
}

// Word 3 of a raw buffer resource on gfx9-family chips (32-bit data format).
constexpr int kRsrcWord3 = 0x00020000;
constexpr int kAuxNT = 2;  // non-temporal: codes and scales are read once

typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef int i32x3 __attribute__((ext_vector_type(3)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

// One chunk of codes: per-lane byte offset voff, wave-uniform byte offset soff.
template <int MODE>
__device__ inline void load_chunk(__amdgpu_buffer_rsrc_t rs, uint32_t voff, uint32_t soff,
                                  uint32_t (&d)[Fmt<MODE>::kWords]) {
  if constexpr (MODE == 0) {
    const i32x2 u = __builtin_amdgcn_raw_buffer_load_b64(rs, int(voff), int(soff), kAuxNT);
    d[0] = uint32_t(u.x);
    d[1] = uint32_t(u.y);
  } else if constexpr (MODE == 1) {
    const i32x3 u = __builtin_amdgcn_raw_buffer_load_b96(rs, int(voff), int(soff), kAuxNT);
    d[0] = uint32_t(u.x);
    d[1] = uint32_t(u.y);
    d[2] = uint32_t(u.z);
  } else {
    const i32x4 u = __builtin_amdgcn_raw_buffer_load_b128(rs, int(voff), int(soff), kAuxNT);
    d[0] = uint32_t(u.x); d[1] = uint32_t(u.y); d[2] = uint32_t(u.z); d[3] = uint32_t(u.w);
    d[4] = uint32_t(__builtin_amdgcn_raw_buffer_load_b32(rs, int(voff + 16), int(soff), kAuxNT));
  }
}

// Sums each of the V values of a lane over the 64 lanes of the wave (V a
// power of two <= 64). Step K exchanges with lane ^ (32 >> K); while more than
// one value is left, each exchange sends half of them to the partner, so the
// count halves per step. Afterwards the total of value k is held by every
// lane whose top log2(V) bits equal k. Steps are compile-time so that every
// value stays in a register.
template <int V, int K>
struct TransposeReduce {
  static __device__ inline void run(float (&v)[V], int lane) {
    constexpr int M = 32 >> K;
    constexpr int C = V >> K;  // values left before this step
    if constexpr (C > 1) {
      const bool upper = (lane & M) != 0;
#pragma unroll
      for (int i = 0; i < C / 2; ++i) {
        const float a = v[i], b = v[i + C / 2];
        const float send = upper ? a : b;
        const float keep = upper ? b : a;
        v[i] = keep + __shfl_xor(send, M, 64);
      }
    } else {
      v[0] += __shfl_xor(v[0], M, 64);
    }
    if constexpr (K < 5) TransposeReduce<V, K + 1>::run(v, lane);
  }
};

template <int V>
__device__ inline float transpose_reduce(float (&v)[V], int lane) {
  static_assert((V & (V - 1)) == 0 && V <= 64, "V must be a power of two <= 64");
  TransposeReduce<V, 0>::run(v, lane);
  return v[0];
}

struct Layout {  // dynamic LDS carve-up, in bytes
  int x, xs, compact, total;
};

template <int B, int MODE>
__host__ __device__ constexpr int lut_bytes() {
  return 4 << (Fmt<MODE>::kEntriesLog2 + replicas_log2<MODE, B>());
}

template <int B, int MODE>
__host__ __device__ inline Layout lds_layout(int nranges, int groups_per_row) {
  Layout L{};
  L.x = 0;
  const int xbytes = B * nranges * 64 * Fmt<MODE>::kCodes * 4;
  L.xs = L.x + xbytes;
  L.compact = L.xs + ((B * groups_per_row * 4 + 15) & ~15);
  L.total = L.compact + (4 << Fmt<MODE>::kEntriesLog2);
  return L;
}

// One group of g = 64*E activations of one batch row, held by one wave (lane l
// has elements l*E .. l*E+E-1): optionally rotated (sigma, FWHT, 1/sqrt(g);
// App. G), rescaled by an exact power of two so that the largest magnitude
// lands in [2^14, 2^15), and written to LDS as fp16 pairs in the layout the
// decode loop reads (chunk-major: lane chunk c of K-range kr at
// ((b * nranges + kr) * 64 + c % 64) * kCodes).
template <int E>
struct XGroup {
  float v[E];

  __device__ inline void load(const void* x, int x_bf16, int64_t off, bool real) {
    if (!real) {
#pragma unroll
      for (int i = 0; i < E; ++i) v[i] = 0.f;
      return;
    }
    if (x_bf16) {
      const uint16_t* p = static_cast<const uint16_t*>(x) + off;
      if constexpr (E % 8 == 0) {
#pragma unroll
        for (int q = 0; q < E / 8; ++q) {
          const u32x4 u = *reinterpret_cast<const u32x4*>(p + 8 * q);
          const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            v[8 * q + 2 * t] = __uint_as_float(w[t] << 16);
            v[8 * q + 2 * t + 1] = __uint_as_float(w[t] & 0xffff0000u);
          }
        }
      } else {
#pragma unroll
        for (int i = 0; i < E; ++i) v[i] = __uint_as_float(uint32_t(p[i]) << 16);
      }
    } else {
      const float* p = static_cast<const float*>(x) + off;
      if constexpr (E % 4 == 0) {
#pragma unroll
        for (int q = 0; q < E / 4; ++q) {
          const float4 f = *reinterpret_cast<const float4*>(p + 4 * q);
          v[4 * q] = f.x; v[4 * q + 1] = f.y; v[4 * q + 2] = f.z; v[4 * q + 3] = f.w;
        }
      } else {
#pragma unroll
        for (int i = 0; i < E; ++i) v[i] = p[i];
      }
    }
  }

  template <int kCodes>
  __device__ inline void stage(int rot, uint64_t seed, int lane, int b, int gblk, int nranges,
                               int groups_per_row, _Float16* s_xh, float* s_xs) {
    constexpr int G = 64 * E;
    if (rot) {
#pragma unroll
      for (int i = 0; i < E; ++i)
        if (rht_sign_negative(seed, uint32_t(lane * E + i))) v[i] = -v[i];
      fwht_wave<E>(v, lane, G);
      // the same constant the separate rotation kernel uses (fp32 of the fp64 value)
      const float rs = float(1.0 / sqrt(double(G)));
#pragma unroll
      for (int i = 0; i < E; ++i) v[i] *= rs;
    }
    float m = 0.f;
#pragma unroll
    for (int i = 0; i < E; ++i) m = fmaxf(m, fabsf(v[i]));
#pragma unroll
    for (int sh = 32; sh >= 1; sh >>= 1) m = fmaxf(m, __shfl_xor(m, sh, 64));
    int e = m > 0.f ? ilogbf(m) - 14 : 0;
    e = e < -126 ? -126 : e;
    constexpr int kCW = 2 * kCodes;  // weights per lane chunk
#pragma unroll
    for (int i = 0; i < E; ++i) {
      const int k = gblk * G + lane * E + i;  // element index in the row
      const int c = k / kCW;
      const int kr = c >> 6, cl = c & 63;
      s_xh[(((b * nranges + kr) * 64 + cl) * kCodes) * 2 + (k % kCW)] =
          static_cast<_Float16>(ldexpf(v[i], -e));
    }
    if (lane == 0) s_xs[b * groups_per_row + gblk] = ldexpf(1.0f, e);
  }
};

constexpr int kDepth = 4;  // items (tile, K-range) whose codes are in flight per wave

// B: batch rows per launch (1, 2, 4, 8; nb <= B are real); RW: rows per wave
// tile; MODE: code format; USC: one scale group spans a whole K-range
// (g >= 64 chunks), so an item's scales are wave-uniform and come through
// scalar loads instead of vector ones.
// The activations x are either already rotated (rot = 0, fp32) or raw
// (rot = 1, fp32 or bf16), in which case the kernel applies the rotation with
// `seed` while staging them.
template <int B, int RW, int MODE, bool USC>
__global__ __launch_bounds__(kThreads) void qgemv_kernel(
    const void* __restrict__ x, int x_bf16, int rot, uint64_t seed, int nb,
    const uint8_t* __restrict__ codes, const uint16_t* __restrict__ scales,
    const float* __restrict__ grid, int pair_table, int log2g, int64_t out, int64_t in,
    float* __restrict__ y) {
  using F = Fmt<MODE>;
  constexpr int RL = replicas_log2<MODE, B>();
  constexpr int kChunkBytes = F::kCodes * F::kBits / 8;
  constexpr int kChunkWeights = 2 * F::kCodes;
  constexpr int kEntries = 1 << F::kEntriesLog2;
  constexpr int kLutWords = kEntries << RL;
  constexpr int kV = RW * B;
  static_assert((kV & (kV - 1)) == 0 && kV <= 64, "RW * B must be a power of two <= 64");

  __shared__ u32x4 s_lut4[kLutWords / 4];
  extern __shared__ u32x4 smem4[];
  char* smem = reinterpret_cast<char*>(smem4);
  uint32_t* s_lut = reinterpret_cast<uint32_t*>(s_lut4);

  const int lane = int(threadIdx.x) & 63;
  // wave index is uniform: keep it (and all row addressing) in scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
  const int nchunks = int(in / kChunkWeights);
  const int nranges = (nchunks + 63) / 64;
  // activations are staged in sub-blocks of min(g, 1024) (one wave each, at
  // most 16 values per lane); each has its own power-of-two rescale
  const int log2sub = log2g < 10 ? log2g : 10;
  const int gpr = int(in >> log2sub);
  const Layout L = lds_layout<B, MODE>(nranges, gpr);
  half2_t* s_x = reinterpret_cast<half2_t*>(smem + L.x);
  float* s_xs = reinterpret_cast<float*>(smem + L.xs);
  uint32_t* s_compact = reinterpret_cast<uint32_t*>(smem + L.compact);

  const uint32_t row_bytes = uint32_t(nchunks) * kChunkBytes;
  const uint32_t groups_per_row = uint32_t(in >> log2g);
  const int64_t ntiles = (out + RW - 1) / RW;
  const int64_t wave_stride = int64_t(gridDim.x) * kWaves;
  const int64_t tile0 = int64_t(blockIdx.x) * kWaves + wave;  // first tile of this wave
  const int64_t my_tiles = tile0 < ntiles ? (ntiles - 1 - tile0) / wave_stride + 1 : 0;
  const int64_t nitems = my_tiles * nranges;

  // ---- 1. small loads first (they are waited on first): grid points for the
  //         table ----
  constexpr int kPer = (kEntries + kThreads - 1) / kThreads;
  float gx[kPer], gy[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {  // branch free: clamped entry index
    const int c = min(int(threadIdx.x) + u * kThreads, kEntries - 1);
    gx[u] = pair_table ? grid[c & 15] : grid[2 * c];
    gy[u] = pair_table ? grid[c >> 4] : grid[2 * c + 1];
  }

  // ---- 2. codes and group scales of the first kDepth items. Items are
  //         (tile, K-range) pairs, K-range fastest; (ft, fk) is the next item
  //         to fetch. Out-of-range lanes / rows read a clamped in-bounds
  //         address and are zeroed later through their scale. ----
  uint32_t buf[kDepth][RW][F::kWords];
  uint32_t sbuf[kDepth][RW];
  int64_t ft = tile0;
  int fk = 0;
  int64_t fetched = 0;
  // Buffer resources over the exact code and scale arrays: every load below
  // uses a clamped in-range offset, so the range check never triggers.
  const __amdgpu_buffer_rsrc_t crs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(codes), 0, int(uint32_t(out) * row_bytes), kRsrcWord3);
  // dword view of the scales, used only when the host has checked that the
  // array is dword aligned and holds an even number of scales
  const uint32_t* __restrict__ scales32 = reinterpret_cast<const uint32_t*>(scales);
  const __amdgpu_buffer_rsrc_t srs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(scales), 0, int(uint32_t(out) * groups_per_row * 2u), kRsrcWord3);
  auto fetch = [&](uint32_t (&d)[RW][F::kWords], uint32_t (&sc)[RW]) {
    if (fetched >= nitems) return;  // uniform
    const int cl = min(fk * 64 + lane, nchunks - 1);  // clamped chunk of this lane
    const uint32_t voff_c = uint32_t(cl - fk * 64) * kChunkBytes;
    const uint32_t voff_s = uint32_t((cl * kChunkWeights) >> log2g) * 2u;
    const uint32_t kofs = uint32_t(fk) * (64u * kChunkBytes);
    const int64_t row0 = ft * RW;
#pragma unroll
    for (int r = 0; r < RW; ++r) {
      const uint32_t rc = uint32_t(min(row0 + r, out - 1));  // uniform
      load_chunk<MODE>(crs, voff_c, rc * row_bytes + kofs, d[r]);
      if constexpr (USC) {
        // the dword holding scale (rc, group of this K-range): scalar load
        const uint32_t idx = rc * groups_per_row + ((uint32_t(fk) * (64u * kChunkWeights)) >> log2g);
        const uint32_t w = __builtin_amdgcn_readfirstlane(scales32[idx >> 1]);
        sc[r] = (idx & 1) ? (w >> 16) : (w & 0xffffu);
      } else {
        sc[r] = uint32_t(uint16_t(__builtin_amdgcn_raw_buffer_load_b16(
            srs, int(voff_s), int(rc * groups_per_row * 2u), kAuxNT)));
      }
    }
    ++fetched;
    if (++fk == nranges) {
      fk = 0;
      ft += wave_stride;
    }
  };
  // ---- 2b/3. this wave's first activation group is requested before the
  //      codes (so waiting for it does not wait for them), then the codes of
  //      the first kDepth items, then the table and the staged activations.
  //      Tasks are (batch row, group) pairs, wave w taking w, w + 8, ... ----
  const int ntasks = B * gpr;
  auto prologue = [&](auto e_tag) {
    constexpr int E = decltype(e_tag)::value;
    XGroup<E> xg;
    auto task_off = [&](int t) { return int64_t(t / gpr) * in + int64_t(t % gpr) * (64 * E) + lane * E; };
    if (wave < ntasks) xg.load(x, x_bf16, task_off(wave), wave / gpr < nb);
#pragma unroll
    for (int s = 0; s < kDepth; ++s) fetch(buf[s], sbuf[s]);
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int c = int(threadIdx.x) + u * kThreads;
      if (c < kEntries) s_compact[c] = pack_half2(gx[u], gy[u]);
    }
    _Float16* s_xh = reinterpret_cast<_Float16*>(s_x);
    for (int t = wave; t < ntasks; t += kWaves) {
      if (t != wave) xg.load(x, x_bf16, task_off(t), t / gpr < nb);
      xg.template stage<F::kCodes>(rot, seed, lane, t / gpr, t % gpr, nranges, gpr, s_xh, s_xs);
    }
  };
  switch (log2sub) {  // the host only rotates here when g <= 1024 (sub = g)
    case 6: prologue(std::integral_constant<int, 1>{}); break;
    case 7: prologue(std::integral_constant<int, 2>{}); break;
    case 8: prologue(std::integral_constant<int, 4>{}); break;
    case 9: prologue(std::integral_constant<int, 8>{}); break;
    default: prologue(std::integral_constant<int, 16>{}); break;
  }
  __syncthreads();
  for (int w4 = int(threadIdx.x) * 4; w4 < kLutWords; w4 += kThreads * 4) {
    const uint32_t e = s_compact[w4 >> RL];
    *reinterpret_cast<u32x4*>(&s_lut[w4]) = u32x4{e, e, e, e};
  }
  __syncthreads();

  // ---- 4. decode: (pt, pk) is the item being processed ----
  const uint32_t copy4 = (uint32_t(lane) & ((1u << RL) - 1)) << 2;
  float acc[RW][B];
#pragma unroll
  for (int r = 0; r < RW; ++r)
#pragma unroll
    for (int b = 0; b < B; ++b) acc[r][b] = 0.f;
  int64_t pt = tile0;
  int pk = 0;

  auto process = [&](const uint32_t (&d)[RW][F::kWords], const uint32_t (&sc)[RW]) {
    const int rvalid = int(min(int64_t(RW), out - pt * RW));
    half2_t xh[B][F::kCodes];
    float xs[B];
    // staging sub-block of this lane's chunk
    const int xg = (min(pk * 64 + lane, nchunks - 1) * kChunkWeights) >> log2sub;
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const half2_t* src = s_x + ((b * nranges + pk) * 64 + lane) * F::kCodes;
#pragma unroll
      for (int j = 0; j < F::kCodes; ++j) xh[b][j] = src[j];
      xs[b] = s_xs[b * gpr + xg];
    }
#pragma unroll
    for (int r = 0; r < RW; ++r) {
      float part[B];
#pragma unroll
      for (int b = 0; b < B; ++b) part[b] = 0.f;
#pragma unroll
      for (int j = 0; j < F::kCodes; ++j) {
        const uint32_t off = lut_offset<MODE, RL>(d[r], j, copy4);
        const half2_t gv = __builtin_bit_cast(
            half2_t, *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(s_lut) + off));
#pragma unroll
        for (int b = 0; b < B; ++b) part[b] = __builtin_amdgcn_fdot2(gv, xh[b][j], part[b], false);
      }
      const float sc_r = float(__builtin_bit_cast(_Float16, uint16_t(sc[r])));
#pragma unroll
      for (int b = 0; b < B; ++b) acc[r][b] = fmaf(part[b], sc_r * xs[b], acc[r][b]);
    }
    if (pk == nranges - 1) {
      float flat[kV];
#pragma unroll
      for (int r = 0; r < RW; ++r)
#pragma unroll
        for (int b = 0; b < B; ++b) {
          flat[r * B + b] = acc[r][b];
          acc[r][b] = 0.f;
        }
      const float total = transpose_reduce<kV>(flat, lane);
      constexpr int kShift = 6 - __builtin_ctz(kV);
      const int k = lane >> kShift;
      const int r = k / B, b = k - (k / B) * B;
      if ((lane & ((1 << kShift) - 1)) == 0 && r < rvalid && b < nb)
        y[int64_t(b) * out + pt * RW + r] = total;
      pk = 0;
      pt += wave_stride;
    } else {
      ++pk;
    }
  };

  for (int64_t i = 0; i < nitems; i += kDepth) {
#pragma unroll
    for (int s = 0; s < kDepth; ++s) {
      if (i + s < nitems) {  // uniform
        process(buf[s], sbuf[s]);
        fetch(buf[s], sbuf[s]);
      }
    }
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

// Activation operand of a launch: already rotated fp32 (rot = 0) or raw
// fp32 / bf16 to be rotated with `seed` (rot = 1).
struct XArg {
  const void* x;
  int x_bf16, rot;
  uint64_t seed;
  const void* rows(int64_t b0, int64_t in) const {
    return static_cast<const char*>(x) + b0 * in * (x_bf16 ? 2 : 4);
  }
};

struct Job {
  XArg xa;
  int nb;
  const uint8_t* codes;
  const uint16_t* scales;
  const float* grid;
  int pair_table, log2g;
  int64_t out, in;
  float* y;
  hipStream_t stream;
};

template <int B, int RW, int MODE, bool USC>
hipError_t launch_rw_usc(const Job& j) {
  using F = Fmt<MODE>;
  const int nchunks = int(j.in / (2 * F::kCodes));
  const int nranges = (nchunks + 63) / 64;
  const Layout L = lds_layout<B, MODE>(nranges, int(j.in >> std::min(j.log2g, 10)));
  static std::once_flag attr_once;
  static hipError_t attr_err = hipSuccess;
  std::call_once(attr_once, [] {
    attr_err = hipFuncSetAttribute(reinterpret_cast<const void*>(&qgemv_kernel<B, RW, MODE, USC>),
                                   hipFuncAttributeMaxDynamicSharedMemorySize,
                                   int(kLdsLimit) - lut_bytes<B, MODE>());
  });
  if (attr_err != hipSuccess) return attr_err;
  const int64_t ntiles = (j.out + RW - 1) / RW;
  const size_t lds = size_t(L.total) + size_t(lut_bytes<B, MODE>());
  const int per_cu = std::max(1, std::min(2, int(kLdsLimit / lds)));
  const int64_t blocks =
      std::max<int64_t>(1, std::min<int64_t>((ntiles + kWaves - 1) / kWaves,
                                             int64_t(device_cus()) * per_cu));
  hipLaunchKernelGGL((qgemv_kernel<B, RW, MODE, USC>), dim3(unsigned(blocks)), dim3(kThreads),
                     size_t(L.total), j.stream, j.xa.x, j.xa.x_bf16, j.xa.rot, j.xa.seed, j.nb,
                     j.codes, j.scales, j.grid, j.pair_table, j.log2g, j.out, j.in, j.y);
  return hipGetLastError();
}

template <int B, int RW, int MODE>
hipError_t launch_rw(const Job& j) {
  constexpr int kRangeWeights = 64 * 2 * Fmt<MODE>::kCodes;
  // scalar path reads whole dwords: needs a dword-aligned array of even length
  if ((int64_t(1) << j.log2g) >= kRangeWeights && reinterpret_cast<uintptr_t>(j.scales) % 4 == 0 &&
      (j.out * (j.in >> j.log2g)) % 2 == 0)
    return launch_rw_usc<B, RW, MODE, true>(j);
  return launch_rw_usc<B, RW, MODE, false>(j);
}

// Rows per wave tile: the largest of 2, 4, 8 that still gives every wave of a
// full-chip launch a tile, within a per-format register budget of
// accumulators (RW * B).
template <int B, int MODE>
hipError_t launch_b(const Job& j) {
  constexpr int kVmax = MODE == 0 ? 32 : MODE == 1 ? 16 : 8;
  constexpr int kRWmax = MODE == 0 ? 8 : 4;
  const int64_t waves = int64_t(device_cus()) * kWaves;  // one block per CU
  if constexpr (8 <= kRWmax && 8 * B <= kVmax) {
    if (j.out / 8 >= 2 * waves) return launch_rw<B, 8, MODE>(j);
  }
  if constexpr (4 * B <= kVmax) {
    if (j.out / 4 >= waves || 2 * B > kVmax) return launch_rw<B, 4, MODE>(j);
  }
  return launch_rw<B, 2, MODE>(j);
}

// Largest batch per launch whose staged activations fit in LDS next to the table.
template <int MODE>
int max_batch_for(int64_t in, int log2g) {
  const int nranges = int((in / (2 * Fmt<MODE>::kCodes) + 63) / 64);
  const int gpr = int(in >> std::min(log2g, 10));
  if (lds_layout<8, MODE>(nranges, gpr).total + lut_bytes<8, MODE>() <= int(kLdsLimit)) return 8;
  if (lds_layout<4, MODE>(nranges, gpr).total + lut_bytes<4, MODE>() <= int(kLdsLimit)) return 4;
  if (lds_layout<2, MODE>(nranges, gpr).total + lut_bytes<2, MODE>() <= int(kLdsLimit)) return 2;
  if (lds_layout<1, MODE>(nranges, gpr).total + lut_bytes<1, MODE>() <= int(kLdsLimit)) return 1;
  return 0;
}

template <int MODE>
hipError_t launch_mode(const Job& j) {
  if (j.nb == 1) return launch_b<1, MODE>(j);
  if (j.nb == 2) return launch_b<2, MODE>(j);
  if (j.nb <= 4) return launch_b<4, MODE>(j);
  return launch_b<8, MODE>(j);
}

hipError_t run_qgemv(const XArg& xa, int64_t batch, const uint8_t* codes, const uint16_t* scales,
                     const float* grid, int p, int n, int g, int64_t out, int64_t in, float* y,
                     hipStream_t stream) {
  const int bits = code_bits(p, n);
  const int mode = bits == 6 ? 1 : bits == 10 ? 2 : 0;
  const int log2g = log2_exact(g);
  const int cap = mode == 0 ? max_batch_for<0>(in, log2g)
                            : mode == 1 ? max_batch_for<1>(in, log2g) : max_batch_for<2>(in, log2g);
  if (cap == 0) return hipErrorInvalidValue;
  for (int64_t b0 = 0; b0 < batch; b0 += cap) {
    Job j{xa, int(std::min<int64_t>(cap, batch - b0)), codes, scales, grid, p == 1 ? 1 : 0,
          log2g, out, in, y + b0 * out, stream};
    j.xa.x = xa.rows(b0, in);
    const hipError_t err = mode == 0 ? launch_mode<0>(j) : mode == 1 ? launch_mode<1>(j)
                                                                    : launch_mode<2>(j);
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

}  // namespace

int64_t qgemv_max_in(int p, int n, int g) {
  const int bits = code_bits(p, n);
  const int log2g = log2_exact(g);
  int64_t best = 0;
  for (int64_t in = g; in <= (int64_t(1) << 20); in += g) {
    const int mb = bits == 6 ? max_batch_for<1>(in, log2g)
                             : bits == 10 ? max_batch_for<2>(in, log2g) : max_batch_for<0>(in, log2g);
    if (mb == 0) break;
    best = in;
  }
  return best;
}

hipError_t launch_qgemv(const float* x_rot, int64_t batch, const uint8_t* codes,
                        const uint16_t* scales, const float* grid, int p, int n, int g,
                        int64_t out, int64_t in, float* y, hipStream_t stream) {
  return run_qgemv(XArg{x_rot, 0, 0, 0}, batch, codes, scales, grid, p, n, g, out, in, y, stream);
}

hipError_t launch_qgemv_rotating(const void* x, int x_bf16, uint64_t seed, int64_t batch,
                                 const uint8_t* codes, const uint16_t* scales, const float* grid,
                                 int p, int n, int g, int64_t out, int64_t in, float* y,
                                 hipStream_t stream) {
  return run_qgemv(XArg{x, x_bf16, 1, seed}, batch, codes, scales, grid, p, n, g, out, in, y,
                   stream);
}

}  // namespace higgs
