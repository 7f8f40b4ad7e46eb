// Lookup-table GEMM for HIGGS layers at larger batches on the matrix cores,
// computed in the rotated space (App. G):
//   y[b][o] = sum_i scale[o][i] * sum_j < G[code(o,i,j)], x_rot[b, ig+jp : ig+(j+1)p] >
// At these batch sizes the layer is a dense contraction, so the dequantised
// weights feed the matrix cores directly (v_mfma_f32_32x32x16_f16 with 32- or
// 64-column batch tiles, v_mfma_f32_16x16x32_f16 with a 16-column tile for
// up to 16 rows). Two kernels per call, and a third when K is split:
//   * xprep_kernel (g < 256: one wave per group) or xprep4_kernel (g >= 256:
//     4 waves per group) converts the activations once: optionally rotating
//     raw activations first (sign flip, fast Walsh-Hadamard transform,
//     1/sqrt(g), the same arithmetic as the separate rotation kernel), then
//     an exact power-of-two rescale per batch row and group so that the group's
//     largest magnitude lands in [2^14, 2^15). fp16 then keeps full
//     precision and cannot overflow. Output: fp16 activations and one
//     power of two per (row, group), in the workspace.
//   * qgemm_kernel: a block owns 128 rows (4 waves x 32) and a K-range; K is
//     split across blocks when the layer has too few rows to fill the chip
//     (partial sums go to the workspace and are added in a fixed order by
//     qgemm_reduce: deterministic), consecutive blocks taking consecutive
//     splits so that each XCD reads the activations of a few splits only.
//     A operand: each lane holds the codes of 32 weights of its row (16
//     codes: 16, 12 or 20 bytes for 8-, 6- or 10-bit codes) per 64-weight
//     K-block and turns them into fp16 pairs through an LDS lookup table
//     replicated against bank conflicts (32 copies of the 256 entries, 64 of
//     64, or 16 of 1024). 8- and 6-bit codes are fetched two stages ahead as
//     whole row pieces (eight lanes read one row's 256 weights: a 128-byte
//     line for 8-bit codes; reading 32 rows x 32 bytes per load instead
//     streamed them at about half the rate) and moved into that layout
//     through the wave's own LDS rows at the stage's start; 10-bit and
//     scalar 8-bit codes are read in the operand layout directly. The MFMA's
//     reduction index is mapped so that lane half h of step s covers weights
//     32h + 8s .. +7 of the K-block, for A and B alike (the 16-column tile's
//     layout is described at qgemm_kernel).
//     B operand: the fp16 activations of one stage (256 weights of K) in
//     LDS; the next stage's are loaded into registers while the current one
//     is multiplied, together with the next stage's group scales and
//     activation exponents.
//     Products accumulate in fp32 MFMA registers; every FOLD K-blocks the
//     group scale and activation exponent are applied and the result is
//     added into fp32 totals (one rounding: an fma by an exactly scaled
//     factor).
// Every global load is unconditional (buffer loads with an out-of-range
// offset return zero without touching memory), so waiting for one load never
// waits for a later-issued one.
// Code formats: 8-bit codes (p = 2, n = 256; p = 1, n = 16 read as byte
// values indexing a table of grid-point pairs), 6-bit (p = 2, n = 64) and
// 10-bit (p = 2, n = 1024) codes, and scalar 8-bit codes (p = 1, n = 256,
// two lookups of single values per pair of weights; "16 bits per pair").

#include <algorithm>
#include <cmath>
#include <type_traits>

#include "internal.h"
#include "wave_fwht.h"

namespace higgs {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kTileRows = 32 * kWaves;  // rows per block
constexpr int kStageK = 256;            // weights of K per staged activation chunk
constexpr int kStageKB = kStageK / 64;  // K-blocks per stage
constexpr int kXRow = kStageK + 8;      // halves per staged activation row (padded)
constexpr int kRing = 2 * kStageKB;     // ring slots of codes in flight per lane (two stages)
constexpr int kMaxGroup = 4;            // layers of one launch (they share the activations)

// Word 3 of a raw buffer resource on gfx9-family chips (32-bit data format).
constexpr int kRsrcWord3 = 0x00020000;
// Cache policy of the code loads: the default. A row's 128-byte line of
// codes is read in four pieces over four K-blocks (or super-blocks), so it
// must stay in L2 between them; with the non-temporal hint it was evicted
// early and a batch-64 product fetched 1.5-1.8x its code bytes.
constexpr int kAuxCodes = 0;
// Per-lane buffer offset beyond any buffer here (< 2^31 bytes): reads zero.
constexpr uint32_t kOffNone = 0x80000000u;

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f16x_acc __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x3 __attribute__((ext_vector_type(3)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

// Code width: table copies (log2), log2 of a table entry's stride in bytes,
// code dwords per lane and K-block (16 codes), and whether codes are read as
// whole 128-byte lines and transposed through LDS (kCT, below).
// 8-bit: 32 copies in the low half of each 256-byte entry slot (64 KiB);
// the slots' high halves hold the code transposition rows. 6-bit: one copy
// per lane (16 KiB) and a separate transposition area. 10-bit: 16 copies
// (64 KiB). Scalar 8-bit codes: one copy per lane (64 KiB).
template <int BITS>
struct GFmt;
template <>
struct GFmt<8> {
  static constexpr int kRL = 5, kStride = 8, kWords = 4;
  static constexpr bool kCT = true;
};
template <>
struct GFmt<6> {
  static constexpr int kRL = 6, kStride = 8, kWords = 3;
  static constexpr bool kCT = true;
};
template <>
struct GFmt<10> {
  static constexpr int kRL = 4, kStride = 6, kWords = 5;
  static constexpr bool kCT = false;
};
// Scalar 8-bit codes (p = 1, n = 256): a pair of weights is two codes, each
// looked up on its own in a table of 256 single values (low half of the
// entry word, same addressing as the 8-bit pair codes).
template <>
struct GFmt<16> {
  static constexpr int kRL = 6, kStride = 8, kWords = 8;
  static constexpr bool kCT = false;
};

// Byte offset in the table of code c (0..15) of a lane's K-block for this
// lane's copy. 8-bit: one v_perm_b32 puts the code byte in byte 1 and the
// lane's copy offset (lane * 4 < 256) in byte 0, which is the address
// code * 256 + lane * 4 of a table with one copy per lane (entry stride 256
// bytes); otherwise the code's bit field, shifted to the entry stride,
// or'ed with copy * 4. lut_off_byte is the 8-bit form for byte b (0 ..
// 4 kWords - 1) of the lane's codes (scalar codes use it per weight).
template <int kWords>
__device__ inline uint32_t lut_off_byte(const uint32_t (&d)[kWords], int b, uint32_t copy_off) {
  const uint32_t sel = 0x0c0c0000u | (uint32_t(4 + (b & 3)) << 8);
  return __builtin_amdgcn_perm(d[b >> 2], copy_off, sel);
}

template <int BITS>
__device__ inline uint32_t lut_off(const uint32_t (&d)[GFmt<BITS>::kWords], int c,
                                   uint32_t copy_off) {
  if constexpr (BITS == 8) {
    return lut_off_byte<GFmt<8>::kWords>(d, c, copy_off);
  } else {
    constexpr int ST = GFmt<BITS>::kStride;
    const int bit = c * BITS, w = bit >> 5, o = bit & 31;
    uint32_t v;
    if (o + BITS <= 32)
      v = d[w] >> o;
    else
      v = __builtin_amdgcn_alignbit(d[w + 1], d[w], o);
    return ((v & ((1u << BITS) - 1u)) << ST) | copy_off;
  }
}

typedef uint32_t u32x3 __attribute__((ext_vector_type(3)));

// kW dwords to / from LDS at a 16-byte aligned byte address (one ds_write /
// ds_read of 12 or 16 bytes).
template <int kW>
__device__ inline void lds_put(char* base, uint32_t off, const uint32_t (&d)[kW]) {
  static_assert(kW == 3 || kW == 4, "12 or 16 bytes");
  if constexpr (kW == 4)
    *reinterpret_cast<u32x4*>(base + off) = u32x4{d[0], d[1], d[2], d[3]};
  else
    *reinterpret_cast<u32x3*>(base + off) = u32x3{d[0], d[1], d[2]};
}
template <int kW>
__device__ inline void lds_get(const char* base, uint32_t off, uint32_t (&d)[kW]) {
  static_assert(kW == 3 || kW == 4, "12 or 16 bytes");
  if constexpr (kW == 4) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(base + off);
    d[0] = v.x; d[1] = v.y; d[2] = v.z; d[3] = v.w;
  } else {
    const u32x3 v = *reinterpret_cast<const u32x3*>(base + off);
    d[0] = v.x; d[1] = v.y; d[2] = v.z;
  }
}

// One lane's codes of one K-block (kWords dwords at byte offset off).
template <int BITS>
__device__ inline void load_codes(__amdgpu_buffer_rsrc_t rs, uint32_t off,
                                  uint32_t (&d)[GFmt<BITS>::kWords]) {
  if constexpr (BITS == 8) {
    const i32x4 u = __builtin_amdgcn_raw_buffer_load_b128(rs, int(off), 0, kAuxCodes);
    d[0] = uint32_t(u.x); d[1] = uint32_t(u.y); d[2] = uint32_t(u.z); d[3] = uint32_t(u.w);
  } else if constexpr (BITS == 16) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const i32x4 u =
          __builtin_amdgcn_raw_buffer_load_b128(rs, int(off + 16u * q), 0, kAuxCodes);
      d[4 * q] = uint32_t(u.x); d[4 * q + 1] = uint32_t(u.y);
      d[4 * q + 2] = uint32_t(u.z); d[4 * q + 3] = uint32_t(u.w);
    }
  } else if constexpr (BITS == 6) {
    const i32x3 u = __builtin_amdgcn_raw_buffer_load_b96(rs, int(off), 0, kAuxCodes);
    d[0] = uint32_t(u.x); d[1] = uint32_t(u.y); d[2] = uint32_t(u.z);
  } else {
    const i32x4 u = __builtin_amdgcn_raw_buffer_load_b128(rs, int(off), 0, kAuxCodes);
    d[0] = uint32_t(u.x); d[1] = uint32_t(u.y); d[2] = uint32_t(u.z); d[3] = uint32_t(u.w);
    d[4] = uint32_t(__builtin_amdgcn_raw_buffer_load_b32(rs, int(off + 16u), 0, kAuxCodes));
  }
}

__device__ inline uint32_t pack_h2(float a, float b) {
  const _Float16 ha = static_cast<_Float16>(a), hb = static_cast<_Float16>(b);
  return uint32_t(__builtin_bit_cast(uint16_t, ha)) |
         (uint32_t(__builtin_bit_cast(uint16_t, hb)) << 16);
}

__device__ inline u32x4 as_u32x4(i32x4 v) {
  return u32x4{uint32_t(v.x), uint32_t(v.y), uint32_t(v.z), uint32_t(v.w)};
}

__device__ inline __amdgpu_buffer_rsrc_t rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, int(bytes), kRsrcWord3);
}

// ---------------------------------------------------------------------------
// Activations -> fp16 + one power of two per (batch row, group).
// One wave per group of g = 64 E elements (lane l holds [lE, (l+1)E)).
// ---------------------------------------------------------------------------
// Rotation seeds of the layers of one launch: layer l's activations go to
// copy l of the fp16 buffer and to xe + l * ngroups (one copy per layer when
// the layers rotate with their own seeds; nl = 1 when they share the copy).
struct XSeeds {
  uint64_t s[kMaxGroup];
  int nl;
};

// Layout of the fp16 activations: per layer copy, 64-row batch chunks; per
// chunk, stage-major: stage s (weights [256 s, 256 s + 256) of a row) of the
// chunk's R = min(batch, 64) rows is one contiguous block (32 KiB at R = 64),
// row after row. A product block
// stages a K-stage of its chunk with fully coalesced 1 KiB reads, and the
// blocks of a layer, which read the same stage at about the same time, fetch
// one contiguous region instead of 64 rows at a stride of the row length
// (a multiple of the memory channel interleave: every row's piece would
// fall in the same channels).
struct XLayout {
  int64_t chunk_halves;  // halves of one chunk: stages * R * 256
  int64_t layer_halves;  // halves of one layer copy: chunks * chunk_halves
  int64_t gpr;           // groups per row
  int64_t rows;          // R
};

__host__ __device__ inline XLayout x_layout(int64_t batch, int64_t in, int g) {
  XLayout xl;
  xl.rows = batch < 64 ? batch : 64;
  xl.chunk_halves = (in + kStageK - 1) / kStageK * xl.rows * kStageK;
  xl.layer_halves = (batch + 63) / 64 * xl.chunk_halves;
  xl.gpr = in / g;
  return xl;
}

__device__ inline int64_t x16_index(const XLayout& xl, int layer, int64_t row, int64_t k) {
  return int64_t(layer) * xl.layer_halves + (row >> 6) * xl.chunk_halves +
         ((k >> 8) * xl.rows + (row & 63)) * kStageK + (k & (kStageK - 1));
}

template <int E, typename InT, bool ROT>
__global__ __launch_bounds__(256) void xprep_kernel(const InT* __restrict__ x, int64_t ngroups,
                                                    XSeeds seeds, XLayout xl, float rscale,
                                                    _Float16* __restrict__ x16,
                                                    float* __restrict__ xe) {
  const int lane = int(threadIdx.x) & 63;
  const int64_t wave0 = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  const int64_t nwaves = int64_t(gridDim.x) * 4;
  constexpr int g = 64 * E;
  // every argument in one round trip (the loop bound would otherwise be read
  // first and the rest after it)
  HIGGS_READ_NOW("s"(x), "s"(ngroups), "s"(seeds.s[0]), "s"(seeds.s[1]), "s"(seeds.s[2]),
                 "s"(seeds.s[3]), "s"(seeds.nl), "s"(xl.chunk_halves), "s"(xl.layer_halves),
                 "s"(xl.gpr), "s"(xl.rows), "s"(rscale), "s"(x16), "s"(xe), "s"(gridDim.x));
  uint64_t neg = 0;
  int neg_layer = -1;  // layer whose signs `neg` holds (uniform)
  for (int64_t item = wave0; item < int64_t(seeds.nl) * ngroups; item += nwaves) {
    const int layer = int(item / ngroups);
    const int64_t grp = item - int64_t(layer) * ngroups;
    if (ROT && layer != neg_layer) {
      uint64_t seed = seeds.s[0];
#pragma unroll
      for (int l = 1; l < kMaxGroup; ++l)
        if (layer == l) seed = seeds.s[l];
      neg = 0;
#pragma unroll
      for (int i = 0; i < E; ++i)
        neg |= uint64_t(rht_sign_negative(seed, uint32_t(lane * E + i))) << i;
      neg_layer = layer;
    }
    const int64_t base = grp * g + int64_t(lane) * E;
    float v[E];
    if constexpr (sizeof(InT) == 4 && E % 4 == 0) {
      const u32x4* p = reinterpret_cast<const u32x4*>(x + base);
#pragma unroll
      for (int q = 0; q < E / 4; ++q) {
        const u32x4 u = p[q];
        v[4 * q] = __uint_as_float(u.x);
        v[4 * q + 1] = __uint_as_float(u.y);
        v[4 * q + 2] = __uint_as_float(u.z);
        v[4 * q + 3] = __uint_as_float(u.w);
      }
    } else if constexpr (sizeof(InT) == 2 && E % 8 == 0) {
      const u32x4* p = reinterpret_cast<const u32x4*>(x + base);
#pragma unroll
      for (int q = 0; q < E / 8; ++q) {
        const u32x4 u = p[q];
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          v[8 * q + 2 * k] = __uint_as_float(w[k] << 16);
          v[8 * q + 2 * k + 1] = __uint_as_float(w[k] & 0xffff0000u);
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < E; ++i) {
        if constexpr (sizeof(InT) == 4)
          v[i] = float(x[base + i]);
        else
          v[i] = __uint_as_float(uint32_t(reinterpret_cast<const uint16_t*>(x)[base + i]) << 16);
      }
    }
    if (ROT) {
#pragma unroll
      for (int i = 0; i < E; ++i)
        if ((neg >> i) & 1) v[i] = -v[i];
      fwht_wave<E>(v, lane, g);
#pragma unroll
      for (int i = 0; i < E; ++i) v[i] *= rscale;
    }
    float m = 0.f;
#pragma unroll
    for (int i = 0; i < E; ++i) m = fmaxf(m, fabsf(v[i]));
    m = wave_max(m, lane);
    int e = m > 0.f ? ilogbf(m) - 14 : 0;
    e = e < -126 ? -126 : (e > 127 ? 127 : e);
    _Float16* dst = x16 + x16_index(xl, layer, grp / xl.gpr,
                                    (grp % xl.gpr) * g + int64_t(lane) * E);
    if constexpr (E % 8 == 0) {
#pragma unroll
      for (int q = 0; q < E / 8; ++q) {
        u32x4 w;
        w.x = pack_h2(ldexpf(v[8 * q], -e), ldexpf(v[8 * q + 1], -e));
        w.y = pack_h2(ldexpf(v[8 * q + 2], -e), ldexpf(v[8 * q + 3], -e));
        w.z = pack_h2(ldexpf(v[8 * q + 4], -e), ldexpf(v[8 * q + 5], -e));
        w.w = pack_h2(ldexpf(v[8 * q + 6], -e), ldexpf(v[8 * q + 7], -e));
        reinterpret_cast<u32x4*>(dst)[q] = w;
      }
    } else {
#pragma unroll
      for (int i = 0; i < E; ++i) dst[i] = static_cast<_Float16>(ldexpf(v[i], -e));
    }
    if (lane == 0) xe[item] = ldexpf(1.0f, e);
  }
}

// The same conversion for g >= 256 with one group per block: thread t of the
// 4 waves holds elements [tE, (t + 1)E) (g = 256 E), so each wave's serial
// chain is a quarter of the one-wave version's. Butterflies over element bits
// below log2(E) run in the lane, the next six across lanes, the top two
// (wave bits) through LDS; the stages run in the same order and each is the
// same (a + b, a - b), so the result is bit-identical to the one-wave
// version and to the separate rotation kernel.
template <int E, typename InT, bool ROT>
__global__ __launch_bounds__(256) void xprep4_kernel(const InT* __restrict__ x, int64_t ngroups,
                                                     XSeeds seeds, XLayout xl, float rscale,
                                                     _Float16* __restrict__ x16,
                                                     float* __restrict__ xe) {
  constexpr int g = 256 * E;
  __shared__ float s_v[2][256 * E];
  __shared__ float s_m[4];
  const int tid = int(threadIdx.x);
  const int lane = tid & 63;
  const int wave = tid >> 6;
  // every argument in one round trip (the loop bound would otherwise be read
  // first and the rest after it)
  HIGGS_READ_NOW("s"(x), "s"(ngroups), "s"(seeds.s[0]), "s"(seeds.s[1]), "s"(seeds.s[2]),
                 "s"(seeds.s[3]), "s"(seeds.nl), "s"(xl.chunk_halves), "s"(xl.layer_halves),
                 "s"(xl.gpr), "s"(xl.rows), "s"(rscale), "s"(x16), "s"(xe), "s"(gridDim.x));
  for (int64_t item = blockIdx.x; item < int64_t(seeds.nl) * ngroups; item += gridDim.x) {
    const int layer = int(item / ngroups);
    const int64_t grp = item - int64_t(layer) * ngroups;
    const int64_t base = grp * g + int64_t(tid) * E;
    float v[E];
    if constexpr (sizeof(InT) == 4 && E % 4 == 0) {
      const u32x4* p = reinterpret_cast<const u32x4*>(x + base);
#pragma unroll
      for (int q = 0; q < E / 4; ++q) {
        const u32x4 u = p[q];
        v[4 * q] = __uint_as_float(u.x);
        v[4 * q + 1] = __uint_as_float(u.y);
        v[4 * q + 2] = __uint_as_float(u.z);
        v[4 * q + 3] = __uint_as_float(u.w);
      }
    } else if constexpr (sizeof(InT) == 2 && E % 8 == 0) {
      const u32x4* p = reinterpret_cast<const u32x4*>(x + base);
#pragma unroll
      for (int q = 0; q < E / 8; ++q) {
        const u32x4 u = p[q];
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          v[8 * q + 2 * k] = __uint_as_float(w[k] << 16);
          v[8 * q + 2 * k + 1] = __uint_as_float(w[k] & 0xffff0000u);
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < E; ++i) {
        if constexpr (sizeof(InT) == 4)
          v[i] = float(x[base + i]);
        else
          v[i] = __uint_as_float(uint32_t(reinterpret_cast<const uint16_t*>(x)[base + i]) << 16);
      }
    }
    if (ROT) {
      uint64_t seed = seeds.s[0];
#pragma unroll
      for (int l = 1; l < kMaxGroup; ++l)
        if (layer == l) seed = seeds.s[l];
#pragma unroll
      for (int i = 0; i < E; ++i)
        if (rht_sign_negative(seed, uint32_t(tid * E + i))) v[i] = -v[i];
      fwht_in_lane<E>(v);
      fwht_cross_lane<E>(v, lane, 64 * E);
      // wave bits 0 and 1: the lower wave of a pair keeps a + b, the upper
      // one a - b (a the lower wave's value)
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        const int bit = 1 << st;
        float* buf = s_v[st];
#pragma unroll
        for (int i = 0; i < E; ++i) buf[tid * E + i] = v[i];
        __syncthreads();
        const float* o = buf + (tid ^ (64 * bit)) * E;
#pragma unroll
        for (int i = 0; i < E; ++i) v[i] = (wave & bit) ? o[i] - v[i] : v[i] + o[i];
      }
#pragma unroll
      for (int i = 0; i < E; ++i) v[i] *= rscale;
    }
    float m = 0.f;
#pragma unroll
    for (int i = 0; i < E; ++i) m = fmaxf(m, fabsf(v[i]));
    m = wave_max(m, lane);
    if (lane == 0) s_m[wave] = m;
    __syncthreads();
    m = fmaxf(fmaxf(s_m[0], s_m[1]), fmaxf(s_m[2], s_m[3]));
    int e = m > 0.f ? ilogbf(m) - 14 : 0;
    e = e < -126 ? -126 : (e > 127 ? 127 : e);
    _Float16* dst = x16 + x16_index(xl, layer, grp / xl.gpr,
                                    (grp % xl.gpr) * g + int64_t(tid) * E);
    if constexpr (E % 8 == 0) {
#pragma unroll
      for (int q = 0; q < E / 8; ++q) {
        u32x4 w;
        w.x = pack_h2(ldexpf(v[8 * q], -e), ldexpf(v[8 * q + 1], -e));
        w.y = pack_h2(ldexpf(v[8 * q + 2], -e), ldexpf(v[8 * q + 3], -e));
        w.z = pack_h2(ldexpf(v[8 * q + 4], -e), ldexpf(v[8 * q + 5], -e));
        w.w = pack_h2(ldexpf(v[8 * q + 6], -e), ldexpf(v[8 * q + 7], -e));
        reinterpret_cast<u32x4*>(dst)[q] = w;
      }
    } else {
#pragma unroll
      for (int i = 0; i < E; ++i) dst[i] = static_cast<_Float16>(ldexpf(v[i], -e));
    }
    if (tid == 0) xe[item] = ldexpf(1.0f, e);
    __syncthreads();  // s_v and s_m are reused by the next item
  }
}

// ---------------------------------------------------------------------------
// The product over one chunk of <= 64 batch rows.
// ---------------------------------------------------------------------------
// One launch covers nl layers (1..kMaxGroup) that read the same activations:
// layer l owns the blocks [blk0[l], blk0[l + 1]) of the 1-D grid, one per
// (row tile, K-split), consecutive blocks taking consecutive splits of a row
// tile: blocks are dealt to the XCDs round-robin in that order, so an XCD
// holds blocks of a few splits only and reads only their activations (with
// 8 or more splits, each split's activations are fetched by one XCD, where a
// tile-major order had all 8 XCDs fetch all of them).
struct QG {
  const _Float16* x16;  // this chunk's stage-major fp16 rows (layer l: + l * x16_stride)
  const float* xe;      // [nb][gpr], powers of two (layer l: + l * xe_stride)
  int64_t x16_stride, xe_stride;
  const float* grid;
  int nb, xrows, pair_table, log2g, in, gpr;  // xrows: R of the fp16 layout
  int nl;
  int kps[kMaxGroup];      // layer l: weights of K per split (a multiple of kStageK)
  int splits[kMaxGroup];   // layer l: K-splits
  const uint8_t* codes[kMaxGroup];
  const uint16_t* scales[kMaxGroup];
  float* dst[kMaxGroup];   // layer l: [splits][nb][out[l]]
  int out[kMaxGroup];
  int blk0[kMaxGroup];
};

// BITS: code bits per pair of weights (8, 6, 10, or 16 for scalar 8-bit
// codes). NB: 32-column batch tiles (1 or 2), or 0 for one 16-column tile
// (at most 16 batch rows, g >= 128) on v_mfma_f32_16x16x32_f16: there a
// lane holds one 32-weight run of each of two rows (its 16-row half's row
// lane % 16 and the one 16 below), run lane / 16 of every 128-weight
// super-block, so that the four lanes that supply one A row hold that row;
// each step of 32 weights feeds two 16x16x32 products, lane group q taking
// weights 32q + 8s .. + 7 of the super-block for A and B alike. FOLD:
// K-blocks per fold (1 or 2: min(g / 64, kStageKB) for g < 256, so a fold
// never spans two groups), or 4: g >= 256, products accumulate in the matrix
// registers over every stage of a scale group and are folded once per group.
// KG: K-groups of 4 waves per block (1 or 2). With 2, the block's 8 waves
// form two groups over the same 128 rows: group q takes stages q, q + 2,
// q + 4, ... of the block's K-range with its own activation staging buffer,
// so each SIMD runs two waves (the second hides the first's latency), and
// the two groups' sums are added in LDS at the end (group 0's + group 1's:
// a fixed order).
template <int BITS, int NB, int FOLD, int KG>
__global__ __launch_bounds__(kThreads * KG) void qgemm_kernel(const QG a) {
  using F = GFmt<BITS>;
  constexpr int kW = F::kWords;
  constexpr int kCopies = 1 << F::kRL;
  constexpr int kEntries = BITS == 16 ? 256 : 1 << BITS;
  constexpr int kEntryU4 = (1 << F::kStride) / 16;  // 16-byte words per table entry slot
  constexpr int kLutU4 = kEntries * kEntryU4;
  constexpr bool kCT = F::kCT;
  constexpr bool k16 = NB == 0;
  static_assert(!k16 || FOLD >= 2, "the 16-column tile folds per 128-weight super-block at least");
  static_assert(KG == 1 || KG == 2, "one or two K-groups");
  constexpr int kBlockThreads = kThreads * KG;
  constexpr bool kGroupFold = FOLD == 4;         // fold once per scale group
  constexpr int kBatch = k16 ? 16 : 32 * NB;
  constexpr int kNBT = k16 ? 1 : NB;             // accumulator tiles per wave
  constexpr int kTPR = kThreads / kBatch;        // staging threads per activation row (per group)
  constexpr int kVec = kStageK / 8 / kTPR;       // 16-byte vectors per staging thread
  constexpr int kFolds = kStageKB / FOLD;        // folds per stage (1 with group folds)
  constexpr int kXWords = kBatch * kXRow / 8;    // u32x4 of one group's staged stage
  // Code transposition rows (kCT): 32 per wave, one per weight row, each the
  // row's codes of one stage (32 kW bytes in eight 16-byte chunk slots). For
  // 8-bit codes they are the high halves of the table's 256-byte entry slots
  // (the table's 32 copies fill the low halves), else an area after the table.
  constexpr uint32_t kTrStride = BITS == 8 ? 256u : 128u;
  constexpr int kTrU4 = (kCT && BITS != 8) ? KG * kWaves * 32 * 128 / 16 : 0;
  static_assert(!kCT || BITS != 8 || KG * kWaves * 32 <= kEntries, "rows fit the table's slots");
  static_assert(!kCT || kW <= 4, "a chunk fits a 16-byte slot");
  // one LDS buffer: the table at address 0 (so a code's table address is the
  // v_perm result itself, with no base to add), the staged activations after
  __shared__ u32x4 s_mem[kLutU4 + kTrU4 + KG * kXWords];
  u32x4* const s_lut4 = s_mem;
  u32x4* const s_x4 = s_mem + kLutU4 + kTrU4;
  const uint32_t* s_lut = reinterpret_cast<const uint32_t*>(s_lut4);
  char* const s_bytes = reinterpret_cast<char*>(s_mem);

  const int tid = int(threadIdx.x);
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kgrp = wave >> 2;  // K-group
  const int rw = wave & 3;     // row wave inside the block's 128 rows
  const int gt = tid & (kThreads - 1);  // thread index inside the K-group
  const _Float16* s_x = reinterpret_cast<const _Float16*>(s_x4 + kgrp * kXWords);
  // the arguments, all requested in one round trip; the block's layer is then
  // picked by selects (an indexed read of the arguments would be a second
  // round trip)
  const uint8_t* codes_l[kMaxGroup];
  const uint16_t* scales_l[kMaxGroup];
  float* dst_l[kMaxGroup];
  int out_l[kMaxGroup], blk0_l[kMaxGroup], kps_l[kMaxGroup], splits_l[kMaxGroup];
#pragma unroll
  for (int l = 0; l < kMaxGroup; ++l) {
    codes_l[l] = a.codes[l];
    scales_l[l] = a.scales[l];
    dst_l[l] = a.dst[l];
    out_l[l] = a.out[l];
    blk0_l[l] = a.blk0[l];
    kps_l[l] = a.kps[l];
    splits_l[l] = a.splits[l];
  }
  const int nl = a.nl;
  static_assert(kMaxGroup == 4, "the read below names four layers");
  HIGGS_READ_NOW("s"(a.x16), "s"(a.xe), "s"(a.x16_stride), "s"(a.xe_stride), "s"(a.grid),
                 "s"(a.nb), "s"(a.xrows), "s"(a.pair_table), "s"(a.log2g), "s"(a.in), "s"(a.gpr),
                 "s"(nl), "s"(codes_l[0]), "s"(codes_l[1]), "s"(codes_l[2]), "s"(codes_l[3]),
                 "s"(scales_l[0]), "s"(scales_l[1]), "s"(scales_l[2]), "s"(scales_l[3]),
                 "s"(dst_l[0]), "s"(dst_l[1]), "s"(dst_l[2]), "s"(dst_l[3]), "s"(out_l[0]),
                 "s"(out_l[1]), "s"(out_l[2]), "s"(out_l[3]), "s"(blk0_l[1]), "s"(blk0_l[2]),
                 "s"(blk0_l[3]), "s"(kps_l[0]), "s"(kps_l[1]), "s"(kps_l[2]), "s"(kps_l[3]),
                 "s"(splits_l[0]), "s"(splits_l[1]), "s"(splits_l[2]), "s"(splits_l[3]));
  // held in registers from here: the compiler would otherwise read these
  // again where registers are short, each read a round trip
  int nbr = a.nb, xrows = a.xrows, log2g = a.log2g, gpr = a.gpr, in = a.in;
  int pair_table = a.pair_table;
  HIGGS_HOLD("+s"(nbr), "+s"(xrows), "+s"(log2g), "+s"(gpr), "+s"(in), "+s"(pair_table));
  int L = 0;
#pragma unroll
  for (int l = 1; l < kMaxGroup; ++l)
    if (l < nl && int(blockIdx.x) >= blk0_l[l]) L = l;
  const uint8_t* codes = codes_l[0];
  const uint16_t* scales = scales_l[0];
  float* dst0 = dst_l[0];
  int out = out_l[0], blk0 = 0, kps = kps_l[0], splits = splits_l[0];
#pragma unroll
  for (int l = 1; l < kMaxGroup; ++l)
    if (L == l) {
      codes = codes_l[l];
      scales = scales_l[l];
      dst0 = dst_l[l];
      out = out_l[l];
      blk0 = blk0_l[l];
      kps = kps_l[l];
      splits = splits_l[l];
    }
  const _Float16* x16 = a.x16 + int64_t(L) * a.x16_stride;
  const float* xe = a.xe + int64_t(L) * a.xe_stride;
  const int wl = int(blockIdx.x) - blk0;  // the block's index in its layer
  const int split = wl % splits;
  const int row0 = (wl / splits) * kTileRows + rw * 32;
  const int kbeg = split * kps;
  const int kend = min(in, kbeg + kps);
  const int nkb = (kend - kbeg) >> 6;                  // K-blocks of this block
  const int nst = (nkb + kStageKB - 1) / kStageKB;     // stages of this block
  const int nit = (nst + KG - 1) / KG;                 // stages of each K-group
  // The block takes its stages in a rotated order, starting at stage rot:
  // blocks of one layer run side by side and would otherwise read the same
  // K-range of codes at the same time; the rotation spreads those reads
  // over the memory channels. It depends on the row tile only (the tile's
  // index inside the layer), so a layer's results are the same in a grouped
  // launch and alone. Stage of this K-group at its iteration `it` (>= nst
  // past the block's range: zero activations, so it adds nothing):
  const int tile = wl / splits;
  const int rot = (tile / 8 + 3 * (tile % 8)) % nst;
  auto stage_of = [&](int it) {
    const int c = it * KG + kgrp;
    if (c >= nst) return c;
    return c + rot >= nst ? c + rot - nst : c + rot;
  };

  // ---- 1. grid points of this thread's table entries: thread t writes the
  //      16-byte stores [t kSPT, (t + 1) kSPT) of the table (numbered over the
  //      copies only), which hold the copies of kEPT consecutive entries (or
  //      part of one entry's) ----
  constexpr int kStoresPerEntry = kCopies / 4;
  constexpr int kSPT = kEntries * kStoresPerEntry / kBlockThreads;
  constexpr int kEPT = kSPT >= kStoresPerEntry ? kSPT / kStoresPerEntry : 1;
  static_assert(kSPT * kBlockThreads == kEntries * kStoresPerEntry, "table stores split evenly");
  const int e0 = tid * kSPT / kStoresPerEntry;
  float gx[kEPT], gy[kEPT];
#pragma unroll
  for (int j = 0; j < kEPT; ++j) {
    const int e = e0 + j;
    if constexpr (BITS == 16) {  // one value per entry, in the low half
      gx[j] = a.grid[e];
      gy[j] = 0.f;
    } else {
      gx[j] = pair_table ? a.grid[e & 15] : a.grid[2 * e];
      gy[j] = pair_table ? a.grid[e >> 4] : a.grid[2 * e + 1];
    }
  }

  // ---- 2. activations of the group's first stage ----
  // A stage of the chunk is one contiguous block (stage-major layout): load v
  // of the group's threads reads its bytes [4096 v, 4096 (v + 1)), 16 per
  // thread (one 1 KiB read per wave); thread gt's piece v is row
  // 8 v + gt / 32, halves [8 (gt % 32), + 8) of the stage.
  const int xk = (gt & 31) * 8;
  const int nstg = (in + kStageK - 1) / kStageK;  // stages of a row
  const __amdgpu_buffer_rsrc_t xrs = rsrc(x16, uint32_t(nstg) * uint32_t(xrows) * kStageK * 2u);
  u32x4 xv[kVec];
  // Weights at or past the end of the block's K-range read zero: the partial
  // last stage of a row, the stages past the block's range that a K-group
  // runs to keep step with the other, and the stage prefetched after a
  // group's last one; so do batch rows past nb.
  auto load_x = [&](int it) {
    const int c = stage_of(it);
    const int k = kbeg + c * kStageK + xk;
    const uint32_t sbase = uint32_t((kbeg >> 8) + c) * uint32_t(xrows) * kStageK;
#pragma unroll
    for (int v = 0; v < kVec; ++v) {
      const int row = 8 * v + (gt >> 5);
      const uint32_t off = (row < nbr && k < kend && c < nst)
                               ? (sbase + uint32_t(row) * kStageK + uint32_t(xk)) * 2u
                               : kOffNone;
      xv[v] = as_u32x4(__builtin_amdgcn_raw_buffer_load_b128(xrs, int(off), 0, 0));
    }
  };
  load_x(0);

  // ---- 3. codes ring ----
  const int ahalf = lane >> 5;
  constexpr uint32_t kKBBytes = 8 * kW;  // bytes of one row's K-block (32 codes)
  const uint32_t row_bytes = uint32_t(in >> 6) * kKBBytes;
  const __amdgpu_buffer_rsrc_t crs = rsrc(codes, uint32_t(out) * row_bytes);
  // kCT: slot j = piece j % 4 of the group's stage j / 4: rows 8 (j % 4) ..
  // + 7 of the wave's 32, lane l reading chunk l % 8 (4 kW bytes: half l % 2
  // of K-block (l % 8) / 2) of row l / 8 of the piece, so that eight lanes
  // read a row's whole stage (a 128-byte line for 8-bit codes): streamed
  // this way a layer's codes arrive at close to twice the rate of pieces of
  // 32 rows x 32 bytes (one row's two chunks of a K-block, the matrix
  // operand's own layout). At the stage's start the wave puts them through
  // its transposition rows into that layout (cod below).
  // Otherwise (10-bit and scalar 8-bit codes) the operand layout is read
  // directly: 32-column tiles: slot j = the group's K-block j, row lane %
  // 32, half lane / 32; 16-column tile: slot j = row (j % 2) of the lane's
  // two, run lane / 16 of the group's super-block j / 2 (g >= 128 and K a
  // multiple of g, so the block holds whole super-blocks).
  uint32_t cbase[kCT ? 4 : 2];
  if constexpr (kCT) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      cbase[i] = uint32_t(min(row0 + 8 * i + (lane >> 3), out - 1)) * row_bytes +
                 uint32_t(kbeg >> 6) * kKBBytes + 4u * kW * uint32_t(lane & 1);
  } else if constexpr (k16) {
#pragma unroll
    for (int m = 0; m < 2; ++m)
      cbase[m] = uint32_t(min(row0 + 16 * m + (lane & 15), out - 1)) * row_bytes +
                 uint32_t(kbeg >> 6) * kKBBytes + 4u * kW * uint32_t(lane >> 4);
  } else {
    cbase[0] = uint32_t(min(row0 + (lane & 31), out - 1)) * row_bytes +
               uint32_t(kbeg >> 6) * kKBBytes + 4u * kW * uint32_t(ahalf);
    cbase[1] = cbase[0];
  }
  uint32_t ring[kRing][kW];
  // the current stage's codes in the operand layout (kCT): 32-column tiles:
  // cod[kb] = K-block kb, row lane % 32, half lane / 32; 16-column tile:
  // cod[2 sb + m] = row m of the lane's two, run lane / 16 of super-block sb
  uint32_t cod[kStageKB][kW];
  // transposition addresses: chunk c of row r sits in slot c ^ (r % 8), so
  // that the eight lanes of a 128-byte LDS access touch distinct banks both
  // when a piece is written (one row, eight chunks) and when the operand
  // layout is read (eight rows, one chunk)
  const uint32_t tr0 =
      (BITS == 8 ? 128u : uint32_t(kLutU4) * 16u) + uint32_t(wave) * 32u * kTrStride;
  const uint32_t tr_put = tr0 + uint32_t(lane >> 3) * kTrStride +
                          (uint32_t((lane & 7) ^ (lane >> 3)) << 4);  // + piece * 8 rows
  const uint32_t tr_get = tr0 + uint32_t(k16 ? (lane & 15) : (lane & 31)) * kTrStride;
  // K-blocks (super-blocks) past the block's range re-read its last one
  // (never used, or multiplied by zero activations)
  auto fetch = [&](int j, uint32_t (&d)[kW]) {
    if constexpr (kCT) {
      const int c = stage_of(j / kStageKB);
      const int kb = min(kStageKB * c + ((lane & 7) >> 1), nkb - 1);
      load_codes<BITS>(crs, cbase[j % kStageKB] + kKBBytes * uint32_t(kb), d);
    } else if constexpr (k16) {
      const int sl = j >> 1;  // the group's super-block
      const int sb = 2 * stage_of(sl >> 1) + (sl & 1);
      load_codes<BITS>(crs, cbase[j & 1] + 2u * kKBBytes * uint32_t(min(sb, nkb / 2 - 1)), d);
    } else {
      const int kb = kStageKB * stage_of(j / kStageKB) + (j % kStageKB);
      load_codes<BITS>(crs, cbase[0] + kKBBytes * uint32_t(min(kb, nkb - 1)), d);
    }
  };
  // With two batch tiles the prologue requests only stage 0's codes and
  // stage 0 requests stage 1's with its other loads: a smaller start-up burst
  // when every block starts at once. With one tile the whole ring is filled
  // here (fewer stages per block, so the early second stage pays off).
  constexpr int kPrologueSlots = NB == 2 ? kStageKB : kRing;
#pragma unroll
  for (int t = 0; t < kPrologueSlots; ++t) fetch(t, ring[t]);

  // ---- 4. scales of each fold of a stage: lane l -> row row0 + l % 32 (group
  //      scale, fp16 bits) and batch row 32t + l % 32 (activation exponent) ----
  const __amdgpu_buffer_rsrc_t srs = rsrc(scales, uint32_t(out) * uint32_t(gpr) * 2u);
  const __amdgpu_buffer_rsrc_t ers = rsrc(xe, uint32_t(nbr) * uint32_t(gpr) * 4u);
  const uint32_t srow = uint32_t(min(row0 + (lane & 31), out - 1));
  uint32_t sc[kFolds];
  float xs[kNBT][kFolds];
  // groups past the row's end (a partial last stage, or a stage past the
  // block's range) re-read the row's last group: finite, and multiplied by
  // zero or never used
  auto load_scales = [&](int it) {
#pragma unroll
    for (int f = 0; f < kFolds; ++f) {
      const int grp = min((kbeg + stage_of(it) * kStageK + f * FOLD * 64) >> log2g, gpr - 1);
      sc[f] = uint32_t(uint16_t(__builtin_amdgcn_raw_buffer_load_b16(
          srs, int((srow * uint32_t(gpr) + uint32_t(grp)) * 2u), 0, 0)));
#pragma unroll
      for (int t = 0; t < kNBT; ++t) {
        // rows past nb read zero (never stored)
        const int b = k16 ? (lane & 15) : 32 * t + (lane & 31);
        xs[t][f] = __builtin_bit_cast(
            float, __builtin_amdgcn_raw_buffer_load_b32(
                       ers, int(b < nbr ? (uint32_t(b) * uint32_t(gpr) + uint32_t(grp)) * 4u
                                         : kOffNone), 0, 0));
      }
    }
  };
  load_scales(0);

  // ---- the table: kCopies copies of each entry ----
#pragma unroll
  for (int k = 0; k < kSPT; ++k) {
    const int n = tid * kSPT + k;
    const int j = n / kStoresPerEntry - e0;  // compile-time after unrolling
    const uint32_t v = pack_h2(gx[j], gy[j]);
    s_lut4[(n / kStoresPerEntry) * kEntryU4 + n % kStoresPerEntry] = u32x4{v, v, v, v};
  }

  // this lane's table copy: with 8-bit codes (and scalar ones) the entry
  // stride is 256 bytes, so one v_perm forms code * 256 + copy * 4
  const uint32_t copy_off = uint32_t(lane & (kCopies - 1)) << 2;
  f16x_acc total[kNBT];
#pragma unroll
  for (int t = 0; t < kNBT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) total[t][r] = 0.f;
  // matrix accumulators; with group folds they carry over the stages of a
  // scale group
  f16x_acc acc[kNBT];
  f32x4 acc16[2];
#pragma unroll
  for (int t = 0; t < kNBT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;
#pragma unroll
  for (int m = 0; m < 2; ++m) acc16[m] = f32x4{0.f, 0.f, 0.f, 0.f};

  // One stage of this K-group: K-blocks 4c .. 4c+3 of c = stage_of(it),
  // codes from ring slots 4H .. 4H+3.
  auto stage = [&](int it, auto H, auto FIRST) {
    constexpr int kSlot0 = decltype(H)::value * kStageKB;
    const int c = stage_of(it);
    // with group folds: fold after this stage when the group's next stage
    // lies in another scale group or past the block's range (uniform)
    const int cn = stage_of(it + 1);  // the group's next stage
    const bool fold_now = cn >= nst ||
                          ((kbeg + cn * kStageK) >> log2g) != ((kbeg + c * kStageK) >> log2g);
    __syncthreads();  // previous stage consumed (first time: table written)
    {
      u32x4* dst = s_x4 + kgrp * kXWords + ((gt >> 5) * kXRow + xk) / 8;
#pragma unroll
      for (int v = 0; v < kVec; ++v) dst[v * (8 * kXRow / 8)] = xv[v];
    }
    uint32_t sc_c[kFolds];
    float xs_c[kNBT][kFolds];
#pragma unroll
    for (int f = 0; f < kFolds; ++f) {
      sc_c[f] = sc[f];
#pragma unroll
      for (int t = 0; t < kNBT; ++t) xs_c[t][f] = xs[t][f];
    }
    __syncthreads();
    if constexpr (kCT) {
      // this stage's codes through the wave's transposition rows into the
      // operand layout (the rows are the wave's own: no block barrier)
#pragma unroll
      for (int i = 0; i < kStageKB; ++i)
        lds_put<kW>(s_bytes, tr_put + uint32_t(i) * 8u * kTrStride, ring[kSlot0 + i]);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
      for (int q = 0; q < kStageKB; ++q) {
        // 32-column tiles: K-block q (chunk 2q + half); 16-column tile:
        // super-block q / 2, row q % 2 of the lane's two (chunk 4 (q / 2) +
        // lane / 16)
        const uint32_t c = k16 ? uint32_t(4 * (q >> 1) + (lane >> 4))
                               : uint32_t(2 * q + (lane >> 5));
        const uint32_t row_off = k16 ? uint32_t(q & 1) * 16u * kTrStride : 0u;
        lds_get<kW>(s_bytes, tr_get + row_off + ((c ^ uint32_t(lane & 7)) << 4), cod[q]);
      }
    }
    // issue the next stage's loads now: the scheduler would otherwise delay
    // them to the end of the stage to save registers
    load_x(it + 1);
    load_scales(it + 1);
    if constexpr (decltype(FIRST)::value && kPrologueSlots < kRing) {
#pragma unroll
      for (int t = kPrologueSlots; t < kRing; ++t) fetch(t, ring[t]);
    }
    if constexpr (kCT) {
      // the slots just transposed take the stage after next
#pragma unroll
      for (int i = 0; i < kStageKB; ++i) fetch(it * kStageKB + kRing + i, ring[kSlot0 + i]);
    }
    __builtin_amdgcn_sched_barrier(0);

    if constexpr (k16) {
      // 8 steps of 32 weights (4 per super-block), two 16x16x32 products
      // each (rows 0-15 and 16-31 of the wave), software-pipelined as below
      constexpr int kSteps = 2 * kStageKB;
      constexpr int kAhead = 2;
      struct Step16 {
        half8 a[2];
        half8 b;
      };
      auto load_step = [&](int st, Step16& o) {
        const int sb = st / 4, s = st % 4;  // super-block inside the stage, step inside it
#pragma unroll
        for (int m = 0; m < 2; ++m) {
          // A: pairs 4s .. 4s+3 of the run -> 8 halves (weights 32q + 8s .. + 7)
          uint32_t a32[4];
          const uint32_t(&cw)[kW] = kCT ? cod[2 * sb + m] : ring[kSlot0 + 2 * sb + m];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if constexpr (BITS == 16) {
              const int cc = 4 * s + q;
              const uint32_t o0 = lut_off_byte<kW>(cw, 2 * cc, copy_off);
              const uint32_t o1 = lut_off_byte<kW>(cw, 2 * cc + 1, copy_off);
              const char* t = reinterpret_cast<const char*>(s_lut);
              a32[q] = uint32_t(*reinterpret_cast<const uint16_t*>(t + o0)) |
                       (uint32_t(*reinterpret_cast<const uint16_t*>(t + o1)) << 16);
            } else {
              const uint32_t off = lut_off<BITS>(cw, 4 * s + q, copy_off);
              a32[q] =
                  *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(s_lut) + off);
            }
          }
          o.a[m] = __builtin_bit_cast(half8, u32x4{a32[0], a32[1], a32[2], a32[3]});
        }
        // B: batch row lane % 16, the same 8 weights
        o.b = *reinterpret_cast<const half8*>(s_x + (lane & 15) * kXRow + sb * 128 +
                                              32 * (lane >> 4) + 8 * s);
      };
      Step16 ops[kSteps];
#pragma unroll
      for (int st = 0; st < kAhead; ++st) load_step(st, ops[st]);
      // fold: register v of product m holds row 16m + 4 (lane / 16) + v
      // of the wave's 32, column lane % 16; lane r holds row r's scale
      auto fold16 = [&](int fo) {
        const float sf = float(__builtin_bit_cast(_Float16, uint16_t(sc_c[fo])));
        const int sfi = __builtin_bit_cast(int, sf);
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int r = 16 * m + 4 * (lane >> 4) + v;
            const float sr = __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(r << 2, sfi));
            total[0][4 * m + v] = fmaf(acc16[m][v], sr * xs_c[0][fo], total[0][4 * m + v]);
          }
#pragma unroll
        for (int m = 0; m < 2; ++m) acc16[m] = f32x4{0.f, 0.f, 0.f, 0.f};
      };
#pragma unroll
      for (int st = 0; st < kSteps; ++st) {
        if (st + kAhead < kSteps) load_step(st + kAhead, ops[st + kAhead]);
        // the last step reading a super-block's codes is issued: refill its
        // two ring slots
        if (!kCT && st + kAhead < kSteps && (st + kAhead) % 4 == 3) {
          const int sb = (st + kAhead) / 4;
          fetch(it * kStageKB + 2 * sb + kRing, ring[kSlot0 + 2 * sb]);
          fetch(it * kStageKB + 2 * sb + 1 + kRing, ring[kSlot0 + 2 * sb + 1]);
        }
#pragma unroll
        for (int m = 0; m < 2; ++m)
          acc16[m] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ops[st].a[m], ops[st].b, acc16[m], 0,
                                                            0, 0);
        if (st % 4 == 3) __builtin_amdgcn_sched_barrier(0);
        if constexpr (!kGroupFold) {
          if (st % (2 * FOLD) == 2 * FOLD - 1) fold16(st / (2 * FOLD));
        }
      }
      if constexpr (kGroupFold) {
        if (fold_now) fold16(0);
      }
      return;
    }

    // The stage's 16 MFMA steps (4 per K-block), software-pipelined: the
    // LDS operands of step st + kAhead are read while step st multiplies.
    constexpr int kSteps = 4 * kStageKB;
    constexpr int kAhead = 2;
    struct Step {
      half8 a;
      half8 b[kNBT];
    };
    auto load_step = [&](int st, Step& o) {
      const int kb = st / 4, s = st % 4;  // K-block inside the stage, step inside it
      // A: codes 4s .. 4s+3 -> 8 halves (weights 32h + 8s .. + 7)
      uint32_t a32[4];
      const uint32_t(&cw)[kW] = kCT ? cod[kb] : ring[kSlot0 + kb];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if constexpr (BITS == 16) {  // weights 2c, 2c + 1: bytes 2c, 2c + 1
          const int cc = 4 * s + q;
          const uint32_t o0 = lut_off_byte<kW>(cw, 2 * cc, copy_off);
          const uint32_t o1 = lut_off_byte<kW>(cw, 2 * cc + 1, copy_off);
          const char* t = reinterpret_cast<const char*>(s_lut);
          a32[q] = uint32_t(*reinterpret_cast<const uint16_t*>(t + o0)) |
                   (uint32_t(*reinterpret_cast<const uint16_t*>(t + o1)) << 16);
        } else {
          const uint32_t off = lut_off<BITS>(cw, 4 * s + q, copy_off);
          a32[q] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(s_lut) + off);
        }
      }
      o.a = __builtin_bit_cast(half8, u32x4{a32[0], a32[1], a32[2], a32[3]});
      // B: batch row 32t + lane % 32, the same 8 weights
#pragma unroll
      for (int t = 0; t < kNBT; ++t)
        o.b[t] = *reinterpret_cast<const half8*>(s_x + (32 * t + (lane & 31)) * kXRow + kb * 64 +
                                                 32 * ahalf + 8 * s);
    };
    // fold: accumulator register r holds row 8 (r / 4) + 4 ahalf + r % 4
    // of the wave's 32, column 32t + lane % 32
    auto fold32 = [&](int fo) {
      const float sf = float(__builtin_bit_cast(_Float16, uint16_t(sc_c[fo])));
      const int sfi = __builtin_bit_cast(int, sf);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = 8 * (r / 4) + (r % 4);
        const float s0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(sfi, rl));
        const float s1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(sfi, rl + 4));
        const float sr = ahalf ? s1 : s0;
#pragma unroll
        for (int t = 0; t < kNBT; ++t) total[t][r] = fmaf(acc[t][r], sr * xs_c[t][fo], total[t][r]);
      }
#pragma unroll
      for (int t = 0; t < kNBT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;
    };
    Step ops[kSteps];
#pragma unroll
    for (int st = 0; st < kAhead; ++st) load_step(st, ops[st]);
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
      if (st + kAhead < kSteps) load_step(st + kAhead, ops[st + kAhead]);
      // the last step reading a K-block's codes is issued: refill its ring slot
      if (!kCT && st + kAhead < kSteps && (st + kAhead) % 4 == 3) {
        const int kb = (st + kAhead) / 4;
        fetch(it * kStageKB + kb + kRing, ring[kSlot0 + kb]);
      }
#pragma unroll
      for (int t = 0; t < kNBT; ++t)
        acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ops[st].a, ops[st].b[t], acc[t], 0, 0, 0);
      if (st % 4 == 3) __builtin_amdgcn_sched_barrier(0);
      if constexpr (!kGroupFold) {
        if (st % (4 * FOLD) == 4 * FOLD - 1) fold32(st / (4 * FOLD));
      }
    }
    if constexpr (kGroupFold) {
      if (fold_now) fold32(0);
    }
  };

  // Pairs of stages with no branch between them (a branch there lets the
  // compiler sink the prefetch loads of one stage down into the next), then
  // the odd last stage. Both K-groups run nit stages (the same barriers).
  // With a deferred ring fill stage 0 comes first on its own (with one tile
  // that peeled form measured slower, so the loop there starts at stage 0).
  if constexpr (kPrologueSlots < kRing) {
    stage(0, std::integral_constant<int, 0>{}, std::true_type{});
    int it = 1;
    for (; it + 1 < nit; it += 2) {
      stage(it, std::integral_constant<int, 1>{}, std::false_type{});
      stage(it + 1, std::integral_constant<int, 0>{}, std::false_type{});
    }
    if (it < nit) stage(it, std::integral_constant<int, 1>{}, std::false_type{});
  } else {
    int it = 0;
    for (; it + 1 < nit; it += 2) {
      stage(it, std::integral_constant<int, 0>{}, std::false_type{});
      stage(it + 1, std::integral_constant<int, 1>{}, std::false_type{});
    }
    if (it < nit) stage(it, std::integral_constant<int, 0>{}, std::false_type{});
  }

  // ---- store through LDS so that lanes write consecutive rows: each wave's
  //      32 rows x kBatch columns go to its slice of the activation buffers
  //      (free once every wave has left the stage loop); with two K-groups,
  //      group 0's waves add group 1's sums for the same rows ----
  constexpr int kORow = 33;  // floats per staged column (32 rows + 1: no bank conflicts)
  static_assert(KG * kWaves * kBatch * kORow * 4 <= KG * kXWords * 16, "output staging fits");
  __syncthreads();
  float* s_o = reinterpret_cast<float*>(s_x4) + (kgrp * kWaves + rw) * (kBatch * kORow);
  if constexpr (k16) {
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        s_o[(lane & 15) * kORow + 16 * m + 4 * (lane >> 4) + v] = total[0][4 * m + v];
  } else {
#pragma unroll
    for (int t = 0; t < kNBT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        s_o[(32 * t + (lane & 31)) * kORow + 8 * (r / 4) + 4 * ahalf + (r % 4)] = total[t][r];
  }
  if constexpr (KG > 1) {
    __syncthreads();
    if (kgrp != 0) return;
  } else {
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  const float* s_o1 = s_o + kWaves * (kBatch * kORow);  // group 1's sums (KG = 2)
  float* dst = dst0 + int64_t(split) * nbr * out + row0;
  const int orow = lane & 31;
#pragma unroll
  for (int i = 0; i < kBatch / 2; ++i) {
    const int b = 2 * i + ahalf;
    float v = s_o[b * kORow + orow];
    if constexpr (KG > 1) v += s_o1[b * kORow + orow];
    if (b < nbr && row0 + orow < out) dst[int64_t(b) * out + orow] = v;
  }
}

// The layers' partial products of one launch: layer l's [splits[l]][n[l]]
// at part[l], its output (n[l] floats) at y[l]; off[l] = n[0] + ... +
// n[l - 1]. A layer without a K-split has n[l] = 0 (its product wrote y), so
// index i belongs to the last layer l with off[l] <= i.
struct RG {
  const float* part[kMaxGroup];
  float* y[kMaxGroup];
  int64_t n[kMaxGroup];
  int64_t off[kMaxGroup + 1];
  int splits[kMaxGroup];
  int nl;
};

// y = sum over splits of the partial products, in split order.
__global__ __launch_bounds__(256) void qgemm_reduce(const RG r) {
  // every argument in one round trip; the layer of an index is then picked
  // by selects (an indexed read would be a second round trip)
  const float* part_l[kMaxGroup];
  float* y_l[kMaxGroup];
  int64_t n_l[kMaxGroup], off_l[kMaxGroup + 1];
  int splits_l[kMaxGroup];
#pragma unroll
  for (int l = 0; l < kMaxGroup; ++l) {
    part_l[l] = r.part[l];
    y_l[l] = r.y[l];
    n_l[l] = r.n[l];
    off_l[l] = r.off[l];
    splits_l[l] = r.splits[l];
  }
  off_l[kMaxGroup] = r.off[kMaxGroup];
  const int nl = r.nl;
  static_assert(kMaxGroup == 4, "the read below names four layers");
  HIGGS_READ_NOW("s"(part_l[0]), "s"(part_l[1]), "s"(part_l[2]), "s"(part_l[3]), "s"(y_l[0]),
                 "s"(y_l[1]), "s"(y_l[2]), "s"(y_l[3]), "s"(n_l[0]), "s"(n_l[1]), "s"(n_l[2]),
                 "s"(n_l[3]), "s"(off_l[1]), "s"(off_l[2]), "s"(off_l[3]), "s"(off_l[4]),
                 "s"(splits_l[0]), "s"(splits_l[1]), "s"(splits_l[2]), "s"(splits_l[3]),
                 "s"(nl), "s"(gridDim.x));
  int64_t total = off_l[1];
#pragma unroll
  for (int l = 2; l <= kMaxGroup; ++l)
    if (l == nl) total = off_l[l];
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < total;
       i += int64_t(gridDim.x) * 256) {
    int L = 0;
#pragma unroll
    for (int l = 1; l < kMaxGroup; ++l)
      if (l < nl && i >= off_l[l]) L = l;
    const float* part = part_l[0];
    float* y = y_l[0];
    int64_t n = n_l[0], j = i;
    int splits = splits_l[0];
#pragma unroll
    for (int l = 1; l < kMaxGroup; ++l)
      if (L == l) {
        part = part_l[l];
        y = y_l[l];
        n = n_l[l];
        j = i - off_l[l];
        splits = splits_l[l];
      }
    // loads eight splits at a time (one memory round trip for up to eight),
    // adds in split order starting from split 0's value
    float s = 0.f;
    for (int k = 0; k < splits; k += 8) {
      float v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = part[int64_t(min(k + q, splits - 1)) * n + j];
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (k + q < splits) s = k + q == 0 ? v[q] : s + v[q];
    }
    y[j] = s;
  }
}

// Throughput of a block with two K-groups relative to the 64-cycle rate of
// one matrix instruction per wave that the split model was built on
// (measured on the 8B shapes at batch 16-64: 1.0 keeps gate/up unsplit and
// splits q/k/v, o and down so that their blocks fill the chip; 1.5 left q
// and o unsplit at batch 64, 0.7 split gate/up).
constexpr double kMfmaGain = 1.0;

// K-split of a layer: stages per split and the number of splits.
struct Split {
  int64_t stages_per_split;
  int64_t splits;
};

// Chooses the K-split for a chunk of nb batch rows from a simple model of
// MI355X (256 compute units, one block of two K-groups each): the time of the busiest
// compute unit at a sustained rate of one matrix instruction per 64 cycles
// per wave, against HBM traffic of codes plus split partial sums (written,
// then read back), plus the reduction launch when there is more than one
// split. A stage of a single 32-column batch tile is priced like one of two
// tiles on layers of at most 64 row tiles: its table decode and staging take
// about as long (measured: at half the price such layers got too few splits
// and left compute units idle), while layers with more rows fill the chip
// anyway, also next to others in a grouped launch. The plan depends only on
// the shapes, so the workspace size is a function of the arguments.
Split plan_split(int64_t out, int64_t in, int64_t nb, int bits) {
  constexpr double kCUs = 256, kClock = 2.4e9, kCyclesPerMfma = 64.0 / kMfmaGain, kHbm = 6e12;
  // the reduction launch measured 4-7 us per call (launch, partial sums read)
  constexpr double kReduceLaunch = 6e-6, kRoundLatency = 1.5e-6;
  const int64_t tiles = (out + kTileRows - 1) / kTileRows;
  const int64_t stages = (in + kStageK - 1) / kStageK;
  const int64_t nbt = (nb > 32 || tiles <= 64) ? 2 : 1;
  double best_t = 1e30;
  Split best{stages, 1};
  for (int64_t s = 1; s <= stages; s *= 2) {
    const int64_t sps = (stages + s - 1) / s;
    const int64_t splits = (stages + sps - 1) / sps;
    const double blocks = double(tiles * splits);
    const double per_block = double(sps * kStageKB * 4 * nbt) * kCyclesPerMfma / kClock;
    const double t_mfma = per_block * std::ceil(blocks / kCUs);
    const double bytes =
        double(out) * double(in) * bits / 16 + (splits > 1 ? 8.0 * splits * nb * out : 0);
    const double t = std::max(t_mfma, bytes / kHbm) + (splits > 1 ? kReduceLaunch : 0) +
                     kRoundLatency * std::ceil(blocks / kCUs);
    if (t < best_t * 0.97) {  // more splits only for a clear gain
      best_t = t;
      best = Split{sps, splits};
    }
    if (sps <= 2) break;
  }
  return best;
}

int64_t align256(int64_t v) { return (v + 255) / 256 * 256; }

template <int E, typename InT, bool ROT>
hipError_t launch_xprep_e(const InT* x, int64_t ngroups, const XSeeds& seeds, const XLayout& xl,
                          float rscale, _Float16* x16, float* xe, hipStream_t stream) {
  const int64_t items = ngroups * seeds.nl;
  if constexpr (E >= 4) {
    // g >= 256: one group per block of 4 waves
    const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>(items, 65536));
    hipLaunchKernelGGL((xprep4_kernel<E / 4, InT, ROT>), dim3(unsigned(blocks)), dim3(256), 0,
                       stream, x, ngroups, seeds, xl, rscale, x16, xe);
  } else {
    const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((items + 3) / 4, 8192));
    hipLaunchKernelGGL((xprep_kernel<E, InT, ROT>), dim3(unsigned(blocks)), dim3(256), 0, stream,
                       x, ngroups, seeds, xl, rscale, x16, xe);
  }
  return hipGetLastError();
}

template <typename InT, bool ROT>
hipError_t launch_xprep(const InT* x, int64_t ngroups, int g, const XSeeds& seed,
                        const XLayout& xl, _Float16* x16, float* xe, hipStream_t stream) {
  const float rscale = float(1.0 / std::sqrt(double(g)));
  switch (g) {
#define HIGGS_XPREP(G) \
  case G:              \
    return launch_xprep_e<G / 64, InT, ROT>(x, ngroups, seed, xl, rscale, x16, xe, stream);
    HIGGS_XPREP(64)
    HIGGS_XPREP(128)
    HIGGS_XPREP(256)
    HIGGS_XPREP(512)
    HIGGS_XPREP(1024)
    HIGGS_XPREP(2048)
    HIGGS_XPREP(4096)
#undef HIGGS_XPREP
    default:
      return hipErrorInvalidValue;
  }
}

// K-groups per block: two everywhere (two waves per SIMD).
constexpr int kKGroups = 2;

template <int BITS, int NB, int FOLD>
hipError_t launch_nb(const QG& a, int64_t blocks, hipStream_t stream) {
  hipLaunchKernelGGL((qgemm_kernel<BITS, NB, FOLD, kKGroups>), dim3(unsigned(blocks)),
                     dim3(kThreads * kKGroups), 0, stream, a);
  return hipGetLastError();
}

template <int BITS, int NB>
hipError_t launch_fold(const QG& a, int g, int64_t blocks, hipStream_t stream) {
  if (g >= 256) return launch_nb<BITS, NB, 4>(a, blocks, stream);
  if (g == 128) return launch_nb<BITS, NB, 2>(a, blocks, stream);
  if constexpr (NB == 0) return hipErrorInvalidValue;  // the 16-column tile needs g >= 128
  else return launch_nb<BITS, NB, 1>(a, blocks, stream);
}

// Batch tile of a chunk of nb rows: one 16-column tile up to 16 rows (when
// g >= 128), else one or two 32-column tiles.
template <int BITS>
hipError_t launch_bits(const QG& a, int g, int64_t blocks, hipStream_t stream) {
  if (a.nb <= 16 && g >= 128) return launch_fold<BITS, 0>(a, g, blocks, stream);
  return a.nb > 32 ? launch_fold<BITS, 2>(a, g, blocks, stream)
                   : launch_fold<BITS, 1>(a, g, blocks, stream);
}

// Workspace layout of a launch over nl layers: fp16 activations
// [nx][batch][in] and exponents [nx][batch][in / g] (nx copies: one per layer
// when the layers rotate with their own seeds, else one), then each layer's
// split partial sums [splits][min(batch, 64)][out] (each 256-byte aligned).
// Each layer keeps its own split plan, so a layer's result does not depend
// on the other layers of the launch.
struct Layout {
  int64_t x16, xe, part[kMaxGroup], total;
};

Layout layout(int64_t batch, const int64_t* outs, int nl, int nx, int64_t in, int g, int bits) {
  Layout L;
  L.x16 = 0;
  L.xe = align256(nx * x_layout(batch, in, g).layer_halves * 2);
  int64_t at = L.xe + align256(nx * batch * (in / g) * 4);
  for (int l = 0; l < nl; ++l) {
    // the larger of the full 64-row chunks and the last one
    int64_t part = 0;
    for (const int64_t nb : {std::min<int64_t>(batch, 64), batch % 64}) {
      if (nb == 0) continue;
      const Split sp = plan_split(outs[l], in, nb, bits);
      if (sp.splits > 1) part = std::max(part, sp.splits * nb * outs[l] * 4);
    }
    L.part[l] = at;
    at += align256(part);
  }
  L.total = at;
  return L;
}

// Bits of code per pair of weights (the kernel's code width): the scalar
// 16-point grid's two 4-bit codes are read as one byte.
int pair_bits(int p, int n) { return p == 1 ? 2 * code_bits(p, n) : code_bits(p, n); }

}  // namespace

int64_t qgemm_workspace_bytes(int64_t batch, int64_t out, int64_t in, int p, int n, int g) {
  return layout(batch, &out, 1, 1, in, g, pair_bits(p, n)).total;
}

int64_t qgemm_group_workspace_bytes(int layers, int64_t batch, const int64_t* outs, int64_t in,
                                    int p, int n, int g) {
  if (layers < 1 || layers > kMaxGroup) return -1;
  return layout(batch, outs, layers, layers, in, g, pair_bits(p, n)).total;
}

hipError_t launch_qgemm_group(const void* x, int x_kind, int layers, const uint64_t* seeds,
                              int64_t batch, const uint8_t* const* codes,
                              const uint16_t* const* scales, const float* grid, int p, int n,
                              int g, const int64_t* outs, int64_t in, float* const* y,
                              void* workspace, hipStream_t stream) {
  if (!qgemm_format(p, n) || layers < 1 || layers > kMaxGroup)
    return hipErrorInvalidValue;
  const int bits = pair_bits(p, n);
  // one rotated copy of the activations per distinct seed arrangement: all
  // layers share it when their seeds agree (or the input is already rotated)
  bool same = true;
  for (int l = 1; l < layers; ++l) same = same && seeds[l] == seeds[0];
  const int nx = (x_kind == kQgemmRotated || same) ? 1 : layers;
  const Layout L = layout(batch, outs, layers, nx, in, g, bits);
  char* ws = static_cast<char*>(workspace);
  _Float16* x16 = reinterpret_cast<_Float16*>(ws + L.x16);
  float* xe = reinterpret_cast<float*>(ws + L.xe);
  const int64_t ngroups = batch * (in / g);
  XSeeds xs{};
  xs.nl = nx;
  for (int l = 0; l < nx; ++l) xs.s[l] = seeds[l];
  const XLayout xl = x_layout(batch, in, g);
  hipError_t err;
  switch (x_kind) {
    case kQgemmRotated:
      err = launch_xprep<float, false>(static_cast<const float*>(x), ngroups, g, xs, xl, x16, xe,
                                       stream);
      break;
    case kQgemmRawF32:
      err = launch_xprep<float, true>(static_cast<const float*>(x), ngroups, g, xs, xl, x16, xe,
                                      stream);
      break;
    case kQgemmRawBF16:
      err = launch_xprep<uint16_t, true>(static_cast<const uint16_t*>(x), ngroups, g, xs, xl,
                                         x16, xe, stream);
      break;
    default:
      return hipErrorInvalidValue;
  }
  if (err != hipSuccess) return err;

  const int gpr = int(in / g);
  for (int64_t b0 = 0; b0 < batch; b0 += 64) {
    const int nb = int(std::min<int64_t>(64, batch - b0));
    QG a{};
    a.x16 = x16 + (b0 / 64) * xl.chunk_halves;
    a.xe = xe + b0 * gpr;
    a.x16_stride = nx > 1 ? xl.layer_halves : 0;
    a.xrows = int(xl.rows);
    a.xe_stride = nx > 1 ? batch * gpr : 0;
    a.grid = grid;
    a.nb = nb;
    a.pair_table = p == 1 ? 1 : 0;
    a.log2g = log2_exact(g);
    a.in = int(in);
    a.gpr = gpr;
    a.nl = layers;
    RG r{};
    r.nl = layers;
    int64_t max_splits = 1, blocks = 0;
    for (int l = 0; l < layers; ++l) {
      const Split sp = plan_split(outs[l], in, nb, bits);
      max_splits = std::max(max_splits, sp.splits);
      a.blk0[l] = int(blocks);
      blocks += (outs[l] + kTileRows - 1) / kTileRows * sp.splits;
      float* part = reinterpret_cast<float*>(ws + L.part[l]);
      a.kps[l] = int(sp.stages_per_split * kStageK);
      a.splits[l] = int(sp.splits);
      r.splits[l] = int(sp.splits);
      a.codes[l] = codes[l];
      a.scales[l] = scales[l];
      a.dst[l] = sp.splits > 1 ? part : y[l] + b0 * outs[l];
      a.out[l] = int(outs[l]);
      r.part[l] = part;
      r.y[l] = y[l] + b0 * outs[l];
      r.n[l] = sp.splits > 1 ? int64_t(nb) * outs[l] : 0;  // unsplit layers: y written directly
      r.off[l + 1] = r.off[l] + r.n[l];
    }
    err = bits == 6    ? launch_bits<6>(a, g, blocks, stream)
          : bits == 10 ? launch_bits<10>(a, g, blocks, stream)
          : bits == 16 ? launch_bits<16>(a, g, blocks, stream)
                       : launch_bits<8>(a, g, blocks, stream);
    if (err != hipSuccess) return err;
    if (max_splits > 1) {
      const int64_t blocks = std::min<int64_t>((r.off[layers] + 255) / 256, 4096);
      hipLaunchKernelGGL(qgemm_reduce, dim3(unsigned(blocks)), dim3(256), 0, stream, r);
      err = hipGetLastError();
      if (err != hipSuccess) return err;
    }
  }
  return hipSuccess;
}

hipError_t launch_qgemm(const void* x, int x_kind, uint64_t seed, int64_t batch,
                        const uint8_t* codes, const uint16_t* scales, const float* grid, int p,
                        int n, int g, int64_t out, int64_t in, float* y, void* workspace,
                        hipStream_t stream) {
  return launch_qgemm_group(x, x_kind, 1, &seed, batch, &codes, &scales, grid, p, n, g, &out, in,
                            &y, workspace, stream);
}

}  // namespace higgs
