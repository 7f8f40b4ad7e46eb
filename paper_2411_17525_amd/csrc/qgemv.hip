// Lookup-table GEMV for HIGGS layers at small batch (1..8 activation rows),
// computed in the rotated space (App. G):
//   y[b][o] = sum_i scale[o][i] * sum_j < G[code(o,i,j)], x_rot[b, ig+jp : ig+(j+1)p] >
// Decoding at this batch is memory bound (Sec. 3.3): the kernel streams the
// packed codes from HBM once, coalesced, and keeps everything else on chip.
//
// Work split. The input dimension is cut into K-slices of 64 lane chunks; a
// lane chunk is 8 (8-bit codes) or 16 (6- and 10-bit codes) consecutive codes
// of a row, so a slice is 1024 or 2048 weights. A block owns a range of rows
// and all of K: each of its waves owns one or two fixed K-slices (kw waves
// cover K) and a row group (rg groups split the rows into tiles of 4 rows,
// 2 at batch 8).
// Because a wave's slices never change, its activations are loaded, rotated
// and converted once, and stay in registers as fp16 pairs for the whole
// kernel; the lane holding weights [16l, 16l + 16) of a slice holds exactly
// the activations it multiplies.
//
// Per block, before decoding:
//   * the codes of the wave's first kDepth items (an item is one tile in one
//     slice) are requested first, so their HBM latency overlaps everything
//     below;
//   * the RHT sign vector (App. G: the activations get the same sigma as the
//     weights) is computed cooperatively, one splitmix64 output per thread,
//     and kept as a bit mask in LDS;
//   * the lookup table of grid points (fp16 pairs) is built in LDS with one
//     copy per lane of a half wave, so the random reads of a wave do not
//     collide in banks (the grid-in-fast-memory constraint of Sec. 3.3,
//     replicated against bank conflicts);
//   * each wave rotates its slices (sign flip, fast Walsh-Hadamard transform,
//     1/sqrt(g)) unless they are already rotated, rescales them by an exact
//     power of two so the largest magnitude lands in [2^14, 2^15) (fp16 keeps
//     full precision without overflow) and converts them to fp16 pairs.
// Decoding: per code one LDS read of the table entry and one v_dot2_f32_f16
// per batch row (fp32 accumulation); per row and slice one group scale. The
// codes of the next tiles are in flight while the current one decodes. A tile
// ends with a fixed butterfly over the lanes; each wave's tile sums go to LDS
// and are added over the kw K-waves in a fixed order at the end of the block
// (deterministic, no atomics).
// Code formats: MODE 0 = 8-bit codes (p = 2, n = 256; also p = 1, n = 16 read
// as 256 byte values indexing a table of grid-point pairs), MODE 1 = 6-bit
// (p = 2, n = 64), MODE 2 = 10-bit (p = 2, n = 1024), MODE 3 = 8-bit scalar
// codes (p = 1, n = 256: the uniform CH8 grid of Sec. 3.3, or any 256-point
// scalar grid), one weight per code: a table entry holds one fp16 value and
// a pair of weights takes two table reads.

#include <algorithm>
#include <atomic>
#include <cmath>
#include <mutex>

#include "internal.h"
#include "wave_fwht.h"

namespace higgs {
namespace {

constexpr int kMaxWaves = 16;     // waves per block (8 for register-heavy shapes)
constexpr int kMinWaves = 4;      // the table fill assumes at least 256 threads
constexpr int kMaxSPW = 2;        // K-slices per wave
constexpr int kPartBytes = 32768; // LDS for the per-wave tile sums of a block
constexpr int kMaxSigWords = 64;  // sign mask of a group of up to 2048
constexpr int kMaxLayers = 4;     // layers of one launch (they share the activations)

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// Rotation modes of a launch (QArgs::rot): none (the activations are already
// rotated), in registers, or through the wave's LDS scratch (g = the slice of
// 16 elements per lane; kRotFloats floats per rotating wave).
constexpr int kRotNone = 0, kRotRegs = 1, kRotLds = 2;
constexpr int kRotFloats = kFwht1024Scratch;

template <int MODE>
struct Fmt;
template <>
struct Fmt<0> {  // 8-bit codes, 256 entries, 32 table copies
  static constexpr int kBits = 8, kCodes = 8, kWords = 2, kEntriesLog2 = 8, kRL = 5;
};
template <>
struct Fmt<1> {  // 6-bit codes, 64 entries, 64 copies
  static constexpr int kBits = 6, kCodes = 16, kWords = 3, kEntriesLog2 = 6, kRL = 6;
};
template <>
struct Fmt<2> {  // 10-bit codes, 1024 entries, 16 copies
  static constexpr int kBits = 10, kCodes = 16, kWords = 5, kEntriesLog2 = 10, kRL = 4;
};
template <>
struct Fmt<3> {  // 8-bit scalar codes, 256 entries, 32 copies; a "code" here is
                 // the pair of weights of two consecutive bytes (16 bits)
  static constexpr int kBits = 16, kCodes = 8, kWords = 4, kEntriesLog2 = 8, kRL = 5;
};

template <int MODE>
constexpr int slice_weights() {
  return 64 * 2 * Fmt<MODE>::kCodes;
}

// Largest batch rows per launch: the fp16 activations of a wave
// (slices x rows x codes-per-chunk registers) stay within 64 registers.
template <int MODE>
constexpr int max_rows_for(int spw) {
  return (MODE == 0 || MODE == 3 ? 8 : 4) / spw;
}

// Waves per block: 16 where a wave fits in 128 registers, else 8 (256).
// 8-bit pair codes up to 4 batch-row slices per wave; CH8 at batch tile 1
// (one or two slices: 72-116 registers), so that both take rows of up to
// 32768 weights.
template <int MODE>
constexpr int max_waves(int b, int spw) {
  return ((MODE == 0 && b * spw <= 4) || (MODE == 3 && b == 1)) ? 16 : 8;
}

// Items (a tile in one slice) whose codes are in flight per wave: deeper at
// batch 1, where registers are free.
template <int B>
constexpr int ring_depth() {
  return 2;
}

// Rows per tile: a tile's sums (rows x batch rows) stay within 16 registers.
template <int B>
constexpr int tile_rows() {
  return B >= 8 ? 2 : 4;
}

// Takes the word by value: __builtin_bit_cast applied directly to a vector
// element (u.y) reads the vector's first element instead.
__device__ inline half2_t as_half2(uint32_t w) { return __builtin_bit_cast(half2_t, w); }

__device__ inline uint32_t pack_half2(float a, float b) {
  const _Float16 ha = static_cast<_Float16>(a), hb = static_cast<_Float16>(b);
  return uint32_t(__builtin_bit_cast(uint16_t, ha)) |
         (uint32_t(__builtin_bit_cast(uint16_t, hb)) << 16);
}

// Byte offset in the table of the entry of code j of a chunk, for this lane's
// copy (entry-major: code * copies + copy, 4 bytes each). `copy_off` is
// copy * 8 for MODE 0 (one v_perm_b32 puts the code byte above it, a shift
// halves the pair: 32 copies, entry stride 128 bytes) and copy * 4 otherwise.
template <int MODE>
__device__ inline uint32_t lut_offset(const uint32_t (&d)[Fmt<MODE>::kWords], int j,
                                      uint32_t copy_off) {
  constexpr int kBits = Fmt<MODE>::kBits, RL = Fmt<MODE>::kRL;
  if constexpr (MODE == 0) {
    static_assert(RL == 5, "the byte-permute addressing assumes 32 copies");
    const uint32_t sel = 0x0c0c0000u | (uint32_t(4 + (j & 3)) << 8);
    return __builtin_amdgcn_perm(d[j >> 2], copy_off, sel) >> 1;
  } else {
    const int bit = j * kBits, word = bit >> 5, off = bit & 31;
    uint32_t v;
    if (off + kBits <= 32)
      v = d[word] >> off;
    else
      v = __builtin_amdgcn_alignbit(d[word + 1], d[word], off);
    return ((v & ((1u << kBits) - 1)) << (RL + 2)) | copy_off;
  }
}

// The fp16 pair of weights j of a chunk. MODE 3 reads the two bytes' entries
// (the value sits in the low half of the table word) with the MODE 0
// addressing; the other formats read one pair entry.
template <int MODE>
__device__ inline half2_t lut_pair(const uint32_t* s_lut, const uint32_t (&d)[Fmt<MODE>::kWords],
                                   int j, uint32_t copy_off) {
  const char* base = reinterpret_cast<const char*>(s_lut);
  if constexpr (MODE == 3) {
    const uint32_t w = d[j >> 1];
    const uint32_t sel_lo = 0x0c0c0000u | (uint32_t(4 + ((2 * j) & 3)) << 8);
    const uint32_t sel_hi = 0x0c0c0000u | (uint32_t(4 + ((2 * j + 1) & 3)) << 8);
    const uint32_t lo = *reinterpret_cast<const uint16_t*>(
        base + (__builtin_amdgcn_perm(w, copy_off, sel_lo) >> 1));
    const uint32_t hi = *reinterpret_cast<const uint16_t*>(
        base + (__builtin_amdgcn_perm(w, copy_off, sel_hi) >> 1));
    return as_half2(lo | (hi << 16));
  } else {
    return as_half2(*reinterpret_cast<const uint32_t*>(base + lut_offset<MODE>(d, j, copy_off)));
  }
}

// Word 3 of a raw buffer resource on gfx9-family chips (32-bit data format).
constexpr int kRsrcWord3 = 0x00020000;
// Per-lane buffer offset beyond any buffer here (< 2^31 bytes): out of range.
constexpr uint32_t kOffNone = 0x80000000u;
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
  } else if constexpr (MODE == 3) {
    const i32x4 u = __builtin_amdgcn_raw_buffer_load_b128(rs, int(voff), int(soff), kAuxNT);
    d[0] = uint32_t(u.x); d[1] = uint32_t(u.y); d[2] = uint32_t(u.z); d[3] = uint32_t(u.w);
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
        v[i] = keep + lane_xor<M>(send, lane);
      }
    } else {
      v[0] += lane_xor<M>(v[0], lane);
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

// One launch covers nl layers (1..kMaxLayers) that read the same
// activations: layer l owns blocks [blk0[l], blk0[l + 1]) (blk0[nl] = grid
// size), each block a range of that layer's rows.
struct QArgs {
  const void* x;  // activations: rotated fp32 (kRotNone) or raw fp32 / bf16 (rotated here)
  const float* grid;
  float rscale;    // 1/sqrt(g) as fp32 (rot = 1)
  int x_bf16, rot, nb, pair_table, log2g;  // rot: kRot*; x_bf16 only with a rotation
  int in;          // input size, shared by the layers
  int kw, rg;      // K-waves and row groups of a block (blockDim = 64 kw rg)
  int rows_per_block;  // a multiple of the tile height
  int part_floats;     // LDS floats of tile sums (rows_per_block * B * kw, rounded up to 4)
  int x_slots;         // (slice, batch row) pairs of shared activations in LDS (rg > 1)
  int nl;              // layers of this launch
  const uint8_t* codes[kMaxLayers];
  const uint16_t* scales[kMaxLayers];
  float* y[kMaxLayers];
  int out[kMaxLayers];  // rows (codes and scales address below 2^31 bytes)
  int blk0[kMaxLayers];
  uint32_t sig[kMaxLayers][kMaxSigWords];  // RHT signs: bit j set iff sigma_j = -1
};

}  // namespace

// Phase stamps (a separate debug build only, compiled with HIGGS_STAMPS): each
// wave of qgemv_kernel records s_memrealtime (a 100 MHz clock common to the
// device) at its phase boundaries into stamps[block][wave][16], set with
// higgs_debug_set_stamps. The product library is built without it.
#ifdef HIGGS_STAMPS
__device__ uint64_t* g_stamps;
#define HIGGS_STAMP(i) (st_[i] = __builtin_amdgcn_s_memrealtime())
#else
#define HIGGS_STAMP(i) ((void)0)
#endif

namespace {

// B: batch rows per launch (nb <= B are real); MODE: code format; SPW:
// K-slices per wave; USC: a scale group spans whole slices (g >= slice), so a
// row's scale in a slice is wave-uniform (one load per tile serves all rows);
// XB: the activations are bf16 (else fp32); RT: rows per tile (tile_rows<B>(),
// or 2 at batch 1 where a block holds few rows: two items per wave instead of
// one, so the first is decoded while the second's codes arrive).
template <int B, int MODE, int SPW, bool USC, bool XB, int RT>
__global__ __launch_bounds__(64 * max_waves<MODE>(B, SPW)) void qgemv_kernel(const QArgs a) {
  using F = Fmt<MODE>;
  constexpr int RL = F::kRL;
  constexpr int kCW = 2 * F::kCodes;  // weights per lane chunk
  constexpr int kSlice = 64 * kCW;
  constexpr int kChunkBytes = F::kCodes * F::kBits / 8;
  constexpr int kEntries = 1 << F::kEntriesLog2;
  constexpr int kLutWords = kEntries << RL;
  constexpr int kRT = RT;
  constexpr int kDepth = ring_depth<B>();
  constexpr int kV = kRT * B;
  static_assert((kV & (kV - 1)) == 0 && kV <= 64, "kRT * B must be a power of two <= 64");
  static_assert(kDepth % SPW == 0, "ring slots must map to fixed slices");

  __shared__ u32x4 s_lut4[kLutWords / 4];
  // dynamic: tile sums [rows_per_block][B][kw], then (rg > 1) the shared
  // activations [slice][B][lane][kCodes fp16 pairs] and their scales
  extern __shared__ u32x4 s_dyn4[];
  float* s_part = reinterpret_cast<float*>(s_dyn4);
  const uint32_t* s_lut = reinterpret_cast<const uint32_t*>(s_lut4);

#ifdef HIGGS_STAMPS
  uint64_t st_[10] = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
#endif
  HIGGS_STAMP(0);
  const int tid = int(threadIdx.x);
  const int lane = tid & 63;
  // wave index is uniform: keep it (and all row addressing) in scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // the arguments of the set-up, all requested in one round trip; the block's
  // layer is then picked by selects (an indexed read of the arguments would
  // be a second round trip)
  const int kw = a.kw, rg = a.rg, nl = a.nl;
  const uint8_t* codes_l[kMaxLayers];
  const uint16_t* scales_l[kMaxLayers];
  float* y_l[kMaxLayers];
  int out_l[kMaxLayers], blk0_l[kMaxLayers];
#pragma unroll
  for (int l = 0; l < kMaxLayers; ++l) {
    codes_l[l] = a.codes[l];
    scales_l[l] = a.scales[l];
    y_l[l] = a.y[l];
    out_l[l] = a.out[l];
    blk0_l[l] = a.blk0[l];
  }
  HIGGS_READ_NOW("s"(kw), "s"(rg), "s"(nl), "s"(a.x), "s"(a.grid), "s"(a.in), "s"(a.log2g),
                 "s"(a.nb), "s"(a.pair_table), "s"(codes_l[0]), "s"(codes_l[1]),
                 "s"(codes_l[2]), "s"(codes_l[3]), "s"(scales_l[0]), "s"(scales_l[1]),
                 "s"(scales_l[2]), "s"(scales_l[3]), "s"(y_l[0]), "s"(y_l[1]), "s"(y_l[2]),
                 "s"(y_l[3]), "s"(out_l[0]), "s"(out_l[1]), "s"(out_l[2]), "s"(out_l[3]),
                 "s"(blk0_l[1]), "s"(blk0_l[2]), "s"(blk0_l[3]), "s"(a.rows_per_block),
                 "s"(a.rot), "s"(a.rscale), "s"(a.part_floats), "s"(a.x_slots));
  int in = a.in, log2g = a.log2g, nb = a.nb, pair_table = a.pair_table, rot = a.rot;
  int rows_per_block = a.rows_per_block, part_floats = a.part_floats, x_slots = a.x_slots;
  float rscale = a.rscale;
  HIGGS_HOLD("+s"(in), "+s"(log2g), "+s"(nb), "+s"(pair_table), "+s"(rot), "+s"(rows_per_block),
             "+s"(part_floats), "+s"(x_slots), "+s"(rscale));
  HIGGS_STAMP(1);
  const int nthreads = 64 * kw * rg;  // the block size (not read from the dispatch)
  const int kslot = wave % kw, rgi = wave / kw;
  int L = 0;
#pragma unroll
  for (int l = 1; l < kMaxLayers; ++l)
    if (l < nl && int(blockIdx.x) >= blk0_l[l]) L = l;
  const uint8_t* codes = codes_l[0];
  const uint16_t* scales = scales_l[0];
  float* y = y_l[0];
  int out = out_l[0], blk0 = 0;
#pragma unroll
  for (int l = 1; l < kMaxLayers; ++l)
    if (L == l) {
      codes = codes_l[l];
      scales = scales_l[l];
      y = y_l[l];
      out = out_l[l];
      blk0 = blk0_l[l];
    }
  const int nchunks = in / kCW;
  const uint32_t row_bytes = uint32_t(nchunks) * kChunkBytes;
  const int gpr = in >> log2g;  // scale groups per row
  const int row0 = (int(blockIdx.x) - blk0) * rows_per_block;
  const int rows_here = min(rows_per_block, out - row0);
  const int ntb = (rows_here + kRT - 1) / kRT;                 // tiles of the block
  const int ntw = ntb > rgi ? (ntb - 1 - rgi) / rg + 1 : 0;   // tiles of this wave
  const int nitems = ntw * SPW;  // item i: tile i / SPW in slice i % SPW

  // ---- 0. grid points for the table (requested first: the table is the
  //         first thing built). The first 256 * P threads build it (P the
  //         largest power of two with 256 * P <= block size), each writing
  //         S consecutive 16-byte stores: entry e's copies are the stores
  //         [e * kStoresPerEntry, (e + 1) * kStoresPerEntry). Every thread
  //         loads, so no branch surrounds a load. ----
  constexpr int kStoresPerEntry = (1 << RL) / 4;
  constexpr int kStores = kEntries * kStoresPerEntry;
  constexpr int kMaxEPT = kEntries >= 256 ? kEntries / 256 : 1;  // entries per thread, at most
  const int tp = nthreads >= 1024 ? 4 : nthreads >= 512 ? 2 : 1;
  const int table_threads = 256 * tp;
  const int spt = kStores / table_threads;  // stores per table thread
  const int tt = min(tid, table_threads - 1);
  float gx[kMaxEPT], gy[kMaxEPT];
#pragma unroll
  for (int j = 0; j < kMaxEPT; ++j) {
    const int e = min((tt * spt) / kStoresPerEntry + j, kEntries - 1);
    if constexpr (MODE == 3) {  // one value per entry, in the low half
      gx[j] = a.grid[e];
      gy[j] = 0.f;
    } else {
      gx[j] = pair_table ? a.grid[e & 15] : a.grid[2 * e];
      gy[j] = pair_table ? a.grid[e >> 4] : a.grid[2 * e + 1];
    }
  }

  // this lane's kCW sign bits (bit i: sigma of element pos0 + i of its group;
  // the lane's elements sit at the same offsets in every group, since kCW
  // divides g), requested first
  const int g = 1 << log2g;
  const int pos0 = (lane * kCW) & (g - 1);
  const uint32_t sig_word = a.sig[L][pos0 >> 5];  // zero without rotation

  // ---- 1. raw activations of this wave's slices: (slice, batch row) pairs
  //         are loaded and converted kRound at a time; the first round is
  //         requested first, before the codes. A lane past K or a batch
  //         row past nb reads an in-range address and is zeroed later. ----
  constexpr int kPairs = SPW * B;
  constexpr int kRawWords = XB ? kCW / 2 : kCW;  // bf16 pairs or fp32 values
  constexpr int kRound = (kPairs >= 2 && 2 * kRawWords <= 32) ? 2 : 1;
  uint32_t raw[kRound][kRawWords];
  auto pair_real = [&](int q) {
    const int s = q / B, b = q % B;
    return b < nb && (kslot + s * kw) * kSlice + lane * kCW < in;
  };
  auto load_pair = [&](int q, uint32_t (&w)[kRawWords]) {
    const int s = q / B, b = q % B;
    const int sl = kslot + s * kw;
    const int e0 = (sl * kSlice + lane * kCW < in) ? sl * kSlice + lane * kCW : 0;
    const int64_t off = int64_t(b < nb ? b : 0) * in + e0;
    const u32x4* p = XB ? reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.x) + off)
                        : reinterpret_cast<const u32x4*>(static_cast<const float*>(a.x) + off);
#pragma unroll
    for (int w4 = 0; w4 < kRawWords / 4; ++w4) {
      const u32x4 u = p[w4];
      w[4 * w4] = u.x; w[4 * w4 + 1] = u.y; w[4 * w4 + 2] = u.z; w[4 * w4 + 3] = u.w;
    }
  };
#pragma unroll
  for (int u = 0; u < kRound; ++u) load_pair(u, raw[u]);

  // ---- 3. codes and scales of the first kDepth items. Rows past the layer
  //         and chunks past K read a clamped in-range address; their
  //         activations are zero or their sums are never stored. ----
  // Buffer resources over the exact code and scale arrays. Loads of items
  // that exist use clamped in-range offsets; loads of items past the wave's
  // last one are still issued (no branch around a load: the compiler's wait
  // counting stays exact) but with a per-lane offset past the end of the
  // buffer, which the hardware range check turns into zeros without a memory
  // access.
  const __amdgpu_buffer_rsrc_t crs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(codes), 0, int(uint32_t(out) * row_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t srs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(scales), 0, int(uint32_t(out) * uint32_t(gpr) * 2u), kRsrcWord3);

  // Scales come through vector loads, in order with the codes: with USC,
  // lane r < kRT holds the scale of row r of the tile (read back with
  // v_readlane); otherwise every lane holds its own group's scale per row.
  // (Scalar loads would share a counter with LDS reads and stall them.)
  constexpr int kScaleRegs = USC ? 1 : kRT;
  uint32_t buf[kDepth][kRT][F::kWords];
  uint32_t sbuf[kDepth][kScaleRegs];
  // ring slot t always holds slice t % SPW (kDepth is a multiple of SPW)
  auto fetch = [&](int item, int s, uint32_t (&d)[kRT][F::kWords], uint32_t (&sc)[kScaleRegs]) {
    const bool live = item < nitems;  // uniform
    const int rbase = row0 + (rgi + (item / SPW) * rg) * kRT;
    const int sl = kslot + s * kw;
    const int cl = min(sl * 64 + lane, nchunks - 1);
    const uint32_t voff = live ? uint32_t(cl) * kChunkBytes : kOffNone;
    // the scales first: they are consumed first
    if constexpr (USC) {
      const int gi = min((sl * kSlice) >> log2g, gpr - 1);
      const uint32_t rl = uint32_t(min(rbase + min(lane, kRT - 1), out - 1));
      sc[0] = uint32_t(uint16_t(__builtin_amdgcn_raw_buffer_load_b16(
          srs, int(live ? (rl * uint32_t(gpr) + uint32_t(gi)) * 2u : kOffNone), 0, kAuxNT)));
    } else {
      const uint32_t gl = live ? (uint32_t(cl * kCW) >> log2g) * 2u : kOffNone;
#pragma unroll
      for (int r = 0; r < kRT; ++r) {
        const uint32_t rc = uint32_t(min(rbase + r, out - 1));
        sc[r] = uint32_t(uint16_t(__builtin_amdgcn_raw_buffer_load_b16(
            srs, int(gl), int(rc * uint32_t(gpr) * 2u), kAuxNT)));
      }
    }
#pragma unroll
    for (int r = 0; r < kRT; ++r) {
      const uint32_t rc = uint32_t(min(rbase + r, out - 1));  // uniform
      load_chunk<MODE>(crs, voff, rc * row_bytes, d[r]);
    }
    // keep each item's loads together and in this order, so that waiting for
    // one item never waits for the next one's
    __builtin_amdgcn_sched_barrier(0);
  };
#pragma unroll
  for (int t = 0; t < kDepth; ++t) fetch(t, t % SPW, buf[t], sbuf[t]);

  // ---- 4. the table ----
  if (tid < table_threads) {
    for (int k = 0; k < spt; ++k) {
      const int si = tid * spt + k;
      const int j = si / kStoresPerEntry - (tid * spt) / kStoresPerEntry;  // < kMaxEPT
      const uint32_t v = pack_half2(gx[0], gy[0]);
      uint32_t vj = v;
#pragma unroll
      for (int q = 1; q < kMaxEPT; ++q)
        if (j == q) vj = pack_half2(gx[q], gy[q]);
      s_lut4[si] = u32x4{vj, vj, vj, vj};
    }
  }

  HIGGS_STAMP(2);

  // ---- 5. the waves of row group 0 rotate and convert the activations of
  //         their slices; with several row groups they leave them in LDS for
  //         the others (one rotation per block) ----
  half2_t xh[SPW][B][F::kCodes];
  float xs[SPW][B];
  const bool converts = rgi == 0;  // uniform
  const bool shares = rg > 1;      // uniform
  constexpr int kXVec = F::kCodes / 4;  // 16-byte vectors of fp16 pairs per lane
  u32x4* s_x = reinterpret_cast<u32x4*>(s_part + part_floats);
  float* s_xs = reinterpret_cast<float*>(s_x + (x_slots * 64 * kXVec));
  // Rotation of one (slice, batch row) pair when g is the slice (1024
  // elements, 16 per lane, lane l holding [16l, 16l + 16)) with every
  // butterfly inside a lane (fwht1024_lds, through the wave's LDS scratch of
  // kRotFloats floats at s_part + kslot * kRotFloats, free before the
  // decode): bit-identical to the register version and to the separate
  // rotation kernel, with about half the instructions. The fp16 pairs then go
  // in the decode layout to the shared activations (several row groups: every
  // wave reads them after the block barrier) or back through the scratch to
  // this wave's registers.
  auto rotate_slice_lds = [&](float (&v)[kCW], int s, int b) {
    if constexpr (kCW == 16) {  // (the call is compiled only then)
      float* wsc = s_part + kslot * kRotFloats;
      fwht1024_lds(v, wsc, lane);
      float m = 0.f;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        v[i] *= rscale;
        m = fmaxf(m, fabsf(v[i]));
      }
      m = wave_max(m, lane);
      int e = m > 0.f ? ilogbf(m) - 14 : 0;
      e = e < -126 ? -126 : e;
      xs[s][b] = ldexpf(1.0f, e);
      // fp16 pair (h, j / 2) of this lane is pair (2 (l % 4) + j / 2) of decode
      // lane 16 h + l / 4: 32-bit word 128 h + 2 l + j / 2 of the slot
      uint32_t pk[8];
#pragma unroll
      for (int k = 0; k < 8; ++k)
        pk[k] = pack_half2(ldexpf(v[2 * k], -e), ldexpf(v[2 * k + 1], -e));
      uint32_t* dw;
      if (shares) {
        const int slot = (kslot + s * kw) * B + b;
        dw = reinterpret_cast<uint32_t*>(s_x + slot * 64 * kXVec);
        if (lane == 0) s_xs[slot] = xs[s][b];
      } else {
        dw = reinterpret_cast<uint32_t*>(wsc);
      }
#pragma unroll
      for (int h = 0; h < 4; ++h)
        *reinterpret_cast<u32x2_t*>(dw + 128 * h + 2 * lane) = u32x2_t{pk[2 * h], pk[2 * h + 1]};
      if (!shares) {
        wave_lds_sync();
#pragma unroll
        for (int k = 0; k < kXVec; ++k) {
          const u32x4 u = reinterpret_cast<const u32x4*>(dw)[lane * kXVec + k];
          xh[s][b][4 * k] = as_half2(u.x);
          xh[s][b][4 * k + 1] = as_half2(u.y);
          xh[s][b][4 * k + 2] = as_half2(u.z);
          xh[s][b][4 * k + 3] = as_half2(u.w);
        }
      }
    }
  };
  auto convert_pair = [&](int q, const uint32_t (&w)[kRawWords]) {
    const int s = q / B, b = q % B;
#ifdef HIGGS_STAMPS
    if (q == 0) {
      __asm__ volatile("" ::"v"(w[0]));  // the first activations have arrived
      HIGGS_STAMP(3);
    }
#endif
    const bool real = pair_real(q);
    float v[kCW];
#pragma unroll
    for (int i = 0; i < kCW; ++i) {
      const uint32_t bits = XB ? ((i & 1) ? (w[i >> 1] & 0xffff0000u) : (w[i >> 1] << 16)) : w[i];
      v[i] = real ? __uint_as_float(bits) : 0.f;
    }
    if constexpr (kCW == 16) {
      if (rot == kRotLds) {  // uniform: g is the slice, 16 elements per lane
        const uint32_t neg = sig_word >> (pos0 & 31);
#pragma unroll
        for (int i = 0; i < kCW; ++i)
          v[i] = __uint_as_float(__float_as_uint(v[i]) ^ ((neg << (31 - i)) & 0x80000000u));
        rotate_slice_lds(v, s, b);
        return;
      }
    }
    if (rot) {
      const uint32_t neg = sig_word >> (pos0 & 31);
#pragma unroll
      for (int i = 0; i < kCW; ++i)  // sign bit of element i ^= bit i of neg
        v[i] = __uint_as_float(__float_as_uint(v[i]) ^ ((neg << (31 - i)) & 0x80000000u));
      fwht_in_lane<kCW>(v);
      // the deferred signs of the cross-lane stages ride on the 1/sqrt(g);
      // g = the slice (every stage runs) takes the branch-free form
      const float rs = rscale * (g == kSlice ? fwht_cross_lane_deferred_fixed<kCW, kSlice>(v, lane)
                                             : fwht_cross_lane_deferred<kCW>(v, lane, g));
#pragma unroll
      for (int i = 0; i < kCW; ++i) v[i] *= rs;
    }
    float m = 0.f;
#pragma unroll
    for (int i = 0; i < kCW; ++i) m = fmaxf(m, fabsf(v[i]));
    m = wave_max(m, lane);
    int e = m > 0.f ? ilogbf(m) - 14 : 0;
    e = e < -126 ? -126 : e;
#pragma unroll
    for (int j = 0; j < F::kCodes; ++j)
      xh[s][b][j] = __builtin_bit_cast(
          half2_t, pack_half2(ldexpf(v[2 * j], -e), ldexpf(v[2 * j + 1], -e)));
    xs[s][b] = ldexpf(1.0f, e);
    if (shares) {
      const int slot = (kslot + s * kw) * B + b;
      u32x4* dst = s_x + (slot * 64 + lane) * kXVec;
#pragma unroll
      for (int k = 0; k < kXVec; ++k)
        dst[k] = u32x4{__builtin_bit_cast(uint32_t, xh[s][b][4 * k]),
                       __builtin_bit_cast(uint32_t, xh[s][b][4 * k + 1]),
                       __builtin_bit_cast(uint32_t, xh[s][b][4 * k + 2]),
                       __builtin_bit_cast(uint32_t, xh[s][b][4 * k + 3])};
      if (lane == 0) s_xs[slot] = xs[s][b];
    }
  };
#pragma unroll
  for (int q0 = 0; q0 < kPairs; q0 += kRound) {
    if (q0 > 0) {
#pragma unroll
      for (int u = 0; u < kRound; ++u) load_pair(q0 + u, raw[u]);
    }
    if (converts) {
#pragma unroll
      for (int u = 0; u < kRound; ++u) convert_pair(q0 + u, raw[u]);
    }
  }
#ifdef HIGGS_STAMPS
  if (converts) {
    __asm__ volatile("" ::"v"(xs[0][0]));  // the conversion is done
    HIGGS_STAMP(4);
  } else {
    st_[3] = st_[4] = st_[2];
  }
#endif
  __syncthreads();
  HIGGS_STAMP(5);
  // the other row groups take the shared activations; so do the converting
  // waves after a rotation through LDS (it leaves them there only)
  if (!converts || (kCW == 16 && rot == kRotLds && shares)) {
#pragma unroll
    for (int q = 0; q < kPairs; ++q) {
      const int s = q / B, b = q % B;
      const int slot = (kslot + s * kw) * B + b;
      const u32x4* src = s_x + (slot * 64 + lane) * kXVec;
#pragma unroll
      for (int k = 0; k < kXVec; ++k) {
        const u32x4 u = src[k];
        xh[s][b][4 * k] = as_half2(u.x);
        xh[s][b][4 * k + 1] = as_half2(u.y);
        xh[s][b][4 * k + 2] = as_half2(u.z);
        xh[s][b][4 * k + 3] = as_half2(u.w);
      }
      xs[s][b] = s_xs[slot];
    }
  }

  // ---- 6. decode the wave's tiles ----
  const uint32_t copy_off = (MODE == 0 || MODE == 3) ? (uint32_t(lane) & 31u) << 3
                                                      : (uint32_t(lane) & ((1u << RL) - 1u)) << 2;
  float acc[kRT][B];
#pragma unroll
  for (int r = 0; r < kRT; ++r)
#pragma unroll
    for (int b = 0; b < B; ++b) acc[r][b] = 0.f;
  // rows whose table entries are read before their products (<= 32 registers)
  constexpr int kRB = (32 / F::kCodes) < kRT ? (32 / F::kCodes) : kRT;
  auto process = [&](int item, int s, const uint32_t (&d)[kRT][F::kWords],
                     const uint32_t (&sc)[kScaleRegs]) {
    // USC: lane r < kRT holds row r's scale; convert once, read per row
    const float sc_lane = float(__builtin_bit_cast(_Float16, uint16_t(sc[0])));
#pragma unroll
    for (int r0 = 0; r0 < kRT; r0 += kRB) {
      half2_t gv[kRB][F::kCodes];
#pragma unroll
      for (int r = 0; r < kRB; ++r)
#pragma unroll
        for (int j = 0; j < F::kCodes; ++j)
          gv[r][j] = lut_pair<MODE>(s_lut, d[r0 + r], j, copy_off);
#pragma unroll
      for (int r = 0; r < kRB; ++r) {
        float part[B];
#pragma unroll
        for (int b = 0; b < B; ++b) part[b] = 0.f;
#pragma unroll
        for (int j = 0; j < F::kCodes; ++j)
#pragma unroll
          for (int b = 0; b < B; ++b)
            part[b] = __builtin_amdgcn_fdot2(gv[r][j], xh[s][b][j], part[b], false);
        float sc_r;
        if constexpr (USC)
          sc_r = __builtin_bit_cast(
              float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, sc_lane), r0 + r));
        else
          sc_r = float(__builtin_bit_cast(_Float16, uint16_t(sc[r0 + r])));
#pragma unroll
        for (int b = 0; b < B; ++b)
          acc[r0 + r][b] = fmaf(part[b], sc_r * xs[s][b], acc[r0 + r][b]);
      }
    }
    if (s == SPW - 1) {  // the tile is complete: reduce over lanes, keep the sums
      float flat[kV];
#pragma unroll
      for (int r = 0; r < kRT; ++r)
#pragma unroll
        for (int b = 0; b < B; ++b) {
          flat[r * B + b] = acc[r][b];
          acc[r][b] = 0.f;
        }
      const float total = transpose_reduce<kV>(flat, lane);
      constexpr int kShift = 6 - __builtin_ctz(kV);
      const int k = lane >> kShift;  // value index r * B + b held by this lane
      if ((lane & ((1 << kShift) - 1)) == 0)
        s_part[((rgi + (item / SPW) * rg) * kRT * B + k) * kw + kslot] = total;
    }
  };

  for (int i = 0; i < nitems; i += kDepth) {
#pragma unroll
    for (int t = 0; t < kDepth; ++t) {
      if (i + t < nitems) process(i + t, t % SPW, buf[t], sbuf[t]);  // uniform
      fetch(i + t + kDepth, t % SPW, buf[t], sbuf[t]);
    }
  }
#ifdef HIGGS_STAMPS
  __builtin_amdgcn_s_waitcnt(0);  // the last tile's sums are in LDS
  HIGGS_STAMP(6);
#endif
  __syncthreads();
  HIGGS_STAMP(7);

  // ---- 7. add the K-waves' sums in a fixed order and store ----
  for (int q = tid; q < rows_here * B; q += nthreads) {
    const int rl = q / B, b = q - (q / B) * B;
    if (b < nb) {
      float t = 0.f;
      for (int k = 0; k < kw; ++k) t += s_part[q * kw + k];
      y[int64_t(b) * out + row0 + rl] = t;
    }
  }
#ifdef HIGGS_STAMPS
  HIGGS_STAMP(8);
  st_[9] = uint64_t(converts ? 1 : 0) | (uint64_t(kw) << 8) | (uint64_t(rg) << 16);
  if (lane == 0 && g_stamps != nullptr) {
    uint64_t* d = g_stamps + (uint64_t(blockIdx.x) * 16 + uint64_t(wave)) * 16;
#pragma unroll
    for (int i = 0; i < 10; ++i) d[i] = st_[i];
  }
#endif
}

typedef _Float16 half4_t __attribute__((ext_vector_type(4)));

// Value of lane (lane & ~3) + i (i = 0..3, compile time): DPP quad broadcast.
template <int I>
__device__ inline float quad_bcast(float v) {
  constexpr int kSel = I | (I << 2) | (I << 4) | (I << 6);
  return __builtin_bit_cast(
      float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), kSel, 0xF, 0xF, true));
}

// Batch >= 2 with 8-bit codes (MODE 0, one K-slice per wave): the same
// product with the multiply-adds on the matrix cores. Above batch 1 the
// small-batch kernel is VALU-bound (one v_dot2 per code and batch row); here
// the VALU work per code is the table addressing only.
// v_mfma_f32_4x4x4_16b_f16 computes 16 independent 4x4x4 products per wave:
// in block b (lanes 4b .. 4b+3), lane 4b+i supplies row i of A and column i
// of B (four fp16 values each, the reduction index in order) and receives
// column i of C (rows 0..3 in its four accumulators). Here A is the 4 weight
// rows of a tile and B 4 batch rows of the activations over the same 4
// weights: lane (b, q) = (lane / 4, lane % 4) holds the codes of tile row q
// and the activations of batch row q (and q + 4 for a batch tile of 8) for
// the 64 weights [64 b, 64 b + 64) of the wave's slice (four lane chunks).
// The 16 blocks' partial products of a tile are summed across lanes at the
// end of the tile; a block's 64 weights lie in one scale group (g >= 64), so
// each lane folds its block's product with its own group's scales.
// Activations are loaded straight into this layout and rotated in it: the
// butterflies run in the same order as in the small-batch kernel and the
// separate rotation kernel (element bits 0-5 in the lane, bits 6-9 across
// lanes 4, 8, 16, 32 apart with deferred signs), so every rotated value is
// bit-identical to theirs.
template <int NBQ, bool XB>
__global__ __launch_bounds__(1024) void qgemv_mfma_kernel(const QArgs a) {
  using F = Fmt<0>;
  constexpr int RL = F::kRL;
  constexpr int B = 4 * NBQ;       // batch rows of the launch
  constexpr int kLW = 64;          // weights of K per lane
  constexpr int kSlice = 16 * kLW;
  constexpr int kLaneBytes = 32;   // codes per lane per tile row
  constexpr int kEntries = 256;
  constexpr int kLutWords = kEntries << RL;
  constexpr int kRT = 4;           // rows per tile (the rows of A)
  constexpr int kDepth = NBQ == 1 ? 2 : 1;  // tiles of codes in flight (registers)

  __shared__ u32x4 s_lut4[kLutWords / 4];
  extern __shared__ u32x4 s_dyn4[];
  float* s_part = reinterpret_cast<float*>(s_dyn4);
  const uint32_t* s_lut = reinterpret_cast<const uint32_t*>(s_lut4);

  const int tid = int(threadIdx.x);
  const int lane = tid & 63;
  const int blk = lane >> 2, q = lane & 3;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // the arguments, all requested in one round trip (as in the small-batch
  // kernel); the block's layer is then picked by selects
  const int kw = a.kw, rg = a.rg, nl = a.nl;
  const uint8_t* codes_l[kMaxLayers];
  const uint16_t* scales_l[kMaxLayers];
  float* y_l[kMaxLayers];
  int out_l[kMaxLayers], blk0_l[kMaxLayers];
#pragma unroll
  for (int l = 0; l < kMaxLayers; ++l) {
    codes_l[l] = a.codes[l];
    scales_l[l] = a.scales[l];
    y_l[l] = a.y[l];
    out_l[l] = a.out[l];
    blk0_l[l] = a.blk0[l];
  }
  HIGGS_READ_NOW("s"(kw), "s"(rg), "s"(nl), "s"(a.x), "s"(a.grid), "s"(a.in), "s"(a.log2g),
                 "s"(a.nb), "s"(a.pair_table), "s"(a.rot), "s"(a.rscale), "s"(codes_l[0]),
                 "s"(codes_l[1]), "s"(codes_l[2]), "s"(codes_l[3]), "s"(scales_l[0]),
                 "s"(scales_l[1]), "s"(scales_l[2]), "s"(scales_l[3]), "s"(y_l[0]),
                 "s"(y_l[1]), "s"(y_l[2]), "s"(y_l[3]), "s"(out_l[0]), "s"(out_l[1]),
                 "s"(out_l[2]), "s"(out_l[3]), "s"(blk0_l[1]), "s"(blk0_l[2]), "s"(blk0_l[3]),
                 "s"(a.rows_per_block), "s"(a.part_floats), "s"(a.x_slots));
  int in = a.in, log2g = a.log2g, nb = a.nb, pair_table = a.pair_table, rot = a.rot;
  int rows_per_block = a.rows_per_block, x_slots = a.x_slots, part_floats = a.part_floats;
  HIGGS_HOLD("+s"(in), "+s"(log2g), "+s"(nb), "+s"(pair_table), "+s"(rot), "+s"(rows_per_block),
             "+s"(x_slots), "+s"(part_floats));
  const int nthreads = 64 * kw * rg;  // the block size (not read from the dispatch)
  const int kslot = wave % kw, rgi = wave / kw;
  int L = 0;
#pragma unroll
  for (int l = 1; l < kMaxLayers; ++l)
    if (l < nl && int(blockIdx.x) >= blk0_l[l]) L = l;
  const uint8_t* codes = codes_l[0];
  const uint16_t* scales = scales_l[0];
  float* y = y_l[0];
  int out = out_l[0], blk0 = 0;
#pragma unroll
  for (int l = 1; l < kMaxLayers; ++l)
    if (L == l) {
      codes = codes_l[l];
      scales = scales_l[l];
      y = y_l[l];
      out = out_l[l];
      blk0 = blk0_l[l];
    }
  const uint32_t row_bytes = uint32_t(in) / 2;  // one byte per two weights
  const int gpr = in >> log2g;
  const int row0 = (int(blockIdx.x) - blk0) * rows_per_block;
  const int rows_here = min(rows_per_block, out - row0);
  const int ntb = (rows_here + kRT - 1) / kRT;
  const int nitems = ntb > rgi ? (ntb - 1 - rgi) / rg + 1 : 0;  // tiles of this wave
  const int k0 = kslot * kSlice + kLW * blk;  // this lane's first weight of K
  const bool k_real = k0 < in;              // uniform per lane (in is a multiple of 64)

  // ---- grid points for the table (as in the small-batch kernel) ----
  constexpr int kStoresPerEntry = (1 << RL) / 4;
  constexpr int kStores = kEntries * kStoresPerEntry;
  const int tp = nthreads >= 1024 ? 4 : nthreads >= 512 ? 2 : 1;
  const int table_threads = 256 * tp;
  const int spt = kStores / table_threads;
  const int tt = min(tid, table_threads - 1);
  const int te = min((tt * spt) / kStoresPerEntry, kEntries - 1);
  const float gx = pair_table ? a.grid[te & 15] : a.grid[2 * te];
  const float gy = pair_table ? a.grid[te >> 4] : a.grid[2 * te + 1];

  // ---- sign bits of this lane's 64 weights (zero without rotation) ----
  const int g = 1 << log2g;
  const int pos = rot ? (k0 & (g - 1)) : 0;  // with rotation g <= 1024: words < 32
  const uint32_t neg_lo = a.sig[L][pos >> 5], neg_hi = a.sig[L][(pos >> 5) + 1];

  // ---- raw activations of batch row q + 4r; the first is requested before the codes ----
  constexpr int kRawWords = XB ? kLW / 2 : kLW;
  uint32_t raw[kRawWords];
  auto load_raw = [&](int r) {
    const int b = q + 4 * r;
    const int64_t off = int64_t(b < nb ? b : 0) * in + (k_real ? k0 : 0);
    const u32x4* p = XB ? reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.x) + off)
                        : reinterpret_cast<const u32x4*>(static_cast<const float*>(a.x) + off);
#pragma unroll
    for (int w4 = 0; w4 < kRawWords / 4; ++w4) {
      const u32x4 u = p[w4];
      raw[4 * w4] = u.x; raw[4 * w4 + 1] = u.y; raw[4 * w4 + 2] = u.z; raw[4 * w4 + 3] = u.w;
    }
  };
  load_raw(0);

  // ---- codes and scales of the first kDepth tiles (branch-free, as in the
  //      small-batch kernel). Lane (b, q): 32 bytes of codes of tile row q;
  //      the scale of tile row q in the lane's group. ----
  const __amdgpu_buffer_rsrc_t crs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(codes), 0, int(uint32_t(out) * row_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t srs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(scales), 0, int(uint32_t(out) * uint32_t(gpr) * 2u), kRsrcWord3);
  const uint32_t kbyte = uint32_t(k_real ? k0 : 0) / 2;
  const uint32_t gi = uint32_t(min((k_real ? k0 : 0) >> log2g, gpr - 1));
  uint32_t buf[kDepth][8];
  uint32_t sbuf[kDepth];
  auto fetch = [&](int item, uint32_t (&d)[8], uint32_t& sc) {
    const bool live = item < nitems;  // uniform
    const int rbase = row0 + (rgi + item * rg) * kRT;
    const uint32_t rc = uint32_t(min(rbase + q, out - 1));
    sc = uint32_t(uint16_t(__builtin_amdgcn_raw_buffer_load_b16(
        srs, int(live ? (rc * uint32_t(gpr) + gi) * 2u : kOffNone), 0, kAuxNT)));
    const uint32_t voff = live ? rc * row_bytes + kbyte : kOffNone;
    const i32x4 u0 = __builtin_amdgcn_raw_buffer_load_b128(crs, int(voff), 0, kAuxNT);
    const i32x4 u1 = __builtin_amdgcn_raw_buffer_load_b128(crs, int(voff + 16u), 0, kAuxNT);
    d[0] = uint32_t(u0.x); d[1] = uint32_t(u0.y); d[2] = uint32_t(u0.z); d[3] = uint32_t(u0.w);
    d[4] = uint32_t(u1.x); d[5] = uint32_t(u1.y); d[6] = uint32_t(u1.z); d[7] = uint32_t(u1.w);
    __builtin_amdgcn_sched_barrier(0);
  };
#pragma unroll
  for (int t = 0; t < kDepth; ++t) fetch(t, buf[t], sbuf[t]);

  // ---- the table ----
  if (tid < table_threads) {
    const uint32_t v = pack_half2(gx, gy);
    for (int k = 0; k < spt; ++k) s_lut4[tid * spt + k] = u32x4{v, v, v, v};
  }

  // ---- rotate and convert: per batch row of the lane, 64 values ----
  uint32_t xa[NBQ][32];  // fp16 pairs of the lane's 64 weights, per batch row
  float xs[NBQ];
  const bool converts = rgi == 0;  // uniform
  const bool shares = rg > 1;      // uniform
  u32x4* s_x = reinterpret_cast<u32x4*>(s_part + part_floats);
  float* s_xs = reinterpret_cast<float*>(s_x + (x_slots * 64 * 2));
  auto convert = [&](int r) {
    const int b = q + 4 * r;
    const bool real = b < nb && k_real;
    float v[kLW];
#pragma unroll
    for (int i = 0; i < kLW; ++i) {
      const uint32_t bits = XB ? ((i & 1) ? (raw[i >> 1] & 0xffff0000u) : (raw[i >> 1] << 16)) : raw[i];
      v[i] = real ? __uint_as_float(bits) : 0.f;
    }
    if (rot) {
#pragma unroll
      for (int i = 0; i < kLW; ++i) {
        const uint32_t nb_ = i < 32 ? neg_lo : neg_hi;
        v[i] = __uint_as_float(__float_as_uint(v[i]) ^ ((nb_ << (31 - (i & 31))) & 0x80000000u));
      }
      // element bits 0..5 inside the lane (only those below g)
#pragma unroll
      for (int h = 1; h < kLW; h <<= 1) {
        if (h < g) {  // uniform
#pragma unroll
          for (int i = 0; i < kLW; ++i)
            if ((i & h) == 0) {
              const float x0 = v[i], x1 = v[i + h];
              v[i] = x0 + x1;
              v[i + h] = x0 - x1;
            }
        }
      }
      // element bits 6..9: lanes 4, 8, 16, 32 apart, signs deferred (16 values at a time)
      int mask = 0;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        float t[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) t[i] = v[16 * c + i];
        if (kLW < g) fwht_lane_stage_deferred<4>(t, lane);
        if (2 * kLW < g) fwht_lane_stage_deferred<8>(t, lane);
        if (4 * kLW < g) fwht_lane_stage_deferred<16>(t, lane);
        if (8 * kLW < g) fwht_lane_stage_deferred<32>(t, lane);
#pragma unroll
        for (int i = 0; i < 16; ++i) v[16 * c + i] = t[i];
      }
      if (kLW < g) mask |= 1;
      if (2 * kLW < g) mask |= 2;
      if (4 * kLW < g) mask |= 4;
      if (8 * kLW < g) mask |= 8;
      const float sgn = (__builtin_popcount(blk & mask) & 1) ? -1.f : 1.f;
      const float rs = a.rscale * sgn;
#pragma unroll
      for (int i = 0; i < kLW; ++i) v[i] *= rs;
    }
    float mx = 0.f;
#pragma unroll
    for (int i = 0; i < kLW; ++i) mx = fmaxf(mx, fabsf(v[i]));
    // over the 16 lanes holding this batch row
    mx = fmaxf(mx, lane_xor<4>(mx, lane));
    mx = fmaxf(mx, lane_xor<8>(mx, lane));
    mx = fmaxf(mx, lane_xor<16>(mx, lane));
    mx = fmaxf(mx, lane_xor<32>(mx, lane));
    int e = mx > 0.f ? ilogbf(mx) - 14 : 0;
    e = e < -126 ? -126 : e;
#pragma unroll
    for (int j = 0; j < 32; ++j) xa[r][j] = pack_half2(ldexpf(v[2 * j], -e), ldexpf(v[2 * j + 1], -e));
    xs[r] = ldexpf(1.0f, e);
    if (shares) {
      const int slot = (kslot * NBQ + r) * 4;
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        u32x4* dst = s_x + ((slot + m) * 64 + lane) * 2;
        dst[0] = u32x4{xa[r][8 * m], xa[r][8 * m + 1], xa[r][8 * m + 2], xa[r][8 * m + 3]};
        dst[1] = u32x4{xa[r][8 * m + 4], xa[r][8 * m + 5], xa[r][8 * m + 6], xa[r][8 * m + 7]};
      }
      if (blk == 0) s_xs[slot + q] = xs[r];
    }
  };
  if (converts) convert(0);
#pragma unroll
  for (int r = 1; r < NBQ; ++r) {
    __builtin_amdgcn_sched_barrier(0);  // keep the next row's loads after the conversion
    load_raw(r);
    if (converts) convert(r);
  }
  __syncthreads();
  if (!converts) {
#pragma unroll
    for (int r = 0; r < NBQ; ++r) {
      const int slot = (kslot * NBQ + r) * 4;
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const u32x4* src = s_x + ((slot + m) * 64 + lane) * 2;
        const u32x4 u0 = src[0], u1 = src[1];
        xa[r][8 * m] = u0.x; xa[r][8 * m + 1] = u0.y; xa[r][8 * m + 2] = u0.z; xa[r][8 * m + 3] = u0.w;
        xa[r][8 * m + 4] = u1.x; xa[r][8 * m + 5] = u1.y; xa[r][8 * m + 6] = u1.z; xa[r][8 * m + 7] = u1.w;
      }
      xs[r] = s_xs[slot + q];
    }
  }

  // ---- decode: per tile 16 steps of v_mfma_f32_4x4x4_16b_f16 ----
  const uint32_t copy_off = (uint32_t(lane) & 31u) << 3;
  auto process = [&](int item, const uint32_t (&d)[8], uint32_t sc) {
    f32x4_t c[NBQ];
#pragma unroll
    for (int r = 0; r < NBQ; ++r) c[r] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const uint32_t dm[2] = {d[2 * m], d[2 * m + 1]};
      half2_t gv[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) gv[j] = lut_pair<0>(s_lut, dm, j, copy_off);
#pragma unroll
      for (int s4 = 0; s4 < 4; ++s4) {
        const half4_t av = half4_t{gv[2 * s4].x, gv[2 * s4].y, gv[2 * s4 + 1].x, gv[2 * s4 + 1].y};
#pragma unroll
        for (int r = 0; r < NBQ; ++r) {
          const half2_t x0 = as_half2(xa[r][8 * m + 2 * s4]), x1 = as_half2(xa[r][8 * m + 2 * s4 + 1]);
          const half4_t bv = half4_t{x0.x, x0.y, x1.x, x1.y};
          c[r] = __builtin_amdgcn_mfma_f32_4x4x4f16(av, bv, c[r], 0, 0, 0);
        }
      }
    }
    // fold: accumulator i is tile row i, whose scale (in the lane's group)
    // sits in lane 4b + i; then sum the 16 blocks (lanes 4 apart)
    const float sc_lane = float(__builtin_bit_cast(_Float16, uint16_t(sc)));
    const float s_row[4] = {quad_bcast<0>(sc_lane), quad_bcast<1>(sc_lane), quad_bcast<2>(sc_lane),
                            quad_bcast<3>(sc_lane)};
    float tot[NBQ][4];
#pragma unroll
    for (int r = 0; r < NBQ; ++r)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float t = c[r][i] * (s_row[i] * xs[r]);
        t += lane_xor<4>(t, lane);
        t += lane_xor<8>(t, lane);
        t += lane_xor<16>(t, lane);
        t += lane_xor<32>(t, lane);
        tot[r][i] = t;
      }
    if (blk == 0) {
      const int tile = rgi + item * rg;
#pragma unroll
      for (int r = 0; r < NBQ; ++r)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          s_part[((tile * kRT + i) * B + q + 4 * r) * kw + kslot] = tot[r][i];
    }
  };

  for (int i = 0; i < nitems; i += kDepth) {
#pragma unroll
    for (int t = 0; t < kDepth; ++t) {
      if (i + t < nitems) process(i + t, buf[t], sbuf[t]);  // uniform
      fetch(i + t + kDepth, buf[t], sbuf[t]);
    }
  }
  __syncthreads();

  // ---- add the K-waves' sums in a fixed order and store ----
  for (int qq = tid; qq < rows_here * B; qq += nthreads) {
    const int rl = qq / B, b = qq - (qq / B) * B;
    if (b < nb) {
      float t = 0.f;
      for (int k = 0; k < kw; ++k) t += s_part[qq * kw + k];
      y[int64_t(b) * out + row0 + rl] = t;
    }
  }
}

// Compute units of the current device, queried once per device. Several
// threads may race to fill an entry: they store the same value, and the
// entries are atomics, so the race is benign.
int device_cus() {
  static std::atomic<int> cus[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int v = cus[dev].load(std::memory_order_relaxed);
  if (v == 0) {
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
      v = 256;
    cus[dev].store(v, std::memory_order_relaxed);
  }
  return v;
}

// Launch shape of one layer: batch rows per launch, slices per wave,
// K-waves, row groups, rows per block and dynamic LDS. One block per compute
// unit, of 4..max_waves waves: the per-block setup (table, rotation) is paid
// once per compute unit.
struct Shape {
  int B, spw, nslices, kw, rg, rt, rows_per_block, blocks, part_floats, x_slots;
  bool lds_rot;  // the rotation goes through LDS (kRotLds)
  size_t lds_bytes;
};

constexpr size_t kLdsBytes = 160 * 1024;
constexpr size_t kMaxSharedX = 64 * 1024;     // LDS for shared activations
constexpr size_t kMaxSharedXMf = 96 * 1024;   // the same for the matrix-core variant

template <int MODE>
constexpr size_t static_lds() {
  return size_t(4) << (Fmt<MODE>::kEntriesLog2 + Fmt<MODE>::kRL);
}

// True when the matrix-core variant takes a small batch: 8-bit codes, batch
// >= 2 (below the batch where the full matrix-core path takes over), one
// K-slice per wave (the 64 weights of a lane lie in one scale group since
// g >= 64).
template <int MODE>
bool mfma_small_batch(int64_t batch, int g, int64_t in) {
  return MODE == 0 && batch >= 2 && g >= 64 && in <= int64_t(slice_weights<0>()) * kMaxWaves;
}

template <int MODE>
bool plan(const int* outs, int nl, int64_t in, int64_t batch, Shape& sh, int* blk0, bool mf,
          bool lds_rot) {
  constexpr int kSlice = slice_weights<MODE>();
  sh.nslices = int((in + kSlice - 1) / kSlice);
  sh.B = 0;
  if (mf) {  // matrix-core variant: batch tiles of 4 or 8, one slice per wave
    sh.B = batch >= 5 ? 8 : 4;
    sh.spw = 1;
    if (sh.nslices > kMaxWaves) return false;
  } else {
    // largest batch tile first (fewest passes over the codes), then one slice
    // per wave if the waves of a block can cover K that way
    const int want = batch >= 8 ? 8 : batch >= 3 ? 4 : int(batch);
    for (int b = want; b >= 1 && sh.B == 0; b >>= 1)
      for (int spw = 1; spw <= kMaxSPW && sh.B == 0; ++spw)
        if (b <= max_rows_for<MODE>(spw) && sh.nslices <= max_waves<MODE>(b, spw) * spw) {
          sh.B = b;
          sh.spw = spw;
        }
  }
  if (sh.B == 0) return false;
  const int wmax = mf ? kMaxWaves : max_waves<MODE>(sh.B, sh.spw);
  sh.kw = (sh.nslices + sh.spw - 1) / sh.spw;
  // rows per tile: 2 for 8-bit codes at batch 1 when the slices of a row
  // span few waves and the blocks hold few rows (q/k/v, o of an 8B block:
  // two items per wave, the first decoded while the second arrives;
  // measured 7.9 -> 7.7 and 6.9 -> 6.6 us), else 4 (2 at batch tiles of 8)
  int kRT = (mf || sh.B < 8) ? 4 : 2;
  if (MODE == 0 && !mf && sh.B == 1 && sh.spw == 1 && sh.kw <= 4) {
    int64_t t4 = 0;
    for (int l = 0; l < nl; ++l) t4 += (outs[l] + 3) / 4;
    if ((t4 + device_cus() - 1) / device_cus() * 4 <= 32) kRT = 2;
  }
  sh.rt = kRT;
  int64_t ntiles = 0;
  for (int l = 0; l < nl; ++l) ntiles += (outs[l] + kRT - 1) / kRT;
  const int64_t cus = device_cus();
  const int64_t tpb_max = std::max<int64_t>(1, kPartBytes / (int64_t(kRT) * sh.B * sh.kw * 4));
  // tiles per block: the fewest with one block per compute unit, blocks never
  // straddling two layers
  auto blocks_for = [&](int64_t t) {
    int64_t b = 0;
    for (int l = 0; l < nl; ++l) b += ((outs[l] + kRT - 1) / kRT + t - 1) / t;
    return b;
  };
  int64_t tpb = std::max<int64_t>(1, std::min<int64_t>((ntiles + cus - 1) / cus, tpb_max));
  while (tpb < tpb_max && blocks_for(tpb) > cus) ++tpb;
  const int rg_max = std::max(1, wmax / sh.kw);
  const int rg_min = std::min(rg_max, (kMinWaves + sh.kw - 1) / sh.kw);
  sh.rg = int(std::min<int64_t>(rg_max, std::max<int64_t>(rg_min, tpb)));
  constexpr size_t kXPerSlot = size_t(64) * Fmt<MODE>::kCodes * 4 + 4;  // fp16 pairs + scale
  size_t xbytes = size_t(sh.kw) * sh.spw * sh.B * kXPerSlot;
  if (sh.rg > 1 && xbytes > (mf ? kMaxSharedXMf : kMaxSharedX)) sh.rg = rg_min;
  if (sh.rg == 1) xbytes = 0;
  sh.x_slots = xbytes ? sh.kw * sh.spw * sh.B : 0;
  sh.rows_per_block = int(kRT * tpb);
  sh.blocks = 0;
  for (int l = 0; l < nl; ++l) {
    blk0[l] = sh.blocks;
    sh.blocks += (outs[l] + sh.rows_per_block - 1) / sh.rows_per_block;
  }
  sh.part_floats = (sh.rows_per_block * sh.B * sh.kw + 3) & ~3;
  sh.lds_bytes = size_t(sh.part_floats) * 4 + xbytes;
  // the rotation scratch of the kw converting waves shares the tile-sum
  // area (written only after the block barrier that ends the rotation)
  sh.lds_rot = false;
  if (lds_rot && !mf && 2 * Fmt<MODE>::kCodes == 16) {
    const int pf = std::max(sh.part_floats, sh.kw * kRotFloats);
    const size_t bytes = size_t(pf) * 4 + xbytes;
    if (bytes + static_lds<MODE>() <= kLdsBytes) {
      sh.part_floats = pf;
      sh.lds_bytes = bytes;
      sh.lds_rot = true;
    }
  }
  return sh.lds_bytes + static_lds<MODE>() <= kLdsBytes;
}

template <int B, int MODE, int SPW, bool USC, bool XB, int RT>
hipError_t launch_k(const QArgs& a, const Shape& sh, hipStream_t stream) {
  static std::once_flag attr_once;
  static hipError_t attr_err = hipSuccess;
  std::call_once(attr_once, [] {
    // the dynamic part (tile sums, shared activations) may pass the 64 KiB default
    attr_err = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&qgemv_kernel<B, MODE, SPW, USC, XB, RT>),
                                   hipFuncAttributeMaxDynamicSharedMemorySize,
                                   int(kLdsBytes - static_lds<MODE>()));
  });
  if (attr_err != hipSuccess) return attr_err;
  hipLaunchKernelGGL((qgemv_kernel<B, MODE, SPW, USC, XB, RT>), dim3(unsigned(sh.blocks)),
                     dim3(unsigned(64 * sh.kw * sh.rg)), sh.lds_bytes, stream, a);
  return hipGetLastError();
}

template <int B, int MODE, int SPW, int RT>
hipError_t launch_rt(const QArgs& a, const Shape& sh, hipStream_t stream) {
  // uniform scales: a group spans whole slices
  const bool usc = (1 << a.log2g) >= slice_weights<MODE>();
  if (a.rot && a.x_bf16)
    return usc ? launch_k<B, MODE, SPW, true, true, RT>(a, sh, stream)
               : launch_k<B, MODE, SPW, false, true, RT>(a, sh, stream);
  return usc ? launch_k<B, MODE, SPW, true, false, RT>(a, sh, stream)
             : launch_k<B, MODE, SPW, false, false, RT>(a, sh, stream);
}

template <int B, int MODE, int SPW>
hipError_t launch_spw(const QArgs& a, const Shape& sh, hipStream_t stream) {
  if constexpr (B == 1 && MODE == 0 && SPW == 1) {
    if (sh.rt == 2) return launch_rt<B, MODE, SPW, 2>(a, sh, stream);
  }
  return launch_rt<B, MODE, SPW, tile_rows<B>()>(a, sh, stream);
}

template <int NBQ, bool XB>
hipError_t launch_mf(const QArgs& a, const Shape& sh, hipStream_t stream) {
  static std::once_flag attr_once;
  static hipError_t attr_err = hipSuccess;
  std::call_once(attr_once, [] {
    attr_err = hipFuncSetAttribute(reinterpret_cast<const void*>(&qgemv_mfma_kernel<NBQ, XB>),
                                   hipFuncAttributeMaxDynamicSharedMemorySize,
                                   int(kLdsBytes - static_lds<0>()));
  });
  if (attr_err != hipSuccess) return attr_err;
  hipLaunchKernelGGL((qgemv_mfma_kernel<NBQ, XB>), dim3(unsigned(sh.blocks)),
                     dim3(unsigned(64 * sh.kw * sh.rg)), sh.lds_bytes, stream, a);
  return hipGetLastError();
}

template <int NBQ>
hipError_t launch_mf_nbq(const QArgs& a, const Shape& sh, hipStream_t stream) {
  return (a.rot && a.x_bf16) ? launch_mf<NBQ, true>(a, sh, stream)
                             : launch_mf<NBQ, false>(a, sh, stream);
}

template <int B, int MODE>
hipError_t launch_b(const QArgs& a, const Shape& sh, hipStream_t stream) {
  if constexpr (B <= max_rows_for<MODE>(1)) {
    if (sh.spw == 1) return launch_spw<B, MODE, 1>(a, sh, stream);
  }
  if constexpr (B <= max_rows_for<MODE>(2)) {
    if (sh.spw == 2) return launch_spw<B, MODE, 2>(a, sh, stream);
  }
  return hipErrorInvalidValue;
}

template <int MODE>
hipError_t run_mode(QArgs a, int64_t batch, hipStream_t stream) {
  Shape sh{};
  const bool mf = mfma_small_batch<MODE>(batch, 1 << a.log2g, a.in);
  // a rotation over groups of exactly one slice goes through LDS
  const bool lds_rot = a.rot != kRotNone && (1 << a.log2g) == slice_weights<MODE>();
  if (!plan<MODE>(a.out, a.nl, a.in, batch, sh, a.blk0, mf, lds_rot))
    return hipErrorInvalidValue;
  if (sh.lds_rot) a.rot = kRotLds;
  const char* x0 = static_cast<const char*>(a.x);
  float* y0[kMaxLayers];
  for (int l = 0; l < kMaxLayers; ++l) y0[l] = a.y[l];
  const int esz = (a.rot && a.x_bf16) ? 2 : 4;
  a.kw = sh.kw;
  a.rg = sh.rg;
  a.rows_per_block = sh.rows_per_block;
  a.part_floats = sh.part_floats;
  a.x_slots = sh.x_slots;
  for (int64_t b0 = 0; b0 < batch; b0 += sh.B) {
    a.nb = int(std::min<int64_t>(sh.B, batch - b0));
    a.x = x0 + b0 * a.in * esz;
    for (int l = 0; l < a.nl; ++l) a.y[l] = y0[l] + b0 * a.out[l];
    hipError_t err = hipErrorInvalidValue;
    if (mf) {
      err = sh.B == 8 ? launch_mf_nbq<2>(a, sh, stream) : launch_mf_nbq<1>(a, sh, stream);
      if (err != hipSuccess) return err;
      continue;
    }
    switch (sh.B) {
      case 1: err = launch_b<1, MODE>(a, sh, stream); break;
      case 2: err = launch_b<2, MODE>(a, sh, stream); break;
      case 4: err = launch_b<4, MODE>(a, sh, stream); break;
      case 8: err = launch_b<8, MODE>(a, sh, stream); break;
      default: break;
    }
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

hipError_t run_qgemv(QArgs a, int64_t batch, int p, int n, hipStream_t stream) {
  const int bits = code_bits(p, n);
  if (bits == 6) return run_mode<1>(a, batch, stream);
  if (bits == 10) return run_mode<2>(a, batch, stream);
  if (p == 1 && n == 256) return run_mode<3>(a, batch, stream);
  return run_mode<0>(a, batch, stream);
}

// The RHT sign mask of (seed, g): bit j set iff sigma_j = -1. Kept in a small
// per-thread cache, since a model calls every layer with its own fixed seed.
void sign_mask(uint64_t seed, int g, uint32_t (&mask)[kMaxSigWords]) {
  struct Entry {
    uint64_t seed = 0;
    int g = 0;
    uint32_t mask[kMaxSigWords];
  };
  constexpr int kEntries = 256;
  thread_local Entry cache[kEntries];
  const uint64_t h = (seed ^ (uint64_t(g) << 32)) * 0x9E3779B97F4A7C15ull;
  Entry& e = cache[h >> 56];
  if (e.g != g || e.seed != seed) {
    for (int w = 0; w < kMaxSigWords; ++w) e.mask[w] = 0;
    for (int j = 0; j < g; ++j)
      if (rht_sign_negative(seed, uint32_t(j))) e.mask[j >> 5] |= 1u << (j & 31);
    e.seed = seed;
    e.g = g;
  }
  for (int w = 0; w < kMaxSigWords; ++w) mask[w] = e.mask[w];
}

QArgs make_args(const void* x, int x_bf16, int rot, int nl, const uint64_t* seeds,
                const uint8_t* const* codes, const uint16_t* const* scales,
                const int64_t* outs, float* const* y, const float* grid, int p, int g,
                int64_t in) {
  QArgs a{};
  a.x = x;
  a.grid = grid;
  a.nl = nl;
  for (int l = 0; l < nl; ++l) {
    a.codes[l] = codes[l];
    a.scales[l] = scales[l];
    a.y[l] = y[l];
    a.out[l] = int(outs[l]);
    if (rot) sign_mask(seeds[l], g, a.sig[l]);
  }
  // the same constant the separate rotation kernel uses (fp32 of the fp64 value)
  a.rscale = float(1.0 / std::sqrt(double(g)));
  a.x_bf16 = x_bf16;
  a.rot = rot ? kRotRegs : kRotNone;
  a.pair_table = p == 1 ? 1 : 0;
  a.log2g = log2_exact(g);
  a.in = int(in);
  return a;
}

}  // namespace

int64_t qgemv_max_in(int p, int n) {
  // batch tile 1 with the most slices a block covers
  const int bits = code_bits(p, n);
  if (bits == 6) return int64_t(slice_weights<1>()) * max_waves<1>(1, kMaxSPW) * kMaxSPW;
  if (bits == 10) return int64_t(slice_weights<2>()) * max_waves<2>(1, kMaxSPW) * kMaxSPW;
  if (p == 1 && n == 256)
    return int64_t(slice_weights<3>()) * max_waves<3>(1, kMaxSPW) * kMaxSPW;
  return int64_t(slice_weights<0>()) * max_waves<0>(1, kMaxSPW) * kMaxSPW;
}

bool qgemv_rotates(int p, int n, int g) {
  const int bits = code_bits(p, n);
  const int slice = bits == 6 ? slice_weights<1>() : bits == 10 ? slice_weights<2>()
                                                                : slice_weights<0>();
  return g <= slice && g <= 32 * kMaxSigWords;
}

hipError_t launch_qgemv(const float* x_rot, int64_t batch, const uint8_t* codes,
                        const uint16_t* scales, const float* grid, int p, int n, int g,
                        int64_t out, int64_t in, float* y, hipStream_t stream) {
  if (in > qgemv_max_in(p, n)) return hipErrorInvalidValue;
  const uint64_t seed = 0;
  const QArgs a = make_args(x_rot, 0, 0, 1, &seed, &codes, &scales, &out, &y, grid, p, g, in);
  return run_qgemv(a, batch, p, n, stream);
}

hipError_t launch_qgemv_rotating(const void* x, int x_bf16, uint64_t seed, int64_t batch,
                                 const uint8_t* codes, const uint16_t* scales, const float* grid,
                                 int p, int n, int g, int64_t out, int64_t in, float* y,
                                 hipStream_t stream) {
  if (in > qgemv_max_in(p, n) || !qgemv_rotates(p, n, g)) return hipErrorInvalidValue;
  const QArgs a = make_args(x, x_bf16, 1, 1, &seed, &codes, &scales, &out, &y, grid, p, g, in);
  return run_qgemv(a, batch, p, n, stream);
}

hipError_t launch_qgemv_rotating_group(const void* x, int x_bf16, int layers,
                                       const uint64_t* seeds, int64_t batch,
                                       const uint8_t* const* codes, const uint16_t* const* scales,
                                       const float* grid, int p, int n, int g, const int64_t* outs,
                                       int64_t in, float* const* y, hipStream_t stream) {
  if (layers < 1 || layers > kMaxLayers || in > qgemv_max_in(p, n) || !qgemv_rotates(p, n, g))
    return hipErrorInvalidValue;
  const QArgs a = make_args(x, x_bf16, 1, layers, seeds, codes, scales, outs, y, grid, p, g, in);
  return run_qgemv(a, batch, p, n, stream);
}

int qgemv_max_layers() { return kMaxLayers; }

}  // namespace higgs

#ifdef HIGGS_STAMPS
// Debug build only: the buffer of qgemv_kernel's phase stamps (NULL: none).
extern "C" int higgs_debug_set_stamps(void* p) {
  return int(hipMemcpyToSymbol(HIP_SYMBOL(higgs::g_stamps), &p, sizeof(p)));
}
#endif
