// Lookup-table GEMM for HIGGS layers at batch >= 16 on the matrix cores,
// computed in the rotated space (App. G):
//   y[b][o] = sum_i scale[o][i] * sum_j < G[code(o,i,j)], x_rot[b, ig+jp : ig+(j+1)p] >
// At these batch sizes the layer is a dense contraction, so the dequantised
// weights feed v_mfma_f32_32x32x16_f16 directly. Two kernels per call:
//   * xprep_kernel converts the activations once: optionally rotating raw
//     activations first (sign flip, fast Walsh-Hadamard transform, 1/sqrt(g),
//     the same arithmetic as the separate rotation kernel), then an exact
//     power-of-two rescale per batch row and group so that the group's
//     largest magnitude lands in [2^14, 2^15). fp16 then keeps full
//     precision and cannot overflow. Output: fp16 activations and one
//     power of two per (row, group), in the workspace.
//   * qgemm_kernel: a block owns 128 rows (4 waves x 32) and a K-range; the
//     grid's second dimension splits K when the layer has too few rows to
//     fill the chip (partial sums go to the workspace and are added in a
//     fixed order by qgemm_reduce: deterministic).
//     A operand: each lane reads 16 bytes of codes of its row (16 codes = 32
//     weights) per 64-weight K-block, kRing K-blocks ahead of use, and turns
//     them into fp16 pairs through an LDS lookup table (32 copies, one per
//     lane of a half wave: no bank conflicts). The MFMA's reduction index is
//     mapped so that lane half h of step s covers weights 32h + 8s .. +7 of
//     the K-block, for A and B alike.
//     B operand: the fp16 activations of one stage (256 weights of K) in
//     LDS; the next stage's are loaded into registers while the current one
//     is multiplied, together with the next stage's group scales and
//     activation exponents.
//     Products accumulate in fp32 MFMA registers; every kFold K-blocks the
//     group scale and activation exponent are applied and the result is
//     added into fp32 totals (one rounding: an fma by an exactly scaled
//     factor).
// Every global load is unconditional (buffer loads with an out-of-range
// offset return zero without touching memory), so waiting for one load never
// waits for a later-issued one.
// Code format: 8-bit codes (p = 2, n = 256; p = 1, n = 16 read as byte
// values indexing a table of grid-point pairs).

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
constexpr int kCopiesLog2 = 5;          // table copies (one per lane of a half wave)
constexpr int kLutWords = 256 << kCopiesLog2;
constexpr int kStageK = 256;            // weights of K per staged activation chunk
constexpr int kStageKB = kStageK / 64;  // K-blocks per stage
constexpr int kXRow = kStageK + 8;      // halves per staged activation row (padded)
constexpr int kRing = 2 * kStageKB;     // K-blocks of codes in flight per lane

// Word 3 of a raw buffer resource on gfx9-family chips (32-bit data format).
constexpr int kRsrcWord3 = 0x00020000;
constexpr int kAuxNT = 2;  // non-temporal: codes are read once
// Per-lane buffer offset beyond any buffer here (< 2^31 bytes): reads zero.
constexpr uint32_t kOffNone = 0x80000000u;

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f16x_acc __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

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
template <int E, typename InT, bool ROT>
__global__ __launch_bounds__(256) void xprep_kernel(const InT* __restrict__ x, int64_t ngroups,
                                                    uint64_t seed, float rscale,
                                                    _Float16* __restrict__ x16,
                                                    float* __restrict__ xe) {
  const int lane = int(threadIdx.x) & 63;
  const int64_t wave0 = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  const int64_t nwaves = int64_t(gridDim.x) * 4;
  constexpr int g = 64 * E;
  uint64_t neg = 0;
  if (ROT) {
#pragma unroll
    for (int i = 0; i < E; ++i)
      neg |= uint64_t(rht_sign_negative(seed, uint32_t(lane * E + i))) << i;
  }
  for (int64_t grp = wave0; grp < ngroups; grp += nwaves) {
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
    _Float16* dst = x16 + base;
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
    if (lane == 0) xe[grp] = ldexpf(1.0f, e);
  }
}

// ---------------------------------------------------------------------------
// The product over one chunk of <= 64 batch rows.
// ---------------------------------------------------------------------------
struct QG {
  const _Float16* x16;  // [nb][in], fp16, rows of this chunk
  const float* xe;      // [nb][gpr], powers of two
  const uint8_t* codes;
  const uint16_t* scales;
  const float* grid;
  float* dst;              // [splits][nb][out]
  int64_t dst_split_stride;
  int nb, pair_table, log2g, out, in, gpr;
  int kps;                 // weights of K per split (a multiple of kStageK)
};

// NB: 32-column batch tiles (1 or 2). FOLD: K-blocks per fold (1, 2 or 4:
// min(g / 64, kStageKB), so a fold never spans two groups).
template <int NB, int FOLD>
__global__ __launch_bounds__(kThreads) void qgemm_kernel(const QG a) {
  constexpr int kBatch = 32 * NB;
  constexpr int kTPR = kThreads / kBatch;       // staging threads per activation row
  constexpr int kVec = kStageK / 8 / kTPR;      // 16-byte vectors per staging thread
  constexpr int kFolds = kStageKB / FOLD;       // folds per stage
  __shared__ u32x4 s_lut4[kLutWords / 4];
  __shared__ u32x4 s_x4[kBatch * kXRow / 8];
  const uint32_t* s_lut = reinterpret_cast<const uint32_t*>(s_lut4);
  const _Float16* s_x = reinterpret_cast<const _Float16*>(s_x4);

  const int tid = int(threadIdx.x);
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int row0 = int(blockIdx.x) * kTileRows + wave * 32;
  const int kbeg = int(blockIdx.y) * a.kps;
  const int kend = min(a.in, kbeg + a.kps);
  const int nkb = (kend - kbeg) >> 6;                  // K-blocks of this block
  const int nst = (nkb + kStageKB - 1) / kStageKB;     // stages of this block

  // ---- 1. grid points of this thread's table entry (256 threads, 256 entries) ----
  const int e = tid;
  const float gx = a.pair_table ? a.grid[e & 15] : a.grid[2 * e];
  const float gy = a.pair_table ? a.grid[e >> 4] : a.grid[2 * e + 1];

  // ---- 2. activations of stage 0: thread row xr, halves [xk, xk + 8 kVec) ----
  const int xr = tid / kTPR;
  const int xk = (tid % kTPR) * (8 * kVec);
  const __amdgpu_buffer_rsrc_t xrs = rsrc(a.x16, uint32_t(a.nb) * uint32_t(a.in) * 2u);
  u32x4 xv[kVec];
  // Stage c = nst (prefetched after the last stage, never used) reads real
  // data or zeros; only weights past the end of the row must read zero.
  auto load_x = [&](int c) {
    const int k = kbeg + c * kStageK + xk;
    const uint32_t off = (xr < a.nb && k < a.in)
                             ? (uint32_t(xr) * uint32_t(a.in) + uint32_t(k)) * 2u
                             : kOffNone;
#pragma unroll
    for (int v = 0; v < kVec; ++v)
      xv[v] = as_u32x4(__builtin_amdgcn_raw_buffer_load_b128(xrs, int(off + 16u * v), 0, 0));
  };
  load_x(0);

  // ---- 3. codes ring: lane row arow, lane half ahalf ----
  const int ahalf = lane >> 5;
  const uint32_t row_bytes = uint32_t(a.in) / 2;  // one byte per 2 weights
  const uint32_t arow = uint32_t(min(row0 + (lane & 31), a.out - 1));
  const __amdgpu_buffer_rsrc_t crs = rsrc(a.codes, uint32_t(a.out) * row_bytes);
  const uint32_t cbase = arow * row_bytes + uint32_t(kbeg >> 1) + 16u * uint32_t(ahalf);
  u32x4 ring[kRing];
  // K-blocks past the block's range re-read its last one (never used: a
  // partial last stage multiplies them by zero activations)
  auto fetch = [&](int j) {
    const uint32_t off = cbase + 32u * uint32_t(min(j, nkb - 1));
    return as_u32x4(__builtin_amdgcn_raw_buffer_load_b128(crs, int(off), 0, kAuxNT));
  };
#pragma unroll
  for (int t = 0; t < kRing; ++t) ring[t] = fetch(t);

  // ---- 4. scales of each fold of a stage: lane l -> row row0 + l % 32 (group
  //      scale, fp16 bits) and batch row 32t + l % 32 (activation exponent) ----
  const __amdgpu_buffer_rsrc_t srs = rsrc(a.scales, uint32_t(a.out) * uint32_t(a.gpr) * 2u);
  const __amdgpu_buffer_rsrc_t ers = rsrc(a.xe, uint32_t(a.nb) * uint32_t(a.gpr) * 4u);
  const uint32_t srow = uint32_t(min(row0 + (lane & 31), a.out - 1));
  uint32_t sc[kFolds];
  float xs[NB][kFolds];
  // groups past the row's end (a partial last stage, or the stage prefetched
  // after the last one) re-read the row's last group: finite, and multiplied
  // by zero or never used
  auto load_scales = [&](int c) {
#pragma unroll
    for (int f = 0; f < kFolds; ++f) {
      const int grp = min((kbeg + c * kStageK + f * FOLD * 64) >> a.log2g, a.gpr - 1);
      sc[f] = uint32_t(uint16_t(__builtin_amdgcn_raw_buffer_load_b16(
          srs, int((srow * uint32_t(a.gpr) + uint32_t(grp)) * 2u), 0, 0)));
#pragma unroll
      for (int t = 0; t < NB; ++t) {
        const int b = 32 * t + (lane & 31);  // rows past nb read zero (never stored)
        xs[t][f] = __builtin_bit_cast(
            float, __builtin_amdgcn_raw_buffer_load_b32(
                       ers, int(b < a.nb ? (uint32_t(b) * uint32_t(a.gpr) + uint32_t(grp)) * 4u
                                         : kOffNone), 0, 0));
      }
    }
  };
  load_scales(0);

  // ---- the table: 32 copies of each entry (8 stores of 16 bytes) ----
  {
    const uint32_t v = pack_h2(gx, gy);
#pragma unroll
    for (int k = 0; k < 8; ++k) s_lut4[e * 8 + k] = u32x4{v, v, v, v};
  }

  const uint32_t copy8 = uint32_t(lane & 31) << 3;  // table copy, pre-shifted for perm + >> 1
  f16x_acc total[NB];
#pragma unroll
  for (int t = 0; t < NB; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) total[t][r] = 0.f;

  // One stage: K-blocks 4c .. 4c+3, codes from ring slots 4H .. 4H+3.
  auto stage = [&](int c, auto H) {
    constexpr int kSlot0 = decltype(H)::value * kStageKB;
    __syncthreads();  // previous stage consumed (first time: table written)
    {
      u32x4* dst = s_x4 + (xr * kXRow + xk) / 8;
#pragma unroll
      for (int v = 0; v < kVec; ++v) dst[v] = xv[v];
    }
    uint32_t sc_c[kFolds];
    float xs_c[NB][kFolds];
#pragma unroll
    for (int f = 0; f < kFolds; ++f) {
      sc_c[f] = sc[f];
#pragma unroll
      for (int t = 0; t < NB; ++t) xs_c[t][f] = xs[t][f];
    }
    __syncthreads();
    // issue the next stage's loads now: the scheduler would otherwise delay
    // them to the end of the stage to save registers
    load_x(c + 1);
    load_scales(c + 1);
    __builtin_amdgcn_sched_barrier(0);

    // The stage's 16 MFMA steps (4 per K-block), software-pipelined: the
    // LDS operands of step st + kAhead are read while step st multiplies.
    constexpr int kSteps = 4 * kStageKB;
    constexpr int kAhead = 2;
    struct Step {
      half8 a;
      half8 b[NB];
    };
    auto load_step = [&](int st, Step& o) {
      const int kb = st / 4, s = st % 4;  // K-block inside the stage, step inside it
      const u32x4 cw = ring[kSlot0 + kb];
      const uint32_t w = s == 0 ? cw.x : s == 1 ? cw.y : s == 2 ? cw.z : cw.w;
      // A: codes 4s .. 4s+3 -> 8 halves (weights 32h + 8s .. + 7)
      uint32_t a32[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t sel = 0x0c0c0000u | (uint32_t(4 + q) << 8);
        const uint32_t off = __builtin_amdgcn_perm(w, copy8, sel) >> 1;
        a32[q] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(s_lut) + off);
      }
      o.a = __builtin_bit_cast(half8, u32x4{a32[0], a32[1], a32[2], a32[3]});
      // B: batch row 32t + lane % 32, the same 8 weights
#pragma unroll
      for (int t = 0; t < NB; ++t)
        o.b[t] = *reinterpret_cast<const half8*>(s_x + (32 * t + (lane & 31)) * kXRow + kb * 64 +
                                                 32 * ahalf + 8 * s);
    };
    Step ops[kSteps];
#pragma unroll
    for (int st = 0; st < kAhead; ++st) load_step(st, ops[st]);
    f16x_acc acc[NB];
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
      if (st % (4 * FOLD) == 0) {
#pragma unroll
        for (int t = 0; t < NB; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;
      }
      if (st + kAhead < kSteps) load_step(st + kAhead, ops[st + kAhead]);
      // the last step reading a K-block's codes is issued: refill its ring slot
      if (st + kAhead < kSteps && (st + kAhead) % 4 == 3) {
        const int kb = (st + kAhead) / 4;
        ring[kSlot0 + kb] = fetch(c * kStageKB + kb + kRing);
      }
#pragma unroll
      for (int t = 0; t < NB; ++t)
        acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ops[st].a, ops[st].b[t], acc[t], 0, 0, 0);
      if (st % 4 == 3) __builtin_amdgcn_sched_barrier(0);
      if (st % (4 * FOLD) == 4 * FOLD - 1) {
        // fold: accumulator register r holds row 8 (r / 4) + 4 ahalf + r % 4
        // of the wave's 32, column 32t + lane % 32
        const int fo = st / (4 * FOLD);
        const float sf = float(__builtin_bit_cast(_Float16, uint16_t(sc_c[fo])));
        const int sfi = __builtin_bit_cast(int, sf);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int rl = 8 * (r / 4) + (r % 4);
          const float s0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(sfi, rl));
          const float s1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(sfi, rl + 4));
          const float sr = ahalf ? s1 : s0;
#pragma unroll
          for (int t = 0; t < NB; ++t) total[t][r] = fmaf(acc[t][r], sr * xs_c[t][fo], total[t][r]);
        }
      }
    }
  };

  // Pairs of stages with no branch between them (a branch there lets the
  // compiler sink the prefetch loads of one stage down into the next), then
  // the odd last stage.
  int c = 0;
  for (; c + 1 < nst; c += 2) {
    stage(c, std::integral_constant<int, 0>{});
    stage(c + 1, std::integral_constant<int, 1>{});
  }
  if (c < nst) stage(c, std::integral_constant<int, 0>{});

  // ---- store through LDS so that lanes write consecutive rows: the wave's
  //      32 rows x kBatch columns go to its slice of the activation buffer
  //      (free once every wave has left the stage loop) ----
  constexpr int kORow = 33;  // floats per staged column (32 rows + 1: no bank conflicts)
  static_assert(kWaves * kBatch * kORow * 4 <= int(sizeof(s_x4)), "output staging fits");
  __syncthreads();
  float* s_o = reinterpret_cast<float*>(s_x4) + wave * (kBatch * kORow);
#pragma unroll
  for (int t = 0; t < NB; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      s_o[(32 * t + (lane & 31)) * kORow + 8 * (r / 4) + 4 * ahalf + (r % 4)] = total[t][r];
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  float* dst = a.dst + int64_t(blockIdx.y) * a.dst_split_stride + row0;
  const int orow = lane & 31;
#pragma unroll
  for (int i = 0; i < kBatch / 2; ++i) {
    const int b = 2 * i + ahalf;
    if (b < a.nb && row0 + orow < a.out) dst[int64_t(b) * a.out + orow] = s_o[b * kORow + orow];
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

// K-split of a layer: stages per split and the number of splits.
struct Split {
  int64_t stages_per_split;
  int64_t splits;
};

// Chooses the K-split for a chunk of nb batch rows from a simple model of
// MI355X (256 compute units, two blocks each): the time of the busiest
// compute unit at a sustained rate of one matrix instruction per 64 cycles
// per wave, against HBM traffic of codes plus split partial sums (written,
// then read back), plus the reduction launch when there is more than one
// split. The plan depends only on the shapes, so the workspace size is a
// function of the arguments.
Split plan_split(int64_t out, int64_t in, int64_t nb) {
  constexpr double kCUs = 256, kClock = 2.4e9, kCyclesPerMfma = 64, kHbm = 6e12;
  constexpr double kReduceLaunch = 3e-6, kRoundLatency = 1.5e-6;
  const int64_t tiles = (out + kTileRows - 1) / kTileRows;
  const int64_t stages = (in + kStageK - 1) / kStageK;
  const int64_t nbt = nb > 32 ? 2 : 1;
  double best_t = 1e30;
  Split best{stages, 1};
  for (int64_t s = 1; s <= stages; s *= 2) {
    const int64_t sps = (stages + s - 1) / s;
    const int64_t splits = (stages + sps - 1) / sps;
    const double blocks = double(tiles * splits);
    const double per_block = double(sps * kStageKB * 4 * nbt) * kCyclesPerMfma / kClock;
    const double t_mfma = per_block * std::ceil(blocks / kCUs);
    const double bytes = double(out) * double(in) / 2 + (splits > 1 ? 8.0 * splits * nb * out : 0);
    const double t = std::max(t_mfma, bytes / kHbm) + (splits > 1 ? kReduceLaunch : 0) +
                     kRoundLatency * std::ceil(blocks / (2 * kCUs));
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
hipError_t launch_xprep_e(const InT* x, int64_t ngroups, uint64_t seed, float rscale,
                          _Float16* x16, float* xe, hipStream_t stream) {
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((ngroups + 3) / 4, 8192));
  hipLaunchKernelGGL((xprep_kernel<E, InT, ROT>), dim3(unsigned(blocks)), dim3(256), 0, stream, x,
                     ngroups, seed, rscale, x16, xe);
  return hipGetLastError();
}

template <typename InT, bool ROT>
hipError_t launch_xprep(const InT* x, int64_t ngroups, int g, uint64_t seed, _Float16* x16,
                        float* xe, hipStream_t stream) {
  const float rscale = float(1.0 / std::sqrt(double(g)));
  switch (g) {
#define HIGGS_XPREP(G) \
  case G:              \
    return launch_xprep_e<G / 64, InT, ROT>(x, ngroups, seed, rscale, x16, xe, stream);
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

template <int NB, int FOLD>
hipError_t launch_nb(const QG& a, int64_t tiles, int64_t splits, hipStream_t stream) {
  hipLaunchKernelGGL((qgemm_kernel<NB, FOLD>), dim3(unsigned(tiles), unsigned(splits)),
                     dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

template <int NB>
hipError_t launch_fold(const QG& a, int g, int64_t tiles, int64_t splits, hipStream_t stream) {
  if (g >= 256) return launch_nb<NB, 4>(a, tiles, splits, stream);
  if (g == 128) return launch_nb<NB, 2>(a, tiles, splits, stream);
  return launch_nb<NB, 1>(a, tiles, splits, stream);
}

// Workspace layout: fp16 activations [batch][in], exponents [batch][in / g],
// split partial sums [splits][min(batch, 64)][out] (each 256-byte aligned).
struct Layout {
  int64_t x16, xe, part, total;
};

Layout layout(int64_t batch, int64_t out, int64_t in, int g) {
  // partial sums: the larger of the full 64-row chunks and the last one
  int64_t part = 0;
  for (const int64_t nb : {std::min<int64_t>(batch, 64), batch % 64}) {
    if (nb == 0) continue;
    const Split sp = plan_split(out, in, nb);
    if (sp.splits > 1) part = std::max(part, sp.splits * nb * out * 4);
  }
  Layout L;
  L.x16 = 0;
  L.xe = align256(batch * in * 2);
  L.part = L.xe + align256(batch * (in / g) * 4);
  L.total = L.part + part;
  return L;
}

}  // namespace

int64_t qgemm_workspace_bytes(int64_t batch, int64_t out, int64_t in, int g) {
  return layout(batch, out, in, g).total;
}

hipError_t launch_qgemm(const void* x, int x_kind, uint64_t seed, int64_t batch,
                        const uint8_t* codes, const uint16_t* scales, const float* grid, int p,
                        int g, int64_t out, int64_t in, float* y, void* workspace,
                        hipStream_t stream) {
  const Layout L = layout(batch, out, in, g);
  char* ws = static_cast<char*>(workspace);
  _Float16* x16 = reinterpret_cast<_Float16*>(ws + L.x16);
  float* xe = reinterpret_cast<float*>(ws + L.xe);
  float* part = reinterpret_cast<float*>(ws + L.part);
  const int64_t ngroups = batch * (in / g);
  hipError_t err;
  switch (x_kind) {
    case kQgemmRotated:
      err = launch_xprep<float, false>(static_cast<const float*>(x), ngroups, g, seed, x16, xe,
                                       stream);
      break;
    case kQgemmRawF32:
      err = launch_xprep<float, true>(static_cast<const float*>(x), ngroups, g, seed, x16, xe,
                                      stream);
      break;
    case kQgemmRawBF16:
      err = launch_xprep<uint16_t, true>(static_cast<const uint16_t*>(x), ngroups, g, seed, x16,
                                         xe, stream);
      break;
    default:
      return hipErrorInvalidValue;
  }
  if (err != hipSuccess) return err;

  const int64_t tiles = (out + kTileRows - 1) / kTileRows;
  const int gpr = int(in / g);
  for (int64_t b0 = 0; b0 < batch; b0 += 64) {
    const int nb = int(std::min<int64_t>(64, batch - b0));
    const Split sp = plan_split(out, in, nb);
    QG a;
    a.x16 = x16 + b0 * in;
    a.xe = xe + b0 * gpr;
    a.codes = codes;
    a.scales = scales;
    a.grid = grid;
    a.dst = sp.splits > 1 ? part : y + b0 * out;
    a.dst_split_stride = int64_t(nb) * out;
    a.nb = nb;
    a.pair_table = p == 1 ? 1 : 0;
    a.log2g = log2_exact(g);
    a.out = int(out);
    a.in = int(in);
    a.gpr = gpr;
    a.kps = int(sp.stages_per_split * kStageK);
    err = nb > 32 ? launch_fold<2>(a, g, tiles, sp.splits, stream)
                  : launch_fold<1>(a, g, tiles, sp.splits, stream);
    if (err != hipSuccess) return err;
    if (sp.splits > 1) {
      const int64_t n = int64_t(nb) * out;
      const int64_t blocks = std::min<int64_t>((n + 255) / 256, 4096);
      hipLaunchKernelGGL(qgemm_reduce, dim3(unsigned(blocks)), dim3(256), 0, stream, part,
                         int(sp.splits), n, y + b0 * out);
      err = hipGetLastError();
      if (err != hipSuccess) return err;
    }
  }
  return hipSuccess;
}

}  // namespace higgs
