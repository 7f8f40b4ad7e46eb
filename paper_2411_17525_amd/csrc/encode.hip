// HIGGS encoder (Alg. 1, RHT-VQ, with the grid of Alg. 2) on the GPU.
//
// One wavefront encodes one group of g consecutive weights of one row:
//   s = ||w||_2                      (fp64 sum of squares, fixed reduction tree)
//   w_dag = H (sigma * (w / s))      (fp64, in-register / cross-lane butterflies)
//   code_j = argmin_k ||w_dag[jp:(j+1)p] - G_k||^2, lowest k on ties
//   scale = fp16(s / sqrt(g))        (one rounding from fp64)
// The search compares c_k = |G_k|^2 / 2 - <v, G_k>, which orders the grid
// points exactly as the squared distance does, in fp64. To take the running
// minimum and its index in one v_min_f64, each candidate's value is shifted
// by a power of two S that makes it positive and its 10 lowest mantissa bits
// are replaced by k: positive doubles order as their bit patterns, so the
// minimum is the smallest value, ties (and values within 1024 ulps of S,
// S 2^-42) going to the lowest k. |v| <= sqrt(g) for a p-vector of a rotated
// group (its squared norm sums to g), so |c_k| <= R^2 / 2 + sqrt(g) R with R
// the largest grid-point norm; each block takes S = the least power of two
// >= max(1024, 2 (R^2 / 2 + sqrt(g) R)) from the grid it loads. Every grid of
// unit-variance points gets S = 1024, where the order differs from the plain
// fp64 distance only at squared-distance gaps below ~5e-10; the band is
// S 2^-41 in general, below 1e-6 for grids whose points have norms <= 1024.
// Codes are packed LSB-first into the row's bit stream through LDS.
// The work is dominated by the n-candidate scan per p-vector: VALU bound.

#include <algorithm>
#include <cmath>

#include "internal.h"
#include "wave_fwht.h"

namespace higgs {
namespace {

constexpr int kWaves = 4;
constexpr int kMaxN = 1024;
constexpr int kMaxG = 4096;
constexpr double kMinShift = 1024.0;   // least shift of the search values
constexpr uint32_t kIndexMask = 1023;  // low mantissa bits that carry the index (n <= 1024)

// min(best, c with its 10 lowest mantissa bits replaced by k). c and best
// are positive and finite, so no NaN handling is needed: one bit-field insert
// on the low word and one v_min_f64 (the compiler's fmin would first quieten
// both operands).
__device__ inline double min_indexed(double best, double c, uint32_t k, uint32_t index_mask) {
  const uint64_t u = __builtin_bit_cast(uint64_t, c);
  uint32_t lo;
  // lo = (k & index_mask) | (low word of c & ~index_mask); index_mask in a VGPR
  __asm__("v_bfi_b32 %0, %1, %2, %3" : "=v"(lo) : "v"(index_mask), "s"(k), "v"(uint32_t(u)));
  const double ck = __builtin_bit_cast(double, (u & 0xffffffff00000000ull) | uint64_t(lo));
  double r;
  __asm__("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(best), "v"(ck));
  return r;
}

// fp64 -> IEEE binary16 bits, round to nearest even, for finite x >= 0.
__device__ inline uint16_t f64_to_f16_rne(double x) {
  if (!(x > 0.0)) return 0;
  if (x >= 65520.0) return 0x7C00;                  // rounds to +infinity
  const int e = ilogb(x);                           // x in [2^e, 2^(e+1))
  const int qe = e - 10 > -24 ? e - 10 : -24;       // fp16 spacing in that binade
  const double r = ldexp(rint(ldexp(x, -qe)), qe);  // exact fp16 value
  const _Float16 h = static_cast<_Float16>(static_cast<float>(r));  // exact conversions
  return __builtin_bit_cast(uint16_t, h);
}

template <typename InT>
__device__ inline double to_f64(InT v);
template <>
__device__ inline double to_f64<float>(float v) { return double(v); }
template <>
__device__ inline double to_f64<uint16_t>(uint16_t v) {
  return double(__uint_as_float(uint32_t(v) << 16));
}

template <int E, typename InT>
__device__ inline void load_group(const InT* __restrict__ src, double (&v)[E]) {
  constexpr int kBytes = E * int(sizeof(InT));
  if constexpr (kBytes % 16 == 0) {
    constexpr int kPer = 16 / int(sizeof(InT));
#pragma unroll
    for (int q = 0; q < kBytes / 16; ++q) {
      const u32x4 u = load_stream16(reinterpret_cast<const char*>(src) + 16 * q);
      const InT* e = reinterpret_cast<const InT*>(&u);
#pragma unroll
      for (int i = 0; i < kPer; ++i) v[q * kPer + i] = to_f64<InT>(e[i]);
    }
  } else {
#pragma unroll
    for (int i = 0; i < E; ++i) v[i] = to_f64<InT>(src[i]);
  }
}

// E: weights per lane (g = 64 E); P: grid dimension; BITS: packed code width.
template <int E, int P, int BITS, typename InT>
__global__ __launch_bounds__(64 * kWaves) void quantize_kernel(
    const InT* __restrict__ w, int64_t rows, int64_t in, uint64_t seed,
    const float* __restrict__ grid, int n, uint8_t* __restrict__ codes, int64_t row_bytes,
    uint16_t* __restrict__ scales) {
  constexpr int G = 64 * E;
  constexpr int kVecPerLane = E / P;
  constexpr int kCodesPerGroup = G / P;
  constexpr int kWordsPerGroup = kCodesPerGroup * BITS / 32;
  static_assert(E % P == 0, "a lane must hold whole p-vectors");
  static_assert((kCodesPerGroup * BITS) % 32 == 0, "group must fill whole dwords");

  // grid point k: P coordinates then |G_k|^2 / 2 + shift (stride P + 1)
  __shared__ double s_grid[kMaxN * (P + 1)];
  __shared__ uint16_t s_codes[kWaves][kMaxG / P];

  const int lane = int(threadIdx.x) & 63;
  const int wave = int(threadIdx.x) >> 6;

  __shared__ double s_r2[kWaves];
  double r2 = 0.0;  // largest squared grid-point norm seen by this thread
  for (int k = int(threadIdx.x); k < n; k += 64 * kWaves) {
    double h = 0.0;
#pragma unroll
    for (int t = 0; t < P; ++t) {
      const double c = double(grid[k * P + t]);
      s_grid[k * (P + 1) + t] = c;
      h += c * c;
    }
    s_grid[k * (P + 1) + P] = 0.5 * h;
    r2 = fmax(r2, h);
  }
  r2 = wave_max(r2, int(threadIdx.x) & 63);
  if ((threadIdx.x & 63) == 0) s_r2[threadIdx.x >> 6] = r2;
  __syncthreads();
  for (int w = 0; w < kWaves; ++w) r2 = fmax(r2, s_r2[w]);
  // the search-value shift: a power of two at least twice the largest |c_k|
  const double bound = 2.0 * (0.5 * r2 + sqrt(double(64 * E)) * sqrt(r2));
  const double shift = bound <= kMinShift ? kMinShift : exp2(ceil(log2(bound)));
  for (int k = int(threadIdx.x); k < n; k += 64 * kWaves) s_grid[k * (P + 1) + P] += shift;

  uint64_t neg = 0;
#pragma unroll
  for (int i = 0; i < E; ++i) neg |= uint64_t(rht_sign_negative(seed, uint32_t(lane * E + i))) << i;

  const int64_t groups_per_row = in / G;
  const int64_t total = rows * groups_per_row;
  const double inv_sqrt_g = 1.0 / sqrt(double(G));
  __syncthreads();

  // Every wave of the block runs the same number of iterations (barriers).
  for (int64_t first = int64_t(blockIdx.x) * kWaves; first < total;
       first += int64_t(gridDim.x) * kWaves) {
    const int64_t grp = first + wave;
    const bool valid = grp < total;
    const int64_t row = valid ? grp / groups_per_row : 0;
    const int64_t gi = valid ? grp - row * groups_per_row : 0;

    double v[E];
    if (valid) {
      load_group<E, InT>(w + row * in + gi * G + lane * E, v);
    } else {
#pragma unroll
      for (int i = 0; i < E; ++i) v[i] = 0.0;
    }

    double ss = 0.0;
#pragma unroll
    for (int i = 0; i < E; ++i) ss += v[i] * v[i];
    ss = wave_sum(ss, lane);
    const double s = sqrt(ss);

#pragma unroll
    for (int i = 0; i < E; ++i) {
      const double u = s > 0.0 ? v[i] / s : 0.0;
      v[i] = ((neg >> i) & 1) ? -u : u;
    }
    fwht_wave<E>(v, lane, G);

    double best[kVecPerLane];
#pragma unroll
    for (int j = 0; j < kVecPerLane; ++j) best[j] = INFINITY;
    const uint32_t index_mask = kIndexMask;
    for (int k = 0; k < n; ++k) {
      double gk[P];
#pragma unroll
      for (int t = 0; t < P; ++t) gk[t] = s_grid[k * (P + 1) + t];
      const double hk = s_grid[k * (P + 1) + P];
#pragma unroll
      for (int j = 0; j < kVecPerLane; ++j) {
        double c = hk;
#pragma unroll
        for (int t = 0; t < P; ++t) c = fma(-v[j * P + t], gk[t], c);
        best[j] = min_indexed(best[j], c, uint32_t(k), index_mask);
      }
    }

#pragma unroll
    for (int j = 0; j < kVecPerLane; ++j)
      s_codes[wave][lane * kVecPerLane + j] =
          uint16_t(__builtin_bit_cast(uint64_t, best[j]) & kIndexMask);
    __syncthreads();

    if (valid) {
      uint32_t* dst = reinterpret_cast<uint32_t*>(codes + row * row_bytes +
                                                  gi * (int64_t(kCodesPerGroup) * BITS / 8));
      for (int wi = lane; wi < kWordsPerGroup; wi += 64) {
        const int bit0 = wi * 32;
        int c = bit0 / BITS;
        uint32_t word = uint32_t(s_codes[wave][c]) >> (bit0 - c * BITS);
        for (++c; c * BITS < bit0 + 32 && c < kCodesPerGroup; ++c)
          word |= uint32_t(s_codes[wave][c]) << (c * BITS - bit0);
        dst[wi] = word;
      }
      if (lane == 0) scales[row * groups_per_row + gi] = f64_to_f16_rne(s * inv_sqrt_g);
    }
    __syncthreads();
  }
}

// Quantization error of a layer, measured in the rotated space: the rotation
// R = H diag(sigma) / sqrt(g) is orthonormal, so per group (Parseval)
//   ||w - w_hat||^2 = || H (sigma * w) / sqrt(g) - scale * concat_j G[code_j] ||^2
// with w_hat the dequantised group (App. G). One wavefront per group writes
// that sum and ||w||^2 as two fp64 values (row-major group order); the layer's
// relative error t^2 (Sec. 3.4) is their ratio of sums. Codes are read from
// the packed row (LSB-first, `bits` per code, up to three bytes per code).
template <int E, int P, typename InT>
__global__ __launch_bounds__(64 * kWaves) void layer_error_kernel(
    const InT* __restrict__ w, int64_t rows, int64_t in, uint64_t seed,
    const float* __restrict__ grid, int bits, const uint8_t* __restrict__ codes, int64_t row_bytes,
    const uint16_t* __restrict__ scales, double* __restrict__ out) {
  constexpr int G = 64 * E;
  static_assert(E % P == 0, "a lane must hold whole p-vectors");
  const int lane = int(threadIdx.x) & 63;
  const int wave = int(threadIdx.x) >> 6;
  uint64_t neg = 0;
#pragma unroll
  for (int i = 0; i < E; ++i) neg |= uint64_t(rht_sign_negative(seed, uint32_t(lane * E + i))) << i;
  const int64_t groups_per_row = in / G;
  const int64_t total = rows * groups_per_row;
  const double inv_sqrt_g = 1.0 / sqrt(double(G));
  const uint32_t mask = (1u << bits) - 1u;
  // no barrier below: each wave walks its own groups
  for (int64_t grp = int64_t(blockIdx.x) * kWaves + wave; grp < total;
       grp += int64_t(gridDim.x) * kWaves) {
    const int64_t row = grp / groups_per_row;
    const int64_t gi = grp - row * groups_per_row;
    double v[E];
    load_group<E, InT>(w + row * in + gi * G + lane * E, v);
    double ss = 0.0;
#pragma unroll
    for (int i = 0; i < E; ++i) ss += v[i] * v[i];
    ss = wave_sum(ss, lane);
#pragma unroll
    for (int i = 0; i < E; ++i)
      if ((neg >> i) & 1) v[i] = -v[i];
    fwht_wave<E>(v, lane, G);
    const double sh = double(__builtin_bit_cast(_Float16, scales[row * groups_per_row + gi]));
    const uint8_t* crow = codes + row * row_bytes;
    double e = 0.0;
#pragma unroll
    for (int t = 0; t < E / P; ++t) {
      const int64_t m = gi * (G / P) + lane * (E / P) + t;  // code index in the row
      const int64_t bit = m * bits;
      const int64_t b0 = bit >> 3;
      uint32_t win = crow[b0];
      if (b0 + 1 < row_bytes) win |= uint32_t(crow[b0 + 1]) << 8;
      if (b0 + 2 < row_bytes) win |= uint32_t(crow[b0 + 2]) << 16;
      const uint32_t code = (win >> (bit & 7)) & mask;
#pragma unroll
      for (int c = 0; c < P; ++c) {
        const double d = v[t * P + c] * inv_sqrt_g - sh * double(grid[code * P + c]);
        e += d * d;
      }
    }
    e = wave_sum(e, lane);
    if (lane == 0) {
      out[2 * grp] = e;
      out[2 * grp + 1] = ss;
    }
  }
}

// t^2 = sum_q err_q / sum_q norm_q over the per-group pairs of
// layer_error_kernel (Sec. 3.4's relative error of the layer). One block:
// thread t adds the pairs t, t + 256, ... in order, then a fixed tree over
// the threads (deterministic). A layer of norm 0 gets t^2 = 0.
__global__ __launch_bounds__(256) void layer_t2_kernel(const double* __restrict__ pairs,
                                                       int64_t groups, double* __restrict__ t2) {
  __shared__ double s_e[256], s_n[256];
  const int tid = int(threadIdx.x);
  double e = 0.0, nrm = 0.0;
  for (int64_t q = tid; q < groups; q += 256) {
    e += pairs[2 * q];
    nrm += pairs[2 * q + 1];
  }
  s_e[tid] = e;
  s_n[tid] = nrm;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (tid < h) {
      s_e[tid] += s_e[tid + h];
      s_n[tid] += s_n[tid + h];
    }
    __syncthreads();
  }
  if (tid == 0) t2[0] = s_n[0] > 0.0 ? s_e[0] / s_n[0] : 0.0;
}

template <int P, typename InT>
hipError_t launch_error_p(const InT* w, int64_t out_rows, int64_t in, const float* grid, int bits,
                          int g, uint64_t seed, const uint8_t* codes, int64_t row_bytes,
                          const uint16_t* scales, double* err, hipStream_t stream) {
  const int64_t total = out_rows * (in / g);
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((total + kWaves - 1) / kWaves, 8192));
  const dim3 grid_dim{unsigned(blocks)}, block{64 * kWaves};
  switch (g) {
#define HIGGS_E_CASE(GV)                                                                     \
  case GV:                                                                                   \
    if constexpr ((GV / 64) % P == 0) {                                                      \
      hipLaunchKernelGGL((layer_error_kernel<GV / 64, P, InT>), grid_dim, block, 0, stream, \
                         w, out_rows, in, seed, grid, bits, codes, row_bytes, scales, err);  \
      return hipGetLastError();                                                              \
    }                                                                                        \
    break;
    HIGGS_E_CASE(64)
    HIGGS_E_CASE(128)
    HIGGS_E_CASE(256)
    HIGGS_E_CASE(512)
    HIGGS_E_CASE(1024)
    HIGGS_E_CASE(2048)
    HIGGS_E_CASE(4096)
#undef HIGGS_E_CASE
    default:
      break;
  }
  return hipErrorInvalidValue;
}

template <int P, int BITS, typename InT>
hipError_t launch_bits(const InT* w, int64_t out, int64_t in, const float* grid, int n, int g,
                       uint64_t seed, uint8_t* codes, int64_t row_bytes, uint16_t* scales,
                       hipStream_t stream) {
  const int64_t total = out * (in / g);
  const int64_t blocks = std::min<int64_t>((total + kWaves - 1) / kWaves, 8192);
  const dim3 grid_dim{unsigned(blocks)}, block{64 * kWaves};
  switch (g) {
#define HIGGS_Q_CASE(GV)                                                                     \
  case GV:                                                                                   \
    if constexpr ((GV / 64) % P == 0) {                                                      \
      hipLaunchKernelGGL((quantize_kernel<GV / 64, P, BITS, InT>), grid_dim, block, 0,       \
                         stream, w, out, in, seed, grid, n, codes, row_bytes, scales);       \
      return hipGetLastError();                                                              \
    }                                                                                        \
    break;
    HIGGS_Q_CASE(64)
    HIGGS_Q_CASE(128)
    HIGGS_Q_CASE(256)
    HIGGS_Q_CASE(512)
    HIGGS_Q_CASE(1024)
    HIGGS_Q_CASE(2048)
    HIGGS_Q_CASE(4096)
#undef HIGGS_Q_CASE
    default:
      break;
  }
  return hipErrorInvalidValue;
}

template <typename InT>
hipError_t launch_typed(const InT* w, int64_t out, int64_t in, const float* grid, int p, int n,
                        int g, uint64_t seed, uint8_t* codes, uint16_t* scales,
                        hipStream_t stream) {
  const int bits = code_bits(p, n);
  const int64_t row_bytes = in / p * bits / 8;
  if (p == 1 && bits == 4)
    return launch_bits<1, 4>(w, out, in, grid, n, g, seed, codes, row_bytes, scales, stream);
  if (p == 1 && bits == 8)
    return launch_bits<1, 8>(w, out, in, grid, n, g, seed, codes, row_bytes, scales, stream);
  if (p == 2 && bits == 6)
    return launch_bits<2, 6>(w, out, in, grid, n, g, seed, codes, row_bytes, scales, stream);
  if (p == 2 && bits == 8)
    return launch_bits<2, 8>(w, out, in, grid, n, g, seed, codes, row_bytes, scales, stream);
  if (p == 2 && bits == 10)
    return launch_bits<2, 10>(w, out, in, grid, n, g, seed, codes, row_bytes, scales, stream);
  return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// GPTQ rounding in place of the nearest-point step (Sec. 3.5), in the rotated
// space: W' = per group H (sigma * w) / sqrt(g), the Hessian of the rotated
// calibration activations, U the upper Cholesky factor of its damped inverse
// (Hinv = U^T U). Columns are taken in order, one p-vector at a time: its
// rotated weights v are rounded like Alg. 1 (nearest grid point of
// v sqrt(g) / s, s the group's norm), the error e = v - (s / sqrt(g)) G[q] is
// scaled, E = e U_pp^-1 (U_pp the p x p diagonal block), and later columns
// move by -E U[p-vector, later]. Within a block of 64 columns the update runs
// here, one wavefront per row (lane j holds column c0 + j); the block's E go
// to `err` and the columns after the block are updated by one GEMM.
// ---------------------------------------------------------------------------

// Rotated weights W' (fp64), each group's norm s (fp64) and the stored scale
// fp16(s / sqrt(g)). One wavefront per group.
template <int E, typename InT>
__global__ __launch_bounds__(64 * kWaves) void gptq_prepare_kernel(
    const InT* __restrict__ w, int64_t rows, int64_t in, uint64_t seed, double* __restrict__ wr,
    double* __restrict__ norms, uint16_t* __restrict__ scales) {
  constexpr int G = 64 * E;
  const int lane = int(threadIdx.x) & 63;
  const int wave = int(threadIdx.x) >> 6;
  uint64_t neg = 0;
#pragma unroll
  for (int i = 0; i < E; ++i) neg |= uint64_t(rht_sign_negative(seed, uint32_t(lane * E + i))) << i;
  const int64_t groups_per_row = in / G;
  const int64_t total = rows * groups_per_row;
  const double inv_sqrt_g = 1.0 / sqrt(double(G));
  for (int64_t grp = int64_t(blockIdx.x) * kWaves + wave; grp < total;
       grp += int64_t(gridDim.x) * kWaves) {
    const int64_t row = grp / groups_per_row;
    const int64_t gi = grp - row * groups_per_row;
    double v[E];
    load_group<E, InT>(w + row * in + gi * G + lane * E, v);
    double ss = 0.0;
#pragma unroll
    for (int i = 0; i < E; ++i) ss += v[i] * v[i];
    ss = wave_sum(ss, lane);
    const double sn = sqrt(ss);
#pragma unroll
    for (int i = 0; i < E; ++i)
      if ((neg >> i) & 1) v[i] = -v[i];
    fwht_wave<E>(v, lane, G);
    double* dst = wr + row * in + gi * G + lane * E;
#pragma unroll
    for (int i = 0; i < E; ++i) dst[i] = v[i] * inv_sqrt_g;
    if (lane == 0) {
      norms[grp] = sn;
      scales[grp] = f64_to_f16_rne(sn * inv_sqrt_g);
    }
  }
}

__device__ inline double readlane_f64(double v, int l) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(u)), l));
  const uint32_t hi = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(u >> 32)), l));
  return __builtin_bit_cast(double, uint64_t(lo) | (uint64_t(hi) << 32));
}

// One block of 64 columns [c0, c0 + 64) for every row (one wavefront per row).
template <int P>
__global__ __launch_bounds__(64 * kWaves) void gptq_block_kernel(
    const double* __restrict__ wr, const double* __restrict__ norms,
    const double* __restrict__ u, const float* __restrict__ grid, int n, int64_t rows,
    int64_t in, int log2g, int64_t c0, int bits, uint8_t* __restrict__ codes, int64_t row_bytes,
    double* __restrict__ err) {
  constexpr int kB = 64;
  constexpr int kVecs = kB / P;
  __shared__ double s_u[kB][kB + 1];
  __shared__ double s_grid[kMaxN * (P + 1)];
  __shared__ uint16_t s_codes[kWaves][kVecs];
  const int tid = int(threadIdx.x);
  const int lane = tid & 63;
  const int wave = tid >> 6;
  for (int i = tid; i < kB * kB; i += 64 * kWaves) {
    const int r = i / kB, c = i % kB;
    s_u[r][c] = c >= r ? u[(c0 + r) * in + c0 + c] : 0.0;  // upper triangle only
  }
  for (int k = tid; k < n; k += 64 * kWaves) {
    double h = 0.0;
#pragma unroll
    for (int t = 0; t < P; ++t) {
      const double c = double(grid[k * P + t]);
      s_grid[k * (P + 1) + t] = c;
      h += c * c;
    }
    s_grid[k * (P + 1) + P] = 0.5 * h;
  }
  __syncthreads();
  const int64_t row = int64_t(blockIdx.x) * kWaves + wave;
  if (row >= rows) return;  // no barrier below
  const int g = 1 << log2g;
  const double sn = norms[row * (in >> log2g) + (c0 >> log2g)];  // the block is in one group
  const double fwd = sn > 0.0 ? sqrt(double(g)) / sn : 0.0;      // W' -> grid units
  const double back = sn / sqrt(double(g));                      // grid units -> W'
  double wv = wr[row * in + c0 + lane];
  double my_err = 0.0;
  for (int t = 0; t < kVecs; ++t) {
    double v[P], uv[P];
#pragma unroll
    for (int k = 0; k < P; ++k) {
      v[k] = readlane_f64(wv, t * P + k);
      uv[k] = v[k] * fwd;
    }
    // nearest grid point: lane l scans candidates l, l + 64, ...; then the
    // wave keeps the least (c, index) pair (lowest index on ties)
    double best = INFINITY;
    int bk = 0;
    for (int k = lane; k < n; k += 64) {
      double c = s_grid[k * (P + 1) + P];
#pragma unroll
      for (int d = 0; d < P; ++d) c = fma(-uv[d], s_grid[k * (P + 1) + d], c);
      if (c < best) {
        best = c;
        bk = k;
      }
    }
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) {
      const double ob = __shfl_xor(best, m, 64);
      const int ok = __shfl_xor(bk, m, 64);
      if (ob < best || (ob == best && ok < bk)) {
        best = ob;
        bk = ok;
      }
    }
    const int q = __builtin_amdgcn_readfirstlane(bk);
    double e[P], es[P];
#pragma unroll
    for (int k = 0; k < P; ++k) e[k] = v[k] - back * s_grid[q * (P + 1) + k];
    // E = e U_pp^-1 (U_pp upper triangular)
    const int i0 = t * P;
    if constexpr (P == 1) {
      es[0] = e[0] / s_u[i0][i0];
    } else {
      es[0] = e[0] / s_u[i0][i0];
      es[1] = (e[1] - es[0] * s_u[i0][i0 + 1]) / s_u[i0 + 1][i0 + 1];
    }
    if (lane >= i0 + P) {
#pragma unroll
      for (int k = 0; k < P; ++k) wv = fma(-es[k], s_u[i0 + k][lane], wv);
    }
#pragma unroll
    for (int k = 0; k < P; ++k)
      if (lane == i0 + k) my_err = es[k];
    if (lane == 0) s_codes[wave][t] = uint16_t(q);
  }
  err[row * kB + lane] = my_err;
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  // pack the block's codes: kVecs * bits bits, whole dwords
  const int words = kVecs * bits / 32;
  uint32_t* dst = reinterpret_cast<uint32_t*>(codes + row * row_bytes + (c0 / P) * bits / 8);
  if (lane < words) {
    const int bit0 = lane * 32;
    int c = bit0 / bits;
    uint32_t word = uint32_t(s_codes[wave][c]) >> (bit0 - c * bits);
    for (++c; c * bits < bit0 + 32 && c < kVecs; ++c)
      word |= uint32_t(s_codes[wave][c]) << (c * bits - bit0);
    dst[lane] = word;
  }
}

__global__ void f32_to_f64_kernel(const float* __restrict__ src, int64_t count,
                                  double* __restrict__ dst) {
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < count;
       i += int64_t(gridDim.x) * 256)
    dst[i] = double(src[i]);
}

// h[i][i] += damp * mean_i h[i][i] (one block; the mean is summed in a fixed
// order: each thread a strided partial, then thread 0 over the partials)
__global__ __launch_bounds__(256) void damp_diag_kernel(double* __restrict__ h, int64_t in,
                                                        double damp) {
  __shared__ double s_part[256];
  double sum = 0.0;
  for (int64_t i = threadIdx.x; i < in; i += 256) sum += h[i * in + i];
  s_part[threadIdx.x] = sum;
  __syncthreads();
  __shared__ double s_add;
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int k = 0; k < 256; ++k) t += s_part[k];
    s_add = damp * t / double(in);
  }
  __syncthreads();
  for (int64_t i = threadIdx.x; i < in; i += 256) h[i * in + i] += s_add;
}

}  // namespace

hipError_t launch_gptq_prepare(const void* w, higgs_dtype dtype, int64_t out, int64_t in, int g,
                               uint64_t seed, double* wr, double* norms, uint16_t* scales,
                               hipStream_t stream) {
  const int64_t total = out * (in / g);
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((total + kWaves - 1) / kWaves, 8192));
  switch (g) {
#define HIGGS_G_CASE(GV)                                                                        \
  case GV:                                                                                      \
    if (dtype == HIGGS_F32)                                                                     \
      hipLaunchKernelGGL((gptq_prepare_kernel<GV / 64, float>), dim3(unsigned(blocks)),        \
                         dim3(64 * kWaves), 0, stream, static_cast<const float*>(w), out, in,  \
                         seed, wr, norms, scales);                                              \
    else                                                                                        \
      hipLaunchKernelGGL((gptq_prepare_kernel<GV / 64, uint16_t>), dim3(unsigned(blocks)),     \
                         dim3(64 * kWaves), 0, stream, static_cast<const uint16_t*>(w), out,   \
                         in, seed, wr, norms, scales);                                          \
    return hipGetLastError();
    HIGGS_G_CASE(64)
    HIGGS_G_CASE(128)
    HIGGS_G_CASE(256)
    HIGGS_G_CASE(512)
    HIGGS_G_CASE(1024)
    HIGGS_G_CASE(2048)
    HIGGS_G_CASE(4096)
#undef HIGGS_G_CASE
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_gptq_block(const double* wr, const double* norms, const double* u,
                             const float* grid, int p, int n, int64_t out, int64_t in, int g,
                             int64_t c0, uint8_t* codes, double* err, hipStream_t stream) {
  const int bits = code_bits(p, n);
  const int64_t row_bytes = in / p * bits / 8;
  const dim3 grid_dim{unsigned((out + kWaves - 1) / kWaves)}, block{64 * kWaves};
  if (p == 1)
    hipLaunchKernelGGL((gptq_block_kernel<1>), grid_dim, block, 0, stream, wr, norms, u, grid, n,
                       out, in, log2_exact(g), c0, bits, codes, row_bytes, err);
  else
    hipLaunchKernelGGL((gptq_block_kernel<2>), grid_dim, block, 0, stream, wr, norms, u, grid, n,
                       out, in, log2_exact(g), c0, bits, codes, row_bytes, err);
  return hipGetLastError();
}

hipError_t launch_to_f64(const float* src, int64_t count, double* dst, hipStream_t stream) {
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((count + 255) / 256, 8192));
  hipLaunchKernelGGL(f32_to_f64_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream, src, count,
                     dst);
  return hipGetLastError();
}

hipError_t launch_damp_diag(double* h, int64_t in, double damp, hipStream_t stream) {
  hipLaunchKernelGGL(damp_diag_kernel, dim3(1), dim3(256), 0, stream, h, in, damp);
  return hipGetLastError();
}

hipError_t launch_layer_error(const void* w, higgs_dtype dtype, int64_t out, int64_t in,
                              const uint8_t* codes, const uint16_t* scales, const float* grid,
                              int p, int n, int g, uint64_t seed, double* err, double* t2,
                              hipStream_t stream) {
  const int bits = code_bits(p, n);
  const int64_t row_bytes = in / p * bits / 8;
  hipError_t st;
  if (dtype == HIGGS_F32) {
    const float* wf = static_cast<const float*>(w);
    st = p == 1 ? launch_error_p<1>(wf, out, in, grid, bits, g, seed, codes, row_bytes, scales,
                                    err, stream)
                : launch_error_p<2>(wf, out, in, grid, bits, g, seed, codes, row_bytes, scales,
                                    err, stream);
  } else {
    const uint16_t* wb = static_cast<const uint16_t*>(w);
    st = p == 1 ? launch_error_p<1>(wb, out, in, grid, bits, g, seed, codes, row_bytes, scales,
                                    err, stream)
                : launch_error_p<2>(wb, out, in, grid, bits, g, seed, codes, row_bytes, scales,
                                    err, stream);
  }
  if (st != hipSuccess || t2 == nullptr) return st;
  hipLaunchKernelGGL(layer_t2_kernel, dim3(1), dim3(256), 0, stream, err, out * (in / g), t2);
  return hipGetLastError();
}

hipError_t launch_quantize(const void* w, higgs_dtype dtype, int64_t out, int64_t in,
                           const float* grid, int p, int n, int g, uint64_t seed, uint8_t* codes,
                           uint16_t* scales, hipStream_t stream) {
  if (dtype == HIGGS_F32)
    return launch_typed(static_cast<const float*>(w), out, in, grid, p, n, g, seed, codes, scales,
                        stream);
  return launch_typed(static_cast<const uint16_t*>(w), out, in, grid, p, n, g, seed, codes, scales,
                      stream);
}

}  // namespace higgs
