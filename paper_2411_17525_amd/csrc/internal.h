// Internal declarations shared by the library's host code and HIP kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/higgs.h"

namespace higgs {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// 16-byte streaming load (non-temporal hint: the data is read once).
__device__ inline u32x4 load_stream16(const void* p) {
  return __builtin_nontemporal_load(static_cast<const u32x4*>(p));
}

// Output j (0-based) of splitmix64 started at state `seed` (Steele, Lea &
// Flood 2014). The generator is counter based: output j mixes
// seed + (j + 1) * 0x9E3779B97F4A7C15.
__host__ __device__ inline uint64_t splitmix64_at(uint64_t seed, uint64_t j) {
  uint64_t z = seed + (j + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// True when sigma_j = -1: the top bit of output j is set.
__host__ __device__ inline bool rht_sign_negative(uint64_t seed, uint32_t j) {
  return (splitmix64_at(seed, j) >> 63) != 0;
}

// Waits once for all the scalar values given (kernel arguments read at the
// top of a kernel): their reads, placed before this statement, are requested
// together, in one round trip to the argument buffer. Left to itself the
// compiler turns a per-layer select into an indexed read whose address
// depends on an earlier read, and defers other reads behind that chain. One
// such statement per kernel: each bounds the scheduler's regions.
#define HIGGS_READ_NOW(...) asm volatile("" ::__VA_ARGS__)
// Holds the integer values given in scalar registers from this point on, as
// values the compiler cannot read again from the argument buffer (it prefers
// re-reading an argument to keeping a register, and each read waits a round
// trip). Integers and floats only: a pointer passed through it loses its
// address space, and loads through it become flat loads.
#define HIGGS_HOLD(...) asm volatile("" : __VA_ARGS__)

inline int log2_exact(int64_t v) {
  if (v <= 0 || (v & (v - 1)) != 0) return -1;
  int l = 0;
  while ((int64_t(1) << l) < v) ++l;
  return l;
}

// Bits per packed code for a supported grid; 0 if (p, n) is not supported.
inline int code_bits(int p, int n) {
  if (p == 1 && n == 16) return 4;
  if (p == 1 && n == 256) return 8;  // CH8: uniform scalar grid, one weight per code
  if (p == 2 && n == 64) return 6;
  if (p == 2 && n == 256) return 8;
  if (p == 2 && n == 1024) return 10;
  return 0;
}

// ---- host grids (grid_lloyd.cpp) ----
int lloyd_grid(int p, int n, uint64_t seed, int64_t num_samples, int max_iters,
               double* grid_out, double* mse_out, int* iters_out);
// Symmetric uniform n-point grid minimising the mean squared error of N(0, 1).
void uniform_grid(int n, double* grid_out, double* step_out, double* mse_out);

// ---- kernel launchers (return the launch status) ----
hipError_t launch_rht_activations(const void* x, higgs_dtype dtype, int64_t batch, int64_t in,
                                  int g, uint64_t seed, float* x_rot, hipStream_t stream);

hipError_t launch_quantize(const void* w, higgs_dtype dtype, int64_t out, int64_t in,
                           const float* grid, int p, int n, const void* index, int g,
                           uint64_t seed, uint8_t* codes, uint16_t* scales, hipStream_t stream);
// The nearest-point search index of a grid (encode.hip): its size in bytes
// and its build (two kernels on `stream`).
int64_t search_index_bytes(int p, int n);
hipError_t launch_search_index(const float* grid, int p, int n, void* index, hipStream_t stream);

// Per-group [err, norm] of a quantized layer (rotated-space error, fp64);
// with t2 != NULL also t^2 = sum(err) / sum(norm) into t2[0] (device).
hipError_t launch_layer_error(const void* w, higgs_dtype dtype, int64_t out, int64_t in,
                              const uint8_t* codes, const uint16_t* scales, const float* grid,
                              int p, int n, int g, uint64_t seed, double* err, double* t2,
                              hipStream_t stream);

// GPTQ rounding (encode.hip kernels, gptq.cpp orchestration).
hipError_t launch_gptq_prepare(const void* w, higgs_dtype dtype, int64_t out, int64_t in, int g,
                               uint64_t seed, double* wr, double* norms, uint16_t* scales,
                               hipStream_t stream);
hipError_t launch_gptq_block(const double* wr, const double* norms, const double* u,
                             const float* grid, int p, int n, int64_t out, int64_t in, int g,
                             int64_t c0, uint8_t* codes, double* err, hipStream_t stream);
hipError_t launch_to_f64(const float* src, int64_t count, double* dst, hipStream_t stream);
hipError_t launch_damp_diag(double* h, int64_t in, double damp, hipStream_t stream);
// Host orchestration; return a higgs_status and fill msg on failure.
int gptq_factor(const float* x_rot, int64_t samples, int64_t in, double damp, double* factor,
                void* workspace, hipStream_t stream, char* msg, int msg_len);
int gptq_quantize(const void* w, higgs_dtype dtype, int64_t out, int64_t in, const float* grid,
                  int p, int n, int g, uint64_t seed, const double* factor, uint8_t* codes,
                  uint16_t* scales, void* workspace, hipStream_t stream, char* msg, int msg_len);
int64_t gptq_factor_workspace_bytes(int64_t samples, int64_t in);
int64_t gptq_quantize_workspace_bytes(int64_t out, int64_t in, int g);

// Exact per-layer choice of quantizers under an average-bits budget
// (bitwidth.cpp); returns a higgs_status and fills msg on failure.
int allocate_bits(int layers, int options, const double* alpha, const double* t2,
                  const double* bits, const int64_t* sizes, double b_max, int32_t* choice,
                  double* objective, double* avg_bits, char* msg, int msg_len);

hipError_t launch_qgemv(const float* x_rot, int64_t batch, const uint8_t* codes,
                        const uint16_t* scales, const float* grid, int p, int n, int g,
                        int64_t out, int64_t in, float* y, hipStream_t stream);

// Same product from raw activations: the rotation is applied while the
// activations are converted (only when qgemv_rotates(p, n, g)).
hipError_t launch_qgemv_rotating(const void* x, int x_bf16, uint64_t seed, int64_t batch,
                                 const uint8_t* codes, const uint16_t* scales, const float* grid,
                                 int p, int n, int g, int64_t out, int64_t in, float* y,
                                 hipStream_t stream);

// Up to qgemv_max_layers() layers that read the same raw activations (same
// in, grid and g; own codes, scales, rows, seed and output) in one launch.
hipError_t launch_qgemv_rotating_group(const void* x, int x_bf16, int layers,
                                       const uint64_t* seeds, int64_t batch,
                                       const uint8_t* const* codes, const uint16_t* const* scales,
                                       const float* grid, int p, int n, int g, const int64_t* outs,
                                       int64_t in, float* const* y, hipStream_t stream);
int qgemv_max_layers();

// Largest input dimension the small-batch kernel handles for this grid.
int64_t qgemv_max_in(int p, int n);
// True when a rotation group fits inside one wave's slice of the small-batch
// kernel, so that it can rotate raw activations itself.
bool qgemv_rotates(int p, int n, int g);

// Matrix-core path (batch >= qgemm_min_batch). The activations are converted
// once into the workspace (kind: already rotated fp32, or raw fp32 / bf16
// rotated on the way with the seed's signs).
constexpr int kQgemmRotated = 0;
constexpr int kQgemmRawF32 = 1;
constexpr int kQgemmRawBF16 = 2;
int64_t qgemm_workspace_bytes(int64_t batch, int64_t out, int64_t in, int p, int n, int g);
hipError_t launch_qgemm(const void* x, int x_kind, uint64_t seed, int64_t batch,
                        const uint8_t* codes, const uint16_t* scales, const float* grid, int p,
                        int n, int g, int64_t out, int64_t in, float* y, void* workspace,
                        hipStream_t stream);

// Up to 4 layers that read the same activations (own codes, scales, rows,
// seed and output) in one activation conversion, one product launch and at
// most one reduction launch per 64 batch rows.
int64_t qgemm_group_workspace_bytes(int layers, int64_t batch, const int64_t* outs, int64_t in,
                                    int p, int n, int g);
hipError_t launch_qgemm_group(const void* x, int x_kind, int layers, const uint64_t* seeds,
                              int64_t batch, const uint8_t* const* codes,
                              const uint16_t* const* scales, const float* grid, int p, int n,
                              int g, const int64_t* outs, int64_t in, float* const* y,
                              void* workspace, hipStream_t stream);

// The library's fixed device scratch (scratch.hip): its device address on
// the current device, resolved once per device (hipGetSymbolAddress).
constexpr int64_t kScratchBytes = HIGGS_NOALLOC_SCRATCH_BYTES;
hipError_t scratch_buffer(void** ptr);

// Code formats the matrix-core kernel reads: grid-point pairs with 6-, 8- or
// 10-bit codes, the scalar 16-point grid read as pairs, and the scalar
// 256-point grid (CH8).
inline bool qgemm_format(int p, int n) {
  if (p == 1) return n == 16 || n == 256;
  return p == 2 && (n == 64 || n == 256 || n == 1024);
}

// Smallest batch at which the matrix-core path replaces the small-batch
// kernel, from launch times measured on MI355X over the Llama-3.1-8B layer
// shapes: the small-batch kernel's time grows with the batch (one v_dot2 per
// code and batch row; for 8-bit pair codes the 4x4x4 matrix variant with
// batch tiles of 4 and 8; a new launch per batch tile), the matrix-core
// product's is nearly flat up to 16 rows (one 16-column tile, g >= 128).
// With g >= 128: batch 5 on rows of up to 8192 weights; on longer rows
// (where the small-batch kernel is slower per row) batch 2 for 8-bit pair
// codes and 3 for the others. With g = 64 (p = 1 only) the matrix-core
// product uses a 32-column tile and takes over later: batch 9, or on longer
// rows 5 for the 16-point grid and 7 for CH8.
inline int64_t qgemm_min_batch(int p, int n, int64_t in, int g) {
  const bool long_rows = in > 8192;
  const bool pairs8 = (p == 2 && n == 256) || (p == 1 && n == 16);
  if (g >= 128) return long_rows ? (pairs8 ? 2 : 3) : 5;
  if (pairs8) return long_rows ? 5 : 9;
  return long_rows ? 7 : 9;
}

// True when higgs_qmatmul takes the matrix-core path for these arguments.
inline bool use_qgemm(int64_t batch, int p, int n, int64_t in, int g) {
  return qgemm_format(p, n) && batch >= qgemm_min_batch(p, n, in, g);
}

}  // namespace higgs
