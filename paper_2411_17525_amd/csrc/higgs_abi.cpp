// C ABI entry points: argument validation on the host, then kernel launches.
// Nothing here calls the HIP runtime before the arguments have been checked,
// and the host-only entry points (grid, signs, sizes) never touch it.

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

#include "internal.h"

namespace {

thread_local std::string g_last_error;

higgs_status fail(higgs_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

higgs_status ok() {
  g_last_error.clear();
  return HIGGS_OK;
}

higgs_status device_status(hipError_t err, const char* what) {
  if (err == hipSuccess) return ok();
  return fail(HIGGS_ERR_DEVICE, "%s: %s", what, hipGetErrorString(err));
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Shared checks of the grid / group configuration used by quantize and qmatmul.
higgs_status check_layer(int p, int n, int g, int64_t out, int64_t in) {
  if (out < 1 || in < 1) return fail(HIGGS_ERR_INVALID_ARG, "out (%lld) and in (%lld) must be >= 1",
                                     (long long)out, (long long)in);
  if (higgs::log2_exact(g) < 0)
    return fail(HIGGS_ERR_INVALID_ARG, "g (%d) must be a power of two", g);
  if (p < 1 || n < 2) return fail(HIGGS_ERR_INVALID_ARG, "invalid grid (p=%d, n=%d)", p, n);
  if (higgs::code_bits(p, n) == 0)
    return fail(HIGGS_ERR_UNSUPPORTED,
                "grid (p=%d, n=%d) not supported: use (1,16), (1,256), (2,64), (2,256) or (2,1024)",
                p, n);
  if (g < 64 * p || g > 4096)
    return fail(HIGGS_ERR_UNSUPPORTED, "g=%d not supported for p=%d: need %d <= g <= 4096", g, p,
                64 * p);
  if (in % g != 0)
    return fail(HIGGS_ERR_INVALID_ARG, "in (%lld) must be a multiple of g (%d)", (long long)in, g);
  // the kernels address codes and scales with 32-bit byte offsets
  if (out * (in / p) * higgs::code_bits(p, n) / 8 >= (int64_t(1) << 31) ||
      out * (in / g) * 2 >= (int64_t(1) << 31))
    return fail(HIGGS_ERR_UNSUPPORTED, "layer too large: codes and scales must each be < 2 GiB");
  return HIGGS_OK;
}

}  // namespace

// Limits of the product kernels beyond check_layer: the small-batch kernel
// keeps a wave's activations in registers, which bounds the input dimension.
static higgs_status check_product(int64_t batch, int p, int n, int64_t in, int g) {
  // the matrix-core path addresses a 64-row chunk of fp16 activations with
  // 32-bit byte offsets
  if (higgs::use_qgemm(batch, p, n, in, g) && in > (int64_t(1) << 23))
    return fail(HIGGS_ERR_UNSUPPORTED, "in (%lld) above 2^23 is not supported at batch %lld",
                (long long)in, (long long)batch);
  if (!higgs::use_qgemm(batch, p, n, in, g) && in > higgs::qgemv_max_in(p, n))
    return fail(HIGGS_ERR_UNSUPPORTED,
                "in (%lld) above %lld is not supported for grid (p=%d, n=%d) at batch %lld",
                (long long)in, (long long)higgs::qgemv_max_in(p, n), p, n, (long long)batch);
  return HIGGS_OK;
}

extern "C" {

int higgs_abi_version(void) { return 3; }

const char* higgs_last_error(void) { return g_last_error.c_str(); }

higgs_status higgs_make_grid(int p, int n, uint64_t seed, int64_t num_samples, int max_iters,
                             float* grid, double* mse_per_dim, int* iters_done) {
  if (grid == nullptr) return fail(HIGGS_ERR_INVALID_ARG, "grid must not be NULL");
  if (p < 1 || p > 2) return fail(HIGGS_ERR_UNSUPPORTED, "p=%d not supported (1 or 2)", p);
  if (n < 2 || n > 4096) return fail(HIGGS_ERR_INVALID_ARG, "n=%d outside [2, 4096]", n);
  if (num_samples < n || num_samples > (int64_t(1) << 28))
    return fail(HIGGS_ERR_INVALID_ARG, "num_samples=%lld must be in [n, 2^28]",
                (long long)num_samples);
  if (max_iters < 0) return fail(HIGGS_ERR_INVALID_ARG, "max_iters must be >= 0");
  std::vector<double> g(size_t(n) * p);
  double mse = 0.0;
  int iters = 0;
  try {
    higgs::lloyd_grid(p, n, seed, num_samples, max_iters, g.data(), &mse, &iters);
  } catch (...) {
    return fail(HIGGS_ERR_DEVICE, "host allocation failed in higgs_make_grid");
  }
  for (size_t i = 0; i < g.size(); ++i) grid[i] = float(g[i]);
  if (mse_per_dim) *mse_per_dim = mse;
  if (iters_done) *iters_done = iters;
  return ok();
}

higgs_status higgs_make_uniform_grid(int n, float* grid, double* step, double* mse) {
  if (grid == nullptr) return fail(HIGGS_ERR_INVALID_ARG, "grid must not be NULL");
  if (n < 2 || n > 4096) return fail(HIGGS_ERR_INVALID_ARG, "n=%d outside [2, 4096]", n);
  std::vector<double> g;
  try {
    g.resize(size_t(n));
  } catch (...) {
    return fail(HIGGS_ERR_DEVICE, "host allocation failed in higgs_make_uniform_grid");
  }
  double st = 0.0, m = 0.0;
  higgs::uniform_grid(n, g.data(), &st, &m);
  for (int k = 0; k < n; ++k) grid[k] = float(g[size_t(k)]);
  if (step) *step = st;
  if (mse) *mse = m;
  return ok();
}

higgs_status higgs_rht_signs(uint64_t seed, int g, int8_t* signs) {
  if (signs == nullptr) return fail(HIGGS_ERR_INVALID_ARG, "signs must not be NULL");
  if (higgs::log2_exact(g) < 0 || g > 4096)
    return fail(HIGGS_ERR_INVALID_ARG, "g (%d) must be a power of two <= 4096", g);
  for (int j = 0; j < g; ++j) signs[j] = higgs::rht_sign_negative(seed, uint32_t(j)) ? -1 : 1;
  return ok();
}

int64_t higgs_codes_row_bytes(int64_t in, int p, int n) {
  const int b = higgs::log2_exact(n);
  if (in < 1 || p < 1 || b < 1 || in % p != 0) return -1;
  const int64_t bits = in / p * b;
  if (bits % 8 != 0) return -1;
  return bits / 8;
}

int64_t higgs_qmatmul_workspace_bytes(int64_t batch, int64_t out, int64_t in, int p, int n,
                                      int g) {
  if (batch < 1 || check_layer(p, n, g, out, in) != HIGGS_OK) return -1;
  if (higgs::use_qgemm(batch, p, n, in, g)) return higgs::qgemm_workspace_bytes(batch, out, in, p, n, g);
  return 0;
}

int64_t higgs_search_index_bytes(int p, int n) {
  if (p < 1 || n < 2 || higgs::code_bits(p, n) == 0) return -1;
  return higgs::search_index_bytes(p, n);
}

higgs_status higgs_search_index(const float* grid, int p, int n, void* index,
                                int64_t index_bytes, void* stream) {
  if (!grid || !index) return fail(HIGGS_ERR_INVALID_ARG, "grid and index must not be NULL");
  if (p < 1 || n < 2 || higgs::code_bits(p, n) == 0)
    return fail(HIGGS_ERR_UNSUPPORTED,
                "grid (p=%d, n=%d) not supported: use (1,16), (1,256), (2,64), (2,256) or (2,1024)",
                p, n);
  if (index_bytes < higgs::search_index_bytes(p, n))
    return fail(HIGGS_ERR_INVALID_ARG, "index too small: %lld bytes needed",
                (long long)higgs::search_index_bytes(p, n));
  if (!aligned(index, 16) || !aligned(grid, 4))
    return fail(HIGGS_ERR_INVALID_ARG, "index must be 16-byte aligned, grid 4");
  const hipError_t err =
      higgs::launch_search_index(grid, p, n, index, static_cast<hipStream_t>(stream));
  return device_status(err, "higgs_search_index launch");
}

higgs_status higgs_quantize(const void* W, higgs_dtype w_dtype, int64_t out, int64_t in,
                            const float* grid, int p, int n, const void* index,
                            int64_t index_bytes, int g, uint64_t rht_seed, uint8_t* codes,
                            uint16_t* scales, void* stream) {
  if (!W || !grid || !codes || !scales)
    return fail(HIGGS_ERR_INVALID_ARG, "W, grid, codes and scales must not be NULL");
  if (w_dtype != HIGGS_F32 && w_dtype != HIGGS_BF16)
    return fail(HIGGS_ERR_INVALID_ARG, "w_dtype must be HIGGS_F32 or HIGGS_BF16");
  const higgs_status st = check_layer(p, n, g, out, in);
  if (st != HIGGS_OK) return st;
  if (!aligned(W, 16) || !aligned(codes, 16) || !aligned(scales, 2) || !aligned(grid, 4))
    return fail(HIGGS_ERR_INVALID_ARG, "W and codes must be 16-byte aligned, scales 2, grid 4");
  if (index != nullptr &&
      (index_bytes < higgs::search_index_bytes(p, n) || !aligned(index, 16)))
    return fail(HIGGS_ERR_INVALID_ARG,
                "index must be 16-byte aligned and hold at least %lld bytes (or be NULL)",
                (long long)higgs::search_index_bytes(p, n));
  const hipError_t err =
      higgs::launch_quantize(W, w_dtype, out, in, grid, p, n, index, g, rht_seed, codes, scales,
                             static_cast<hipStream_t>(stream));
  return device_status(err, "higgs_quantize launch");
}

higgs_status higgs_layer_error(const void* W, higgs_dtype w_dtype, int64_t out, int64_t in,
                               const uint8_t* codes, const uint16_t* scales, const float* grid,
                               int p, int n, int g, uint64_t rht_seed, double* group_err,
                               double* t2, void* stream) {
  if (!W || !codes || !scales || !grid || !group_err)
    return fail(HIGGS_ERR_INVALID_ARG, "W, codes, scales, grid and group_err must not be NULL");
  if (w_dtype != HIGGS_F32 && w_dtype != HIGGS_BF16)
    return fail(HIGGS_ERR_INVALID_ARG, "w_dtype must be HIGGS_F32 or HIGGS_BF16");
  const higgs_status st = check_layer(p, n, g, out, in);
  if (st != HIGGS_OK) return st;
  if (!aligned(W, 16) || !aligned(scales, 2) || !aligned(grid, 4) || !aligned(group_err, 8) ||
      !aligned(t2, 8))
    return fail(HIGGS_ERR_INVALID_ARG,
                "W must be 16-byte aligned, group_err and t2 8, grid 4, scales 2");
  const hipError_t err =
      higgs::launch_layer_error(W, w_dtype, out, in, codes, scales, grid, p, n, g, rht_seed,
                                group_err, t2, static_cast<hipStream_t>(stream));
  return device_status(err, "higgs_layer_error launch");
}

int64_t higgs_gptq_factor_workspace_bytes(int64_t samples, int64_t in) {
  if (samples < 1 || in < 64 || in % 64 != 0) return -1;
  return higgs::gptq_factor_workspace_bytes(samples, in);
}

higgs_status higgs_gptq_factor(const float* x_rot, int64_t samples, int64_t in, double damp,
                               double* factor, void* workspace, int64_t workspace_bytes,
                               void* stream) {
  if (!x_rot || !factor || !workspace)
    return fail(HIGGS_ERR_INVALID_ARG, "x_rot, factor and workspace must not be NULL");
  if (samples < 1 || in < 64 || in % 64 != 0 || in > 65536)
    return fail(HIGGS_ERR_INVALID_ARG, "need samples >= 1 and in a multiple of 64 in [64, 65536]");
  if (samples * in >= (int64_t(1) << 31))
    return fail(HIGGS_ERR_UNSUPPORTED, "samples * in must be below 2^31");
  if (!(damp >= 0.0) || !std::isfinite(damp))
    return fail(HIGGS_ERR_INVALID_ARG, "damp must be finite and >= 0");
  if (workspace_bytes < higgs::gptq_factor_workspace_bytes(samples, in))
    return fail(HIGGS_ERR_INVALID_ARG, "workspace too small: %lld bytes needed",
                (long long)higgs::gptq_factor_workspace_bytes(samples, in));
  if (!aligned(x_rot, 4) || !aligned(factor, 8) || !aligned(workspace, 256))
    return fail(HIGGS_ERR_INVALID_ARG, "x_rot 4-, factor 8-, workspace 256-byte aligned");
  char msg[256] = {0};
  const int st = higgs::gptq_factor(x_rot, samples, in, damp, factor, workspace,
                                    static_cast<hipStream_t>(stream), msg, int(sizeof(msg)));
  if (st != HIGGS_OK) return fail(higgs_status(st), "%s", msg);
  return ok();
}

int64_t higgs_quantize_gptq_workspace_bytes(int64_t out, int64_t in, int g) {
  if (out < 1 || in < 1 || higgs::log2_exact(g) < 6 || in % g != 0) return -1;
  return higgs::gptq_quantize_workspace_bytes(out, in, g);
}

higgs_status higgs_quantize_gptq(const void* W, higgs_dtype w_dtype, int64_t out, int64_t in,
                                 const float* grid, int p, int n, int g, uint64_t rht_seed,
                                 const double* factor, uint8_t* codes, uint16_t* scales,
                                 void* workspace, int64_t workspace_bytes, void* stream) {
  if (!W || !grid || !factor || !codes || !scales || !workspace)
    return fail(HIGGS_ERR_INVALID_ARG,
                "W, grid, factor, codes, scales and workspace must not be NULL");
  if (w_dtype != HIGGS_F32 && w_dtype != HIGGS_BF16)
    return fail(HIGGS_ERR_INVALID_ARG, "w_dtype must be HIGGS_F32 or HIGGS_BF16");
  const higgs_status st = check_layer(p, n, g, out, in);
  if (st != HIGGS_OK) return st;
  if (out * in >= (int64_t(1) << 31) || in > 65536)
    return fail(HIGGS_ERR_UNSUPPORTED, "GPTQ rounding needs out * in < 2^31 and in <= 65536");
  const int64_t need = higgs::gptq_quantize_workspace_bytes(out, in, g);
  if (workspace_bytes < need)
    return fail(HIGGS_ERR_INVALID_ARG, "workspace too small: %lld bytes needed", (long long)need);
  if (!aligned(W, 16) || !aligned(codes, 16) || !aligned(scales, 2) || !aligned(grid, 4) ||
      !aligned(factor, 8) || !aligned(workspace, 256))
    return fail(HIGGS_ERR_INVALID_ARG,
                "W and codes 16-, factor 8-, workspace 256-byte aligned, grid 4, scales 2");
  char msg[256] = {0};
  const int rs = higgs::gptq_quantize(W, w_dtype, out, in, grid, p, n, g, rht_seed, factor, codes,
                                      scales, workspace, static_cast<hipStream_t>(stream), msg,
                                      int(sizeof(msg)));
  if (rs != HIGGS_OK) return fail(higgs_status(rs), "%s", msg);
  return ok();
}

higgs_status higgs_allocate_bits(int layers, int options, const double* alpha, const double* t2,
                                 const double* bits, const int64_t* sizes, double b_max,
                                 int32_t* choice, double* objective, double* avg_bits) {
  if (!alpha || !t2 || !bits || !sizes || !choice)
    return fail(HIGGS_ERR_INVALID_ARG, "alpha, t2, bits, sizes and choice must not be NULL");
  for (int l = 0; l < layers; ++l)
    if (!(alpha[l] >= 0.0) || !std::isfinite(alpha[l]))
      return fail(HIGGS_ERR_INVALID_ARG, "alpha[%d] must be finite and >= 0", l);
  for (int64_t i = 0; i < int64_t(layers) * options; ++i)
    if (!(t2[i] >= 0.0) || !std::isfinite(t2[i]))
      return fail(HIGGS_ERR_INVALID_ARG, "t2[%lld] must be finite and >= 0", (long long)i);
  char msg[256] = {0};
  const int st = higgs::allocate_bits(layers, options, alpha, t2, bits, sizes, b_max, choice,
                                      objective, avg_bits, msg, int(sizeof(msg)));
  if (st != HIGGS_OK) return fail(higgs_status(st), "%s", msg);
  return ok();
}

higgs_status higgs_rht_activations(const void* x, higgs_dtype x_dtype, int64_t batch, int64_t in,
                                   int g, uint64_t rht_seed, float* x_rot, void* stream) {
  if (!x || !x_rot) return fail(HIGGS_ERR_INVALID_ARG, "x and x_rot must not be NULL");
  if (x_dtype != HIGGS_F32 && x_dtype != HIGGS_BF16)
    return fail(HIGGS_ERR_INVALID_ARG, "x_dtype must be HIGGS_F32 or HIGGS_BF16");
  if (batch < 1 || in < 1)
    return fail(HIGGS_ERR_INVALID_ARG, "batch and in must be >= 1");
  if (higgs::log2_exact(g) < 1 || g > 4096)
    return fail(HIGGS_ERR_UNSUPPORTED, "g (%d) must be a power of two in [2, 4096]", g);
  if (in % g != 0)
    return fail(HIGGS_ERR_INVALID_ARG, "in (%lld) must be a multiple of g (%d)", (long long)in, g);
  if (!aligned(x, 16) || !aligned(x_rot, 16))
    return fail(HIGGS_ERR_INVALID_ARG, "x and x_rot must be 16-byte aligned");
  const size_t esz = x_dtype == HIGGS_F32 ? 4 : 2;
  const char* xb = static_cast<const char*>(x);
  const char* yb = reinterpret_cast<const char*>(x_rot);
  const size_t nx = size_t(batch * in) * esz, ny = size_t(batch * in) * 4;
  if (xb < yb + ny && yb < xb + nx)
    return fail(HIGGS_ERR_INVALID_ARG, "x and x_rot must not overlap");
  const hipError_t err = higgs::launch_rht_activations(x, x_dtype, batch, in, g, rht_seed, x_rot,
                                                       static_cast<hipStream_t>(stream));
  return device_status(err, "higgs_rht_activations launch");
}

higgs_status higgs_qmatmul(const float* x_rot, int64_t batch, const uint8_t* codes,
                           const uint16_t* scales, const float* grid, int p, int n, int g,
                           int64_t out, int64_t in, float* y, void* workspace,
                           int64_t workspace_bytes, void* stream) {
  if (!x_rot || !codes || !scales || !grid || !y)
    return fail(HIGGS_ERR_INVALID_ARG, "x_rot, codes, scales, grid and y must not be NULL");
  if (batch < 1) return fail(HIGGS_ERR_INVALID_ARG, "batch must be >= 1");
  higgs_status st = check_layer(p, n, g, out, in);
  if (st == HIGGS_OK) st = check_product(batch, p, n, in, g);
  if (st != HIGGS_OK) return st;
  const int64_t need = higgs_qmatmul_workspace_bytes(batch, out, in, p, n, g);
  if (workspace_bytes < need || (need > 0 && workspace == nullptr))
    return fail(HIGGS_ERR_INVALID_ARG, "workspace too small: %lld bytes needed",
                (long long)need);
  if (!aligned(x_rot, 16) || !aligned(codes, 16) || !aligned(scales, 2) || !aligned(grid, 4) ||
      !aligned(y, 4) || !aligned(workspace, 16))
    return fail(HIGGS_ERR_INVALID_ARG,
                "x_rot, codes and workspace must be 16-byte aligned, y and grid 4, scales 2");
  const hipError_t err =
      higgs::use_qgemm(batch, p, n, in, g)
          ? higgs::launch_qgemm(x_rot, higgs::kQgemmRotated, 0, batch, codes, scales, grid, p, n, g,
                                out, in, y, workspace, static_cast<hipStream_t>(stream))
          : higgs::launch_qgemv(x_rot, batch, codes, scales, grid, p, n, g, out, in, y,
                                static_cast<hipStream_t>(stream));
  return device_status(err, "higgs_qmatmul launch");
}

int64_t higgs_qmatmul_fused_workspace_bytes(int64_t batch, int64_t out, int64_t in, int p, int n,
                                            int g) {
  if (batch < 1 || check_layer(p, n, g, out, in) != HIGGS_OK) return -1;
  if (higgs::use_qgemm(batch, p, n, in, g))  // rotation inside the activation conversion
    return higgs::qgemm_workspace_bytes(batch, out, in, p, n, g);
  if (higgs::qgemv_rotates(p, n, g)) return 0;  // rotation inside the product
  // rotated activations (16-byte aligned) followed by the product's workspace
  const int64_t xrot = (batch * in * 4 + 255) / 256 * 256;
  return xrot + higgs_qmatmul_workspace_bytes(batch, out, in, p, n, g);
}

}  // extern "C"

// Validation of higgs_qmatmul_fused's arguments (also per layer of
// higgs_qmatmul_fused_multi); returns the workspace the call needs in *need.
// check_ws = false skips the checks of the caller's workspace (the
// allocation-free entry point brings its own).
static higgs_status check_fused(const void* x, higgs_dtype x_dtype, int64_t batch,
                                const uint8_t* codes, const uint16_t* scales, const float* grid,
                                int p, int n, int g, int64_t out, int64_t in, const float* y,
                                const void* workspace, int64_t workspace_bytes, int64_t* need,
                                bool check_ws = true) {
  if (!x || !codes || !scales || !grid || !y)
    return fail(HIGGS_ERR_INVALID_ARG, "x, codes, scales, grid and y must not be NULL");
  if (x_dtype != HIGGS_F32 && x_dtype != HIGGS_BF16)
    return fail(HIGGS_ERR_INVALID_ARG, "x_dtype must be HIGGS_F32 or HIGGS_BF16");
  if (batch < 1) return fail(HIGGS_ERR_INVALID_ARG, "batch must be >= 1");
  higgs_status st = check_layer(p, n, g, out, in);
  if (st == HIGGS_OK) st = check_product(batch, p, n, in, g);
  if (st != HIGGS_OK) return st;
  *need = higgs_qmatmul_fused_workspace_bytes(batch, out, in, p, n, g);
  if (check_ws && (workspace_bytes < *need || (*need > 0 && workspace == nullptr)))
    return fail(HIGGS_ERR_INVALID_ARG, "workspace too small: %lld bytes needed",
                (long long)*need);
  if (!aligned(x, 16) || !aligned(codes, 16) || !aligned(scales, 2) || !aligned(grid, 4) ||
      !aligned(y, 4) || (check_ws && !aligned(workspace, 16)))
    return fail(HIGGS_ERR_INVALID_ARG,
                "x, codes and workspace must be 16-byte aligned, y and grid 4, scales 2");
  return HIGGS_OK;
}

// Launches of one checked higgs_qmatmul_fused call.
static higgs_status run_fused(const void* x, higgs_dtype x_dtype, int64_t batch,
                              const uint8_t* codes, const uint16_t* scales, const float* grid,
                              int p, int n, int g, uint64_t rht_seed, int64_t out, int64_t in,
                              float* y, void* workspace, int64_t need, hipStream_t s) {
  if (higgs::use_qgemm(batch, p, n, in, g)) {
    const hipError_t err = higgs::launch_qgemm(
        x, x_dtype == HIGGS_BF16 ? higgs::kQgemmRawBF16 : higgs::kQgemmRawF32, rht_seed, batch,
        codes, scales, grid, p, n, g, out, in, y, workspace, s);
    return device_status(err, "higgs_qmatmul_fused launch");
  }
  if (need == 0) {
    const hipError_t err = higgs::launch_qgemv_rotating(x, x_dtype == HIGGS_BF16 ? 1 : 0, rht_seed,
                                                        batch, codes, scales, grid, p, n, g, out,
                                                        in, y, s);
    return device_status(err, "higgs_qmatmul_fused launch");
  }
  float* x_rot = static_cast<float*>(workspace);
  hipError_t err = higgs::launch_rht_activations(x, x_dtype, batch, in, g, rht_seed, x_rot, s);
  if (err != hipSuccess) return device_status(err, "higgs_qmatmul_fused rotation launch");
  err = higgs::launch_qgemv(x_rot, batch, codes, scales, grid, p, n, g, out, in, y, s);
  return device_status(err, "higgs_qmatmul_fused launch");
}

extern "C" {

higgs_status higgs_qmatmul_fused(const void* x, higgs_dtype x_dtype, int64_t batch,
                                 const uint8_t* codes, const uint16_t* scales, const float* grid,
                                 int p, int n, int g, uint64_t rht_seed, int64_t out, int64_t in,
                                 float* y, void* workspace, int64_t workspace_bytes, void* stream) {
  int64_t need = 0;
  const higgs_status st = check_fused(x, x_dtype, batch, codes, scales, grid, p, n, g, out, in, y,
                                      workspace, workspace_bytes, &need);
  if (st != HIGGS_OK) return st;
  return run_fused(x, x_dtype, batch, codes, scales, grid, p, n, g, rht_seed, out, in, y,
                   workspace, need, static_cast<hipStream_t>(stream));
}

higgs_status higgs_qmatmul_fused_noalloc(const void* x, higgs_dtype x_dtype, int64_t batch,
                                         const uint8_t* codes, const uint16_t* scales,
                                         const float* grid, int p, int n, int g,
                                         uint64_t rht_seed, int64_t out, int64_t in, float* y,
                                         void* stream) {
  int64_t need = 0;
  const higgs_status st = check_fused(x, x_dtype, batch, codes, scales, grid, p, n, g, out, in, y,
                                      nullptr, 0, &need, false);
  if (st != HIGGS_OK) return st;
  if (need > higgs::kScratchBytes)
    return fail(HIGGS_ERR_UNSUPPORTED,
                "this call needs %lld bytes of workspace; the fixed scratch holds %lld "
                "(use higgs_qmatmul_fused with a workspace)",
                (long long)need, (long long)higgs::kScratchBytes);
  void* ws = nullptr;
  if (need > 0) {
    const hipError_t err = higgs::scratch_buffer(&ws);
    if (err != hipSuccess) return device_status(err, "higgs_qmatmul_fused_noalloc scratch");
  }
  return run_fused(x, x_dtype, batch, codes, scales, grid, p, n, g, rht_seed, out, in, y, ws,
                   need, static_cast<hipStream_t>(stream));
}

int64_t higgs_qmatmul_fused_multi_workspace_bytes(int layers, int64_t batch, const int64_t* out,
                                                  int64_t in, int p, int n, int g) {
  if (layers < 1 || layers > 4 || out == nullptr || batch < 1) return -1;
  for (int l = 0; l < layers; ++l)
    if (check_layer(p, n, g, out[l], in) != HIGGS_OK) return -1;
  if (higgs::use_qgemm(batch, p, n, in, g))
    return higgs::qgemm_group_workspace_bytes(layers, batch, out, in, p, n, g);
  int64_t need = 0;
  for (int l = 0; l < layers; ++l)
    need = std::max(need, higgs_qmatmul_fused_workspace_bytes(batch, out[l], in, p, n, g));
  return need;
}

higgs_status higgs_qmatmul_fused_multi(int layers, const void* x, higgs_dtype x_dtype,
                                       int64_t batch, const uint8_t* const* codes,
                                       const uint16_t* const* scales, const float* grid, int p,
                                       int n, int g, const uint64_t* rht_seeds,
                                       const int64_t* out, int64_t in, float* const* y,
                                       void* workspace, int64_t workspace_bytes, void* stream) {
  if (layers < 1 || layers > std::min(4, higgs::qgemv_max_layers()))
    return fail(HIGGS_ERR_INVALID_ARG, "layers (%d) must be in [1, %d]", layers,
                higgs::qgemv_max_layers());
  if (!codes || !scales || !rht_seeds || !out || !y)
    return fail(HIGGS_ERR_INVALID_ARG, "codes, scales, rht_seeds, out and y must not be NULL");
  // per-layer checks; the workspace is checked against the whole call's need
  int64_t need[4] = {0, 0, 0, 0};
  for (int l = 0; l < layers; ++l) {
    const higgs_status st =
        check_fused(x, x_dtype, batch, codes[l], scales[l], grid, p, n, g, out[l], in, y[l],
                    workspace, INT64_MAX, &need[l]);
    if (st != HIGGS_OK) return fail(st, "layer %d: %s", l, higgs_last_error());
  }
  const int64_t need_all =
      higgs_qmatmul_fused_multi_workspace_bytes(layers, batch, out, in, p, n, g);
  if (workspace_bytes < need_all || (need_all > 0 && workspace == nullptr))
    return fail(HIGGS_ERR_INVALID_ARG, "workspace too small: %lld bytes needed",
                (long long)need_all);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const int x_bf16 = x_dtype == HIGGS_BF16 ? 1 : 0;
  if (higgs::use_qgemm(batch, p, n, in, g)) {  // one conversion, one product launch per 64 rows
    const hipError_t err = higgs::launch_qgemm_group(
        x, x_bf16 ? higgs::kQgemmRawBF16 : higgs::kQgemmRawF32, layers, rht_seeds, batch, codes,
        scales, grid, p, n, g, out, in, y, workspace, s);
    return device_status(err, "higgs_qmatmul_fused_multi launch");
  }
  if (need_all == 0) {  // rotation inside the small-batch product: one launch
    const hipError_t err = higgs::launch_qgemv_rotating_group(
        x, x_bf16, layers, rht_seeds, batch, codes, scales, grid, p, n, g, out, in, y, s);
    return device_status(err, "higgs_qmatmul_fused_multi launch");
  }
  for (int l = 0; l < layers; ++l) {
    const higgs_status st = run_fused(x, x_dtype, batch, codes[l], scales[l], grid, p, n, g,
                                      rht_seeds[l], out[l], in, y[l], workspace, need[l], s);
    if (st != HIGGS_OK) return st;
  }
  return ok();
}

}  // extern "C"
