// GPTQ rounding for HIGGS (Sec. 3.5): the nearest-point step of Alg. 1
// replaced by the GPTQ error-feedback rounding, in the rotated space, with the
// same output format (codes + fp16 group scales).
//
// Factor: H = X'^T X' over the rotated calibration activations X' (samples x
// in, as higgs_rht_activations writes them), damped by damp * mean(diag H) on
// the diagonal (the usual GPTQ damping), then Hinv = H^-1 and its Cholesky
// factor Hinv = U^T U, all in fp64 (rocBLAS syrk, rocSOLVER potrf / potri /
// potrf). rocSOLVER leaves a column-major lower factor L with Hinv = L L^T;
// read row-major, that buffer is exactly U = L^T.
//
// Quantize: the rotated weights W' and group norms (one kernel), then per
// block of 64 columns the block kernel (rounding, in-block error feedback,
// codes) and one fp64 GEMM  W'[:, after] -= E_block U[block, after].

#include <rocblas/rocblas.h>
#include <rocsolver/rocsolver.h>

#include <cstdio>
#include <mutex>

#include "internal.h"

namespace higgs {
namespace {

// One rocBLAS handle per (thread, device); rocSOLVER uses the same handle.
rocblas_handle blas_handle(char* msg, int msg_len) {
  struct Slot {
    int device = -1;
    rocblas_handle h = nullptr;
  };
  thread_local Slot slots[16];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 16) {
    std::snprintf(msg, size_t(msg_len), "no usable HIP device");
    return nullptr;
  }
  Slot& s = slots[dev];
  if (s.h == nullptr) {
    if (rocblas_create_handle(&s.h) != rocblas_status_success) {
      std::snprintf(msg, size_t(msg_len), "rocblas_create_handle failed");
      s.h = nullptr;
      return nullptr;
    }
    s.device = dev;
  }
  return s.h;
}

int64_t align256(int64_t v) { return (v + 255) / 256 * 256; }

}  // namespace

int64_t gptq_factor_workspace_bytes(int64_t samples, int64_t in) {
  return align256(samples * in * 8) + 256;  // fp64 activations + the info word
}

int64_t gptq_quantize_workspace_bytes(int64_t out, int64_t in, int g) {
  return align256(out * in * 8) + align256(out * (in / g) * 8) + align256(out * 64 * 8);
}

int gptq_factor(const float* x_rot, int64_t samples, int64_t in, double damp, double* factor,
                void* workspace, hipStream_t stream, char* msg, int msg_len) {
  rocblas_handle h = blas_handle(msg, msg_len);
  if (!h) return HIGGS_ERR_DEVICE;
  if (rocblas_set_stream(h, stream) != rocblas_status_success) {
    std::snprintf(msg, size_t(msg_len), "rocblas_set_stream failed");
    return HIGGS_ERR_DEVICE;
  }
  double* x64 = static_cast<double*>(workspace);
  rocblas_int* info =
      reinterpret_cast<rocblas_int*>(static_cast<char*>(workspace) + align256(samples * in * 8));
  if (launch_to_f64(x_rot, samples * in, x64, stream) != hipSuccess) {
    std::snprintf(msg, size_t(msg_len), "activation conversion launch failed");
    return HIGGS_ERR_DEVICE;
  }
  // row-major X' [samples][in] is column-major in x samples: H = A A^T
  const double one = 1.0, zero = 0.0;
  const rocblas_int n = rocblas_int(in), k = rocblas_int(samples);
  if (rocblas_dsyrk(h, rocblas_fill_lower, rocblas_operation_none, n, k, &one, x64, n, &zero,
                    factor, n) != rocblas_status_success) {
    std::snprintf(msg, size_t(msg_len), "rocblas_dsyrk failed");
    return HIGGS_ERR_DEVICE;
  }
  if (launch_damp_diag(factor, in, damp, stream) != hipSuccess) {
    std::snprintf(msg, size_t(msg_len), "damping launch failed");
    return HIGGS_ERR_DEVICE;
  }
  const char* steps[3] = {"Cholesky factorisation of H", "inversion of H",
                          "Cholesky factorisation of H^-1"};
  for (int step = 0; step < 3; ++step) {
    const rocblas_status st =
        step == 1 ? rocsolver_dpotri(h, rocblas_fill_lower, n, factor, n, info)
                  : rocsolver_dpotrf(h, rocblas_fill_lower, n, factor, n, info);
    if (st != rocblas_status_success) {
      std::snprintf(msg, size_t(msg_len), "rocSOLVER failed in the %s", steps[step]);
      return HIGGS_ERR_DEVICE;
    }
    rocblas_int host_info = 0;
    if (hipMemcpyAsync(&host_info, info, sizeof(host_info), hipMemcpyDeviceToHost, stream) !=
            hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess) {
      std::snprintf(msg, size_t(msg_len), "reading the factorisation status failed");
      return HIGGS_ERR_DEVICE;
    }
    if (host_info != 0) {
      std::snprintf(msg, size_t(msg_len),
                    "%s failed at column %d: the damped Hessian is not positive definite",
                    steps[step], int(host_info));
      return HIGGS_ERR_INVALID_ARG;
    }
  }
  return HIGGS_OK;
}

int gptq_quantize(const void* w, higgs_dtype dtype, int64_t out, int64_t in, const float* grid,
                  int p, int n, int g, uint64_t seed, const double* factor, uint8_t* codes,
                  uint16_t* scales, void* workspace, hipStream_t stream, char* msg, int msg_len) {
  rocblas_handle h = blas_handle(msg, msg_len);
  if (!h) return HIGGS_ERR_DEVICE;
  if (rocblas_set_stream(h, stream) != rocblas_status_success) {
    std::snprintf(msg, size_t(msg_len), "rocblas_set_stream failed");
    return HIGGS_ERR_DEVICE;
  }
  char* ws = static_cast<char*>(workspace);
  double* wr = reinterpret_cast<double*>(ws);
  double* norms = reinterpret_cast<double*>(ws + align256(out * in * 8));
  double* err = reinterpret_cast<double*>(ws + align256(out * in * 8) + align256(out * (in / g) * 8));
  if (launch_gptq_prepare(w, dtype, out, in, g, seed, wr, norms, scales, stream) != hipSuccess) {
    std::snprintf(msg, size_t(msg_len), "rotation launch failed");
    return HIGGS_ERR_DEVICE;
  }
  const double minus_one = -1.0, one = 1.0;
  for (int64_t c0 = 0; c0 < in; c0 += 64) {
    if (launch_gptq_block(wr, norms, factor, grid, p, n, out, in, g, c0, codes, err, stream) !=
        hipSuccess) {
      std::snprintf(msg, size_t(msg_len), "block launch failed at column %lld", (long long)c0);
      return HIGGS_ERR_DEVICE;
    }
    const int64_t rest = in - (c0 + 64);
    if (rest <= 0) break;
    // column-major views: W'^T[c0+64:, :] (rest x out, ld in) -=
    //   U[c0:c0+64, c0+64:]^T (rest x 64, ld in) * E^T (64 x out, ld 64)
    if (rocblas_dgemm(h, rocblas_operation_none, rocblas_operation_none, rocblas_int(rest),
                      rocblas_int(out), 64, &minus_one, factor + c0 * in + c0 + 64,
                      rocblas_int(in), err, 64, &one, wr + c0 + 64,
                      rocblas_int(in)) != rocblas_status_success) {
      std::snprintf(msg, size_t(msg_len), "rocblas_dgemm failed at column %lld", (long long)c0);
      return HIGGS_ERR_DEVICE;
    }
  }
  return HIGGS_OK;
}

}  // namespace higgs
