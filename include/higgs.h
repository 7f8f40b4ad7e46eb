/*
 * higgs.h - C ABI of the HIGGS quantized linear-layer library for MI355X (gfx950).
 *
 * HIGGS (arXiv 2411.17525, Sec. 3) quantizes a weight matrix by rotating each
 * group of g consecutive input-dimension weights with a random Hadamard
 * transform (RHT), dividing by the group's L2 norm and rounding every p
 * consecutive rotated values to the nearest point of an n-point grid that is
 * MSE-optimal for the standard normal distribution (Alg. 1, Alg. 2). Inference
 * applies the same RHT to the activations and multiplies in the rotated space
 * (App. G), dequantising grid indices through a lookup table (Sec. 3.3).
 *
 * Conventions (fixed where the paper leaves a choice open):
 *   - W is row-major [out][in]; groups are contiguous along `in` (App. G
 *     groups W[0, 0:g], W[0, g:2g], ...). in % g == 0, g a power of two.
 *   - The rotation of a group is R = H diag(sigma) / sqrt(g), H the unnormalised
 *     Sylvester Hadamard matrix in natural order (H[r][c] = (-1)^popcount(r&c)).
 *     sigma in {+1,-1}^g is shared by every group, row and activation block:
 *     sigma_j = +1 iff the top bit of output j of splitmix64 started at the
 *     rotation seed is 0 (see higgs_rht_signs).
 *   - Codes are 0-based grid indices; code m of a row (m = i*(g/p) + j for
 *     group i, p-vector j) occupies bits [m*b, (m+1)*b) of the row's byte
 *     string, b = log2(n), bit t being bit (t % 8) of byte t / 8 (LSB first).
 *   - scales[o][i] is the fp16 (IEEE binary16, round to nearest even, one
 *     rounding from the exact value) of s / sqrt(g), s = ||W[o, ig:(i+1)g]||_2.
 *   - Supported grids (p, n): (1,16), (2,64), (2,256), (2,1024), i.e. 4, 3,
 *     4 and 5 bits per weight, and (1,256), 8 bits per weight (the CH8
 *     format with the grid of higgs_make_uniform_grid(256); any 256-point
 *     scalar grid works); grid is fp32 [n][p], point k at grid[k*p].
 *     Grids are MSE-optimal for N(0, I_p), so their points have norms of a
 *     few units; the encoder's search is exact for point norms up to 1024
 *     (see higgs_quantize).
 *
 * Memory: the caller owns every buffer. Device pointers must point to device
 * memory of the current HIP device; host pointers to host memory. The library
 * allocates no device memory, with one exception: the GPTQ entry points
 * (higgs_gptq_factor, higgs_quantize_gptq) call rocBLAS and rocSOLVER, whose
 * handle (one per calling thread and device, created on first use and kept
 * until the process ends) allocates its own device workspace. The library
 * keeps no pointer to a caller's buffer after a call returns.
 * Streams: `stream` is a hipStream_t (NULL = the legacy default stream). Device
 * calls only enqueue work; outputs are valid once the stream is synchronised.
 *
 * Errors: every call validates its arguments on the host before launching
 * anything and returns HIGGS_ERR_INVALID_ARG (malformed sizes or pointers) or
 * HIGGS_ERR_UNSUPPORTED (a well-formed configuration this build does not
 * implement) with no work enqueued. A failed launch returns HIGGS_ERR_DEVICE.
 * higgs_last_error() returns a thread-local message for the last failure of
 * the calling thread. No C++ exception crosses this interface; calls keep no
 * global mutable state apart from that message and per-process caches that
 * are filled once (compute-unit counts, RHT sign masks per thread, the GPTQ
 * handles above), and are safe to make from several threads.
 */
#ifndef HIGGS_H_
#define HIGGS_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum higgs_status {
  HIGGS_OK = 0,
  HIGGS_ERR_INVALID_ARG = 1,
  HIGGS_ERR_UNSUPPORTED = 2,
  HIGGS_ERR_DEVICE = 3
} higgs_status;

typedef enum higgs_dtype {
  HIGGS_F32 = 0,  /* IEEE binary32 */
  HIGGS_BF16 = 1, /* bfloat16 bit patterns (uint16) */
  /* Range markers, not element types: they give the enumeration the full
   * range of int, so that any int a C caller passes is a valid value that
   * the library can check and reject (HIGGS_ERR_INVALID_ARG). */
  HIGGS_DTYPE_RANGE_MIN_ = -2147483647 - 1,
  HIGGS_DTYPE_RANGE_MAX_ = 2147483647
} higgs_dtype;

/* Version of this interface (incremented on any incompatible change). */
int higgs_abi_version(void);

/* Message describing the last failed call on this thread ("" if none). The
 * pointer stays valid until the next call on the same thread. */
const char *higgs_last_error(void);

/* ---------------------------------------------------------------------------
 * higgs_make_grid - the MSE-optimal Gaussian grid G_n^p (Sec. 3.2; Alg. 2,
 * "computed once" per (n, p)). Host only, synchronous, deterministic.
 *
 * Lloyd's algorithm on num_samples standard-normal p-vectors: normals come
 * from splitmix64(seed) outputs turned into 53-bit uniforms u = (z >> 11)
 * 2^-53, paired (u1, u2) into r = sqrt(-2 ln(1-u1)), theta = 2 pi u2 ->
 * r cos(theta), r sin(theta), filled row-major into the [num_samples][p]
 * sample matrix. Start: the first n samples. Each iteration assigns every
 * sample to its nearest point (squared Euclidean distance, lowest index on
 * ties) and moves each point to the mean of its cell; an empty cell keeps its
 * point. Stops when an assignment repeats the previous one or after max_iters
 * mean updates. The paper's CLVQ procedure is not spelled out; this Lloyd
 * iteration minimises the same objective.
 *
 *   grid         [out] host, n*p floats (fp32 of the fp64 result).
 *   mse_per_dim  [out] host, nullable: mean over samples of the squared
 *                distance to the final grid, divided by p.
 *   iters_done   [out] host, nullable: number of mean updates performed.
 * Requires 1 <= p <= 2, 2 <= n <= 4096, num_samples >= n, max_iters >= 0.
 * ------------------------------------------------------------------------- */
higgs_status higgs_make_grid(int p, int n, uint64_t seed, int64_t num_samples, int max_iters,
                             float *grid, double *mse_per_dim, int *iters_done);

/* ---------------------------------------------------------------------------
 * higgs_make_uniform_grid - the uniform scalar grid of the CH8 format
 * (Sec. 3.3: for bit widths beyond the lookup-table grids, the grid is
 * constrained to be uniform, its position and scale chosen to minimise the
 * expected squared error over N(0, 1); with n = 256 and p = 1 this is CH8).
 * Host only, synchronous, deterministic.
 *
 * Points grid[k] = step * (k - (n - 1) / 2), k < n (symmetric about 0, the
 * optimum for the symmetric density); step minimises E[(X - Q(X))^2] for
 * X ~ N(0, 1) with nearest-point rounding, computed exactly (closed-form
 * Gaussian integrals, root of the derivative by bisection).
 *
 *   grid  [out] host, n floats (fp32 of the fp64 points), usable as the
 *         (p, n) = (1, n) grid of higgs_quantize / higgs_qmatmul.
 *   step  [out] host, nullable: the fp64 step.
 *   mse   [out] host, nullable: the fp64 mean squared error at that step.
 * Requires 2 <= n <= 4096.
 * ------------------------------------------------------------------------- */
higgs_status higgs_make_uniform_grid(int n, float *grid, double *step, double *mse);

/* The RHT sign vector sigma (Alg. 1, seed xi): signs[j] = +1 or -1 for
 * j < g, host buffer of g int8. Host only. g must be a power of two <= 4096. */
higgs_status higgs_rht_signs(uint64_t seed, int g, int8_t *signs);

/* Bytes of one packed code row: (in / p) * log2(n) / 8; -1 if the arguments
 * are invalid or the row does not fill whole bytes. Sec. 3.3, Constraint 1:
 * codes are stored as bit-packed indices of log2(n) bits; here one contiguous
 * LSB-first stream per row serves every code width. Host only, pure. */
int64_t higgs_codes_row_bytes(int64_t in, int p, int n);

/* Bytes of device workspace higgs_qmatmul needs for these sizes (0 if none;
 * -1 if the arguments are invalid). The workspace holds what the product of
 * App. G / Sec. 3.3 keeps between its kernels on the matrix-core path: the
 * activations converted to fp16 with one power of two per batch row and scale
 * group, and the partial sums of a K-split (the codes themselves, Constraint
 * 1's packed indices, are read in place). Host only, pure. */
int64_t higgs_qmatmul_workspace_bytes(int64_t batch, int64_t out, int64_t in, int p, int n, int g);

/* ---------------------------------------------------------------------------
 * higgs_search_index - the nearest-point search index of a grid, for
 * higgs_quantize (the search of Alg. 1 over the grid of Alg. 2). Device,
 * asynchronous on `stream` (two kernel launches).
 *
 * The index cuts the square [-4, 4)^p into buckets (128 x 128 for p = 2 with
 * n >= 256, 64 x 64 for n = 64, 512 for p = 1) and lists, per bucket, every
 * grid point that can be the nearest one to a vector in it: a point is left
 * out only when another point is nearer to the whole bucket by a margin far
 * above the search's rounding, so the codes of higgs_quantize are the same
 * with and without it. It records a hash of the grid's values;
 * higgs_quantize ignores an index whose hash does not match the grid it is
 * given, or whose lists would not fit its on-chip table, and then scans all
 * n points for every vector.
 *
 *   grid   [in]  device, n*p floats (the grid passed to higgs_quantize).
 *   index  [out] device, >= higgs_search_index_bytes(p, n) bytes, 16-byte
 *                aligned; owned by the caller, reused for every layer
 *                quantized with this grid (until the grid's values change).
 * Errors: HIGGS_ERR_UNSUPPORTED for an unsupported (p, n);
 * HIGGS_ERR_INVALID_ARG for NULL pointers, misalignment or a short buffer.
 * ------------------------------------------------------------------------- */
int64_t higgs_search_index_bytes(int p, int n); /* -1 for an unsupported grid; host only */
higgs_status higgs_search_index(const float *grid, int p, int n, void *index,
                                int64_t index_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * higgs_quantize - Alg. 1 (RHT-VQ) with the grid of Alg. 2, on the GPU.
 *
 * For every row o and group i: s = ||w||_2 of w = W[o, ig:(i+1)g];
 * w_dag = H (sigma * (w / s)) (entries ~ N(0,1), ||w_dag||^2 = g); each
 * p-vector w_dag[jp:(j+1)p] gets the index of its nearest grid point (lowest
 * index on ties); scales[o][i] = fp16(s / sqrt(g)). A group with s == 0 gets
 * scale 0 and, for every p-vector, the grid point nearest the origin.
 * Rotation and search are done in fp64. The search may resolve candidates
 * whose squared distances differ by less than S 2^-41 to the lower index,
 * S the least power of two >= max(1024, R^2 + 2 sqrt(g) R) for the largest
 * grid-point norm R: below 5e-10 for every unit-variance grid (S = 1024), and
 * below 1e-6 for any grid with R <= 1024.
 *
 *   W        [in]  device, out*in values of w_dtype (HIGGS_F32 or HIGGS_BF16).
 *   grid     [in]  device, n*p floats.
 *   index    [in]  device, the grid's search index (higgs_search_index) of
 *                  index_bytes bytes, or NULL: every vector then scans all
 *                  n points (same codes, slower).
 *   codes    [out] device, out * higgs_codes_row_bytes(in, p, n) bytes.
 *   scales   [out] device, out * (in/g) fp16 bit patterns.
 * Requires out >= 1, in >= g, in % g == 0, g a power of two with
 * 64*p <= g <= 4096, (p, n) supported. W must hold finite values.
 * ------------------------------------------------------------------------- */
higgs_status higgs_quantize(const void *W, higgs_dtype w_dtype, int64_t out, int64_t in,
                            const float *grid, int p, int n, const void *index,
                            int64_t index_bytes, int g, uint64_t rht_seed, uint8_t *codes,
                            uint16_t *scales, void *stream);

/* ---------------------------------------------------------------------------
 * higgs_layer_error - the quantization error of a layer (Sec. 3.4: the
 * relative squared error t^2 = ||W - W_hat||_F^2 / ||W||_F^2 that, weighted
 * by a per-layer coefficient, predicts the loss increase; Sec. 4 uses it per
 * layer and quantizer). Device, asynchronous on `stream`.
 *
 * For each group i of each row o (row-major group order) writes two fp64
 * values: group_err[2q] = ||W[o, ig:(i+1)g] - W_hat[o, ig:(i+1)g]||^2 and
 * group_err[2q+1] = ||W[o, ig:(i+1)g]||^2, q = o*(in/g) + i. W_hat is the
 * dequantised layer (codes, scales, grid, g and rht_seed as in
 * higgs_quantize); the error is computed in the rotated space, where the
 * orthonormal rotation leaves it unchanged: || H diag(sigma) w / sqrt(g) -
 * scale * concat_j G[code_j] ||^2, in fp64.
 *   W          [in]  device, out*in fp32 or bf16 (as for higgs_quantize).
 *   group_err  [out] device, 2*out*(in/g) doubles, 8-byte aligned.
 *   t2         [out] device, nullable, one double, 8-byte aligned: the
 *              layer's t^2 = sum(err) / sum(norm) over its groups (0 for an
 *              all-zero layer), summed on the GPU in a fixed order
 *              (deterministic).
 * Requires the higgs_quantize layer conditions; W 16-byte aligned.
 * ------------------------------------------------------------------------- */
higgs_status higgs_layer_error(const void *W, higgs_dtype w_dtype, int64_t out, int64_t in,
                               const uint8_t *codes, const uint16_t *scales, const float *grid,
                               int p, int n, int g, uint64_t rht_seed, double *group_err,
                               double *t2, void *stream);

/* ---------------------------------------------------------------------------
 * GPTQ rounding (Sec. 3.5: the nearest-point step of Alg. 1 replaced by a
 * rounding that uses layer activations; the output format is unchanged).
 * Works in the rotated space, where the layer computes (W R^T)(R x) with the
 * orthonormal blockwise rotation R of higgs_rht_activations.
 *
 * higgs_gptq_factor - from rotated calibration activations X' (row-major
 * [samples][in], e.g. higgs_rht_activations of the layer's inputs with the
 * layer's g and rht_seed): H = X'^T X', H[i][i] += damp * mean_i H[i][i],
 * and the upper triangular U with H^-1 = U^T U, all fp64. Device; synchronises
 * `stream` to read the factorisation status.
 *   factor     [out] device, in*in doubles, row-major; U is its upper triangle
 *              (the strict lower triangle is left unspecified).
 *   workspace  device, >= higgs_gptq_factor_workspace_bytes(samples, in),
 *              256-byte aligned.
 * Requires in a multiple of 64 in [64, 65536], samples * in < 2^31, damp >= 0
 * (GPTQ uses 0.01). HIGGS_ERR_INVALID_ARG if the damped H is not positive
 * definite (e.g. all-zero activations with damp 0).
 *
 * higgs_quantize_gptq - codes and scales of W in the higgs_quantize format.
 * Scales as higgs_quantize (fp16(s / sqrt(g)) of the original group norms).
 * Codes: columns of the rotated weights W' (per group H (sigma * w) / sqrt(g))
 * are taken in order, one p-vector v at a time; its code q is the nearest grid
 * point of v sqrt(g) / s (lowest index on ties), and with e = v - (s /
 * sqrt(g)) G[q] and E = e U_pp^-1 (U_pp the diagonal p x p block of U) every
 * later column j moves by -E U[p-vector, j]. fp64 throughout; the update of a
 * block of 64 columns runs in the block, later columns get one GEMM per
 * block. With a diagonal H the codes are those of higgs_quantize (up to the
 * fp64 rounding of the normalisation).
 *   factor     [in]  device, as written by higgs_gptq_factor for this `in`.
 *   workspace  device, >= higgs_quantize_gptq_workspace_bytes(out, in, g),
 *              256-byte aligned (rotated weights, norms, block errors: fp64).
 * Requires the higgs_quantize conditions, out * in < 2^31, in <= 65536.
 * ------------------------------------------------------------------------- */
int64_t higgs_gptq_factor_workspace_bytes(int64_t samples, int64_t in);
higgs_status higgs_gptq_factor(const float *x_rot, int64_t samples, int64_t in, double damp,
                               double *factor, void *workspace, int64_t workspace_bytes,
                               void *stream);
int64_t higgs_quantize_gptq_workspace_bytes(int64_t out, int64_t in, int g);
higgs_status higgs_quantize_gptq(const void *W, higgs_dtype w_dtype, int64_t out, int64_t in,
                                 const float *grid, int p, int n, int g, uint64_t rht_seed,
                                 const double *factor, uint8_t *codes, uint16_t *scales,
                                 void *workspace, int64_t workspace_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * higgs_allocate_bits - per-layer quantizer choice under an average-bits
 * budget (Sec. 4, "Variable Bitwidth Quantization": minimise
 * sum_l alpha_l * t2[l][j_l] subject to sum_l bits[j_l] * d_l <= b_max *
 * sum_l d_l). Host only, synchronous, deterministic, exact.
 *
 * Solved as a multiple-choice knapsack by dynamic programming over integer
 * costs: bits[j] must be multiples of 2^-8 (every HIGGS option log2(n)/p +
 * 16/g with g >= 64 is), so costs bits[j] * 256 * d_l are integers; ties
 * keep the lower option index.
 *   layers, options  L >= 1 layers, 1 <= J <= 255 quantizer options.
 *   alpha      [in]  host, L finite coefficients >= 0.
 *   t2         [in]  host, L*J errors >= 0, row-major [layer][option].
 *   bits       [in]  host, J bits per weight of each option.
 *   sizes      [in]  host, L weight counts d_l in [1, 2^40].
 *   b_max      the average bits per weight allowed.
 *   choice     [out] host, L option indices.
 *   objective  [out] host, nullable: sum_l alpha_l * t2[l][choice[l]].
 *   avg_bits   [out] host, nullable: the chosen average bits per weight.
 * Returns HIGGS_ERR_INVALID_ARG when the budget is below the cheapest
 * assignment, HIGGS_ERR_UNSUPPORTED when the budget table would exceed
 * 512 MiB (L times the budget range in units of the costs' common divisor).
 * ------------------------------------------------------------------------- */
higgs_status higgs_allocate_bits(int layers, int options, const double *alpha, const double *t2,
                                 const double *bits, const int64_t *sizes, double b_max,
                                 int32_t *choice, double *objective, double *avg_bits);

/* ---------------------------------------------------------------------------
 * higgs_rht_activations - the activation side of App. G ("rotating
 * activations"): x_rot[b, block i] = H (sigma * x[b, block i]) / sqrt(g), in
 * fp32, with the same g and rotation seed as the layer's higgs_quantize call.
 *
 *   x      [in]  device, batch*in values of x_dtype, row-major [batch][in].
 *   x_rot  [out] device, batch*in floats. Must not overlap x.
 * Requires batch >= 1, in % g == 0, g a power of two with 2 <= g <= 4096.
 * ------------------------------------------------------------------------- */
higgs_status higgs_rht_activations(const void *x, higgs_dtype x_dtype, int64_t batch, int64_t in,
                                   int g, uint64_t rht_seed, float *x_rot, void *stream);

/* ---------------------------------------------------------------------------
 * higgs_qmatmul - the layer product in the rotated space (App. G; Sec. 3.3's
 * lookup-table matmul):
 *   y[b][o] = sum_i scales[o][i] * sum_j < grid[code(o,i,j)], x_rot[b, ig+jp : ig+(j+1)p] >
 * which equals x W_hat^T for x_rot = higgs_rht_activations(x). Grid points
 * and activations enter the products as fp16 (activations after an exact
 * power-of-two rescaling per batch row and block of inputs: 1024 inputs,
 * 2048 for 6- and 10-bit codes, on the small-batch path; one scale group of
 * g inputs on the matrix-core path), products are accumulated in fp32; y is
 * fp32.
 *
 *   x_rot     [in]  device, batch*in floats, row-major [batch][in].
 *   codes     [in]  device, packed codes as written by higgs_quantize.
 *   scales    [in]  device, out*(in/g) fp16 bit patterns.
 *   grid      [in]  device, n*p floats.
 *   y         [out] device, batch*out floats, row-major [batch][out].
 *   workspace [in]  device scratch of at least
 *                   higgs_qmatmul_workspace_bytes(...) bytes (may be NULL
 *                   when that is 0); its contents are not preserved.
 * Requires batch >= 1, out >= 1, in % g == 0, (p, n) supported, 64*p <= g
 * <= 4096, x_rot finite with magnitudes below 2^100. in <= 32768 for every
 * format unless the call takes the matrix-core path (in <= 2^23 there);
 * larger inputs return HIGGS_ERR_UNSUPPORTED. The matrix-core path serves every supported (p, n)
 * from a batch that depends on g, the format and the row length (measured
 * crossovers with the small-batch kernel): with g >= 128, batch 5 for
 * in <= 8192, else 2 for (2,256) and (1,16) and 3 for the other formats;
 * with g = 64 (p = 1), batch 9 for in <= 8192, else 5 for (1,16) and 7 for
 * (1,256).
 * ------------------------------------------------------------------------- */
higgs_status higgs_qmatmul(const float *x_rot, int64_t batch, const uint8_t *codes,
                           const uint16_t *scales, const float *grid, int p, int n, int g,
                           int64_t out, int64_t in, float *y, void *workspace,
                           int64_t workspace_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * higgs_qmatmul_fused - the layer output from raw activations:
 *   y = x W_hat^T = higgs_qmatmul(higgs_rht_activations(x, g, rht_seed), ...)
 * App. G: the activation rotation is asymptotically free next to the product;
 * here it runs inside the product kernel, while the activations are converted
 * (one launch), whenever the small-batch kernel runs (batches below the
 * matrix-core path's) and g <= 1024 (2048 for 6- and 10-bit codes);
 * on the matrix-core path inside its activation conversion
 * pass; as a separate pass into the workspace otherwise. Same numerics as the
 * two-call sequence.
 *
 *   x         [in]  device, batch*in values of x_dtype, row-major [batch][in].
 *   rht_seed  the layer's rotation seed (the one given to higgs_quantize).
 *   workspace [in]  device scratch of at least
 *                   higgs_qmatmul_fused_workspace_bytes(...) bytes.
 * Other arguments and requirements as for higgs_qmatmul.
 * ------------------------------------------------------------------------- */
int64_t higgs_qmatmul_fused_workspace_bytes(int64_t batch, int64_t out, int64_t in, int p, int n,
                                            int g);

higgs_status higgs_qmatmul_fused(const void *x, higgs_dtype x_dtype, int64_t batch,
                                 const uint8_t *codes, const uint16_t *scales, const float *grid,
                                 int p, int n, int g, uint64_t rht_seed, int64_t out, int64_t in,
                                 float *y, void *workspace, int64_t workspace_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * higgs_qmatmul_fused_noalloc - higgs_qmatmul_fused for callers that cannot
 * allocate device memory (code under HIP stream capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same product, the same kernels and
 * bit-identical results, with the workspace taken from a fixed scratch array
 * inside the library instead of the caller.
 *
 * The scratch is a device array of HIGGS_NOALLOC_SCRATCH_BYTES (32 MiB) in
 * the library's code object: each device the library runs on holds its own
 * copy until the process ends. This call allocates nothing (no hipMalloc, no
 * allocating library routine); the first call on a device resolves the
 * array's device address (hipGetSymbolAddress) and keeps it.
 *   - Calls whose workspace (higgs_qmatmul_fused_workspace_bytes) exceeds
 *     the scratch return HIGGS_ERR_UNSUPPORTED with nothing enqueued.
 *   - All calls on one device share its scratch: calls that overlap on one
 *     device (concurrent streams, several host threads) race and may corrupt
 *     each other's results. Serialise them, e.g. on one stream.
 *   - The scratch keeps the last call's contents; nothing in it has to start
 *     at zero.
 * Arguments, requirements and errors otherwise as for higgs_qmatmul_fused.
 * ------------------------------------------------------------------------- */
#define HIGGS_NOALLOC_SCRATCH_BYTES (32ll << 20)
higgs_status higgs_qmatmul_fused_noalloc(const void *x, higgs_dtype x_dtype, int64_t batch,
                                         const uint8_t *codes, const uint16_t *scales,
                                         const float *grid, int p, int n, int g,
                                         uint64_t rht_seed, int64_t out, int64_t in, float *y,
                                         void *stream);

/* ---------------------------------------------------------------------------
 * higgs_qmatmul_fused_multi - the outputs of up to 4 layers that read the
 * same activations (a transformer's q, k and v projections, or its gate and
 * up projections), each quantized on its own (own codes, scales, rows and
 * rotation seed, App. G):
 *   y[l] = x W_hat_l^T,  l < layers.
 * Bit-identical to one higgs_qmatmul_fused call per layer. When the rotation
 * runs inside the small-batch product kernel (see higgs_qmatmul_fused) all
 * layers are computed by ONE launch: each block of the launch takes rows of
 * one layer, so the launch and prologue cost is paid once. On the
 * matrix-core path the layers share one activation conversion
 * launch (one rotated copy per distinct seed), one product launch and at most
 * one reduction launch per 64 batch rows. Otherwise the layers are computed
 * one after another on the stream, sharing the workspace.
 *
 *   layers     1..4.
 *   x          [in]  device, batch*in values of x_dtype, row-major, shared.
 *   codes, scales, rht_seeds, out, y
 *              [in]  HOST arrays of `layers` entries: layer l's device codes
 *                    and scales (as for higgs_qmatmul), rotation seed, rows,
 *                    and device output (batch*out[l] floats).
 *   grid, p, n, g, in: shared by the layers.
 *   workspace  [in]  device scratch of at least
 *                    higgs_qmatmul_fused_multi_workspace_bytes(...) bytes
 *                    (may be NULL when that is 0).
 * Requirements and errors per layer as for higgs_qmatmul_fused; layers
 * outside 1..4 or a NULL array return HIGGS_ERR_INVALID_ARG. Outputs must
 * not overlap each other or x. The workspace query (host, pure) takes the
 * host array out[layers] and returns -1 for invalid arguments.
 * ------------------------------------------------------------------------- */
int64_t higgs_qmatmul_fused_multi_workspace_bytes(int layers, int64_t batch,
                                                  const int64_t *out, int64_t in, int p, int n,
                                                  int g);

higgs_status higgs_qmatmul_fused_multi(int layers, const void *x, higgs_dtype x_dtype,
                                       int64_t batch, const uint8_t *const *codes,
                                       const uint16_t *const *scales, const float *grid, int p,
                                       int n, int g, const uint64_t *rht_seeds,
                                       const int64_t *out, int64_t in, float *const *y,
                                       void *workspace, int64_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* HIGGS_H_ */
