"""CPU oracle for the HIGGS inference path (test infrastructure only).

This is a plain, slow, fp64 NumPy implementation of what the quantized
linear-layer path computes. It exists to check the HIP library: only the
tests, the smoke check and the benchmark's CPU-baseline leg use it. The
product path never imports it, and it shares no code, table or constant
generator with the library.

Every function cites the passage of the paper (arXiv 2411.17525, "Pushing
the Limits of Large Language Model Quantization via the Linearity Theorem")
that it follows. Conventions the paper leaves open are fixed here and listed
with the reason in the design notes:

* the Hadamard matrix is the unnormalised Sylvester matrix in natural order;
* the rotation of a group is R = H diag(sigma) / sqrt(g); one sign vector
  sigma of length g is shared by every group, row and activation block;
* sigma_j = +1 when the top bit of the j-th splitmix64 output (state started
  at the seed) is 0, else -1;
* codes are 0-based; ties in the nearest-point search go to the lowest
  index; consecutive rotated coordinates [j*p, (j+1)*p) form one p-vector;
* the stored scale is fp16(round-to-nearest-even of s / sqrt(g)), converted
  from fp64 in one step; codes use the exact s;
* codes are packed LSB-first, log2(n) bits each, row after row;
* the grid is built by seeded Lloyd iterations on N Gaussian p-vectors drawn
  by splitmix64 + Box-Muller (the paper uses CLVQ, whose steps it does not
  give, and does not print its grids).

Parity status: exact grid values, the sign mapping and the Hadamard order are
conventions; the paper fixes none of them ("parity unpinned" for those three
choices). Everything else is pinned by the CPU tests against closed forms,
library routines, brute force and the bits-per-weight figures the paper
prints.
"""
from __future__ import annotations

import math

import numpy as np

MASK64 = (1 << 64) - 1
_GAMMA = 0x9E3779B97F4A7C15
_MIX1 = 0xBF58476D1CE4E5B9
_MIX2 = 0x94D049BB133111EB


# ---------------------------------------------------------------------------
# Random numbers (the rotation seed xi of Alg. 1, and the grid's samples)
# ---------------------------------------------------------------------------

def splitmix64(seed: int, count: int, start: int = 0) -> np.ndarray:
    """Outputs start .. start+count-1 of splitmix64 (Steele, Lea & Flood, 2014).

    The generator is counter based: output j mixes state seed + (j+1)*gamma.
    """
    j = np.arange(start + 1, start + count + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(seed & MASK64) + j * np.uint64(_GAMMA)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(_MIX1)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(_MIX2)
        z = z ^ (z >> np.uint64(31))
    return z


def rht_signs(seed: int, g: int) -> np.ndarray:
    """The diagonal sign vector of the random Hadamard transform (Alg. 1, seed xi).

    sigma_j = +1 if the top bit of splitmix64 output j is 0, else -1.
    """
    z = splitmix64(seed, g)
    return np.where((z >> np.uint64(63)) == 0, 1, -1).astype(np.int8)


def uniforms(seed: int, count: int) -> np.ndarray:
    """53-bit uniforms in [0, 1): (z >> 11) * 2^-53."""
    z = splitmix64(seed, count)
    return (z >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)


def gaussian_samples(seed: int, num: int, p: int) -> np.ndarray:
    """num standard-normal p-vectors, row-major (num, p), by Box-Muller.

    Normals come in pairs from consecutive uniforms (u1, u2):
    r = sqrt(-2 ln(1 - u1)), theta = 2 pi u2, giving r cos(theta), r sin(theta).
    """
    total = num * p
    pairs = (total + 1) // 2
    u = uniforms(seed, 2 * pairs)
    u1 = u[0::2]
    u2 = u[1::2]
    r = np.sqrt(-2.0 * np.log(1.0 - u1))
    theta = 2.0 * math.pi * u2
    out = np.empty(2 * pairs, dtype=np.float64)
    out[0::2] = r * np.cos(theta)
    out[1::2] = r * np.sin(theta)
    return out[:total].reshape(num, p)


# ---------------------------------------------------------------------------
# Grid: MSE-optimal Gaussian grid G_n^p (Sec. 3.2, Alg. 2; built once per (n, p))
# ---------------------------------------------------------------------------

def nearest(points: np.ndarray, grid: np.ndarray, chunk: int = 4096,
            with_gap: bool = True):
    """Brute-force nearest grid point for each row of points.

    Squared Euclidean distance d_k = sum_t (v_t - G_kt)^2 (terms added in
    order t = 0, 1, ...), first index on ties. Returns (index, best distance,
    gap from the best to the second-best distance; None if not asked for).
    """
    points = np.asarray(points, dtype=np.float64)
    grid = np.asarray(grid, dtype=np.float64)
    m, p = points.shape
    idx = np.empty(m, dtype=np.int64)
    best = np.empty(m, dtype=np.float64)
    gap = np.empty(m, dtype=np.float64) if with_gap else None
    for a in range(0, m, chunk):
        v = points[a:a + chunk]
        rows = np.arange(len(v))
        d = (v[:, 0:1] - grid[None, :, 0]) ** 2
        for t in range(1, p):
            d += (v[:, t:t + 1] - grid[None, :, t]) ** 2
        k = np.argmin(d, axis=1)
        idx[a:a + chunk] = k
        b = d[rows, k]
        best[a:a + chunk] = b
        if with_gap:
            if grid.shape[0] > 1:
                d[rows, k] = np.inf
                gap[a:a + chunk] = d.min(axis=1) - b
            else:
                gap[a:a + chunk] = np.inf
    return idx, best, gap


def code_distances(points: np.ndarray, grid: np.ndarray, codes: np.ndarray) -> np.ndarray:
    """Squared Euclidean distance from each point to the grid point its code
    names, with the terms added in the same order as in nearest(). Where
    several codes are acceptable (a near-tie), this is what a candidate code
    is judged by: its distance against the best one."""
    points = np.asarray(points, dtype=np.float64)
    grid = np.asarray(grid, dtype=np.float64)
    q = grid[np.asarray(codes, dtype=np.int64)]
    d = (points[:, 0] - q[:, 0]) ** 2
    for t in range(1, points.shape[1]):
        d += (points[:, t] - q[:, t]) ** 2
    return d


def lloyd_grid(p: int, n: int, seed: int, num_samples: int = 1 << 20,
               max_iters: int = 300):
    """Lloyd's algorithm for an n-point grid minimising E||x - Q(x)||^2, x ~ N(0, I_p).

    Start: the first n samples. Each iteration assigns every sample to its
    nearest point and then moves each point to the mean of its cell (a cell
    with no sample keeps its point). Stops when an assignment repeats the
    previous one, or after max_iters mean updates.

    Returns (grid (n, p) fp64, per-dimension MSE of the final grid on the
    samples, number of mean updates done).
    """
    x = gaussian_samples(seed, num_samples, p)
    grid = x[:n].copy()
    prev = None
    iters = 0
    while True:
        assign, _, _ = nearest(x, grid, with_gap=False)
        if prev is not None and np.array_equal(assign, prev):
            break
        if iters >= max_iters:
            break
        counts = np.bincount(assign, minlength=n)
        new = grid.copy()
        for t in range(p):
            sums = np.bincount(assign, weights=x[:, t], minlength=n)
            nz = counts > 0
            new[nz, t] = sums[nz] / counts[nz]
        grid = new
        prev = assign
        iters += 1
    _, best, _ = nearest(x, grid, with_gap=False)
    mse = float(best.sum() / (num_samples * p))
    return grid, mse, iters


def grid_mse(grid: np.ndarray, samples: np.ndarray) -> float:
    """Per-dimension MSE of rounding the given samples to the grid."""
    _, best, _ = nearest(samples, grid, with_gap=False)
    return float(best.sum() / (samples.shape[0] * samples.shape[1]))


def uniform_grid_mse(n: int, step: float) -> float:
    """E[(X - Q(X))^2] for X ~ N(0, 1) and Q rounding to the nearest of the n
    points step * (k - (n - 1) / 2): the integral of (x - c_k)^2 phi(x) over
    each point's cell (bounded by the midpoints between points), by numerical
    quadrature (scipy.integrate.quad), summed over the cells."""
    from scipy import integrate

    def density(x):
        return math.exp(-0.5 * x * x) / math.sqrt(2.0 * math.pi)

    total = 0.0
    for k in range(n):
        c = step * (k - 0.5 * (n - 1))
        lo = -math.inf if k == 0 else step * (k - 0.5 * n)
        hi = math.inf if k == n - 1 else step * (k + 1 - 0.5 * n)
        val, _ = integrate.quad(lambda x: (x - c) ** 2 * density(x), lo, hi,
                                epsabs=1e-15, epsrel=1e-13, limit=200)
        total += val
    return total


def uniform_grid(n: int):
    """The CH8-style grid of Sec. 3.3: a uniform grid whose position and
    scale minimise the expected squared error over N(0, 1). For the symmetric
    density the optimal uniform grid is symmetric about 0, so only the step is
    free: minimise uniform_grid_mse(n, step) over the step (bounded scalar
    minimisation, scipy.optimize.minimize_scalar).

    Returns (points (n,) fp64, step, mse)."""
    from scipy import optimize

    res = optimize.minimize_scalar(lambda st: uniform_grid_mse(n, st), bounds=(1e-4, 4.0),
                                   method="bounded", options={"xatol": 1e-12, "maxiter": 500})
    step = float(res.x)
    points = step * (np.arange(n, dtype=np.float64) - 0.5 * (n - 1))
    return points, step, uniform_grid_mse(n, step)


# ---------------------------------------------------------------------------
# Hadamard transform (Alg. 1; App. G)
# ---------------------------------------------------------------------------

def hadamard(g: int) -> np.ndarray:
    """Unnormalised Sylvester Hadamard matrix of order g (a power of 2), fp64."""
    if g < 1 or g & (g - 1):
        raise ValueError("g must be a power of 2")
    h = np.ones((1, 1), dtype=np.float64)
    while h.shape[0] < g:
        h = np.kron(np.array([[1.0, 1.0], [1.0, -1.0]]), h)
    return h


def bits_per_code(n: int) -> int:
    b = int(round(math.log2(n)))
    if 1 << b != n:
        raise ValueError("n must be a power of 2 for packed codes")
    return b


def bits_per_weight(p: int, n: int, g: int) -> float:
    """Storage cost: log2(n)/p bits of code plus one 16-bit scale per g weights (App. H)."""
    return math.log2(n) / p + 16.0 / g


# ---------------------------------------------------------------------------
# Alg. 1 (RHT-VQ): rotate, scale and round one layer
# ---------------------------------------------------------------------------

def rotate_groups(w_rows: np.ndarray, g: int, seed: int):
    """Per group: s = ||w||_2 and w_dag = H (sigma * (w / s)) (Alg. 1).

    w_rows: (rows, in). Returns (s of shape (rows, in/g), w_dag of shape
    (rows, in/g, g)). A group with s = 0 gets w_dag = 0.
    """
    rows, inp = w_rows.shape
    if inp % g:
        raise ValueError("in must be a multiple of g")
    h = hadamard(g)
    sigma = rht_signs(seed, g).astype(np.float64)
    w = np.asarray(w_rows, dtype=np.float64).reshape(rows, inp // g, g)
    s = np.sqrt((w * w).sum(axis=2))
    safe = np.where(s > 0, s, 1.0)
    unit = w / safe[:, :, None]                        # w_i / s_i
    w_dag = (unit * sigma[None, None, :]) @ h.T        # H (sigma * (w_i / s_i))
    w_dag[s == 0] = 0.0
    return s, w_dag


def f64_to_f16(x: np.ndarray) -> np.ndarray:
    """fp64 -> fp16, round to nearest even, in one step (NumPy's cast)."""
    return np.asarray(x, dtype=np.float64).astype(np.float16)


def quantize(w_rows: np.ndarray, grid: np.ndarray, g: int, seed: int):
    """HIGGS quantization of a layer (Alg. 1 with the grid of Alg. 2).

    w_rows: (rows, in) with exact input values; grid: (n, p).
    Returns a dict with
      codes  (rows, in/p) int64, 0-based, nearest p-vector of the grid;
      best   (rows, in/p) the nearest point's squared distance;
      gap    (rows, in/p) second-best minus best squared distance;
      scales (rows, in/g) fp16 = fp16(s / sqrt(g));
      s      (rows, in/g) fp64 exact group norms;
      w_dag  (rows, in/g, g) rotated unit-norm-times-sqrt(g) groups.
    """
    grid = np.asarray(grid, dtype=np.float64)
    n, p = grid.shape
    if g % p:
        raise ValueError("g must be a multiple of p")
    rows, inp = w_rows.shape
    s, w_dag = rotate_groups(w_rows, g, seed)
    vecs = w_dag.reshape(-1, p)
    idx, best, gap = nearest(vecs, grid)
    scales = f64_to_f16(s / np.sqrt(float(g)))
    return {
        "codes": idx.reshape(rows, inp // p),
        "best": best.reshape(rows, inp // p),
        "gap": gap.reshape(rows, inp // p),
        "scales": scales,
        "s": s,
        "w_dag": w_dag,
    }


def pack_codes(codes: np.ndarray, n: int) -> np.ndarray:
    """Pack 0-based codes LSB-first: code m of a row fills bits [m*b, (m+1)*b).

    Bit t of the row's stream is bit (t mod 8) of byte floor(t / 8).
    codes: (rows, codes_per_row); the row's bit count must be a multiple of 8.
    """
    b = bits_per_code(n)
    rows, m = codes.shape
    if (m * b) % 8:
        raise ValueError("row does not fill whole bytes")
    bits = np.zeros((rows, m * b), dtype=np.uint8)
    c = np.asarray(codes, dtype=np.int64)
    for t in range(b):
        bits[:, t::b] = (c >> t) & 1
    return np.packbits(bits, axis=1, bitorder="little")


def unpack_codes(packed: np.ndarray, n: int, codes_per_row: int) -> np.ndarray:
    b = bits_per_code(n)
    bits = np.unpackbits(np.asarray(packed, dtype=np.uint8), axis=1, bitorder="little")
    bits = bits[:, :codes_per_row * b].astype(np.int64)
    codes = np.zeros((packed.shape[0], codes_per_row), dtype=np.int64)
    for t in range(b):
        codes |= bits[:, t::b] << t
    return codes


def codes_row_bytes(inp: int, p: int, n: int) -> int:
    return inp // p * bits_per_code(n) // 8


# ---------------------------------------------------------------------------
# App. G: dequantization in the original space, and the reference product
# ---------------------------------------------------------------------------

def dequantize(codes: np.ndarray, scales_f16: np.ndarray, grid: np.ndarray, g: int,
               seed: int) -> np.ndarray:
    """W_hat[o, block i] = scale[o, i] * sigma * (H concat_j G[q_oij]) / sqrt(g).

    This is the inverse rotation R^-1 = diag(sigma) H / sqrt(g) applied to the
    looked-up grid points, then the stored scale (App. G, dequantization paragraph).
    codes: (rows, in/p); scales_f16: (rows, in/g) fp16.
    """
    grid = np.asarray(grid, dtype=np.float64)
    n, p = grid.shape
    rows, m = codes.shape
    inp = m * p
    h = hadamard(g)
    sigma = rht_signs(seed, g).astype(np.float64)
    q = grid[np.asarray(codes, dtype=np.int64)].reshape(rows, inp // g, g)
    back = (q @ h.T) * sigma[None, None, :] / math.sqrt(g)
    sc = np.asarray(scales_f16, dtype=np.float16).astype(np.float64)
    return (back * sc[:, :, None]).reshape(rows, inp)


def rht_activations(x: np.ndarray, g: int, seed: int) -> np.ndarray:
    """x_rot[b, block i] = H (sigma * x[b, block i]) / sqrt(g) (App. G, rotating activations)."""
    x = np.asarray(x, dtype=np.float64)
    batch, inp = x.shape
    if inp % g:
        raise ValueError("in must be a multiple of g")
    h = hadamard(g)
    sigma = rht_signs(seed, g).astype(np.float64)
    xb = x.reshape(batch, inp // g, g) * sigma[None, None, :]
    return (xb @ h.T / math.sqrt(g)).reshape(batch, inp)


def qmatmul(x: np.ndarray, codes: np.ndarray, scales_f16: np.ndarray, grid: np.ndarray,
            g: int, seed: int) -> np.ndarray:
    """Reference layer output y = x W_hat^T in fp64, in the original space.

    x: (batch, in) activations (not rotated). Returns (batch, rows).
    """
    w_hat = dequantize(codes, scales_f16, grid, g, seed)
    return np.asarray(x, dtype=np.float64) @ w_hat.T


def layer_error(w: np.ndarray, w_hat: np.ndarray) -> float:
    """Relative squared Frobenius error t_l^2 = ||W_hat - W||_F^2 / ||W||_F^2 (Thm. 1)."""
    w = np.asarray(w, dtype=np.float64)
    return float(((w_hat - w) ** 2).sum() / (w ** 2).sum())


# ---------------------------------------------------------------------------
# Variable bitwidth (Sec. 4): per-layer quantizer choice under a budget
# ---------------------------------------------------------------------------

def allocate_bits_brute(alpha, t2, bits, sizes, b_max: float):
    """Eq. (objective) of Sec. 4 by enumeration: over every assignment j_1..j_L
    of options to layers with sum_l bits[j_l] * d_l <= b_max * sum_l d_l,
    the least sum_l alpha_l * t2[l][j_l]. For small L only (J^L assignments).

    Returns (best objective, list of every optimal assignment as tuples, the
    optimal assignments' average bits per weight); objective None when no
    assignment fits."""
    import itertools
    alpha = np.asarray(alpha, dtype=np.float64)
    t2 = np.asarray(t2, dtype=np.float64)
    bits = np.asarray(bits, dtype=np.float64)
    sizes = np.asarray(sizes, dtype=np.float64)
    L, J = t2.shape
    budget = b_max * sizes.sum()
    best, arg = None, []
    for ch in itertools.product(range(J), repeat=L):
        cost = sum(bits[j] * sizes[l] for l, j in enumerate(ch))
        if cost > budget:
            continue
        obj = sum(alpha[l] * t2[l, j] for l, j in enumerate(ch))
        if best is None or obj < best * (1 - 1e-12):
            best, arg = obj, [ch]
        elif obj <= best * (1 + 1e-12):
            arg.append(ch)
    avg = [sum(bits[j] * sizes[l] for l, j in enumerate(ch)) / sizes.sum() for ch in arg]
    return best, arg, avg


# ---------------------------------------------------------------------------
# GPTQ rounding in place of the nearest-point step (Sec. 3.5)
# ---------------------------------------------------------------------------

def gptq_factor(x_rot, damp: float = 0.01) -> np.ndarray:
    """Upper triangular U with (H + damp * mean(diag H) * I)^-1 = U^T U, where
    H = X'^T X' over the rotated calibration activations X' (samples, in).
    GPTQ's damped Hessian and the Cholesky factor of its inverse (fp64: the
    plain inverse, then numpy's Cholesky)."""
    x = np.asarray(x_rot, dtype=np.float64)
    h = x.T @ x
    h[np.diag_indices_from(h)] += damp * float(np.mean(np.diag(h)))
    hinv = np.linalg.inv(h)
    hinv = 0.5 * (hinv + hinv.T)
    return np.linalg.cholesky(hinv).T


def rotated_weights(w_rows: np.ndarray, g: int, seed: int):
    """W' = per group H (sigma * w) / sqrt(g) (the orthonormal rotation R of
    App. G applied to each group) and the group norms s."""
    rows, inp = w_rows.shape
    h = hadamard(g)
    sigma = rht_signs(seed, g).astype(np.float64)
    w = np.asarray(w_rows, dtype=np.float64).reshape(rows, inp // g, g)
    s = np.sqrt((w * w).sum(axis=2))
    wr = ((w * sigma[None, None, :]) @ h.T) / math.sqrt(g)
    return wr.reshape(rows, inp), s


def quantize_gptq(w_rows: np.ndarray, grid: np.ndarray, g: int, seed: int, u: np.ndarray,
                  follow=None, follow_tol: float = 0.0):
    """HIGGS with GPTQ rounding (Sec. 3.5): Alg. 1's normalisation and output
    format, with the rounding of each p-vector feeding its error forward.

    In the rotated space, column p-vectors are taken in order. For p-vector
    j (columns c = [jp, (j+1)p)) of every row: v = W'[:, c]; its code is the
    nearest grid point of v sqrt(g) / s (s the group's norm; lowest index on
    ties); the error e = v - (s / sqrt(g)) G[code] is scaled, E = e
    U[c, c]^-1, and every later column moves: W'[:, later] -= E U[c, later].

    follow: optional candidate codes (rows, in/p) from another implementation.
    Where a candidate differs from the nearest point but its squared distance
    (grid units) is within follow_tol of the best, the rounding is ambiguous
    and the recursion continues from the candidate, so the later columns are
    still compared; a candidate outside that band is recorded in "mismatch"
    and the oracle keeps its own code. Without follow the result is the plain
    recursion above.

    Returns codes (rows, in/p), gap (rows, in/p) of each rounding, scales
    (fp16(s / sqrt(g))), the original rotated weights, the scaled errors E
    (rows, in), the dequantised rotated weights and mismatch (rows, in/p)."""
    grid = np.asarray(grid, dtype=np.float64)
    n, p = grid.shape
    rows, inp = w_rows.shape
    w0, s = rotated_weights(w_rows, g, seed)
    w = w0.copy()
    codes = np.zeros((rows, inp // p), dtype=np.int64)
    gaps = np.zeros((rows, inp // p))
    errs = np.zeros((rows, inp))
    deq = np.zeros((rows, inp))
    mismatch = np.zeros((rows, inp // p), dtype=bool)
    for j in range(inp // p):
        c = slice(j * p, (j + 1) * p)
        sg = s[:, (j * p) // g]
        v = w[:, c]
        unit = np.where(sg[:, None] > 0, v * math.sqrt(g) / np.where(sg > 0, sg, 1.0)[:, None],
                        0.0)
        idx, best, gap = nearest(unit, grid)
        if follow is not None:
            cand = np.asarray(follow[:, j], dtype=np.int64)
            tie = (cand != idx) & (code_distances(unit, grid, cand) - best <= follow_tol)
            mismatch[:, j] = (cand != idx) & ~tie
            idx = np.where(tie, cand, idx)
        codes[:, j], gaps[:, j] = idx, gap
        q = (sg / math.sqrt(g))[:, None] * grid[idx]
        deq[:, c] = q
        e = v - q
        es = e @ np.linalg.inv(u[c, c])
        errs[:, c] = es
        w[:, (j + 1) * p:] -= es @ u[c, (j + 1) * p:]
    return {"codes": codes, "gap": gaps, "scales": f64_to_f16(s / math.sqrt(float(g))),
            "w_rot": w0, "err_scaled": errs, "deq_rot": deq, "mismatch": mismatch}

