"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these checks re-derive a value through the oracle's own formula:
they use closed forms, independent library routines (SciPy's Hadamard
matrix, normal CDF), brute force, published generator test vectors and the
bits-per-weight figures the paper prints.
"""
import math
import os

import numpy as np
import pytest
import scipy.linalg
import scipy.stats

from conftest import GOLDEN, load_grid_fixture
from oracle import higgs_oracle as O


# --------------------------------------------------------------------------
# splitmix64 and the Gaussian sampler
# --------------------------------------------------------------------------

def test_splitmix64_published_vectors():
    # The generator's widely published check outputs (Steele, Lea & Flood
    # 2014; the same values appear in every public implementation's tests).
    assert [int(v) for v in O.splitmix64(1234567, 5)] == [
        6457827717110365317, 3203168211198807973, 9817491932198370423,
        4593380528125082431, 16408922859458223821]
    assert int(O.splitmix64(0, 1)[0]) == 0xE220A8397B1DCDAF
    # counter form: skipping ahead equals continuing the stream
    full = O.splitmix64(42, 20)
    assert np.array_equal(full[7:], O.splitmix64(42, 13, start=7))


def test_sign_vector_balanced_and_seeded():
    s = O.rht_signs(7, 4096)
    assert set(np.unique(s)) <= {-1, 1}
    assert abs(int(s.sum())) < 4 * math.sqrt(4096)
    assert not np.array_equal(O.rht_signs(7, 64), O.rht_signs(8, 64))
    # sigma_j depends on the top bit of output j only
    z = O.splitmix64(7, 16)
    for j in range(16):
        assert s[j] == (1 if int(z[j]) < (1 << 63) else -1)


def test_gaussian_samples_are_standard_normal():
    x = O.gaussian_samples(3, 1 << 16, 2)
    for t in range(2):
        res = scipy.stats.kstest(x[:, t], scipy.stats.norm.cdf)
        assert res.pvalue > 1e-4, res
    assert abs(x.mean()) < 0.02
    assert abs(x.var() - 1.0) < 0.02
    # the two coordinates of a vector are uncorrelated
    assert abs(np.corrcoef(x[:, 0], x[:, 1])[0, 1]) < 0.02
    # radius^2 of a 2-d standard normal is exponential with mean 2
    r2 = (x ** 2).sum(axis=1)
    assert scipy.stats.kstest(r2, scipy.stats.expon(scale=2.0).cdf).pvalue > 1e-4


# --------------------------------------------------------------------------
# Hadamard matrix and the random Hadamard transform (Alg. 1, App. G)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("g", [1, 2, 4, 8, 64, 1024])
def test_hadamard_is_sylvester(g):
    h = O.hadamard(g)
    assert np.array_equal(h, scipy.linalg.hadamard(g).astype(np.float64))
    assert np.array_equal(h @ h.T, g * np.eye(g))
    assert np.array_equal(h, h.T)
    # entry (r, c) = (-1)^popcount(r & c)
    r, c = np.meshgrid(np.arange(g), np.arange(g), indexing="ij")
    pc = np.vectorize(lambda v: bin(int(v)).count("1"))(r & c)
    assert np.array_equal(h, np.where(pc % 2 == 0, 1.0, -1.0))
    if g == 2:
        assert np.array_equal(h, np.array([[1.0, 1.0], [1.0, -1.0]]))


@pytest.mark.parametrize("g", [8, 64, 1024])
def test_rht_round_trip_and_norm(g):
    rng = np.random.default_rng(g)
    w = rng.standard_t(5, size=(3, 4 * g))
    w[1, g:2 * g] = 0.0                     # one all-zero group
    s, w_dag = O.rotate_groups(w, g, seed=11)
    assert np.allclose(s, np.sqrt((w.reshape(3, 4, g) ** 2).sum(axis=2)), rtol=1e-15, atol=0)
    # Parseval: every non-zero group has ||w_dag||^2 = g (entries ~ N(0, 1))
    norms = (w_dag ** 2).sum(axis=2)
    nz = s > 0
    assert np.allclose(norms[nz], g, rtol=1e-12)
    assert np.all(w_dag[~nz] == 0)
    # inverse RHT recovers W exactly (before rounding): w = (s/sqrt g) sigma * (H w_dag) / sqrt g
    h = scipy.linalg.hadamard(g).astype(np.float64)
    sigma = O.rht_signs(11, g).astype(np.float64)
    back = (w_dag @ h) * sigma / math.sqrt(g) * (s / math.sqrt(g))[:, :, None]
    err = np.abs(back.reshape(3, -1) - w).max() / np.abs(w).max()
    assert err < 1e-13


def test_one_hot_group_worked_example():
    # w = a e_k  =>  s = |a| and w_dag = sign(a) sigma_k H[:, k], exactly.
    g, k, a = 16, 5, -0.75
    w = np.zeros((1, g))
    w[0, k] = a
    s, w_dag = O.rotate_groups(w, g, seed=3)
    sigma = O.rht_signs(3, g)
    col = np.array([(-1) ** bin(r & k).count("1") for r in range(g)], dtype=np.float64)
    assert s[0, 0] == abs(a)
    assert np.array_equal(w_dag[0, 0], -1.0 * sigma[k] * col)
    # The rotated group holds only the vectors (+-1, +-1); with the 4-point
    # grid {(+-1, +-1)} listed in this order, the code of (u, v) is
    # 2*(u < 0) + (v < 0), worked by hand.
    grid = np.array([[1.0, 1.0], [1.0, -1.0], [-1.0, 1.0], [-1.0, -1.0]])
    q = O.quantize(w, grid, g, seed=3)
    v = w_dag[0, 0].reshape(-1, 2)
    expect = 2 * (v[:, 0] < 0) + (v[:, 1] < 0)
    assert np.array_equal(q["codes"][0], expect)
    assert np.all(q["gap"] > 0)
    # exact reconstruction: the grid contains every rotated vector
    w_hat = O.dequantize(q["codes"], q["scales"], grid, g, seed=3)
    assert np.allclose(w_hat, w, rtol=0, atol=abs(a) * 2 ** -11)


def test_activation_rht_is_orthogonal():
    g = 256
    rng = np.random.default_rng(1)
    x = rng.standard_normal((3, 2 * g))
    xr = O.rht_activations(x, g, seed=9)
    assert np.allclose((xr.reshape(3, 2, g) ** 2).sum(2), (x.reshape(3, 2, g) ** 2).sum(2),
                       rtol=1e-13)
    # one-hot input: x = e_k -> x_rot = sigma_k H[:, k] / sqrt(g)
    e = np.zeros((1, g))
    e[0, 17] = 1.0
    sigma = O.rht_signs(9, g)
    col = scipy.linalg.hadamard(g)[:, 17].astype(np.float64)
    assert np.allclose(O.rht_activations(e, g, 9)[0], sigma[17] * col / math.sqrt(g),
                       rtol=0, atol=1e-15)


# --------------------------------------------------------------------------
# Encoding (Alg. 1): optimality by brute force, zero groups, scales
# --------------------------------------------------------------------------

@pytest.mark.parametrize("p,n,g", [(1, 2, 8), (1, 4, 8), (2, 4, 8), (2, 16, 4), (1, 16, 4),
                                   (2, 2, 8)])
def test_encode_is_optimal_by_brute_force(p, n, g):
    rng = np.random.default_rng(100 * p + n + g)
    grid = rng.standard_normal((n, p))
    w = rng.standard_t(5, size=(3, g))
    q = O.quantize(w, grid, g, seed=5)
    s = np.sqrt((w ** 2).sum(axis=1))
    h = scipy.linalg.hadamard(g).astype(np.float64)
    sigma = O.rht_signs(5, g).astype(np.float64)
    m = g // p
    # enumerate every code vector of a group; reconstruct in the ORIGINAL space
    # with the exact scale s/sqrt(g): w_hat = (s/sqrt g) * sigma * (H G[c]) / sqrt g
    combos = np.array(np.meshgrid(*[np.arange(n)] * m, indexing="ij")).reshape(m, -1).T
    pts = grid[combos].reshape(len(combos), g)
    recon = (pts @ h) * sigma / math.sqrt(g)
    for r in range(3):
        errs = (((s[r] / math.sqrt(g)) * recon - w[r]) ** 2).sum(axis=1)
        mine = (((s[r] / math.sqrt(g)) * recon[np.ravel_multi_index(
            tuple(q["codes"][r]), (n,) * m)] - w[r]) ** 2).sum()
        assert mine <= errs.min() * (1 + 1e-12) + 1e-300


def test_zero_group():
    grid = np.array([[0.5, 0.5], [0.1, -0.1], [-0.1, 0.1], [2.0, 2.0]])
    w = np.zeros((2, 8))
    w[1] = np.arange(8) - 3.5
    q = O.quantize(w, grid, 8, seed=1)
    # zero group: scale 0, every code is the grid point nearest the origin
    # (points 1 and 2 tie at distance 0.02; the lower index wins)
    assert q["scales"][0, 0] == 0
    assert np.all(q["codes"][0] == 1)
    assert np.all(q["gap"][0] == 0)
    w_hat = O.dequantize(q["codes"], q["scales"], grid, 8, seed=1)
    assert np.all(w_hat[0] == 0)


def test_scale_is_fp16_of_fp64_in_one_step():
    # 1 + 2^-11 + 2^-30 lies above the fp16 midpoint 1 + 2^-11, so one-step
    # rounding gives 1 + 2^-10; rounding through fp32 first would give 1.0.
    x = 1.0 + 2.0 ** -11 + 2.0 ** -30
    assert float(O.f64_to_f16(np.array([x]))[0]) == 1.0 + 2.0 ** -10
    assert float(np.float16(np.float32(x))) == 1.0
    # scale of a group with known norm: s = 32 * 3 for g = 1024 -> s/sqrt(g) = 3
    w = np.full((1, 1024), 3.0)
    q = O.quantize(w, np.array([[0.0, 0.0], [1.0, 1.0]]), 1024, seed=0)
    assert q["scales"][0, 0] == np.float16(3.0)


# --------------------------------------------------------------------------
# App. F and App. G identities
# --------------------------------------------------------------------------

def _small_grid(p, n, samples=1 << 13, seed=0):
    fx = load_grid_fixture(p, n)
    if fx is not None:
        return fx[0]
    return O.lloyd_grid(p, n, seed, samples, 100)[0]


def test_layer_error_equals_rotated_space_error():
    grid = _small_grid(2, 64)
    g = 256
    rng = np.random.default_rng(4)
    w = rng.standard_t(5, size=(8, 2 * g)) * 0.02
    q = O.quantize(w, grid, g, seed=2)
    w_hat = O.dequantize(q["codes"], q["scales"], grid, g, seed=2)
    direct = ((w - w_hat) ** 2).sum()
    sc = q["scales"].astype(np.float64)
    pts = grid[q["codes"]].reshape(8, 2, g)
    rot = ((sc[:, :, None] * pts - (q["s"] / math.sqrt(g))[:, :, None] * q["w_dag"]) ** 2).sum()
    assert abs(direct - rot) <= 1e-10 * direct


def test_rotated_space_product_equals_original_space():
    # App. G: multiply in the rotated space with the same seed on activations.
    grid = _small_grid(2, 256)
    g = 128
    rng = np.random.default_rng(5)
    w = rng.standard_t(5, size=(16, 3 * g)) * 0.02
    x = rng.standard_normal((4, 3 * g))
    q = O.quantize(w, grid, g, seed=13)
    y = O.qmatmul(x, q["codes"], q["scales"], grid, g, seed=13)
    xr = O.rht_activations(x, g, seed=13).reshape(4, 3, g)
    pts = grid[q["codes"]].reshape(16, 3, g)
    sc = q["scales"].astype(np.float64)
    y_rot = np.einsum("bif,oif,oi->bo", xr, pts, sc)
    assert np.abs(y - y_rot).max() <= 1e-12 * np.abs(y).max()


def test_app_f_error_matches_grid_mse():
    # t_l^2 ~= per-dimension MSE of the grid on N(0, I_p), independent of W.
    fx = load_grid_fixture(2, 256)
    grid = fx[0] if fx is not None else O.lloyd_grid(2, 256, 0, 1 << 14, 150)[0]
    mse = O.grid_mse(grid, O.gaussian_samples(999, 1 << 16, 2))
    rng = np.random.default_rng(6)
    g = 1024
    w = rng.standard_normal((128, g))
    q = O.quantize(w, grid, g, seed=1)
    t2 = O.layer_error(w, O.dequantize(q["codes"], q["scales"], grid, g, seed=1))
    assert abs(t2 / mse - 1) < 0.05, (t2, mse)
    # heavy-tailed weights give a similar error after the rotation
    wt = rng.standard_t(5, size=(128, g))
    qt = O.quantize(wt, grid, g, seed=1)
    t2t = O.layer_error(wt, O.dequantize(qt["codes"], qt["scales"], grid, g, seed=1))
    assert abs(t2t / mse - 1) < 0.10, (t2t, mse)


# --------------------------------------------------------------------------
# Grids (Sec. 3.2): closed forms, textbook values, invariants
# --------------------------------------------------------------------------

def _lloyd_max_exact(levels, iters=20000):
    """Exact Lloyd-Max quantizer of N(0, 1) by the centroid / midpoint conditions."""
    c = np.linspace(-2.5, 2.5, levels)
    pdf, cdf = scipy.stats.norm.pdf, scipy.stats.norm.cdf
    for _ in range(iters):
        t = np.concatenate([[-np.inf], (c[:-1] + c[1:]) / 2, [np.inf]])
        mass = cdf(t[1:]) - cdf(t[:-1])
        c = (pdf(t[:-1]) - pdf(t[1:])) / mass
    t = np.concatenate([[-np.inf], (c[:-1] + c[1:]) / 2, [np.inf]])
    mass = cdf(t[1:]) - cdf(t[:-1])
    mse = 1.0 - ((pdf(t[:-1]) - pdf(t[1:])) ** 2 / mass).sum()
    return c, mse


def test_grid_two_points_closed_form():
    grid, mse, _ = O.lloyd_grid(1, 2, seed=1, num_samples=1 << 16, max_iters=50)
    pts = np.sort(grid[:, 0])
    a = math.sqrt(2 / math.pi)
    assert np.allclose(pts, [-a, a], rtol=0.01)
    assert abs(mse - (1 - 2 / math.pi)) < 0.005


def test_grid_sixteen_levels_matches_lloyd_max():
    c, mse_exact = _lloyd_max_exact(16)
    assert abs(mse_exact - 0.009497) < 2e-5          # Max (1960), 16 levels
    fx = load_grid_fixture(1, 16)
    if fx is not None:
        grid = fx[0]
    else:
        grid = O.lloyd_grid(1, 16, 0, 1 << 16, 300)[0]
    mse = O.grid_mse(grid, O.gaussian_samples(12345, 1 << 17, 1))
    assert abs(mse / mse_exact - 1) < 0.03, (mse, mse_exact)
    assert np.allclose(np.sort(grid[:, 0]), c, atol=0.06)


def test_grid_p2_between_shannon_and_product_bounds():
    for n, levels in [(64, 8), (256, 16)]:
        grid = _small_grid(2, n)
        mse = O.grid_mse(grid, O.gaussian_samples(777, 1 << 15, 2))
        shannon = 2.0 ** (-2 * math.log2(n) / 2)
        product = _lloyd_max_exact(levels, 5000)[1]
        assert shannon < mse < product, (n, shannon, mse, product)


def test_grid_fixed_point_and_energy_identity():
    x = O.gaussian_samples(21, 4096, 2)
    grid, mse, iters = O.lloyd_grid(2, 16, seed=21, num_samples=4096, max_iters=1000)
    assert iters < 1000                                  # converged: assignment repeated
    idx, best, _ = O.nearest(x, grid)
    for k in range(16):
        cell = x[idx == k]
        assert len(cell) > 0
        assert np.allclose(grid[k], cell.mean(axis=0), rtol=0, atol=1e-12)
    q = grid[idx]
    lhs = (q ** 2).sum(axis=1).mean()
    rhs = (x ** 2).sum(axis=1).mean() - 2 * mse
    assert abs(lhs - rhs) < 1e-10
    assert abs(best.mean() / 2 - mse) < 1e-15


def test_grid_mse_decreases_with_n():
    samples = O.gaussian_samples(31, 1 << 14, 2)
    mses = []
    for n in (4, 16, 64):
        grid = O.lloyd_grid(2, n, seed=3, num_samples=1 << 13, max_iters=60)[0]
        mses.append(O.grid_mse(grid, samples))
    fx = load_grid_fixture(2, 256)
    if fx is not None:
        mses.append(O.grid_mse(fx[0], samples))
    assert all(a > b for a, b in zip(mses, mses[1:])), mses


# --------------------------------------------------------------------------
# Storage format: bits per weight (App. H) and packing
# --------------------------------------------------------------------------

# ---------------------------------------------------------------------------
# Uniform grid of the CH8 format (Sec. 3.3)
# ---------------------------------------------------------------------------

def test_uniform_grid_two_points_closed_form():
    """With two points the optimal quantizer is uniform: +-sqrt(2/pi), MSE 1 - 2/pi."""
    pts, step, mse = O.uniform_grid(2)
    assert abs(step / (2 * math.sqrt(2 / math.pi)) - 1) < 1e-6
    assert abs(mse - (1 - 2 / math.pi)) < 1e-9
    assert np.allclose(pts, [-step / 2, step / 2])


@pytest.mark.parametrize("n,step_ref,mse_ref", [(4, 0.9957, 0.1188), (8, 0.5860, 0.03744),
                                                (16, 0.3352, 0.01154)])
def test_uniform_grid_matches_max_1960(n, step_ref, mse_ref):
    """Optimum uniform quantizers of N(0, 1) as tabulated by Max (1960)."""
    pts, step, mse = O.uniform_grid(n)
    assert abs(step / step_ref - 1) < 5e-4
    assert abs(mse / mse_ref - 1) < 5e-4
    assert np.allclose(pts, step * (np.arange(n) - (n - 1) / 2), rtol=0, atol=1e-15)


def test_uniform_grid_mse_by_sampling():
    """Rounding seeded Gaussian samples to the 256-point grid reproduces the
    quadrature MSE (an estimate independent of the integration)."""
    pts, step, mse = O.uniform_grid(256)
    x = O.gaussian_samples(99, 1 << 20, 1)
    emp = O.grid_mse(pts[:, None], x)
    assert abs(emp / mse - 1) < 0.01, (emp, mse)


def test_uniform_grid_is_feasible_lloyd_max_is_lower():
    """A uniform grid is one of the grids Lloyd-Max optimises over, so its MSE
    is at least the optimum's; both fall as n grows."""
    _, lloyd_max = _lloyd_max_exact(16)
    assert lloyd_max < O.uniform_grid(16)[2]
    ms = [O.uniform_grid(n)[2] for n in (2, 4, 8, 16, 32)]
    assert all(a > b for a, b in zip(ms, ms[1:]))


# ---------------------------------------------------------------------------
# Variable bitwidth (Sec. 4)
# ---------------------------------------------------------------------------

def test_allocation_hand_example():
    """Two layers, two options (2 and 4 bits), b_max = 3: (4, 2) bits cost 6
    and score 0.1 + 0.3; (2, 4) also fits and scores 0.6; (2, 2) scores 0.7;
    (4, 4) does not fit."""
    best, arg, avg = O.allocate_bits_brute([1.0, 1.0], [[0.4, 0.1], [0.3, 0.2]], [2.0, 4.0],
                                           [1, 1], 3.0)
    assert abs(best - 0.4) < 1e-15 and arg == [(1, 0)] and avg == [3.0]


def _random_instance(seed, L=5, J=4):
    rng = np.random.default_rng(seed)
    t2 = np.sort(rng.uniform(1e-3, 5e-2, (L, J)), axis=1)[:, ::-1]  # more bits, less error
    alpha = rng.uniform(0.2, 3.0, L)
    bits = np.array([3.25, 4.015625, 5.015625, 8.015625])[:J]
    sizes = rng.integers(1, 15, L) * (1 << 22)
    return alpha, t2, bits, sizes


def test_allocation_extreme_budgets():
    alpha, t2, bits, sizes = _random_instance(3)
    # budget for everything: every layer takes its least-error option
    best, _, _ = O.allocate_bits_brute(alpha, t2, bits, sizes, bits.max())
    assert abs(best - (alpha * t2.min(axis=1)).sum()) < 1e-15
    # budget for the cheapest option only
    best, arg, _ = O.allocate_bits_brute(alpha, t2, bits, sizes, bits.min())
    assert arg == [tuple([int(np.argmin(bits))] * len(alpha))]
    # below every assignment: nothing fits
    assert O.allocate_bits_brute(alpha, t2, bits, sizes, bits.min() * 0.99)[0] is None


@pytest.mark.parametrize("seed", [1, 2, 5])
def test_allocation_respects_lagrangian_bound(seed):
    """Weak duality: for every lam >= 0, sum_l min_j (alpha_l t2_lj + lam bits_j
    d_l) - lam b_max D <= optimum <= the objective of any fitting assignment."""
    alpha, t2, bits, sizes = _random_instance(seed)
    b_max = 4.4
    best, arg, avg = O.allocate_bits_brute(alpha, t2, bits, sizes, b_max)
    assert all(a <= b_max + 1e-12 for a in avg)
    D = sizes.sum()
    for lam in np.linspace(0.0, 2e-9, 21):
        dual = (alpha[:, None] * t2 + lam * bits[None, :] * sizes[:, None]).min(axis=1).sum() \
            - lam * b_max * D
        assert dual <= best * (1 + 1e-12)
    cheapest = (alpha * t2[:, int(np.argmin(bits))]).sum()
    assert best <= cheapest


# ---------------------------------------------------------------------------
# GPTQ rounding (Sec. 3.5)
# ---------------------------------------------------------------------------

def _gptq_case(seed, rows=12, inp=128, g=64, samples=512, mix=True):
    rng = np.random.default_rng(seed)
    w = rng.standard_normal((rows, inp)) * 0.02
    x = rng.standard_normal((samples, inp))
    if mix:  # correlated inputs: a random mixing of the features
        x = x @ (np.eye(inp) + 0.8 * rng.standard_normal((inp, inp)) / math.sqrt(inp))
    return w, x


@pytest.mark.parametrize("p,n", [(1, 16), (2, 64)])
def test_gptq_error_identity(p, n):
    """The recursion's bookkeeping: W'_orig - W'_hat = E U (U upper), so the
    damped proxy loss tr(dW H dW^T) equals ||E||^2. A dropped term, a wrong
    index or a transposed factor breaks both."""
    w, x = _gptq_case(1)
    g, seed = 64, 3
    grid = _small_grid(p, n)
    xr = np.concatenate([O.rht_activations(x[:, b:b + g], g, seed) for b in range(0, x.shape[1], g)],
                        axis=1)
    u = O.gptq_factor(xr, 0.01)
    assert np.allclose(np.tril(u, -1), 0)
    r = O.quantize_gptq(w, grid, g, seed, u)
    dw = r["w_rot"] - r["deq_rot"]
    assert np.allclose(dw, r["err_scaled"] @ u, rtol=0, atol=1e-12)
    h = xr.T @ xr
    h[np.diag_indices_from(h)] += 0.01 * np.mean(np.diag(h))
    loss = np.einsum("ij,jk,ik->", dw, h, dw)
    assert abs(loss / (r["err_scaled"] ** 2).sum() - 1) < 1e-9


def test_gptq_with_diagonal_hessian_is_round_to_nearest():
    """H proportional to I: U is diagonal, nothing is fed forward, and the
    codes are Alg. 1's nearest points."""
    w, _ = _gptq_case(2)
    g, seed = 64, 5
    grid = _small_grid(2, 64)
    u = O.gptq_factor(np.eye(w.shape[1]) * 3.0, 0.0)
    assert np.allclose(u, np.eye(w.shape[1]) / 3.0)
    r = O.quantize_gptq(w, grid, g, seed, u)
    ref = O.quantize(w, grid, g, seed)
    diff = r["codes"] != ref["codes"]
    assert not (diff & (ref["gap"] >= 1e-9)).any()
    assert np.array_equal(r["scales"].view(np.uint16), ref["scales"].view(np.uint16))


@pytest.mark.parametrize("seed", [4, 6])
def test_gptq_lowers_calibration_loss(seed):
    """On correlated calibration inputs GPTQ's rounding leaves less output
    error than round-to-nearest (the purpose of the method)."""
    w, x = _gptq_case(seed)
    g, s0 = 64, 9
    grid = _small_grid(2, 64)
    xr = np.concatenate([O.rht_activations(x[:, b:b + g], g, s0) for b in range(0, x.shape[1], g)],
                        axis=1)
    r = O.quantize_gptq(w, grid, g, s0, O.gptq_factor(xr, 0.01))
    ref = O.quantize(w, grid, g, s0)
    w_gptq = O.dequantize(r["codes"], r["scales"], grid, g, s0)
    w_rtn = O.dequantize(ref["codes"], ref["scales"], grid, g, s0)
    assert ((w_gptq - w) @ x.T).var() < 0.9 * ((w_rtn - w) @ x.T).var()


def test_code_distances_brute_force():
    """The distance of a named code equals the direct sum of squares, and
    for the nearest code it is nearest()'s best distance."""
    rng = np.random.default_rng(8)
    grid = rng.standard_normal((16, 2))
    pts = rng.standard_normal((40, 2))
    codes = rng.integers(0, 16, 40)
    d = O.code_distances(pts, grid, codes)
    for i in range(40):
        want = sum((pts[i, t] - grid[codes[i], t]) ** 2 for t in range(2))
        assert d[i] == want
    idx, best, _ = O.nearest(pts, grid)
    assert np.array_equal(O.code_distances(pts, grid, idx), best)


def test_gptq_follow_mode():
    """Following candidate codes: the oracle's own codes change nothing; a
    candidate away from a tie is reported and not adopted; at an exact tie
    (a grid point duplicated at a higher index) the candidate is adopted,
    and since both points are equal the recursion is unchanged."""
    w, x = _gptq_case(11)
    g, seed = 64, 2
    grid = _small_grid(2, 64)
    xr = np.concatenate([O.rht_activations(x[:, b:b + g], g, seed) for b in range(0, x.shape[1], g)],
                        axis=1)
    u = O.gptq_factor(xr, 0.01)
    r = O.quantize_gptq(w, grid, g, seed, u)
    assert not r["mismatch"].any()
    same = O.quantize_gptq(w, grid, g, seed, u, follow=r["codes"], follow_tol=1e-6)
    assert np.array_equal(same["codes"], r["codes"]) and not same["mismatch"].any()
    wrong = r["codes"].copy()
    wrong[3, 5] = (wrong[3, 5] + 1) % 64           # a different, farther point
    bad = O.quantize_gptq(w, grid, g, seed, u, follow=wrong, follow_tol=1e-6)
    assert bad["mismatch"][3, 5] and bad["mismatch"].sum() == 1
    assert np.array_equal(bad["codes"], r["codes"])
    # exact ties: point 64 duplicates point k; the oracle picks k (lower
    # index), the candidate names 64
    k = int(r["codes"][0, 0])
    grid2 = np.concatenate([grid, grid[k:k + 1]])
    base = O.quantize_gptq(w, grid2, g, seed, u)
    assert np.array_equal(base["codes"], r["codes"])
    alt = base["codes"].copy()
    alt[alt == k] = 64
    tied = O.quantize_gptq(w, grid2, g, seed, u, follow=alt, follow_tol=0.0)
    assert not tied["mismatch"].any()
    assert np.array_equal(tied["codes"], alt)
    assert np.array_equal(tied["deq_rot"], base["deq_rot"])


def test_bits_per_weight_matches_paper():
    with open(os.path.join(GOLDEN, "bits_per_weight_app_h.txt")) as f:
        rows = [line.split() for line in f if line.strip() and not line.startswith("#")]
    assert len(rows) == 5
    for p, n, g, printed in rows:
        bpw = O.bits_per_weight(int(p), int(n), int(g))
        assert round(bpw, 2) == float(printed), (p, n, g, bpw)


def test_pack_matches_hand_example():
    with open(os.path.join(GOLDEN, "pack_example.txt")) as f:
        cases = [line for line in f if line.strip() and not line.startswith("#")]
    assert len(cases) == 4
    for line in cases:
        n, codes, packed = (part.split() for part in line.split("|"))
        n = int(n[0])
        codes = np.array([[int(c) for c in codes]])
        expect = np.array([[int(b, 16) for b in packed]], dtype=np.uint8)
        got = O.pack_codes(codes, n)
        assert np.array_equal(got, expect), (n, got, expect)
        assert np.array_equal(O.unpack_codes(got, n, codes.shape[1]), codes)


@pytest.mark.parametrize("n", [16, 64, 256, 1024])
def test_pack_round_trip(n):
    rng = np.random.default_rng(n)
    codes = rng.integers(0, n, size=(5, 64))
    packed = O.pack_codes(codes, n)
    assert packed.shape == (5, 64 * O.bits_per_code(n) // 8)
    assert np.array_equal(O.unpack_codes(packed, n, 64), codes)
