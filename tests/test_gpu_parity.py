"""GPU parity: the HIP library (through its C ABI) against the CPU oracle.

Bars (from the method's definition and the fp formats involved):
  * codes: bit-exact, except at near-ties: where the GPU's index differs from
    the oracle's, its fp64 squared distance must be within 1e-6 of the best
    one (an equally valid rounding);
  * scales: bit-exact fp16;
  * activation rotation: |x_rot - ref| <= (log2(g) + 1) * 2^-23 * ||x_block||_2
    per element (fp32 butterflies: one rounding per stage);
  * qmatmul: relative Frobenius error <= 2e-3 against the fp64 oracle
    (fp16 grid points and activations, fp32 accumulation), over the whole
    output and also for every batch row on its own and every block of 32
    output features (there against the output's overall RMS), so that a bad
    row or tile is not diluted by the rest.
"""
import math
import sys

import numpy as np
import pytest

from conftest import load_grid_fixture
from oracle import higgs_oracle as O
from paper_2411_17525_amd import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

GAP_EXEMPT = 1e-6
QMM_TOL = 2e-3


def announce(msg):
    print(f"[gpu-case] {msg}", file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def H():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2411_17525_amd import higgs
    higgs.lib()  # raises if the library is missing: no fallback
    return higgs


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def grid_f32(p, n):
    if (p, n) == (1, 256):  # CH8: the oracle's uniform MSE-optimal grid
        return O.uniform_grid(256)[0].astype(np.float32)[:, None]
    fx = load_grid_fixture(p, n)
    if fx is None:
        pytest.skip(f"grid fixture p={p} n={n} not generated (tests/golden/make_grids.py)")
    return fx[0].astype(np.float32)


def weight_dev(wt):
    return dev_bf16(wt.bits) if wt.dtype == "bf16" else dev(wt.values)


def check_codes(gpu_codes, gpu_scales, ref, n, rows=None, grid=None):
    """Compare GPU codes / scales (device tensors) with the oracle's dict:
    a differing code must be a near-tie, i.e. name a grid point whose fp64
    squared distance to the rotated p-vector is within GAP_EXEMPT of the
    nearest one's (grid: the (n, p) grid the codes index)."""
    codes_np = gpu_codes.cpu().numpy()
    scales_np = gpu_scales.cpu().numpy()
    if rows is not None:
        codes_np, scales_np = codes_np[rows], scales_np[rows]
    got = O.unpack_codes(codes_np, n, ref["codes"].shape[1])
    diff = got != ref["codes"]
    if diff.any():
        assert grid is not None, "codes differ and no grid was given to judge the ties"
        p = np.asarray(grid).shape[1]
        vecs = ref["w_dag"].reshape(-1, p)
        d_gpu = O.code_distances(vecs, np.asarray(grid, dtype=np.float64), got.reshape(-1))
        excess = d_gpu.reshape(got.shape) - ref["best"]
        bad = diff & (excess >= GAP_EXEMPT)
        assert not bad.any(), (f"{int(bad.sum())} codes differ beyond the tie band; "
                               f"first at {np.argwhere(bad)[0]}")
    assert np.array_equal(scales_np.view(np.uint16), ref["scales"].view(np.uint16)), \
        "scales differ"
    return int(diff.sum())


def rel_fro(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def check_qmm(y, y_ref, tol=QMM_TOL):
    """The product bar: relative Frobenius error over the whole output, over
    each batch row, and over each block of 32 output features (all batch
    rows) measured against the output's overall RMS."""
    y = np.asarray(y, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    err = rel_fro(y, y_ref)
    assert err <= tol, err
    for r in range(y.shape[0]):
        e = rel_fro(y[r], y_ref[r])
        assert e <= tol, (r, e)
    rms = np.sqrt(np.mean(y_ref ** 2))
    for c0 in range(0, y.shape[1], 32):
        blk = y[:, c0:c0 + 32] - y_ref[:, c0:c0 + 32]
        e = float(np.sqrt(np.mean(blk ** 2)) / rms)
        assert e <= tol, (c0, e)
    return err


# ---------------------------------------------------------------------------
# activation rotation
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("g,batch,blocks,dtype", [
    (1024, 1, 4, "bf16"), (1024, 3, 2, "f32"), (4096, 2, 2, "bf16"), (64, 5, 3, "f32"),
    (128, 1, 7, "bf16"), (8, 3, 5, "f32"), (2, 1, 33, "f32"), (32, 7, 3, "bf16"),
    (2048, 8, 7, "bf16")])
def test_rht_activations(H, g, batch, blocks, dtype):
    inp = g * blocks
    announce(f"rht g={g} batch={batch} in={inp} dtype={dtype}")
    act = synth.activations(batch, inp, seed=g + batch)
    x_np = act.values if dtype == "f32" else act.values
    x_dev = dev(act.values) if dtype == "f32" else dev_bf16(act.bits)
    seed = 1000 + g
    out = H.rht_activations(x_dev, g, seed)
    torch.cuda.synchronize()
    ref = O.rht_activations(x_np.astype(np.float64), g, seed)
    got = out.cpu().numpy().astype(np.float64)
    norms = np.sqrt((x_np.astype(np.float64).reshape(batch, blocks, g) ** 2).sum(axis=2))
    bound = (math.log2(g) + 1) * 2.0 ** -23 * np.repeat(norms, g, axis=1).reshape(batch, inp)
    assert np.all(np.abs(got - ref) <= bound + 1e-30)


def test_rht_llama_shapes_batch64(H):
    for inp in (4096, 14336):
        announce(f"rht full shape in={inp} batch=64")
        act = synth.activations(64, inp, seed=inp)
        out = H.rht_activations(dev_bf16(act.bits), 1024, 3)
        torch.cuda.synchronize()
        rows = [0, 17, 63]
        ref = O.rht_activations(act.values[rows].astype(np.float64), 1024, 3)
        got = out.cpu().numpy()[rows].astype(np.float64)
        assert np.abs(got - ref).max() <= 11 * 2.0 ** -23 * np.sqrt(1024) * 6


# ---------------------------------------------------------------------------
# encoder
# ---------------------------------------------------------------------------

ENC_CASES = [
    # p, n, g, out, in, dtype
    (2, 256, 1024, 16, 2048, "bf16"),
    (2, 256, 128, 5, 1024, "f32"),
    (2, 64, 1024, 9, 2048, "bf16"),
    (2, 64, 256, 3, 512, "f32"),
    (2, 1024, 1024, 4, 2048, "bf16"),
    (2, 1024, 4096, 2, 4096, "f32"),
    (1, 16, 1024, 7, 2048, "bf16"),
    (1, 16, 64, 3, 640, "f32"),
    (2, 256, 4096, 3, 8192, "bf16"),
    (1, 256, 1024, 6, 2048, "bf16"),      # CH8
    (1, 256, 64, 3, 640, "f32"),
]


@pytest.mark.parametrize("p,n,g,out,inp,dtype", ENC_CASES)
def test_quantize_matches_oracle(H, p, n, g, out, inp, dtype):
    announce(f"quantize p={p} n={n} g={g} out={out} in={inp} {dtype}")
    grid = grid_f32(p, n)
    wt = synth.student_t_weight(out, inp, seed=out * 7 + inp, dtype=dtype, outliers=True)
    seed = 77 + g
    codes, scales = H.quantize(weight_dev(wt), dev(grid), g, seed)
    torch.cuda.synchronize()
    ref = O.quantize(wt.values.astype(np.float64), grid.astype(np.float64), g, seed)
    check_codes(codes, scales, ref, n, grid=grid)


@pytest.mark.parametrize("scale,g", [(12.0, 4096), (30.0, 1024)])
def test_quantize_large_norm_grid(H, scale, g):
    """A grid whose points are far from unit variance (the (2,256) grid times
    `scale`): the search values need a shift above 1024 to stay positive,
    which the encoder derives from the grid it loads."""
    p, n = 2, 256
    announce(f"quantize grid x{scale} g={g}")
    grid = (grid_f32(p, n) * np.float32(scale)).astype(np.float32)
    wt = synth.student_t_weight(6, 2 * g, seed=int(scale), dtype="f32", outliers=True)
    codes, scales = H.quantize(dev(wt.values), dev(grid), g, 9)
    torch.cuda.synchronize()
    ref = O.quantize(wt.values.astype(np.float64), grid.astype(np.float64), g, 9)
    check_codes(codes, scales, ref, n, grid=grid)


def test_quantize_special_groups(H):
    """Zero groups, one-hot groups and an exact fp16 rounding tie in the scale."""
    p, n, g = 2, 256, 1024
    announce("quantize special groups")
    grid = grid_f32(p, n)
    w = synth.student_t_weight(6, 2 * g, seed=5, dtype="f32", outliers=False).values.copy()
    w[0, :g] = 0.0                        # zero group
    w[1, :] = 0.0
    w[1, 37] = -2.5                       # one-hot group: rotated values are exactly +-1
    w[2, :] = 0.0
    w[2, 5] = 32.0 * (1 + 2.0 ** -11)     # s / sqrt(g) = 1 + 2^-11: fp16 tie -> even (1.0)
    w[2, g + 9] = 32.0 * (1 + 3 * 2.0 ** -11)  # tie -> even (1 + 2^-9)
    codes, scales = H.quantize(dev(w), dev(grid), g, 11)
    torch.cuda.synchronize()
    ref = O.quantize(w.astype(np.float64), grid.astype(np.float64), g, 11)
    assert float(ref["scales"][2, 0]) == 1.0
    assert float(ref["scales"][2, 1]) == 1.0 + 2.0 ** -9
    check_codes(codes, scales, ref, n, grid=grid)


def test_quantize_cfg1_full(H):
    """1024 x 1024 fp32 Student-t layer, grid (2, 256), g = 1024, seed 0."""
    announce("quantize cfg1 1024x1024")
    grid = grid_f32(2, 256)
    wt = synth.student_t_weight(1024, 1024, seed=0, dtype="f32", outliers=False)
    codes, scales = H.quantize(dev(wt.values), dev(grid), 1024, 0)
    torch.cuda.synchronize()
    ref = O.quantize(wt.values.astype(np.float64), grid.astype(np.float64), 1024, 0)
    ties = check_codes(codes, scales, ref, 256, grid=grid)
    assert ties <= 5
    # the layer's relative error is the grid's MSE (App. F)
    w_hat = O.dequantize(ref["codes"], ref["scales"], grid.astype(np.float64), 1024, 0)
    t2 = O.layer_error(wt.values, w_hat)
    assert 0.006 < t2 < 0.010


@pytest.mark.parametrize("layer", range(7))
def test_quantize_llama8b_sampled_rows(H, layer):
    name, out, inp = synth.LLAMA8B_LAYERS[layer]
    announce(f"quantize 8B {name} {out}x{inp}")
    grid = grid_f32(2, 256)
    wt = synth.student_t_weight(out, inp, seed=4000 + layer, dtype="bf16")
    codes, scales = H.quantize(dev_bf16(wt.bits), dev(grid), 1024, layer)
    torch.cuda.synchronize()
    rows = sorted({0, out - 1, *np.random.default_rng(layer).integers(0, out, 4).tolist()})
    ref = O.quantize(wt.values[rows].astype(np.float64), grid.astype(np.float64), 1024, layer)
    check_codes(codes, scales, ref, 256, rows=rows, grid=grid)


# ---------------------------------------------------------------------------
# the encoder's search index (exact pruning of the nearest-point search)
# ---------------------------------------------------------------------------

INDEX_GRIDS = [(2, 64), (2, 256), (2, 1024), (1, 16), (1, 256)]


def read_index(idx, p, n):
    """Header and lists of an index read back from the device. Layout: a
    64-byte header (u32 magic, p, n, buckets per axis, list entries, usable
    flag, two reserved; u64 grid hash; f64 margin, half side), then u16
    offsets (one per bucket, plus the end) and the u16 lists, each region
    16-byte aligned; buckets per axis^p buckets in all."""
    raw = idx.cpu().numpy()
    u32 = raw[:24].view(np.uint32)
    f64 = raw[40:56].view(np.float64)
    cells = int(u32[3]) ** p
    o0 = 64
    l0 = o0 + (2 * (cells + 1) + 15) // 16 * 16
    offs = raw[o0:o0 + 2 * (cells + 1)].view(np.uint16).astype(np.int64)
    total = int(u32[4])
    lists = raw[l0:l0 + 2 * total].view(np.uint16).astype(np.int64)
    return {"magic": int(u32[0]), "p": int(u32[1]), "n": int(u32[2]), "nb": int(u32[3]),
            "total": total, "usable": int(u32[5]), "margin": float(f64[0]),
            "half_side": float(f64[1]), "offs": offs, "lists": lists}


@pytest.mark.parametrize("p,n", INDEX_GRIDS)
def test_search_index_lists_hold_the_nearest_point(H, p, n):
    """For random points of every bucket and for every bucket corner, the
    grid point nearest to it (fp64 brute force, the oracle's search) is in
    that bucket's list: the pruning never drops the answer."""
    announce(f"search index p={p} n={n}")
    grid = grid_f32(p, n)
    ix = read_index(H.search_index(dev(grid)), p, n)
    nb = ix["nb"]
    assert nb == (512 if p == 1 else (128 if n >= 256 else 64))
    assert (ix["magic"], ix["p"], ix["n"], ix["usable"]) == (0x49534748, p, n, 1)
    assert ix["half_side"] == 4.0 and 0 < ix["margin"] < 1e-5
    offs, lists = ix["offs"], ix["lists"]
    cells = nb ** p
    assert offs[0] == 0 and offs[cells] == ix["total"]
    assert np.all(np.diff(offs) >= 1)                    # no empty list
    assert np.all((lists >= 0) & (lists < n))
    w = 8.0 / nb
    rng = np.random.default_rng(n + p)
    per = 6
    cell = np.arange(cells)
    lo = np.stack([-4.0 + w * (cell % nb), -4.0 + w * (cell // nb)], 1)[:, :p] if p == 2 \
        else (-4.0 + w * cell)[:, None]
    pts = [lo[:, None, :] + w * rng.random((cells, per, p))]
    corners = [[0.0], [1.0 - 1e-12]] if p == 1 else \
        [[0.0, 0.0], [0.0, 1.0 - 1e-12], [1.0 - 1e-12, 0.0], [1.0 - 1e-12, 1.0 - 1e-12]]
    pts.append(lo[:, None, :] + w * np.array(corners)[None])
    pts = np.concatenate(pts, axis=1)                    # [cells, samples, p]
    k, _, _ = O.nearest(pts.reshape(-1, p), grid.astype(np.float64), with_gap=False)
    k = k.reshape(cells, -1)
    member = np.zeros((cells, n), dtype=bool)
    owner = np.repeat(cell, np.diff(offs))
    member[owner, lists] = True
    missing = ~member[cell[:, None], k]
    assert not missing.any(), f"{int(missing.sum())} nearest points missing, first bucket " \
        f"{int(np.argwhere(missing)[0][0])}"


def spiked_rows(g, seed, rows, groups, rng):
    """Rows whose groups rotate (Alg. 1) to vectors outside the bucketed
    square: w = sigma * (H e_j) scaled, plus a little noise, so that w_dag
    has one coordinate near sqrt(g) (for half the groups), or a mix of a
    spike and noise."""
    sig = O.rht_signs(seed, g).astype(np.float64)
    h = O.hadamard(g)
    w = rng.standard_normal((rows, groups * g)) * 0.02
    for r in range(rows):
        for q in range(groups):
            j = int(rng.integers(0, g))
            amp = 0.5 if (r + q) % 2 == 0 else 0.02
            w[r, q * g:(q + 1) * g] += amp * sig * h[j]
    return w.astype(np.float32)


@pytest.mark.parametrize("p,n", INDEX_GRIDS)
def test_quantize_index_matches_full_scan(H, p, n):
    """Codes and scales with the grid's index, without an index, and with
    the index of another grid (ignored: its hash does not match) are
    identical and match the oracle, on a layer that mixes Student-t rows
    with rows whose rotated vectors leave the bucketed square."""
    g = 1024
    announce(f"quantize index vs full scan p={p} n={n}")
    grid = grid_f32(p, n)
    rng = np.random.default_rng(3 * n + p)
    wt = synth.student_t_weight(6, 2 * g, seed=n + p, dtype="f32", outliers=True).values
    w = np.concatenate([wt, spiked_rows(g, 5, 4, 2, rng)], axis=0)
    seed = 5
    gd = dev(grid)
    idx = H.search_index(gd)
    other = H.search_index(dev((grid * np.float32(1.5)).astype(np.float32)))
    c1, s1 = H.quantize(dev(w), gd, g, seed, index=idx)
    c2, s2 = H.quantize(dev(w), gd, g, seed, index=False)
    c3, s3 = H.quantize(dev(w), gd, g, seed, index=other)
    torch.cuda.synchronize()
    assert torch.equal(c1, c2) and torch.equal(c1, c3)
    assert torch.equal(s1, s2) and torch.equal(s1, s3)
    ref = O.quantize(w.astype(np.float64), grid.astype(np.float64), g, seed)
    assert np.abs(ref["w_dag"]).max() > 8.0      # some vectors do leave the square
    check_codes(c1, s1, ref, n, grid=grid)


def test_quantize_index_overflow_and_duplicate_points(H):
    """Two grids the index cannot help with or must not mislead: (a) every
    point in a tiny cluster, so that buckets far from it list more points
    than the index holds (it marks itself unusable and every vector scans
    the grid); (b) a grid with a repeated point, where the lower index must
    win as in a full scan."""
    g = 1024
    announce("quantize index overflow / duplicate points")
    base = grid_f32(2, 1024)
    tiny = (base * np.float32(1e-3) + np.float32(0.5)).astype(np.float32)
    ix = read_index(H.search_index(dev(tiny)), 2, 1024)
    assert ix["usable"] == 0
    w = synth.student_t_weight(4, 2 * g, seed=17, dtype="f32", outliers=True).values
    c, s = H.quantize(dev(w), dev(tiny), g, 3)
    c2, s2 = H.quantize(dev(w), dev(tiny), g, 3, index=False)
    torch.cuda.synchronize()
    assert torch.equal(c, c2) and torch.equal(s, s2)
    ref = O.quantize(w.astype(np.float64), tiny.astype(np.float64), g, 3)
    check_codes(c, s, ref, 1024, grid=tiny)

    dup = grid_f32(2, 256).copy()
    ref0 = O.quantize(w.astype(np.float64), dup.astype(np.float64), g, 4)
    used = np.bincount(ref0["codes"].reshape(-1), minlength=256)
    src = int(np.argmax(used))                   # the most used point
    dst = 255 if src != 255 else 254
    lo_i, hi_i = min(src, dst), max(src, dst)
    dup[dst] = dup[src]
    c, s = H.quantize(dev(w), dev(dup), g, 4)
    torch.cuda.synchronize()
    ref = O.quantize(w.astype(np.float64), dup.astype(np.float64), g, 4)
    got = O.unpack_codes(c.cpu().numpy(), 256, ref["codes"].shape[1])
    assert not np.any(got == hi_i) and np.any(got == lo_i)
    check_codes(c, s, ref, 256, grid=dup)


# ---------------------------------------------------------------------------
# layer error (Sec. 3.4 / Sec. 4): rotated-space error on the GPU against the
# oracle's original-space ||W - W_hat||^2 of the GPU's own codes and scales
# ---------------------------------------------------------------------------

ERR_CASES = [
    # p, n, g, out, in, dtype
    (2, 256, 1024, 16, 2048, "bf16"),
    (2, 64, 256, 9, 1024, "f32"),
    (1, 16, 64, 5, 640, "bf16"),
    (2, 1024, 1024, 4, 2048, "f32"),
    (1, 256, 128, 7, 1024, "bf16"),
    (2, 256, 4096, 3, 8192, "f32"),
]


@pytest.mark.parametrize("p,n,g,out,inp,dtype", ERR_CASES)
def test_layer_error_matches_oracle(H, p, n, g, out, inp, dtype):
    announce(f"layer_error p={p} n={n} g={g} out={out} in={inp} {dtype}")
    grid = grid_f32(p, n)
    wt = synth.student_t_weight(out, inp, seed=out * 11 + inp, dtype=dtype, outliers=True)
    seed = 5 + g
    w_dev = weight_dev(wt)
    codes, scales = H.quantize(w_dev, dev(grid), g, seed)
    t2, ge = H.layer_error(w_dev, codes, scales, dev(grid), g, seed)
    ge = ge.cpu().numpy()
    w = wt.values.astype(np.float64)
    w_hat = O.dequantize(O.unpack_codes(codes.cpu().numpy(), n, inp // p), scales.cpu().numpy(),
                         grid.astype(np.float64), g, seed)
    t2_ref = O.layer_error(w, w_hat)
    assert abs(t2 - t2_ref) <= 1e-9 * t2_ref, (t2, t2_ref)
    err_ref = ((w - w_hat) ** 2).reshape(out, inp // g, g).sum(axis=2).ravel()
    norm_ref = (w ** 2).reshape(out, inp // g, g).sum(axis=2).ravel()
    assert np.allclose(ge[:, 0], err_ref, rtol=1e-9, atol=1e-300)
    assert np.allclose(ge[:, 1], norm_ref, rtol=1e-12, atol=0)


# ---------------------------------------------------------------------------
# GPTQ rounding (Sec. 3.5)
# ---------------------------------------------------------------------------

def _calib(samples, inp, seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((samples, inp))
    x = x @ (np.eye(inp) + 0.8 * rng.standard_normal((inp, inp)) / math.sqrt(inp))
    return x.astype(np.float32)


@pytest.mark.parametrize("samples,inp,damp", [(512, 256, 0.01), (2048, 1024, 0.01), (300, 512, 0.1)])
def test_gptq_factor_matches_oracle(H, samples, inp, damp):
    announce(f"gptq factor samples={samples} in={inp}")
    xr = _calib(samples, inp, inp)
    u = H.gptq_factor(dev(xr), damp).cpu().numpy()
    u_ref = O.gptq_factor(xr.astype(np.float64), damp)
    up = np.triu(u)
    assert np.linalg.norm(up - u_ref) <= 1e-9 * np.linalg.norm(u_ref)


GPTQ_CASES = [
    # p, n, g, out, in, dtype
    (2, 256, 256, 24, 512, "bf16"),
    (2, 64, 1024, 16, 2048, "f32"),
    (1, 16, 64, 20, 256, "bf16"),
    (2, 1024, 128, 8, 512, "f32"),
    (1, 256, 256, 12, 512, "bf16"),
]


@pytest.mark.parametrize("p,n,g,out,inp,dtype", GPTQ_CASES)
def test_quantize_gptq_matches_oracle(H, p, n, g, out, inp, dtype):
    """Every code of every row against the oracle's own recursion on its own
    factor. The calibration activations (already in the rotated space) are
    the shared input of both factors. Where the library's rounding differs
    from the oracle's, it must be a near-tie (its squared distance within
    GAP_EXEMPT of the nearest point's); the oracle then continues from the
    library's choice, so the rest of the row is still compared."""
    announce(f"gptq quantize p={p} n={n} g={g} out={out} in={inp} {dtype}")
    grid = grid_f32(p, n)
    wt = synth.student_t_weight(out, inp, seed=out + 3 * inp, dtype=dtype)
    seed = 13 + g
    x_rot = _calib(4 * inp, inp, out)
    factor = H.gptq_factor(dev(x_rot), 0.01)
    codes, scales = H.quantize_gptq(weight_dev(wt), dev(grid), g, seed, factor)
    torch.cuda.synchronize()
    got = O.unpack_codes(codes.cpu().numpy(), n, inp // p)
    u_ref = O.gptq_factor(x_rot.astype(np.float64), 0.01)
    ref = O.quantize_gptq(wt.values.astype(np.float64), grid.astype(np.float64), g, seed, u_ref,
                          follow=got, follow_tol=GAP_EXEMPT)
    assert np.array_equal(scales.cpu().numpy().view(np.uint16), ref["scales"].view(np.uint16))
    mism = ref["mismatch"]
    assert not mism.any(), (int(mism.sum()), np.argwhere(mism)[0])
    assert np.array_equal(got, ref["codes"])


def test_quantize_gptq_diagonal_hessian_is_round_to_nearest(H):
    p, n, g, out, inp = 2, 256, 1024, 16, 2048
    announce("gptq with a diagonal Hessian")
    grid = grid_f32(p, n)
    wt = synth.student_t_weight(out, inp, seed=7, dtype="bf16")
    x_rot = dev((np.eye(inp) * 2.0).astype(np.float32))
    factor = H.gptq_factor(x_rot, 0.0)
    c1, s1 = H.quantize_gptq(weight_dev(wt), dev(grid), g, 3, factor)
    c2, s2 = H.quantize(weight_dev(wt), dev(grid), g, 3)
    torch.cuda.synchronize()
    ref = O.quantize(wt.values.astype(np.float64), grid.astype(np.float64), g, 3)
    assert torch.equal(s1, s2)
    a = O.unpack_codes(c1.cpu().numpy(), n, inp // p)
    b = O.unpack_codes(c2.cpu().numpy(), n, inp // p)
    assert not ((a != b) & (ref["gap"] >= GAP_EXEMPT)).any()


def test_gptq_lowers_product_error_end_to_end(H):
    """Encode with GPTQ rounding on the GPU, multiply with the LUT product:
    on the calibration inputs the output error is below round-to-nearest's."""
    p, n, g, out, inp = 2, 256, 1024, 64, 2048
    announce("gptq end to end")
    grid = dev(grid_f32(p, n))
    wt = synth.student_t_weight(out, inp, seed=21, dtype="f32")
    x = _calib(1024, inp, 5)
    xd = dev(x)
    x_rot = H.rht_activations(xd, g, 2)
    cg, sg = H.quantize_gptq(dev(wt.values), grid, g, 2, H.gptq_factor(x_rot, 0.01))
    cr, sr = H.quantize(dev(wt.values), grid, g, 2)
    y_true = x.astype(np.float64) @ wt.values.astype(np.float64).T
    e_g = H.qmatmul(x_rot, cg, sg, grid, g, out).cpu().numpy() - y_true
    e_r = H.qmatmul(x_rot, cr, sr, grid, g, out).cpu().numpy() - y_true
    assert (e_g ** 2).sum() < 0.8 * (e_r ** 2).sum()


# ---------------------------------------------------------------------------
# qmatmul (rotated-space LUT product)
# ---------------------------------------------------------------------------

def run_layer(H, x_bits, codes_np, scales_f16, grid, g, seed, out):
    x_dev = dev_bf16(x_bits)
    x_rot = H.rht_activations(x_dev, g, seed)
    y = H.qmatmul(x_rot, dev(codes_np), dev(scales_f16), dev(grid), g, out)
    torch.cuda.synchronize()
    return y.cpu().numpy().astype(np.float64)


QMM_CASES = [
    # p, n, g, out, in, batch
    (2, 256, 1024, 64, 2048, 1),
    (2, 256, 1024, 37, 4096, 4),
    (2, 256, 1024, 16, 1024, 3),     # partial K-range
    (2, 256, 128, 21, 3072, 8),
    (2, 256, 1024, 40, 2048, 9),     # two batch chunks
    (2, 256, 1024, 33, 2048, 16),
    (2, 64, 1024, 24, 2048, 2),
    (2, 64, 256, 13, 6144, 5),
    (2, 1024, 1024, 24, 2048, 1),
    (2, 1024, 2048, 11, 4096, 7),
    (1, 16, 1024, 24, 2048, 8),
    (1, 16, 64, 9, 1024, 1),
    # matrix-core path: ragged rows, K not a multiple of the 256-weight
    # stage, group sizes below / above the stage, both batch tile widths,
    # a second batch chunk
    (2, 256, 128, 200, 1152, 17),
    (1, 16, 64, 130, 1088, 40),
    (2, 256, 2048, 300, 4096, 64),
    (2, 256, 4096, 64, 4096, 32),
    (2, 256, 1024, 129, 8192, 70),
    # matrix-core path with 6- and 10-bit codes (codes straddling dwords)
    (2, 64, 1024, 200, 2048, 17),
    (2, 64, 128, 130, 1152, 40),
    (2, 1024, 1024, 129, 4096, 64),
    (2, 1024, 256, 70, 1280, 33),
    (2, 1024, 2048, 40, 8192, 70),
    # three full 64-row chunks and an 8-row remainder (16-column tile)
    (2, 256, 256, 40, 1024, 200),
    # the 16-column tile (up to 16 batch rows, g >= 128): every code width,
    # both fold lengths, ragged rows, K not a multiple of the stage
    (2, 256, 256, 129, 2304, 16),
    (2, 64, 128, 130, 1152, 10),
    (2, 1024, 256, 70, 1280, 12),
    (1, 16, 512, 33, 2560, 14),
    (1, 256, 128, 45, 1152, 11),
    # small batches on the matrix-core small-batch variant (batch tiles of 4
    # and 8 (the 8-row tile: g = 64, below that grid's crossover), every
    # group size, K not a multiple of the 1024-weight slice)
    (2, 256, 256, 70, 3072, 3),
    (1, 16, 64, 45, 1152, 7),
    (2, 256, 512, 9, 2048, 2),
    (2, 256, 2048, 21, 4096, 4),
    # either side of the batch where the matrix-core path takes over: with
    # g >= 128 at 5 on rows <= 8192, on longer rows at 2 for 8-bit pair codes
    # and 3 for the others; with g = 64 at 9 (longer rows: 5 for (1,16), 7
    # for CH8)
    (2, 256, 1024, 40, 4096, 4),
    (2, 256, 1024, 40, 4096, 5),
    (2, 256, 1024, 40, 12288, 1),
    (2, 256, 1024, 40, 12288, 2),
    (2, 64, 512, 33, 2048, 4),
    (2, 64, 512, 33, 2048, 5),
    (2, 64, 1024, 33, 12288, 2),
    (2, 64, 1024, 33, 12288, 3),
    (2, 1024, 1024, 20, 2048, 4),
    (2, 1024, 1024, 20, 2048, 5),
    (2, 1024, 1024, 20, 12288, 3),
    (1, 256, 1024, 20, 2048, 5),
    (1, 256, 1024, 20, 12288, 2),
    (1, 256, 1024, 20, 12288, 3),
    (1, 16, 64, 40, 2048, 8),
    (1, 16, 64, 40, 2048, 9),
    (1, 256, 64, 20, 12288, 7),
    # CH8 (p = 1, n = 256): one weight per 8-bit code
    (1, 256, 1024, 24, 2048, 1),
    (1, 256, 128, 13, 1152, 5),
    (1, 256, 64, 40, 2048, 8),
    # CH8 on the matrix-core path: every fold length, both batch tile widths,
    # ragged rows, K not a multiple of the stage, a second batch chunk
    (1, 256, 1024, 33, 4096, 17),
    (1, 256, 64, 70, 1088, 40),
    (1, 256, 128, 129, 2304, 64),
    (1, 256, 4096, 33, 8192, 70),
    # the small-batch kernel on rotated input with two K-slices per wave
    # (rows above 16384 weights at batch 1; the 70B down layer's path), every
    # pair-code width
    (2, 256, 1024, 40, 20480, 1),
    (2, 256, 1024, 40, 28672, 1),
    (2, 64, 1024, 33, 28672, 1),
    (2, 1024, 1024, 24, 20480, 1),
    # CH8 rows above 16384 weights: 16 waves at batch 1, batch 2 as two
    # launches of batch tile 1
    (1, 256, 1024, 20, 28672, 1),
    (1, 256, 1024, 20, 20480, 2),
    # K-splits whose last split is short: one 128-weight super-block of the
    # 16-column tile, a partial 256-weight stage
    (2, 256, 128, 21, 3200, 16),
    (2, 256, 128, 21, 2432, 8),
]


@pytest.mark.parametrize("p,n,g,out,inp,batch", QMM_CASES)
def test_qmatmul_matches_oracle(H, p, n, g, out, inp, batch):
    announce(f"qmatmul p={p} n={n} g={g} out={out} in={inp} batch={batch}")
    grid = grid_f32(p, n)
    wt = synth.student_t_weight(out, inp, seed=out + inp + batch, dtype="bf16")
    seed = 3 + batch
    ref = O.quantize(wt.values.astype(np.float64), grid.astype(np.float64), g, seed)
    packed = O.pack_codes(ref["codes"], n)
    act = synth.activations(batch, inp, seed=99 + batch)
    y = run_layer(H, act.bits, packed, ref["scales"], grid, g, seed, out)
    y_ref = O.qmatmul(act.values.astype(np.float64), ref["codes"], ref["scales"],
                      grid.astype(np.float64), g, seed)
    check_qmm(y, y_ref)


def test_qmatmul_end_to_end_cfg1(H):
    """W -> GPU encode -> GPU RHT + qmatmul against the oracle's W_hat, x."""
    announce("end-to-end cfg1")
    grid = grid_f32(2, 256)
    wt = synth.student_t_weight(1024, 1024, seed=0, dtype="f32", outliers=False)
    act = synth.activations(1, 1024, seed=1)
    codes, scales = H.quantize(dev(wt.values), dev(grid), 1024, 0)
    x_rot = H.rht_activations(dev_bf16(act.bits), 1024, 0)
    y = H.qmatmul(x_rot, codes, scales, dev(grid), 1024, 1024)
    torch.cuda.synchronize()
    ref = O.quantize(wt.values.astype(np.float64), grid.astype(np.float64), 1024, 0)
    y_ref = O.qmatmul(act.values.astype(np.float64), ref["codes"], ref["scales"],
                      grid.astype(np.float64), 1024, 0)
    check_qmm(y.cpu().numpy(), y_ref)
    # and against the unquantized layer: the error is the quantization error
    y_w = act.values.astype(np.float64) @ wt.values.astype(np.float64).T
    assert rel_fro(y.cpu().numpy().astype(np.float64), y_w) < 0.2


@pytest.mark.parametrize("batch", [2, 12, 40])
def test_qmatmul_activation_scaling(H, batch):
    """Zero, huge and tiny activations, also mixed across the rows of one batch
    (each row and group gets its own power of two): exact power-of-two
    rescaling keeps precision, on the small-batch kernel (batch 2) and on the
    matrix-core path's 16- and 64-column tiles (12, 40)."""
    p, n, g, out, inp = 2, 256, 1024, 16, 2048
    grid = grid_f32(p, n)
    codes = synth.random_codes(out, inp // p, n, seed=1)
    scales = synth.random_scales_f16(out, inp // g, seed=2).view(np.float16)
    packed = O.pack_codes(codes, n)
    rng = np.random.default_rng(3)
    w_rot = grid.astype(np.float64)[codes].reshape(out, inp // g, g) \
        * scales.astype(np.float64)[:, :, None]
    row_mags = np.array([1e30, 1e-30, 1.0, 0.0] * batch)[:batch]
    for mag in (0.0, 1e30, 1e-30, "mixed"):
        announce(f"qmatmul activation magnitude {mag} batch {batch}")
        m = row_mags[:, None] if mag == "mixed" else mag
        x_rot = (rng.standard_normal((batch, inp)) * m).astype(np.float32)
        y = H.qmatmul(dev(x_rot), dev(packed), dev(scales), dev(grid), g, out)
        torch.cuda.synchronize()
        y_ref = x_rot.astype(np.float64) @ w_rot.reshape(out, inp).T
        got = y.cpu().numpy().astype(np.float64)
        if mag == 0.0:
            assert np.all(got == 0)
        elif mag == "mixed":
            for r in range(batch):  # every row to its own relative tolerance
                if row_mags[r] == 0.0:
                    assert np.all(got[r] == 0)
                else:
                    assert rel_fro(got[r], y_ref[r]) <= QMM_TOL, r
        else:
            assert rel_fro(got, y_ref) <= QMM_TOL


@pytest.mark.parametrize("batch", [4, 12, 64])
def test_qmatmul_deterministic(H, batch):
    """Two calls give the same bits (fixed reduction orders, no atomics): the
    small-batch kernel's K-wave sums, the matrix-core path's split partial
    sums added in split order (16- and 64-column tiles)."""
    p, n, g, out, inp = 2, 256, 1024, 4096, 4096
    announce(f"qmatmul determinism 4096x4096 batch {batch}")
    codes = synth.random_codes(out, inp // p, n, seed=4)
    scales = synth.random_scales_f16(out, inp // g, seed=5).view(np.float16)
    grid = dev(grid_f32(p, n))
    x_rot = dev(np.random.default_rng(6).standard_normal((batch, inp)).astype(np.float32))
    c, s = dev(O.pack_codes(codes, n)), dev(scales)
    y1 = H.qmatmul(x_rot, c, s, grid, g, out).clone()
    y2 = H.qmatmul(x_rot, c, s, grid, g, out)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)


FULL_CASES = [
    # p, n, batches: the Llama-3.1-8B shapes at the benchmark's batch sizes
    (2, 256, (1, 4)),
    (2, 64, (1, 2, 8)),
    (1, 16, (1, 2, 8)),
    (2, 256, (16, 32, 64)),
    (1, 256, (1, 8)),
]


@pytest.mark.parametrize("layer", range(7))
@pytest.mark.parametrize("case", range(len(FULL_CASES)))
def test_qmatmul_llama8b_sampled_outputs(H, layer, case):
    p, n, batches = FULL_CASES[case]
    name, out, inp = synth.LLAMA8B_LAYERS[layer]
    g = 1024
    grid = grid_f32(p, n)
    codes = synth.random_codes(out, inp // p, n, seed=layer)
    scales = synth.random_scales_f16(out, inp // g, seed=layer + 100).view(np.float16)
    c_dev, s_dev, g_dev = dev(O.pack_codes(codes, n)), dev(scales), dev(grid)
    rows = sorted({0, out - 1, *np.random.default_rng(layer).integers(0, out, 30).tolist()})
    w_hat = O.dequantize(codes[rows], scales[rows], grid.astype(np.float64), g, layer)
    for batch in batches:
        announce(f"qmatmul 8B {name} {out}x{inp} p={p} n={n} batch={batch}")
        act = synth.activations(batch, inp, seed=layer + 500 + batch)
        x_rot = H.rht_activations(dev_bf16(act.bits), g, layer)
        y = H.qmatmul(x_rot, c_dev, s_dev, g_dev, g, out)
        torch.cuda.synchronize()
        got = y.cpu().numpy().astype(np.float64)[:, rows]
        y_ref = act.values.astype(np.float64) @ w_hat.T
        check_qmm(got, y_ref)


# ---------------------------------------------------------------------------
# fused rotation + product (raw activations in, y out)
# ---------------------------------------------------------------------------

FUSED_CASES = [
    # p, n, g, out, in, batch, dtype
    (2, 256, 1024, 48, 4096, 1, "bf16"),
    (2, 256, 1024, 37, 2048, 3, "f32"),
    (2, 256, 128, 21, 1024, 8, "bf16"),
    (2, 64, 512, 19, 3072, 2, "bf16"),
    (2, 1024, 1024, 24, 2048, 5, "f32"),
    (1, 16, 64, 9, 1024, 1, "bf16"),
    (1, 16, 1024, 33, 2048, 4, "bf16"),
    (2, 256, 2048, 16, 4096, 2, "bf16"),     # g > 1024: separate rotation pass
    (2, 256, 1024, 40, 2048, 16, "bf16"),    # matrix-core path
    (2, 256, 4096, 40, 8192, 33, "f32"),
    (2, 256, 128, 70, 1152, 20, "f32"),
    (1, 16, 64, 33, 1088, 48, "bf16"),
    (1, 256, 1024, 37, 2048, 3, "bf16"),
    (1, 256, 256, 20, 1024, 8, "f32"),
    (2, 64, 512, 40, 3072, 20, "bf16"),
    (2, 1024, 1024, 33, 2048, 48, "f32"),
    (2, 256, 512, 50, 2560, 7, "bf16"),
    (2, 256, 128, 33, 1152, 11, "f32"),
    (1, 16, 1024, 130, 4096, 2, "bf16"),
    (1, 256, 1024, 40, 2048, 16, "bf16"),    # CH8, matrix-core path
    (1, 256, 256, 20, 1280, 48, "f32"),
]


@pytest.mark.parametrize("p,n,g,out,inp,batch,dtype", FUSED_CASES)
def test_qmatmul_fused_matches_oracle(H, p, n, g, out, inp, batch, dtype):
    announce(f"qmatmul_fused p={p} n={n} g={g} out={out} in={inp} batch={batch} {dtype}")
    grid = grid_f32(p, n)
    wt = synth.student_t_weight(out, inp, seed=out * 3 + inp, dtype="bf16")
    seed = 41 + g + batch
    ref = O.quantize(wt.values.astype(np.float64), grid.astype(np.float64), g, seed)
    act = synth.activations(batch, inp, seed=7 + batch)
    x_dev = dev_bf16(act.bits) if dtype == "bf16" else dev(act.values)
    y = H.qmatmul_fused(x_dev, dev(O.pack_codes(ref["codes"], n)), dev(ref["scales"]), dev(grid),
                        g, seed, out)
    torch.cuda.synchronize()
    y_ref = O.qmatmul(act.values.astype(np.float64), ref["codes"], ref["scales"],
                      grid.astype(np.float64), g, seed)
    check_qmm(y.cpu().numpy(), y_ref)


@pytest.mark.parametrize("g,batch", [(1024, 1), (1024, 4), (256, 2), (128, 8), (1024, 16),
                                     (128, 64), (4096, 40), (512, 5), (256, 12), (1024, 7),
                                     (256, 20), (512, 33), (2048, 64)])
def test_qmatmul_fused_equals_two_step(H, g, batch):
    """Rotation inside the product's staging = separate rotation + product, bit for bit."""
    p, n, out, inp = 2, 256, 64, 4096
    announce(f"fused vs two-step g={g} batch={batch}")
    grid = dev(grid_f32(p, n))
    codes = dev(O.pack_codes(synth.random_codes(out, inp // p, n, seed=g), n))
    scales = dev(synth.random_scales_f16(out, inp // g, seed=g + 1).view(np.float16))
    act = synth.activations(batch, inp, seed=g + batch)
    x = dev_bf16(act.bits)
    y1 = H.qmatmul_fused(x, codes, scales, grid, g, 5, out)
    y2 = H.qmatmul(H.rht_activations(x, g, 5), codes, scales, grid, g, out)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)


@pytest.mark.parametrize("p,n,out,inp,dtype", [
    (2, 256, 2100, 4096, "bf16"),    # four row groups: one wave rotates, the others share
    (2, 256, 2100, 3072, "f32"),
    (2, 256, 64, 14336, "f32"),      # one row group: every wave rotates its own slice
    (1, 256, 64, 16384, "bf16"),     # scalar codes, sixteen slices
    (1, 256, 600, 2048, "f32"),
    (1, 16, 64, 28672, "bf16"),      # two slices per wave
    (2, 256, 3000, 1024, "bf16"),    # one slice, six row groups share one rotation
    (1, 256, 5000, 1024, "f32"),
])
def test_qmatmul_fused_equals_two_step_batch1(H, p, n, out, inp, dtype):
    """Batch 1, g = 1024 (the rotation group is a wave's slice, rotated through LDS):
    the fused product equals the separate rotation + product bit for bit, for
    bf16 and fp32 activations, shared and per-wave rotations, one and two
    slices per wave (App. G)."""
    g = 1024
    announce(f"fused vs two-step batch 1 p={p} n={n} out={out} in={inp} {dtype}")
    grid = dev(grid_f32(p, n))
    codes = dev(O.pack_codes(synth.random_codes(out, inp // p, n, seed=inp + out), n))
    scales = dev(synth.random_scales_f16(out, inp // g, seed=inp).view(np.float16))
    act = synth.activations(1, inp, seed=inp + 3)
    x = dev_bf16(act.bits) if dtype == "bf16" else dev(act.values)
    y1 = H.qmatmul_fused(x, codes, scales, grid, g, 9, out)
    y2 = H.qmatmul(H.rht_activations(x, g, 9), codes, scales, grid, g, out)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)


@pytest.mark.parametrize("layer", range(7))
def test_qmatmul_fused_llama8b_sampled_outputs(H, layer):
    name, out, inp = synth.LLAMA8B_LAYERS[layer]
    p, n, g = 2, 256, 1024
    grid = grid_f32(p, n)
    codes = synth.random_codes(out, inp // p, n, seed=layer + 20)
    scales = synth.random_scales_f16(out, inp // g, seed=layer + 120).view(np.float16)
    c_dev, s_dev, g_dev = dev(O.pack_codes(codes, n)), dev(scales), dev(grid)
    rows = sorted({0, out - 1, *np.random.default_rng(layer + 9).integers(0, out, 30).tolist()})
    w_hat = O.dequantize(codes[rows], scales[rows], grid.astype(np.float64), g, layer)
    for batch in (1, 4, 64):
        announce(f"qmatmul_fused 8B {name} {out}x{inp} batch={batch}")
        act = synth.activations(batch, inp, seed=layer + 700 + batch)
        y = H.qmatmul_fused(dev_bf16(act.bits), c_dev, s_dev, g_dev, g, layer, out)
        torch.cuda.synchronize()
        got = y.cpu().numpy().astype(np.float64)[:, rows]
        check_qmm(got, act.values.astype(np.float64) @ w_hat.T)


# ---------------------------------------------------------------------------
# Llama-3.1-70B shapes with per-layer bitwidths drawn by seed from p = 2,
# n in {64, 256, 1024}, g = 1024: full-size launches (the benchmark's fused
# call at batch 1 and 64), checked on sampled rows
# ---------------------------------------------------------------------------

N70 = synth.mixed_n_for_70b()


@pytest.mark.parametrize("layer", range(7))
def test_quantize_llama70b_sampled_rows(H, layer):
    name, out, inp = synth.LLAMA70B_LAYERS[layer]
    n = N70[layer]
    announce(f"quantize 70B {name} {out}x{inp} p=2 n={n}")
    grid = grid_f32(2, n)
    w_dev, _ = synth.student_t_weight_device(out, inp, 5000 + layer, "cuda")
    codes, scales = H.quantize(w_dev, dev(grid), 1024, layer)
    torch.cuda.synchronize()
    rows = sorted({0, out - 1, *np.random.default_rng(layer + 70).integers(0, out, 3).tolist()})
    idx = torch.tensor(rows, device="cuda")
    w_rows = w_dev[idx].float().cpu().numpy().astype(np.float64)
    ref = O.quantize(w_rows, grid.astype(np.float64), 1024, layer)
    check_codes(codes[idx], scales[idx], ref, n, grid=grid)


@pytest.mark.parametrize("layer", range(7))
def test_qmatmul_fused_llama70b_sampled_outputs(H, layer):
    name, out, inp = synth.LLAMA70B_LAYERS[layer]
    p, n, g = 2, N70[layer], 1024
    grid = grid_f32(p, n)
    packed = synth.random_code_bytes(out, O.codes_row_bytes(inp, p, n), seed=layer + 5100)
    scales = synth.random_scales_f16(out, inp // g, seed=layer + 5200).view(np.float16)
    c_dev, s_dev, g_dev = dev(packed), dev(scales), dev(grid)
    rows = sorted({0, out - 1, *np.random.default_rng(layer + 71).integers(0, out, 24).tolist()})
    codes = O.unpack_codes(packed[rows], n, inp // p)
    w_hat = O.dequantize(codes, scales[rows], grid.astype(np.float64), g, layer)
    for batch in (1, 64):
        announce(f"qmatmul_fused 70B {name} {out}x{inp} p=2 n={n} batch={batch}")
        act = synth.activations(batch, inp, seed=5000 + layer + 500 + batch)
        y = H.qmatmul_fused(dev_bf16(act.bits), c_dev, s_dev, g_dev, g, layer, out)
        torch.cuda.synchronize()
        got = y.cpu().numpy().astype(np.float64)[:, rows]
        check_qmm(got, act.values.astype(np.float64) @ w_hat.T)


# ---------------------------------------------------------------------------
# several layers that read the same activations (q/k/v, gate/up) in one call
# ---------------------------------------------------------------------------

MULTI_CASES = [
    # p, n, g, outs, in, batch, dtype
    (2, 256, 1024, (96, 24, 24), 4096, 1, "bf16"),
    (2, 256, 1024, (4096, 1024, 1024), 4096, 1, "bf16"),   # the 8B q, k, v
    (2, 256, 1024, (14336, 14336), 4096, 1, "bf16"),       # the 8B gate, up
    (2, 256, 1024, (14336, 14336), 4096, 4, "bf16"),
    (1, 16, 256, (33, 70), 2048, 4, "f32"),
    (2, 64, 512, (19, 40, 8, 3), 3072, 2, "bf16"),
    (2, 1024, 1024, (24, 9), 2048, 5, "f32"),
    (1, 256, 1024, (37, 20), 2048, 3, "bf16"),
    (2, 256, 1024, (7,), 1024, 8, "bf16"),
    (2, 256, 1024, (4096, 1024, 1024), 4096, 5, "bf16"),
    (2, 256, 1024, (14336, 14336), 4096, 12, "bf16"),
    (2, 256, 2048, (16, 8), 4096, 2, "bf16"),     # g above the slice: per-layer rotation passes
    # matrix-core path: one conversion, one product launch per 64 batch rows,
    # layers with different K-splits (and none) in one reduction
    (2, 256, 1024, (40, 72), 2048, 20, "bf16"),
    (2, 256, 1024, (4096, 1024, 1024), 4096, 64, "bf16"),
    (2, 256, 1024, (14336, 14336), 4096, 64, "bf16"),
    (2, 1024, 1024, (130, 64), 2048, 70, "f32"),
    (1, 16, 64, (130, 33, 7, 250), 1088, 40, "bf16"),
    (2, 64, 128, (300, 20), 1152, 17, "f32"),
    (1, 256, 1024, (40, 129, 8), 2048, 24, "bf16"),
    # the 16-column tile in a grouped launch whose layers have different
    # K-split counts (blocks of each layer in turn, splits innermost)
    (2, 256, 1024, (4096, 1024, 1024), 4096, 12, "bf16"),
    (1, 256, 1024, (40, 129), 12288, 4, "f32"),
    (2, 64, 256, (300, 20, 77), 2048, 16, "bf16"),
]


@pytest.mark.parametrize("p,n,g,outs,inp,batch,dtype", MULTI_CASES)
def test_qmatmul_fused_multi_equals_per_layer(H, p, n, g, outs, inp, batch, dtype):
    announce(f"qmatmul_fused_multi p={p} n={n} g={g} outs={outs} in={inp} batch={batch} {dtype}")
    grid = dev(grid_f32(p, n))
    rb = O.codes_row_bytes(inp, p, n)
    layers = []
    for l, o in enumerate(outs):
        c = dev(synth.random_code_bytes(o, rb, seed=o + 13 * l))
        sc = dev(synth.random_scales_f16(o, inp // g, seed=o + 17 * l).view(np.float16))
        layers.append((c, sc, 30 + l, o))
    act = synth.activations(batch, inp, seed=inp + batch)
    x = dev_bf16(act.bits) if dtype == "bf16" else dev(act.values)
    ys = H.qmatmul_fused_multi(x, layers, grid, g)
    torch.cuda.synchronize()
    for (c, sc, seed, o), y in zip(layers, ys):
        y1 = H.qmatmul_fused(x, c, sc, grid, g, seed, o)
        torch.cuda.synchronize()
        assert torch.equal(y, y1), f"layer of {o} rows differs from its own fused call"


@pytest.mark.parametrize("batch", [16, 64, 150])
def test_qmatmul_split_outputs_all_written(H, batch):
    """Layers split along K (q/k/v at 4096 columns), over one, one full and
    more than two 64-row chunks: the outputs land in memory that held NaN
    (freed poison of the same shapes), so an element the split reduction
    misses fails; a second call must give the same bits."""
    p, n, g, inp, outs = 2, 256, 1024, 4096, (4096, 1024, 1024)
    announce(f"qmatmul split outputs all written batch={batch}")
    grid = dev(grid_f32(p, n))
    rb = O.codes_row_bytes(inp, p, n)
    layers = []
    for l, o in enumerate(outs):
        c = dev(synth.random_code_bytes(o, rb, seed=o + 7 * l))
        sc = dev(synth.random_scales_f16(o, inp // g, seed=o + 11 * l).view(np.float16))
        layers.append((c, sc, 50 + l, o))
    x = dev_bf16(synth.activations(batch, inp, seed=batch + 1).bits)
    results = []
    for _ in range(2):
        junk = [torch.full((batch, o), float("nan"), device="cuda") for o in outs]
        del junk
        ys = H.qmatmul_fused_multi(x, layers, grid, g)
        torch.cuda.synchronize()
        assert all(bool(torch.isfinite(y).all()) for y in ys)
        results.append([y.clone() for y in ys])
    for y1, y2 in zip(*results):
        assert torch.equal(y1, y2)


@pytest.mark.parametrize("batch", [2, 32])
def test_qmatmul_fused_multi_shared_seed(H, batch):
    """Layers quantized with one seed share the rotated activations."""
    p, n, g, inp = 2, 256, 1024, 4096
    announce(f"qmatmul_fused_multi shared seed batch={batch}")
    grid = dev(grid_f32(p, n))
    rb = O.codes_row_bytes(inp, p, n)
    layers = [(dev(synth.random_code_bytes(o, rb, seed=o)),
               dev(synth.random_scales_f16(o, inp // g, seed=o + 1).view(np.float16)), 77, o)
              for o in (256, 96, 96)]
    act = synth.activations(batch, inp, seed=3)
    x = dev_bf16(act.bits)
    ys = H.qmatmul_fused_multi(x, layers, grid, g)
    torch.cuda.synchronize()
    for (c, sc, seed, o), y in zip(layers, ys):
        assert torch.equal(y, H.qmatmul_fused(x, c, sc, grid, g, seed, o))


def test_qmatmul_fused_multi_matches_oracle(H):
    p, n, g, inp, batch = 2, 256, 1024, 2048, 2
    grid = grid_f32(p, n)
    act = synth.activations(batch, inp, seed=5)
    layers, refs = [], []
    for l, o in enumerate((40, 13, 13)):
        wt = synth.student_t_weight(o, inp, seed=600 + l, dtype="bf16")
        ref = O.quantize(wt.values.astype(np.float64), grid.astype(np.float64), g, 50 + l)
        layers.append((dev(O.pack_codes(ref["codes"], n)), dev(ref["scales"]), 50 + l, o))
        refs.append(O.qmatmul(act.values.astype(np.float64), ref["codes"], ref["scales"],
                              grid.astype(np.float64), g, 50 + l))
    ys = H.qmatmul_fused_multi(dev_bf16(act.bits), layers, dev(grid), g)
    torch.cuda.synchronize()
    for y, y_ref in zip(ys, refs):
        check_qmm(y.cpu().numpy(), y_ref)
