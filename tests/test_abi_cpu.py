"""CPU-side checks of libhiggs.so: it loads, exports what include/higgs.h
declares, its host-only entry points agree with the oracle, and invalid
arguments are rejected on the host before anything reaches the GPU.

No call here launches a kernel: every device entry point is called only with
arguments its host-side validation refuses.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from conftest import ROOT, load_grid_fixture
from oracle import higgs_oracle as O

H = pytest.importorskip("paper_2411_17525_amd.higgs")

INVALID, UNSUPPORTED = 1, 2
FAKE = 1 << 20          # an aligned, never-dereferenced stand-in for a device pointer


def _gpu_visible():
    try:
        import torch
        return torch.cuda.device_count() > 0
    except Exception:
        return False


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(H.LIB_PATH):
        pytest.fail("libhiggs.so is not built (run __graft_entry__.build())")
    return H.lib()


# The argument-validation tests pass fake device pointers. They only use
# argument sets the host rejects, but as a second line of defence they never
# run where a GPU is visible.
no_gpu = pytest.mark.skipif(_gpu_visible(), reason="fake-pointer tests run only without a GPU")


def test_exports_every_declared_symbol(L):
    with open(os.path.join(ROOT, "include", "higgs.h")) as f:
        text = f.read()
    declared = set(re.findall(r"\b(higgs_[a-z0-9_]+)\s*\(", text))
    assert {"higgs_make_grid", "higgs_quantize", "higgs_rht_activations",
            "higgs_qmatmul"} <= declared
    for name in sorted(declared):
        assert hasattr(L, name), name
    assert H.abi_version() == 3


@pytest.mark.parametrize("n", [2, 16, 256])
def test_uniform_grid_matches_oracle(n):
    g, step, mse = H.make_uniform_grid(n)
    pts, step_o, mse_o = O.uniform_grid(n)
    # the oracle minimises the quadrature MSE directly (flat minimum: ~1e-8 in
    # the step); the library solves the stationarity condition exactly
    assert abs(step / step_o - 1) < 1e-6
    assert abs(mse / mse_o - 1) < 1e-10
    assert np.array_equal(g[:, 0], (step * (np.arange(n) - (n - 1) / 2)).astype(np.float32))
    assert np.allclose(g[:, 0], pts, rtol=1e-6, atol=0)


def test_uniform_grid_rejects_bad_n(L):
    buf = np.zeros(8, dtype=np.float32)
    for n in (0, 1, 4097):
        assert L.higgs_make_uniform_grid(n, buf.ctypes.data_as(ctypes.c_void_p), None, None) == INVALID
    assert L.higgs_make_uniform_grid(4, None, None, None) == INVALID


@pytest.mark.parametrize("seed,L,J,b_max", [(0, 5, 4, 4.4), (1, 6, 5, 4.1), (2, 7, 3, 5.0),
                                             (3, 4, 5, 6.5), (4, 6, 2, 3.7), (5, 1, 3, 4.5)])
def test_allocate_bits_matches_brute_force(seed, L, J, b_max):
    """The library's DP against enumeration of every assignment."""
    rng = np.random.default_rng(seed)
    bits = np.array([3.25, 4.015625, 4.015625, 5.015625, 8.015625])[:J]
    t2 = rng.uniform(1e-3, 6e-2, (L, J))
    alpha = rng.uniform(0.1, 3.0, L)
    sizes = rng.integers(1, 15, L) * (1 << 22)
    best, arg, _ = O.allocate_bits_brute(alpha, t2, bits, sizes, b_max)
    choice, obj, avg = H.allocate_bits(alpha, t2, bits, sizes, b_max)
    assert best is not None
    assert abs(obj - best) <= 1e-12 * best
    assert tuple(int(c) for c in choice) in arg      # one of the optimal assignments
    assert avg <= b_max + 1e-12
    assert abs(avg - (bits[choice] * sizes).sum() / sizes.sum()) < 1e-12


def test_allocate_bits_rejects(L):
    t2 = np.full((2, 2), 0.01)
    with pytest.raises(H.HiggsError) as e:
        H.allocate_bits([1.0, 1.0], t2, [3.25, 4.0], [1 << 20, 1 << 20], 3.0)  # below cheapest
    assert e.value.status == INVALID
    with pytest.raises(H.HiggsError) as e:
        H.allocate_bits([1.0, 1.0], t2, [3.3, 4.0], [1 << 20, 1 << 20], 4.0)   # not k / 256
    assert e.value.status == INVALID
    with pytest.raises(H.HiggsError) as e:
        H.allocate_bits([1.0, -1.0], t2, [3.25, 4.0], [1 << 20, 1 << 20], 4.0)  # alpha < 0
    assert e.value.status == INVALID
    with pytest.raises(H.HiggsError) as e:   # coprime sizes: the table would be too large
        H.allocate_bits(np.ones(64), np.tile([0.01, 0.005], (64, 1)), [1 / 256, 1.0],
                        (1 << 30) + 1 + 2 * np.arange(64), 0.9)
    assert e.value.status == UNSUPPORTED
    # near-2^40 sizes with no common divisor and a 4000-bit option: the slack
    # is ~2^61 cost units, so slack * layers passes 2^63; refused, not wrapped
    with pytest.raises(H.HiggsError) as e:
        H.allocate_bits(np.ones(4), np.tile([0.01, 0.001], (4, 1)), [1 / 256, 4000.0],
                        (1 << 40) - 1 - 2 * np.arange(4), 4000.0)
    assert e.value.status == UNSUPPORTED


def test_layer_error_rejects_bad_args_before_launch(L):
    def f(w=FAKE, dt=1, out=16, inp=2048, codes=FAKE, scales=FAKE, grid=FAKE, p=2, n=256, g=1024,
          err=FAKE, t2=FAKE + 4096):
        return L.higgs_layer_error(w, dt, out, inp, codes, scales, grid, p, n, g, 0, err, t2,
                                   None)
    assert f(w=None) == INVALID
    assert f(dt=7) == INVALID
    assert f(n=100) == UNSUPPORTED
    assert f(inp=1000) == INVALID
    assert f(err=FAKE + 4) == INVALID
    assert f(t2=FAKE + 4) == INVALID


@pytest.mark.parametrize("seed,g", [(0, 64), (5, 1024), (2 ** 63 + 7, 4096), (123, 2)])
def test_signs_match_oracle(seed, g):
    assert np.array_equal(H.rht_signs(seed, g), O.rht_signs(seed, g))


@pytest.mark.parametrize("p,n,inp", [(1, 16, 4096), (2, 64, 4096), (2, 256, 14336),
                                     (2, 1024, 8192), (2, 256, 1024)])
def test_row_bytes_match_oracle(p, n, inp):
    assert H.codes_row_bytes(inp, p, n) == O.codes_row_bytes(inp, p, n)


def test_row_bytes_invalid():
    assert H.codes_row_bytes(3, 2, 256) == -1       # in % p != 0
    assert H.codes_row_bytes(6, 2, 8) == -1          # 3 codes * 3 bits: not whole bytes
    assert H.codes_row_bytes(64, 2, 100) == -1       # n not a power of two


@pytest.mark.parametrize("p,n,samples,iters", [(2, 16, 4096, 1000), (2, 64, 1 << 14, 40),
                                               (1, 16, 1 << 14, 300), (1, 2, 4096, 100)])
def test_make_grid_matches_oracle(p, n, samples, iters):
    g_lib, mse_lib, it_lib = H.make_grid(p, n, 7, samples, iters)
    g_or, mse_or, it_or = O.lloyd_grid(p, n, 7, samples, iters)
    assert it_lib == it_or
    np.testing.assert_allclose(g_lib, g_or.astype(np.float32), rtol=0, atol=1e-6)
    assert abs(mse_lib - mse_or) <= 1e-12 * mse_or


@pytest.mark.parametrize("p,n", [(1, 16), (2, 64)])
def test_make_grid_full_size_matches_fixture(p, n):
    fx = load_grid_fixture(p, n)
    if fx is None:
        pytest.skip("grid fixture not generated")
    grid, meta = fx
    g_lib, mse_lib, it_lib = H.make_grid(p, n, int(meta.get("seed", 0)),
                                         1 << 20, int(meta.get("max_iters", 300)))
    assert it_lib == int(meta["iters"])
    np.testing.assert_allclose(g_lib, grid.astype(np.float32), rtol=0, atol=1e-5)
    assert abs(mse_lib / float(meta["mse_per_dim"]) - 1) < 1e-9


def test_make_grid_rejects_bad_args():
    out = np.zeros(64, dtype=np.float32)
    ptr = out.ctypes.data_as(ctypes.c_void_p)
    L = H.lib()
    assert L.higgs_make_grid(3, 16, 0, 1024, 10, ptr, None, None) == UNSUPPORTED
    assert L.higgs_make_grid(2, 16, 0, 8, 10, ptr, None, None) == INVALID   # samples < n
    assert L.higgs_make_grid(2, 16, 0, 1024, -1, ptr, None, None) == INVALID
    assert L.higgs_make_grid(2, 16, 0, 1024, 10, None, None, None) == INVALID
    assert "grid" in L.higgs_last_error().decode()


@no_gpu
def test_quantize_rejects_bad_args_before_launch(L):
    def q(w=FAKE, dt=1, out=8, inp=1024, grid=FAKE, p=2, n=256, g=1024, codes=FAKE, scales=FAKE,
          index=None, index_bytes=0):
        return L.higgs_quantize(w, dt, out, inp, grid, p, n, index, index_bytes, g, 0, codes,
                                scales, None)
    assert q(w=None) == INVALID
    assert q(codes=None) == INVALID
    assert q(dt=7) == INVALID
    assert q(out=0) == INVALID
    assert q(g=1000) == INVALID                     # not a power of two
    assert q(inp=1536) == INVALID                   # in % g
    assert q(p=2, n=128) == UNSUPPORTED             # grid not supported
    assert q(p=3, n=64) == UNSUPPORTED
    assert q(g=64, inp=1024) == UNSUPPORTED         # p = 2 needs g >= 128
    assert q(g=8192, inp=8192) == UNSUPPORTED
    assert q(w=FAKE + 2) == INVALID                 # misaligned
    assert "aligned" in L.higgs_last_error().decode()
    need = L.higgs_search_index_bytes(2, 256)
    assert q(index=FAKE, index_bytes=need - 1) == INVALID   # short index
    assert q(index=FAKE + 8, index_bytes=need) == INVALID   # misaligned index
    assert "index" in L.higgs_last_error().decode()


@no_gpu
def test_search_index_rejects_bad_args_before_launch(L):
    def si(grid=FAKE, p=2, n=256, index=FAKE, nbytes=None):
        nb = L.higgs_search_index_bytes(p, n) if nbytes is None else nbytes
        return L.higgs_search_index(grid, p, n, index, nb, None)
    assert L.higgs_search_index_bytes(2, 128) == -1
    assert L.higgs_search_index_bytes(3, 64) == -1
    for p, n in [(1, 16), (1, 256), (2, 64), (2, 256), (2, 1024)]:
        assert L.higgs_search_index_bytes(p, n) > 0
    assert si(grid=None) == INVALID
    assert si(index=None) == INVALID
    assert si(p=2, n=128, nbytes=1 << 20) == UNSUPPORTED
    assert si(nbytes=L.higgs_search_index_bytes(2, 256) - 1) == INVALID
    assert si(index=FAKE + 4) == INVALID
    assert "aligned" in L.higgs_last_error().decode()


@no_gpu
def test_rht_rejects_bad_args_before_launch(L):
    def r(x=FAKE, dt=1, batch=1, inp=1024, g=1024, xr=FAKE * 4):
        return L.higgs_rht_activations(x, dt, batch, inp, g, 0, xr, None)
    assert r(x=None) == INVALID
    assert r(batch=0) == INVALID
    assert r(g=1) == UNSUPPORTED
    assert r(g=8192, inp=8192) == UNSUPPORTED
    assert r(inp=1001, g=8) == INVALID
    assert r(xr=FAKE + 1024) == INVALID             # overlaps x
    assert "overlap" in L.higgs_last_error().decode()


@no_gpu
def test_qmatmul_rejects_bad_args_before_launch(L):
    def m(x=FAKE, batch=1, codes=FAKE, scales=FAKE, grid=FAKE, p=2, n=256, g=1024, out=16,
          inp=2048, y=FAKE, ws=None, wsb=0):
        return L.higgs_qmatmul(x, batch, codes, scales, grid, p, n, g, out, inp, y, ws, wsb, None)
    assert m(x=None) == INVALID
    assert m(batch=0) == INVALID
    assert m(inp=1000) == INVALID
    assert m(n=512) == UNSUPPORTED
    assert m(codes=FAKE + 4) == INVALID
    assert H.qmatmul_workspace_bytes(1, 16, 2048, 2, 256, 1024) >= 0
    assert H.qmatmul_workspace_bytes(0, 16, 2048, 2, 256, 1024) == -1
    # size limits, checked before any launch: the small-batch kernel's K
    # (32768 weights), the matrix-core path's (2^23), 2 GiB of codes
    assert m(inp=32768, y=FAKE + 2) == INVALID                # size allowed; y misaligned
    assert "aligned" in L.higgs_last_error().decode()
    assert m(inp=65536) == UNSUPPORTED
    assert "65536" in L.higgs_last_error().decode()
    assert m(batch=16, inp=65536) == INVALID                # allowed; no workspace given
    assert "workspace" in L.higgs_last_error().decode()
    assert m(batch=16, inp=1 << 24) == UNSUPPORTED
    assert m(batch=16, out=1 << 20, inp=8192) == UNSUPPORTED
    assert "2 GiB" in L.higgs_last_error().decode()
    # every format takes rows of up to 32768 weights on the small-batch
    # kernel (CH8 included, at batch 1 and 2), none above
    for p, n in ((1, 16), (1, 256), (2, 64), (2, 256), (2, 1024)):
        for batch in (1, 2):
            if H.qmatmul_workspace_bytes(batch, 16, 32768, p, n, 1024) != 0:
                continue  # the matrix-core path takes this batch
            assert m(batch=batch, p=p, n=n, inp=32768, y=FAKE + 2) == INVALID, (p, n, batch)
            assert "aligned" in L.higgs_last_error().decode()
            assert m(batch=batch, p=p, n=n, inp=33792) == UNSUPPORTED, (p, n, batch)


@no_gpu
def test_qmatmul_fused_rejects_bad_args_before_launch(L):
    def f(x=FAKE, dt=1, batch=1, codes=FAKE, scales=FAKE, grid=FAKE, p=2, n=256, g=1024, out=16,
          inp=2048, y=FAKE, ws=None, wsb=0):
        return L.higgs_qmatmul_fused(x, dt, batch, codes, scales, grid, p, n, g, 0, out, inp, y,
                                     ws, wsb, None)
    assert f(x=None) == INVALID
    assert f(dt=5) == INVALID
    assert f(batch=0) == INVALID
    assert f(n=100) == UNSUPPORTED
    assert f(x=FAKE + 8) == INVALID
    # a separate rotation pass needs workspace: refused without it
    assert H.qmatmul_fused_workspace_bytes(1, 16, 4096, 2, 256, 2048) > 0
    assert f(g=2048, inp=4096) == INVALID
    assert "workspace" in L.higgs_last_error().decode()
    assert H.qmatmul_fused_workspace_bytes(1, 16, 4096, 2, 256, 1024) == 0
    # 6- and 10-bit codes and CH8 take the matrix-core path too (workspace
    # for the fp16 copy), from a batch that depends on the format (and for
    # 8-bit pair codes on the row length); below it the small-batch kernel
    # runs without workspace
    for n in (64, 1024):
        assert H.qmatmul_workspace_bytes(32, 4096, 4096, 2, n, 1024) >= 32 * 4096 * 2
    assert H.qmatmul_workspace_bytes(32, 4096, 4096, 1, 256, 1024) >= 32 * 4096 * 2
    for batch, p, n, inp, gemm in ((4, 1, 256, 4096, False), (5, 1, 256, 4096, True),
                                   (4, 2, 64, 4096, False), (5, 2, 64, 4096, True),
                                   (4, 2, 1024, 4096, False), (5, 2, 1024, 4096, True),
                                   (4, 2, 256, 4096, False), (5, 2, 256, 4096, True),
                                   (1, 2, 256, 12288, False), (2, 2, 256, 12288, True),
                                   (4, 1, 16, 8192, False), (2, 1, 16, 8192 + 1024, True),
                                   (2, 2, 64, 12288, False), (3, 2, 64, 12288, True),
                                   (2, 1, 256, 12288, False), (3, 1, 256, 12288, True),
                                   (2, 2, 1024, 12288, False), (3, 2, 1024, 12288, True)):
        ws = H.qmatmul_workspace_bytes(batch, 4096, inp, p, n, 1024)
        assert (ws >= batch * inp * 2) if gemm else ws == 0, (batch, p, n, inp, ws)
    # g = 64 (p = 1): the matrix-core product runs a 32-column tile and takes
    # over later
    for batch, n, inp, gemm in ((8, 16, 4096, False), (9, 16, 4096, True),
                                (4, 16, 12288, False), (5, 16, 12288, True),
                                (6, 256, 12288, False), (7, 256, 12288, True)):
        ws = H.qmatmul_workspace_bytes(batch, 4096, inp, 1, n, 64)
        assert (ws >= batch * inp * 2) if gemm else ws == 0, (batch, n, inp, ws)
    # matrix-core path: the rotation happens in its activation conversion, so
    # both entry points need the same workspace (at least the fp16 copy)
    need = H.qmatmul_fused_workspace_bytes(32, 4096, 4096, 2, 256, 1024)
    assert need == H.qmatmul_workspace_bytes(32, 4096, 4096, 2, 256, 1024) >= 32 * 4096 * 2
    assert f(batch=32, out=4096, inp=4096) == INVALID
    assert "workspace" in L.higgs_last_error().decode()


@no_gpu
def test_qmatmul_fused_noalloc_rejects_before_any_device_call(L):
    """The allocation-free entry point checks its arguments and the size of
    the workspace it would take from the fixed scratch before touching the
    device."""
    def f(x=FAKE, dt=1, batch=1, p=2, n=256, g=1024, out=16, inp=2048, y=FAKE):
        return L.higgs_qmatmul_fused_noalloc(x, dt, batch, FAKE, FAKE, FAKE, p, n, g, 0, out,
                                             inp, y, None)
    assert f(x=None) == INVALID
    assert f(y=FAKE + 2) == INVALID
    assert f(inp=1000) == INVALID
    assert f(n=100) == UNSUPPORTED
    need = H.qmatmul_fused_workspace_bytes(8192, 64, 4096, 2, 256, 1024)
    assert need > (32 << 20)
    assert f(batch=8192, out=64, inp=4096) == UNSUPPORTED
    assert "scratch" in L.higgs_last_error().decode()


@no_gpu
def test_qmatmul_fused_multi_rejects_bad_args_before_launch(L):
    import ctypes
    vp3 = ctypes.c_void_p * 3

    def f(layers=3, x=FAKE, batch=1, codes=(FAKE, FAKE, FAKE), outs=(16, 16, 16), g=1024,
          inp=2048, ys=(FAKE, FAKE, FAKE), arrays=True, ws=None, wsb=0):
        c = vp3(*codes) if arrays else None
        sc = vp3(FAKE, FAKE, FAKE)
        seeds = (ctypes.c_uint64 * 3)(1, 2, 3)
        o = (ctypes.c_int64 * 3)(*outs)
        y = vp3(*ys)
        return L.higgs_qmatmul_fused_multi(layers, x, 1, batch, c, sc, FAKE, 2, 256, g, seeds, o,
                                           inp, y, ws, wsb, None)
    assert f(layers=0) == INVALID
    assert f(layers=5) == INVALID
    assert f(arrays=False) == INVALID
    assert f(x=None) == INVALID
    assert f(codes=(FAKE, FAKE + 4, FAKE)) == INVALID
    assert "layer 1" in L.higgs_last_error().decode()
    assert f(outs=(16, 0, 16)) == INVALID
    assert f(ys=(FAKE, FAKE, None)) == INVALID
    assert "layer 2" in L.higgs_last_error().decode()
    assert f(inp=1000) == INVALID
    # per-layer rotation passes (g above the slice) need the workspace
    assert f(g=2048, inp=4096) == INVALID
    assert "workspace" in L.higgs_last_error().decode()
    # the matrix-core path needs one rotated copy per layer plus each layer's
    # split partial sums: more than any single layer
    outs = [4096, 1024, 1024]
    multi = H.qmatmul_fused_multi_workspace_bytes(64, outs, 4096, 2, 256, 1024)
    single = max(H.qmatmul_fused_workspace_bytes(64, o, 4096, 2, 256, 1024) for o in outs)
    assert multi > single > 0
    assert f(batch=64, outs=tuple(outs), inp=4096, ws=FAKE, wsb=single) == INVALID
    assert "workspace" in L.higgs_last_error().decode()
    assert H.qmatmul_fused_multi_workspace_bytes(1, outs, 4096, 2, 256, 1024) == 0
    assert H.qmatmul_fused_multi_workspace_bytes(1, [], 4096, 2, 256, 1024) == -1
    assert H.qmatmul_fused_multi_workspace_bytes(1, [16] * 5, 4096, 2, 256, 1024) == -1
