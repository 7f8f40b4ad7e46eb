"""Python binding of libhiggs.so (ctypes): argument marshalling only.

Every computation runs in the library's HIP kernels (or, for the grid and the
sign vector, in its host C++). PyTorch provides device memory and the current
stream. If the library is not built, every entry point raises.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
# HIGGS_LIB names another build of the library (e.g. one with host sanitizers)
LIB_PATH = os.environ.get("HIGGS_LIB") or os.path.join(_PKG, "libhiggs.so")

HIGGS_F32 = 0
HIGGS_BF16 = 1
SUPPORTED_GRIDS = ((1, 16), (1, 256), (2, 64), (2, 256), (2, 1024))

_lib = None


class HiggsError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"higgs status {status}: {message}")
        self.status = status


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it first "
                           "(python -c 'import __graft_entry__ as g; g.build()')")
    L = ctypes.CDLL(LIB_PATH)
    i64, i32, u64, vp = ctypes.c_int64, ctypes.c_int, ctypes.c_uint64, ctypes.c_void_p
    L.higgs_abi_version.restype = i32
    L.higgs_last_error.restype = ctypes.c_char_p
    L.higgs_make_grid.argtypes = [i32, i32, u64, i64, i32, vp, vp, vp]
    L.higgs_make_grid.restype = i32
    L.higgs_make_uniform_grid.argtypes = [i32, vp, vp, vp]
    L.higgs_make_uniform_grid.restype = i32
    L.higgs_layer_error.argtypes = [vp, i32, i64, i64, vp, vp, vp, i32, i32, i32, u64, vp, vp,
                                    vp]
    L.higgs_layer_error.restype = i32
    L.higgs_allocate_bits.argtypes = [i32, i32, vp, vp, vp, vp, ctypes.c_double, vp, vp, vp]
    L.higgs_allocate_bits.restype = i32
    L.higgs_gptq_factor_workspace_bytes.argtypes = [i64, i64]
    L.higgs_gptq_factor_workspace_bytes.restype = i64
    L.higgs_gptq_factor.argtypes = [vp, i64, i64, ctypes.c_double, vp, vp, i64, vp]
    L.higgs_gptq_factor.restype = i32
    L.higgs_quantize_gptq_workspace_bytes.argtypes = [i64, i64, i32]
    L.higgs_quantize_gptq_workspace_bytes.restype = i64
    L.higgs_quantize_gptq.argtypes = [vp, i32, i64, i64, vp, i32, i32, i32, u64, vp, vp, vp, vp,
                                      i64, vp]
    L.higgs_quantize_gptq.restype = i32
    L.higgs_rht_signs.argtypes = [u64, i32, vp]
    L.higgs_rht_signs.restype = i32
    L.higgs_codes_row_bytes.argtypes = [i64, i32, i32]
    L.higgs_codes_row_bytes.restype = i64
    L.higgs_qmatmul_workspace_bytes.argtypes = [i64, i64, i64, i32, i32, i32]
    L.higgs_qmatmul_workspace_bytes.restype = i64
    L.higgs_search_index_bytes.argtypes = [i32, i32]
    L.higgs_search_index_bytes.restype = i64
    L.higgs_search_index.argtypes = [vp, i32, i32, vp, i64, vp]
    L.higgs_search_index.restype = i32
    L.higgs_quantize.argtypes = [vp, i32, i64, i64, vp, i32, i32, vp, i64, i32, u64, vp, vp, vp]
    L.higgs_quantize.restype = i32
    L.higgs_rht_activations.argtypes = [vp, i32, i64, i64, i32, u64, vp, vp]
    L.higgs_rht_activations.restype = i32
    L.higgs_qmatmul.argtypes = [vp, i64, vp, vp, vp, i32, i32, i32, i64, i64, vp, vp, i64, vp]
    L.higgs_qmatmul.restype = i32
    L.higgs_qmatmul_fused_workspace_bytes.argtypes = [i64, i64, i64, i32, i32, i32]
    L.higgs_qmatmul_fused_workspace_bytes.restype = i64
    L.higgs_qmatmul_fused.argtypes = [vp, i32, i64, vp, vp, vp, i32, i32, i32, u64, i64, i64, vp,
                                      vp, i64, vp]
    L.higgs_qmatmul_fused.restype = i32
    L.higgs_qmatmul_fused_noalloc.argtypes = [vp, i32, i64, vp, vp, vp, i32, i32, i32, u64, i64,
                                              i64, vp, vp]
    L.higgs_qmatmul_fused_noalloc.restype = i32
    L.higgs_qmatmul_fused_multi.argtypes = [i32, vp, i32, i64, vp, vp, vp, i32, i32, i32, vp, vp,
                                            i64, vp, vp, i64, vp]
    L.higgs_qmatmul_fused_multi.restype = i32
    L.higgs_qmatmul_fused_multi_workspace_bytes.argtypes = [i32, i64, vp, i64, i32, i32, i32]
    L.higgs_qmatmul_fused_multi_workspace_bytes.restype = i64
    _lib = L
    return L


def _check(status: int):
    if status != 0:
        raise HiggsError(status, lib().higgs_last_error().decode())


def _ptr(t) -> int:
    return int(t.data_ptr())


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(int(stream.cuda_stream))


def _need_cuda(name, t, dtypes):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} must have dtype in {dtypes}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _dtype_code(t):
    import torch
    return HIGGS_F32 if t.dtype == torch.float32 else HIGGS_BF16


# ---------------------------------------------------------------------------
# host entry points
# ---------------------------------------------------------------------------

def abi_version() -> int:
    return int(lib().higgs_abi_version())


def make_grid(p: int, n: int, seed: int = 0, num_samples: int = 1 << 20, max_iters: int = 300):
    """Lloyd grid for N(0, I_p) (host). Returns (grid float32 (n, p), mse_per_dim, iters)."""
    grid = np.zeros((n, p), dtype=np.float32)
    mse = ctypes.c_double(0.0)
    iters = ctypes.c_int(0)
    _check(lib().higgs_make_grid(p, n, seed, num_samples, max_iters,
                                 grid.ctypes.data_as(ctypes.c_void_p),
                                 ctypes.addressof(mse), ctypes.addressof(iters)))
    return grid, mse.value, iters.value


def make_uniform_grid(n: int):
    """Uniform MSE-optimal grid for N(0, 1) (host; CH8 with n = 256).
    Returns (grid float32 (n, 1), step, mse)."""
    grid = np.zeros((n, 1), dtype=np.float32)
    step = ctypes.c_double(0.0)
    mse = ctypes.c_double(0.0)
    _check(lib().higgs_make_uniform_grid(n, grid.ctypes.data_as(ctypes.c_void_p),
                                         ctypes.addressof(step), ctypes.addressof(mse)))
    return grid, step.value, mse.value


def rht_signs(seed: int, g: int) -> np.ndarray:
    out = np.zeros(g, dtype=np.int8)
    _check(lib().higgs_rht_signs(seed, g, out.ctypes.data_as(ctypes.c_void_p)))
    return out


def codes_row_bytes(inp: int, p: int, n: int) -> int:
    return int(lib().higgs_codes_row_bytes(inp, p, n))


def qmatmul_workspace_bytes(batch: int, out: int, inp: int, p: int, n: int, g: int) -> int:
    return int(lib().higgs_qmatmul_workspace_bytes(batch, out, inp, p, n, g))


def qmatmul_fused_workspace_bytes(batch: int, out: int, inp: int, p: int, n: int, g: int) -> int:
    return int(lib().higgs_qmatmul_fused_workspace_bytes(batch, out, inp, p, n, g))


# ---------------------------------------------------------------------------
# device entry points (torch tensors on the current HIP device)
# ---------------------------------------------------------------------------

def search_index_bytes(p: int, n: int) -> int:
    """Bytes of the nearest-point search index of a (p, n) grid."""
    b = int(lib().higgs_search_index_bytes(p, n))
    if b < 0:
        raise HiggsError(2, f"grid (p={p}, n={n}) not supported")
    return b


def search_index(grid, index=None, stream=None):
    """The grid's search index (device uint8 tensor), built on the GPU.

    grid: [n, p] float32 on the device. Build it once per grid and pass it to
    every quantize() call that uses that grid.
    """
    import torch
    _need_cuda("grid", grid, (torch.float32,))
    n, p = grid.shape
    nb = search_index_bytes(p, n)
    if index is None:
        index = torch.empty(nb, dtype=torch.uint8, device=grid.device)
    _need_cuda("index", index, (torch.uint8,))
    if index.numel() < nb:
        raise ValueError("index buffer too small")
    _check(lib().higgs_search_index(_ptr(grid), p, n, _ptr(index), index.numel(), _stream(stream)))
    return index


def quantize(w, grid, g: int, seed: int, codes=None, scales=None, stream=None, index=None):
    """Alg. 1 on the GPU. w: [out, in] float32 or bfloat16; grid: [n, p] float32.

    index: the grid's search_index(); None builds one for this call, False
    passes none (every vector then scans all n points; same codes).
    Returns (codes uint8 [out, row_bytes], scales float16 [out, in/g]).
    """
    import torch
    _need_cuda("w", w, (torch.float32, torch.bfloat16))
    _need_cuda("grid", grid, (torch.float32,))
    out, inp = w.shape
    n, p = grid.shape
    rb = codes_row_bytes(inp, p, n)
    if rb <= 0:
        raise HiggsError(1, f"invalid code row for in={inp}, p={p}, n={n}")
    if codes is None:
        codes = torch.empty((out, rb), dtype=torch.uint8, device=w.device)
    if scales is None:
        scales = torch.empty((out, inp // g if g > 0 else 0), dtype=torch.float16, device=w.device)
    _need_cuda("codes", codes, (torch.uint8,))
    _need_cuda("scales", scales, (torch.float16,))
    if codes.numel() < out * rb or scales.numel() < out * (inp // g):
        raise ValueError("codes or scales buffer too small")
    if index is None:
        index = search_index(grid, stream=stream)
    if index is False:
        ip, ib = None, 0
    else:
        _need_cuda("index", index, (torch.uint8,))
        ip, ib = _ptr(index), index.numel()
    _check(lib().higgs_quantize(_ptr(w), _dtype_code(w), out, inp, _ptr(grid), p, n, ip, ib, g,
                                seed, _ptr(codes), _ptr(scales), _stream(stream)))
    return codes, scales


def layer_error(w, codes, scales, grid, g: int, seed: int, group_err=None, t2=None,
                stream=None):
    """Per-group [err, norm] of a quantized layer and its t^2 on the GPU
    (fp64 device tensors [out * in/g, 2] and [1]). Returns (t2 as a float,
    group_err); reading t2 synchronises the stream."""
    import torch
    _need_cuda("w", w, (torch.float32, torch.bfloat16))
    _need_cuda("grid", grid, (torch.float32,))
    _need_cuda("codes", codes, (torch.uint8,))
    _need_cuda("scales", scales, (torch.float16,))
    out, inp = w.shape
    n, p = grid.shape
    if group_err is None:
        group_err = torch.empty((out * (inp // g), 2), dtype=torch.float64, device=w.device)
    if t2 is None:
        t2 = torch.empty(1, dtype=torch.float64, device=w.device)
    _need_cuda("group_err", group_err, (torch.float64,))
    _need_cuda("t2", t2, (torch.float64,))
    _check(lib().higgs_layer_error(_ptr(w), _dtype_code(w), out, inp, _ptr(codes), _ptr(scales),
                                   _ptr(grid), p, n, g, seed, _ptr(group_err), _ptr(t2),
                                   _stream(stream)))
    return float(t2.item()), group_err


def allocate_bits(alpha, t2, bits, sizes, b_max: float):
    """Exact per-layer option choice: min sum alpha_l t2[l, j_l] s.t. sum
    bits[j_l] d_l <= b_max sum d_l (host). Returns (choice int32 [L],
    objective, avg_bits)."""
    alpha = np.ascontiguousarray(alpha, dtype=np.float64)
    t2 = np.ascontiguousarray(t2, dtype=np.float64)
    bits = np.ascontiguousarray(bits, dtype=np.float64)
    sizes = np.ascontiguousarray(sizes, dtype=np.int64)
    L, J = t2.shape
    if alpha.shape != (L,) or bits.shape != (J,) or sizes.shape != (L,):
        raise ValueError("alpha [L], t2 [L, J], bits [J], sizes [L]")
    choice = np.zeros(L, dtype=np.int32)
    obj = ctypes.c_double(0.0)
    avg = ctypes.c_double(0.0)
    vp = ctypes.c_void_p
    _check(lib().higgs_allocate_bits(L, J, alpha.ctypes.data_as(vp), t2.ctypes.data_as(vp),
                                     bits.ctypes.data_as(vp), sizes.ctypes.data_as(vp),
                                     float(b_max), choice.ctypes.data_as(vp),
                                     ctypes.addressof(obj), ctypes.addressof(avg)))
    return choice, obj.value, avg.value


def gptq_factor(x_rot, damp: float = 0.01, factor=None, stream=None):
    """U (upper, row-major in a [in, in] float64 tensor) with (H + damping)^-1 =
    U^T U, H = x_rot^T x_rot over rotated calibration activations [samples, in]."""
    import torch
    _need_cuda("x_rot", x_rot, (torch.float32,))
    samples, inp = x_rot.shape
    if factor is None:
        factor = torch.empty((inp, inp), dtype=torch.float64, device=x_rot.device)
    _need_cuda("factor", factor, (torch.float64,))
    need = int(lib().higgs_gptq_factor_workspace_bytes(samples, inp))
    if need < 0:
        raise HiggsError(1, f"invalid shape samples={samples} in={inp}")
    ws = torch.empty(need, dtype=torch.uint8, device=x_rot.device)
    _check(lib().higgs_gptq_factor(_ptr(x_rot), samples, inp, float(damp), _ptr(factor), _ptr(ws),
                                   need, _stream(stream)))
    return factor


def quantize_gptq(w, grid, g: int, seed: int, factor, codes=None, scales=None, stream=None):
    """GPTQ rounding in place of Alg. 1's nearest point (same code / scale format)."""
    import torch
    _need_cuda("w", w, (torch.float32, torch.bfloat16))
    _need_cuda("grid", grid, (torch.float32,))
    _need_cuda("factor", factor, (torch.float64,))
    out, inp = w.shape
    n, p = grid.shape
    rb = codes_row_bytes(inp, p, n)
    if rb <= 0:
        raise HiggsError(1, f"invalid code row for in={inp}, p={p}, n={n}")
    if codes is None:
        codes = torch.empty((out, rb), dtype=torch.uint8, device=w.device)
    if scales is None:
        scales = torch.empty((out, inp // g), dtype=torch.float16, device=w.device)
    need = int(lib().higgs_quantize_gptq_workspace_bytes(out, inp, g))
    if need < 0:
        raise HiggsError(1, f"invalid shape out={out} in={inp} g={g}")
    ws = torch.empty(need, dtype=torch.uint8, device=w.device)
    _check(lib().higgs_quantize_gptq(_ptr(w), _dtype_code(w), out, inp, _ptr(grid), p, n, g, seed,
                                     _ptr(factor), _ptr(codes), _ptr(scales), _ptr(ws), need,
                                     _stream(stream)))
    return codes, scales


def rht_activations(x, g: int, seed: int, out=None, stream=None):
    """x_rot = H (sigma * x_block) / sqrt(g) per block; x: [batch, in] float32 or bfloat16."""
    import torch
    _need_cuda("x", x, (torch.float32, torch.bfloat16))
    batch, inp = x.shape
    if out is None:
        out = torch.empty((batch, inp), dtype=torch.float32, device=x.device)
    _need_cuda("out", out, (torch.float32,))
    if out.numel() < batch * inp:
        raise ValueError("out buffer too small")
    _check(lib().higgs_rht_activations(_ptr(x), _dtype_code(x), batch, inp, g, seed, _ptr(out),
                                       _stream(stream)))
    return out


def qmatmul(x_rot, codes, scales, grid, g: int, out_features: int, y=None, workspace=None,
            stream=None):
    """y = rotated-space LUT product; x_rot: [batch, in] float32. Returns y [batch, out] float32."""
    import torch
    _need_cuda("x_rot", x_rot, (torch.float32,))
    _need_cuda("codes", codes, (torch.uint8,))
    _need_cuda("scales", scales, (torch.float16,))
    _need_cuda("grid", grid, (torch.float32,))
    batch, inp = x_rot.shape
    n, p = grid.shape
    if y is None:
        y = torch.empty((batch, out_features), dtype=torch.float32, device=x_rot.device)
    _need_cuda("y", y, (torch.float32,))
    if y.numel() < batch * out_features:
        raise ValueError("y buffer too small")
    need = qmatmul_workspace_bytes(batch, out_features, inp, p, n, g)
    ws_ptr, ws_bytes = None, 0
    if need > 0:
        if workspace is None:
            workspace = torch.empty(need, dtype=torch.uint8, device=x_rot.device)
        ws_ptr, ws_bytes = _ptr(workspace), workspace.numel() * workspace.element_size()
    _check(lib().higgs_qmatmul(_ptr(x_rot), batch, _ptr(codes), _ptr(scales), _ptr(grid), p, n, g,
                               out_features, inp, _ptr(y), ws_ptr, ws_bytes, _stream(stream)))
    return y


def qmatmul_fused(x, codes, scales, grid, g: int, seed: int, out_features: int, y=None,
                  workspace=None, stream=None):
    """y = x W_hat^T from raw activations x: [batch, in] float32 or bfloat16."""
    import torch
    _need_cuda("x", x, (torch.float32, torch.bfloat16))
    _need_cuda("codes", codes, (torch.uint8,))
    _need_cuda("scales", scales, (torch.float16,))
    _need_cuda("grid", grid, (torch.float32,))
    batch, inp = x.shape
    n, p = grid.shape
    if y is None:
        y = torch.empty((batch, out_features), dtype=torch.float32, device=x.device)
    _need_cuda("y", y, (torch.float32,))
    if y.numel() < batch * out_features:
        raise ValueError("y buffer too small")
    need = qmatmul_fused_workspace_bytes(batch, out_features, inp, p, n, g)
    ws_ptr, ws_bytes = None, 0
    if need > 0:
        if workspace is None:
            workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
        ws_ptr, ws_bytes = _ptr(workspace), workspace.numel() * workspace.element_size()
    _check(lib().higgs_qmatmul_fused(_ptr(x), _dtype_code(x), batch, _ptr(codes), _ptr(scales),
                                     _ptr(grid), p, n, g, seed, out_features, inp, _ptr(y),
                                     ws_ptr, ws_bytes, _stream(stream)))
    return y


def qmatmul_fused_noalloc(x, codes, scales, grid, g: int, seed: int, out_features: int, y=None,
                          stream=None):
    """qmatmul_fused with the library's fixed scratch as the workspace (no
    device allocation by the library; calls on one device must not overlap)."""
    import torch
    _need_cuda("x", x, (torch.float32, torch.bfloat16))
    _need_cuda("codes", codes, (torch.uint8,))
    _need_cuda("scales", scales, (torch.float16,))
    _need_cuda("grid", grid, (torch.float32,))
    batch, inp = x.shape
    n, p = grid.shape
    if y is None:
        y = torch.empty((batch, out_features), dtype=torch.float32, device=x.device)
    _need_cuda("y", y, (torch.float32,))
    if y.numel() < batch * out_features:
        raise ValueError("y buffer too small")
    _check(lib().higgs_qmatmul_fused_noalloc(_ptr(x), _dtype_code(x), batch, _ptr(codes),
                                             _ptr(scales), _ptr(grid), p, n, g, seed,
                                             out_features, inp, _ptr(y), _stream(stream)))
    return y


def qmatmul_fused_multi_workspace_bytes(batch: int, outs, inp: int, p: int, n: int,
                                        g: int) -> int:
    arr = (ctypes.c_int64 * max(len(outs), 1))(*outs)
    return int(lib().higgs_qmatmul_fused_multi_workspace_bytes(len(outs), batch, arr, inp, p, n,
                                                               g))


def qmatmul_fused_multi(x, layers, grid, g: int, ys=None, workspace=None, stream=None):
    """Outputs of up to 4 layers that read the same raw activations x:
    layers = [(codes, scales, seed, out_features), ...]; returns [y_l]."""
    import torch
    _need_cuda("x", x, (torch.float32, torch.bfloat16))
    _need_cuda("grid", grid, (torch.float32,))
    batch, inp = x.shape
    n, p = grid.shape
    k = len(layers)
    if ys is None:
        ys = [torch.empty((batch, o), dtype=torch.float32, device=x.device)
              for _, _, _, o in layers]
    for (c, sc, _, o), y in zip(layers, ys):
        _need_cuda("codes", c, (torch.uint8,))
        _need_cuda("scales", sc, (torch.float16,))
        _need_cuda("y", y, (torch.float32,))
        if y.numel() < batch * o:
            raise ValueError("y buffer too small")
    need = qmatmul_fused_multi_workspace_bytes(batch, [o for *_, o in layers], inp, p, n, g)
    ws_ptr, ws_bytes = None, 0
    if need > 0:
        if workspace is None:
            workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
        ws_ptr, ws_bytes = _ptr(workspace), workspace.numel() * workspace.element_size()
    vpk = ctypes.c_void_p * max(k, 1)
    codes_a = vpk(*[_ptr(c) for c, *_ in layers])
    scales_a = vpk(*[_ptr(sc) for _, sc, *_ in layers])
    ys_a = vpk(*[_ptr(y) for y in ys])
    seeds_a = (ctypes.c_uint64 * max(k, 1))(*[sd for _, _, sd, _ in layers])
    outs_a = (ctypes.c_int64 * max(k, 1))(*[o for *_, o in layers])
    _check(lib().higgs_qmatmul_fused_multi(k, _ptr(x), _dtype_code(x), batch, codes_a, scales_a,
                                           _ptr(grid), p, n, g, seeds_a, outs_a, inp, ys_a,
                                           ws_ptr, ws_bytes, _stream(stream)))
    return ys


@dataclasses.dataclass
class QuantizedLinear:
    """A HIGGS-quantized linear layer: codes, scales, grid, group size and rotation seed."""

    codes: object
    scales: object
    grid: object
    g: int
    seed: int
    out_features: int
    in_features: int

    @classmethod
    def from_weight(cls, w, grid, g: int, seed: int):
        codes, scales = quantize(w, grid, g, seed)
        return cls(codes, scales, grid, g, seed, w.shape[0], w.shape[1])

    def forward(self, x, y=None, workspace=None):
        """y = x W_hat^T (rotation fused into the product when it fits)."""
        return qmatmul_fused(x, self.codes, self.scales, self.grid, self.g, self.seed,
                             self.out_features, y=y, workspace=workspace)

    def forward_two_step(self, x, x_rot=None, y=None):
        """Same output through the separate rotation and product calls."""
        x_rot = rht_activations(x, self.g, self.seed, out=x_rot)
        return qmatmul(x_rot, self.codes, self.scales, self.grid, self.g, self.out_features, y=y)
