"""Seeded synthetic inputs for tests and benchmarks.

This module holds no arithmetic of the quantization method: it only draws
weights and activations with NumPy's ``default_rng`` and rounds them to the
storage dtype. Both the CPU oracle (through the tests) and the HIP path take
their inputs from here.

Weight recipe (stand-in for real Llama weights, whose incoherence processing
makes them near-Gaussian after the rotation, Sec. 3.1 of the paper):
  * Student-t with 5 degrees of freedom, multiplied by 0.02 / sqrt(5/3) so the
    population standard deviation is 0.02;
  * optionally round(0.001 * in) input columns, drawn without replacement,
    multiplied by 20 (outlier channels), applied after the scaling;
  * rounded to bf16 (round to nearest even) or kept in fp32.
Activations: N(0, 1), rounded to bf16.
"""
from __future__ import annotations

import dataclasses
import numpy as np

# Llama-3.1-8B and 70B linear layer shapes, (name, out, in).
LLAMA8B_LAYERS = (
    ("q", 4096, 4096),
    ("k", 1024, 4096),
    ("v", 1024, 4096),
    ("o", 4096, 4096),
    ("gate", 14336, 4096),
    ("up", 14336, 4096),
    ("down", 4096, 14336),
)
LLAMA70B_LAYERS = (
    ("q", 8192, 8192),
    ("k", 1024, 8192),
    ("v", 1024, 8192),
    ("o", 8192, 8192),
    ("gate", 28672, 8192),
    ("up", 28672, 8192),
    ("down", 8192, 28672),
)


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); return the uint16 bit patterns."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    rounding = ((u >> 16) & 1) + 0x7FFF
    out = ((u + rounding) >> 16).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass
class Weight:
    """A synthetic weight matrix [out][in] in row-major order.

    ``values`` holds the exact values as fp32 (bf16 values are exact in fp32);
    ``bits`` holds the uint16 bf16 patterns when dtype == "bf16", else None.
    """

    values: np.ndarray
    dtype: str
    bits: np.ndarray | None
    outlier_cols: np.ndarray


def student_t_weight(out: int, inp: int, seed: int, dtype: str = "bf16",
                     outliers: bool = True, std: float = 0.02) -> Weight:
    rng = np.random.default_rng(seed)
    w = rng.standard_t(5.0, size=(out, inp)) * (std / np.sqrt(5.0 / 3.0))
    cols = np.zeros(0, dtype=np.int64)
    if outliers:
        k = int(round(0.001 * inp))
        if k > 0:
            cols = np.sort(rng.choice(inp, size=k, replace=False))
            w[:, cols] *= 20.0
    w32 = w.astype(np.float32)
    if dtype == "bf16":
        bits = f32_to_bf16_bits(w32)
        return Weight(bf16_bits_to_f32(bits), "bf16", bits, cols)
    if dtype == "f32":
        return Weight(w32, "f32", None, cols)
    raise ValueError(f"unknown dtype {dtype}")


def student_t_weight_device(out: int, inp: int, seed: int, device, outliers: bool = True,
                            std: float = 0.02):
    """The same recipe as ``student_t_weight`` (bf16), drawn on a GPU with a
    seeded torch generator, for layers too large to draw on the host in
    reasonable time (the 70B shapes). Student-t(5) is drawn as Z / sqrt(V / 5)
    with Z ~ N(0, 1) and V ~ chi2(5) = 2 * Gamma(5/2). Returns
    (bf16 tensor [out][in] on ``device``, outlier columns as a NumPy array).
    The values differ from the host recipe's (another generator); a test takes
    the oracle's copy of the rows it checks from this tensor."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    z = torch.randn((out, inp), device=device, generator=gen, dtype=torch.float32)
    conc = torch.full((out, inp), 2.5, device=device, dtype=torch.float32)
    v = 2.0 * torch._standard_gamma(conc, generator=gen)
    del conc
    w = z * torch.rsqrt(v / 5.0) * (std / np.sqrt(5.0 / 3.0))
    del z, v
    cols = np.zeros(0, dtype=np.int64)
    if outliers:
        k = int(round(0.001 * inp))
        if k > 0:
            perm = torch.randperm(inp, device=device, generator=gen)[:k]
            cols = np.sort(perm.cpu().numpy().astype(np.int64))
            w[:, torch.from_numpy(cols).to(device)] *= 20.0
    return w.to(torch.bfloat16), cols


def gaussian_weight(out: int, inp: int, seed: int) -> Weight:
    """fp32 N(0,1) weights (used where a purely Gaussian layer is wanted)."""
    rng = np.random.default_rng(seed)
    return Weight(rng.standard_normal((out, inp)).astype(np.float32), "f32", None,
                  np.zeros(0, dtype=np.int64))


@dataclasses.dataclass
class Activation:
    values: np.ndarray          # [batch][in] fp32 holding bf16-exact values
    bits: np.ndarray            # uint16 bf16 patterns


def activations(batch: int, inp: int, seed: int) -> Activation:
    rng = np.random.default_rng(seed)
    bits = f32_to_bf16_bits(rng.standard_normal((batch, inp)).astype(np.float32))
    return Activation(bf16_bits_to_f32(bits), bits)


def random_codes(out: int, n_codes_per_row: int, n: int, seed: int) -> np.ndarray:
    """Uniform code indices in [0, n), shape [out][n_codes_per_row] (int32)."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, n, size=(out, n_codes_per_row), dtype=np.int32)


def random_code_bytes(out: int, row_bytes: int, seed: int) -> np.ndarray:
    """Uniform random packed code rows, shape [out][row_bytes] (uint8). With
    n a power of two every bit pattern is a valid code stream, so these stand
    for encoded codes wherever only their traffic or their decoding matters."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, 256, size=(out, row_bytes), dtype=np.uint8)


def random_scales_f16(out: int, groups: int, seed: int, lo: float = 5e-4,
                      hi: float = 2e-3) -> np.ndarray:
    """Positive fp16 scales, shape [out][groups], returned as uint16 bit patterns."""
    rng = np.random.default_rng(seed)
    return rng.uniform(lo, hi, size=(out, groups)).astype(np.float16).view(np.uint16)


# Seeds used by the Llama-shaped workloads: base + layer index for weights,
# weight seed + 500 + batch for activations, rotation seed = layer index.
def layer_seeds(base: int, layer_index: int, batch: int) -> tuple[int, int, int]:
    w_seed = base + layer_index
    return w_seed, w_seed + 500 + batch, layer_index


def mixed_n_for_70b(seed: int = 5) -> list[int]:
    """Per-layer grid sizes for the mixed-bitwidth 70B workload (p = 2)."""
    choice = np.random.default_rng(seed).integers(0, 3, len(LLAMA70B_LAYERS))
    return [(64, 256, 1024)[int(c)] for c in choice]
