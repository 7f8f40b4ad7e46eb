"""The allocation-free product entry point against the one that takes a
workspace: same inputs, same bits, on two calls in a row (the second with a
smaller input), through the C ABI."""
import ctypes
import sys

import numpy as np
import pytest

from conftest import load_grid_fixture
from oracle import higgs_oracle as O
from paper_2411_17525_amd import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def announce(msg):
    print(f"[gpu-case] {msg}", file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def H():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2411_17525_amd import higgs
    higgs.lib()
    return higgs


def _layer(p, n, g, out, inp, seed):
    grid = load_grid_fixture(p, n)[0].astype(np.float32)
    rb = O.codes_row_bytes(inp, p, n)
    codes = torch.from_numpy(synth.random_code_bytes(out, rb, seed=seed)).cuda()
    scales = torch.from_numpy(synth.random_scales_f16(out, inp // g, seed=seed + 1)
                              .view(np.float16)).cuda()
    return codes, scales, torch.from_numpy(grid).cuda()


# pairs of calls, the second smaller: the matrix-core path with K-splits (its
# workspace holds the fp16 activations and the split partial sums), and the
# small-batch path with a separate rotation pass (g above the kernel's slice:
# the workspace holds the rotated activations)
CALLS = [
    ((2, 256, 1024, 4096, 4096, 64), (2, 256, 1024, 1024, 2048, 20)),
    ((2, 64, 1024, 14336, 4096, 33), (2, 64, 1024, 4096, 14336, 16)),
    ((2, 256, 2048, 512, 8192, 3), (2, 256, 2048, 64, 4096, 1)),
]


@pytest.mark.parametrize("pair", range(len(CALLS)))
def test_noalloc_matches_workspace_entry_point(H, pair):
    for step, (p, n, g, out, inp, batch) in enumerate(CALLS[pair]):
        announce(f"noalloc call {step}: p={p} n={n} g={g} out={out} in={inp} batch={batch}")
        need = H.qmatmul_fused_workspace_bytes(batch, out, inp, p, n, g)
        assert 0 < need <= (32 << 20)
        codes, scales, grid = _layer(p, n, g, out, inp, seed=100 * pair + step)
        x = torch.from_numpy(synth.activations(batch, inp, seed=7 * pair + step).bits
                             .view(np.int16)).cuda().view(torch.bfloat16)
        y_ws = H.qmatmul_fused(x, codes, scales, grid, g, 11 + step, out)
        y_na = torch.full((batch, out), float("nan"), device="cuda")
        H.qmatmul_fused_noalloc(x, codes, scales, grid, g, 11 + step, out, y=y_na)
        torch.cuda.synchronize()
        assert torch.equal(y_na, y_ws), (pair, step)


def test_noalloc_refuses_oversized_call(H):
    p, n, g, out, inp, batch = 2, 256, 1024, 64, 4096, 8192
    need = H.qmatmul_fused_workspace_bytes(batch, out, inp, p, n, g)
    assert need > (32 << 20)
    codes, scales, grid = _layer(p, n, g, out, inp, seed=5)
    x = torch.zeros((batch, inp), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(H.HiggsError) as e:
        H.qmatmul_fused_noalloc(x, codes, scales, grid, g, 1, out)
    assert e.value.status == 2
