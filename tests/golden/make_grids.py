"""Writes the grid fixtures tests/golden/grid_p{p}_n{n}.txt.

Each grid is the oracle's seeded Lloyd grid (oracle.higgs_oracle.lloyd_grid):
2^20 Gaussian p-vectors from splitmix64(seed 0) + Box-Muller, at most 300
mean updates. These grids are the MSE-optimal Gaussian grids G_n^p of
Alg. 2 ("computed once" per (n, p), Sec. 3.2) under the Lloyd reading of the
paper's CLVQ step. Only the oracle is called here.

usage: python tests/golden/make_grids.py [p n] ...
"""
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import higgs_oracle as O  # noqa: E402

SEED = 0
SAMPLES = 1 << 20
MAX_ITERS = 300
DEFAULT = [(1, 16), (2, 64), (2, 256), (2, 1024)]


def write(p, n):
    t0 = time.time()
    grid, mse, iters = O.lloyd_grid(p, n, SEED, SAMPLES, MAX_ITERS)
    path = os.path.join(HERE, f"grid_p{p}_n{n}.txt")
    with open(path, "w") as f:
        f.write(f"# HIGGS grid G_n^p, p={p} n={n}: oracle Lloyd on {SAMPLES} Gaussian samples, "
                f"seed={SEED}, max_iters={MAX_ITERS}\n")
        f.write(f"# iters={iters} mse_per_dim={mse!r}\n")
        f.write("# written by tests/golden/make_grids.py (calls oracle.higgs_oracle only)\n")
        for row in grid:
            f.write(" ".join(repr(float(v)) for v in row) + "\n")
    print(f"p={p} n={n}: iters={iters} mse={mse:.6g} ({time.time() - t0:.0f} s) -> {path}",
          flush=True)


if __name__ == "__main__":
    args = [int(a) for a in sys.argv[1:]]
    todo = list(zip(args[0::2], args[1::2])) if args else DEFAULT
    for p, n in todo:
        write(p, n)
