"""Write the float64-oracle gradients of the mixer backward at 2^18 tokens.

Calls only the oracle and the seeded input generator.  The workload is
grid2d's widths (C = 128, H = 8, M = 128) over N = 2^18 tokens of one batch
entry, bf16 storage (the fp32 path reads the same stored values).  The
oracle needs a few minutes on a CPU at this size, so the GPU test compares
against this stored copy: the seed gradient, the five weight gradients, the
summed latent and query gradients dZ, dQ, and the input gradient dX at one
token of every 512-token block (at a position within the block drawn per
block) plus the first and the last token.

    python tests/golden/make_backward_expected.py
"""

import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import flarepp_oracle as orc  # noqa: E402
from paper_2608_11519_amd import inputs as inp  # noqa: E402

OUT = os.path.join(HERE, "backward_quartermega_expected.npz")
BLOCK = 512
INPUT_SEED, DO_SEED = 30, 31


def workload():
    return inp.Workload("bwd-quartermega", 1, 1 << 18, 128, 8, 128, "bf16", "normal")


def sample_tokens(N):
    nblk = (N + BLOCK - 1) // BLOCK
    off = np.random.Generator(np.random.PCG64(2)).integers(0, BLOCK, size=nblk)
    idx = np.minimum(np.arange(nblk) * BLOCK + off, N - 1)
    return np.unique(np.concatenate([idx, [0, N - 1]]))


def main():
    w = workload()
    d = inp.make_inputs(w, INPUT_SEED)
    dO = inp.make_tensor((w.B, w.N, w.C), DO_SEED, w.dtype)
    g = orc.mixer_backward(d["X"], d["Wk"], d["Wv"], d["Wkt"], d["Wvt"], d["Wo"], d["seeds"], w.H, dO)
    tok = sample_tokens(w.N)
    out = {k: g[k].astype(np.float32) for k in ("dseeds", "dWk", "dWv", "dWkt", "dWvt", "dWo", "dZ", "dQ")}
    np.savez_compressed(OUT, tokens=tok, dX=g["dX"][:, tok].astype(np.float32), **out)
    print("wrote", OUT)


if __name__ == "__main__":
    main()
