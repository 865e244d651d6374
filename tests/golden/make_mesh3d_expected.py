"""Write the float64-oracle expected values for the 2^20-token workload.

Calls only the oracle and the seeded input generator.  The oracle needs
minutes on a CPU for this size (every synthesised query and latent reduces
over all 2^20 tokens), so the GPU test compares against this stored sample:
every route of Q(X) and Z for every head, and the decoded tokens Y and the
output O at one token of every 256-token block (at a position within the
block drawn per block, so that every lane position of the decode's tiles is
covered), plus the first and the last token.

    python tests/golden/make_mesh3d_expected.py
"""

import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import flarepp_oracle as orc  # noqa: E402
from paper_2608_11519_amd import inputs as inp  # noqa: E402

OUT = os.path.join(HERE, "mesh3d_expected.npz")
BLOCK = 256  # tokens per sampled block


def sample_tokens(N):
    nblk = (N + BLOCK - 1) // BLOCK
    off = np.random.Generator(np.random.PCG64(1)).integers(0, BLOCK, size=nblk)
    idx = np.minimum(np.arange(nblk) * BLOCK + off, N - 1)
    return np.unique(np.concatenate([idx, [0, N - 1]]))


def main():
    w = inp.workload("mesh3d")
    d = inp.make_inputs(w, 0)
    X = d["X"].astype(np.float64)
    H = w.H
    Kt = orc.project(X, d["Wkt"], H)
    Vt = orc.project(X, d["Wvt"], H)
    Q, L1 = orc.sdpa(d["seeds"][None], Kt, Vt)
    del Kt, Vt
    K = orc.project(X, d["Wk"], H)
    V = orc.project(X, d["Wv"], H)
    Z, L2 = orc.sdpa(Q, K, V)
    del V
    tok = sample_tokens(w.N)
    Yh, _ = orc.sdpa(K[:, :, tok], Q, Z)
    Y = orc.merge_heads(Yh)
    O = Y @ d["Wo"].astype(np.float64)
    np.savez_compressed(OUT, tokens=tok, Q=Q.astype(np.float32), Z=Z.astype(np.float32),
                        Y=Y.astype(np.float32), O=O.astype(np.float32))
    print("wrote", OUT)


if __name__ == "__main__":
    main()
