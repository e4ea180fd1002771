"""Writes chain_splitmix_tokens.txt: token blocks whose chain reproduces the
published SplitMix64 outputs.

With pool seed S = 0 and block size 16 the chain starts at h_{-1} = 0, so
h_0 = splitmix64(0 xor M_0) is the stream's first output when block 0 is all
zero tokens (M_0 = 0).  Step j gives h_j = mix64((h_{j-1} xor M_j) + gamma),
which is the (j+1)-th output of the stream seeded at 0, mix64((j+1) gamma),
exactly when h_{j-1} xor M_j = j gamma, that is when
    M_j = out_{j-1} xor (j gamma mod 2^64),
where out_i are the published outputs (splitmix64_seed0.txt).  So the four
blocks written here make h_0 .. h_3 equal the four published words, and a
test that runs any implementation of the chain over them checks its
structure (the xor with the previous hash, the added gamma, the block index
of M_j, the start value S) against values published outside this project.

M_j = sum_m tok_m t_m mod 2^64 with the oracle's token keys t_m (odd).  Two
tokens absorb the target: with the other fourteen fixed (small seeded
values), tok_0 t_0 + tok_1 t_1 = R needs tok_0 = c - x u, tok_1 = x, where
u = t_1 / t_0 and c = R / t_0 mod 2^64, and both in [0, 2^32).  The pairs
(x, x u + k 2^64) form a two-dimensional lattice; a Lagrange-Gauss reduced
basis and rounding of the target (2^31, c - 2^31) find a point in that box
(a few seeds of the fixed tokens are tried if needed).

Only the oracle's token keys are used.  Run from the repository root:
    python tests/golden/make_chain_tokens.py
"""

from __future__ import annotations

import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import oracle as O  # noqa: E402
from tests.chain_tokens import solve_block  # noqa: E402

M64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
BS = 16
SEED = 0
OUT = os.path.join(HERE, "chain_splitmix_tokens.txt")


def published():
    with open(os.path.join(HERE, "splitmix64_seed0.txt")) as f:
        return [int(ln.split()[0], 16) for ln in f if ln.strip() and not ln.startswith("#")]


def main():
    out = published()
    keys = [O.token_key(SEED, m) for m in range(BS)]
    rng = np.random.default_rng(20261202)
    blocks = [[0] * BS]
    for j in range(1, len(out)):
        blocks.append(solve_block(out[j - 1] ^ (j * GAMMA & M64), keys, rng))
    toks = np.array([t for blk in blocks for t in blk], np.uint32)
    h = O.chain(toks, BS, SEED)
    assert [int(x) for x in h] == out, "chain does not reproduce the published outputs"
    with open(OUT, "w") as f:
        f.write("# Token blocks (block size 16, pool seed 0) whose chain h_0 .. h_3 equals the\n")
        f.write("# published SplitMix64 outputs for seed 0 (splitmix64_seed0.txt): block 0 is\n")
        f.write("# all zero, block j makes M_j = out_{j-1} xor j*gamma.  Written by\n")
        f.write("# make_chain_tokens.py from the oracle's token keys; one block per line,\n")
        f.write("# 16 decimal u32 tokens.\n")
        for blk in blocks:
            f.write(" ".join(str(t) for t in blk) + "\n")
    print(f"wrote {OUT}")


if __name__ == "__main__":
    main()
