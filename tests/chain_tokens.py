"""Token blocks with a chosen multilinear: the lattice solver behind the
chain fixtures.

M = sum_m tok_m t_m mod 2^64 over a block's 16 tokens with odd token keys
t_m.  Two tokens absorb any target R: with the other fourteen fixed (small
seeded values), tok_0 t_0 + tok_1 t_1 = R needs tok_0 = c - x u and
tok_1 = x, where u = t_1 / t_0 and c = R / t_0 mod 2^64, both in [0, 2^32).
The pairs (x, x u + k 2^64) form a two-dimensional lattice; a
Lagrange-Gauss reduced basis and rounding of the target (2^31, c - 2^31)
find a point in that box (a few seeds of the fixed tokens are tried if
needed).  The keys are passed in (the oracle's token keys), so nothing here
computes the method's arithmetic.
"""

from __future__ import annotations

BS = 16


def gauss_reduce(b1, b2):
    def n2(v):
        return v[0] * v[0] + v[1] * v[1]

    if n2(b1) > n2(b2):
        b1, b2 = b2, b1
    while True:
        den = n2(b1)
        num = b1[0] * b2[0] + b1[1] * b2[1]
        mu = (2 * num + den) // (2 * den)  # nearest integer to num / den
        b2 = (b2[0] - mu * b1[0], b2[1] - mu * b1[1])
        if n2(b2) >= n2(b1):
            return b1, b2
        b1, b2 = b2, b1


def near_points(b1, b2, t):
    """Lattice points a b1 + b b2 around the real solution of t = a b1 + b b2."""
    det = b1[0] * b2[1] - b1[1] * b2[0]
    a_num = t[0] * b2[1] - t[1] * b2[0]
    b_num = b1[0] * t[1] - b1[1] * t[0]
    a0, b0 = a_num // det, b_num // det
    for da in (-1, 0, 1, 2):
        for db in (-1, 0, 1, 2):
            a, b = a0 + da, b0 + db
            yield (a * b1[0] + b * b2[0], a * b1[1] + b * b2[1])


def solve_block(target, keys, rng):
    """16 u32 tokens whose multilinear with `keys` is `target` mod 2^64."""
    t0inv = pow(keys[0], -1, 1 << 64)
    u = keys[1] * t0inv % (1 << 64)
    b1, b2 = gauss_reduce((1, u), (0, 1 << 64))
    for _ in range(64):
        rest = [int(x) for x in rng.integers(0, 32000, size=BS - 2)]
        r = (target - sum(t * k for t, k in zip(rest, keys[2:]))) % (1 << 64)
        c = r * t0inv % (1 << 64)
        for x, y in near_points(b1, b2, (1 << 31, c - (1 << 31))):
            tok0 = c - y
            if 0 <= x < (1 << 32) and 0 <= tok0 < (1 << 32):
                toks = [tok0, x] + rest
                assert sum(t * k for t, k in zip(toks, keys)) % (1 << 64) == target
                return toks
    raise RuntimeError("no token block found")
