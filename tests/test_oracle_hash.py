"""Pins for the oracle's arithmetic: key schedule, block digest, token chain.

Each test checks the oracle against something other than itself: published
SplitMix64 outputs, closed forms of the multilinear digest, exhaustive single
bit flips, and structural properties of the chain.
"""

import numpy as np
import pytest

from oracle import oracle as O
from tests.conftest import golden_lines

M64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
GOLD = [int(x[0], 16) for x in golden_lines("splitmix64_seed0.txt")]


def words_to_bytes(words):
    return np.asarray(words, dtype="<u8").view(np.uint8)


# ------------------------------------------------------------------ SplitMix64


def test_splitmix64_matches_published_outputs():
    for i, g in enumerate(GOLD):
        assert O.splitmix64_at(0, i) == g
    # the one-step form is the first output from a state
    assert O.splitmix64(0) == GOLD[0]
    # a stream advanced by i gammas continues the same sequence
    assert O.splitmix64_at(GAMMA, 0) == GOLD[1]
    assert O.splitmix64_at((2 * GAMMA) & M64, 1) == GOLD[3]


def test_mix64_fixes_zero_and_is_injective_on_sample():
    assert O.mix64(0) == 0
    rng = np.random.default_rng(1)
    xs = [int(x) for x in rng.integers(0, 2**63, size=4000, dtype=np.int64)]
    assert len({O.mix64(x) for x in xs}) == len(set(xs))


def _unxorshift(y: int, s: int) -> int:
    """Inverse of y = x ^ (x >> s) on 64-bit words: recover x from its top
    bits down, s bits at a time."""
    x = y
    for _ in range(64 // s + 1):
        x = y ^ (x >> s)
    return x & M64


def _mix64_inverse(z: int) -> int:
    """The SplitMix64 finaliser run backwards: each step is a bijection (xor
    with a right shift, multiplication by an odd constant mod 2^64)."""
    c1, c2 = 0xBF58476D1CE4E5B9, 0x94D049BB133111EB
    z = _unxorshift(z, 31)
    z = z * pow(c2, -1, 1 << 64) & M64
    z = _unxorshift(z, 27)
    z = z * pow(c1, -1, 1 << 64) & M64
    return _unxorshift(z, 30)


def test_mix64_is_the_published_bijection():
    # the oracle's finaliser undone step by step by the inverse of the
    # published steps: a changed shift, constant or step order breaks it
    rng = np.random.default_rng(3)
    xs = [0, 1, M64, GAMMA] + [int(v) for v in rng.integers(0, 2**64, size=300, dtype=np.uint64)]
    for x in xs:
        assert _mix64_inverse(O.mix64(x)) == x
    # and the published outputs come from the states (i+1) * gamma
    for i, g in enumerate(GOLD):
        assert _mix64_inverse(g) == (i + 1) * GAMMA & M64


def test_key_schedules_are_odd_stream_outputs():
    for i, g in enumerate(GOLD):
        assert O.kv_key(0, i) == g | 1
        # token keys use the complemented seed: seed 2^64-1 -> stream from 0
        assert O.token_key(M64, i) == g | 1
    rng = np.random.default_rng(2)
    for s in rng.integers(0, 2**63, size=20, dtype=np.int64):
        for i in (0, 1, 7, 4095, 262143):
            assert O.kv_key(int(s), i) & 1 == 1


# ---------------------------------------------------------------- block digest


def test_digest_of_zero_block_is_zero():
    assert O.block_digest(np.zeros(4096, np.uint8), 1234) == 0


def test_digest_of_unit_word_is_its_key():
    # D(e_i) = k_i: with seed 0 these are the published stream outputs
    for i, g in enumerate(GOLD):
        w = np.zeros(8, np.uint64)
        w[i] = 1
        assert O.block_digest(words_to_bytes(w), 0) == g | 1


def test_words_are_little_endian():
    seed = 99
    k0 = O.kv_key(seed, 0)
    k1 = O.kv_key(seed, 1)
    for q in range(16):
        buf = np.zeros(16, np.uint8)
        buf[q] = 0xA5
        k = k0 if q < 8 else k1
        assert O.block_digest(buf, seed) == (0xA5 << (8 * (q % 8))) * k & M64


def test_digest_is_additive_and_scales():
    rng = np.random.default_rng(3)
    seed = 7
    a = rng.integers(0, 2**64, size=512, dtype=np.uint64)
    b = rng.integers(0, 2**64, size=512, dtype=np.uint64)
    da = O.block_digest(words_to_bytes(a), seed)
    db = O.block_digest(words_to_bytes(b), seed)
    assert O.block_digest(words_to_bytes(a + b), seed) == (da + db) & M64
    c = 0x1234567
    assert O.block_digest(words_to_bytes(a * np.uint64(c)), seed) == (c * da) & M64


def test_digest_against_python_bigint_sum():
    rng = np.random.default_rng(4)
    seed = 0xDEADBEEF
    w = rng.integers(0, 2**64, size=300, dtype=np.uint64)
    expect = sum(int(x) * O.kv_key(seed, i) for i, x in enumerate(w)) % (1 << 64)
    assert O.block_digest(words_to_bytes(w), seed) == expect


def test_every_single_bit_flip_is_detected_exhaustive():
    """All 131072 single-bit flips of a 16 KiB block (the tiny pool's block
    size): the digest changes by exactly +-2^beta * k_i, never by 0."""
    rng = np.random.default_rng(5)
    seed = 1001
    block = rng.integers(0, 256, size=16384, dtype=np.uint8)
    d0 = O.block_digest(block, seed)
    words = block.view("<u8")
    keys = [O.kv_key(seed, i) for i in range(words.size)]
    for bit in range(8 * block.size):
        i, beta = divmod(bit, 64)
        flipped = block.copy()
        flipped[bit // 8] ^= np.uint8(1 << (bit % 8))
        d1 = O.block_digest(flipped, seed)
        was_set = (int(words[i]) >> beta) & 1
        delta = (-(1 << beta) if was_set else (1 << beta)) * keys[i] & M64
        assert (d1 - d0) & M64 == delta
        assert d1 != d0


def test_two_sign_bit_flips_can_cancel():
    """The documented limit: bit 63 flipped in two words of one block changes
    the digest by 2^63 (k_i +- k_j), which is 0 mod 2^64 since keys are odd."""
    block = np.zeros(64, np.uint8)
    d0 = O.block_digest(block, 5)
    block[7] ^= 0x80
    block[15] ^= 0x80
    assert O.block_digest(block, 5) == d0


# ------------------------------------------------------------- head shards


def _full_and_shard(full, first, heads):
    """(full canonical bytes, the shard's own canonical bytes) of a block
    given as [plane][token][head][row byte]."""
    return full.reshape(-1), np.ascontiguousarray(full[:, :, first:first + heads, :]).reshape(-1)


@pytest.mark.parametrize("heads", [1, 2, 4, 8])
def test_head_shards_add_up_to_the_block_digest(heads):
    """Under tensor parallelism by KV head each GPU holds a slice of every
    block's heads.  Shard digests (each word keyed by its position in the
    full block) over a partition of the heads add up to the full block's
    digest, and each equals the full digest of the block with every other
    head's bytes zeroed (linearity: zero words contribute nothing)."""
    rng = np.random.default_rng(40 + heads)
    planes, bs, total, row = 3, 4, 8, 24
    seed = 777
    full = rng.integers(0, 256, size=(planes, bs, total, row), dtype=np.uint8)
    d_full = O.block_digest(full.reshape(-1), seed)
    acc = 0
    for first in range(0, total, heads):
        _, shard = _full_and_shard(full, first, heads)
        d = O.shard_digest(shard, seed, planes, bs, heads, row, total, first)
        masked = np.zeros_like(full)
        masked[:, :, first:first + heads, :] = full[:, :, first:first + heads, :]
        assert d == O.block_digest(masked.reshape(-1), seed)
        acc = (acc + d) & M64
    assert acc == d_full


def test_unsharded_shard_digest_is_the_block_digest():
    rng = np.random.default_rng(48)
    full = rng.integers(0, 256, size=(2, 16, 2, 128), dtype=np.uint8)
    assert O.shard_digest(full.reshape(-1), 5, 2, 16, 2, 128, 2, 0) == O.block_digest(full.reshape(-1), 5)


# ----------------------------------------------------------- canonical layout


def test_canonical_block_is_plane_major_concatenation():
    planes, nb, chunk = 3, 5, 32
    pool = np.zeros(planes * nb * chunk, np.uint8)
    p, b, q = 2, 3, 11
    pool[(p * nb + b) * chunk + q] = 0x5C
    canon = O.canonical_block(pool, planes, nb, chunk, b)
    assert canon.size == planes * chunk
    assert np.flatnonzero(canon).tolist() == [p * chunk + q]
    idx = p * chunk + q
    assert O.block_digest(canon, 17) == (0x5C << (8 * (idx % 8))) * O.kv_key(17, idx // 8) & M64
    # other blocks see nothing
    for other in range(nb):
        if other != b:
            assert not O.canonical_block(pool, planes, nb, chunk, other).any()


def test_whole_pool_digests_are_the_single_block_digests():
    rng = np.random.default_rng(12)
    for planes, nb, chunk in ((1, 7, 16), (3, 5, 32), (4, 9, 8)):
        pool = rng.integers(0, 256, size=planes * nb * chunk, dtype=np.uint8)
        whole = O.pool_digests(pool, planes, nb, chunk, 23)
        one = [O.block_digest(O.canonical_block(pool, planes, nb, chunk, b), 23) for b in range(nb)]
        assert whole.tolist() == one
    # one set byte reaches only its own block, weighted by its word's key
    planes, nb, chunk = 3, 5, 32
    pool = np.zeros(planes * nb * chunk, np.uint8)
    pool[(2 * nb + 3) * chunk + 11] = 0x5C
    idx = 2 * chunk + 11
    want = (0x5C << (8 * (idx % 8))) * O.kv_key(17, idx // 8) & M64
    assert O.pool_digests(pool, planes, nb, chunk, 17).tolist() == [0, 0, 0, want, 0]


def test_apply_flip_addresses_canonical_bits():
    planes, nb, chunk = 4, 3, 16
    rng = np.random.default_rng(6)
    pool = rng.integers(0, 256, size=planes * nb * chunk, dtype=np.uint8)
    for b in range(nb):
        for bit in (0, 7, 8, 127, 128, 8 * planes * chunk - 1):
            before = O.canonical_block(pool, planes, nb, chunk, b)
            O.apply_flip(pool, planes, nb, chunk, b, bit)
            after = O.canonical_block(pool, planes, nb, chunk, b)
            diff = np.flatnonzero(before != after)
            assert diff.tolist() == [bit // 8]
            assert int(before[bit // 8] ^ after[bit // 8]) == 1 << (bit % 8)
    with pytest.raises(ValueError):
        O.apply_flip(pool, planes, nb, chunk, 0, 8 * planes * chunk)


# ---------------------------------------------------------------- token chain


def test_token_multilinear_unit_tokens_give_token_keys():
    for m, g in enumerate(GOLD):
        tok = np.zeros(16, np.uint32)
        tok[m] = 1
        assert O.token_multilinear(tok, M64) == g | 1
        tok[m] = 31999
        assert O.token_multilinear(tok, M64) == 31999 * (g | 1) & M64


def test_chain_first_step_on_zero_tokens_is_published_output():
    # h_0 = splitmix64(S xor 0) = first stream output from state S = 0
    h = O.chain(np.zeros(16, np.uint32), 16, 0)
    assert int(h[0]) == GOLD[0]
    assert O.chain_hash(np.zeros(0, np.uint32), 16, 12345) == 12345


def chain_fixture():
    """Token blocks (block size 16, pool seed 0) whose chain is the published
    SplitMix64 stream (tests/golden/make_chain_tokens.py)."""
    return np.array([int(t) for row in golden_lines("chain_splitmix_tokens.txt") for t in row],
                    np.uint32)


def test_chain_reproduces_published_outputs():
    # block 0 is zero tokens and block j has M_j = out_{j-1} xor j*gamma, so
    # h_j = splitmix64(h_{j-1} xor M_j) = mix64((j+1) gamma) = out_j: the
    # whole chain (xor with the previous hash, added gamma, block index of
    # M_j, start value S = 0) against the four published outputs
    toks = chain_fixture()
    assert toks.size == 4 * 16
    assert [int(h) for h in O.chain(toks, 16, 0)] == GOLD
    for k in range(1, 5):
        assert O.chain_hash(toks[: 16 * k], 16, 0) == GOLD[k - 1]
    # the same tokens in another block order, or under another seed, leave
    # the stream
    swapped = np.concatenate([toks[:16], toks[32:48], toks[16:32], toks[48:]])
    assert [int(h) for h in O.chain(swapped, 16, 0)][1:] != GOLD[1:]
    assert [int(h) for h in O.chain(toks, 16, 1)] != GOLD


def test_chain_is_prefix_closed_and_shared_prefixes_collide():
    rng = np.random.default_rng(7)
    bs, seed = 16, 1002
    base = rng.integers(0, 32000, size=16 * 9, dtype=np.uint32)
    h_full = O.chain(base, bs, seed)
    for k in range(1, 9):
        assert np.array_equal(O.chain(base[: k * bs], bs, seed), h_full[:k])
        other = np.concatenate([base[: k * bs], rng.integers(0, 32000, size=40, dtype=np.uint32)])
        h_other = O.chain(other, bs, seed)
        assert np.array_equal(h_other[:k], h_full[:k])
        assert h_other[k] != h_full[k]


def test_chain_depends_on_every_token_and_on_seed():
    rng = np.random.default_rng(8)
    tok = rng.integers(0, 32000, size=50, dtype=np.uint32)
    h0 = O.chain_hash(tok, 16, 5)
    for pos in range(tok.size):
        t2 = tok.copy()
        t2[pos] ^= 1
        assert O.chain_hash(t2, 16, 5) != h0
    assert O.chain_hash(tok, 16, 6) != h0


def test_chain_ragged_tail_counts_only_present_tokens():
    # a trailing zero token inside the last block adds 0 * t_m: documented
    # collision of the partial-block reading
    tok = np.array([3, 1, 4, 1, 5], np.uint32)
    assert O.chain_hash(tok, 16, 9) == O.chain_hash(np.append(tok, 0), 16, 9)
    assert O.chain_hash(tok, 16, 9) != O.chain_hash(np.append(tok, 2), 16, 9)
    # block boundaries matter: 16 tokens then 1 token is two blocks
    t17 = np.arange(17, dtype=np.uint32)
    assert O.chain(t17, 16, 9).size == 2
