"""Pins for the oracle's cache identity: the per-position identity check at
claim_check, the identity table built at offload and the reuse lookup.

The expected values never use a hash: a chain hash h_j names the token
prefix of blocks 0..j, so every expectation here is computed by comparing
token blocks directly (section 5 cache identity; Table 5 fixed cache
identity and joinable block hashes; section 7 reuse lookup E1; Table 2
ambiguity rule for duplicate ownership and cache-identity mismatch).
Tokens are drawn from [1, vocab): a trailing token 0 leaves a block's
multilinear unchanged, a documented limit of the token hash.
"""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_01387_amd.synth import from_claims
from tests.conftest import golden_lines

BS = 4
NB = 64
SEED = 4242
RNG = np.random.default_rng(99)
D0 = (np.arange(NB, dtype=np.uint64) * np.uint64(0x9E3779B1) + np.uint64(3))


def blocks_of(tokens):
    return [tuple(int(x) for x in tokens[i:i + BS]) for i in range(0, len(tokens), BS)]


def first_block_difference(a, b):
    """First block index where two token sequences differ in content or
    length, or None."""
    ba, bb = blocks_of(a), blocks_of(b)
    for j in range(max(len(ba), len(bb))):
        if j >= len(ba) or j >= len(bb) or ba[j] != bb[j]:
            return j
    return None


def rand_tokens(n):
    return RNG.integers(1, 32000, size=n, dtype=np.uint32)


def variants(tk):
    """Token sequences presented at reuse: same, one token changed, cut,
    extended, cut to a block boundary."""
    out = [tk.copy()]
    for _ in range(3):
        m = int(RNG.integers(0, tk.size))
        v = tk.copy()
        v[m] = v[m] % 31999 + 1 if v[m] != 31999 else 1
        out.append(v)
    out.append(tk[: int(RNG.integers(1, tk.size + 1))].copy())
    out.append(np.concatenate([tk, rand_tokens(int(RNG.integers(1, 2 * BS + 1)))]))
    out.append(tk[: (tk.size // BS) * BS].copy() if tk.size >= BS else tk.copy())
    return out


def test_identity_position_matches_token_comparison():
    """For each presented token sequence, against the same accepted footprint:
    the outcome is UNKNOWN at the first block whose tokens differ (or where
    the block table and the token blocks part, whichever comes first), and
    MATERIALIZED when nothing differs."""
    for trial in range(60):
        ntok = int(RNG.integers(1, 9 * BS))
        tk = rand_tokens(ntok)
        n = -(-ntok // BS)
        blocks = list(range(n))
        acc = from_claims([(7, blocks, tk)])
        for pres in variants(tk):
            op = O.OraclePool(NB, BS, SEED)
            assert op.offload(acc, D0) == O.OK
            op.restore(acc)
            out = op.check(from_claims([(7, blocks, pres)]), D0)[0]
            diff = first_block_difference(tk, pres)
            npres = -(-pres.size // BS)
            shape = min(n, npres) if npres != n else None
            cands = [x for x in (diff, shape) if x is not None]
            if not cands:
                assert out["code"] == O.MATERIALIZED and out["reasons"] == 0
                assert out["intact_blocks"] == n
                continue
            want = min(cands)
            assert out["code"] == O.UNKNOWN, (trial, tk.size, pres.size)
            assert out["first_failing_block"] == want, (trial, tk.size, pres.size, diff, shape)
            assert bool(out["reasons"] & O.R_TOKEN_MISMATCH) == (diff is not None)
            assert out["intact_blocks"] == min(want, n)


def registered_prefixes(claims, holders=None):
    """prefix (tuple of token blocks 0..j) -> set of physical blocks at j,
    over the offloaded claims, by direct comparison.  With ``holders`` (a
    dict), also record the prefix each physical block holds: that of its
    latest registration, in offload order (claims in order, positions in
    order)."""
    reg = {}
    for _, blks, tk in claims:
        tb = blocks_of(tk)
        for j in range(len(blks)):
            reg.setdefault(tuple(tb[: j + 1]), set()).add(int(blks[j]))
            if holders is not None:
                holders[int(blks[j])] = tuple(tb[: j + 1])
    return reg


def brute_lookup(reg, tk, holders=None):
    """Leading token blocks whose prefix is registered to exactly one block
    that (with ``holders``) still holds that prefix; a prefix registered to
    two blocks stops the walk as ambiguous."""
    tb = blocks_of(tk)
    hit = 0
    while hit < len(tb):
        prefix = tuple(tb[: hit + 1])
        owners = reg.get(prefix)
        if owners is None:
            return hit, None, False
        if len(owners) > 1:
            return hit, None, True
        if holders is not None and holders[next(iter(owners))] != prefix:
            return hit, None, False  # the block was registered since under another prefix
        hit += 1
    return hit, None, False


def make_family_claims():
    """Claims with shared prefixes (same tokens and blocks, as a prefix cache
    stores them), one duplicate owner (same tokens, another block) and
    unrelated claims."""
    root = rand_tokens(6 * BS + 2)
    claims = [(100, list(range(0, 7)), root)]
    # shares 3 full blocks with the root, then its own blocks
    t1 = np.concatenate([root[: 3 * BS], rand_tokens(2 * BS)])
    claims.append((101, [0, 1, 2, 10, 11], t1))
    # shares 2 blocks, then repeats the root's third block's tokens in another
    # physical block: duplicate ownership of the 3-block prefix
    t2 = np.concatenate([root[: 3 * BS], rand_tokens(BS)])
    claims.append((102, [0, 1, 20, 21], t2))
    # identical copy of the first claim's first 4 blocks (dedup)
    claims.append((103, [0, 1, 2, 3], root[: 4 * BS].copy()))
    for k in range(4):
        t = rand_tokens(int(RNG.integers(1, 5 * BS)))
        claims.append((200 + k, list(range(30 + 6 * k, 30 + 6 * k + -(-t.size // BS))), t))
    return claims


def test_lookup_matches_prefix_brute_force():
    claims = make_family_claims()
    op = O.OraclePool(NB, BS, SEED)
    assert op.offload(from_claims(claims), D0) == O.OK
    holders = {}
    reg = registered_prefixes(claims, holders)
    entries, ambiguous = op.identity_stats()
    assert entries == len(reg)
    assert ambiguous == sum(1 for v in reg.values() if len(v) > 1) == 1

    reqs = []
    for _, _, tk in claims:
        reqs.extend(variants(tk))
    reqs.append(rand_tokens(3 * BS))
    reqs.append(np.zeros(0, np.uint32))
    batch = from_claims([(1000 + i, [], t) for i, t in enumerate(reqs)])
    got = op.lookup(batch)
    for i, t in enumerate(reqs):
        hit, _, amb = brute_lookup(reg, t, holders)
        r = got[i]
        assert r["request_id"] == 1000 + i
        assert r["hit_blocks"] == hit, (i, t.size)
        assert r["hit_tokens"] == min(hit * BS, t.size)
        nt = -(-t.size // BS)
        if amb:
            want = O.LK_UNKNOWN
        elif hit == nt and hit > 0:
            want = O.LK_HIT
        elif hit == 0:
            want = O.LK_MISS
        else:
            want = O.LK_PARTIAL
        assert r["status"] == want, (i, hit, nt, amb)
        if hit:
            owners = reg[tuple(blocks_of(t)[:hit])]
            assert r["last_block"] == next(iter(owners))
            assert r["chain_hash_at_hit"] == O.chain(t, BS, SEED)[hit - 1]
        else:
            assert r["last_block"] == O.NONE32 and r["chain_hash_at_hit"] == SEED
    # the lookup changes nothing: a second lookup gives the same, no events
    assert np.array_equal(op.lookup(batch), got)


def test_ambiguous_identity_fails_the_lookup_closed():
    """The 3-block prefix shared by claims 100 and 102 sits in two different
    physical blocks: a request through it is UNKNOWN with 2 hit blocks,
    never a 3-block (or longer) hit."""
    claims = make_family_claims()
    op = O.OraclePool(NB, BS, SEED)
    op.offload(from_claims(claims), D0)
    root = claims[0][2]
    r = op.lookup(from_claims([(1, [], root)]))[0]
    assert (r["status"], r["hit_blocks"]) == (O.LK_UNKNOWN, 2)
    # a prefix that stops before the ambiguous block is a plain hit
    r = op.lookup(from_claims([(2, [], root[: 2 * BS])]))[0]
    assert (r["status"], r["hit_blocks"], r["last_block"]) == (O.LK_HIT, 2, 1)


def test_lookup_ignores_claims_that_were_not_offloaded():
    """A claim with a missing block-table entry is accepted but never
    offloaded: none of its identities are registered."""
    tk = rand_tokens(3 * BS)
    op = O.OraclePool(NB, BS, SEED)
    op.offload(from_claims([(9, [1, 0xFFFFFFFF, 2], tk)]), D0)
    assert op.identity_stats() == (0, 0)
    assert op.lookup(from_claims([(9, [], tk)]))[0]["status"] == O.LK_MISS


def test_malformed_lookup_rows_are_unknown():
    b = from_claims([(1, [], rand_tokens(5)), (0xFFFFFFFFFFFFFFFF, [], rand_tokens(5)),
                     (3, [], rand_tokens(2))])
    b.token_offsets[3] = b.tokens.size + 7  # row 2 runs past the token array
    op = O.OraclePool(NB, BS, SEED)
    got = op.lookup(b)
    assert got["status"].tolist() == [O.LK_MISS, O.LK_UNKNOWN, O.LK_UNKNOWN]
    b.token_offsets[3] = b.token_offsets[2]
    b.token_offsets[2] = b.token_offsets[1] - 1  # row 1 now runs backwards
    assert op.lookup(b)["status"][1] == O.LK_UNKNOWN


def test_reuse_lookup_of_the_running_example_hits_448_tokens():
    """Section 7 paths A and B: the reuse lookup of the offloaded 448-token
    claim reports hit = 448 (28 blocks of 16 tokens)."""
    rows = {r[0]: int(r[1]) for r in golden_lines("paper_event_paths.txt") if r[1].isdigit()}
    k, bs = rows["LOOKUP_HIT_TOKENS"], rows["PREDICATE_BLOCK_SIZE"]
    tk = RNG.integers(1, 32000, size=k, dtype=np.uint32)
    op = O.OraclePool(NB, bs, SEED)
    c = from_claims([(0x448, list(range(k // bs)), tk)])
    op.offload(c, D0)
    r = op.lookup(c)[0]
    assert (r["status"], r["hit_tokens"], r["hit_blocks"]) == (O.LK_HIT, 448, 28)
    # a reuse request that continues the conversation still hits the 448
    longer = np.concatenate([tk, RNG.integers(1, 32000, size=37, dtype=np.uint32)])
    r = op.lookup(from_claims([(0x449, [], longer)]))[0]
    assert (r["status"], r["hit_tokens"]) == (O.LK_PARTIAL, 448)


def test_reassigned_block_no_longer_hits_its_old_identity():
    """Claim 1 offloads block 5 holding prefix P; claim 2 then offloads block
    5 holding prefix Q.  Block 5 no longer holds P: a lookup of P must not
    report a hit on it (section 7 E1 reports what is resident; Table 2, an
    ambiguous or stale mapping must not be served), while Q hits.  A third
    claim storing P in block 5 again makes P hit and Q stale."""
    p_tok, q_tok = rand_tokens(BS), rand_tokens(BS)
    op = O.OraclePool(NB, BS, SEED)
    assert op.offload(from_claims([(1, [5], p_tok)]), D0) == O.OK
    r = op.lookup(from_claims([(10, [], p_tok)]))[0]
    assert (r["status"], r["hit_blocks"], r["last_block"]) == (O.LK_HIT, 1, 5)
    assert op.offload(from_claims([(2, [5], q_tok)]), D0) == O.OK
    assert op.identity_stats() == (2, 0)
    got = op.lookup(from_claims([(10, [], p_tok), (11, [], q_tok)]))
    assert (got[0]["status"], got[0]["hit_blocks"], got[0]["last_block"]) == (O.LK_MISS, 0, O.NONE32)
    assert (got[1]["status"], got[1]["hit_blocks"], got[1]["last_block"]) == (O.LK_HIT, 1, 5)
    # the same within one batch: the later row holds the block
    op2 = O.OraclePool(NB, BS, SEED)
    op2.offload(from_claims([(1, [5], p_tok), (2, [5], q_tok)]), D0)
    got = op2.lookup(from_claims([(10, [], p_tok), (11, [], q_tok)]))
    assert got["status"].tolist() == [O.LK_MISS, O.LK_HIT]
    # P stored in block 5 again
    assert op.offload(from_claims([(3, [5], p_tok.copy())]), D0) == O.OK
    got = op.lookup(from_claims([(10, [], p_tok), (11, [], q_tok)]))
    assert got["status"].tolist() == [O.LK_HIT, O.LK_MISS]
    # a longer prefix through a reassigned block stops there
    tk = rand_tokens(3 * BS)
    op3 = O.OraclePool(NB, BS, SEED)
    op3.offload(from_claims([(1, [0, 1, 2], tk)]), D0)
    op3.offload(from_claims([(2, [1], rand_tokens(BS))]), D0)
    r = op3.lookup(from_claims([(10, [], tk)]))[0]
    assert (r["status"], r["hit_blocks"], r["last_block"]) == (O.LK_PARTIAL, 1, 0)


@pytest.mark.parametrize("seed", range(8))
def test_lookup_with_block_reuse_matches_brute_force(seed):
    """Claims drawn over only a few physical blocks, so that blocks are
    registered under many prefixes, offloaded in one to three batches; every
    lookup equals the brute-force walk over token-prefix tuples with block
    holders (the latest registration of each block)."""
    rng = np.random.default_rng(500 + seed)
    nphys = 6
    roots = [rand_tokens(int(rng.integers(1, 6 * BS))) for _ in range(3)]
    claims = []
    for k in range(14):
        root = roots[int(rng.integers(len(roots)))]
        cut = int(rng.integers(0, root.size + 1))
        tk = np.concatenate([root[:cut], rand_tokens(int(rng.integers(0, 3 * BS)))])
        if tk.size == 0:
            tk = rand_tokens(1)
        n = -(-tk.size // BS)
        claims.append((300 + k, [int(x) for x in rng.integers(0, nphys, size=n)], tk))
    cuts = sorted(rng.choice(np.arange(1, len(claims)), size=int(rng.integers(0, 3)), replace=False))
    op = O.OraclePool(NB, BS, SEED)
    start = 0
    for end in list(cuts) + [len(claims)]:
        assert op.offload(from_claims(claims[start:end]), D0) == O.OK
        start = end
    holders = {}
    reg = registered_prefixes(claims, holders)
    assert op.identity_stats() == (len(reg), sum(1 for v in reg.values() if len(v) > 1))
    reqs = []
    for _, _, tk in claims:
        reqs.extend(variants(tk))
    got = op.lookup(from_claims([(1000 + i, [], t) for i, t in enumerate(reqs)]))
    stale_stops = 0
    for i, t in enumerate(reqs):
        hit, _, amb = brute_lookup(reg, t, holders)
        r = got[i]
        assert (int(r["hit_blocks"]), r["status"] == O.LK_UNKNOWN) == (hit, amb), (seed, i)
        nt = -(-t.size // BS)
        if not amb:
            want = O.LK_HIT if hit == nt and hit > 0 else O.LK_MISS if hit == 0 else O.LK_PARTIAL
            assert r["status"] == want
        if hit:
            assert r["last_block"] == next(iter(reg[tuple(blocks_of(t)[:hit])]))
        plain_hit, _, plain_amb = brute_lookup(reg, t)
        stale_stops += int(plain_hit > hit and not amb)
    assert stale_stops > 0  # block reuse did stop some walks
