"""The seeded input generator: Philox known answers, content statistics and
the structure of the generated claim batches."""

from dataclasses import replace

import numpy as np
import pytest

from paper_2606_01387_amd.synth import FULL, MISSING, TINY, FaultSpec, content, make_batch, make_faults, scaled
from tests.conftest import golden_lines


def test_philox_known_answers():
    for row in golden_lines("philox4x32_10_kat.txt"):
        v = [int(x, 16) for x in row]
        assert content.philox4x32_10(v[0:4], v[4:6]) == v[6:10]


def test_bf16_content_is_standard_normal_like():
    g = TINY.geometry
    pool = content.pool_host(g, TINY.content_seed).view("<u2")
    f = (pool.astype(np.uint32) << 16).view(np.float32)
    assert abs(f.mean()) < 0.01 and abs(f.var() - 1.0) < 0.02
    assert np.abs(f).max() <= 3.0


def test_fp8_content_is_uniform_bytes():
    g = scaled(FULL["mla-fp8"], 4, 4).geometry
    pool = content.pool_host(g, 5)
    hist = np.bincount(pool, minlength=256)
    assert hist.min() > 0.8 * pool.size / 256 and hist.max() < 1.2 * pool.size / 256


def test_canonical_block_matches_pool_layout():
    g = TINY.geometry
    pool = content.pool_host(g, TINY.content_seed)
    for b in (0, 17, 63):
        canon = content.block_canonical(g, TINY.content_seed, b)
        for p in range(g.planes):
            off = (p * g.num_blocks + b) * g.chunk_bytes
            assert np.array_equal(canon[p * g.chunk_bytes:(p + 1) * g.chunk_bytes],
                                  pool[off:off + g.chunk_bytes])


@pytest.mark.parametrize("name", ["tiny", "llama3-8b", "mla-fp8"])
def test_batch_structure(name):
    w = FULL[name]
    b = make_batch(w)
    g = w.geometry
    assert np.array_equal(b.claim_ids, make_batch(w).claim_ids)  # deterministic
    assert np.unique(b.claim_ids).size == b.num_claims
    n = np.diff(b.block_offsets.astype(np.int64))
    t = np.diff(b.token_offsets.astype(np.int64))
    assert (n >= 1).all() and np.array_equal(n, (t + g.block_size - 1) // g.block_size)
    ok = b.block_ids[b.block_ids != MISSING]
    assert (ok < g.num_blocks).all()
    # over-subscribed: every pool block is referenced
    assert b.unique_blocks(g.num_blocks).size == g.num_blocks


def test_prefix_sharing_copies_tokens_and_blocks():
    w = FULL["llama3-8b"]
    b = make_batch(w)
    bs = w.geometry.block_size
    seen = {}
    shared = 0
    for c in range(b.num_claims):
        _, blks, toks = b.claim(c)
        key = tuple(toks[:bs])
        if key in seen:
            _, blks0, toks0 = b.claim(seen[key])
            k = 0
            while (k + 1) * bs <= min(len(toks), len(toks0)) and np.array_equal(
                    toks[k * bs:(k + 1) * bs], toks0[k * bs:(k + 1) * bs]):
                k += 1
            assert np.array_equal(blks[:k], blks0[:k])
            shared += 1
        else:
            seen[key] = c
    assert shared > 50


def test_missing_entries_and_faults():
    w = scaled(FULL["llama3-70b"], 2000, 400)
    b = make_batch(w)
    assert (b.block_ids == MISSING).sum() == round(0.02 * 400)
    f = make_faults(w, b)
    assert f.flip_blocks.size == round(0.001 * 2000)
    assert np.unique(f.flip_blocks).size == f.flip_blocks.size
    assert (f.flip_bits < 8 * w.geometry.block_bytes).all()


def test_changed_blocks_cancels_repeated_flips():
    f = FaultSpec(np.array([3, 3, 5, 7, 7], np.uint32), np.array([10, 10, 1, 2, 3], np.uint64),
                  np.zeros(0, np.uint32))
    assert f.changed_blocks().tolist() == [5, 7]


def test_predicates_cover_a_leading_prefix():
    """With a predicate fraction, the selected claims get k in [1, T_c]
    tokens and the rest exactly T_c; without one, no predicate array."""
    assert make_batch(TINY).predicate_tokens is None
    w = replace(TINY, num_claims=400, predicate_fraction=0.5)
    b = make_batch(w)
    T = np.diff(b.token_offsets.astype(np.int64))
    k = b.predicate_tokens.astype(np.int64)
    assert k.shape == T.shape and (k >= 1).all() and (k <= T).all()
    assert 0.3 < np.mean(k < T) < 0.6
    again = make_batch(w)
    assert np.array_equal(again.predicate_tokens, b.predicate_tokens)
    sub = b.subset([5, 2])
    assert sub.predicate_tokens.tolist() == [b.predicate_tokens[5], b.predicate_tokens[2]]


def test_requests_follow_their_kinds():
    """Lookup requests: same / cut / changed / extended copies of claim
    token rows, or fresh rows, with the stated lengths."""
    from paper_2606_01387_amd.synth import make_requests

    w = replace(TINY, num_claims=200)
    b = make_batch(w)
    req, kind = make_requests(w, b, num_requests=500)
    assert req.num_claims == 500 and req.num_refs == 0
    assert np.unique(req.claim_ids).size == 500
    counts = np.bincount(kind, minlength=5)
    assert (counts > 40).all()
    L = np.diff(req.token_offsets.astype(np.int64))
    bs = w.geometry.block_size
    rows = [req.tokens[int(req.token_offsets[i]):int(req.token_offsets[i + 1])] for i in range(500)]
    claims = {tuple(b.claim(c)[2].tolist()) for c in range(b.num_claims)}
    for i, k in enumerate(kind):
        t = tuple(rows[i].tolist())
        if k == 0:
            assert t in claims
        elif k == 1:
            assert any(c[: len(t)] == t for c in claims) and len(t) >= 1
        elif k == 2:
            assert t not in claims or len(t) == 0
        elif k == 3:
            assert any(t[: len(c)] == c and 1 <= len(t) - len(c) <= 2 * bs for c in claims)
    again, kind2 = make_requests(w, b, num_requests=500)
    assert np.array_equal(again.tokens, req.tokens) and np.array_equal(kind, kind2)
