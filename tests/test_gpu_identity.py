"""Cache identity on the GPU against the oracle, element by element: the
identity table built at offload (entries and ambiguous entries), the reuse
lookup (section 7 E1: hit blocks and tokens, status, last block, chain hash
at the hit) and the per-position identity compare of claim_check (Table 2:
cache-identity mismatch and duplicate ownership fail closed)."""

from __future__ import annotations

from dataclasses import replace

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_01387_amd.synth import (FULL, TINY, Geometry, Workload, from_claims, make_batch,
                                        make_faults, make_requests, scaled)
from tests.helpers import apply_flips, digests
from tests.test_gpu_parity import (LONG_CLAIMS, MAX_BS_LONG, MAX_BS_SHORT, MIN_BS, capacities,
                                   free_gpu, gpu_pool_tensor, note, same_events, same_outcomes)

pytestmark = pytest.mark.gpu

LK_FIELDS = [n for n in O.LOOKUP_DTYPE.names if n != "pad"]


@pytest.fixture(scope="module")
def torch():
    import torch as t

    assert t.cuda.is_available(), "GPU tests need a GPU"
    return t


@pytest.fixture(scope="module")
def ck():
    from paper_2606_01387_amd import claimkv

    claimkv.lib()
    return claimkv


def same_lookups(got, want):
    assert len(got) == len(want)
    for f in LK_FIELDS:
        if not np.array_equal(got[f], want[f]):
            bad = np.flatnonzero(got[f] != want[f])[:5]
            raise AssertionError(f"lookup field {f} differs at rows {bad.tolist()}: "
                                 f"gpu {got[f][bad].tolist()} oracle {want[f][bad].tolist()}")


LOOKUP_CASES = [
    TINY,
    scaled(FULL["llama3-8b"], 48, 60),
    scaled(FULL["llama3-70b"], 24, 40, missing_claim_rate=0.1),
    scaled(FULL["small-claim-stress"], 256, 30000),
    scaled(FULL["mla-fp8"], 40, 60),
    LONG_CLAIMS,
    MAX_BS_SHORT,
    MAX_BS_LONG,
    MIN_BS,
]


@pytest.mark.parametrize("w", LOOKUP_CASES, ids=lambda w: w.name)
def test_lookup_parity(torch, ck, w):
    g = w.geometry
    batch = make_batch(w)
    reqs, kind = make_requests(w, batch, num_requests=max(2 * batch.num_claims, 64))
    note(f"lookup parity {w.name}: {batch.num_claims} claims, {reqs.num_claims} requests, "
         f"{reqs.num_tokens} request tokens")
    kv = torch.zeros(g.pool_bytes, dtype=torch.uint8, device="cuda")
    with ck.Pool(g, w.seed, kv, **capacities(batch)) as pool:
        pool.offload(ck.DeviceBatch(batch))
        got = pool.lookup(ck.DeviceBatch(reqs))
        stats = pool.identity_stats()
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    assert op.offload(batch, np.zeros(g.num_blocks, np.uint64)) == O.OK
    want = op.lookup(reqs)
    same_lookups(got, want)
    assert stats == op.identity_stats()
    st = np.bincount(got["status"], minlength=4)
    note(f"  status unknown/hit/partial/miss = {st.tolist()}, identities {stats}")
    assert st[ck.LOOKUP_HIT] and st[ck.LOOKUP_PARTIAL] and st[ck.LOOKUP_MISS]
    del kv
    free_gpu(torch)


def test_duplicate_ownership_and_edge_rows(torch, ck):
    """Equal registrations stored once, one identity in two blocks, an
    identity registered by a claim in a later offload, a claim that is never
    offloaded, empty and malformed request rows."""
    w = TINY
    g = w.geometry
    bs = g.block_size
    rng = np.random.default_rng(5)

    def toks(n):
        return rng.integers(1, 32000, size=n, dtype=np.uint32)

    root = toks(5 * bs + 3)
    first = from_claims([
        (100, [0, 1, 2, 3, 4, 5], root),
        (101, [0, 1, 2, 9], np.concatenate([root[: 3 * bs], toks(bs)])),    # shares 3 blocks
        (103, [0, 1, 2, 3], root[: 4 * bs].copy()),                           # equal copy
        (104, [7, 0xFFFFFFFF, 8], toks(3 * bs)),                              # never offloaded
    ])
    later = from_claims([
        (102, [0, 1, 20, 21], np.concatenate([root[: 3 * bs], toks(bs)])),   # block 2's identity in 20
        (105, [30, 31], toks(2 * bs)),
    ])
    reqs = [root, root[: 2 * bs], root[: 3 * bs + 1], np.concatenate([root, toks(7)]),
            later.claim(1)[2], first.claim(3)[2], toks(40), np.zeros(0, np.uint32),
            first.claim(1)[2]]
    rb = from_claims([(900 + i, [], t) for i, t in enumerate(reqs)] +
                     [(0xFFFFFFFFFFFFFFFF, [], toks(3)), (950, [], toks(2))])
    rb.token_offsets[-1] = rb.tokens.size + 5  # the last row runs past the tokens

    kv = gpu_pool_tensor(torch, w)
    op = O.OraclePool(g.num_blocks, bs, w.seed)
    zero = np.zeros(g.num_blocks, np.uint64)
    with ck.Pool(g, w.seed, kv, max_claims=64, max_footprint=256, event_capacity=256) as pool:
        pool.offload(ck.DeviceBatch(first))
        op.offload(first, zero)
        same_lookups(pool.lookup(ck.DeviceBatch(rb)), op.lookup(rb))
        assert pool.identity_stats() == op.identity_stats() == (7, 0)
        pool.offload(ck.DeviceBatch(later))
        op.offload(later, zero)
        got = pool.lookup(ck.DeviceBatch(rb))
        same_lookups(got, op.lookup(rb))
        assert pool.identity_stats() == op.identity_stats() == (10, 1)
    assert got["status"][0] == ck.LOOKUP_UNKNOWN and got["hit_blocks"][0] == 2
    assert got["status"][1] == ck.LOOKUP_HIT and got["last_block"][1] == 1
    assert got["status"][-2:].tolist() == [ck.LOOKUP_UNKNOWN, ck.LOOKUP_UNKNOWN]
    del kv
    free_gpu(torch)


def vary_tokens(batch, rng, frac=0.5):
    """The same claims (ids and block rows) presenting other tokens: for a
    fraction of them one token changed, a cut, or an extension."""
    parts = []
    for c in range(batch.num_claims):
        cid, blks, tk = batch.claim(c)
        tk = tk.copy()
        if tk.size and rng.random() < frac:
            k = rng.integers(0, 3)
            if k == 0:
                m = rng.integers(0, tk.size)
                tk[m] = (int(tk[m]) + 1 + int(rng.integers(0, 31999))) % 32000
            elif k == 1:
                tk = tk[: int(rng.integers(0, tk.size))]
            else:
                tk = np.concatenate([tk, rng.integers(0, 32000, size=int(rng.integers(1, 40)),
                                                      dtype=np.uint32)])
        parts.append((cid, blks, tk))
    return from_claims(parts)


ID_CASES = [
    replace(TINY, num_load_failed=1),
    scaled(FULL["llama3-8b"], 48, 60, corrupt_rate=0.1, num_load_failed=2),
    scaled(FULL["small-claim-stress"], 256, 20000, corrupt_rate=0.02),
    LONG_CLAIMS,
]


@pytest.mark.parametrize("w", ID_CASES, ids=lambda w: w.name)
def test_identity_check_parity(torch, ck, w):
    """Offload, restore, then check with half of the claims presenting other
    tokens: outcomes (first failing block = the first block whose identity
    differs, unless an earlier problem wins) and events equal the oracle's."""
    g = w.geometry
    batch = make_batch(w)
    faults = make_faults(w, batch)
    pres = vary_tokens(batch, np.random.default_rng(w.gen_seed + 3))
    note(f"identity check {w.name}: {batch.num_claims} claims")
    kv = gpu_pool_tensor(torch, w)
    with ck.Pool(g, w.seed, kv, **capacities(batch)) as pool:
        pool.offload(ck.DeviceBatch(batch))
        pool.restore(ck.DeviceBatch(batch), faults=faults)
        pool.read(max_outcomes=1)
        pool.check(ck.DeviceBatch(pres))
        out, ev = pool.read()
    host = __import__("paper_2606_01387_amd.synth", fromlist=["content"]).content.pool_host(
        g, w.content_seed)
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    assert op.offload(batch, digests(host, w)) == O.OK
    assert op.restore(batch, faults.load_failed) == O.OK
    op.events(clear=True)
    want = op.check(pres, digests(apply_flips(host, w, faults), w))
    same_outcomes(out, want)
    same_events(ev, op.events())
    tm = (out["reasons"] & ck.R_TOKEN_MISMATCH) != 0
    positioned = tm & (out["first_failing_block"] != ck.NONE)
    note(f"  token mismatch in {int(tm.sum())} claims, {int(positioned.sum())} at a block position")
    assert positioned.any()
    del kv
    free_gpu(torch)
