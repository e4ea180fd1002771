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
from paper_2606_01387_amd.synth import (FULL, TINY, FaultSpec, Geometry, Workload, from_claims,
                                        make_batch, make_faults, make_requests, scaled)
from tests.helpers import apply_flips, digests
from tests.test_gpu_parity import (LONG_CLAIMS, MAX_BS_LONG, MAX_BS_SHORT, MIN_BS, capacities,
                                   free_gpu, gpu_pool_tensor, note, same_events, same_outcomes)

pytestmark = pytest.mark.gpu

LK_FIELDS = [n for n in O.LOOKUP_DTYPE.names if n != "pad"]


def same_lookups(got, want):
    assert len(got) == len(want)
    for f in LK_FIELDS:
        if not np.array_equal(got[f], want[f]):
            bad = np.flatnonzero(got[f] != want[f])[:5]
            raise AssertionError(f"lookup field {f} differs at rows {bad.tolist()}: "
                                 f"gpu {got[f][bad].tolist()} oracle {want[f][bad].tolist()}")


def unaliased(w: Workload) -> Workload:
    """The workload's claims over a pool of tiny blocks large enough that
    the generator never gives two unrelated claims one physical block.  The
    benchmark workloads reference several times more blocks than their pools
    hold, so unrelated prefixes share blocks and each block holds only its
    latest registration's identity (most identities go stale); with distinct
    blocks the lookups reach hits, partial hits and misses.  A lookup reads
    no KV bytes, so 16-byte rows per token keep the pool small."""
    g = w.geometry
    refs = make_batch(w).num_refs
    geo = Geometry(1, 1, g.block_size, 1, 8, 2, 2 * refs + 64)
    return replace(w, name=w.name + "-unaliased", geometry=geo)


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
LOOKUP_CASES += [unaliased(w) for w in LOOKUP_CASES[1:]]


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
    if w.name.endswith("-unaliased") or w is TINY:
        assert st[ck.LOOKUP_HIT] and st[ck.LOOKUP_PARTIAL] and st[ck.LOOKUP_MISS]
    else:
        assert st[ck.LOOKUP_MISS]  # aliased blocks: stale identities stop lookups
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


def _positioned_cases(W: int, bs: int, rng):
    """Claims of 2W + W/2 + 3 blocks (several windows of a W-wide group)
    whose presented tokens differ from the accepted ones at chosen block
    positions: window edges, the last block, two places, cuts, extensions,
    an accepted claim shorter than its rows, and digest faults, reported
    failures or missing entries before or after the first identity
    mismatch.  Returns (accepted parts, presented parts, flips (position),
    load failures (position)) per claim, plus filler claims that bring the
    mean row length to W."""
    n = 2 * W + W // 2 + 3
    r = 5  # the accepted claims end 5 tokens short of their last block

    def toks(k):
        return rng.integers(1, 32000, size=k, dtype=np.uint32)

    def chg(t, blocks):
        t = t.copy()
        for j in blocks:
            m = j * bs + int(rng.integers(0, bs if (j + 1) * bs <= t.size else t.size - j * bs))
            t[m] = (int(t[m]) + 1 + int(rng.integers(0, 31998))) % 32000
        return t

    specs = [  # (name, presented(t), flip positions, load-failed positions, missing positions, accepted cut)
        ("same", lambda t: t, [], [], [], None),
        ("chg@0", lambda t: chg(t, [0]), [], [], [], None),
        ("chg@W-1", lambda t: chg(t, [W - 1]), [], [], [], None),
        ("chg@W", lambda t: chg(t, [W]), [], [], [], None),
        ("chg@last", lambda t: chg(t, [n - 1]), [], [], [], None),
        ("chg@2,n-2", lambda t: chg(t, [2, n - 2]), [], [], [], None),
        ("cut@W", lambda t: t[: W * bs], [], [], [], None),
        ("cut@W+7tok", lambda t: t[: W * bs + 7], [], [], [], None),
        ("cut@0", lambda t: t[:0], [], [], [], None),
        ("ext+3", lambda t: np.concatenate([t, toks(3)]), [], [], [], None),
        ("ext+bs+5", lambda t: np.concatenate([t, toks(bs + 5)]), [], [], [], None),
        ("acc-short", lambda t: t, [], [], [], (W + 1) * bs),
        ("flip@1,chg@W+1", lambda t: chg(t, [W + 1]), [1], [], [], None),
        ("flip@n-3", lambda t: t, [n - 3], [], [], None),
        ("acc-short,flip@W+2", lambda t: t, [W + 2], [], [], W * bs),
        ("lf@1,ext", lambda t: np.concatenate([t, toks(2 * bs)]), [], [1], [], None),
        ("miss@1,chg@W+2", lambda t: chg(t, [W + 2]), [], [], [1], None),
        ("chg@W+3,flip@W+5", lambda t: chg(t, [W + 3]), [W + 5], [], [], None),
    ]
    cases = []
    for name, pres, flips, lfs, miss, acc_cut in specs:
        full = toks(n * bs - r)
        acc = full if acc_cut is None else full[:acc_cut]
        cases.append((name, n, acc, pres(full), flips, lfs, miss))
    # fillers: 1-block claims that bring the mean row length into (W/2, W]
    refs = len(cases) * n
    k = 0
    while -(-(refs + k) // (len(cases) + k)) > W:
        k += 1
    fill = [toks(bs - 3) for _ in range(k)]
    return cases, fill


@pytest.mark.parametrize("W", [4, 16, 64])
def test_identity_positions(torch, ck, W):
    """Per-position identity at chosen positions, against the oracle: the
    parallel compare's first mismatch, the values it takes from the
    accepted chain below it, and the serial chain from the first mismatch
    (or from the end of a shorter accepted claim) on."""
    g = Geometry(1, 1, 16, 1, 8, 2, 4096)  # 256-byte blocks
    bs = g.block_size
    w = Workload(name=f"identity-positions-w{W}", geometry=g, seed=77 + W, num_claims=1,
                 length=("blocks", 1, 1, False), sharing=("fraction", 0.0), corrupt_rate=0.0,
                 content_seed=5 + W)
    rng = np.random.default_rng(400 + W)
    cases, fill = _positioned_cases(W, bs, rng)
    acc_parts, pres_parts, flips, lfs = [], [], [], []
    nxt = 0
    for i, (name, n, acc, pres, fl, lf, miss) in enumerate(cases):
        blks = np.arange(nxt, nxt + n, dtype=np.uint32)
        nxt += n
        pblks = blks.copy()
        pblks[miss] = 0xFFFFFFFF
        acc_parts.append((1000 + i, blks, acc))
        pres_parts.append((1000 + i, pblks, pres))
        flips += [(int(blks[j]), int(rng.integers(0, 8 * g.block_bytes))) for j in fl]
        lfs += [int(blks[j]) for j in lf]
    for i, t in enumerate(fill):
        part = (5000 + i, np.array([nxt], np.uint32), t)
        nxt += 1
        acc_parts.append(part)
        pres_parts.append(part)
    assert nxt <= g.num_blocks
    accepted, presented = from_claims(acc_parts), from_claims(pres_parts)
    mean = -(-presented.num_refs // presented.num_claims)
    assert W // 2 < mean <= W or (W == 4 and mean <= 4)
    faults = FaultSpec(np.array([f[0] for f in flips], np.uint32),
                       np.array([f[1] for f in flips], np.uint64), np.array(lfs, np.uint32))
    note(f"identity positions W={W}: {len(cases)} positioned claims of {cases[0][1]} blocks, "
         f"{len(fill)} fillers")
    kv = gpu_pool_tensor(torch, w)
    with ck.Pool(g, w.seed, kv, **capacities(accepted)) as pool:
        pool.offload(ck.DeviceBatch(accepted))
        pool.restore(ck.DeviceBatch(accepted), faults=faults)
        pool.read(max_outcomes=1)
        pool.check(ck.DeviceBatch(presented))
        out, ev = pool.read()
    host = __import__("paper_2606_01387_amd.synth", fromlist=["content"]).content.pool_host(
        g, w.content_seed)
    op = O.OraclePool(g.num_blocks, bs, w.seed)
    assert op.offload(accepted, digests(host, w)) == O.OK
    assert op.restore(accepted, faults.load_failed) == O.OK
    op.events(clear=True)
    want = op.check(presented, digests(apply_flips(host, w, faults), w))
    for i, case in enumerate(cases):
        note(f"  {case[0]}: code {int(want['code'][i])} block {int(want['first_failing_block'][i])} "
             f"reasons {int(want['reasons'][i]):#x}")
    same_outcomes(out, want)
    same_events(ev, op.events())
    # the cases reach what they are for: a mismatch at the changed block
    names = [c[0] for c in cases]
    ffb = out["first_failing_block"]
    assert ffb[names.index("chg@0")] == 0
    assert ffb[names.index("chg@W")] == W
    assert ffb[names.index("chg@last")] == cases[0][1] - 1
    assert ffb[names.index("flip@1,chg@W+1")] == W + 1
    assert ffb[names.index("miss@1,chg@W+2")] == 1
    assert out["code"][names.index("same")] == ck.MATERIALIZED
    del kv
    free_gpu(torch)


def test_chain_reproduces_published_outputs_on_gpu(torch, ck):
    """The library's chain against values published outside this project:
    on a pool with seed 0 and 16-token blocks, the token blocks of
    tests/golden/chain_splitmix_tokens.txt chain to the four published
    SplitMix64 outputs for seed 0.  Checked in acceptance (ACCEPTED carries
    the chain hash), in the check (outcome chain hash, per-position identity)
    and in the lookup (chain hash at the hit, for every prefix length)."""
    from tests.test_oracle_hash import GOLD, chain_fixture

    note("chain against published SplitMix64 outputs")
    toks = chain_fixture()
    g = Geometry(1, 2, 16, 1, 8, 2, 16)
    kv = torch.zeros(g.pool_bytes, dtype=torch.uint8, device="cuda")
    blocks = [3, 5, 7, 9]
    claim = from_claims([(0x5EED, blocks, toks)])
    changed = toks.copy()
    changed[40] += 1  # a token of block 2
    reqs = from_claims([(0x100 + k, [], toks[: 16 * k]) for k in range(1, 5)])
    with ck.Pool(g, 0, kv, max_claims=64, max_footprint=256, event_capacity=256) as pool:
        db = ck.DeviceBatch(claim)
        pool.offload(db)
        _, ev_acc = pool.read(max_outcomes=1)
        pool.restore(db)
        pool.check(db)
        out, _ = pool.read()
        lk = pool.lookup(ck.DeviceBatch(reqs))
        pool.check(ck.DeviceBatch(from_claims([(0x5EED, blocks, changed)])))
        out_changed, _ = pool.read()
    acc = ev_acc[ev_acc["kind"] == ck.EV_ACCEPTED]
    assert acc["aux"].tolist() == [GOLD[3]]
    assert out["code"].tolist() == [ck.MATERIALIZED]
    assert int(out[0]["chain_hash"]) == GOLD[3]
    assert lk["hit_blocks"].tolist() == [1, 2, 3, 4]
    assert lk["last_block"].tolist() == blocks
    assert lk["chain_hash_at_hit"].tolist() == GOLD
    # identities h_0, h_1 still match; block 2 is the first that differs
    assert out_changed["code"].tolist() == [ck.UNKNOWN]
    assert int(out_changed[0]["first_failing_block"]) == 2
    assert int(out_changed[0]["reasons"]) & ck.R_TOKEN_MISMATCH
    del kv
    free_gpu(torch)


def test_same_batch_duplicate_ownership(torch, ck):
    """Registrants of one identity racing inside one offload batch: pairs of
    claims with the same tokens, half of them with a different first block
    (duplicate ownership of h_0, so h_0 is ambiguous; their later identities
    have the same blocks and stay plain), half with identical blocks (stored
    once).  The GPU registers concurrently, the oracle in batch order; the
    identity counts and every lookup must agree."""
    note("same-batch duplicate ownership")
    w = TINY
    g = w.geometry
    bs = g.block_size
    rng = np.random.default_rng(17)
    parts, reqs = [], []
    for i in range(100):
        nblk = int(rng.integers(2, 5))
        t = rng.integers(1, 32000, size=nblk * bs - int(rng.integers(0, bs)), dtype=np.uint32)
        blocks = [int(x) for x in rng.integers(0, g.num_blocks, size=nblk)]
        other = list(blocks)
        if i % 2 == 0:
            other[0] = (blocks[0] + 1 + int(rng.integers(0, g.num_blocks - 1))) % g.num_blocks
        parts += [(1000 + 2 * i, blocks, t), (1001 + 2 * i, other, t.copy())]
        reqs += [t, t[: bs], np.concatenate([t, rng.integers(1, 32000, size=bs, dtype=np.uint32)])]
    order = rng.permutation(len(parts))
    batch = from_claims([parts[k] for k in order])
    rb = from_claims([(5000 + i, [], r) for i, r in enumerate(reqs)])
    kv = gpu_pool_tensor(torch, w)
    op = O.OraclePool(g.num_blocks, bs, w.seed)
    zero = np.zeros(g.num_blocks, np.uint64)
    with ck.Pool(g, w.seed, kv, max_claims=512, max_footprint=2048, event_capacity=2048) as pool:
        pool.offload(ck.DeviceBatch(batch))
        assert op.offload(batch, zero) == O.OK
        stats = pool.identity_stats()
        got = pool.lookup(ck.DeviceBatch(rb))
    assert stats == op.identity_stats()
    assert stats[1] == 50  # h_0 of every pair with a different first block
    same_lookups(got, op.lookup(rb))
    assert (got["status"] == ck.LOOKUP_UNKNOWN).sum() >= 100
    del kv
    free_gpu(torch)


@pytest.mark.parametrize("batches", [1, 3])
def test_lookup_source_switching(torch, ck, batches):
    """Long requests (wide groups) that leave one accepted claim's identities
    for another's: a tree of claims that share prefixes of different lengths
    (offloaded in one batch, or in three), and requests that follow one
    branch, switch branches at a divergence, run past a shorter claim's end
    onto a longer one, or leave every claim.  Every lookup field against the
    oracle."""
    note(f"lookup source switching, {batches} offload batches")
    w = replace(TINY, geometry=replace(TINY.geometry, num_blocks=1024))
    g = w.geometry
    bs = g.block_size
    rng = np.random.default_rng(23 + batches)

    def toks(nblk):
        return rng.integers(1, 32000, size=nblk * bs, dtype=np.uint32)

    root = toks(90)
    branches = [root]
    for cut in (7, 20, 33, 64, 80):  # branches diverging from earlier ones at block `cut`
        base = branches[int(rng.integers(0, len(branches)))]
        cut = min(cut, base.size // bs - 1)
        branches.append(np.concatenate([base[: cut * bs], toks(int(rng.integers(10, 70)))]))
    short = root[: 30 * bs].copy()  # a shorter claim inside the root
    claims = branches + [short]
    parts = []
    perm = iter(rng.permutation(g.num_blocks).tolist())  # distinct blocks: none goes stale
    for i, t in enumerate(claims):
        nblk = t.size // bs
        parts.append((700 + i, [next(perm) for _ in range(nblk)], t))
    # shared prefixes keep the same physical blocks as the claim they copy
    by_tokens = {}
    for k, (cid, blks, t) in enumerate(parts):
        for j in range(len(blks)):
            key = t[: (j + 1) * bs].tobytes()
            if key in by_tokens:
                blks[j] = by_tokens[key]
            else:
                by_tokens[key] = blks[j]
    reqs = []
    for t in claims:
        reqs.append(t)
        reqs.append(np.concatenate([t, toks(3)]))
        cut = int(rng.integers(1, t.size))
        reqs.append(t[:cut])
        changed = t.copy()
        changed[int(rng.integers(0, t.size))] += 1
        reqs.append(changed)
    # follow the short claim, then continue along the root past its end
    reqs.append(root[: 60 * bs])
    rb = from_claims([(9000 + i, [], r) for i, r in enumerate(reqs)])
    assert rb.num_tokens // rb.num_claims >= 16 * bs  # wide lookup groups
    groups = np.array_split(rng.permutation(len(parts)), batches)
    kv = gpu_pool_tensor(torch, w)
    op = O.OraclePool(g.num_blocks, bs, w.seed)
    zero = np.zeros(g.num_blocks, np.uint64)
    with ck.Pool(g, w.seed, kv, max_claims=64, max_footprint=4096, event_capacity=512) as pool:
        for grp in groups:
            bt = from_claims([parts[k] for k in grp])
            pool.offload(ck.DeviceBatch(bt))
            assert op.offload(bt, zero) == O.OK
        got = pool.lookup(ck.DeviceBatch(rb))
        stats = pool.identity_stats()
    want = op.lookup(rb)
    same_lookups(got, want)
    assert stats == op.identity_stats()
    assert (got["status"] == ck.LOOKUP_HIT).sum() >= len(claims)
    del kv
    free_gpu(torch)


@pytest.mark.parametrize("zero_at,nblocks", [(1, 3), (20, 40)])
def test_identity_zero(torch, ck, zero_at, nblocks):
    """A claim whose chain reaches the identity 0 at a chosen block (that
    block's tokens solved on the lattice of the token keys, so that
    h_{j-1} xor M_j = -gamma and h_j = mix64(0) = 0).  The library keeps that
    identity in a table entry of its own; registration (new, then present),
    lookups that hit, follow and stop at it (narrow and wide groups),
    ambiguity from a second block and the check, against the oracle."""
    from tests.chain_tokens import solve_block

    note(f"identity 0 at block {zero_at} of {nblocks}")
    m64, gamma = (1 << 64) - 1, 0x9E3779B97F4A7C15
    w = TINY
    g, seed, bs = w.geometry, w.seed, w.geometry.block_size
    rng = np.random.default_rng(5000 + zero_at)
    prefix = rng.integers(0, 32000, size=zero_at * bs, dtype=np.uint32)
    h_prev = int(O.chain(prefix, bs, seed)[-1])
    keys = [O.token_key(seed, k) for k in range(bs)]
    zb = np.array(solve_block(h_prev ^ (-gamma & m64), keys, rng), np.uint32)
    rest = rng.integers(0, 32000, size=(nblocks - zero_at - 1) * bs, dtype=np.uint32)
    toks = np.concatenate([prefix, zb, rest])
    assert int(O.chain(toks, bs, seed)[zero_at]) == 0
    blocks = [int(b) for b in rng.permutation(g.num_blocks)[:nblocks]]
    upto = (zero_at + 1) * bs
    first = from_claims([(0x51, blocks, toks), (0x52, blocks[: zero_at + 1], toks[:upto])])
    other = toks.copy()
    other[upto + 3] ^= 1  # a token of the block after the identity 0
    at_zero = toks.copy()
    at_zero[upto - 2] ^= 1  # a token of the identity-0 block
    reqs = from_claims([(0x101, [], toks), (0x102, [], toks[:upto]), (0x103, [], toks[: upto - 5]),
                        (0x104, [], other), (0x105, [], at_zero), (0x106, [], toks[upto:])])
    second = from_claims([(0x53, [(b + 1) % g.num_blocks for b in blocks[: zero_at + 1]],
                           toks[:upto])])
    kv = gpu_pool_tensor(torch, w)
    host = __import__("paper_2606_01387_amd.synth", fromlist=["content"]).content.pool_host(
        g, w.content_seed)
    op = O.OraclePool(g.num_blocks, bs, seed)
    with ck.Pool(g, seed, kv, max_claims=64, max_footprint=1024, event_capacity=1024) as pool:
        pool.offload(ck.DeviceBatch(first))
        assert op.offload(first, digests(host, w)) == O.OK
        assert pool.identity_stats() == op.identity_stats() == (nblocks, 0)
        got = pool.lookup(ck.DeviceBatch(reqs))
        same_lookups(got, op.lookup(reqs))
        assert got["status"][0] == ck.LOOKUP_HIT and int(got["chain_hash_at_hit"][1]) == 0
        pool.restore(ck.DeviceBatch(first))
        assert op.restore(first) == O.OK
        pool.read(max_outcomes=1)
        op.events(clear=True)
        pool.check(ck.DeviceBatch(first))
        out, ev = pool.read()
        same_outcomes(out, op.check(first, digests(host, w)))
        same_events(ev, op.events(clear=True))
        assert out["code"].tolist() == [ck.MATERIALIZED] * 2
        # the identity 0 (and the prefix before it) registered to other blocks
        pool.offload(ck.DeviceBatch(second))
        assert op.offload(second, digests(host, w)) == O.OK
        assert pool.identity_stats() == op.identity_stats() == (nblocks, zero_at + 1)
        got = pool.lookup(ck.DeviceBatch(reqs))
        same_lookups(got, op.lookup(reqs))
        assert got["status"][0] == ck.LOOKUP_UNKNOWN
    del kv
    free_gpu(torch)
