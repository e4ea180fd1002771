"""GPU parity: the HIP library (through its C ABI) against the CPU oracle.

Every comparison is exact: outcomes, events, offload / restored digests and
first-failing-block indices are integers and must match bit for bit.

* scaled workloads (real digests of every block on both sides, several
  digest tiles, ragged chunks and ragged claim tails);
* the paper's lifecycle controls, replayed step by step on both sides;
* the staged offload / restore round trip (device and pinned host staging);
* the full-size workloads in the benchmark's launch configuration: all
  outcomes and events, and the offload and restored digests of every
  referenced block, against real oracle digests of every one of them (their
  bytes generated on the host threads, block by block); and a reuse lookup
  of as many requests as claims, with the identity-table counts.
"""

from __future__ import annotations

import gc
import sys
from dataclasses import replace

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_01387_amd.synth import (FULL, MISSING, SHARDS, TINY, Batch, FaultSpec, Geometry, Workload, content,
                                        from_claims, make_batch, make_faults, make_requests, scaled)
from tests.helpers import apply_flips, digests, real_digests, validate_lifecycle

pytestmark = pytest.mark.gpu

OUT_FIELDS = [n for n in O.OUTCOME_DTYPE.names if n != "pad"]
EV_FIELDS = [n for n in O.EVENT_DTYPE.names if n != "pad"]


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def free_gpu(torch):
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def gpu_pool_tensor(torch, w: Workload):
    g = w.geometry
    kv = torch.empty(g.pool_bytes, dtype=torch.uint8, device="cuda")
    content.fill_pool_gpu(kv.data_ptr(), kv.numel(), g, w.content_seed,
                          torch.cuda.current_stream().cuda_stream)
    return kv


def same_outcomes(got, want):
    assert len(got) == len(want)
    for f in OUT_FIELDS:
        if not np.array_equal(got[f], want[f]):
            bad = np.flatnonzero(got[f] != want[f])[:5]
            raise AssertionError(f"outcome field {f} differs at claims {bad.tolist()}: "
                                 f"gpu {got[f][bad].tolist()} oracle {want[f][bad].tolist()}")


def same_events(got, want):
    assert len(got) == len(want), (len(got), len(want))
    for f in EV_FIELDS:
        if not np.array_equal(got[f], want[f]):
            bad = np.flatnonzero(got[f] != want[f])[:5]
            raise AssertionError(f"event field {f} differs at {bad.tolist()}: "
                                 f"gpu {got[f][bad].tolist()} oracle {want[f][bad].tolist()}")


def capacities(batch):
    return dict(max_claims=max(64, 2 * batch.num_claims), max_footprint=max(256, 4 * batch.num_refs),
                event_capacity=max(256, 8 * batch.num_claims))


# --------------------------------------------------------------- fill parity


@pytest.mark.parametrize("w", [TINY, scaled(FULL["llama3-8b"], 6, 4), scaled(FULL["mla-fp8"], 5, 4)],
                         ids=lambda w: w.name)
def test_gpu_fill_matches_host_generator(torch, w):
    note(f"fill parity {w.name}")
    kv = gpu_pool_tensor(torch, w)
    got = kv.cpu().numpy()
    want = content.pool_host(w.geometry, w.content_seed)
    assert np.array_equal(got, want)


# ------------------------------------------------- scaled workloads, real bytes

RAGGED = Workload(
    name="ragged-chunk", geometry=Geometry(3, 2, 16, 3, 40, 2, 37), seed=77, num_claims=300,
    length=("blocks", 1, 3, True), sharing=("zipf", 1.2, 8), corrupt_rate=0.2, num_load_failed=2,
    gen_seed=11, content_seed=12)  # 3840-byte chunks: not a multiple of 1 KiB
TINY_CHUNK = Workload(
    name="48-byte-chunk", geometry=Geometry(2, 1, 3, 1, 8, 2, 19), seed=5, num_claims=50,
    length=("blocks", 1, 12, True), sharing=("fraction", 0.3), corrupt_rate=0.3, num_load_failed=1,
    gen_seed=3, content_seed=4)
LONG_CLAIMS = Workload(
    name="long-claims", geometry=Geometry(4, 2, 16, 2, 64, 2, 50), seed=99, num_claims=12,
    length=("blocks", 100, 300, True), sharing=("fraction", 0.5), corrupt_rate=0.1,
    missing_claim_rate=0.25, num_load_failed=1, gen_seed=21, content_seed=22)

# block-size extremes: 1024-token blocks (the largest a pool accepts) with
# short claims (narrow groups) and long ones (one claim per wave), and
# 1-token blocks, whose 16-byte chunks are the smallest possible
MAX_BS_SHORT = Workload(
    name="bs1024-short", geometry=Geometry(1, 1, 1024, 1, 8, 2, 12), seed=31, num_claims=40,
    length=("blocks", 1, 3, True), sharing=("fraction", 0.3), corrupt_rate=0.25, num_load_failed=1,
    gen_seed=32, content_seed=33)
MAX_BS_LONG = Workload(
    name="bs1024-long", geometry=Geometry(1, 1, 1024, 1, 8, 2, 12), seed=34, num_claims=6,
    length=("blocks", 40, 70, True), sharing=("fraction", 0.5), corrupt_rate=0.2, num_load_failed=1,
    gen_seed=35, content_seed=36)
MIN_BS = Workload(
    name="bs1-16-byte-chunk", geometry=Geometry(1, 2, 1, 1, 8, 2, 40), seed=37, num_claims=30,
    length=("blocks", 1, 90, True), sharing=("zipf", 1.2, 5), corrupt_rate=0.1, num_load_failed=2,
    gen_seed=38, content_seed=39)

# Many planes with few digest workgroups each: the digest reads its piece
# groups in phases so that the grid stays full.  320 planes of 32 KiB chunks
# in four 8 KiB pieces each (320 piece groups, four phases of 80) and 122
# planes of 36 KiB chunks in three 12 KiB pieces each (92 piece groups, the
# last with two pieces; two phases of 46).
MANY_PLANES = Workload(
    name="320-planes-phased", geometry=Geometry(160, 2, 16, 8, 128, 2, 24), seed=41, num_claims=30,
    length=("blocks", 1, 6, True), sharing=("fraction", 0.3), corrupt_rate=0.15, num_load_failed=1,
    gen_seed=42, content_seed=43)
MANY_PLANES_RAGGED = Workload(
    name="122-planes-phased-short-last-group", geometry=Geometry(122, 1, 64, 1, 576, 1, 10),
    seed=44, num_claims=12, length=("blocks", 1, 4, True), sharing=("fraction", 0.3),
    corrupt_rate=0.2, num_load_failed=1, gen_seed=45, content_seed=46)

# 2^22 blocks (two 16-byte chunks each, a 128 MiB pool) under 100 000
# claims of 1-80 blocks: 3.8 M unique blocks, so the mark array is
# compacted in many passes, each digest workgroup flushes its partials
# many times, and the event scan runs over many tiles.
MANY_BLOCKS = Workload(
    name="4m-blocks", geometry=Geometry(1, 2, 1, 1, 8, 2, 1 << 22), seed=51, num_claims=100_000,
    length=("blocks", 1, 80, True), sharing=("fraction", 0.2), corrupt_rate=0.0005,
    num_load_failed=3, gen_seed=52, content_seed=53)

SCALED = [
    replace(TINY, num_load_failed=1),
    scaled(FULL["llama3-8b"], 48, 60, corrupt_rate=0.1, num_load_failed=2),
    scaled(FULL["llama3-70b"], 24, 40, corrupt_rate=0.1, missing_claim_rate=0.1, num_load_failed=1),
    scaled(FULL["small-claim-stress"], 256, 30000, corrupt_rate=0.02, num_load_failed=3),
    scaled(FULL["mla-fp8"], 40, 60, corrupt_rate=0.1, num_load_failed=1),
    RAGGED,
    TINY_CHUNK,
    LONG_CLAIMS,
    # leading_prefix_at_least(k) predicates on part of the claims: one-claim-
    # per-wave groups, mid-size groups and two-lane groups
    replace(LONG_CLAIMS, name="long-claims-predicate", num_claims=16, predicate_fraction=0.7,
            missing_claim_rate=0.0, corrupt_rate=0.005, num_load_failed=1,
            geometry=replace(LONG_CLAIMS.geometry, num_blocks=400)),
    replace(scaled(FULL["llama3-8b"], 48, 60, corrupt_rate=0.25, num_load_failed=4,
                   predicate_fraction=0.6), name="llama3-8b-predicate"),
    replace(scaled(FULL["small-claim-stress"], 256, 30000, corrupt_rate=0.05, num_load_failed=3,
                   predicate_fraction=0.5), name="stress-predicate"),
    MAX_BS_SHORT,
    MAX_BS_LONG,
    MIN_BS,
    # one GPU's head shard of the 70B pool under 8-way tensor parallelism
    scaled(SHARDS["llama3-70b-tp8-shard"], 24, 40, corrupt_rate=0.1, missing_claim_rate=0.1,
           num_load_failed=1),
    MANY_PLANES,
    MANY_PLANES_RAGGED,
    MANY_BLOCKS,
]


def run_both_real(torch, ck, w, batch, faults):
    """Whole lifecycle on both sides with real digests of every block."""
    g = w.geometry
    kv = gpu_pool_tensor(torch, w)
    db = ck.DeviceBatch(batch)
    with ck.Pool(g, w.seed, kv, **capacities(batch)) as pool:
        pool.offload(db)
        pool.restore(db, faults=faults)
        pool.check(db)
        out, ev = pool.read()
        st = pool.block_state()
    host = content.pool_host(g, w.content_seed)
    d0 = digests(host, w)
    restored = apply_flips(host, w, faults)
    d1 = digests(restored, w)
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    assert op.offload(batch, d0) == O.OK
    assert op.restore(batch, faults.load_failed) == O.OK
    want = op.check(batch, d1)
    return out, ev, st, want, op.events(), op.block_state(), kv


@pytest.mark.parametrize("w", SCALED, ids=lambda w: w.name)
def test_parity_scaled_real_digests(torch, ck, w):
    batch = make_batch(w)
    faults = make_faults(w, batch)
    note(f"scaled parity {w.name}: {batch.num_claims} claims, {batch.num_refs} refs, "
         f"{w.geometry.num_blocks} blocks of {w.geometry.block_bytes} B, "
         f"{faults.flip_blocks.size} flips, {faults.load_failed.size} load failures")
    out, ev, st, want, want_ev, want_st, kv = run_both_real(torch, ck, w, batch, faults)
    same_outcomes(out, want)
    same_events(ev, want_ev)
    for f in ("d_off", "d_res", "valid_off", "load_failed"):
        assert np.array_equal(st[f], want_st[f]), f
    # the restored pool holds exactly the flipped bytes
    host = apply_flips(content.pool_host(w.geometry, w.content_seed), w, faults)
    assert np.array_equal(kv.cpu().numpy(), host)
    codes = np.bincount(out["code"], minlength=3)
    note(f"  outcomes unknown/materialized/failed = {codes.tolist()}")
    if w.predicate_fraction:
        # the case must reach the predicate's own branch: a claim that is
        # materialized although one of its blocks failed past the predicate
        beyond = (out["reasons"] & ck.R_BEYOND_PREDICATE) != 0
        assert (beyond & (out["code"] == ck.MATERIALIZED)).any()
        assert (out["intact_blocks"] <= out["num_blocks"]).all()
    del kv
    free_gpu(torch)


# ------------------------------------------------------ paper controls, mirrored


class Mirror:
    """The same lifecycle steps on the GPU library and on the oracle (tiny
    pool, real bytes on both sides)."""

    def __init__(self, torch, ck, event_capacity=4096, w=TINY, stream=None, max_claims=256,
                 max_footprint=8192):
        self.w = w
        g = self.w.geometry
        self.torch, self.ck = torch, ck
        self.kv = gpu_pool_tensor(torch, self.w)
        self.host = content.pool_host(g, self.w.content_seed)
        self.pool = ck.Pool(g, self.w.seed, self.kv, stream=stream, max_claims=max_claims,
                            max_footprint=max_footprint, event_capacity=event_capacity)
        self.op = O.OraclePool(g.num_blocks, g.block_size, self.w.seed)

    def offload(self, batch):
        try:
            self.pool.offload(self.ck.DeviceBatch(batch))
            rc = self.ck.OK
        except self.ck.ClaimError as e:
            rc = e.status
        want = self.op.offload(batch, digests(self.host, self.w))
        assert rc == want, (rc, want)
        return rc

    def restore(self, batch, flips=(), load_failed=()):
        f = FaultSpec(np.array([b for b, _ in flips], np.uint32),
                      np.array([bit for _, bit in flips], np.uint64),
                      np.array(load_failed, np.uint32))
        # a temporary batch: the pool keeps its device arrays alive until
        # the work queued on its stream (which may not be torch's) is done
        self.pool.restore(self.ck.DeviceBatch(batch), faults=f)
        self.host = apply_flips(self.host, self.w, f)
        assert self.op.restore(batch, f.load_failed) == O.OK

    def rewrite(self, block, canon):
        """Replace block's bytes (canonical order) on the GPU pool and the host copy."""
        g = self.w.geometry
        self.pool.stream.synchronize()
        src = self.torch.from_numpy(np.ascontiguousarray(canon).reshape(g.planes, g.chunk_bytes)).cuda()
        self.kv.view(g.planes, g.num_blocks, g.chunk_bytes)[:, block, :] = src
        self.torch.cuda.synchronize()
        self.host.reshape(g.planes, g.num_blocks, g.chunk_bytes)[:, block, :] = \
            np.ascontiguousarray(canon).reshape(g.planes, g.chunk_bytes)

    def canonical(self, block):
        g = self.w.geometry
        return O.canonical_block(self.host, g.planes, g.num_blocks, g.chunk_bytes, block)

    def lookup(self, batch):
        got = self.pool.lookup(self.ck.DeviceBatch(batch))
        want = self.op.lookup(batch)
        for f in want.dtype.names:
            if f != "pad":
                assert np.array_equal(got[f], want[f]), f
        assert self.pool.identity_stats() == self.op.identity_stats()
        return got

    def check(self, batch):
        self.pool.check(self.ck.DeviceBatch(batch))
        want = self.op.check(batch, digests(self.host, self.w))
        got, ev = self.pool.read()
        same_outcomes(got, want)
        same_events(ev, self.op.events(clear=True))
        return got

    def finish(self):
        st = self.pool.block_state()
        want = self.op.block_state()
        for f in st:
            assert np.array_equal(st[f], want[f]), f
        self.pool.close()


RNG = np.random.default_rng(77)


def toks(nblocks, tail=16):
    return RNG.integers(0, 32000, size=(nblocks - 1) * 16 + tail if nblocks else 0, dtype=np.uint32)


def test_controls_mirrored(torch, ck):
    note("controls mirrored on gpu and oracle")
    m = Mirror(torch, ck)
    ck_ = ck
    # path A and B and C in one pool
    tA, tB, tN = toks(3, 5), toks(4), toks(3)
    a = from_claims([(0xA, [3, 9, 27], tA)])
    b = from_claims([(0xB, [5, 6, 7, 8], tB), (0xD, [40, 41, 42], tN)])
    m.offload(a)
    m.offload(b)
    m.restore(a)
    m.restore(b, flips=[(41, 1234)], load_failed=[7])
    out = m.check(from_claims([(0xA, [3, 9, 27], tA), (0xB, [5, 6, 7, 8], tB),
                               (0xD, [40, 41, 42], tN)]))
    assert out["code"].tolist() == [ck_.MATERIALIZED, ck_.RESTORE_FAILED_FAIL_CLOSED,
                                    ck_.RESTORE_FAILED_FAIL_CLOSED]
    # unclaimed failure, not accepted, reuse without restore, identity mismatch
    m.restore(from_claims([]), flips=[(60, 7)], load_failed=[61])
    c = from_claims([(0xC, [10, 11], toks(2))])
    m.offload(c)
    tk = toks(3)
    e = from_claims([(0xE, [12, 13, 14], tk)])
    m.offload(e)
    m.restore(e)
    m.check(from_claims([(0xF, [10, 11], c.claim(0)[2]),  # never accepted
                         (0xC, [10, 11], c.claim(0)[2]),  # no restore
                         (0xE, [12, 13, 14], np.where(np.arange(tk.size) == 20, tk + 1, tk)),
                         (0xE, [12, 99 % 64, 14], tk),  # footprint mismatch
                         (0xE, [12, 13], tk[:32]),
                         (0xE, [12, 13, 14], tk)]))
    # missing entries, empty and malformed rows, shared block
    f = from_claims([(0x10, [20, MISSING, 21], toks(3)), (0x11, [], toks(0)),
                     (0xFFFFFFFFFFFFFFFF, [22], toks(1)), (0x12, [23, 24], toks(3)),
                     (0x13, [30, 31, 32], toks(3)), (0x14, [30, 31, 33], toks(3))])
    m.offload(f)
    m.restore(f, flips=[(31, 999)])
    m.check(f)
    # duplicates refuse acceptance on both sides
    assert m.offload(from_claims([(0x20, [1], toks(1)), (0x20, [2], toks(1))])) == ck_.EDUP
    assert m.offload(from_claims([(0x21, [1], toks(1)), (0xA, [2], toks(1))])) == ck_.EDUP
    # the running example: 448 tokens = 28 blocks, failure in the 28th block
    p = from_claims([(0x448, list(range(28, 56)), toks(28))])
    m.offload(p)
    m.restore(p, load_failed=[55])
    out = m.check(p)
    assert out[0]["first_failing_block"] == 27
    # the same example with a longer claim and its predicate fixed at
    # acceptance: a failure past block 28 leaves it materialized
    tp = toks(36)
    lp = from_claims([(0x44A, list(range(20, 56)), tp), (0x44B, list(range(20, 56)), tp)])
    lp.predicate_tokens = np.array([448, 449], np.uint64)
    m.offload(lp)
    m.restore(lp, flips=[(48, 77)])
    lp.predicate_tokens = None
    out = m.check(lp)
    assert out["code"].tolist() == [ck_.MATERIALIZED, ck_.RESTORE_FAILED_FAIL_CLOSED]
    assert out["intact_blocks"].tolist() == [28, 28]
    assert out[0]["reasons"] == ck_.R_BEYOND_PREDICATE
    # a later offload of the failed block by another claim records that
    # claim's own offload: it is materialized, the first claim stays failed
    q = from_claims([(0x449, [55], toks(1))])
    m.offload(q)
    m.restore(q)
    m.restore(p)
    out = m.check(from_claims([p.claim(0), q.claim(0)]))
    assert out["code"].tolist() == [ck_.RESTORE_FAILED_FAIL_CLOSED, ck_.MATERIALIZED]
    # block 48 (position 20 of the 448 claim) was flipped after its offload,
    # by the restore of the longer claims: that now decides first
    assert out[0]["first_failing_block"] == 20
    assert out[0]["reasons"] == ck_.R_LOAD_FAILED | ck_.R_DIGEST_MISMATCH
    # malformed offsets in a device batch never fault and give UNKNOWN
    bad = from_claims([(0x30, [1, 2], toks(2)), (0x31, [3], toks(1))])
    bad.block_offsets[1] = 3
    bad.block_offsets[2] = 2
    m.offload(bad)
    m.restore(bad)
    m.check(bad)
    # an empty batch on every call
    empty = from_claims([])
    m.offload(empty)
    m.restore(empty)
    m.check(empty)
    assert m.lookup(empty).size == 0
    m.finish()
    del m
    free_gpu(torch)


def test_claim_scoped_records_mirrored(torch, ck):
    """Section 5 storage_restorability row and Table 9 (fallback-recompute
    and wrong-claim rows), on the GPU against the oracle with real bytes:
    (1) claim C's restore reports block 6 lost; the block is recomputed with
    the same bytes and stored by another claim X's offload: C still fails
    closed at position 1, X is materialized; (2) claim D is restored intact,
    then its block 12 receives other bytes that claim Y offloads: D fails
    closed at position 1 against its own offload digest, Y is materialized."""
    note("claim-scoped offload records mirrored")
    m = Mirror(torch, ck)
    c = from_claims([(0xC0, [5, 6, 7], toks(3))])
    m.offload(c)
    m.restore(c, load_failed=[6])
    out = m.check(c)
    assert (int(out[0]["code"]), int(out[0]["first_failing_block"])) == (ck.RESTORE_FAILED_FAIL_CLOSED, 1)
    x = from_claims([(0xA0, [6], toks(1))])
    m.rewrite(6, m.canonical(6).copy())  # the recompute: the same bytes written again
    m.offload(x)
    m.restore(x)
    m.restore(c)
    out = m.check(from_claims([c.claim(0), x.claim(0)]))
    assert out["code"].tolist() == [ck.RESTORE_FAILED_FAIL_CLOSED, ck.MATERIALIZED]
    assert int(out[0]["reasons"]) == ck.R_LOAD_FAILED

    d = from_claims([(0xD0, [11, 12, 13], toks(3))])
    m.offload(d)
    m.restore(d)
    assert m.check(d)[0]["code"] == ck.MATERIALIZED
    before = m.canonical(12).copy()
    m.rewrite(12, np.random.default_rng(3).integers(0, 256, size=before.size, dtype=np.uint8))
    y = from_claims([(0xB0, [12], toks(1))])
    m.offload(y)
    m.restore(y)
    out = m.check(from_claims([d.claim(0), y.claim(0)]))
    assert out["code"].tolist() == [ck.RESTORE_FAILED_FAIL_CLOSED, ck.MATERIALIZED]
    assert int(out[0]["first_failing_block"]) == 1 and int(out[0]["reasons"]) == ck.R_DIGEST_MISMATCH
    assert int(out[0]["expected_digest"]) == O.block_digest(before, m.w.seed)
    # C and D presented in one batch with a shared block of another claim
    z = from_claims([(0xE0, [6, 12, 20], toks(3))])
    m.offload(z)
    m.restore(z)
    out = m.check(from_claims([c.claim(0), d.claim(0), z.claim(0)]))
    assert out["code"].tolist() == [ck.RESTORE_FAILED_FAIL_CLOSED, ck.RESTORE_FAILED_FAIL_CLOSED,
                                    ck.MATERIALIZED]
    m.finish()
    del m
    free_gpu(torch)


def test_reassigned_block_identity_mirrored(torch, ck):
    """A block registered under a second identity no longer answers lookups
    of the first (section 7 E1; Table 2), across offload calls and within
    one batch, on the GPU against the oracle; a later registration of the
    first identity in the block makes it hit again."""
    note("block reassignment and stale identities mirrored")
    m = Mirror(torch, ck)
    p_tok, q_tok, long_tok = toks(1), toks(1), toks(3)
    m.offload(from_claims([(1, [5], p_tok), (10, [30, 31, 32], long_tok)]))
    reqs = from_claims([(100, [], p_tok), (101, [], q_tok), (102, [], long_tok)])
    got = m.lookup(reqs)
    assert got["status"].tolist() == [ck.LOOKUP_HIT, ck.LOOKUP_MISS, ck.LOOKUP_HIT]
    m.offload(from_claims([(2, [5], q_tok), (11, [31], toks(1))]))
    got = m.lookup(reqs)
    assert got["status"].tolist() == [ck.LOOKUP_MISS, ck.LOOKUP_HIT, ck.LOOKUP_PARTIAL]
    assert int(got[2]["hit_blocks"]) == 1
    m.offload(from_claims([(3, [5], p_tok.copy()), (4, [7], q_tok.copy()), (5, [7], p_tok.copy())]))
    got = m.lookup(reqs)
    # p: registered to 5 and 7 (ambiguous); q: registered to 5 and 7 as well
    assert got["status"].tolist() == [ck.LOOKUP_UNKNOWN, ck.LOOKUP_UNKNOWN, ck.LOOKUP_PARTIAL]
    m.finish()
    del m
    free_gpu(torch)


@pytest.mark.parametrize("heads", [1, 2])
def test_head_shards_add_up(torch, ck, heads):
    """A pool of 4-head blocks cut into head shards of 1 or 2 heads (each
    shard pool holding its heads' bytes of every block, as one GPU does
    under tensor parallelism by KV head): every shard's offload digests
    equal the oracle's shard digests, and for every block the shards'
    digests add up, mod 2^64, to the digest the whole pool records."""
    note(f"head shards of {heads}")
    gf = Geometry(2, 2, 16, 4, 64, 2, 64)
    wf = replace(TINY, name="four-heads", geometry=gf)
    batch = make_batch(wf)
    kv = gpu_pool_tensor(torch, wf)
    host = content.pool_host(gf, wf.content_seed)
    caps = capacities(batch)
    with ck.Pool(gf, wf.seed, kv, **caps) as pool:
        pool.offload(ck.DeviceBatch(batch))
        whole = pool.block_state()["d_off"]
    ref = batch.unique_blocks(gf.num_blocks)
    assert np.array_equal(whole[ref], digests(host, wf)[ref])
    view = kv.view(gf.planes, gf.num_blocks, gf.block_size, 4, gf.row_bytes)
    host_view = host.reshape(gf.planes, gf.num_blocks, gf.block_size, 4, gf.row_bytes)
    acc = np.zeros(gf.num_blocks, dtype=np.uint64)
    for first in range(0, 4, heads):
        gs = replace(gf, num_kv_heads=heads, total_kv_heads=4, first_kv_head=first)
        ws = replace(wf, geometry=gs)
        shard = view[:, :, :, first:first + heads, :].contiguous().view(-1)
        with ck.Pool(gs, ws.seed, shard, **caps) as pool:
            pool.offload(ck.DeviceBatch(batch))
            d = pool.block_state()["d_off"]
        host_shard = np.ascontiguousarray(host_view[:, :, :, first:first + heads, :]).reshape(-1)
        assert np.array_equal(d[ref], digests(host_shard, ws)[ref]), first
        acc += d  # wraps mod 2^64
        del shard
    assert np.array_equal(acc, whole)
    del kv
    free_gpu(torch)


def test_rows_sharing_entries(torch, ck):
    """Block rows that share block-table entries, which compressed rows
    allow only around a row whose offsets run backwards (itself malformed):
    each well-formed claim keeps its own accepted footprint and identities,
    as the oracle does, through offload, restore, check and lookup."""
    note("rows sharing block-table entries")
    m = Mirror(torch, ck)
    tA, tC, tE = toks(4), toks(3, 7), toks(3)
    # A = entries [0, 4), B = [4, 1) malformed, C = [1, 4) (A's last three,
    # other tokens), D = [4, 2) malformed, E = [2, 5) (shares two with A and C)
    batch = Batch(claim_ids=np.array([0xA1, 0xB1, 0xC1, 0xD1, 0xE1], np.uint64),
                  block_offsets=np.array([0, 4, 1, 4, 2, 5], np.uint32),
                  block_ids=np.array([3, 9, 27, 30, 44], np.uint32),
                  token_offsets=np.array([0, 64, 64, 64 + tC.size, 64 + tC.size,
                                          64 + tC.size + tE.size], np.uint64),
                  tokens=np.concatenate([tA, tC, tE]).astype(np.uint32))
    m.offload(batch)
    m.restore(batch, flips=[(44, 1000)])
    out = m.check(batch)
    assert out["code"].tolist() == [ck.MATERIALIZED, ck.UNKNOWN, ck.MATERIALIZED, ck.UNKNOWN,
                                    ck.RESTORE_FAILED_FAIL_CLOSED]
    assert int(out["first_failing_block"][4]) == 2
    # the same claims presented as plain consecutive rows
    out = m.check(from_claims([(0xA1, [3, 9, 27, 30], tA), (0xC1, [9, 27, 30], tC),
                               (0xE1, [27, 30, 44], tE)]))
    assert out["code"].tolist() == [ck.MATERIALIZED, ck.MATERIALIZED,
                                    ck.RESTORE_FAILED_FAIL_CLOSED]
    reqs = from_claims([(0x1, [], tA), (0x2, [], tC), (0x3, [], tE),
                        (0x4, [], np.concatenate([tC[:32], tA[32:]]))])
    want = m.op.lookup(reqs)
    got = m.pool.lookup(ck.DeviceBatch(reqs))
    for f in [n for n in O.LOOKUP_DTYPE.names if n != "pad"]:
        assert np.array_equal(got[f], want[f]), (f, got[f].tolist(), want[f].tolist())
    # the rows register blocks 9, 27 and 30 under A's, then C's, then E's
    # prefixes: each block holds its latest registration, so A and C hit
    # only their first block and E all three
    assert got["status"][:3].tolist() == [ck.LOOKUP_PARTIAL, ck.LOOKUP_PARTIAL, ck.LOOKUP_HIT]
    assert got["hit_blocks"][:3].tolist() == [1, 1, 3]
    assert m.pool.identity_stats() == m.op.identity_stats()
    m.finish()
    free_gpu(torch)


def with_shared_rows(base, first, count, rng):
    """The base batch, then a row whose block offsets run backwards, then
    `count` claims with fresh ids that reuse the block rows of base claims
    first .. first+count-1 (sharing their block-table entries) and present
    fresh tokens of the same lengths."""
    C = base.num_claims
    bo, to = base.block_offsets.astype(np.int64), base.token_offsets.astype(np.int64)
    lens = to[first + 1: first + count + 1] - to[first: first + count]
    fresh = rng.integers(0, 32000, size=int(lens.sum()), dtype=np.uint32)
    ids = np.concatenate([base.claim_ids, [np.uint64(0xBAC0000000000000)],
                          0xC1A0000000000000 + np.arange(count, dtype=np.uint64)]).astype(np.uint64)
    new_bo = np.concatenate([bo, bo[first: first + count + 1]])
    new_to = np.concatenate([to, [to[C]], to[C] + np.cumsum(lens)])
    return Batch(claim_ids=ids, block_offsets=new_bo.astype(np.uint32), block_ids=base.block_ids,
                 token_offsets=new_to.astype(np.uint64),
                 tokens=np.concatenate([base.tokens, fresh]).astype(np.uint32))


def test_shared_rows_at_scale(torch, ck):
    """A scaled stress batch of 3000 claims followed by a backwards row and
    500 claims that share block-table entries with 500 earlier claims but
    present other tokens (3501 rows: several claims per thread in the
    store-offset scan).  Whole lifecycle with real digests and lookups of
    the shared-row claims' tokens, against the oracle."""
    w = scaled(FULL["small-claim-stress"], 256, 3000, corrupt_rate=0.05, num_load_failed=2)
    base = make_batch(w)
    batch = with_shared_rows(base, 1000, 500, np.random.default_rng(7))
    assert batch.block_offsets[3001] < batch.block_offsets[3000]  # the backwards row
    faults = make_faults(w, batch)
    note(f"shared rows at scale: {batch.num_claims} claims, {batch.num_refs} entries")
    out, ev, st, want, want_ev, want_st, kv = run_both_real(torch, ck, w, batch, faults)
    same_outcomes(out, want)
    same_events(ev, want_ev)
    for f in st:
        assert np.array_equal(st[f], want_st[f]), f
    codes = out["code"][3001:]
    assert (codes == ck.MATERIALIZED).any() and (codes == ck.RESTORE_FAILED_FAIL_CLOSED).any()
    assert out["code"][3000] == ck.UNKNOWN
    del kv
    free_gpu(torch)


def test_scratch_growth_and_two_pools(torch, ck):
    """Two pools with different content and seeds, one on torch's stream and
    one on a stream of its own, driven in turn; pool A sees batches of 20,
    3000 and 20 claims (its per-claim scratch, sized for 1024 claims at
    first, grows in the middle of its life) and checks a small batch again
    after the large one.  Each pool against its own oracle."""
    note("scratch growth and two pools")
    wa = replace(TINY, name="pool-a")
    wb = replace(TINY, name="pool-b", seed=4242, content_seed=4343)
    caps = dict(event_capacity=40000, max_claims=8192, max_footprint=65536)
    side = torch.cuda.Stream()
    a = Mirror(torch, ck, w=wa, **caps)
    b = Mirror(torch, ck, w=wb, stream=side, **caps)
    torch.cuda.synchronize()  # pool content filled on torch's stream before pool B's stream reads it
    small1 = make_batch(replace(wa, num_claims=20, gen_seed=301))
    large = make_batch(replace(wa, num_claims=3000, gen_seed=302))
    small2 = make_batch(replace(wa, num_claims=20, gen_seed=303))
    other = make_batch(replace(wb, num_claims=50, gen_seed=304))
    flips = [(3, 77), (40, 131071)]
    a.offload(small1)
    b.offload(other)
    a.restore(small1, flips=flips)
    b.restore(other, flips=[(5, 1)], load_failed=[9])
    a.check(small1)
    b.check(other)
    a.offload(large)
    a.restore(large)
    got = a.check(large)
    assert len(got) == 3000
    b.check(other)
    a.offload(small2)
    a.restore(small2, load_failed=[12])
    a.check(small2)
    a.check(small1)  # the first batch again, after the scratch grew
    b.check(other)
    side.synchronize()
    a.finish()
    b.finish()
    free_gpu(torch)


def test_repeated_checks_append_events_in_order(torch, ck):
    note("repeated checks")
    m = Mirror(torch, ck)
    w = TINY
    batch = make_batch(w)
    faults = make_faults(w, batch)
    m.offload(batch)
    m.restore(batch, flips=list(zip(faults.flip_blocks.tolist(), faults.flip_bits.tolist())))
    first = m.check(batch)
    for _ in range(3):
        again = m.check(batch)
        assert np.array_equal(first, again)  # deterministic
    m.finish()
    free_gpu(torch)


def test_capacity_errors(torch, ck):
    note("capacity errors")
    w = TINY
    g = w.geometry
    kv = gpu_pool_tensor(torch, w)
    batch = make_batch(w)
    db = ck.DeviceBatch(batch)
    with ck.Pool(g, w.seed, kv, max_claims=8, event_capacity=4096) as pool:
        with pytest.raises(ck.ClaimError) as ei:
            pool.offload(db)  # 16 claims > 8
        assert ei.value.status == ck.ENOSPC
    with ck.Pool(g, w.seed, kv, max_claims=64, event_capacity=40) as pool:
        pool.offload(db)  # 16..32 events
        with pytest.raises(ck.ClaimError) as ei:
            pool.check(db)  # could need 32 more
        assert ei.value.status == ck.ENOSPC
        pool.read()  # drains the log
        pool.restore(db)
        pool.read()
        pool.check(db)
        out, ev = pool.read()
        assert len(out) == 16 and len(ev) >= 16
    with ck.Pool(g, w.seed, kv, max_claims=64, event_capacity=4096) as pool:
        small = torch.empty(g.block_bytes, dtype=torch.uint8, device="cuda")
        with pytest.raises(ck.ClaimError) as ei:
            pool.offload(db, staging=small)
        assert ei.value.status == ck.ENOSPC
        pool.offload(db)  # the refused call changed nothing
        with pytest.raises(ck.ClaimError) as ei:
            pool.offload(db)
        assert ei.value.status == ck.EDUP
        bad = FaultSpec(np.array([g.num_blocks], np.uint32), np.array([0], np.uint64),
                        np.zeros(0, np.uint32))
        with pytest.raises(ck.ClaimError) as ei:
            pool.restore(db, faults=bad)
        assert ei.value.status == ck.EINVAL
        bad = FaultSpec(np.array([0], np.uint32), np.array([8 * g.block_bytes], np.uint64),
                        np.zeros(0, np.uint32))
        with pytest.raises(ck.ClaimError) as ei:
            pool.restore(db, faults=bad)
        assert ei.value.status == ck.EINVAL
        # restoring from staging needs the whole staged size
        U = batch.unique_blocks(g.num_blocks).size
        big = torch.empty(U * g.block_bytes, dtype=torch.uint8, device="cuda")
        pool2 = ck.Pool(g, w.seed, kv, max_claims=64, event_capacity=4096)
        pool2.offload(db, staging=big)
        with pytest.raises(ck.ClaimError) as ei:
            pool2.restore(db, staging=big, staging_bytes=big.numel() - 16)
        assert ei.value.status == ck.EINVAL
        pool2.restore(db, staging=big)
        pool2.close()
    del kv
    free_gpu(torch)


# ------------------------------------------------------------- staged round trip


STAGED = [
    scaled(FULL["mla-fp8"], 30, 40, corrupt_rate=0.1, num_load_failed=1),  # 3 pieces per chunk
    scaled(FULL["small-claim-stress"], 96, 300, corrupt_rate=0.1, num_load_failed=1),  # 1 piece
    TINY_CHUNK,  # 48-byte chunks: one ragged piece
    MANY_PLANES_RAGGED,  # staging written in two phases
]


@pytest.mark.parametrize("where", ["device", "pinned-host"])
@pytest.mark.parametrize("w", STAGED, ids=lambda w: w.name)
def test_staged_round_trip(torch, ck, w, where):
    g = w.geometry
    batch = make_batch(w)
    faults = make_faults(w, batch)
    U = batch.unique_blocks(g.num_blocks).size
    note(f"staged round trip via {where}: {U} blocks of {g.block_bytes} B")
    kv = gpu_pool_tensor(torch, w)
    if where == "device":
        staging = torch.empty(U * g.block_bytes, dtype=torch.uint8, device="cuda")
    else:
        staging = torch.empty(U * g.block_bytes, dtype=torch.uint8, pin_memory=True)
    db = ck.DeviceBatch(batch)
    host = content.pool_host(g, w.content_seed)
    with ck.Pool(g, w.seed, kv, **capacities(batch)) as pool:
        pool.offload(db, staging=staging)
        torch.cuda.synchronize()
        # staging holds the canonical bytes, ascending block order
        st_bytes = staging.cpu().numpy()
        uniq = batch.unique_blocks(g.num_blocks)
        for k in (0, U // 2, U - 1):
            want = O.canonical_block(host, g.planes, g.num_blocks, g.chunk_bytes, int(uniq[k]))
            assert np.array_equal(st_bytes[k * g.block_bytes:(k + 1) * g.block_bytes], want)
        kv.zero_()  # the device copy is gone
        pool.restore(db, staging=staging, faults=faults)
        pool.check(db)
        out, ev = pool.read()
    restored = apply_flips(host, w, faults)
    assert np.array_equal(kv.cpu().numpy(), restored)
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    op.offload(batch, digests(host, w))
    op.restore(batch, faults.load_failed)
    same_outcomes(out, op.check(batch, digests(restored, w)))
    same_events(ev, op.events())
    del kv, staging
    free_gpu(torch)


@pytest.mark.parametrize("where", ["device", "pinned-host"])
def test_two_staged_offloads(torch, ck, where):
    """A staged offload into another staging buffer starts a new generation:
    after two staged offloads into two buffers only the second's blocks can
    be copied back.  Batch A (claims over blocks 0..23) is offloaded with
    staging, then batch B (claims over blocks 16..39) with a second staging
    buffer; every staged
    block's device copy is then lost (zeroed).  A restore of A and B from
    B's staging copies back blocks 16..39 only: B's claims and A's claims
    inside 16..23 are materialized, A's claims touching 0..15 fail closed on
    the digest compare (their bytes are gone), never a false success.  GPU
    against the oracle, with the pool bytes after the restore against the
    host model."""
    note(f"two staged offloads via {where}")
    w = TINY
    g = w.geometry
    rng = np.random.default_rng(41)

    def rows(first_id, lo, hi, n):
        out = []
        for k in range(n):
            m = int(rng.integers(1, 4))
            out.append((first_id + k, [int(x) for x in rng.integers(lo, hi, size=m)],
                        rng.integers(0, 32000, size=m * g.block_size, dtype=np.uint32)))
        return out

    a_rows = rows(0xA000, 0, 24, 12) + [(0xAF00, [16, 17, 23], rng.integers(0, 32000, size=48,
                                                                           dtype=np.uint32))]
    b_rows = rows(0xB000, 16, 40, 12)
    a, b, both = from_claims(a_rows), from_claims(b_rows), from_claims(a_rows + b_rows)
    ua, ub = a.unique_blocks(g.num_blocks), b.unique_blocks(g.num_blocks)
    kv = gpu_pool_tensor(torch, w)

    def staging_for(n):
        if where == "device":
            return torch.empty(n * g.block_bytes, dtype=torch.uint8, device="cuda")
        return torch.empty(n * g.block_bytes, dtype=torch.uint8, pin_memory=True)

    st_a, st_b = staging_for(ua.size), staging_for(ub.size)
    host = content.pool_host(g, w.content_seed)
    with ck.Pool(g, w.seed, kv, max_claims=128, max_footprint=1024, event_capacity=1024) as pool:
        pool.offload(ck.DeviceBatch(a), staging=st_a)
        pool.offload(ck.DeviceBatch(b), staging=st_b)
        pool.stream.synchronize()
        lost = np.union1d(ua, ub)
        idx = torch.as_tensor(lost.astype(np.int64), device="cuda")
        kv.view(g.planes, g.num_blocks, g.chunk_bytes)[:, idx, :] = 0
        torch.cuda.synchronize()
        db = ck.DeviceBatch(both)
        pool.restore(db, staging=st_b)
        pool.read()
        pool.check(db)
        out, ev = pool.read()
    model = host.copy()
    gone = np.setdiff1d(ua, ub)  # staged only by the first offload
    model.reshape(g.planes, g.num_blocks, g.chunk_bytes)[:, gone, :] = 0
    assert np.array_equal(kv.cpu().numpy(), model)
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    op.offload(a, digests(host, w))
    op.offload(b, digests(host, w))
    op.restore(both)
    op.events(clear=True)
    same_outcomes(out, op.check(both, digests(model, w)))
    same_events(ev, op.events())
    gone_set = set(int(x) for x in gone)
    for c, (cid, blks, _) in enumerate(a_rows + b_rows):
        hit = [j for j, x in enumerate(blks) if x in gone_set]
        if hit:
            assert (int(out[c]["code"]), int(out[c]["first_failing_block"])) == \
                (ck.RESTORE_FAILED_FAIL_CLOSED, hit[0]), cid
            assert out[c]["reasons"] & ck.R_DIGEST_MISMATCH
        else:
            assert out[c]["code"] == ck.MATERIALIZED, cid
    assert (out["code"] == ck.MATERIALIZED).any() and (out["code"] == ck.RESTORE_FAILED_FAIL_CLOSED).any()
    del kv, st_a, st_b
    free_gpu(torch)


# ----------------------------------------------------------- full-size workloads


@pytest.mark.parametrize("case", ["append", "too-small", "reset", "unstaged-between"])
@pytest.mark.parametrize("where", ["device", "pinned-host"])
def test_staging_buffer_accumulates(torch, ck, where, case):
    """Staged offloads into one staging buffer accumulate (section 7 paths A
    and B: the offload tier holds the blocks of every staged offload).
    Batch A (claims over blocks 0..23) is staged, then batch B (blocks
    16..39) into the same buffer; every staged block's device copy is then
    lost (zeroed), and A and B are restored from the buffer.
      append:           every block comes back; every claim is materialized.
      too-small:        the buffer lacks one block for B: B's offload is
                        refused with ENOSPC and changes nothing; A still
                        comes back whole.
      reset:            claim_staging_reset between the offloads: B starts a
                        new generation at the start of the buffer, so the
                        blocks only A staged are lost and A's claims on them
                        fail closed.
      unstaged-between: an offload of blocks 0..7 without staging between A
                        and B drops their staged copies, so they are lost.
    GPU against the oracle, with the pool bytes after the restore against
    the host model."""
    note(f"staging buffer accumulates: {case} via {where}")
    w = TINY
    g = w.geometry
    rng = np.random.default_rng(43)

    def rows(first_id, lo, hi, n):
        out = []
        for k in range(n):
            m = int(rng.integers(1, 4))
            out.append((first_id + k, [int(x) for x in rng.integers(lo, hi, size=m)],
                        rng.integers(0, 32000, size=m * g.block_size, dtype=np.uint32)))
        return out

    a_rows = rows(0xA000, 0, 24, 12) + [(0xAF00, [0, 8, 23], rng.integers(0, 32000, size=48,
                                                                          dtype=np.uint32))]
    b_rows = rows(0xB000, 16, 40, 12)
    c_rows = [(0xC000, list(range(0, 8)), rng.integers(0, 32000, size=8 * g.block_size,
                                                        dtype=np.uint32))]
    a, b, c = from_claims(a_rows), from_claims(b_rows), from_claims(c_rows)
    ua, ub = a.unique_blocks(g.num_blocks), b.unique_blocks(g.num_blocks)
    slots = ua.size + ub.size - (1 if case == "too-small" else 0)
    if where == "device":
        arena = torch.empty(slots * g.block_bytes, dtype=torch.uint8, device="cuda")
    else:
        arena = torch.empty(slots * g.block_bytes, dtype=torch.uint8, pin_memory=True)
    host = content.pool_host(g, w.content_seed)
    kv = gpu_pool_tensor(torch, w)
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    staged_a = ck.DeviceBatch(a)
    with ck.Pool(g, w.seed, kv, max_claims=128, max_footprint=1024, event_capacity=1024) as pool:
        pool.offload(staged_a, staging=arena)
        assert op.offload(a, digests(host, w)) == O.OK
        if case == "reset":
            pool.staging_reset()
        if case == "unstaged-between":
            pool.offload(ck.DeviceBatch(c))
            assert op.offload(c, digests(host, w)) == O.OK
        offloaded = [a] + ([c] if case == "unstaged-between" else [])
        if case == "too-small":
            with pytest.raises(ck.ClaimError) as e:
                pool.offload(ck.DeviceBatch(b), staging=arena)
            assert e.value.status == ck.ENOSPC
        else:
            pool.offload(ck.DeviceBatch(b), staging=arena)
            assert op.offload(b, digests(host, w)) == O.OK
            offloaded.append(b)
        pool.stream.synchronize()
        lost = np.union1d(ua, ub)
        idx = torch.as_tensor(lost.astype(np.int64), device="cuda")
        kv.view(g.planes, g.num_blocks, g.chunk_bytes)[:, idx, :] = 0
        torch.cuda.synchronize()
        every = from_claims(a_rows + (c_rows if case == "unstaged-between" else [])
                            + (b_rows if case != "too-small" else []))
        db = ck.DeviceBatch(every)
        pool.restore(db, staging=arena)
        pool.read()
        pool.check(db)
        out, ev = pool.read()
    # blocks without a staged copy stay zero
    if case == "append":
        gone = np.zeros(0, np.int64)
    elif case == "too-small":
        gone = np.setdiff1d(ub, ua)  # B was refused: only A's blocks were staged
    elif case == "reset":
        gone = np.setdiff1d(ua, ub)
    else:  # A's blocks among C's, whose staged copies C dropped (B stages none of them)
        gone = np.setdiff1d(np.intersect1d(ua, np.arange(8)), ub)
    model = host.copy()
    model.reshape(g.planes, g.num_blocks, g.chunk_bytes)[:, gone, :] = 0
    assert np.array_equal(kv.cpu().numpy(), model)
    assert op.restore(every) == O.OK
    op.events(clear=True)
    same_outcomes(out, op.check(every, digests(model, w)))
    same_events(ev, op.events())
    codes = out["code"]
    if case in ("append", "too-small"):
        assert (codes[: len(a_rows)] == ck.MATERIALIZED).all()
    else:
        assert (codes == ck.RESTORE_FAILED_FAIL_CLOSED).any()
        assert (codes == ck.MATERIALIZED).any()
    del kv, arena
    free_gpu(torch)


@pytest.mark.parametrize("name", ["llama3-8b", "llama3-70b", "small-claim-stress", "mla-fp8",
                                  "llama3-70b-tp8-shard"])
def test_full_size_parity(torch, ck, name):
    w = FULL[name] if name in FULL else SHARDS[name]
    g = w.geometry
    batch = make_batch(w)
    faults = make_faults(w, batch)
    note(f"full size {name}: {batch.num_claims} claims, {batch.num_refs} refs, "
         f"{batch.num_tokens} tokens, pool {g.pool_bytes / 1e9:.2f} GB")
    kv = gpu_pool_tensor(torch, w)
    db = ck.DeviceBatch(batch)
    ref = batch.unique_blocks(g.num_blocks)
    reqs, _ = make_requests(w, batch)
    with ck.Pool(g, w.seed, kv, **capacities(batch)) as pool:
        pool.offload(db)
        pool.restore(db, faults=faults)
        _, ev_pre = pool.read(max_outcomes=1)
        pool.check(db)
        out, ev = pool.read()
        st = pool.block_state()
        lk = pool.lookup(ck.DeviceBatch(reqs))
        stats = pool.identity_stats()
    del kv, db
    free_gpu(torch)
    note(f"  gpu done; oracle digests of all {ref.size} referenced blocks on the host")
    last = [0.0]

    def progress(done, total):
        if done == total or done / total >= last[0] + 0.25:
            last[0] = done / total
            note(f"    {done}/{total} blocks digested")

    d0, d1 = real_digests(w, faults, ref, progress=progress)
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    assert op.offload(batch, d0) == O.OK
    assert op.restore(batch, faults.load_failed) == O.OK
    want_pre = op.events(clear=True)
    want = op.check(batch, d1)
    same_events(ev_pre, want_pre)
    same_outcomes(out, want)
    same_events(ev, op.events())
    validate_lifecycle(batch, ev_pre, ev, out)  # the paper's lifecycle order, from the paper alone
    want_lk = op.lookup(reqs)
    for f in want_lk.dtype.names:
        if f != "pad":
            assert np.array_equal(lk[f], want_lk[f]), f
    assert stats == op.identity_stats()
    note(f"  lookup status unknown/hit/partial/miss = {np.bincount(lk['status'], minlength=4).tolist()}, "
         f"identities {stats}")
    # every referenced block's offload and restored digest, bit for bit
    for f, want_d in (("d_off", d0), ("d_res", d1)):
        if not np.array_equal(st[f][ref], want_d[ref]):
            bad = ref[st[f][ref] != want_d[ref]][:5]
            raise AssertionError(f"{f} differs at blocks {bad.tolist()}")
    assert st["valid_off"][ref].all()
    codes = np.bincount(out["code"], minlength=3)
    note(f"  outcomes unknown/materialized/failed = {codes.tolist()}")
    if w.predicate_fraction:
        # the case must reach the predicate's own branch: a claim that is
        # materialized although one of its blocks failed past the predicate
        beyond = (out["reasons"] & ck.R_BEYOND_PREDICATE) != 0
        assert (beyond & (out["code"] == ck.MATERIALIZED)).any()
        assert (out["intact_blocks"] <= out["num_blocks"]).all()


def test_digest_of_unit_words_is_published_key(torch, ck):
    """The library's digest against published values: with pool seed 0, a
    block whose only non-zero canonical word is w_i = 1 digests to
    k_i = splitmix64(0, i) | 1, the i-th published SplitMix64 output with
    its low bit set; w_i = 2^b gives 2^b k_i.  Blocks 0..3 carry the unit
    word at canonical index 0..3 (plane 0); block 4 carries 2^63 at index 1."""
    from tests.test_oracle_hash import GOLD

    note("digest of unit words against published outputs")
    g = Geometry(1, 2, 16, 1, 8, 2, 8)  # 256-byte chunks, 2 planes
    kv = torch.zeros(g.pool_bytes, dtype=torch.uint8, device="cuda")
    words = kv.view(torch.int64)
    chunk_words = g.chunk_bytes // 8
    for b in range(4):  # plane 0, block b, word b of its chunk
        words[b * chunk_words + b] = 1
    words[4 * chunk_words + 1] = -(1 << 63)  # bit 63 of word 1 of block 4
    claim = from_claims([(0xD1, [0, 1, 2, 3, 4], np.arange(5 * 16, dtype=np.uint32))])
    with ck.Pool(g, 0, kv, max_claims=16, max_footprint=64, event_capacity=64) as pool:
        pool.offload(ck.DeviceBatch(claim))
        st = pool.block_state()
    assert [int(x) for x in st["d_off"][:4]] == [x | 1 for x in GOLD]
    assert int(st["d_off"][4]) == ((GOLD[1] | 1) << 63) & ((1 << 64) - 1)
    assert int(st["d_off"][5]) == 0 and not st["valid_off"][5]
    del kv
    free_gpu(torch)
