"""Pins for the oracle's claim lifecycle: outcomes, attribution, event order.

The expected results come from the paper's semantics (section 1 running
example, section 7 witness paths and controls, Table 2 ambiguity rule,
Tables 8 and 9 false-positive controls), stated independently of the
oracle's min-reduction: sequential scans, enumeration, memcmp brute force.
"""

import itertools
from dataclasses import replace

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_01387_amd.synth import FULL, MISSING, TINY, FaultSpec, from_claims, make_batch, make_faults, scaled
from tests.conftest import golden_lines
from tests.helpers import NONE32, apply_flips, digests, expected_by_scan, host_pool, modeled_digests, oracle_lifecycle

KIND = {
    "ACCEPTED": O.EV_ACCEPTED,
    "OFFLOADED": O.EV_OFFLOADED,
    "RESTORE_REQUIRED": O.EV_RESTORE_REQUIRED,
    "RESTORED": O.EV_RESTORED,
    "RESTORATION_FAILED": O.EV_RESTORATION_FAILED,
    "ACTIVE_REQUEST_REFUSED": O.EV_ACTIVE_REQUEST_REFUSED,
    "OUTCOME_UNKNOWN": O.EV_OUTCOME_UNKNOWN,
}
PATHS = {row[0]: [KIND[k] for k in row[1:]] for row in golden_lines("paper_event_paths.txt")
         if row[0] in ("A", "B", "C_target", "C_nontarget")}

BS = TINY.geometry.block_size
NB = TINY.geometry.num_blocks
RNG = np.random.default_rng(2024)


def toks(nblocks, tail=BS):
    return RNG.integers(0, 32000, size=(nblocks - 1) * BS + tail if nblocks else 0, dtype=np.uint32)


def kinds_for(events, cid):
    return [int(e["kind"]) for e in events if int(e["claim_id"]) == cid]


@pytest.fixture(scope="module")
def pool():
    return host_pool(TINY)


@pytest.fixture(scope="module")
def d0(pool):
    return digests(pool, TINY)


def fresh():
    return O.OraclePool(NB, BS, TINY.seed)


# ------------------------------------------------------- outcome enumeration


def test_outcome_enumeration_matches_sequential_scan():
    """Every assignment of ok / failed / missing to the blocks of a claim of
    n <= 7 blocks: missing (no outcome) dominates failure, and the smallest
    position of the dominating kind is reported."""
    nb = 16
    base = np.arange(nb, dtype=np.uint64) * np.uint64(1000003) + np.uint64(17)
    for n in range(0, 8):
        for state in itertools.product("ofm", repeat=n):
            blocks = [j if s != "m" else MISSING for j, s in enumerate(state)]
            tk = np.arange(n * 4, dtype=np.uint32)  # block size 4 -> n token blocks
            b = from_claims([(42, blocks, tk)])
            op = O.OraclePool(nb, 4, 77)
            assert op.offload(b, base) == O.OK
            assert op.restore(b) == O.OK
            after = base.copy()
            for j, s in enumerate(state):
                if s == "f":
                    after[j] ^= np.uint64(1)
            out = op.check(b, after)[0]
            if n == 0:
                assert (out["code"], out["first_failing_block"]) == (O.UNKNOWN, NONE32)
                assert out["reasons"] & O.R_EMPTY
                continue
            if "m" in state:
                want = (O.UNKNOWN, state.index("m"))
            elif "f" in state:
                want = (O.RESTORE_FAILED_FAIL_CLOSED, state.index("f"))
            else:
                want = (O.MATERIALIZED, NONE32)
            assert (int(out["code"]), int(out["first_failing_block"])) == want, state
            assert bool(out["reasons"] & O.R_MISSING_ENTRY) == ("m" in state)
            assert bool(out["reasons"] & O.R_DIGEST_MISMATCH) == ("f" in state)


# ------------------------------------------------------ paper witness paths


def test_path_a_success_order(pool, d0):
    cid = 0xC1A1
    b = from_claims([(cid, [3, 9, 27], toks(3, 5))])
    op = fresh()
    assert op.offload(b, d0) == O.OK
    assert op.restore(b) == O.OK
    out = op.check(b, d0)[0]
    ev = op.events()
    assert kinds_for(ev, cid) == PATHS["A"]
    assert out["code"] == O.MATERIALIZED and out["reasons"] == 0
    assert out["first_failing_block"] == NONE32 and out["phys_block"] == NONE32
    h = O.chain_hash(b.claim(0)[2], BS, TINY.seed)
    assert out["chain_hash"] == h
    assert ev[0]["aux"] == h and ev[-1]["aux"] == h  # accepted identity == restored identity
    assert list(ev["seq"]) == list(range(len(ev)))


def test_path_b_same_claim_reported_load_failure(pool, d0):
    cid = 0xC1B2
    b = from_claims([(cid, [5, 6, 7, 8], toks(4))])
    op = fresh()
    op.offload(b, d0)
    op.restore(b, load_failed_blocks=[7])
    out = op.check(b, d0)[0]
    ev = op.events()
    assert kinds_for(ev, cid) == PATHS["B"]
    assert out["code"] == O.RESTORE_FAILED_FAIL_CLOSED
    assert out["first_failing_block"] == 2 and out["phys_block"] == 7
    assert out["reasons"] == O.R_LOAD_FAILED
    assert out["expected_digest"] == out["observed_digest"] == d0[7]
    refused = ev[ev["kind"] == O.EV_ACTIVE_REQUEST_REFUSED]
    assert len(refused) == 1 and refused[0]["aux"] == cid  # blocking_claim_ids = [C]
    failed = ev[ev["kind"] == O.EV_RESTORATION_FAILED]
    assert failed[0]["seq"] < refused[0]["seq"]
    h = O.chain(b.claim(0)[2], BS, TINY.seed)
    assert out["chain_hash_at_fail"] == h[2]


def test_path_b_silent_corruption(pool, d0):
    cid = 0xC1B3
    b = from_claims([(cid, [10, 11, 12], toks(3))])
    f = FaultSpec(np.array([11], np.uint32), np.array([12345], np.uint64), np.zeros(0, np.uint32))
    op, out, ev, _, d1 = oracle_lifecycle(TINY, b, f, pool)
    assert kinds_for(ev, cid) == PATHS["B"]
    o = out[0]
    assert o["code"] == O.RESTORE_FAILED_FAIL_CLOSED and o["first_failing_block"] == 1
    assert o["expected_digest"] == d0[11] and o["observed_digest"] == d1[11] != d0[11]
    assert o["reasons"] == O.R_DIGEST_MISMATCH


def test_path_c_target_only_attribution(pool):
    target, nontarget = 0x7A, 0x7B
    b = from_claims([(target, [1, 2, 3], toks(3)), (nontarget, [4, 5, 6], toks(3))])
    f = FaultSpec(np.array([2], np.uint32), np.array([77], np.uint64), np.zeros(0, np.uint32))
    op, out, ev, _, _ = oracle_lifecycle(TINY, b, f, pool)
    assert kinds_for(ev, target) == PATHS["C_target"]
    assert kinds_for(ev, nontarget) == PATHS["C_nontarget"]
    refused = ev[ev["kind"] == O.EV_ACTIVE_REQUEST_REFUSED]
    assert set(int(x) for x in refused["aux"]) == {target}
    assert out["code"].tolist() == [O.RESTORE_FAILED_FAIL_CLOSED, O.MATERIALIZED]


# ------------------------------------------- false-positive controls (Table 9)


def test_unclaimed_failure_gives_no_claim_outcome(pool):
    b = from_claims([(1, [0, 1], toks(2)), (2, [2, 3], toks(2))])
    f = FaultSpec(np.array([40], np.uint32), np.array([5], np.uint64), np.array([41], np.uint32))
    op, out, ev, _, _ = oracle_lifecycle(TINY, b, f, pool)
    assert (out["code"] == O.MATERIALIZED).all()
    assert not (ev["kind"] == O.EV_RESTORATION_FAILED).any()


def test_fallback_recompute_does_not_restore_the_claim(pool, d0):
    """A reported load failure stays a failure of the claim even if the bytes
    are later rewritten correctly (Table 9, fallback-recompute row: a
    recompute after a failed load is not evidence that the claim was
    restored)."""
    b = from_claims([(9, [20, 21], toks(2))])
    op = fresh()
    op.offload(b, d0)
    op.restore(b, load_failed_blocks=[21])
    out = op.check(b, d0)[0]  # bytes equal to the original
    assert out["code"] == O.RESTORE_FAILED_FAIL_CLOSED and out["first_failing_block"] == 1
    # a second restore without a reported failure does not clear it either
    op.restore(b)
    out = op.check(b, d0)[0]
    assert out["code"] == O.RESTORE_FAILED_FAIL_CLOSED and out["reasons"] == O.R_LOAD_FAILED


def test_recompute_stored_by_another_claim_does_not_restore_the_first():
    """Section 5 storage_restorability row (store and load name the same
    claim; a hook must not relabel a fallback recompute as restoration) and
    Table 9's fallback-recompute row.  Claim C = [5, 6, 7] is offloaded and
    its restore reports block 6 lost; the block is recomputed (the same
    bytes) and stored by an offload of another claim X = [6], which is then
    restored.  C's reuse still fails closed at position 1; X, whose own
    offload recorded the recomputed bytes, is materialized."""
    d = np.arange(NB, dtype=np.uint64) * np.uint64(7919) + np.uint64(11)
    c = from_claims([(0xC, [5, 6, 7], toks(3))])
    x = from_claims([(0xA, [6], toks(1))])
    op = fresh()
    assert op.offload(c, d) == O.OK
    assert op.restore(c, load_failed_blocks=[6]) == O.OK
    first = op.check(c, d)[0]
    assert (first["code"], first["first_failing_block"]) == (O.RESTORE_FAILED_FAIL_CLOSED, 1)
    assert op.offload(x, d) == O.OK  # the recompute, stored under X
    assert op.restore(x) == O.OK
    op.events(clear=True)
    out_c = op.check(c, d)[0]
    assert (out_c["code"], out_c["first_failing_block"], out_c["phys_block"]) == \
        (O.RESTORE_FAILED_FAIL_CLOSED, 1, 6)
    assert out_c["reasons"] == O.R_LOAD_FAILED
    assert kinds_for(op.events(), 0xC) == [O.EV_RESTORATION_FAILED, O.EV_ACTIVE_REQUEST_REFUSED]
    out_x = op.check(x, d)[0]
    assert out_x["code"] == O.MATERIALIZED and out_x["reasons"] == 0
    # C restored again, after X's offload: still failed, never RESTORED
    op.restore(c)
    assert op.check(c, d)[0]["code"] == O.RESTORE_FAILED_FAIL_CLOSED
    assert O.EV_RESTORED not in kinds_for(op.events(), 0xC)


def test_another_claims_offload_record_does_not_satisfy_the_claim():
    """Section 5 storage_restorability row (store and load name the same
    claim) and Table 9's wrong-claim row.  Claim C = [5, 6, 7] is offloaded,
    restored and materialized.  Block 6 then receives other bytes, which a
    second claim X = [6] offloads.  C's next check compares block 6 with C's
    own offload, not X's: it fails closed at position 1, with C's digest as
    the expected one and the new bytes' digest as the observed one.  X is
    materialized."""
    d = np.arange(NB, dtype=np.uint64) * np.uint64(7919) + np.uint64(11)
    c = from_claims([(0xC, [5, 6, 7], toks(3))])
    x = from_claims([(0xA, [6], toks(1))])
    op = fresh()
    op.offload(c, d)
    op.restore(c)
    assert op.check(c, d)[0]["code"] == O.MATERIALIZED
    d2 = d.copy()
    d2[6] = np.uint64(0x5EED)  # block 6 now holds X's bytes
    op.offload(x, d2)
    op.restore(x)
    out = op.check(c, d2)[0]
    assert (out["code"], out["first_failing_block"], out["phys_block"]) == \
        (O.RESTORE_FAILED_FAIL_CLOSED, 1, 6)
    assert out["reasons"] == O.R_DIGEST_MISMATCH
    assert (int(out["expected_digest"]), int(out["observed_digest"])) == (int(d[6]), 0x5EED)
    assert op.check(x, d2)[0]["code"] == O.MATERIALIZED
    # the block state keeps the latest offload's digest (X's): evidence only
    assert int(op.block_state()["d_off"][6]) == 0x5EED


def test_failure_reported_before_a_claim_is_not_its_failure():
    """A load failure reported before a claim's offload belongs to the claims
    that had recorded the block then; the later claim recorded the block's
    bytes itself (section 7 path C: only the claim's own failure counts)."""
    d = np.arange(NB, dtype=np.uint64) + np.uint64(5)
    a = from_claims([(1, [3, 4], toks(2))])
    b = from_claims([(2, [4, 8], toks(2))])
    op = fresh()
    op.offload(a, d)
    op.restore(a, load_failed_blocks=[4])
    op.offload(b, d)
    op.restore(from_claims([(1, [3, 4], a.claim(0)[2]), (2, [4, 8], b.claim(0)[2])]))
    out = op.check(from_claims([(1, [3, 4], a.claim(0)[2]), (2, [4, 8], b.claim(0)[2])]), d)
    assert out["code"].tolist() == [O.RESTORE_FAILED_FAIL_CLOSED, O.MATERIALIZED]
    # a failure reported after both offloads fails both
    op.restore(from_claims([(2, [4, 8], b.claim(0)[2])]), load_failed_blocks=[4])
    out = op.check(from_claims([(1, [3, 4], a.claim(0)[2]), (2, [4, 8], b.claim(0)[2])]), d)
    assert out["code"].tolist() == [O.RESTORE_FAILED_FAIL_CLOSED] * 2
    assert out["first_failing_block"].tolist() == [1, 0]
    assert op.block_state()["load_failed"][4] == 1


def _write_block(pool, g, b, canon):
    """Put canonical bytes into block b of a host pool array ([plane][block][chunk])."""
    flat = pool.reshape(-1)
    for p in range(g.planes):
        at = (p * g.num_blocks + b) * g.chunk_bytes
        flat[at:at + g.chunk_bytes] = canon[p * g.chunk_bytes:(p + 1) * g.chunk_bytes]


@pytest.mark.parametrize("seed", range(12))
def test_multi_offload_lifecycles_match_a_claim_ledger(seed):
    """Random lifecycles over a few shared blocks: offloads of new claims,
    block rewrites between them (recomputes of earlier bytes, other bytes,
    single-bit flips), restores with reported load failures, and checks.
    The expectation is a ledger written from the paper with no digest: each
    claim's offload stores a copy of its blocks' bytes (the claim's own
    offload, section 5 storage_restorability); a check of a restored claim
    fails closed at the first position whose current bytes differ from the
    claim's own stored copy, or whose block had a load failure reported by a
    restore call after the claim's offload (Table 9: a recompute is not a
    restore, a wrong claim's record does not count); a claim never restored
    has no outcome."""
    rng = np.random.default_rng(7000 + seed)
    w = TINY
    g = w.geometry
    pool = host_pool(w).copy()
    hot = rng.choice(g.num_blocks, size=6, replace=False)
    op = fresh()
    ledger = {}  # claim id -> [blocks, tokens, stored copies, call index, restored]
    reports = []  # (block, call index)
    calls = 0
    seen_outcomes = set()
    for step in range(14):
        act = rng.choice(["offload", "rewrite", "restore", "check"], p=[0.3, 0.3, 0.2, 0.2])
        if step == 13:
            act = "restore"  # the last step restores and then checks every claim
        if act == "offload" or not ledger:
            calls += 1
            rows = []
            for _ in range(int(rng.integers(1, 4))):
                cid = 100 + len(ledger) + len(rows)
                n = int(rng.integers(1, 4))
                blks = [int(x) for x in rng.choice(hot, size=n)]
                rows.append((cid, blks, toks(n)))
            batch = from_claims(rows)
            assert op.offload(batch, digests(pool, w)) == O.OK
            for cid, blks, tk in rows:
                copies = [O.canonical_block(pool, g.planes, g.num_blocks, g.chunk_bytes, b).copy()
                          for b in blks]
                ledger[cid] = [blks, tk, copies, calls, False]
        elif act == "rewrite":
            b = int(rng.choice(hot))
            u = rng.random()
            if u < 0.4:  # a recompute: bytes equal to some claim's stored copy of b
                copies = [c[2][j] for c in ledger.values() for j, x in enumerate(c[0]) if x == b]
                if not copies:
                    continue
                _write_block(pool, g, b, copies[int(rng.integers(len(copies)))])
            elif u < 0.7:  # other bytes
                _write_block(pool, g, b, rng.integers(0, 256, size=g.block_bytes, dtype=np.uint8))
            else:  # a silent single-bit flip
                O.apply_flip(pool, g.planes, g.num_blocks, g.chunk_bytes, b,
                             int(rng.integers(0, 8 * g.block_bytes)))
        elif act == "restore":
            calls += 1
            cids = [c for c in ledger if rng.random() < 0.8 or step == 13]
            lost = [int(b) for b in hot if rng.random() < 0.15]
            batch = from_claims([(c, ledger[c][0], ledger[c][1]) for c in cids])
            assert op.restore(batch, load_failed_blocks=lost) == O.OK
            reports += [(b, calls) for b in lost]
            for c in cids:
                ledger[c][4] = True
        if act == "check" or step == 13:
            cids = list(ledger)
            rng.shuffle(cids)
            batch = from_claims([(c, ledger[c][0], ledger[c][1]) for c in cids])
            out = op.check(batch, digests(pool, w))
            for o, c in zip(out, cids):
                blks, _, copies, at, restored = ledger[c]
                if not restored:
                    assert (int(o["code"]), int(o["first_failing_block"])) == (O.UNKNOWN, NONE32)
                    assert o["reasons"] & O.R_NO_RESTORE
                    continue
                bad = []
                for j, b in enumerate(blks):
                    now = O.canonical_block(pool, g.planes, g.num_blocks, g.chunk_bytes, b)
                    lost = any(rb == b and rc > at for rb, rc in reports)
                    if lost or not np.array_equal(now, copies[j]):
                        bad.append(j)
                if not bad:
                    assert o["code"] == O.MATERIALIZED and o["reasons"] == 0, (seed, step, c)
                else:
                    j = bad[0]
                    assert (int(o["code"]), int(o["first_failing_block"])) == \
                        (O.RESTORE_FAILED_FAIL_CLOSED, j), (seed, step, c, bad)
                    assert int(o["expected_digest"]) == O.block_digest(copies[j], w.seed)
                seen_outcomes.add(int(o["code"]))
    assert seen_outcomes  # restored claims were checked


def test_event_payloads_against_independent_values(pool, d0):
    """Each event's aux payload (section 7 event list, paths A and B),
    against a value computed without the lifecycle code: OFFLOADED carries
    the number of block-table entries offloaded; RESTORE_REQUIRED the
    accepted number, whatever the restore batch presents; RESTORATION_FAILED
    the restored (observed) digest at the failing block, here from the exact
    single-flip delta D_off + (w' - w) * k_i mod 2^64; OUTCOME_UNKNOWN the
    reason bits; a malformed row's chain hash is the seed (no tokens are
    read)."""
    cid = 0xB0B
    blocks = [10, 11, 12]
    tk = toks(3)
    b = from_claims([(cid, blocks, tk)])
    bit = 8 * 4096 * 2 + 64 * 37 + 61  # plane 2 of the 4 planes, word 37 there, bit 61
    f = FaultSpec(np.array([11], np.uint32), np.array([bit], np.uint64), np.zeros(0, np.uint32))
    op = fresh()
    assert op.offload(b, d0) == O.OK
    # the restore presents the claim with a shorter row: aux is the accepted count
    assert op.restore(from_claims([(cid, blocks[:2], tk[: 2 * BS])])) == O.OK
    restored = apply_flips(pool, TINY, f)
    out = op.check(b, digests(restored, TINY))[0]
    ev = op.events()
    aux = {int(e["kind"]): int(e["aux"]) for e in ev}
    assert aux[O.EV_OFFLOADED] == len(blocks)
    assert aux[O.EV_RESTORE_REQUIRED] == len(blocks)
    g = TINY.geometry
    canon = O.canonical_block(pool, g.planes, g.num_blocks, g.chunk_bytes, 11)
    i = bit // 64
    w_old = int.from_bytes(bytes(canon[8 * i:8 * i + 8]), "little")
    w_new = w_old ^ (1 << (bit % 64))
    want = (int(d0[11]) + (w_new - w_old) * O.kv_key(TINY.seed, i)) % (1 << 64)
    assert want != int(d0[11])
    assert (int(out["code"]), int(out["first_failing_block"])) == (O.RESTORE_FAILED_FAIL_CLOSED, 1)
    assert aux[O.EV_RESTORATION_FAILED] == want  # the observed digest, not the expected one
    assert int(out["observed_digest"]) == want and int(out["expected_digest"]) == int(d0[11])
    assert aux[O.EV_ACTIVE_REQUEST_REFUSED] == cid

    # OUTCOME_UNKNOWN carries the reason bits (the header's values)
    op2 = fresh()
    rows = [(1, [4, MISSING, 5], toks(3)), (2, [6, 7], toks(2)), (0xFFFFFFFFFFFFFFFF, [8], toks(1))]
    op2.offload(from_claims(rows[:2]), d0)
    op2.events(clear=True)
    out2 = op2.check(from_claims(rows), d0)
    ev2 = op2.events()
    assert [int(e["kind"]) for e in ev2] == [O.EV_OUTCOME_UNKNOWN] * 3
    assert [int(e["aux"]) for e in ev2] == [0x020 | 0x002 | 0x004, 0x004, 0x200]
    assert [int(e["block_index"]) for e in ev2] == [1, NONE32, NONE32]
    assert int(out2[2]["chain_hash"]) == TINY.seed and int(out2[2]["num_blocks"]) == 0
    empty = op2.check(from_claims([(3, [], toks(0))]), d0)[0]
    assert int(empty["chain_hash"]) == TINY.seed


def test_ordinary_offload_without_claim_is_not_an_outcome(d0):
    """Claim Y was never accepted; its blocks were offloaded by claim X."""
    tk = toks(2)
    x = from_claims([(100, [30, 31], tk)])
    y = from_claims([(200, [30, 31], tk)])
    op = fresh()
    op.offload(x, d0)
    op.restore(x)
    out = op.check(y, d0)[0]
    assert out["code"] == O.UNKNOWN and out["first_failing_block"] == NONE32
    assert out["reasons"] & O.R_NOT_ACCEPTED
    assert kinds_for(op.events(), 200) == [O.EV_OUTCOME_UNKNOWN]


def test_wrong_claim_failure_is_not_attributed(pool):
    b = from_claims([(1, [12, 13], toks(2)), (2, [14, 15], toks(2))])
    f = FaultSpec(np.zeros(0, np.uint32), np.zeros(0, np.uint64), np.array([15], np.uint32))
    op, out, ev, _, _ = oracle_lifecycle(TINY, b, f, pool)
    assert out["code"].tolist() == [O.MATERIALIZED, O.RESTORE_FAILED_FAIL_CLOSED]
    assert kinds_for(ev, 1)[-1] == O.EV_RESTORED


def test_reuse_without_restore_is_ambiguous(d0):
    b = from_claims([(5, [1, 2], toks(2))])
    op = fresh()
    op.offload(b, d0)
    out = op.check(b, d0)[0]
    assert out["code"] == O.UNKNOWN and out["reasons"] == O.R_NO_RESTORE


def test_cache_identity_mismatch_is_ambiguous(d0):
    tk = toks(3)
    b = from_claims([(5, [1, 2, 3], tk)])
    op = fresh()
    op.offload(b, d0)
    op.restore(b)
    tk2 = tk.copy()
    tk2[20] += 1
    out = op.check(from_claims([(5, [1, 2, 3], tk2)]), d0)[0]
    assert out["code"] == O.UNKNOWN and out["reasons"] == O.R_TOKEN_MISMATCH
    # the identity is compared block by block: token 20 lies in block 1
    assert out["first_failing_block"] == 20 // BS and out["intact_blocks"] == 1
    out = op.check(from_claims([(5, [1, 9, 3], tk)]), d0)[0]
    assert out["code"] == O.UNKNOWN and out["first_failing_block"] == 1
    # block 9 differs from the accepted footprint and has no offload record
    assert out["reasons"] == O.R_FOOTPRINT_MISMATCH | O.R_NO_OFFLOAD_RECORD
    out = op.check(from_claims([(5, [1, 2], tk[: 2 * BS])]), d0)[0]
    assert out["code"] == O.UNKNOWN and out["first_failing_block"] == 2
    assert out["reasons"] & O.R_FOOTPRINT_MISMATCH and out["reasons"] & O.R_TOKEN_MISMATCH


def test_missing_entry_blocks_offload_and_outcome(d0):
    b = from_claims([(6, [4, MISSING, 5], toks(3))])
    op = fresh()
    op.offload(b, d0)
    op.restore(b)
    out = op.check(b, d0)[0]
    assert kinds_for(op.events(), 6) == [O.EV_ACCEPTED, O.EV_OUTCOME_UNKNOWN]
    assert out["code"] == O.UNKNOWN and out["first_failing_block"] == 1
    assert out["phys_block"] == MISSING
    assert out["reasons"] & O.R_MISSING_ENTRY and out["reasons"] & O.R_NOT_OFFLOADED
    assert op.claim_state(6) == O.ST_ACCEPTED


def test_unknown_dominates_earlier_failure(pool):
    b = from_claims([(8, [16, 17, 18, MISSING], toks(4))])
    f = FaultSpec(np.array([16], np.uint32), np.array([3], np.uint64), np.zeros(0, np.uint32))
    _, out, _, _, _ = oracle_lifecycle(TINY, b, f, pool)
    assert out[0]["code"] == O.UNKNOWN and out[0]["first_failing_block"] == 3
    assert out[0]["reasons"] & O.R_DIGEST_MISMATCH


def test_shared_block_corruption_fails_every_referencing_claim(pool):
    tk = toks(3)
    b = from_claims([(1, [50, 51, 52], tk), (2, [50, 51, 60], np.concatenate([tk[: 2 * BS], toks(1)])),
                     (3, [61, 62], toks(2))])
    f = FaultSpec(np.array([51], np.uint32), np.array([999], np.uint64), np.zeros(0, np.uint32))
    _, out, _, _, _ = oracle_lifecycle(TINY, b, f, pool)
    assert out["code"].tolist() == [O.RESTORE_FAILED_FAIL_CLOSED, O.RESTORE_FAILED_FAIL_CLOSED,
                                    O.MATERIALIZED]
    assert out["first_failing_block"].tolist()[:2] == [1, 1]
    assert out[0]["chain_hash_at_fail"] == out[1]["chain_hash_at_fail"]  # shared prefix identity


def test_duplicate_ownership_refuses_acceptance(d0):
    op = fresh()
    dup = from_claims([(1, [1], toks(1)), (1, [2], toks(1))])
    assert op.offload(dup, d0) == O.EDUP
    assert len(op.events()) == 0 and op.claim_state(1) == 0
    ok = from_claims([(1, [1], toks(1))])
    assert op.offload(ok, d0) == O.OK
    assert op.offload(from_claims([(2, [2], toks(1)), (1, [3], toks(1))]), d0) == O.EDUP
    assert op.claim_state(2) == 0


def test_malformed_rows_and_empty_claims(d0):
    b = from_claims([(1, [1, 2], toks(2)), (2, [], toks(0)), (0xFFFFFFFFFFFFFFFF, [3], toks(1)),
                     (4, [4, 5], toks(3))])
    op = fresh()
    assert op.offload(b, d0) == O.OK
    op.restore(b)
    out = op.check(b, d0)
    assert out["code"].tolist() == [O.MATERIALIZED, O.UNKNOWN, O.UNKNOWN, O.UNKNOWN]
    assert out[1]["reasons"] & O.R_EMPTY and out[1]["first_failing_block"] == NONE32
    assert out[2]["reasons"] == O.R_MALFORMED and out[2]["num_blocks"] == 0
    assert out[3]["reasons"] & O.R_SHAPE_MISMATCH and out[3]["first_failing_block"] == 2
    assert op.claim_state(0xFFFFFFFFFFFFFFFF) == 0
    # offsets that run backwards make a row malformed, never an error
    bad = from_claims([(7, [1, 2], toks(2)), (8, [3], toks(1))])
    bad.block_offsets[1] = 3  # offsets [0, 3, 2]: row 1 runs backwards
    bad.block_offsets[2] = 2
    op2 = fresh()
    assert op2.offload(bad, d0) == O.OK
    op2.restore(bad)
    out = op2.check(bad, d0)
    assert out[1]["reasons"] == O.R_MALFORMED


def test_predicate_prefix_of_running_example(d0):
    """The running example's predicate covers 448 tokens = 28 full blocks;
    a failure in the 28th block fails the claim, and the chain hash before
    it identifies the intact 27-block prefix."""
    rows = {r[0]: int(r[1]) for r in golden_lines("paper_event_paths.txt") if r[0].startswith("PRED")}
    nblk = rows["PREDICATE_TOKENS"] // rows["PREDICATE_BLOCK_SIZE"]
    assert nblk == 28 and rows["PREDICATE_BLOCK_SIZE"] == BS
    tk = toks(nblk)
    b = from_claims([(0xC, list(range(nblk)), tk)])
    op = fresh()
    op.offload(b, d0)
    op.restore(b, load_failed_blocks=[27])
    out = op.check(b, d0)[0]
    assert out["code"] == O.RESTORE_FAILED_FAIL_CLOSED and out["first_failing_block"] == 27
    h = O.chain(tk, BS, TINY.seed)
    assert out["chain_hash_at_fail"] == h[27] and out["chain_hash"] == h[27]
    assert O.chain_hash(tk[: 27 * BS], BS, TINY.seed) == h[26]


def _scan_with_predicate(state, pred_blocks):
    """Expected (code, first_failing_block, beyond, intact) by a plain left to
    right scan: any ambiguity ('m') decides UNKNOWN at its first position;
    else the first failure ('f') among the predicate's leading blocks fails
    the claim; failures past them leave it MATERIALIZED and only mark
    BEYOND_PREDICATE; intact is the first position that is not 'o'."""
    intact = next((j for j, s in enumerate(state) if s != "o"), len(state))
    beyond = any(s == "f" for s in state[pred_blocks:])
    if "m" in state:
        return O.UNKNOWN, state.index("m"), beyond, intact
    for j, s in enumerate(state[:pred_blocks]):
        if s == "f":
            return O.RESTORE_FAILED_FAIL_CLOSED, j, beyond, intact
    return O.MATERIALIZED, NONE32, beyond, intact


def test_predicate_enumeration_matches_sequential_scan():
    """Every ok / failed / missing assignment to a claim of 1..5 blocks of 4
    tokens, under every predicate length k from 0 tokens to past the claim:
    the predicate covers ceil(k / 4) leading blocks (section 1 running
    example: the blocks holding the first k tokens)."""
    nb, bs = 16, 4
    base = np.arange(nb, dtype=np.uint64) * np.uint64(1000003) + np.uint64(17)
    for n in range(1, 6):
        for state in itertools.product("ofm", repeat=n):
            blocks = [j if s != "m" else MISSING for j, s in enumerate(state)]
            after = base.copy()
            for j, s in enumerate(state):
                if s == "f":
                    after[j] ^= np.uint64(1 << (j % 64))
            for k in range(0, bs * n + 3):
                b = from_claims([(42, blocks, np.arange(n * bs, dtype=np.uint32))])
                b.predicate_tokens = np.array([k], np.uint64)
                op = O.OraclePool(nb, bs, 77)
                assert op.offload(b, base) == O.OK
                assert op.restore(b) == O.OK
                out = op.check(b, after)[0]
                pred_blocks = min(-(-k // bs), n)
                assert op.claim_predicate(42) == pred_blocks
                code, first, beyond, intact = _scan_with_predicate(state, pred_blocks)
                got = (int(out["code"]), int(out["first_failing_block"]),
                       bool(out["reasons"] & O.R_BEYOND_PREDICATE), int(out["intact_blocks"]))
                assert got == (code, first, beyond, intact), (state, k)
                # a failure inside the predicate is the only source of these bits
                assert bool(out["reasons"] & O.R_DIGEST_MISMATCH) == ("f" in state[:pred_blocks])


def test_predicate_running_example_on_a_longer_claim(d0):
    """A 36-block claim whose predicate is leading_prefix_at_least(448): only
    the first 28 blocks decide.  A lost block 30 leaves the claim
    MATERIALIZED (path A events) with the loss recorded as beyond the
    predicate and 30 intact leading blocks; a lost block 27 fails it (path
    B); k = 449 stretches the predicate to block 28."""
    rows = {r[0]: int(r[1]) for r in golden_lines("paper_event_paths.txt") if r[0].startswith("PRED")}
    k = rows["PREDICATE_TOKENS"]
    tk = toks(36)
    cid = 0xC0DE
    for pred_tokens, lost, want_code, want_first in [
        (k, 30, O.MATERIALIZED, NONE32),
        (k, 27, O.RESTORE_FAILED_FAIL_CLOSED, 27),
        (k, 28, O.MATERIALIZED, NONE32),
        (k + 1, 28, O.RESTORE_FAILED_FAIL_CLOSED, 28),
    ]:
        b = from_claims([(cid, list(range(36)), tk)])
        b.predicate_tokens = np.array([pred_tokens], np.uint64)
        op = fresh()
        assert op.offload(b, d0) == O.OK
        assert op.claim_predicate(cid) == -(-pred_tokens // BS)
        op.restore(b, load_failed_blocks=[lost])
        # the predicate was fixed at acceptance: the check's batch carries none
        b.predicate_tokens = None
        out = op.check(b, d0)[0]
        assert (int(out["code"]), int(out["first_failing_block"])) == (want_code, want_first)
        assert out["intact_blocks"] == lost
        if want_code == O.MATERIALIZED:
            assert out["reasons"] == O.R_BEYOND_PREDICATE
            assert kinds_for(op.events(), cid) == PATHS["A"]
        else:
            assert out["reasons"] == O.R_LOAD_FAILED
            assert kinds_for(op.events(), cid) == PATHS["B"]


def test_predicate_of_section_6_2(d0):
    """leading_prefix_at_least(17) over a 35-token claim: the predicate
    covers blocks 0 and 1 only, so a failed partial tail block still leaves
    32 >= 17 intact leading tokens and the claim materialized."""
    rows = {r[0]: int(r[1]) for r in golden_lines("paper_event_paths.txt") if r[0].startswith("PRED")}
    k, T = rows["PREDICATE2_TOKENS"], rows["PREDICATE2_CLAIM_TOKENS"]
    tk = RNG.integers(0, 32000, size=T, dtype=np.uint32)
    for lost, want_code in [(2, O.MATERIALIZED), (1, O.RESTORE_FAILED_FAIL_CLOSED),
                            (0, O.RESTORE_FAILED_FAIL_CLOSED)]:
        b = from_claims([(0x17, [40, 41, 42], tk)])
        b.predicate_tokens = np.array([k], np.uint64)
        op = fresh()
        assert op.offload(b, d0) == O.OK
        assert op.claim_predicate(0x17) == 2
        op.restore(b, load_failed_blocks=[40 + lost])
        out = op.check(b, d0)[0]
        assert out["code"] == want_code and out["intact_blocks"] == lost
        assert min(int(out["intact_blocks"]) * BS, T) >= k or want_code != O.MATERIALIZED


def test_whole_claim_predicate_equals_no_predicate(pool):
    """k >= the claim's token count, or no predicate array at all, both
    cover the whole claim: outcomes and events are identical."""
    w = replace(TINY, num_load_failed=2)
    batch = make_batch(w)
    faults = make_faults(w, batch)
    T = np.diff(batch.token_offsets.astype(np.int64))
    runs = []
    for pred in (None, T.astype(np.uint64), (T + 1000).astype(np.uint64)):
        batch.predicate_tokens = pred
        _, out, ev, _, _ = oracle_lifecycle(w, batch, faults, pool)
        runs.append((out, ev))
        assert np.array_equal(out["intact_blocks"] <= out["num_blocks"], np.ones(len(out), bool))
    for out, ev in runs[1:]:
        assert np.array_equal(out, runs[0][0]) and np.array_equal(ev, runs[0][1])


# --------------------------------------------------- tiny-pool brute force


def test_tiny_workload_matches_memcmp_brute_force():
    """The tiny workload end to end: the failing set is computed by comparing
    restored and original bytes block by block, plus the reported failures,
    with no digest involved; the digest-based outcomes must agree."""
    w = TINY
    b = make_batch(w)
    f = make_faults(w, b)
    f = FaultSpec(f.flip_blocks, f.flip_bits, np.array([int(b.block_ids[5])], np.uint32))
    pool = host_pool(w)
    op, out, ev, d0, d1 = oracle_lifecycle(w, b, f, pool)
    restored = apply_flips(pool, w, f)
    g = w.geometry
    failing = set(int(x) for x in f.load_failed)
    for blk in range(g.num_blocks):
        a = O.canonical_block(pool, g.planes, g.num_blocks, g.chunk_bytes, blk)
        r = O.canonical_block(restored, g.planes, g.num_blocks, g.chunk_bytes, blk)
        if not np.array_equal(a, r):
            failing.add(blk)
    assert failing  # the workload does exercise failures
    want = expected_by_scan(b, g.num_blocks, g.block_size, failing)
    got = [(int(o["code"]), int(o["first_failing_block"])) for o in out]
    assert got == want
    # events: one terminal event per outcome, two for a failure, claim order
    term = ev[ev["kind"] >= O.EV_RESTORED]
    assert len(term) == b.num_claims + int((out["code"] == O.RESTORE_FAILED_FAIL_CLOSED).sum())
    assert list(ev["seq"]) == list(range(len(ev)))


def test_modeled_digests_reproduce_real_digest_outcomes():
    """Large pools are checked with real digests only for blocks whose bytes
    change (and a sample); every other block's before/after digests are
    equal placeholders.  On the tiny workload this gives exactly the
    outcomes and events of digesting every block."""
    w = TINY
    b = make_batch(w)
    f = make_faults(w, b)
    f = FaultSpec(f.flip_blocks, f.flip_bits, np.array([int(b.block_ids[7])], np.uint32))
    _, out_real, ev_real, _, _ = oracle_lifecycle(w, b, f)
    m0, m1 = modeled_digests(w, f, blocks_needed=[])
    op = O.OraclePool(w.geometry.num_blocks, w.geometry.block_size, w.seed)
    op.offload(b, m0)
    op.restore(b, f.load_failed)
    out_mod = op.check(b, m1)
    assert np.array_equal(out_real, out_mod)
    assert np.array_equal(ev_real, op.events())


@pytest.mark.parametrize("w", [TINY, scaled(FULL["llama3-70b"], 24, 40, missing_claim_rate=0.1),
                               scaled(FULL["small-claim-stress"], 256, 30000)],
                         ids=lambda w: w.name)
def test_event_log_follows_the_lifecycle_at_scale(w):
    """The oracle's event log over a whole workload, checked against the
    paper's lifecycle order by a validator written from the paper alone
    (tests.helpers.validate_lifecycle): consecutive sequence numbers,
    ACCEPTED (+ OFFLOADED) in batch order, RESTORE_REQUIRED for the
    offloaded claims, one terminal outcome per claim that agrees with its
    code, the claim itself as the blocking id."""
    from tests.helpers import modeled_digests, validate_lifecycle

    b = make_batch(w)
    f = make_faults(w, b)
    d0, d1 = modeled_digests(w, f, [])
    op = O.OraclePool(w.geometry.num_blocks, w.geometry.block_size, w.seed)
    assert op.offload(b, d0) == O.OK
    assert op.restore(b, f.load_failed) == O.OK
    pre = op.events(clear=True)
    out = op.check(b, d1)
    validate_lifecycle(b, pre, op.events(), out)
    assert len(set(out["code"].tolist())) >= 2


@pytest.mark.parametrize("seed", range(4))
def test_mutation_controls_oracle(seed):
    """The oracle on the mutation controls (clean restore, then each claim
    presented with its footprint order, a token, an entry or an offload
    record changed): every outcome equals the one the mutation alone
    predicts (UNKNOWN at the mutated position, else MATERIALIZED)."""
    from paper_2606_01387_amd.synth import content
    from tests.test_gpu_attribution import MUTATIONS, mutated, seeded

    w, batch, _ = seeded(100 + seed)
    g = w.geometry
    unref = np.setdiff1d(np.arange(g.num_blocks), batch.unique_blocks(g.num_blocks))
    pres, expected, kinds = mutated(batch, unref, np.random.default_rng(seed), g.block_size)
    assert all(kinds.count(k) >= 10 for k in MUTATIONS)
    host = content.pool_host(g, w.content_seed)
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    assert op.offload(batch, digests(host, w)) == O.OK
    assert op.restore(batch) == O.OK
    out = op.check(pres, digests(host, w))
    assert [(int(a), int(b)) for a, b in zip(out["code"], out["first_failing_block"])] == expected


def test_fuzz_cases_run_on_the_oracle():
    """The irregular lifecycles the GPU differential test replays run on the
    oracle with every offload accepted, and mix all three outcomes."""
    from paper_2606_01387_amd.synth import content
    from tests.fuzz_cases import SEEDS, make_case

    codes = np.zeros(3, dtype=np.int64)
    for seed in SEEDS:
        case = make_case(seed)
        w, g = case.w, case.w.geometry
        host = content.pool_host(g, w.content_seed)
        op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
        for i, b in enumerate(case.offload):
            if i == 1:
                assert op.restore(case.mid, case.mid_faults.load_failed) == O.OK
                host = apply_flips(host, w, case.mid_faults)
            assert op.offload(b, digests(host, w)) == O.OK
        assert op.restore(case.restore, case.faults.load_failed) == O.OK
        op.events(clear=True)
        out = op.check(case.check, digests(apply_flips(host, w, case.faults), w))
        assert out.size == case.check.num_claims
        failed = int((out["code"] == O.RESTORE_FAILED_FAIL_CLOSED).sum())
        assert op.events().size == out.size + failed
        codes += np.bincount(out["code"], minlength=3)
    assert (codes > 20).all(), codes


@pytest.mark.parametrize("seed", range(80))
def test_sequences_follow_the_claim_ledger(seed):
    """The oracle over the multi-step lifecycles the GPU differential test
    replays (tests/fuzz_cases.make_sequence): at every check, each claim that
    was offloaded whole, restored since, and is presented as accepted has
    the outcome a byte ledger gives, with no digest: it fails closed at the
    first position inside its predicate whose bytes differ from its own
    offload-time copy, or whose block had a load failure reported by a later
    restore; otherwise it is materialized (section 5 storage_restorability;
    Table 9; section 1 predicate)."""
    from tests.fuzz_cases import make_sequence

    seq = make_sequence(seed)
    w, g = seq.w, seq.w.geometry
    bs = g.block_size
    host = host_pool(w).copy()
    op = O.OraclePool(g.num_blocks, bs, w.seed)
    ledger = {}  # id -> (blocks, tokens, copies, call, pred_blocks, offloaded)
    restored = set()
    reports = []
    judged = 0
    for call, st in enumerate(seq.steps):
        b = st.batch
        if st.kind == "offload":
            assert op.offload(b, digests(host, w)) == O.OK
            for c in range(b.num_claims):
                cid, blks, tk = b.claim(c)
                n = len(blks)
                whole = n > 0 and (blks < g.num_blocks).all() and n == -(-len(tk) // bs)
                k = None if b.predicate_tokens is None else int(b.predicate_tokens[c])
                pred = n if k is None else min(n, -(-k // bs))
                copies = [O.canonical_block(host, g.planes, g.num_blocks, g.chunk_bytes, int(x)).copy()
                          if x < g.num_blocks else None for x in blks]
                ledger[int(cid)] = (blks.copy(), tk.copy(), copies, call, pred, whole)
        elif st.kind == "restore":
            assert op.restore(b, st.faults.load_failed) == O.OK
            host = apply_flips(host, w, st.faults)
            reports += [(int(x), call) for x in st.faults.load_failed]
            restored |= {int(x) for x in b.claim_ids if int(x) in ledger and ledger[int(x)][5]}
        elif st.kind == "check":
            out = op.check(b, digests(host, w))
            for c in range(b.num_claims):
                cid, blks, tk = b.claim(c)
                cid = int(cid)
                if cid not in ledger or cid not in restored:
                    continue
                a_blks, a_tk, copies, at, pred, _ = ledger[cid]
                if not (np.array_equal(blks, a_blks) and np.array_equal(tk, a_tk)):
                    continue
                bad = [j for j in range(pred)
                       if any(rb == int(a_blks[j]) and rc > at for rb, rc in reports)
                       or not np.array_equal(O.canonical_block(host, g.planes, g.num_blocks,
                                                               g.chunk_bytes, int(a_blks[j])), copies[j])]
                o = out[c]
                if bad:
                    assert (int(o["code"]), int(o["first_failing_block"])) == \
                        (O.RESTORE_FAILED_FAIL_CLOSED, bad[0]), (seed, call, cid, bad)
                else:
                    assert o["code"] == O.MATERIALIZED, (seed, call, cid)
                judged += 1
        else:
            op.lookup(b)
    assert judged > 0
