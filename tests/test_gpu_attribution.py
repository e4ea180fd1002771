"""Claim attribution and false-positive controls at scale, on the GPU.

The paper's section 7 path C and its Table 8 / Table 9 controls as a
property test over many seeded pools: each pool has silently corrupted
blocks (referenced or not), reported load failures, flips that cancel, and
blocks no claim references.  For every seed the GPU result must equal the
oracle's bit for bit, and the outcomes must satisfy the paper's attribution
rules against a failing set computed by comparing bytes:

* a claim fails closed iff one of its own blocks is in the failing set
  (target-only attribution; unclaimed and wrong-claim failures never count);
* every ACTIVE_REQUEST_REFUSED names its own claim as the blocking claim and
  follows that claim's RESTORATION_FAILED;
* a claim none of whose blocks failed is MATERIALIZED (generic failure
  elsewhere in the pool does not touch it).
"""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_01387_amd.synth import FaultSpec, Geometry, Workload, content, make_batch, make_faults
from tests.helpers import apply_flips, digests
from tests.test_gpu_parity import free_gpu

pytestmark = pytest.mark.gpu


def seeded(seed):
    w = Workload(
        name=f"attribution-{seed}", geometry=Geometry(2, 2, 16, 2, 32, 2, 400), seed=9000 + seed,
        num_claims=120, length=("blocks", 1, 6, True), sharing=("zipf", 1.2, 6),
        corrupt_rate=0.05, num_load_failed=4, gen_seed=seed * 31 + 1, content_seed=seed * 17 + 3)
    batch = make_batch(w)
    f = make_faults(w, batch)
    rng = np.random.default_rng(seed)
    # a flip applied twice cancels; a second flip in an already corrupted block
    b0, bit0 = int(f.flip_blocks[0]), int(rng.integers(0, 8 * w.geometry.block_bytes))
    # and one flip in a block no claim references (an unclaimed failure)
    unref = np.setdiff1d(np.arange(w.geometry.num_blocks), batch.unique_blocks(w.geometry.num_blocks))
    assert unref.size, "the pool must have unreferenced blocks"
    bu = int(rng.choice(unref))
    blocks = np.concatenate([f.flip_blocks, [b0, b0, bu]]).astype(np.uint32)
    bits = np.concatenate([f.flip_bits, [bit0, bit0, 12345]]).astype(np.uint64)
    return w, batch, FaultSpec(blocks, bits, f.load_failed)


@pytest.mark.parametrize("seed", range(12))
def test_attribution_and_controls(torch, ck, seed):
    w, batch, faults = seeded(seed)
    g = w.geometry
    print(f"attribution seed {seed}: {batch.num_claims} claims, "
          f"{batch.unique_blocks(g.num_blocks).size}/{g.num_blocks} blocks referenced", flush=True)
    kv = torch.empty(g.pool_bytes, dtype=torch.uint8, device="cuda")
    content.fill_pool_gpu(kv.data_ptr(), kv.numel(), g, w.content_seed,
                          torch.cuda.current_stream().cuda_stream)
    db = ck.DeviceBatch(batch)
    with ck.Pool(g, w.seed, kv, max_claims=256, max_footprint=4096, event_capacity=4096) as pool:
        pool.offload(db)
        pool.restore(db, faults=faults)
        pool.read(max_outcomes=1)
        pool.check(db)
        out, ev = pool.read()

    host = content.pool_host(g, w.content_seed)
    restored = apply_flips(host, w, faults)
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    op.offload(batch, digests(host, w))
    op.restore(batch, faults.load_failed)
    op.events(clear=True)
    want = op.check(batch, digests(restored, w))
    for f in want.dtype.names:
        if f != "pad":
            assert np.array_equal(out[f], want[f]), f
    want_ev = op.events()
    for f in ("seq", "claim_id", "aux", "kind", "block_index", "phys_block"):
        assert np.array_equal(ev[f] - (ev["seq"][0] if f == "seq" else 0),
                              want_ev[f] - (want_ev["seq"][0] if f == "seq" else 0)), f

    # failing set by comparing bytes, plus reported failures
    failing = set(int(b) for b in faults.load_failed)
    for b in range(g.num_blocks):
        if not np.array_equal(O.canonical_block(host, g.planes, g.num_blocks, g.chunk_bytes, b),
                              O.canonical_block(restored, g.planes, g.num_blocks, g.chunk_bytes, b)):
            failing.add(b)
    assert int(faults.flip_blocks[0]) in failing  # the cancelled pair left the first flip
    referenced = set(int(b) for b in batch.unique_blocks(g.num_blocks))
    assert failing - referenced, "the seed must also exercise unclaimed failures"

    for c in range(batch.num_claims):
        cid, blks, _ = batch.claim(c)
        own = [j for j, b in enumerate(blks) if int(b) in failing]
        if own:
            assert out[c]["code"] == ck.RESTORE_FAILED_FAIL_CLOSED
            assert out[c]["first_failing_block"] == own[0]
        else:
            assert out[c]["code"] == ck.MATERIALIZED
    failed_ids = {int(x) for x in out["claim_id"][out["code"] == ck.RESTORE_FAILED_FAIL_CLOSED]}
    for i, e in enumerate(ev):
        if e["kind"] == ck.EV_ACTIVE_REQUEST_REFUSED:
            assert int(e["aux"]) == int(e["claim_id"]) and int(e["claim_id"]) in failed_ids
            prev = ev[i - 1]
            assert prev["kind"] == ck.EV_RESTORATION_FAILED and prev["claim_id"] == e["claim_id"]
        if e["kind"] == ck.EV_RESTORATION_FAILED:
            assert int(e["claim_id"]) in failed_ids
    del kv


MUTATIONS = ("none", "swap", "token", "missing", "unrecorded")


def mutated(batch, unref, rng, bs):
    """The claims of `batch` presented again at check time, claim c with
    mutation c mod 5 at a seeded position (when its shape allows it):
    two different block-table entries swapped, one token changed, one entry
    replaced by the missing marker, or one entry replaced by a pool block
    that was never offloaded.  Returns the presented batch and, from the
    mutation alone, each claim's expected (code, first failing block): the
    restore was clean, so a mutation at p makes the claim UNKNOWN at p
    (swap: the first of the two positions; token: its token block)."""
    from paper_2606_01387_amd.synth import MISSING, from_claims

    parts, expected, kinds = [], [], []
    for c in range(batch.num_claims):
        cid, blks, tk = batch.claim(c)
        blks, tk = blks.copy(), tk.copy()
        kind, exp = MUTATIONS[c % len(MUTATIONS)], (1, 0xFFFFFFFF)  # MATERIALIZED
        n = blks.size
        if kind == "swap":
            pairs = [(p, q) for p in range(n) for q in range(p + 1, n) if blks[p] != blks[q]]
            if pairs:
                p, q = pairs[int(rng.integers(len(pairs)))]
                blks[p], blks[q] = blks[q], blks[p]
                exp = (0, p)
            else:
                kind = "none"
        elif kind == "token" and tk.size:
            m = int(rng.integers(tk.size))
            tk[m] = (int(tk[m]) + 1 + int(rng.integers(31999))) % 32000
            exp = (0, m // bs)
        elif kind in ("missing", "unrecorded") and n:
            p = int(rng.integers(n))
            blks[p] = MISSING if kind == "missing" else int(rng.choice(unref))
            exp = (0, p)
        else:
            kind = "none"
        parts.append((cid, blks, tk))
        expected.append(exp)
        kinds.append(kind)
    return from_claims(parts), expected, kinds


@pytest.mark.parametrize("seed", range(4))
def test_mutation_controls(torch, ck, seed):
    """Mutation controls: after a clean offload and restore, every claim is
    checked again with one thing changed (footprint order, a token, a
    missing entry, a block without an offload record).  Each mutated claim
    must fail closed as UNKNOWN at the mutated position and every other
    claim stay MATERIALIZED, with the GPU equal to the oracle bit for bit."""
    w, batch, _ = seeded(100 + seed)
    g = w.geometry
    unref = np.setdiff1d(np.arange(g.num_blocks), batch.unique_blocks(g.num_blocks))
    pres, expected, kinds = mutated(batch, unref, np.random.default_rng(seed), g.block_size)
    print(f"mutation controls seed {seed}: " +
          ", ".join(f"{k} {kinds.count(k)}" for k in MUTATIONS), flush=True)
    kv = torch.empty(g.pool_bytes, dtype=torch.uint8, device="cuda")
    content.fill_pool_gpu(kv.data_ptr(), kv.numel(), g, w.content_seed,
                          torch.cuda.current_stream().cuda_stream)
    db = ck.DeviceBatch(batch)
    with ck.Pool(g, w.seed, kv, max_claims=256, max_footprint=4096, event_capacity=4096) as pool:
        pool.offload(db)
        pool.restore(db)
        pool.read(max_outcomes=1)
        pool.check(ck.DeviceBatch(pres))
        out, ev = pool.read()
    host = content.pool_host(g, w.content_seed)
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    op.offload(batch, digests(host, w))
    op.restore(batch)
    op.events(clear=True)
    want = op.check(pres, digests(host, w))
    for f in want.dtype.names:
        if f != "pad":
            assert np.array_equal(out[f], want[f]), f
    assert [(int(a), int(b)) for a, b in zip(out["code"], out["first_failing_block"])] == expected
    assert all(k != "none" for k, (code, _) in zip(kinds, expected) if code == 0)
    assert sum(k != "none" for k in kinds) >= 0.7 * batch.num_claims
    token = np.array([k == "token" for k in kinds])
    assert (out["reasons"][token] & ck.R_TOKEN_MISMATCH).all()
    assert len(ev) == batch.num_claims  # one terminal event each, none refused
    del kv


@pytest.mark.parametrize("seed", range(8))
def test_attribution_after_reoffload(torch, ck, seed):
    """The controls when blocks are offloaded again (section 5
    storage_restorability row; Table 9 fallback-recompute and wrong-claim
    rows).  Batch A is offloaded, restored with faults and checked; then
    some corrupted blocks are rewritten to their original bytes (a
    recompute), other blocks get new flips, and batch B (new claims)
    re-offloads blocks of A, among them blocks whose load failed; then A
    and B are restored (a few more reported failures) and checked together.
    GPU equals oracle, and every claim's outcome follows a ledger of its own
    offload-time bytes: it fails closed at the first position whose bytes
    now differ from its own offload's, or whose block had a load failure
    reported after its offload; otherwise it is materialized."""
    w, batch_a, faults = seeded(100 + seed)
    g = w.geometry
    rng = np.random.default_rng(seed)
    host0 = content.pool_host(g, w.content_seed)
    after1 = apply_flips(host0, w, faults)
    # the rewrite: cancel half of the first flips (recompute of the original
    # bytes), add new flips on referenced blocks
    half = faults.flip_blocks.size // 2
    ref_a = batch_a.unique_blocks(g.num_blocks)
    new_blocks = rng.choice(ref_a, size=6, replace=False).astype(np.uint32)
    rewrite = FaultSpec(np.concatenate([faults.flip_blocks[:half], new_blocks]).astype(np.uint32),
                        np.concatenate([faults.flip_bits[:half],
                                        rng.integers(0, 8 * g.block_bytes, size=6)]).astype(np.uint64),
                        np.zeros(0, np.uint32))
    after2 = apply_flips(after1, w, rewrite)
    # batch B: new claims over blocks of A (failed, rewritten, others)
    hot = np.unique(np.concatenate([faults.load_failed, faults.flip_blocks, new_blocks])).astype(np.int64)
    rows = []
    for k in range(40):
        n = int(rng.integers(1, 5))
        pick = np.where(rng.random(n) < 0.5, rng.choice(hot, size=n), rng.choice(ref_a, size=n))
        rows.append((int(5_000_000 + k), pick.astype(np.uint32),
                     rng.integers(0, 32000, size=n * g.block_size, dtype=np.uint32)))
    from paper_2606_01387_amd.synth import from_claims
    batch_b = from_claims(rows)
    both = from_claims([batch_a.claim(c) for c in range(batch_a.num_claims)] + rows)
    late_lost = rng.choice(hot, size=2, replace=False).astype(np.uint32)
    final = FaultSpec(np.zeros(0, np.uint32), np.zeros(0, np.uint64), late_lost)
    print(f"re-offload seed {seed}: A {batch_a.num_claims} claims, B {batch_b.num_claims}, "
          f"{half} flips cancelled, 6 new flips, late failures {late_lost.tolist()}", flush=True)

    kv = torch.empty(g.pool_bytes, dtype=torch.uint8, device="cuda")
    content.fill_pool_gpu(kv.data_ptr(), kv.numel(), g, w.content_seed,
                          torch.cuda.current_stream().cuda_stream)
    with ck.Pool(g, w.seed, kv, max_claims=512, max_footprint=8192, event_capacity=8192) as pool:
        pool.offload(ck.DeviceBatch(batch_a))
        pool.restore(ck.DeviceBatch(batch_a), faults=faults)
        pool.check(ck.DeviceBatch(batch_a))
        out1, _ = pool.read()
        pool.restore(ck.DeviceBatch(from_claims([])), faults=rewrite)
        pool.offload(ck.DeviceBatch(batch_b))
        pool.restore(ck.DeviceBatch(both), faults=final)
        pool.read()  # drop the events before the check
        pool.check(ck.DeviceBatch(both))
        out2, ev2 = pool.read()
        pool.stream.synchronize()
        assert np.array_equal(kv.cpu().numpy(), after2)

    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    op.offload(batch_a, digests(host0, w))
    op.restore(batch_a, faults.load_failed)
    want1 = op.check(batch_a, digests(after1, w))
    op.restore(from_claims([]), rewrite.load_failed)
    op.offload(batch_b, digests(after2, w))
    op.restore(both, final.load_failed)
    op.events(clear=True)
    want2 = op.check(both, digests(after2, w))
    for f in want2.dtype.names:
        if f != "pad":
            assert np.array_equal(out1[f], want1[f]), f
            assert np.array_equal(out2[f], want2[f]), f
    want_ev = op.events()
    for f in ("claim_id", "aux", "kind", "block_index", "phys_block"):
        assert np.array_equal(ev2[f], want_ev[f]), f

    # the ledger: call 1 offload A, 2 restore (first failures), 3 rewrite,
    # 4 offload B, 5 restore (late failures)
    reported = [(int(b), 2) for b in faults.load_failed] + [(int(b), 5) for b in late_lost]
    canon = {}

    def block_bytes(pool_bytes, b):
        key = (id(pool_bytes), b)
        if key not in canon:
            canon[key] = O.canonical_block(pool_bytes, g.planes, g.num_blocks, g.chunk_bytes, b)
        return canon[key]

    kinds = {"materialized": 0, "failed_a": 0, "failed_b": 0, "a_kept_failed_after_b": 0}
    b_blocks = set(int(x) for x in batch_b.block_ids)
    for c in range(both.num_claims):
        _, blks, _ = both.claim(c)
        in_a = c < batch_a.num_claims
        snap, at = (host0, 1) if in_a else (after2, 4)
        bad = [j for j, b in enumerate(blks)
               if any(rb == int(b) and rc > at for rb, rc in reported)
               or not np.array_equal(block_bytes(after2, int(b)), block_bytes(snap, int(b)))]
        if bad:
            assert out2[c]["code"] == ck.RESTORE_FAILED_FAIL_CLOSED, (seed, c, bad)
            assert out2[c]["first_failing_block"] == bad[0]
            kinds["failed_a" if in_a else "failed_b"] += 1
            if in_a and int(blks[bad[0]]) in b_blocks:
                kinds["a_kept_failed_after_b"] += 1
        else:
            assert out2[c]["code"] == ck.MATERIALIZED, (seed, c)
            kinds["materialized"] += 1
    print(f"  {kinds}", flush=True)
    assert kinds["a_kept_failed_after_b"] > 0  # B re-offloaded a block A failed on
    del kv
    free_gpu(torch)
