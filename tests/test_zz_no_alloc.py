"""claim_check_static, the check that allocates nothing, through the C ABI
against claim_check on the same pool and batches (and the oracle): two
calls in a row, the second with a smaller batch, so the fixed scratch holds
the first call's larger contents when the second runs.  Outcomes must be
equal field by field, and the events each call appends equal claim_check's
(apart from their global sequence numbers, which keep counting)."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_01387_amd.synth import FULL, from_claims, make_batch, make_faults, scaled
from tests.helpers import apply_flips, digests
from tests.test_gpu_parity import free_gpu, gpu_pool_tensor, note, same_events, same_outcomes

pytestmark = pytest.mark.gpu

EV_FIELDS = ("claim_id", "aux", "kind", "block_index", "phys_block")


def test_check_static_matches_check(torch, ck):
    # 20000 claims (the tiled event scan), then 3000 of them (one workgroup)
    w = scaled(FULL["small-claim-stress"], 256, 20000, corrupt_rate=0.05, num_load_failed=3)
    g = w.geometry
    batch = make_batch(w)
    faults = make_faults(w, batch)
    small = from_claims([batch.claim(c) for c in range(0, 6000, 2)])
    note(f"check_static: {batch.num_claims} then {small.num_claims} claims over {g.num_blocks} blocks")
    kv = gpu_pool_tensor(torch, w)
    with ck.Pool(g, w.seed, kv, max_claims=2 * batch.num_claims, max_footprint=4 * batch.num_refs,
                 event_capacity=8 * batch.num_claims) as pool:
        db = ck.DeviceBatch(batch)
        pool.offload(db)
        pool.restore(db, faults=faults)
        pool.read()
        results = []
        for b in (batch, small):
            d = ck.DeviceBatch(b)
            pool.check(d)
            want, want_ev = pool.read()
            out = pool.check_static(d)
            got_none, got_ev = pool.read()
            assert got_none.size == 0  # the outcomes are in `out`
            got = out.cpu().numpy().view(ck.OUTCOME_DTYPE)[: b.num_claims].copy()
            same_outcomes(got, want)
            assert got_ev.size == want_ev.size
            for f in EV_FIELDS:
                assert np.array_equal(got_ev[f], want_ev[f]), f
            assert np.array_equal(got_ev["seq"], want_ev["seq"] + want_ev.size)
            results.append((b, got, got_ev))
            note(f"  {b.num_claims} claims: outcomes and {got_ev.size} events equal claim_check's")
        # sizes past the fixed scratch, or an output too small, queue nothing
        big = ck.DeviceBatch(from_claims([(i + 1, [], np.zeros(0, np.uint32))
                                          for i in range(ck.STATIC_MAX_CLAIMS + 1)]))
        with pytest.raises(ck.ClaimError) as e:
            pool.check_static(big)
        assert e.value.status == ck.ELIMIT
        tiny_out = torch.empty(64 * 10, dtype=torch.uint8, device="cuda")
        with pytest.raises(ck.ClaimError) as e:
            pool.check_static(ck.DeviceBatch(small), out=tiny_out)
        assert e.value.status == ck.ENOSPC
        _, ev_after = pool.read()
        assert ev_after.size == 0
    # and the oracle agrees with both
    from paper_2606_01387_amd.synth import content
    host = content.pool_host(g, w.content_seed)
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    op.offload(batch, digests(host, w))
    op.restore(batch, faults.load_failed)
    d1 = digests(apply_flips(host, w, faults), w)
    for b, got, _ in results:
        op.events(clear=True)
        same_outcomes(got, op.check(b, d1))
    del kv
    free_gpu(torch)


def test_check_static_at_its_limit(torch, ck):
    # exactly CLAIM_STATIC_MAX_CLAIMS claims: every byte of the fixed scratch
    w = scaled(FULL["small-claim-stress"], 256, ck.STATIC_MAX_CLAIMS, corrupt_rate=0.05,
               num_load_failed=3)
    g = w.geometry
    batch = make_batch(w)
    faults = make_faults(w, batch)
    assert batch.num_claims == ck.STATIC_MAX_CLAIMS
    note(f"check_static at its limit: {batch.num_claims} claims over {g.num_blocks} blocks")
    kv = gpu_pool_tensor(torch, w)
    with ck.Pool(g, w.seed, kv, max_claims=2 * batch.num_claims, max_footprint=2 * batch.num_refs,
                 event_capacity=6 * batch.num_claims) as pool:
        db = ck.DeviceBatch(batch)
        pool.offload(db)
        pool.restore(db, faults=faults)
        pool.read()
        pool.check(db)
        want, want_ev = pool.read()
        out = pool.check_static(db)
        _, got_ev = pool.read()
        got = out.cpu().numpy().view(ck.OUTCOME_DTYPE)[: batch.num_claims].copy()
        same_outcomes(got, want)
        assert got_ev.size == want_ev.size
        for f in EV_FIELDS:
            assert np.array_equal(got_ev[f], want_ev[f]), f
        codes = np.bincount(got["code"], minlength=3)
        note(f"  outcomes unknown/materialized/failed = {codes.tolist()}, {got_ev.size} events")
        assert codes[1] and codes[2]
    del kv
    free_gpu(torch)


def test_check_static_empty_batch(torch, ck):
    # no claims: nothing to write, no events, and the log stays as it was
    w = scaled(FULL["small-claim-stress"], 64, 8)
    kv = gpu_pool_tensor(torch, w)
    with ck.Pool(w.geometry, w.seed, kv, max_claims=64, max_footprint=256,
                 event_capacity=256) as pool:
        empty = ck.DeviceBatch(from_claims([]))
        out = pool.check_static(empty)
        got, ev = pool.read()
        assert got.size == 0 and ev.size == 0
        assert out.numel() >= ck.OUTCOME_DTYPE.itemsize
    del kv
    free_gpu(torch)
