"""Differential test of the library against the oracle over seeded irregular
lifecycles (tests/fuzz_cases.py): five pool geometries (one a head shard, one
whose digest runs in four phases), offload batches with empty, long, missing,
out-of-range, malformed and entry-sharing rows, reserved ids and predicates,
shared and duplicate-owned identities, faults, a partial restore (in a third
of the cases from device staging, after the staged blocks' device copies are
zeroed: staging written by the second offload into a new buffer, or by both
offloads into one buffer, which accumulates and so keeps the first offload's
bytes of blocks the second does not restage), a check batch that presents the
claims again reordered, repeated and changed, and lookups; between the two
offloads a restore of first-batch claims reports load failures and flips
bytes of their blocks, which the second batch re-offloads under another
claim. The pool's bytes after the restore must equal the host model, and
every status, outcome field, event, per-block digest, lookup field and
identity count the oracle's."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_01387_amd.synth import content
from tests.fuzz_cases import SEEDS, capacities, make_case, well_formed_blocks
from tests.helpers import apply_flips, digests
from tests.test_gpu_parity import free_gpu, gpu_pool_tensor, same_events, same_outcomes

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seed", SEEDS)
def test_fuzz_lifecycle(torch, ck, seed):
    case = make_case(seed)
    w = case.w
    g = w.geometry
    print(f"fuzz seed {seed} ({case.size}{', staged' if case.staged else ''}): heads {g.num_kv_heads}/{g.total_kv_heads or g.num_kv_heads}, "
          f"offload {[b.num_claims for b in case.offload]}, check {case.check.num_claims}, "
          f"lookup {case.lookup.num_claims}", flush=True)
    host = content.pool_host(g, w.content_seed)
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    kv = gpu_pool_tensor(torch, w)
    # staged cases alternate: the second offload stages into a new buffer,
    # or both offloads stage into one buffer, which accumulates
    accumulate = case.staged and (seed // 3) % 2 == 1
    staging = None
    if accumulate:
        slots = sum(well_formed_blocks(b, g.num_blocks).size for b in case.offload)
        staging = torch.empty(max(1, slots) * g.block_bytes, dtype=torch.uint8, device="cuda")
    snap = {}  # block -> its bytes at its latest staged offload (its staged copy)
    print(f"  mid restore {case.mid.num_claims} claims, {case.mid_faults.flip_blocks.size} flips, "
          f"{case.mid_faults.load_failed.size} load failures{', one staging buffer' if accumulate else ''}",
          flush=True)
    with ck.Pool(g, w.seed, kv, **capacities(case)) as pool:
        for i, b in enumerate(case.offload):
            if i == 1:  # the restore between the offloads: failures, changed bytes
                pool.restore(ck.DeviceBatch(case.mid), faults=case.mid_faults)
                assert op.restore(case.mid, case.mid_faults.load_failed) == O.OK
                host = apply_flips(host, w, case.mid_faults)
            want = op.offload(b, digests(host, w))
            blocks = well_formed_blocks(b, g.num_blocks)
            use = None
            if accumulate:
                use = staging
            elif case.staged and i == len(case.offload) - 1:
                staging = torch.empty(max(1, blocks.size) * g.block_bytes, dtype=torch.uint8,
                                      device="cuda")
                use = staging
            try:
                pool.offload(ck.DeviceBatch(b), staging=use)
                got = ck.OK
            except ck.ClaimError as e:
                got = e.status
            assert got == want
            if got == ck.OK:
                if use is not None and not accumulate:
                    snap = {}  # a new buffer: a new staging generation
                host3 = host.reshape(g.planes, g.num_blocks, g.chunk_bytes)
                for blk in blocks.tolist():
                    if use is not None:
                        snap[blk] = host3[:, blk, :].copy()
                    else:
                        snap.pop(blk, None)  # an unstaged offload drops the staged copy
        restored = host.copy()
        if case.staged:
            # the staged blocks' device copies are gone; the restore copies
            # back, from their staged copies, those its well-formed rows
            # reference
            staged = np.array(sorted(snap), dtype=np.int64)
            pool.stream.synchronize()
            idx = torch.as_tensor(staged, device="cuda")
            kv.view(g.planes, g.num_blocks, g.chunk_bytes)[:, idx, :] = 0
            torch.cuda.synchronize()
            r3 = restored.reshape(g.planes, g.num_blocks, g.chunk_bytes)
            r3[:, staged, :] = 0
            for blk in np.intersect1d(staged, well_formed_blocks(case.restore, g.num_blocks)).tolist():
                r3[:, blk, :] = snap[blk]
        pool.restore(ck.DeviceBatch(case.restore), staging=staging, faults=case.faults)
        assert op.restore(case.restore, case.faults.load_failed) == O.OK
        restored = apply_flips(restored, w, case.faults)
        pool.stream.synchronize()
        assert np.array_equal(kv.cpu().numpy(), restored)
        _, ev_pre = pool.read(max_outcomes=1)
        same_events(ev_pre, op.events(clear=True))
        pool.check(ck.DeviceBatch(case.check))
        out, ev = pool.read()
        same_outcomes(out, op.check(case.check, digests(restored, w)))
        same_events(ev, op.events(clear=True))
        st = pool.block_state()
        for f, v in op.block_state().items():
            assert np.array_equal(st[f], v), f
        got = pool.lookup(ck.DeviceBatch(case.lookup))
        want = op.lookup(case.lookup)
        for f in want.dtype.names:
            if f != "pad":
                assert np.array_equal(got[f], want[f]), f
        assert pool.identity_stats() == op.identity_stats()
    del kv, staging
    free_gpu(torch)
