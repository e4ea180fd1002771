"""Multi-step lifecycles on the GPU against the oracle, step by step
(tests/fuzz_cases.make_sequence): several offloads over a few hot blocks
(claims sharing blocks, re-offloading blocks whose loads failed or whose
bytes changed, registering other prefixes in them; predicates), restores
of random subsets with reported failures and bit flips, some undoing
earlier flips (recomputes), checks of random subsets presented as accepted
or changed, and lookups. In half of the sequences the offloads stage into
one staging buffer (device or page-locked host memory), which accumulates
(some offloads unstaged, which drops their blocks' staged copies, and an
occasional staging reset), and some restores first lose the device copies
of staged blocks and copy them back from their latest staged bytes. After
every step the pool bytes equal the host model; every check's outcomes and
events, every lookup and the identity counts, and at the end the per-block
state, equal the oracle's."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_01387_amd.synth import content
from tests.fuzz_cases import SEQUENCE_SEEDS, make_sequence, well_formed_blocks
from tests.helpers import apply_flips, digests
from tests.test_gpu_parity import free_gpu, gpu_pool_tensor, same_events, same_outcomes

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seed", SEQUENCE_SEEDS)
def test_lifecycle_sequence(torch, ck, seed):
    seq = make_sequence(seed)
    w, g = seq.w, seq.w.geometry
    print(f"sequence {seed}: {''.join(s.kind[0] for s in seq.steps)}, {seq.claims} claims, "
          f"{g.num_blocks} blocks", flush=True)
    host = content.pool_host(g, w.content_seed)
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    kv = gpu_pool_tensor(torch, w)
    rng = np.random.default_rng(90_000 + seed)
    arena = None
    if rng.random() < 0.5:  # one staging buffer for the whole sequence
        slots = sum(well_formed_blocks(st.batch, g.num_blocks).size
                    for st in seq.steps if st.kind == "offload")
        if rng.random() < 0.5:
            arena = torch.empty(max(1, slots) * g.block_bytes, dtype=torch.uint8, device="cuda")
        else:  # page-locked host memory, which the kernels write and read over the link
            arena = torch.empty(max(1, slots) * g.block_bytes, dtype=torch.uint8, pin_memory=True)
    snap = {}  # block -> its bytes at its latest staged offload
    with ck.Pool(g, w.seed, kv, max_claims=4 * seq.claims + 64, max_footprint=4 * seq.refs + 64,
                 event_capacity=64 * seq.claims + 1024) as pool:
        for st in seq.steps:
            db = ck.DeviceBatch(st.batch)
            if st.kind == "offload":
                stage = arena is not None and rng.random() < 0.6
                if stage and rng.random() < 0.15:
                    pool.staging_reset()
                    snap = {}
                pool.offload(db, staging=arena if stage else None)
                assert op.offload(st.batch, digests(host, w)) == O.OK
                h3 = host.reshape(g.planes, g.num_blocks, g.chunk_bytes)
                for blk in well_formed_blocks(st.batch, g.num_blocks).tolist():
                    if stage:
                        snap[blk] = h3[:, blk, :].copy()
                    else:
                        snap.pop(blk, None)
            elif st.kind == "restore":
                from_staging = arena is not None and snap and rng.random() < 0.5
                if from_staging:
                    # some staged blocks lose their device copies first
                    staged = np.array(sorted(snap), dtype=np.int64)
                    gone = staged[rng.random(staged.size) < 0.5]
                    pool.stream.synchronize()
                    kv.view(g.planes, g.num_blocks, g.chunk_bytes)[
                        :, torch.as_tensor(gone, device="cuda"), :] = 0
                    torch.cuda.synchronize()
                    h3 = host.reshape(g.planes, g.num_blocks, g.chunk_bytes)
                    h3[:, gone, :] = 0
                    for blk in np.intersect1d(staged, well_formed_blocks(st.batch, g.num_blocks)).tolist():
                        h3[:, blk, :] = snap[blk]
                pool.restore(db, staging=arena if from_staging else None, faults=st.faults)
                assert op.restore(st.batch, st.faults.load_failed) == O.OK
                host = apply_flips(host, w, st.faults)
            elif st.kind == "check":
                pool.check(db)
                out, ev = pool.read()
                same_outcomes(out, op.check(st.batch, digests(host, w)))
                want_ev = op.events(clear=True)
                same_events(ev, want_ev)
            else:
                got = pool.lookup(db)
                want = op.lookup(st.batch)
                for f in want.dtype.names:
                    if f != "pad":
                        assert np.array_equal(got[f], want[f]), f
                assert pool.identity_stats() == op.identity_stats()
        pool.stream.synchronize()
        assert np.array_equal(kv.cpu().numpy(), host)
        stb = pool.block_state()
        for f, v in op.block_state().items():
            assert np.array_equal(stb[f], v), f
    del kv
    free_gpu(torch)
