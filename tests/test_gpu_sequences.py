"""Multi-step lifecycles on the GPU against the oracle, step by step
(tests/fuzz_cases.make_sequence): several offloads over a few hot blocks
(claims sharing blocks, re-offloading blocks whose loads failed or whose
bytes changed, registering other prefixes in them; predicates), restores
of random subsets with reported failures and bit flips, some undoing
earlier flips (recomputes), checks of random subsets presented as accepted
or changed, and lookups.  After every step the pool bytes equal the host
model; every check's outcomes and events, every lookup and the identity
counts, and at the end the per-block state, equal the oracle's."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_01387_amd.synth import content
from tests.fuzz_cases import SEQUENCE_SEEDS, make_sequence
from tests.helpers import apply_flips, digests
from tests.test_gpu_parity import free_gpu, gpu_pool_tensor, same_events, same_outcomes

pytestmark = pytest.mark.gpu


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


@pytest.mark.parametrize("seed", SEQUENCE_SEEDS)
def test_lifecycle_sequence(torch, ck, seed):
    seq = make_sequence(seed)
    w, g = seq.w, seq.w.geometry
    print(f"sequence {seed}: {''.join(s.kind[0] for s in seq.steps)}, {seq.claims} claims, "
          f"{g.num_blocks} blocks", flush=True)
    host = content.pool_host(g, w.content_seed)
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    kv = gpu_pool_tensor(torch, w)
    with ck.Pool(g, w.seed, kv, max_claims=4 * seq.claims + 64, max_footprint=4 * seq.refs + 64,
                 event_capacity=64 * seq.claims + 1024) as pool:
        for st in seq.steps:
            db = ck.DeviceBatch(st.batch)
            if st.kind == "offload":
                pool.offload(db)
                assert op.offload(st.batch, digests(host, w)) == O.OK
            elif st.kind == "restore":
                pool.restore(db, faults=st.faults)
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
