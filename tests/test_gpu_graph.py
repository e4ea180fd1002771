"""claim_check_static captured into a HIP graph and replayed (the callers
it serves include code under graph capture): every replay, with eager work
and synchronizations between replays, must give the eager call's outcomes
and events; and replays that the host cannot bound must never write past
the event log: a replay whose events do not fit appends none, and the next
outcomes_read reports it (CLAIM_ENOSPC) with the events that fit intact."""

import ctypes

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_01387_amd.synth import FULL, content, make_batch, make_faults, scaled
from tests.helpers import apply_flips, digests
from tests.test_gpu_parity import free_gpu, gpu_pool_tensor, note, same_outcomes

pytestmark = pytest.mark.gpu

EV_FIELDS = ("claim_id", "aux", "kind", "block_index", "phys_block")
CAPTURE_RELAXED = 2  # hipStreamCaptureModeRelaxed


@pytest.fixture(scope="module")
def hip():
    h = ctypes.CDLL("libamdhip64.so")
    vp = ctypes.c_void_p
    h.hipStreamBeginCapture.argtypes = [vp, ctypes.c_int]
    h.hipStreamEndCapture.argtypes = [vp, ctypes.POINTER(vp)]
    h.hipGraphInstantiate.argtypes = [ctypes.POINTER(vp), vp, vp, ctypes.c_char_p, ctypes.c_size_t]
    h.hipGraphLaunch.argtypes = [vp, vp]
    h.hipGraphExecDestroy.argtypes = [vp]
    h.hipGraphDestroy.argtypes = [vp]
    return h


def same_events_but_seq(got, want, seq_shift):
    assert got.size == want.size, (got.size, want.size)
    for f in EV_FIELDS:
        assert np.array_equal(got[f], want[f]), f
    assert np.array_equal(got["seq"], want["seq"] + np.uint64(seq_shift))


@pytest.mark.parametrize("claims", [1500, 6000], ids=["one-workgroup-events", "tiled-events"])
def test_check_static_graph_replays(torch, ck, hip, claims):
    w = scaled(FULL["small-claim-stress"], 256, claims, corrupt_rate=0.05, num_load_failed=2)
    g = w.geometry
    batch = make_batch(w)
    faults = make_faults(w, batch)
    C = batch.num_claims
    # the oracle first: its outcomes, and the events one check appends
    host = content.pool_host(g, w.content_seed)
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    op.offload(batch, digests(host, w))
    op.restore(batch, faults.load_failed)
    want = op.check(batch, digests(apply_flips(host, w, faults), w))
    E = C + int((want["code"] == O.RESTORE_FAILED_FAIL_CLOSED).sum())
    cap = 2 * E + E // 2  # two checks' events fit, three do not
    note(f"graph replays: {C} claims, {E} events per check, log of {cap}")
    kv = gpu_pool_tensor(torch, w)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    db = ck.DeviceBatch(batch)
    buf = torch.empty(C * ck.OUTCOME_DTYPE.itemsize, dtype=torch.uint8, device="cuda")

    def outcomes():
        return buf.cpu().numpy().view(ck.OUTCOME_DTYPE)[:C].copy()

    with ck.Pool(g, w.seed, kv, stream=s, max_claims=2 * C, max_footprint=2 * batch.num_refs,
                 event_capacity=cap) as pool:
        pool.offload(db)
        pool.read(max_outcomes=1)
        pool.restore(db, faults=faults)
        pool.read(max_outcomes=1)
        pool.check_static(db, out=buf)
        s.synchronize()
        ref = outcomes()
        same_outcomes(ref, want)
        _, ev_ref = pool.read()
        assert ev_ref.size == E

        graph, gexec = ctypes.c_void_p(), ctypes.c_void_p()
        assert hip.hipStreamBeginCapture(ctypes.c_void_p(s.cuda_stream), CAPTURE_RELAXED) == 0
        try:
            pool.check_static(db, out=buf)
        finally:
            rc_end = hip.hipStreamEndCapture(ctypes.c_void_p(s.cuda_stream), ctypes.byref(graph))
        assert rc_end == 0 and graph.value
        assert hip.hipGraphInstantiate(ctypes.byref(gexec), graph, None, None, 0) == 0
        try:
            for r in range(3):  # eager work and a synchronization between replays
                buf.zero_()
                torch.cuda.synchronize()
                assert hip.hipGraphLaunch(gexec, ctypes.c_void_p(s.cuda_stream)) == 0
                s.synchronize()
                same_outcomes(outcomes(), ref)
                _, ev = pool.read()
                same_events_but_seq(ev, ev_ref, (r + 1) * E)
                note(f"  replay {r}: outcomes and {ev.size} events equal the eager call's")
            # three replays without reading the log: the third's events do not fit
            for _ in range(3):
                assert hip.hipGraphLaunch(gexec, ctypes.c_void_p(s.cuda_stream)) == 0
            s.synchronize()
            same_outcomes(outcomes(), ref)  # outcomes are written whatever the log holds
            evs = np.zeros(cap, ck.EVENT_DTYPE)
            n_ev = ctypes.c_uint64()
            rc = ck.lib().outcomes_read(pool._h, None, 0, None, evs.ctypes.data, evs.size,
                                        ctypes.byref(n_ev))
            assert rc == ck.ENOSPC
            assert n_ev.value == 2 * E
            same_events_but_seq(evs[:E], ev_ref, 4 * E)
            same_events_but_seq(evs[E:2 * E], ev_ref, 5 * E)
            note(f"  third replay of {E} events dropped; log held {n_ev.value}, reported ENOSPC")
            # the read cleared the mark: the next replay appends as usual
            assert hip.hipGraphLaunch(gexec, ctypes.c_void_p(s.cuda_stream)) == 0
            s.synchronize()
            _, ev = pool.read()
            same_events_but_seq(ev, ev_ref, 6 * E)
        finally:
            hip.hipGraphExecDestroy(gexec)
            hip.hipGraphDestroy(graph)
    del kv, buf
    free_gpu(torch)
