"""The C boundary on its own: a plain C99 program (tests/c_abi/lifecycle.c)
creates a pool over hipMalloc'd memory on the default stream and runs
offload, restore (with bit flips and reported load failures), check and
outcomes_read through libclaimkv.so, with no Python or PyTorch in its
process.  Its outcomes and events must equal the oracle's."""

import os
import struct
import subprocess

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_01387_amd.synth import FULL, TINY, content, make_batch, make_faults, scaled
from tests.helpers import apply_flips, digests

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLIENT = os.path.join(ROOT, "tests", "c_abi", "lifecycle")
OUT_FIELDS = [n for n in O.OUTCOME_DTYPE.names if n != "pad"]
EV_FIELDS = [n for n in O.EVENT_DTYPE.names if n != "pad"]


def write_input(path, w, batch, faults, pool):
    g = w.geometry
    with open(path, "wb") as f:
        f.write(struct.pack("<7I", g.num_layers, g.planes_per_layer, g.block_size, g.num_kv_heads,
                            g.head_dim, g.elem_bytes, g.num_blocks))
        f.write(struct.pack("<2Q", w.seed, pool.size))
        f.write(pool.tobytes())
        f.write(struct.pack("<I2Q", batch.num_claims, batch.num_refs, batch.num_tokens))
        for a, dt in ((batch.claim_ids, "<u8"), (batch.block_offsets, "<u4"), (batch.block_ids, "<u4"),
                      (batch.token_offsets, "<u8"), (batch.tokens, "<u4")):
            f.write(np.ascontiguousarray(a, dtype=dt).tobytes())
        f.write(struct.pack("<2I", faults.flip_blocks.size, faults.load_failed.size))
        f.write(np.ascontiguousarray(faults.flip_blocks, "<u4").tobytes())
        f.write(np.ascontiguousarray(faults.flip_bits, "<u8").tobytes())
        f.write(np.ascontiguousarray(faults.load_failed, "<u4").tobytes())


@pytest.mark.parametrize("w", [TINY, scaled(FULL["small-claim-stress"], 256, 3000, corrupt_rate=0.05,
                                            num_load_failed=3)], ids=lambda w: w.name)
def test_c_client_lifecycle(tmp_path, w):
    assert os.path.exists(CLIENT), f"{CLIENT} is not built: run __graft_entry__.build()"
    g = w.geometry
    batch = make_batch(w)
    faults = make_faults(w, batch)
    pool = content.pool_host(g, w.content_seed)
    inp, outp = tmp_path / "in.bin", tmp_path / "out.bin"
    write_input(inp, w, batch, faults, pool)
    print(f"C client on {w.name}: {batch.num_claims} claims", flush=True)
    run = subprocess.run([CLIENT, str(inp), str(outp)], capture_output=True, text=True, timeout=120)
    print(run.stdout.strip(), run.stderr.strip()[-400:], flush=True)
    assert run.returncode == 0
    raw = outp.read_bytes()
    status = struct.unpack_from("<5i", raw, 0)
    assert status == (0, 0, 0, 0, 0), status
    n_out, n_ev = struct.unpack_from("<IQ", raw, 20)
    at = 32
    got = np.frombuffer(raw, O.OUTCOME_DTYPE, n_out, at)
    ev = np.frombuffer(raw, O.EVENT_DTYPE, n_ev, at + 64 * n_out)
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    assert op.offload(batch, digests(pool, w)) == O.OK
    assert op.restore(batch, faults.load_failed) == O.OK
    op.events(clear=True)
    want = op.check(batch, digests(apply_flips(pool, w, faults), w))
    want_ev = op.events()
    assert n_out == batch.num_claims and n_ev == want_ev.size
    for f in OUT_FIELDS:
        assert np.array_equal(got[f], want[f]), f
    for f in EV_FIELDS:
        assert np.array_equal(ev[f], want_ev[f]), f
    assert (got["code"] == O.RESTORE_FAILED_FAIL_CLOSED).any() and (got["code"] == O.MATERIALIZED).any()
