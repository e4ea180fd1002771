"""The digest grid each workload's launches take (claim_digest_grid) on a
256-CU MI355X: one phase for the 13 GB MLA and head-shard pools, two for
the 17 GB 8B and 30 GB stress pools (14 to 32 GiB, split in two at a plane
chunk's edge; one for an odd number of piece groups, and one for an MLA pool
whose halves would end inside a chunk), and for the 105 GB 70B
pool two piece groups at a time in phases of 1.3 GB; the many-plane pools of the parity and fuzz tests, and a
launch of the 70B pool over few blocks, in the phases that keep the grid
full.
The pools are allocated at full size but never read."""

import pytest

from paper_2606_01387_amd.synth import FULL, LLAMA3_70B_TP8, Geometry
from tests.fuzz_cases import GEOMETRIES
from tests.test_gpu_parity import MANY_PLANES, MANY_PLANES_RAGGED, free_gpu, note

pytestmark = pytest.mark.gpu

# (geometry, refs) -> (words per lane, segments, piece groups, slots,
#                      piece groups at a time, workgroups on each)
CASES = [
    ("llama3-8b", FULL["llama3-8b"].geometry, None, (16, 4, 64, 256, 32, 8)),
    ("llama3-70b", FULL["llama3-70b"].geometry, None, (16, 4, 160, 256, 2, 128)),
    ("small-claim-stress", FULL["small-claim-stress"].geometry, None, (16, 2, 28, 256, 14, 18)),
    ("mla-fp8", FULL["mla-fp8"].geometry, None, (24, 3, 46, 256, 46, 5)),
    ("llama3-70b-tp8-shard", LLAMA3_70B_TP8.geometry, None, (8, 1, 40, 512, 40, 12)),
    # the 70B pool under a batch of 300 entries: 1.6 GB, within one phase's
    # bound, read in the two phases that fill the grid
    ("llama3-70b-300-refs", FULL["llama3-70b"].geometry, 300, (16, 4, 160, 256, 80, 3)),
    # 17.1 GB of 36 KiB chunks in three 12 KiB pieces: half of the 46 piece
    # groups would end inside a chunk, so one phase
    ("mla-shaped-17.1GB", Geometry(61, 1, 64, 1, 576, 1, 7600), None, (24, 3, 46, 256, 46, 5)),
    # 15.9 GB in an odd number of piece groups (27): one phase
    ("odd-piece-groups-15.9GB", Geometry(27, 2, 16, 4, 128, 2, 18000), None, (16, 2, 27, 256, 27, 9)),
    (MANY_PLANES.name, MANY_PLANES.geometry, None, (16, 4, 320, 256, 80, 3)),
    (MANY_PLANES_RAGGED.name, MANY_PLANES_RAGGED.geometry, None, (24, 3, 92, 256, 46, 5)),
    ("600-planes-fuzz", GEOMETRIES[4], None, (16, 2, 300, 256, 75, 3)),
]
FIELDS = ("words_per_lane", "segments", "piece_groups", "slots", "pga", "groups")


@pytest.mark.parametrize("name,g,refs,want", CASES, ids=[c[0] for c in CASES])
def test_digest_grid(torch, ck, name, g: Geometry, refs, want):
    if torch.cuda.get_device_properties(0).multi_processor_count != 256:
        pytest.skip("grid expectations are for 256 compute units")
    kv = torch.empty(g.pool_bytes, dtype=torch.uint8, device="cuda")
    with ck.Pool(g, 1, kv, max_claims=64, max_footprint=256, event_capacity=256) as pool:
        got = pool.digest_grid(refs)
    note(f"{name}: {got}")
    assert tuple(got[f] for f in FIELDS) == want
    phases = got["piece_groups"] // got["pga"]
    assert phases * got["pga"] == got["piece_groups"]
    del kv
    free_gpu(torch)
