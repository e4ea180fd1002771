"""The digest kernel over seeded random pool geometries, against the
oracle: block sizes, head counts, head widths and element sizes that give
chunks from 16 bytes to 72 KiB (every words-per-lane width the kernel
instantiates, whole and ragged chunks, one or several segments per chunk),
planes from 1 to 12, and head shards at random offsets; and pools of 100 to
860 planes over 8 to 16 blocks, whose digest mostly reads its piece groups
in phases (one phase would leave much of the grid idle).  Every block's
offload digest, and its restore digest after seeded flips, must equal the
oracle's."""

import os

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_01387_amd.synth import TINY, FaultSpec, Geometry, Workload, content, from_claims
from tests.helpers import apply_flips, digests
from tests.test_gpu_parity import free_gpu, gpu_pool_tensor

pytestmark = pytest.mark.gpu


def random_geometry(rng) -> Geometry:
    while True:
        layers, ppl = int(rng.integers(1, 7)), int(rng.choice([1, 2]))
        bs = int(rng.choice([1, 2, 3, 4, 5, 8, 16, 32, 64]))
        heads = int(rng.choice([1, 1, 2, 3, 4, 8]))
        dim = int(rng.choice([8, 16, 24, 40, 64, 96, 128, 576]))
        eb = int(rng.choice([1, 2]))
        chunk = bs * heads * dim * eb
        if chunk % 16 or chunk > 72 * 1024:
            continue
        nb = int(rng.integers(8, 40))
        if rng.random() < 0.3 and dim * eb % 8 == 0:
            total = heads * int(rng.integers(2, 5))
            first = int(rng.integers(0, total - heads + 1))
            return Geometry(layers, ppl, bs, heads, dim, eb, nb, total_kv_heads=total,
                            first_kv_head=first)
        return Geometry(layers, ppl, bs, heads, dim, eb, nb)


# Chunks of 12 to 72 words per lane (6 to 36 KiB) and the segments they
# split into: pieces of 12, 16, 24 or 32 words per lane, one digest
# workgroup per CU.
_PLANE_CHUNKS = [(6144, 1), (8192, 1), (12288, 1), (16384, 1), (24576, 2), (32768, 2), (36864, 3)]


def many_plane_geometry(rng) -> Geometry:
    """Planes enough for 87-108 or 130-216 piece groups of 4 pieces (the
    last group often short): one phase would fill at most 85 % of a grid of
    one workgroup per CU on 256 CUs."""
    while True:
        chunk, segs = _PLANE_CHUNKS[int(rng.integers(len(_PLANE_CHUNKS)))]
        pgs = int(rng.integers(87, 109)) if rng.random() < 0.3 else int(rng.integers(130, 217))
        planes = max(1, (4 * pgs - int(rng.integers(0, 4))) // segs)
        ppl = 2 if planes % 2 == 0 and rng.random() < 0.5 else 1
        bs = int(rng.choice([1, 2, 4, 8, 16]))
        nb = int(rng.integers(8, 17))  # enough blocks for several workgroups per phase
        if planes * chunk * nb > 160 << 20:
            continue
        return Geometry(planes // ppl, ppl, bs, 1, chunk // bs, 1, nb)


# CLAIMKV_SHAPE_SEEDS widens a one-off run; the suite runs the first 60
@pytest.mark.parametrize("seed", range(int(os.environ.get("CLAIMKV_SHAPE_SEEDS", "60"))))
def test_digest_shapes(torch, ck, seed):
    rng = np.random.default_rng(70_000 + seed)
    run_shape(torch, ck, random_geometry(rng), rng, seed)


@pytest.mark.parametrize("seed", range(int(os.environ.get("CLAIMKV_PLANE_SEEDS", "16"))))
def test_digest_shapes_many_planes(torch, ck, seed):
    rng = np.random.default_rng(80_000 + seed)
    run_shape(torch, ck, many_plane_geometry(rng), rng, seed)


def run_shape(torch, ck, g, rng, seed):
    w = Workload(name=f"shape-{seed}", geometry=g, seed=int(rng.integers(0, 2**63)), num_claims=0,
                 length=TINY.length, sharing=TINY.sharing, corrupt_rate=0.0, gen_seed=seed,
                 content_seed=int(rng.integers(0, 2**31)))
    print(f"digest shape seed {seed}: planes {g.planes}, chunk {g.chunk_bytes} B "
          f"(bs {g.block_size}, heads {g.num_kv_heads}/{g.total_kv_heads or g.num_kv_heads}, "
          f"dim {g.head_dim}, elem {g.elem_bytes}), {g.num_blocks} blocks", flush=True)
    # every block, one claim each (a few blocks twice)
    blocks = list(range(g.num_blocks)) + [int(b) for b in rng.integers(0, g.num_blocks, 3)]
    batch = from_claims([(i + 1, [b], rng.integers(0, 32000, g.block_size, dtype=np.uint32))
                         for i, b in enumerate(blocks)])
    nflip = int(rng.integers(1, 6))
    faults = FaultSpec(rng.integers(0, g.num_blocks, nflip).astype(np.uint32),
                       rng.integers(0, 8 * g.block_bytes, nflip).astype(np.uint64),
                       np.zeros(0, np.uint32))
    kv = gpu_pool_tensor(torch, w)
    host = content.pool_host(g, w.content_seed)
    with ck.Pool(g, w.seed, kv, max_claims=128, max_footprint=256, event_capacity=512) as pool:
        db = ck.DeviceBatch(batch)
        pool.offload(db)
        pool.restore(db, faults=faults)
        pool.check(db)
        out, _ = pool.read()
        st = pool.block_state()
    assert np.array_equal(st["d_off"], digests(host, w))
    assert np.array_equal(st["d_res"], digests(apply_flips(host, w, faults), w))
    failed = set(int(b) for b in faults.changed_blocks())
    assert [int(c) for c in out["code"]] == [2 if b in failed else 1 for b in blocks]
    del kv
    free_gpu(torch)
