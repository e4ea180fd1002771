"""The block-by-block oracle digests used at full size equal the digests of
the whole generated pool, before and after the flips (CPU)."""

import numpy as np
import pytest

from oracle.pool_digests import modeled_digests, real_digests
from paper_2606_01387_amd.synth import SHARDS, TINY, make_batch, make_faults, scaled
from tests.helpers import apply_flips, digests, host_pool


@pytest.mark.parametrize("w", [TINY, scaled(SHARDS["llama3-70b-tp8-shard"], 24, 10, corrupt_rate=0.2)],
                         ids=lambda w: w.name)
def test_real_digests_equal_whole_pool_digests(w):
    batch = make_batch(w)
    faults = make_faults(w, batch)
    assert faults.flip_blocks.size
    pool = host_pool(w)
    want0 = digests(pool, w)
    want1 = digests(apply_flips(pool, w, faults), w)
    every = np.arange(w.geometry.num_blocks)
    d0, d1 = real_digests(w, faults, every, threads=4)
    assert np.array_equal(d0, want0) and np.array_equal(d1, want1)
    # a subset: listed blocks real, the rest equal placeholders (as modeled)
    some = every[::3]
    s0, s1 = real_digests(w, faults, some, threads=3)
    m0, m1 = modeled_digests(w, faults, some)
    assert np.array_equal(s0[some], want0[some]) and np.array_equal(s1[some], want1[some])
    rest = np.setdiff1d(every, np.union1d(some, faults.changed_blocks()))
    assert np.array_equal(s0[rest], s1[rest]) and np.array_equal(s0[rest], m0[rest])
