"""Seeded synthetic inputs: workloads, claim batches, faults and pool content.

This subpackage only builds inputs.  It holds none of the checker's
arithmetic and is shared by the product's tests, the oracle side and the
benchmark.
"""

from .claims import MISSING, REQUEST_KINDS, Batch, FaultSpec, from_claims, make_batch, make_faults, make_requests  # noqa: F401
from .workloads import FULL, LLAMA3_8B, LLAMA3_70B, LLAMA3_70B_TP8, MLA_FP8, SHARDS, STRESS, TINY, Geometry, Workload, scaled  # noqa: F401
