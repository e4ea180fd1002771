"""Workload shapes for the claim-scoped KV materialization checker.

Each workload names a paged KV pool geometry (the cache identity's block
geometry, Table 5 "fixed cache identity") and the shape of a synthetic claim
batch: claim count, length distribution, prefix sharing, corruption rate and
missing block-table entries.  Sizes follow the model shapes they are named
after (layers x KV heads x head_dim x block_size x element size); nothing
here depends on weights, tokenizers or datasets.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field, replace


@dataclass(frozen=True)
class Geometry:
    """Paged KV pool geometry.  Layout in HBM: [plane][block][chunk], where a
    plane is one layer's K or V (or one layer's MLA latent) and a chunk is
    block_size x num_kv_heads x head_dim elements in [token][head][dim]
    order."""

    num_layers: int
    planes_per_layer: int  # 2 = K and V, 1 = MLA latent
    block_size: int  # tokens per block
    num_kv_heads: int  # 1 for an MLA latent
    head_dim: int  # latent width for MLA
    elem_bytes: int  # 2 = bf16, 1 = fp8 e4m3 (bytes are never interpreted)
    num_blocks: int
    # a head shard (tensor parallel by KV head): this pool holds heads
    # [first_kv_head, first_kv_head + num_kv_heads) of blocks that have
    # total_kv_heads heads; 0 = whole blocks
    total_kv_heads: int = 0
    first_kv_head: int = 0

    @property
    def sharded(self) -> bool:
        return self.total_kv_heads not in (0, self.num_kv_heads)

    @property
    def row_bytes(self) -> int:
        """One head's bytes of one token."""
        return self.head_dim * self.elem_bytes

    @property
    def planes(self) -> int:
        return self.num_layers * self.planes_per_layer

    @property
    def chunk_bytes(self) -> int:
        return self.block_size * self.num_kv_heads * self.head_dim * self.elem_bytes

    @property
    def block_bytes(self) -> int:
        return self.planes * self.chunk_bytes

    @property
    def pool_bytes(self) -> int:
        return self.block_bytes * self.num_blocks

    @property
    def raw_bytes(self) -> bool:
        """True when content is uniform random bytes (fp8), else bf16 values."""
        return self.elem_bytes == 1


@dataclass(frozen=True)
class Workload:
    name: str
    geometry: Geometry
    seed: int  # cache-identity seed S of the pool (keys and chain)
    num_claims: int
    # claim length: ("blocks", lo, hi, ragged_tail) or
    #               ("lognormal_tokens", median, sigma, lo, hi)
    length: tuple
    # prefix sharing: ("fraction", f) -> a fraction f of claims share with an
    # earlier root claim; ("zipf", a, claims_per_family) -> family sizes
    # follow Zipf(a) over ceil(C / claims_per_family) families.
    sharing: tuple
    corrupt_rate: float  # fraction of pool blocks with one flipped bit
    missing_claim_rate: float = 0.0  # fraction of claims with one missing entry
    num_load_failed: int = 0  # reported load failures (referenced blocks)
    predicate_fraction: float = 0.0  # claims whose predicate covers only a prefix
    gen_seed: int = 0  # seed of the claim / fault generator
    content_seed: int = 0  # seed of the pool content generator
    vocab: int = 32000
    notes: str = field(default="", compare=False)

    @property
    def num_corrupt(self) -> int:
        return int(round(self.corrupt_rate * self.geometry.num_blocks))


def _w(name, geom, seed, **kw) -> Workload:
    kw.setdefault("gen_seed", seed * 7 + 1)
    kw.setdefault("content_seed", seed * 13 + 5)
    return Workload(name=name, geometry=geom, seed=seed, **kw)


TINY = _w(
    "tiny",
    Geometry(2, 2, 16, 2, 64, 2, 64),
    seed=1001,
    num_claims=16,
    length=("blocks", 1, 8, True),
    sharing=("fraction", 0.25),
    corrupt_rate=0.05,
    notes="64 blocks of 16 KiB; parity case the oracle runs in seconds",
)

LLAMA3_8B = _w(
    "llama3-8b",
    Geometry(32, 2, 16, 8, 128, 2, 8192),
    seed=1002,
    num_claims=1024,
    length=("lognormal_tokens", 512, math.log(64) / 6, 64, 4096),
    sharing=("zipf", 1.1, 4),
    corrupt_rate=0.01,
    notes="2 MiB blocks, 16 GiB pool; the benchmark workload",
)

LLAMA3_70B = _w(
    "llama3-70b",
    Geometry(80, 2, 16, 8, 128, 2, 20000),
    seed=1003,
    num_claims=4096,
    length=("lognormal_tokens", 4096, math.log(64) / 6, 512, 32768),
    sharing=("zipf", 1.1, 4),
    corrupt_rate=0.001,
    missing_claim_rate=0.02,
    notes="5 MiB blocks, ~105 GB pool on one GPU",
)

STRESS = _w(
    "small-claim-stress",
    Geometry(28, 2, 16, 4, 128, 2, 32768),
    seed=1004,
    num_claims=1_000_000,
    length=("blocks", 1, 4, False),
    sharing=("zipf", 1.3, 64),
    corrupt_rate=0.005,
    notes="896 KiB blocks, 1M claims of 1-4 blocks",
)

MLA_FP8 = _w(
    "mla-fp8",
    Geometry(61, 1, 64, 1, 576, 1, 6000),
    seed=1005,
    num_claims=512,
    length=("lognormal_tokens", 1448, math.log(512) / 6, 64, 32768),
    sharing=("zipf", 1.1, 4),
    corrupt_rate=0.001,
    notes="576-byte fp8 latent per token, 64-token blocks; staged round trip",
)

FULL = {w.name: w for w in (TINY, LLAMA3_8B, LLAMA3_70B, STRESS, MLA_FP8)}

# One GPU's share of the 70B pool under tensor parallelism by KV head over 8
# GPUs: the same blocks and claims, each block holding one of the 8 heads
# (640 KiB per block, 4 KiB chunks, a 13.1 GB pool).  Its digests are the
# head shard's part of the full blocks' digests.
LLAMA3_70B_TP8 = replace(
    LLAMA3_70B, name="llama3-70b-tp8-shard",
    geometry=Geometry(80, 2, 16, 1, 128, 2, 20000, total_kv_heads=8, first_kv_head=0),
    notes="one GPU's head shard of the 70B pool under 8-way tensor parallelism")

SHARDS = {w.name: w for w in (LLAMA3_70B_TP8,)}


def scaled(w: Workload, num_blocks: int, num_claims: int, **kw) -> Workload:
    """The same geometry per block with a smaller pool and batch: parity cases
    that the oracle finishes in seconds but that still span many tiles."""
    g = replace(w.geometry, num_blocks=num_blocks)
    return replace(w, name=f"{w.name}-scaled", geometry=g, num_claims=num_claims, **kw)
