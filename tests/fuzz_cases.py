"""Seeded irregular lifecycles for differential tests of the library against
the oracle: small pools of several geometries and batches with every
irregularity the batch format allows (empty and long rows, missing and
out-of-range entries, rows whose offsets run backwards or past the arrays,
rows that share entries, reserved and repeated ids, token rows that do not
match the block rows, predicates), faults, and check and lookup batches
that present the claims again with changes.  Between the two offloads a
restore of the first batch reports load failures and changes bytes, and the
second batch re-offloads some of those blocks under other claims (a
recompute stored by another claim, or other bytes).  Inputs only: nothing
here computes the method's arithmetic."""

from __future__ import annotations

import os
from dataclasses import dataclass

import numpy as np

from paper_2606_01387_amd.synth import MISSING, TINY, Batch, FaultSpec, Geometry, Workload, from_claims

RESERVED = 0xFFFFFFFFFFFFFFFF

GEOMETRIES = [
    Geometry(2, 2, 16, 2, 64, 2, 64),  # bf16 K/V, 16 KiB blocks
    Geometry(1, 2, 4, 1, 16, 2, 32),  # 4-token blocks, 128-byte chunks
    Geometry(3, 1, 8, 1, 24, 1, 48),  # fp8 latent, 192-byte chunks
    Geometry(2, 2, 16, 1, 64, 2, 40, total_kv_heads=4, first_kv_head=2),  # a head shard
]


@dataclass
class Case:
    w: Workload
    size: str
    staged: bool  # the second offload stages its blocks, the restore copies them back
    offload: list  # batches offloaded in turn
    mid: Batch  # restored (with mid_faults) after the first offload, before the second
    mid_faults: FaultSpec
    restore: Batch
    faults: FaultSpec
    check: Batch
    lookup: Batch


def _tokens(rng, n):
    return rng.integers(0, 32000, size=n, dtype=np.uint32)


SIZES = {"short": [0, 1, 1, 2, 3, 4, 6, 9], "long": [0, 3, 20, 40, 70, 120], "many": [0, 1, 1, 2, 3]}


def _claims(rng, g, count, ids, size="short"):
    bs = g.block_size
    parts = []
    for cid in ids[:count]:
        n = int(rng.choice(SIZES[size]))
        blks = rng.integers(0, g.num_blocks, size=n).astype(np.int64)
        for j in range(n):
            u = rng.random()
            if u < 0.02:
                blks[j] = MISSING
            elif u < 0.03:
                blks[j] = g.num_blocks + int(rng.integers(0, 5))
        nt = n if rng.random() < 0.92 else max(0, n + int(rng.choice([-1, 1])))
        ntok = nt * bs - (int(rng.integers(0, bs)) if nt and rng.random() < 0.4 else 0)
        parts.append((int(cid), blks.astype(np.uint32), _tokens(rng, ntok)))
    return parts


def _bend(rng, b: Batch) -> Batch:
    """Make some rows malformed: offsets that run backwards (so later rows
    may share entries) or past the arrays."""
    bo, to = b.block_offsets.astype(np.int64), b.token_offsets.astype(np.int64)
    C = b.num_claims
    if C >= 3 and rng.random() < 0.5:
        c = int(rng.integers(1, C))
        bo[c] = int(rng.integers(0, bo[c] + 1)) if rng.random() < 0.5 else bo[c]
        bo[c] = max(0, bo[c] - int(rng.integers(0, 6)))
    if C >= 2 and rng.random() < 0.3:
        to[int(rng.integers(1, C))] += int(rng.integers(1, 40))  # a row past the tokens or backwards
    if C >= 1 and rng.random() < 0.2:
        bo[C] = b.num_refs + 3  # the last row runs past the entries
    # offsets stay within their types; rows past the arrays are malformed
    return Batch(b.claim_ids, np.clip(bo, 0, 2**32 - 1).astype(np.uint32), b.block_ids,
                 np.clip(to, 0, None).astype(np.uint64), b.tokens)


def _present(rng, g, accepted, extra_ids, size):
    """The claims again, reordered, some repeated, some changed (a token, an
    entry, a cut or an extension), plus claims never accepted."""
    parts = []
    order = rng.permutation(len(accepted)) if accepted else []
    for i in order:
        cid, blks, tk = accepted[i]
        blks, tk = blks.copy(), tk.copy()
        u = rng.random()
        if u < 0.06 and tk.size:
            tk[int(rng.integers(tk.size))] ^= 1
        elif u < 0.12 and blks.size:
            blks[int(rng.integers(blks.size))] = int(rng.integers(0, g.num_blocks))
        elif u < 0.16:
            tk = tk[: int(rng.integers(0, tk.size + 1))]
        elif u < 0.20:
            tk = np.concatenate([tk, _tokens(rng, int(rng.integers(1, 2 * g.block_size)))])
        parts.append((cid, blks, tk))
        if rng.random() < 0.1:
            parts.append((cid, blks, tk))  # the same claim presented twice
    parts += _claims(rng, g, len(extra_ids), extra_ids, size)
    return from_claims(parts)


def make_case(seed: int) -> Case:
    rng = np.random.default_rng(80_000 + seed)
    g = GEOMETRIES[seed % len(GEOMETRIES)]
    w = Workload(name=f"fuzz-{seed}", geometry=g, seed=int(rng.integers(0, 2**63)),
                 num_claims=0, length=TINY.length, sharing=TINY.sharing, corrupt_rate=0.0,
                 gen_seed=seed, content_seed=int(rng.integers(0, 2**31)))
    # most cases are short claims; some have long claims (the wide group
    # paths) or thousands of claims (the tiled event scan)
    size = {6: "long", 7: "many"}.get(seed % 8, "short")
    n_first = {"short": int(rng.integers(0, 30)), "long": int(rng.integers(1, 12)),
               "many": int(rng.integers(4200, 6000))}[size]
    ids = rng.permutation(np.arange(1, 20000, dtype=np.uint64))
    if rng.random() < 0.3:
        ids[int(rng.integers(0, 10))] = RESERVED
    first = _claims(rng, g, n_first, ids[:n_first], size)
    second = _claims(rng, g, int(rng.integers(0, 12)), ids[10000:10012], size)
    # a later claim with an earlier claim's tokens (shared identities; with
    # another block row, duplicate ownership)
    if first and rng.random() < 0.7:
        src = first[int(rng.integers(len(first)))]
        blks = src[1].copy()
        if blks.size and rng.random() < 0.5:
            blks[0] = int(rng.integers(0, g.num_blocks))
        second.append((int(ids[10100]), blks, src[2].copy()))
    # between the offloads: a restore of some first-batch claims that reports
    # load failures and flips bytes of blocks they hold; the second batch then
    # re-offloads some of those blocks under a new claim
    held = [int(x) for _, blks, _ in first for x in blks if x < g.num_blocks]
    mid_rows = [r for r in first if rng.random() < 0.7]
    touched = (rng.choice(held, size=min(len(held), int(rng.integers(1, 4))), replace=False)
               if held and rng.random() < 0.8 else np.zeros(0, np.int64))
    lost = touched[: int(rng.integers(0, touched.size + 1))]
    flipped = np.setdiff1d(touched, lost) if rng.random() < 0.5 else touched
    mid_faults = FaultSpec(np.asarray(flipped, np.uint32),
                           rng.integers(0, 8 * g.block_bytes, size=flipped.size).astype(np.uint64),
                           np.asarray(lost, np.uint32))
    if touched.size:
        n_re = int(rng.integers(1, 4))
        blks = np.concatenate([touched, rng.integers(0, g.num_blocks, size=n_re)]).astype(np.uint32)
        rng.shuffle(blks)
        second.append((int(ids[10150]), blks, _tokens(rng, blks.size * g.block_size)))
    b1 = _bend(rng, from_claims(first))
    b1.predicate_tokens = (rng.integers(0, 80, size=b1.num_claims).astype(np.uint64)
                           if rng.random() < 0.4 else None)
    b2 = from_claims(second)
    accepted = first + second
    nflip = int(rng.integers(0, 6))
    flips = FaultSpec(rng.integers(0, g.num_blocks, size=nflip).astype(np.uint32),
                      rng.integers(0, 8 * g.block_bytes, size=nflip).astype(np.uint64),
                      rng.integers(0, g.num_blocks, size=int(rng.integers(0, 3))).astype(np.uint32))
    keep = len(accepted) if rng.random() < 0.8 else int(rng.integers(0, len(accepted) + 1))
    restore = from_claims(accepted[:keep])
    check = _bend(rng, _present(rng, g, accepted, ids[10200:10204], size))
    reqs = [(int(i), [], p[2][: int(rng.integers(0, p[2].size + 1))] if rng.random() < 0.3 else p[2])
            for i, p in zip(ids[12000:], accepted)]
    lookup = _bend(rng, from_claims(reqs + [(int(ids[10300]), [], _tokens(rng, 3 * g.block_size))]))
    return Case(w, size, seed % 3 == 0, [b1, b2], from_claims(mid_rows), mid_faults, restore, flips,
                check, lookup)



def well_formed_blocks(b: Batch, num_blocks: int) -> np.ndarray:
    """In-range blocks referenced by the batch's well-formed rows (the
    blocks an offload stages and a restore copies back), ascending."""
    bo, to = b.block_offsets.astype(np.int64), b.token_offsets.astype(np.int64)
    out = []
    for c in range(b.num_claims):
        if (int(b.claim_ids[c]) == RESERVED or bo[c] > bo[c + 1] or bo[c + 1] > b.num_refs
                or to[c] > to[c + 1] or to[c + 1] > b.num_tokens):
            continue
        blks = b.block_ids[bo[c]:bo[c + 1]]
        out.append(blks[blks < num_blocks])
    return np.unique(np.concatenate(out)) if out else np.zeros(0, np.uint32)


def capacities(case: Case) -> dict:
    claims = sum(b.num_claims for b in case.offload)
    refs = sum(b.num_refs for b in case.offload)
    return dict(max_claims=2 * claims + 64, max_footprint=4 * refs + 256,
                event_capacity=4 * (claims + case.check.num_claims) + 1024)


# CLAIMKV_FUZZ_SEEDS widens a one-off run; the suite replays the first 160
SEEDS = range(int(os.environ.get("CLAIMKV_FUZZ_SEEDS", "160")))
