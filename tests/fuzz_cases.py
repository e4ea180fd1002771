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
    # 600 planes of 16 KiB chunks over 4 blocks: 300 piece groups of 8 KiB
    # pieces, whose digest runs in four phases of 75 (fewer phases would
    # leave a quarter or more of the digest grid idle)
    Geometry(300, 2, 16, 4, 128, 2, 4),
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


# ------------------------------------------------- multi-step lifecycles


@dataclass
class Step:
    kind: str  # "offload", "restore", "check" or "lookup"
    batch: Batch
    faults: FaultSpec | None = None


@dataclass
class Sequence:
    w: Workload
    steps: list
    claims: int  # claims offloaded over the whole sequence
    refs: int


def make_sequence(seed: int, num_steps: int = 12) -> Sequence:
    """A random lifecycle of several offloads over a few hot blocks, so that
    claims share blocks, re-offload blocks whose loads failed or whose bytes
    changed, and register other prefixes in them; restores of random subsets
    of the claims with reported failures and bit flips (some flips undo
    earlier ones: a recompute of the original bytes); checks of random
    subsets, some presented changed or never accepted; lookups of their
    tokens.  Inputs only."""
    rng = np.random.default_rng(90_000 + seed)
    g = GEOMETRIES[seed % len(GEOMETRIES)]
    w = Workload(name=f"seq-{seed}", geometry=g, seed=int(rng.integers(0, 2**63)),
                 num_claims=0, length=TINY.length, sharing=TINY.sharing, corrupt_rate=0.0,
                 gen_seed=seed, content_seed=int(rng.integers(0, 2**31)))
    bs = g.block_size
    hot = rng.choice(g.num_blocks, size=min(g.num_blocks, int(rng.integers(6, 16))), replace=False)
    accepted = []  # (id, blocks, tokens)
    flips_done = []  # (block, bit) applied so far
    steps = []
    next_id = 1
    refs = 0
    for k in range(num_steps):
        kind = "offload" if k == 0 else str(rng.choice(["offload", "restore", "check", "lookup"],
                                                        p=[0.3, 0.3, 0.3, 0.1]))
        if kind == "offload":
            rows = []
            for _ in range(int(rng.integers(1, 7))):
                n = int(rng.integers(0, 6))
                blks = rng.choice(hot, size=n).astype(np.int64)
                if n and rng.random() < 0.05:
                    blks[int(rng.integers(n))] = MISSING
                if accepted and rng.random() < 0.35:  # an earlier claim's tokens (shared identities)
                    src = accepted[int(rng.integers(len(accepted)))]
                    tk = src[2][: int(rng.integers(0, src[2].size + 1))].copy()
                    n = -(-tk.size // bs)
                    blks = np.concatenate([src[1][:n], rng.choice(hot, size=max(0, n - src[1].size))])
                    if n and rng.random() < 0.5:
                        blks[int(rng.integers(n))] = int(rng.choice(hot))
                else:
                    tk = _tokens(rng, n * bs - (int(rng.integers(0, bs)) if n and rng.random() < 0.3 else 0))
                rows.append((next_id, blks.astype(np.uint32), tk))
                next_id += 1
            b = from_claims(rows)
            if rng.random() < 0.3:
                b.predicate_tokens = rng.integers(0, 6 * bs, size=b.num_claims).astype(np.uint64)
            accepted += rows
            refs += b.num_refs
            steps.append(Step("offload", b))
        elif kind == "restore":
            sub = [r for r in accepted if rng.random() < 0.7]
            fb, fbits = [], []
            for _ in range(int(rng.integers(0, 4))):
                if flips_done and rng.random() < 0.4:  # undo an earlier flip: a recompute
                    b0, bit0 = flips_done.pop(int(rng.integers(len(flips_done))))
                else:
                    b0, bit0 = int(rng.choice(hot)), int(rng.integers(0, 8 * g.block_bytes))
                    flips_done.append((b0, bit0))
                fb.append(b0)
                fbits.append(bit0)
            lost = rng.choice(hot, size=int(rng.integers(0, 3)), replace=False)
            steps.append(Step("restore", from_claims(sub),
                              FaultSpec(np.array(fb, np.uint32), np.array(fbits, np.uint64),
                                        np.asarray(lost, np.uint32))))
        elif kind == "check":
            pres = []
            for r in accepted:
                if rng.random() < 0.8:
                    cid, blks, tk = r[0], r[1].copy(), r[2].copy()
                    if rng.random() < 0.08 and blks.size:
                        blks[int(rng.integers(blks.size))] = int(rng.choice(hot))
                    elif rng.random() < 0.08 and tk.size:
                        tk[int(rng.integers(tk.size))] ^= 3
                    pres.append((cid, blks, tk))
            rng.shuffle(pres)
            pres.append((int(50_000 + k), rng.choice(hot, size=2).astype(np.uint32), _tokens(rng, 2 * bs)))
            steps.append(Step("check", from_claims(pres)))
        else:
            reqs = [(int(60_000 + 100 * k + i), [], r[2][: int(rng.integers(0, r[2].size + 1))])
                    for i, r in enumerate(accepted)]
            reqs.append((int(70_000 + k), [], _tokens(rng, 3 * bs)))
            steps.append(Step("lookup", from_claims(reqs)))
    steps.append(Step("restore", from_claims(accepted), FaultSpec(np.zeros(0, np.uint32), np.zeros(0, np.uint64),
                                                                   np.zeros(0, np.uint32))))
    steps.append(Step("check", from_claims(accepted)))
    return Sequence(w, steps, len(accepted), refs)


SEQUENCE_SEEDS = range(int(os.environ.get("CLAIMKV_SEQUENCE_SEEDS", "80")))
