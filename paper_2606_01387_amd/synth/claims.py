"""Seeded synthetic claim batches and fault specifications.

A batch is a compressed-row table of claims: stable 64-bit claim ids,
per-claim block-table rows (physical block ids, 0xFFFFFFFF = missing) and
per-claim token ids.  Prefix sharing copies the leading full blocks of a
family root, both its token ids and its physical block ids, as a prefix
cache does.  Blocks that are not shared take physical ids from a seeded
permutation of the pool, cycling: the batches reference several times more
logical blocks than the pool holds, so unrelated claims alias physical
blocks, and nearly every pool block is referenced.

All randomness comes from numpy's PCG64 generator with a fixed seed.  The
generator holds none of the checker's arithmetic: it only builds inputs.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

from .workloads import Workload

MISSING = 0xFFFFFFFF


@dataclass
class Batch:
    claim_ids: np.ndarray  # u64 [C]
    block_offsets: np.ndarray  # u32 [C+1]
    block_ids: np.ndarray  # u32 [N]
    token_offsets: np.ndarray  # u64 [C+1]
    tokens: np.ndarray  # u32 [T]
    predicate_tokens: np.ndarray | None = None  # u64 [C]: leading_prefix_at_least(k)

    @property
    def num_claims(self) -> int:
        return int(self.claim_ids.size)

    @property
    def num_refs(self) -> int:
        return int(self.block_ids.size)

    @property
    def num_tokens(self) -> int:
        return int(self.tokens.size)

    def claim(self, c: int):
        """(claim id, block ids, tokens) of claim c."""
        b0, b1 = int(self.block_offsets[c]), int(self.block_offsets[c + 1])
        t0, t1 = int(self.token_offsets[c]), int(self.token_offsets[c + 1])
        return int(self.claim_ids[c]), self.block_ids[b0:b1], self.tokens[t0:t1]

    def subset(self, idx) -> "Batch":
        """A batch made of the listed claims, in the listed order."""
        parts = [self.claim(int(c)) for c in idx]
        b = from_claims(parts)
        if self.predicate_tokens is not None:
            b.predicate_tokens = self.predicate_tokens[np.asarray(idx, dtype=np.int64)]
        return b

    def unique_blocks(self, num_blocks: int) -> np.ndarray:
        b = self.block_ids[self.block_ids < num_blocks]
        return np.unique(b)


def from_claims(parts) -> Batch:
    """Build a batch from a list of (claim id, block ids, tokens)."""
    ids = np.array([p[0] for p in parts], dtype=np.uint64)
    nb = np.array([len(p[1]) for p in parts], dtype=np.int64)
    nt = np.array([len(p[2]) for p in parts], dtype=np.int64)
    bo = np.zeros(len(parts) + 1, dtype=np.uint32)
    bo[1:] = np.cumsum(nb)
    to = np.zeros(len(parts) + 1, dtype=np.uint64)
    to[1:] = np.cumsum(nt)
    bi = (np.concatenate([np.asarray(p[1], np.uint32) for p in parts])
          if parts and nb.sum() else np.zeros(0, np.uint32))
    tk = (np.concatenate([np.asarray(p[2], np.uint32) for p in parts])
          if parts and nt.sum() else np.zeros(0, np.uint32))
    return Batch(ids, bo, bi.astype(np.uint32), to, tk.astype(np.uint32))


@dataclass
class FaultSpec:
    flip_blocks: np.ndarray  # u32 [F]   physical block of each flip
    flip_bits: np.ndarray  # u64 [F]   canonical bit index within the block
    load_failed: np.ndarray  # u32 [L]   blocks whose load is reported failed

    @staticmethod
    def none() -> "FaultSpec":
        return FaultSpec(np.zeros(0, np.uint32), np.zeros(0, np.uint64), np.zeros(0, np.uint32))

    def changed_blocks(self) -> np.ndarray:
        """Blocks whose bytes differ after the flips (an even number of flips
        of the same bit cancels)."""
        if self.flip_blocks.size == 0:
            return np.zeros(0, np.uint32)
        key = self.flip_blocks.astype(np.uint64) << np.uint64(40) | self.flip_bits
        uniq, counts = np.unique(key, return_counts=True)
        odd = uniq[counts % 2 == 1]
        return np.unique((odd >> np.uint64(40)).astype(np.uint32))


def _token_counts(w: Workload, rng: np.random.Generator) -> np.ndarray:
    bs = w.geometry.block_size
    kind = w.length[0]
    C = w.num_claims
    if kind == "blocks":
        _, lo, hi, ragged = w.length
        n = rng.integers(lo, hi + 1, size=C)
        if ragged:
            return (n - 1) * bs + rng.integers(1, bs + 1, size=C)
        return n * bs
    if kind == "lognormal_tokens":
        _, median, sigma, lo, hi = w.length
        t = np.exp(rng.normal(math.log(median), sigma, size=C))
        return np.clip(np.rint(t), lo, hi).astype(np.int64)
    raise ValueError(kind)


def _roots(w: Workload, rng: np.random.Generator) -> np.ndarray:
    """root[c] = the claim whose prefix c shares (c itself for a root)."""
    C = w.num_claims
    kind = w.sharing[0]
    idx = np.arange(C)
    if kind == "fraction":
        k = int(round(w.sharing[1] * C))
        sharers = np.sort(rng.choice(np.arange(1, C), size=min(k, C - 1), replace=False))
        root = idx.copy()
        is_sharer = np.zeros(C, bool)
        is_sharer[sharers] = True
        for c in sharers:
            cands = np.flatnonzero(~is_sharer[:c])
            root[c] = cands[rng.integers(0, cands.size)]
        return root
    if kind == "zipf":
        _, a, per_family = w.sharing
        F = max(1, math.ceil(C / per_family))
        p = np.arange(1, F + 1, dtype=np.float64) ** (-a)
        fam = rng.choice(F, size=C, p=p / p.sum())
        _, first, inverse = np.unique(fam, return_index=True, return_inverse=True)
        return first[inverse]
    raise ValueError(kind)


def make_batch(w: Workload) -> Batch:
    """The workload's claim batch (deterministic in w.gen_seed)."""
    g = w.geometry
    bs, nb, C = g.block_size, g.num_blocks, w.num_claims
    rng = np.random.default_rng(w.gen_seed)

    T = _token_counts(w, rng).astype(np.int64)
    n = (T + bs - 1) // bs
    root = _roots(w, rng)
    full = T // bs
    m = np.minimum(full, full[root])
    u = rng.random(C)
    share = np.minimum(np.floor(u * (m + 1)).astype(np.int64), m)
    share[root == np.arange(C)] = 0

    bo = np.zeros(C + 1, np.int64)
    bo[1:] = np.cumsum(n)
    to = np.zeros(C + 1, np.int64)
    to[1:] = np.cumsum(T)
    N, TT = int(bo[-1]), int(to[-1])
    if N >= MISSING:
        raise ValueError("too many block references")

    # claim-relative position of every block entry / token
    claim_of_ref = np.repeat(np.arange(C), n)
    j_of_ref = np.arange(N) - bo[claim_of_ref]
    claim_of_tok = np.repeat(np.arange(C), T)
    m_of_tok = np.arange(TT) - to[claim_of_tok]

    shared_ref = j_of_ref < share[claim_of_ref]
    shared_tok = m_of_tok < share[claim_of_tok] * bs

    # physical ids: fresh entries cycle through a seeded permutation
    perm = rng.permutation(nb).astype(np.int64)
    blk = np.empty(N, np.int64)
    fresh = np.flatnonzero(~shared_ref)
    blk[fresh] = perm[np.arange(fresh.size) % nb]
    src = bo[root[claim_of_ref[shared_ref]]] + j_of_ref[shared_ref]
    blk[shared_ref] = blk[src]  # roots never share, so sources are fresh

    tok = rng.integers(0, w.vocab, size=TT, dtype=np.int64)
    tsrc = to[root[claim_of_tok[shared_tok]]] + m_of_tok[shared_tok]
    tok[shared_tok] = tok[tsrc]

    # missing block-table entries
    k = int(round(w.missing_claim_rate * C))
    if k:
        victims = rng.choice(C, size=k, replace=False)
        jj = (rng.random(k) * n[victims]).astype(np.int64)
        blk[bo[victims] + jj] = MISSING

    # stable 64-bit claim ids, distinct from batch positions
    ids = rng.integers(1, np.iinfo(np.int64).max, size=C, dtype=np.int64).astype(np.uint64)
    while np.unique(ids).size != C:
        _, first = np.unique(ids, return_index=True)
        dup = np.setdiff1d(np.arange(C), first)
        ids[dup] = rng.integers(1, np.iinfo(np.int64).max, size=dup.size, dtype=np.int64)

    pred = None
    if w.predicate_fraction > 0:
        # a fraction of the claims covers only a leading prefix: k uniform in
        # [1, T_c]; the rest cover the whole claim
        pred = T.astype(np.uint64).copy()
        sel = rng.random(C) < w.predicate_fraction
        pred[sel] = (1 + (rng.random(int(sel.sum())) * T[sel]).astype(np.int64)).astype(np.uint64)

    return Batch(
        claim_ids=ids,
        block_offsets=bo.astype(np.uint32),
        block_ids=blk.astype(np.uint32),
        token_offsets=to.astype(np.uint64),
        tokens=tok.astype(np.uint32),
        predicate_tokens=pred,
    )


REQUEST_KINDS = ("same", "cut", "changed", "extended", "fresh")


def make_requests(w: Workload, batch: Batch, num_requests: int | None = None,
                  mix=(0.3, 0.2, 0.2, 0.15, 0.15)) -> tuple[Batch, np.ndarray]:
    """Reuse-lookup requests against an offloaded claim batch (token rows
    only; block rows are empty).  Each request takes a uniformly chosen
    source claim and is, with the probabilities in ``mix``: the same tokens;
    a cut to a uniform length in [1, T]; the same length with one uniformly
    chosen token changed; the tokens followed by 1..2*block_size fresh ones;
    or T fresh tokens.  Returns the batch and the kind index of each row."""
    bs = w.geometry.block_size
    rng = np.random.default_rng(w.gen_seed ^ 0x10C0)
    C = batch.num_claims
    R = C if num_requests is None else num_requests
    to = batch.token_offsets.astype(np.int64)
    Tc = np.diff(to)
    src = rng.integers(0, C, size=R)
    kind = rng.choice(len(REQUEST_KINDS), size=R, p=np.asarray(mix) / np.sum(mix))
    Ts = Tc[src]
    L = Ts.copy()
    cut = kind == 1
    L[cut] = 1 + (rng.random(int(cut.sum())) * np.maximum(Ts[cut], 1)).astype(np.int64)
    ext = kind == 3
    L[ext] = Ts[ext] + rng.integers(1, 2 * bs + 1, size=int(ext.sum()))
    L = np.maximum(L, 0)

    ro = np.zeros(R + 1, np.int64)
    ro[1:] = np.cumsum(L)
    TT = int(ro[-1])
    req_of_tok = np.repeat(np.arange(R), L)
    m = np.arange(TT) - ro[req_of_tok]
    copied = (kind[req_of_tok] != 4) & (m < Ts[req_of_tok])
    tok = rng.integers(0, w.vocab, size=TT, dtype=np.int64)
    tok[copied] = batch.tokens[(to[src[req_of_tok]] + m)[copied]]

    # one changed token per "changed" request (never left equal)
    ch = np.flatnonzero((kind == 2) & (L > 0))
    pos = ro[ch] + (rng.random(ch.size) * L[ch]).astype(np.int64)
    tok[pos] = (tok[pos] + 1 + rng.integers(0, w.vocab - 1, size=ch.size)) % w.vocab

    ids = rng.integers(1, np.iinfo(np.int64).max, size=R, dtype=np.int64).astype(np.uint64)
    req = Batch(
        claim_ids=ids,
        block_offsets=np.zeros(R + 1, np.uint32),
        block_ids=np.zeros(0, np.uint32),
        token_offsets=ro.astype(np.uint64),
        tokens=tok.astype(np.uint32),
    )
    return req, kind


def make_faults(w: Workload, batch: Batch | None = None) -> FaultSpec:
    """One flipped bit in each of round(rate * num_blocks) distinct pool
    blocks (referenced or not), plus num_load_failed reported load failures
    on referenced blocks."""
    g = w.geometry
    rng = np.random.default_rng(w.gen_seed ^ 0x5A5A5A5A)
    k = w.num_corrupt
    blocks = rng.choice(g.num_blocks, size=k, replace=False).astype(np.uint32)
    bits = rng.integers(0, 8 * g.block_bytes, size=k, dtype=np.int64).astype(np.uint64)
    lf = np.zeros(0, np.uint32)
    if w.num_load_failed:
        if batch is None:
            batch = make_batch(w)
        ref = batch.unique_blocks(g.num_blocks)
        lf = rng.choice(ref, size=min(w.num_load_failed, ref.size), replace=False)
        lf = lf.astype(np.uint32)
    return FaultSpec(blocks, bits, lf)
