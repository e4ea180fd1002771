"""Python handle on the C++ reference oracle (``oracle/oracle.cpp``).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``; the product path never imports it.

The oracle is a plain single-threaded statement of the checker's
definitions; see the header of ``oracle.cpp`` for what is computed and which
passage of the paper each part follows.  This module only marshals numpy
arrays into it.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "oracle.cpp")
LIBRARY = os.path.join(_HERE, "liboracle.so")

NONE32 = 0xFFFFFFFF

# The oracle's own record layouts (declared independently of the product).
OUTCOME_DTYPE = np.dtype(
    [
        ("claim_id", "<u8"),
        ("code", "<u4"),
        ("first_failing_block", "<u4"),
        ("phys_block", "<u4"),
        ("num_blocks", "<u4"),
        ("reasons", "<u4"),
        ("intact_blocks", "<u4"),
        ("expected_digest", "<u8"),
        ("observed_digest", "<u8"),
        ("chain_hash", "<u8"),
        ("chain_hash_at_fail", "<u8"),
    ]
)
EVENT_DTYPE = np.dtype(
    [
        ("seq", "<u8"),
        ("claim_id", "<u8"),
        ("aux", "<u8"),
        ("kind", "<u4"),
        ("block_index", "<u4"),
        ("phys_block", "<u4"),
        ("pad", "<u4"),
    ]
)
LOOKUP_DTYPE = np.dtype(
    [
        ("request_id", "<u8"),
        ("hit_tokens", "<u8"),
        ("chain_hash_at_hit", "<u8"),
        ("status", "<u4"),
        ("hit_blocks", "<u4"),
        ("last_block", "<u4"),
        ("pad", "<u4"),
    ]
)
assert OUTCOME_DTYPE.itemsize == 64 and EVENT_DTYPE.itemsize == 40 and LOOKUP_DTYPE.itemsize == 40

# vocabulary (the oracle's own copy)
UNKNOWN, MATERIALIZED, RESTORE_FAILED_FAIL_CLOSED = 0, 1, 2
EV_ACCEPTED, EV_OFFLOADED, EV_RESTORE_REQUIRED = 1, 2, 3
EV_RESTORED, EV_RESTORATION_FAILED, EV_ACTIVE_REQUEST_REFUSED, EV_OUTCOME_UNKNOWN = 4, 5, 6, 7
ST_ACCEPTED, ST_OFFLOADED, ST_RESTORE_REQUIRED = 1, 2, 4
R_NOT_ACCEPTED = 0x001
R_NOT_OFFLOADED = 0x002
R_NO_RESTORE = 0x004
R_TOKEN_MISMATCH = 0x008
R_FOOTPRINT_MISMATCH = 0x010
R_MISSING_ENTRY = 0x020
R_NO_OFFLOAD_RECORD = 0x040
R_SHAPE_MISMATCH = 0x080
R_EMPTY = 0x100
R_MALFORMED = 0x200
R_LOAD_FAILED = 0x400
R_DIGEST_MISMATCH = 0x800
R_BEYOND_PREDICATE = 0x1000
OK, EINVAL, EDUP = 0, -1, -5
LK_UNKNOWN, LK_HIT, LK_PARTIAL, LK_MISS = 0, 1, 2, 3


def build(force: bool = True) -> str:
    """Compile the oracle with g++ (single-threaded, no special flags)."""
    if force or not os.path.exists(LIBRARY):
        tmp = LIBRARY + ".tmp"
        subprocess.run(
            ["g++", "-O2", "-std=c++17", "-shared", "-fPIC", SOURCE, "-o", tmp], check=True
        )
        os.replace(tmp, LIBRARY)
    return LIBRARY


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIBRARY):
            build()
        L = ctypes.CDLL(LIBRARY)
        u64, u32, vp = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p
        for name, args, res in [
            ("orc_mix64", [u64], u64),
            ("orc_splitmix64", [u64], u64),
            ("orc_splitmix64_at", [u64, u64], u64),
            ("orc_kv_key", [u64, u64], u64),
            ("orc_token_key", [u64, u64], u64),
            ("orc_block_digest", [vp, u64, u64], u64),
            ("orc_pool_digests", [vp, u32, u32, u64, u64, vp], ctypes.c_int),
            ("orc_shard_digest", [vp, u32, u32, u32, u32, u32, u32, u64], u64),
            ("orc_token_multilinear", [vp, u64, u64], u64),
            ("orc_chain", [vp, u64, u32, u64, vp], u64),
            ("orc_canonical_block", [vp, u32, u32, u64, u32, vp], ctypes.c_int),
            ("orc_apply_flip", [vp, u32, u32, u64, u32, u64], ctypes.c_int),
            ("orc_pool_new", [u32, u32, u64], vp),
            ("orc_pool_free", [vp], None),
            ("orc_offload", [vp, u32, u64, u64, vp, vp, vp, vp, vp, vp, vp], ctypes.c_int),
            ("orc_restore", [vp, u32, u64, u64, vp, vp, vp, vp, vp, u32, vp], ctypes.c_int),
            ("orc_check", [vp, u32, u64, u64, vp, vp, vp, vp, vp, vp, vp], ctypes.c_int),
            ("orc_num_events", [vp], u64),
            ("orc_events", [vp, vp], None),
            ("orc_events_clear", [vp], None),
            ("orc_block_state", [vp, vp, vp, vp, vp], None),
            ("orc_claim_state", [vp, u64], u32),
            ("orc_claim_predicate", [vp, u64], u32),
            ("orc_lookup", [vp, u32, u64, vp, vp, vp, vp], ctypes.c_int),
            ("orc_identity_stats", [vp, vp, vp], None),
        ]:
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def _arr(a, dtype):
    return np.ascontiguousarray(np.asarray(a, dtype=dtype))


# ------------------------------------------------------------ pure functions


def mix64(z: int) -> int:
    return lib().orc_mix64(z)


def splitmix64(x: int) -> int:
    return lib().orc_splitmix64(x)


def splitmix64_at(s: int, i: int) -> int:
    return lib().orc_splitmix64_at(s, i)


def kv_key(seed: int, i: int) -> int:
    return lib().orc_kv_key(seed, i)


def token_key(seed: int, m: int) -> int:
    return lib().orc_token_key(seed, m)


def block_digest(canon: np.ndarray, seed: int) -> int:
    c = _arr(canon, np.uint8)
    assert c.size % 8 == 0
    return lib().orc_block_digest(_ptr(c), c.size, seed)


def shard_digest(canon: np.ndarray, seed: int, planes: int, block_size: int, heads: int,
                 row_bytes: int, heads_total: int, first_head: int) -> int:
    """Digest of a head shard of a block: its words with the keys of their
    positions in the full block (``canon``: the shard's own canonical
    bytes, planes chunks of [token][head][row_bytes])."""
    c = _arr(canon, np.uint8)
    assert c.size == planes * block_size * heads * row_bytes and row_bytes % 8 == 0
    assert first_head + heads <= heads_total
    return lib().orc_shard_digest(_ptr(c), planes, block_size, heads, row_bytes, heads_total,
                                  first_head, seed)


def token_multilinear(tokens, seed: int) -> int:
    t = _arr(tokens, np.uint32)
    return lib().orc_token_multilinear(_ptr(t), t.size, seed)


def chain(tokens, block_size: int, seed: int) -> np.ndarray:
    """h_0 .. h_{nt-1} for one claim's tokens."""
    t = _arr(tokens, np.uint32)
    nt = -(-t.size // block_size)
    h = np.zeros(nt, dtype=np.uint64)
    lib().orc_chain(_ptr(t), t.size, block_size, seed, _ptr(h))
    return h


def chain_hash(tokens, block_size: int, seed: int) -> int:
    t = _arr(tokens, np.uint32)
    return lib().orc_chain(_ptr(t), t.size, block_size, seed, None)


def canonical_block(pool: np.ndarray, planes: int, num_blocks: int, chunk_bytes: int, b: int):
    p = _arr(pool, np.uint8).reshape(-1)
    out = np.zeros(planes * chunk_bytes, dtype=np.uint8)
    rc = lib().orc_canonical_block(_ptr(p), planes, num_blocks, chunk_bytes, b, _ptr(out))
    if rc != OK:
        raise ValueError("block out of range")
    return out


def apply_flip(pool: np.ndarray, planes: int, num_blocks: int, chunk_bytes: int, b: int, bit: int):
    """Flip one canonical bit of block b in the host pool array (in place)."""
    assert pool.dtype == np.uint8 and pool.flags["C_CONTIGUOUS"]
    rc = lib().orc_apply_flip(_ptr(pool), planes, num_blocks, chunk_bytes, b, bit)
    if rc != OK:
        raise ValueError("flip out of range")


def pool_digests(pool: np.ndarray, planes: int, num_blocks: int, chunk_bytes: int, seed: int,
                 blocks=None) -> np.ndarray:
    """Digest of every (or of each listed) block of a host pool array."""
    out = np.zeros(num_blocks, dtype=np.uint64)
    if blocks is None:  # every block, in one loop of the oracle library
        p = _arr(pool, np.uint8).reshape(-1)
        assert p.size >= planes * num_blocks * chunk_bytes
        rc = lib().orc_pool_digests(_ptr(p), planes, num_blocks, chunk_bytes, seed, _ptr(out))
        if rc != OK:
            raise ValueError("block bytes not a whole number of 64-bit words")
        return out
    for b in blocks:
        out[b] = block_digest(canonical_block(pool, planes, num_blocks, chunk_bytes, int(b)), seed)
    return out


# ------------------------------------------------------------------ lifecycle


class OraclePool:
    """The oracle's claim pool: registry, offload records and event log.

    Block digests are supplied by the caller (computed with
    :func:`block_digest`) as an array indexed by physical block id.
    """

    def __init__(self, num_blocks: int, block_size: int, seed: int):
        self.num_blocks = num_blocks
        self.block_size = block_size
        self.seed = seed
        self._free = lib().orc_pool_free  # kept: module globals may be gone at exit
        self._h = lib().orc_pool_new(num_blocks, block_size, seed)
        if not self._h:
            raise ValueError("bad pool geometry")

    def __del__(self):
        h = getattr(self, "_h", None)
        if h:
            self._free(h)
            self._h = None

    @staticmethod
    def _batch_args(batch):
        ids = _arr(batch.claim_ids, np.uint64)
        bo = _arr(batch.block_offsets, np.uint32)
        bi = _arr(batch.block_ids, np.uint32)
        to = _arr(batch.token_offsets, np.uint64)
        tk = _arr(batch.tokens, np.uint32)
        keep = (ids, bo, bi, to, tk)
        return keep, [ids.size, bi.size, tk.size, _ptr(ids), _ptr(bo), _ptr(bi), _ptr(to), _ptr(tk)]

    def offload(self, batch, digest_now: np.ndarray) -> int:
        """Accept and offload; ``batch.predicate_tokens`` (optional, u64 per
        claim) sets each claim's leading_prefix_at_least(k)."""
        keep, args = self._batch_args(batch)
        d = _arr(digest_now, np.uint64)
        assert d.size == self.num_blocks
        pred = getattr(batch, "predicate_tokens", None)
        pred = None if pred is None else _arr(pred, np.uint64)
        return lib().orc_offload(self._h, *args, _ptr(pred), _ptr(d))

    def restore(self, batch, load_failed_blocks=()) -> int:
        keep, args = self._batch_args(batch)
        f = _arr(load_failed_blocks, np.uint32)
        return lib().orc_restore(self._h, *args, f.size, _ptr(f) if f.size else None)

    def check(self, batch, digest_now: np.ndarray) -> np.ndarray:
        keep, args = self._batch_args(batch)
        d = _arr(digest_now, np.uint64)
        assert d.size == self.num_blocks
        out = np.zeros(keep[0].size, dtype=OUTCOME_DTYPE)
        rc = lib().orc_check(self._h, *args, _ptr(d), _ptr(out))
        if rc != OK:
            raise RuntimeError(f"orc_check failed: {rc}")
        return out

    def events(self, clear: bool = False) -> np.ndarray:
        n = lib().orc_num_events(self._h)
        out = np.zeros(n, dtype=EVENT_DTYPE)
        if n:
            lib().orc_events(self._h, _ptr(out))
        if clear:
            lib().orc_events_clear(self._h)
        return out

    def block_state(self):
        nb = self.num_blocks
        d_off = np.zeros(nb, np.uint64)
        d_res = np.zeros(nb, np.uint64)
        valid = np.zeros(nb, np.uint8)
        failed = np.zeros(nb, np.uint8)
        lib().orc_block_state(self._h, _ptr(d_off), _ptr(d_res), _ptr(valid), _ptr(failed))
        return {"d_off": d_off, "d_res": d_res, "valid_off": valid, "load_failed": failed}

    def claim_state(self, claim_id: int) -> int:
        return lib().orc_claim_state(self._h, claim_id)

    def claim_predicate(self, claim_id: int) -> int:
        return lib().orc_claim_predicate(self._h, claim_id)

    def lookup(self, batch) -> np.ndarray:
        """Identity lookup of each row's tokens (block rows are not read)."""
        ids = _arr(batch.claim_ids, np.uint64)
        to = _arr(batch.token_offsets, np.uint64)
        tk = _arr(batch.tokens, np.uint32)
        out = np.zeros(ids.size, dtype=LOOKUP_DTYPE)
        rc = lib().orc_lookup(self._h, ids.size, tk.size, _ptr(ids), _ptr(to), _ptr(tk), _ptr(out))
        if rc != OK:
            raise RuntimeError(f"orc_lookup failed: {rc}")
        return out

    def identity_stats(self) -> tuple[int, int]:
        """(registered identities, ambiguous identities)."""
        e, a = ctypes.c_uint64(), ctypes.c_uint64()
        lib().orc_identity_stats(self._h, ctypes.byref(e), ctypes.byref(a))
        return int(e.value), int(a.value)
