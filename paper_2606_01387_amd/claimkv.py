"""Python binding of ``libclaimkv.so`` (the C ABI in ``include/claimkv.h``).

Argument marshalling only: every step of offload, restore and check runs in
the library's HIP kernels.  PyTorch provides device memory and the stream.
There is no fallback: if the library is missing, loading it raises.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(_HERE)
SOURCE = os.path.join(_HERE, "csrc", "claimkv.hip")
LIBRARY = os.path.join(_HERE, "libclaimkv.so")
INCLUDE = os.path.join(ROOT, "include")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-shared", "-std=c++17",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]

# ------------------------------------------------------------ vocabulary
OK, EINVAL, ENOMEM, EHIP, ENOSPC, EDUP, ELIMIT = 0, -1, -2, -3, -4, -5, -6
STATIC_MAX_CLAIMS = 262144
UNKNOWN, MATERIALIZED, RESTORE_FAILED_FAIL_CLOSED = 0, 1, 2
EV_ACCEPTED, EV_OFFLOADED, EV_RESTORE_REQUIRED, EV_RESTORED = 1, 2, 3, 4
EV_RESTORATION_FAILED, EV_ACTIVE_REQUEST_REFUSED, EV_OUTCOME_UNKNOWN = 5, 6, 7
R_NOT_ACCEPTED, R_NOT_OFFLOADED, R_NO_RESTORE, R_TOKEN_MISMATCH = 0x001, 0x002, 0x004, 0x008
R_FOOTPRINT_MISMATCH, R_MISSING_ENTRY, R_NO_OFFLOAD_RECORD, R_SHAPE_MISMATCH = 0x010, 0x020, 0x040, 0x080
R_EMPTY, R_MALFORMED, R_LOAD_FAILED, R_DIGEST_MISMATCH = 0x100, 0x200, 0x400, 0x800
R_BEYOND_PREDICATE = 0x1000
LOOKUP_UNKNOWN, LOOKUP_HIT, LOOKUP_PARTIAL, LOOKUP_MISS = 0, 1, 2, 3
NONE = 0xFFFFFFFF
RESERVED_ID = 0xFFFFFFFFFFFFFFFF
POOL_TIMING = 0x1
POOL_STAGE_TIMING = 0x2

OUTCOME_DTYPE = np.dtype(
    [("claim_id", "<u8"), ("code", "<u4"), ("first_failing_block", "<u4"), ("phys_block", "<u4"),
     ("num_blocks", "<u4"), ("reasons", "<u4"), ("intact_blocks", "<u4"), ("expected_digest", "<u8"),
     ("observed_digest", "<u8"), ("chain_hash", "<u8"), ("chain_hash_at_fail", "<u8")])
EVENT_DTYPE = np.dtype(
    [("seq", "<u8"), ("claim_id", "<u8"), ("aux", "<u8"), ("kind", "<u4"), ("block_index", "<u4"),
     ("phys_block", "<u4"), ("reserved", "<u4")])

LOOKUP_DTYPE = np.dtype(
    [("request_id", "<u8"), ("hit_tokens", "<u8"), ("chain_hash_at_hit", "<u8"), ("status", "<u4"),
     ("hit_blocks", "<u4"), ("last_block", "<u4"), ("reserved", "<u4")])

EXPORTS = ("claim_pool_create", "claim_pool_destroy", "claim_offload", "claim_restore",
           "claim_staging_reset", "claim_check", "claim_check_static", "claim_lookup",
           "claim_identity_stats", "outcomes_read", "claim_timing_read", "claim_block_state_read",
           "claim_digest_grid", "claim_strerror")


class PoolDesc(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_uint32), ("planes_per_layer", ctypes.c_uint32),
                ("block_size", ctypes.c_uint32), ("num_kv_heads", ctypes.c_uint32),
                ("head_dim", ctypes.c_uint32), ("elem_bytes", ctypes.c_uint32),
                ("num_blocks", ctypes.c_uint32), ("flags", ctypes.c_uint32),
                ("seed", ctypes.c_uint64), ("kv_base", ctypes.c_void_p),
                ("kv_bytes", ctypes.c_uint64), ("stream", ctypes.c_void_p),
                ("max_claims", ctypes.c_uint64), ("max_footprint", ctypes.c_uint64),
                ("event_capacity", ctypes.c_uint64), ("total_kv_heads", ctypes.c_uint32),
                ("first_kv_head", ctypes.c_uint32)]


class CBatch(ctypes.Structure):
    _fields_ = [("num_claims", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
                ("num_refs", ctypes.c_uint64), ("num_tokens", ctypes.c_uint64),
                ("claim_ids", ctypes.c_void_p), ("block_offsets", ctypes.c_void_p),
                ("block_ids", ctypes.c_void_p), ("token_offsets", ctypes.c_void_p),
                ("tokens", ctypes.c_void_p), ("predicate_tokens", ctypes.c_void_p)]


class CFaults(ctypes.Structure):
    _fields_ = [("num_flips", ctypes.c_uint32), ("num_load_failed", ctypes.c_uint32),
                ("flip_blocks", ctypes.c_void_p), ("flip_bits", ctypes.c_void_p),
                ("load_failed_blocks", ctypes.c_void_p)]


class CTiming(ctypes.Structure):
    _fields_ = [("calls", ctypes.c_uint32), ("last_unique", ctypes.c_uint32),
                ("total_ms", ctypes.c_double), ("digest_ms", ctypes.c_double),
                ("select_ms", ctypes.c_double), ("finalize_ms", ctypes.c_double),
                ("claims_ms", ctypes.c_double), ("events_ms", ctypes.c_double)]


class CGridInfo(ctypes.Structure):
    _fields_ = [("words_per_lane", ctypes.c_uint32), ("segments", ctypes.c_uint32),
                ("piece_groups", ctypes.c_uint32), ("slots", ctypes.c_uint32),
                ("pga", ctypes.c_uint32), ("groups", ctypes.c_uint32)]


assert ctypes.sizeof(PoolDesc) == 96 and ctypes.sizeof(CBatch) == 72
assert OUTCOME_DTYPE.itemsize == 64 and EVENT_DTYPE.itemsize == 40 and LOOKUP_DTYPE.itemsize == 40


class ClaimError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {strerror(status)} ({status})")


def build() -> str:
    """Compile libclaimkv.so for gfx950 in-tree."""
    tmp = LIBRARY + ".tmp"
    subprocess.run([HIPCC, *HIP_FLAGS, f"-I{INCLUDE}", SOURCE, "-o", tmp], check=True)
    os.replace(tmp, LIBRARY)
    return LIBRARY


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library.  Raises if it has not been built: there is no
    fallback path."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIBRARY):
            raise RuntimeError(f"{LIBRARY} is missing: build it (__graft_entry__.build())")
        L = ctypes.CDLL(LIBRARY)
        vp, i32, u32, u64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_uint32, ctypes.c_uint64
        sig = {
            "claim_pool_create": ([ctypes.POINTER(PoolDesc), ctypes.POINTER(vp)], i32),
            "claim_pool_destroy": ([vp], i32),
            "claim_offload": ([vp, ctypes.POINTER(CBatch), vp, u64], i32),
            "claim_restore": ([vp, ctypes.POINTER(CBatch), vp, u64, ctypes.POINTER(CFaults)], i32),
            "claim_staging_reset": ([vp], i32),
            "claim_check": ([vp, ctypes.POINTER(CBatch)], i32),
            "claim_check_static": ([vp, ctypes.POINTER(CBatch), vp, u32], i32),
            "claim_lookup": ([vp, ctypes.POINTER(CBatch), vp, u32], i32),
            "claim_identity_stats": ([vp, ctypes.POINTER(u64), ctypes.POINTER(u64)], i32),
            "outcomes_read": ([vp, vp, u32, ctypes.POINTER(u32), vp, u64, ctypes.POINTER(u64)], i32),
            "claim_timing_read": ([vp, ctypes.POINTER(CTiming)], i32),
            "claim_block_state_read": ([vp, u32, u32, vp, vp, vp, vp], i32),
            "claim_digest_grid": ([vp, u64, ctypes.POINTER(CGridInfo)], i32),
            "claim_strerror": ([i32], ctypes.c_char_p),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def strerror(status: int) -> str:
    return lib().claim_strerror(status).decode()


def _check(status: int, what: str) -> None:
    if status != OK:
        raise ClaimError(status, what)


def _torch():
    import torch

    return torch


class DeviceBatch:
    """A claim batch in device memory (torch tensors) plus its C struct.

    ``batch`` is any object with numpy arrays ``claim_ids`` (u64),
    ``block_offsets`` (u32), ``block_ids`` (u32), ``token_offsets`` (u64)
    and ``tokens`` (u32), and optionally ``predicate_tokens`` (u64 per claim
    or None).  The upload is complete when the constructor returns, so a
    pool on any stream may use the batch."""

    def __init__(self, batch, device="cuda"):
        torch = _torch()

        def up(a, np_dtype, t_dtype):
            a = np.ascontiguousarray(np.asarray(a, dtype=np_dtype))
            t = torch.from_numpy(a.view(t_dtype_np[t_dtype])).to(device)
            return t

        t_dtype_np = {torch.int64: np.int64, torch.int32: np.int32}
        self.ids = up(batch.claim_ids, np.uint64, torch.int64)
        self.bo = up(batch.block_offsets, np.uint32, torch.int32)
        self.bi = up(batch.block_ids, np.uint32, torch.int32)
        self.to = up(batch.token_offsets, np.uint64, torch.int64)
        self.tok = up(batch.tokens, np.uint32, torch.int32)
        pred = getattr(batch, "predicate_tokens", None)
        self.pred = None if pred is None else up(pred, np.uint64, torch.int64)
        # copies from pageable memory may still be in flight on the current
        # stream; the pool's kernels can run on another one
        torch.cuda.current_stream(self.ids.device).synchronize()
        n_claims = int(self.ids.numel())
        # the kernels read offsets[c + 1] and predicate[c] for every claim c
        if n_claims and (self.bo.numel() != n_claims + 1 or self.to.numel() != n_claims + 1):
            raise ValueError("block_offsets and token_offsets need num_claims + 1 entries")
        if self.pred is not None and self.pred.numel() != n_claims:
            raise ValueError("predicate_tokens needs one entry per claim")
        self.struct = CBatch(
            num_claims=n_claims, reserved=0, num_refs=int(self.bi.numel()),
            num_tokens=int(self.tok.numel()),
            claim_ids=self.ids.data_ptr() or None, block_offsets=self.bo.data_ptr() or None,
            block_ids=self.bi.data_ptr() or None, token_offsets=self.to.data_ptr() or None,
            tokens=self.tok.data_ptr() or None,
            predicate_tokens=(self.pred.data_ptr() or None) if self.pred is not None else None)

    @property
    def num_claims(self) -> int:
        return int(self.struct.num_claims)


class Pool:
    """A claim pool over a caller-owned KV tensor on the current GPU.

    ``geometry`` has num_layers, planes_per_layer, block_size, num_kv_heads,
    head_dim, elem_bytes and num_blocks, and for a head shard total_kv_heads
    and first_kv_head (e.g. ``synth.Geometry``); ``kv`` is a
    contiguous CUDA tensor of at least planes x num_blocks x chunk bytes laid
    out [plane][block][chunk]."""

    def __init__(self, geometry, seed: int, kv, *, stream=None, max_claims: int = 1 << 16,
                 max_footprint: int = 1 << 22, event_capacity: int = 1 << 20, timing: bool = False,
                 stage_timing: bool = False):
        torch = _torch()
        if not kv.is_cuda or not kv.is_contiguous():
            raise ValueError("kv must be a contiguous device tensor")
        if stream is None:
            stream = torch.cuda.current_stream(kv.device)
        self.kv = kv
        self.stream = stream
        self.geometry = geometry
        self.seed = seed
        d = PoolDesc(
            num_layers=geometry.num_layers, planes_per_layer=geometry.planes_per_layer,
            block_size=geometry.block_size, num_kv_heads=geometry.num_kv_heads,
            head_dim=geometry.head_dim, elem_bytes=geometry.elem_bytes,
            num_blocks=geometry.num_blocks,
            flags=(POOL_TIMING if timing else 0) | (POOL_STAGE_TIMING if stage_timing else 0), seed=seed,
            kv_base=kv.data_ptr(), kv_bytes=kv.numel() * kv.element_size(),
            stream=stream.cuda_stream, max_claims=max_claims, max_footprint=max_footprint,
            event_capacity=event_capacity,
            total_kv_heads=getattr(geometry, "total_kv_heads", 0),
            first_kv_head=getattr(geometry, "first_kv_head", 0))
        h = ctypes.c_void_p()
        with torch.cuda.device(kv.device):
            _check(lib().claim_pool_create(ctypes.byref(d), ctypes.byref(h)), "claim_pool_create")
        self._h = h
        self.event_capacity = event_capacity
        # device arrays of calls still queued on the pool's stream: the C ABI
        # needs them alive until that work completes, which the next call
        # that waits for the stream guarantees
        self._inflight = []

    def close(self) -> None:
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            _check(lib().claim_pool_destroy(h), "claim_pool_destroy")
        self._h = None
        self._inflight = []

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # --------------------------------------------------------------- calls
    def offload(self, batch: DeviceBatch, staging=None, staging_bytes: int | None = None) -> None:
        ptr, nbytes = _staging_args(staging, staging_bytes)
        _check(lib().claim_offload(self._h, ctypes.byref(batch.struct), ptr, nbytes), "claim_offload")
        self._inflight = []  # claim_offload ends by waiting for the stream

    def restore(self, batch: DeviceBatch, staging=None, faults=None,
                staging_bytes: int | None = None) -> None:
        ptr, nbytes = _staging_args(staging, staging_bytes)
        keep = []
        fs = None
        if faults is not None:
            fb = np.ascontiguousarray(faults.flip_blocks, dtype=np.uint32)
            fbits = np.ascontiguousarray(faults.flip_bits, dtype=np.uint64)
            lf = np.ascontiguousarray(faults.load_failed, dtype=np.uint32)
            keep = [fb, fbits, lf]
            fs = CFaults(num_flips=fb.size, num_load_failed=lf.size,
                         flip_blocks=fb.ctypes.data if fb.size else None,
                         flip_bits=fbits.ctypes.data if fbits.size else None,
                         load_failed_blocks=lf.ctypes.data if lf.size else None)
        _check(lib().claim_restore(self._h, ctypes.byref(batch.struct), ptr, nbytes,
                                   ctypes.byref(fs) if fs is not None else None), "claim_restore")
        del keep  # host fault lists: read before claim_restore returns
        self._inflight += [batch, staging]

    def staging_reset(self) -> None:
        """claim_staging_reset: the next staged offload starts a new
        staging generation."""
        _check(lib().claim_staging_reset(self._h), "claim_staging_reset")

    def check(self, batch: DeviceBatch) -> None:
        _check(lib().claim_check(self._h, ctypes.byref(batch.struct)), "claim_check")
        self._inflight.append(batch)

    def check_static(self, batch: DeviceBatch, out=None):
        """claim_check_static: the check with no allocation by the library;
        outcomes go to ``out`` (a device uint8 tensor of 64 bytes per claim,
        made here if None), which is returned."""
        torch = _torch()
        n = batch.num_claims
        if out is None:
            out = torch.empty(max(1, n) * OUTCOME_DTYPE.itemsize, dtype=torch.uint8,
                              device=self.kv.device)
        cap = out.numel() // OUTCOME_DTYPE.itemsize
        _check(lib().claim_check_static(self._h, ctypes.byref(batch.struct), out.data_ptr(), cap),
               "claim_check_static")
        self._inflight += [batch, out]
        return out

    def lookup_async(self, batch: DeviceBatch, out=None):
        """Queue a reuse lookup of the batch's token rows on the pool stream;
        returns the device tensor (uint8, 40 bytes per row) it fills."""
        torch = _torch()
        n = batch.num_claims
        if out is None:
            out = torch.empty(max(1, n) * LOOKUP_DTYPE.itemsize, dtype=torch.uint8,
                              device=self.kv.device)
        cap = out.numel() // LOOKUP_DTYPE.itemsize
        _check(lib().claim_lookup(self._h, ctypes.byref(batch.struct), out.data_ptr(), cap),
               "claim_lookup")
        self._inflight += [batch, out]
        return out

    def lookup(self, batch: DeviceBatch) -> np.ndarray:
        """Reuse lookup of the batch's token rows, read back to the host."""
        out = self.lookup_async(batch)
        self.stream.synchronize()
        self._inflight = []
        return out.cpu().numpy().view(LOOKUP_DTYPE)[: batch.num_claims].copy()

    def identity_stats(self) -> tuple[int, int]:
        """(registered identities, ambiguous identities)."""
        e, a = ctypes.c_uint64(), ctypes.c_uint64()
        _check(lib().claim_identity_stats(self._h, ctypes.byref(e), ctypes.byref(a)),
               "claim_identity_stats")
        self._inflight = []  # waited for the stream
        return int(e.value), int(a.value)

    def read(self, max_outcomes: int = 1 << 22, max_events: int | None = None, out=None,
             events=None):
        """(outcomes of the last check, events since the last read).

        With ``out`` / ``events`` (host arrays of OUTCOME_DTYPE / EVENT_DTYPE,
        for instance views of page-locked memory) the records are written
        there and views of them are returned; otherwise into new arrays."""
        if out is None:
            out = np.zeros(max_outcomes, dtype=OUTCOME_DTYPE)
            fresh_out = True
        else:
            assert out.dtype == OUTCOME_DTYPE and out.flags["C_CONTIGUOUS"]
            fresh_out = False
        if events is None:
            events = np.zeros(self.event_capacity if max_events is None else max_events,
                              dtype=EVENT_DTYPE)
            fresh_ev = True
        else:
            assert events.dtype == EVENT_DTYPE and events.flags["C_CONTIGUOUS"]
            fresh_ev = False
        n_out = ctypes.c_uint32()
        n_ev = ctypes.c_uint64()
        _check(lib().outcomes_read(self._h, out.ctypes.data, out.size, ctypes.byref(n_out),
                                   events.ctypes.data, events.size, ctypes.byref(n_ev)),
               "outcomes_read")
        self._inflight = []  # waited for the stream
        o, e = out[: n_out.value], events[: n_ev.value]
        return (o.copy() if fresh_out else o), (e.copy() if fresh_ev else e)

    def block_state(self, first: int = 0, count: int | None = None) -> dict:
        """Per-block digests and flags of blocks [first, first + count)."""
        if count is None:
            count = self.geometry.num_blocks - first
        d_off = np.zeros(count, np.uint64)
        d_res = np.zeros(count, np.uint64)
        valid = np.zeros(count, np.uint8)
        failed = np.zeros(count, np.uint8)
        _check(lib().claim_block_state_read(self._h, first, count, d_off.ctypes.data,
                                            d_res.ctypes.data, valid.ctypes.data,
                                            failed.ctypes.data), "claim_block_state_read")
        self._inflight = []  # waited for the stream
        return {"d_off": d_off, "d_res": d_res, "valid_off": valid, "load_failed": failed}

    def digest_grid(self, refs: int | None = None) -> dict:
        """The digest grid of a launch over ``refs`` block-table entries
        (default: as many as the pool has blocks)."""
        g = CGridInfo()
        n = self.geometry.num_blocks if refs is None else refs
        _check(lib().claim_digest_grid(self._h, n, ctypes.byref(g)), "claim_digest_grid")
        return {name: getattr(g, name) for name, _ in CGridInfo._fields_}

    def timing(self) -> dict:
        t = CTiming()
        _check(lib().claim_timing_read(self._h, ctypes.byref(t)), "claim_timing_read")
        return {name: getattr(t, name) for name, _ in CTiming._fields_}


def _staging_args(staging, nbytes):
    if staging is None:
        return None, 0
    if hasattr(staging, "data_ptr"):
        return staging.data_ptr(), nbytes if nbytes is not None else staging.numel() * staging.element_size()
    return int(staging), int(nbytes or 0)
