"""Synthetic pool content: host generator (C) and GPU fill (HIP).

Both implement the definition in ``content_host.c`` (Philox4x32-10 counters
per 16-byte unit).  The host side serves the oracle (canonical bytes of the
blocks it digests); the GPU side fills pools that are too large to build on
the host.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from .workloads import Geometry

_HERE = os.path.dirname(os.path.abspath(__file__))
HOST_SRC = os.path.join(_HERE, "content_host.c")
HOST_LIB = os.path.join(_HERE, "libsynth_host.so")
FILL_SRC = os.path.join(_HERE, "fill.hip")
FILL_LIB = os.path.join(_HERE, "libsynth_fill.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-shared", "-std=c++17",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def build() -> None:
    """Compile the host generator (gcc) and the GPU fill (hipcc, gfx950)."""
    tmp = HOST_LIB + ".tmp"
    subprocess.run(["gcc", "-O3", "-std=c99", "-shared", "-fPIC", HOST_SRC, "-o", tmp], check=True)
    os.replace(tmp, HOST_LIB)
    tmp = FILL_LIB + ".tmp"
    subprocess.run([HIPCC, *HIP_FLAGS, FILL_SRC, "-o", tmp], check=True)
    os.replace(tmp, FILL_LIB)


_host = None
_fill = None


def _host_lib():
    global _host
    if _host is None:
        if not os.path.exists(HOST_LIB):
            raise RuntimeError(f"{HOST_LIB} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(HOST_LIB)
        vp, u32, u64 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64
        L.synth_philox4x32_10.argtypes = [vp, vp, vp]
        L.synth_philox4x32_10.restype = None
        L.synth_block_canonical.argtypes = [u64, ctypes.c_int, u32, u64, u32, vp]
        L.synth_block_canonical.restype = ctypes.c_int
        L.synth_pool_host.argtypes = [u64, ctypes.c_int, u32, u32, u64, vp]
        L.synth_pool_host.restype = ctypes.c_int
        _host = L
    return _host


def _fill_lib():
    global _fill
    if _fill is None:
        if not os.path.exists(FILL_LIB):
            raise RuntimeError(f"{FILL_LIB} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(FILL_LIB)
        vp, u32, u64 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64
        L.synth_fill_pool.argtypes = [vp, u64, u64, ctypes.c_int, u32, u32, u64, vp]
        L.synth_fill_pool.restype = ctypes.c_int
        L.synth_copy_probe.argtypes = [vp, vp, u64, vp]
        L.synth_copy_probe.restype = ctypes.c_int
        L.synth_read_probe.argtypes = [vp, u64, u32, vp, vp]
        L.synth_read_probe.restype = ctypes.c_int
        _fill = L
    return _fill


def philox4x32_10(ctr, key) -> list[int]:
    c = np.asarray(ctr, dtype=np.uint32)
    k = np.asarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    _host_lib().synth_philox4x32_10(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return [int(x) for x in out]


def block_canonical(g: Geometry, content_seed: int, b: int) -> np.ndarray:
    """Canonical bytes (planes concatenated) of pool block b."""
    out = np.empty(g.block_bytes, dtype=np.uint8)
    rc = _host_lib().synth_block_canonical(content_seed, int(g.raw_bytes), g.planes,
                                           g.chunk_bytes, b, out.ctypes.data)
    if rc:
        raise ValueError("chunk size must be a multiple of 16 bytes")
    return out


def pool_host(g: Geometry, content_seed: int) -> np.ndarray:
    """The whole pool, [plane][block][chunk] bytes (small pools only)."""
    if g.pool_bytes > (1 << 31):
        raise ValueError("pool too large to build on the host")
    out = np.empty(g.pool_bytes, dtype=np.uint8)
    rc = _host_lib().synth_pool_host(content_seed, int(g.raw_bytes), g.planes, g.num_blocks,
                                     g.chunk_bytes, out.ctypes.data)
    if rc:
        raise ValueError("chunk size must be a multiple of 16 bytes")
    return out


def fill_pool_gpu(ptr: int, nbytes: int, g: Geometry, content_seed: int, stream: int) -> None:
    """Fill device memory at ``ptr`` with the pool's content on ``stream``."""
    rc = _fill_lib().synth_fill_pool(ptr, nbytes, content_seed, int(g.raw_bytes), g.planes,
                                     g.num_blocks, g.chunk_bytes, stream)
    if rc:
        raise RuntimeError(f"synth_fill_pool failed ({rc})")


def copy_probe(dst: int, src: int, nbytes: int, stream: int) -> None:
    """Plain streaming copy (the checker's load form), for counter calibration."""
    rc = _fill_lib().synth_copy_probe(dst, src, nbytes, stream)
    if rc:
        raise RuntimeError(f"synth_copy_probe failed ({rc})")


def read_probe(src: int, nbytes: int, cus: int, sink: int, stream: int) -> None:
    """Plain streaming read of a buffer (the measured bandwidth ceiling)."""
    rc = _fill_lib().synth_read_probe(src, nbytes, cus, sink, stream)
    if rc:
        raise RuntimeError(f"synth_read_probe failed ({rc})")
