"""The C ABI library on the CPU: it loads, exports every declared entry
point, its record layouts match the header, and argument errors are reported
before any GPU work (none of these calls touches a GPU)."""

import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2606_01387_amd import claimkv as ck

HEADER = os.path.join(ck.INCLUDE, "claimkv.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(ck.LIBRARY):
        ck.build()
    return ck.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)))


def test_every_declared_function_is_exported(L):
    names = declared_functions()
    assert set(names) == set(ck.EXPORTS)
    for n in names:
        assert hasattr(L, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", ck.LIBRARY], capture_output=True,
                         text=True, check=True).stdout
    exported = {ln.split()[-1] for ln in out.splitlines() if " T " in ln}
    assert exported == set(names)


def test_record_layouts_match_header(tmp_path):
    fields = {
        "claim_outcome": list(ck.OUTCOME_DTYPE.names),
        "claim_event": list(ck.EVENT_DTYPE.names),
        "claim_lookup_result": list(ck.LOOKUP_DTYPE.names),
        "claim_pool_desc": [f for f, _ in ck.PoolDesc._fields_],
        "claim_batch": [f for f, _ in ck.CBatch._fields_],
        "claim_fault_spec": [f for f, _ in ck.CFaults._fields_],
        "claim_timing": [f for f, _ in ck.CTiming._fields_],
        "claim_grid_info": [f for f, _ in ck.CGridInfo._fields_],
    }
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "claimkv.h"', "int main(void){"]
    for st, fs in fields.items():
        lines.append(f'printf("{st} %zu\\n", sizeof({st}));')
        for f in fs:
            lines.append(f'printf("{st}.{f} %zu\\n", offsetof({st}, {f}));')
    lines.append("return 0;}")
    src = tmp_path / "probe.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "probe"
    subprocess.run(["gcc", f"-I{ck.INCLUDE}", str(src), "-o", str(exe)], check=True)
    got = dict(ln.split() for ln in subprocess.run([str(exe)], capture_output=True, text=True,
                                                   check=True).stdout.splitlines())
    for dt, st in ((ck.OUTCOME_DTYPE, "claim_outcome"), (ck.EVENT_DTYPE, "claim_event"),
                   (ck.LOOKUP_DTYPE, "claim_lookup_result")):
        assert int(got[st]) == dt.itemsize
        for f in dt.names:
            assert int(got[f"{st}.{f}"]) == dt.fields[f][1], (st, f)
    for cls, st in ((ck.PoolDesc, "claim_pool_desc"), (ck.CBatch, "claim_batch"),
                    (ck.CFaults, "claim_fault_spec"), (ck.CTiming, "claim_timing"),
                    (ck.CGridInfo, "claim_grid_info")):
        assert int(got[st]) == ctypes.sizeof(cls)
        for f, _ in cls._fields_:
            assert int(got[f"{st}.{f}"]) == getattr(cls, f).offset, (st, f)


def test_strerror(L):
    for code in (ck.OK, ck.EINVAL, ck.ENOMEM, ck.EHIP, ck.ENOSPC, ck.EDUP, ck.ELIMIT):
        assert ck.strerror(code) != "unknown status"
    assert ck.strerror(-99) == "unknown status"
    assert "duplicate" in ck.strerror(ck.EDUP)


def _desc(**kw):
    d = dict(num_layers=2, planes_per_layer=2, block_size=16, num_kv_heads=2, head_dim=64,
             elem_bytes=2, num_blocks=64, flags=0, seed=1, kv_base=0x10000, kv_bytes=1 << 20,
             stream=None, max_claims=16, max_footprint=128, event_capacity=64)
    d.update(kw)
    return ck.PoolDesc(**d)


@pytest.mark.parametrize("bad", [
    dict(num_layers=0), dict(planes_per_layer=3), dict(block_size=0), dict(block_size=2048),
    dict(num_kv_heads=0), dict(head_dim=0), dict(elem_bytes=0), dict(num_blocks=0),
    dict(num_blocks=0xFFFFFFFF), dict(kv_base=None), dict(kv_base=0x10008),
    dict(kv_bytes=(1 << 20) - 1), dict(max_claims=0), dict(event_capacity=0), dict(flags=0x80),
    dict(flags=0x4),
    # head shards: past the full block's heads, or head rows that are not whole words
    dict(total_kv_heads=4, first_kv_head=3), dict(first_kv_head=1), dict(total_kv_heads=1),
    dict(head_dim=2, elem_bytes=1, total_kv_heads=4),
])
def test_pool_create_rejects_bad_descriptions(L, bad):
    d = _desc(**bad)
    h = ctypes.c_void_p()
    rc = L.claim_pool_create(ctypes.byref(d), ctypes.byref(h))
    assert rc == ck.EINVAL and not h.value


@pytest.mark.parametrize("ok", [dict(total_kv_heads=8, first_kv_head=6), dict(total_kv_heads=2),
                                dict(total_kv_heads=0, first_kv_head=0),
                                dict(flags=ck.POOL_TIMING | ck.POOL_STAGE_TIMING)])
def test_pool_create_accepts_head_shards(L, ok):
    """Valid head-shard descriptions and flags pass validation (without a GPU the
    call then fails in the runtime, never with EINVAL)."""
    d = _desc(**ok)
    h = ctypes.c_void_p()
    rc = L.claim_pool_create(ctypes.byref(d), ctypes.byref(h))
    assert rc != ck.EINVAL
    if rc == ck.OK:
        L.claim_pool_destroy(h)


def test_chunk_must_be_multiple_of_16_bytes(L):
    d = _desc(head_dim=3, elem_bytes=1, num_kv_heads=1, block_size=5)  # 15-byte chunk
    h = ctypes.c_void_p()
    assert L.claim_pool_create(ctypes.byref(d), ctypes.byref(h)) == ck.EINVAL


def test_null_arguments_are_rejected(L):
    h = ctypes.c_void_p()
    assert L.claim_pool_create(None, ctypes.byref(h)) == ck.EINVAL
    assert L.claim_pool_create(ctypes.byref(_desc()), None) == ck.EINVAL
    b = ck.CBatch()
    assert L.claim_offload(None, ctypes.byref(b), None, 0) == ck.EINVAL
    assert L.claim_restore(None, ctypes.byref(b), None, 0, None) == ck.EINVAL
    assert L.claim_staging_reset(None) == ck.EINVAL
    assert L.claim_check(None, ctypes.byref(b)) == ck.EINVAL
    assert L.claim_check_static(None, ctypes.byref(b), None, 0) == ck.EINVAL
    assert L.outcomes_read(None, None, 0, None, None, 0, None) == ck.EINVAL
    assert L.claim_timing_read(None, None) == ck.EINVAL
    assert L.claim_block_state_read(None, 0, 0, None, None, None, None) == ck.EINVAL
    assert L.claim_lookup(None, ctypes.byref(b), None, 0) == ck.EINVAL
    assert L.claim_identity_stats(None, None, None) == ck.EINVAL
    g = ck.CGridInfo()
    assert L.claim_digest_grid(None, 0, ctypes.byref(g)) == ck.EINVAL
    assert L.claim_pool_destroy(None) == ck.OK


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(ck, "LIBRARY", str(tmp_path / "missing.so"))
    monkeypatch.setattr(ck, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        ck.lib()
