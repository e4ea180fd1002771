"""Benchmark: verified claim-KV bandwidth of claim_check on one MI355X.

One step = one claim_check call over the whole batch: select the unique
referenced blocks, gather + digest them (the HBM-bound kernel), combine the
block digests, then per claim chain the token hash, compare, min-reduce to
the outcome and append the ordered events.  The pool, the batch and the
offload record are resident in HBM before the timed region starts.

Prints one JSON line.  ``value`` is the physical verified bandwidth: unique
physical block bytes digested and checked per second (each physical block
is read once however many claims alias it).
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "verified claim-KV GB/s (gather+digest+compare) and claims/s; % of HBM peak"
HBM_PEAK_GBPS = 8000.0  # MI355X published HBM3E bandwidth


def digest_traffic(workload: str):
    """Calibrated HBM bytes per digest launch from the committed counter
    summary, or None if there is none or the kernel source changed since."""
    import hashlib

    path = os.path.join(ROOT, "profiles", f"k_digest_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    if "```json" not in text:
        return None
    data = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
    src = os.path.join(ROOT, data["source"])
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != data["source_sha256"]:
        return None
    return int(data["traffic_bytes_per_launch"])


def cpu_baseline(w, batch, faults, sample_gb: float):
    """The oracle as it stands, single-threaded, on a bounded sample of the
    workload: the unique blocks are taken in order up to `sample_gb` of block
    bytes (all of them when they fit), their content is generated untimed on
    all host threads and their restored bytes (the flips applied) are
    digested by the oracle, timed; the per-byte rate is extrapolated to the
    whole unique set.  The claim stage (chain, compare, min-reduction,
    events) runs on the whole batch, timed.  Digests of blocks outside the
    sample are modeled (equal before and after, real for changed blocks).
    Returns the baseline record, the oracle's outcomes and events, its
    per-block digests and the blocks whose digests are real."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    from oracle import oracle as O
    from paper_2606_01387_amd.synth import content
    from oracle.pool_digests import canon_digest, modeled_digests

    g = w.geometry
    uniq = batch.unique_blocks(g.num_blocks)
    n_sample = int(min(uniq.size, max(1, sample_gb * 1e9 // g.block_bytes)))
    blocks = uniq[:n_sample]
    changed = set(int(b) for b in faults.changed_blocks())
    flips = {}
    for b, bit in zip(faults.flip_blocks, faults.flip_bits):
        flips.setdefault(int(b), []).append(int(bit))
    d0, d1 = modeled_digests(w, faults, blocks_needed=[])
    threads = max(1, min(16, os.cpu_count() or 1))
    t_digest = 0.0
    t_gen = time.perf_counter()
    with ThreadPoolExecutor(threads) as ex:
        for lo in range(0, n_sample, 256):
            part = [int(b) for b in blocks[lo:lo + 256]]
            canon = list(ex.map(lambda b: content.block_canonical(g, w.content_seed, b), part))
            for b, c in zip(part, canon):
                for bit in flips.get(b, []):  # restored bytes
                    c[bit // 8] ^= np.uint8(1 << (bit % 8))
            t0 = time.perf_counter()
            for b, c in zip(part, canon):
                d1[b] = canon_digest(c, w)
            t_digest += time.perf_counter() - t0
            for b in part:  # a changed block's d0 is already its real pre-flip digest
                if b not in changed:
                    d0[b] = d1[b]
    t_gen = time.perf_counter() - t_gen - t_digest
    op = O.OraclePool(g.num_blocks, g.block_size, w.seed)
    op.offload(batch, d0)
    op.restore(batch, faults.load_failed)
    op.events(clear=True)
    t0 = time.perf_counter()
    out = op.check(batch, d1)
    t_claims = time.perf_counter() - t0
    ev = op.events()
    per_byte = t_digest / (n_sample * g.block_bytes)
    t_check = per_byte * uniq.size * g.block_bytes + t_claims
    gbps = uniq.size * g.block_bytes / t_check / 1e9
    whole = n_sample == uniq.size
    real = np.union1d(blocks, np.array(sorted(changed | set(int(b) for b in faults.load_failed)),
                                       dtype=np.int64)).astype(np.int64)
    sample = (f"single-threaded oracle: digest of the restored bytes of "
              f"{'all ' if whole else ''}{n_sample} of {uniq.size} unique blocks "
              f"({n_sample * g.block_bytes / 1e9:.2f} GB) timed in {t_digest:.2f} s"
              + ("" if whole else " and extrapolated per byte to the whole unique set")
              + f"; claim stage on all {batch.num_claims} claims timed in {t_claims:.3f} s; "
              f"content generated untimed on {threads} host threads in {t_gen:.1f} s")
    return {
        "value": round(gbps, 4),
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "sample": sample,
        "claims_per_s": round(batch.num_claims / t_check, 2),
        "host_cpus": os.cpu_count(),
        "host_cpu_model": _cpu_model(),
    }, out, ev, d0, d1, real


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama3-8b")
    ap.add_argument("--geometry", default=None,
                    help="layers,planes_per_layer,block_size,kv_heads,head_dim,elem_bytes,num_blocks: "
                         "the workload's claims and faults over a pool of this geometry")
    ap.add_argument("--cpu-sample-gb", type=float, default=20.0,
                    help="block bytes the oracle digests for the CPU baseline (whole unique set "
                         "if it is smaller)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--round-trip", action="store_true",
                    help="offload through pinned host staging, drop the device copy, restore from "
                         "staging; time the two transfers separately from the on-device verify")
    ap.add_argument("--stages", action="store_true",
                    help="also time every stage of the check (two more hipEvents per stage)")
    ap.add_argument("--copy-probe-gib", type=float, default=0.0,
                    help="run one plain device copy of this size first (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this checker runs one pool per GPU and has no "
              "multi-GPU path; run it with --gpus 1", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2606_01387_amd import claimkv as ck
    from paper_2606_01387_amd.synth import FULL, SHARDS, content, make_batch, make_faults, make_requests

    w = FULL[args.workload] if args.workload in FULL else SHARDS[args.workload]
    if args.geometry:
        from dataclasses import replace

        from paper_2606_01387_amd.synth import Geometry

        dims = [int(x) for x in args.geometry.split(",")]
        w = replace(w, name=f"{w.name}-claims-on-{'x'.join(map(str, dims))}", geometry=Geometry(*dims))
    g = w.geometry
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)

    batch = make_batch(w)
    faults = make_faults(w, batch)
    uniq = batch.unique_blocks(g.num_blocks)
    U, C = int(uniq.size), batch.num_claims
    present_refs = int((batch.block_ids < g.num_blocks).sum())

    if args.copy_probe_gib > 0:
        # a plain copy kernel that reads and writes exactly n bytes with the
        # checker's load form: the reference for scaling the HBM counters
        n = int(args.copy_probe_gib * (1 << 30))
        a = torch.zeros(n, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        content.copy_probe(b.data_ptr(), a.data_ptr(), n, stream.cuda_stream)
        torch.cuda.synchronize()
        del a, b

    kv = torch.empty(g.pool_bytes, dtype=torch.uint8, device=dev)
    content.fill_pool_gpu(kv.data_ptr(), kv.numel(), g, w.content_seed, stream.cuda_stream)

    # measured streaming-read ceiling of this machine (context for the roofline)
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    sink = torch.zeros(1, dtype=torch.int32, device=dev)
    probe_ms = []
    for _ in range(4):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        content.read_probe(kv.data_ptr(), kv.numel(), cus, sink.data_ptr(), stream.cuda_stream)
        e1.record(stream)
        e1.synchronize()
        probe_ms.append(e0.elapsed_time(e1))
    probe_bytes = kv.numel() // 32768 * 32768
    read_ceiling = probe_bytes / (sorted(probe_ms)[1] * 1e-3) / 1e9
    db = ck.DeviceBatch(batch, device=dev)
    steps, warm = args.steps, args.warmup
    pool = ck.Pool(g, w.seed, kv, stream=stream, max_claims=2 * C, max_footprint=2 * batch.num_refs,
                   event_capacity=2 * C * (steps + warm + 2) + 4 * C, timing=True,
                   stage_timing=args.stages)
    round_trip = None
    lifecycle = None
    if args.round_trip:
        # the host-link leg of the lifecycle: gather + digest straight into
        # pinned host memory, lose the device copy, scatter back from host
        staging = torch.empty(U * g.block_bytes, dtype=torch.uint8, pin_memory=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        pool.offload(db, staging=staging)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        kv.zero_()
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        pool.restore(db, staging=staging, faults=faults)
        torch.cuda.synchronize()
        t3 = time.perf_counter()
        moved = U * g.block_bytes
        # the copy engine's own rates over the same pinned buffer and bytes:
        # the host-link ceiling the kernels are measured against
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        scratch_dev = torch.empty(moved, dtype=torch.uint8, device=kv.device)  # not the pool
        ev[0].record(stream)
        staging.copy_(kv[:moved], non_blocking=True)  # reads the pool, writes the spent staging
        ev[1].record(stream)
        scratch_dev.copy_(staging, non_blocking=True)
        ev[2].record(stream)
        ev[2].synchronize()
        del scratch_dev
        d2h = moved / (ev[0].elapsed_time(ev[1]) * 1e-3) / 1e9
        h2d = moved / (ev[1].elapsed_time(ev[2]) * 1e-3) / 1e9
        off_gbps = moved / (t1 - t0) / 1e9
        res_gbps = moved / (t3 - t2) / 1e9
        round_trip = {
            "staging": "pinned host memory (hipHostMalloc), written and read by the kernels",
            "bytes": moved,
            "offload_ms": round((t1 - t0) * 1e3, 3),
            "offload_GBps": round(off_gbps, 2),
            "restore_ms": round((t3 - t2) * 1e3, 3),
            "restore_GBps": round(res_gbps, 2),
            "copy_engine_d2h_GBps": round(d2h, 2),
            "copy_engine_h2d_GBps": round(h2d, 2),
            "offload_frac_of_copy_engine": round(off_gbps / d2h, 4),
            "restore_frac_of_copy_engine": round(res_gbps / h2d, 4),
            "host_link_nominal_GBps": 64.0,
            "note": "whole claim_offload / claim_restore calls (acceptance, digest, events "
                    "included); copy-engine rates are plain pinned<->device copies of the "
                    "same bytes; nominal link is PCIe Gen5 x16 per direction; the timed "
                    "verify below runs on the restored pool",
        }
        del staging
    else:
        # the lifecycle steps before the checks, timed once (whole calls,
        # including their waits on the stream); not part of the check's value
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        pool.offload(db)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        pool.restore(db, faults=faults)
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        lifecycle = {"offload_ms": round((t1 - t0) * 1e3, 3), "restore_ms": round((t2 - t1) * 1e3, 3),
                     "note": "claim_offload (acceptance, identity registration, offload digest) and "
                             "claim_restore (faults, RESTORE_REQUIRED) on the device-resident pool, "
                             "wall time of one call each, including the offload's host waits"}
    pool.read(max_outcomes=1)
    grid = pool.digest_grid(batch.num_refs)

    for _ in range(warm):
        pool.check(db)
    torch.cuda.synchronize()
    pool.timing()  # discard warm-up stage times

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        pool.check(db)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    stages = pool.timing()
    out, ev = pool.read()
    state = pool.block_state()

    # outcomes_read of one check (its outcomes and events, D2H), timed apart:
    # into page-locked host buffers, then into new pageable arrays
    out_pin = torch.empty(max(1, C) * ck.OUTCOME_DTYPE.itemsize, dtype=torch.uint8, pin_memory=True)
    ev_pin = torch.empty((2 * C + 16) * ck.EVENT_DTYPE.itemsize, dtype=torch.uint8, pin_memory=True)
    read = {}
    for kind in ("pinned", "pageable"):
        pool.check(db)
        torch.cuda.synchronize()
        r0 = time.perf_counter()
        if kind == "pinned":
            o1, e1 = pool.read(out=out_pin.numpy().view(ck.OUTCOME_DTYPE),
                               events=ev_pin.numpy().view(ck.EVENT_DTYPE))
        else:
            o1, e1 = pool.read(max_outcomes=max(1, C), max_events=2 * C + 16)
        r1 = time.perf_counter()
        assert np.array_equal(o1, out), "a repeated check read back other outcomes"
        nbytes = o1.size * ck.OUTCOME_DTYPE.itemsize + e1.size * ck.EVENT_DTYPE.itemsize
        read[kind] = (r1 - r0, nbytes, int(e1.size))
    del out_pin, ev_pin

    # spread of single checks, in a separate pass after the timed region:
    # hipEvents on the pool stream around each check
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    marks[0].record(stream)
    for i in range(steps):
        pool.check(db)
        marks[i + 1].record(stream)
    marks[-1].synchronize()
    per_check = np.array([marks[i].elapsed_time(marks[i + 1]) for i in range(steps)])

    # reuse lookup of as many requests as claims, timed apart from the check
    reqs, _ = make_requests(w, batch)
    dreq = ck.DeviceBatch(reqs)
    lk_buf = pool.lookup_async(dreq)
    l0, l1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    l0.record(stream)
    for _ in range(steps):
        pool.lookup_async(dreq, out=lk_buf)
    l1.record(stream)
    l1.synchronize()
    lookup_ms = l0.elapsed_time(l1) / steps
    lk = lk_buf.cpu().numpy().view(ck.LOOKUP_DTYPE)[: reqs.num_claims]
    identities = pool.identity_stats()
    pool.close()

    ms_per_step = (t1 - t0) * 1e3 / steps
    phys_bytes = U * g.block_bytes
    meta_bytes = (8 * C + 4 * (C + 1) + 4 * batch.num_refs + 8 * (C + 1) + 4 * batch.num_tokens
                  + 64 * C + 40 * len(ev) // max(1, steps + warm))
    value = phys_bytes / (ms_per_step * 1e-3) / 1e9
    digest_ms = stages["digest_ms"] / max(1, stages["calls"])
    achieved = phys_bytes / (digest_ms * 1e-3) / 1e9
    n_fail = int((out["code"] == ck.RESTORE_FAILED_FAIL_CLOSED).sum())

    line = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warm,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "num_blocks": g.num_blocks,
            "block_bytes": g.block_bytes,
            "unique_blocks": U,
            "claims": C,
            "block_refs": batch.num_refs,
            **({"kv_heads": f"{g.first_kv_head}..{g.first_kv_head + g.num_kv_heads - 1} of "
                            f"{g.total_kv_heads} (head shard)"} if g.sharded else {}),
            "tokens": batch.num_tokens,
            "corrupted_blocks": int(faults.flip_blocks.size),
        },
        "check_ms_p10_p50_p90": [round(float(np.percentile(per_check, q)), 4) for q in (10, 50, 90)],
        "claims_per_s": round(C / (ms_per_step * 1e-3), 1),
        "logical_GBps": round(present_refs * g.block_bytes / (ms_per_step * 1e-3) / 1e9, 2),
        "pct_hbm_peak": round(100 * (phys_bytes + meta_bytes) / (ms_per_step * 1e-3) / 1e9
                              / HBM_PEAK_GBPS, 2),
        "stage_ms": {k: round(stages[k] / max(1, stages["calls"]), 4)
                     for k in (("select_ms", "digest_ms", "finalize_ms", "claims_ms", "events_ms")
                               if args.stages else ("digest_ms",))},
        "outcomes": {"failed_closed": n_fail, "materialized": int((out["code"] == ck.MATERIALIZED).sum()),
                     "unknown": int((out["code"] == ck.UNKNOWN).sum())},
        "roofline": {
            "bound": "hbm",
            "kernel": "k_digest",
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": digest_traffic(w.name),
            "traffic_unit": "bytes/launch",
            "bytes_per_launch": phys_bytes,
            "avg_launch_ms": round(digest_ms, 4),
            "measured_read_ceiling": round(read_ceiling, 1),
            "frac_of_read_ceiling": round(achieved / read_ceiling, 4),
            "digest_grid": {
                "words_per_lane": grid["words_per_lane"],
                "piece_groups": grid["piece_groups"],
                "piece_groups_at_a_time": grid["pga"],
                "workgroups_each": grid["groups"],
                "phases": grid["piece_groups"] // grid["pga"],
                "workgroups": grid["pga"] * grid["groups"],
            },
        },
    }
    line["lookup"] = {
        "requests": reqs.num_claims,
        "request_tokens": reqs.num_tokens,
        "ms": round(lookup_ms, 4),
        "requests_per_s": round(reqs.num_claims / (lookup_ms * 1e-3), 1),
        "tokens_per_s": round(reqs.num_tokens / (lookup_ms * 1e-3), 1),
        "hit_tokens": int(lk["hit_tokens"].sum()),
        "status_unknown_hit_partial_miss": np.bincount(lk["status"], minlength=4).tolist(),
        "identities_registered_ambiguous": list(identities),
    }
    line["outcomes_read"] = {
        "bytes": read["pinned"][1],
        "outcomes": int(out.size),
        "events": read["pinned"][2],
        "pinned_ms": round(read["pinned"][0] * 1e3, 3),
        "pinned_GBps": round(read["pinned"][1] / read["pinned"][0] / 1e9, 2),
        "pageable_ms": round(read["pageable"][0] * 1e3, 3),
        "pageable_GBps": round(read["pageable"][1] / read["pageable"][0] / 1e9, 2),
        "note": "one outcomes_read call after one more check: that check's outcomes and events, "
                "D2H into page-locked host buffers, then into new pageable arrays (synchronous "
                "copies, host wall time)",
    }
    if round_trip is not None:
        line["round_trip"] = round_trip
    if lifecycle is not None:
        line["lifecycle"] = lifecycle
    if not args.no_cpu_baseline:
        base, want, want_ev, d0, d1, real = cpu_baseline(w, batch, faults, args.cpu_sample_gb)
        line["cpu_baseline"] = base
        # the last timed check against the oracle: every outcome field, that
        # check's events, and the digests of every block the oracle digested
        same_out = all(np.array_equal(out[f], want[f]) for f in want.dtype.names)
        k = len(want_ev)
        last = ev[len(ev) - k:]
        same_ev = len(ev) == k * (steps + warm) and all(
            np.array_equal(last[f], want_ev[f])
            for f in ("claim_id", "aux", "kind", "block_index", "phys_block"))
        same_d = bool(np.array_equal(state["d_off"][real], d0[real]) and
                      np.array_equal(state["d_res"][real], d1[real]))
        line["verified_against_oracle"] = bool(same_out and same_ev and same_d)
        line["oracle_comparison"] = {"outcome_fields": bool(same_out), "events": bool(same_ev),
                                     "block_digests": same_d, "blocks_with_real_digests": int(real.size)}
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
