#!/usr/bin/env python3
"""Benchmark of the Cascade scheduling step on one MI355X.

One timed step = the whole hot path on one synthetic queue, inputs resident in
HBM: cascade_step (budgets, actions, least-budget-first order, admission,
preemption, move lists), then the KV copies it emitted, on one stream: by
default cascade_pack_unpack (spills and restores in one launch, ordered by the
step's hazard pairs); with --copy separate, cascade_pack then cascade_unpack.

Prints one JSON line: requests/s of the whole step, the step (parts 1-3)
latency, copy GB/s, a roofline record for the dominant kernel (the KV copy,
measured with HIP events on its stream) and the CPU oracle timed on this host
as a reported baseline.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("scheduling-step latency (µs) & requests/s at N=65536; "
          "KV pack/unpack GB/s vs HBM peak")
HBM_PEAK_GBPS = 8000.0
WORKLOADS = {
    0: ("256 chat requests, 3 SLO classes (2/10/60 s), waits U[0, SLO], 8B-class KV "
        "(32 layers), 4096-block pool, token cap 8192"),
    1: ("8192 chat requests, 5 SLO classes (2/10/60/120/300 s), waits U[0, SLO], 8B-class KV, "
        "65536-block (128 GiB) pool, token cap 16384, restore cap 512 blocks"),
    2: ("65536 requests, 80% chat / 20% agentic, 5 SLO classes (1/2/10/30/60 s, bound to the "
        "application), waits U[0, SLO/2], 8B-class KV (32 layers x 8 heads x 128 x bf16, "
        "16-token blocks), 200 GB pool, token cap 16384, ~2 GB packed and unpacked"),
    3: ("65536 requests, 50% reasoning / 25% chat / 25% agentic, 30% in families of 4 "
        "parallel reasoning samples sharing one of 512 prefixes of 1k-32k tokens, high load "
        "(127 co-scheduled decodes), waits of SLO - (20 ms + prompt at 10k tok/s) +- 20 ms, "
        "exact budget ties, 200 GB pool, token cap 16384"),
    4: ("262144 requests, 80% chat / 20% agentic, 5 SLO classes (2/5/10/30/60 s), waits "
        "U[0, SLO/2], 70B-class KV (80 layers), 250 GB pool, token cap 32768, "
        "~8 GB packed and unpacked"),
}

# Bytes a step must move through HBM per request: its input fields (id 8,
# class / state / queue tier / prefix tier 1 each, arrival 8, four 4-byte
# lengths, its block-table row offset 4) and its outputs (budget 8, action
# 1, tier 1, tokens granted / restore blocks / order position / allocation
# begin and count 4 each).  Block-table slots, free slots and emitted moves
# are counted per entry on top.
STEP_IN_BYTES_PER_REQUEST = 8 + 4 * 1 + 8 + 4 * 4 + 4
STEP_OUT_BYTES_PER_REQUEST = 8 + 1 + 1 + 5 * 4


def step_compulsory_bytes(w, res):
    """HBM bytes one scheduling step (parts 1-3) cannot avoid: every
    request's fields in and outputs out, every block-table and free-list
    slot read once (range checks, victims' rows), the slot list and both
    move lists (16-byte records) written once."""
    n = len(w["id"])
    return (n * (STEP_IN_BYTES_PER_REQUEST + STEP_OUT_BYTES_PER_REQUEST)
            + 4 * int(w["row_offsets"][-1]) + 4 * len(w["free_slots"])
            + 4 * int(res["n_slot_list"]) + 16 * int(res["n_unpack"] + res["n_pack"])
            + 4 * int(res["n_admitted"]))


def host_cpu():
    """This host's CPU as the oracle baseline sees it."""
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count()
    return {"model": model, "nproc": os.cpu_count(), "usable_cpus": usable}


def measured_traffic(cfg, layout, kernel, chunk_bytes):
    """HBM bytes per KV-copy launch from the committed rocprofv3 counter
    passes (FETCH_SIZE and WRITE_SIZE, each scaled by what it reads for a
    plain copy of known size), or None when the workload or kernel differs or
    the kernel source has changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "kvmove_counters_65536req_8b_200gb.md")
    try:
        text = open(path).read()
        rec = json.loads(text.rsplit("```json", 1)[1].split("```", 1)[0])
        src = open(os.path.join(ROOT, rec["source"]), "rb").read()
    except (OSError, IndexError, ValueError, KeyError):
        return None
    if (cfg != 2 or layout != "layer_major" or chunk_bytes != 32768
            or rec.get("kernel") != kernel):
        return None
    if hashlib.sha256(src).hexdigest() != rec["source_sha256"]:
        return None
    return float(rec["traffic_bytes_per_launch"])


def progress(msg):
    """One line per phase on stderr (the JSON line alone goes to stdout)."""
    print(f"bench: {msg}", file=sys.stderr, flush=True)


def measure_prefix_probe(cfg, stream, reps=20):
    """The step's inputs n_prefix / prefix_tier from block hashes: index build
    (clear + insert) and lookup on the workload's requests, HIP events on the
    stream that runs them (outside the step's timed region)."""
    import torch
    import paper_2608_06557_amd.synth as synth
    from paper_2608_06557_amd import device
    pw = synth.make_prefix_workload(cfg, shared_frac=0.3)
    d = device.DevicePrefix(pw)
    assert d.build(stream) == 0 and d.probe(stream) == 0
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    tb, tp = [], []
    for _ in range(reps):
        ev[0].record(stream)
        assert d.build(stream) == 0
        ev[1].record(stream)
        assert d.probe(stream) == 0
        ev[2].record(stream)
        torch.cuda.synchronize()
        tb.append(ev[0].elapsed_time(ev[1]) * 1e3)
        tp.append(ev[1].elapsed_time(ev[2]) * 1e3)
    g = d.fetch()
    assert g["status"] == 0
    n = d.n
    bt = pw["block_tokens"]
    full = np.diff(pw["block_offsets"])
    lim = np.minimum(full, (pw["n_in"] - 1) // bt)
    matched = g["n_prefix"] // bt
    looked = np.minimum(lim, matched + 1)       # blocks a lookup must examine
    us = float(np.median(tp))
    progress("prefix lookup measured")
    return {"requests": n, "index_facts": d.n_entries, "index_slots": d.capacity,
            "prompt_blocks": int(full.sum()), "blocks_examined": int(looked.sum()),
            "matched_blocks": int(matched.sum()),
            "build_us_p50": float(np.median(tb)), "probe_us_p50": us,
            "probe_req_per_s": n / (us * 1e-6),
            "blocks_examined_per_s": float(looked.sum()) / (us * 1e-6)}


def measure_reclaim(cfg, stream, reps=20):
    """Per-tier LRU reclamation, HBM -> DRAM -> NVMe, at the configuration's
    tier sizes: HIP events around each tier's call on the stream that runs
    them, tables and index restored from pristine copies between repetitions
    (outside the timed region).  The oracle's chain is timed once beside it."""
    import torch
    import paper_2608_06557_amd.synth as synth
    from paper_2608_06557_amd import device
    w = synth.make_tier_workload(cfg)
    d = device.DeviceTiers(w["tables"], w["needs"], w["index_keys"], w["index_masks"])
    keep = ([b.clone() for b in d.bh], [x.clone() for x in d.lu], d.index.clone())
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    per, tot = [[], [], []], []

    def restore():
        for t in range(3):
            d.bh[t].copy_(keep[0][t])
            d.lu[t].copy_(keep[1][t])
        d.index.copy_(keep[2])
        d.status.zero_()

    for r in range(reps + 2):
        restore()
        ev[0].record(stream)
        for t in range(3):
            assert d.call(t, stream) == 0
            ev[t + 1].record(stream)
        torch.cuda.synchronize()
        if r >= 2:  # two warm-ups
            for t in range(3):
                per[t].append(ev[t].elapsed_time(ev[t + 1]) * 1e3)
            tot.append(ev[0].elapsed_time(ev[3]) * 1e3)
    g = d.fetch()
    assert g["status"] == 0
    # the same chain replayed from a graph: the host enqueues nothing between
    # the tiers; the replay's results must equal the eager chain's
    graph = torch.cuda.CUDAGraph()
    cs = torch.cuda.Stream()
    restore()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=cs):
        assert d.run(cs) == 0
    gtot = []
    for r in range(reps + 2):
        restore()
        ev[0].record(stream)
        graph.replay()
        ev[3].record(stream)
        torch.cuda.synchronize()
        if r >= 2:
            gtot.append(ev[0].elapsed_time(ev[3]) * 1e3)
    gg = d.fetch()
    assert gg["status"] == 0
    for t in range(3):
        for k in ["freed", "placed", "block_hash", "last_use_ns"]:
            assert np.array_equal(gg["tiers"][t][k], g["tiers"][t][k]), (t, k)
    # the same chain as one cascade_tier_reclaim_chain call (the three tables'
    # count and histogram passes launched together); results equal the
    # per-tier calls'
    d.chain_args()
    ctot = []
    for r in range(reps + 2):
        restore()
        ev[0].record(stream)
        assert d.run_chain(stream) == 0
        ev[3].record(stream)
        torch.cuda.synchronize()
        if r >= 2:
            ctot.append(ev[0].elapsed_time(ev[3]) * 1e3)
    gc = d.fetch()
    assert gc["status"] == 0
    for t in range(3):
        for k in ["freed", "placed", "block_hash", "last_use_ns"]:
            assert np.array_equal(gc["tiers"][t][k], g["tiers"][t][k]), (t, k)
    n_rec = [len(g["tiers"][t]["freed"]) + len(g["tiers"][t]["placed"]) for t in range(3)]
    slots = int(sum(w["sizes"]))
    us = float(np.median(tot))
    # compulsory traffic: every slot's hash, stamp and held flag read once
    compulsory = 17 * slots
    progress("tier reclamation measured")
    return {"tier_slots": list(w["sizes"]), "needs": list(w["needs"]),
            "compulsory_bytes": compulsory,
            "compulsory_us_at_peak": compulsory / (HBM_PEAK_GBPS * 1e3),
            "reclaimed": n_rec, "demoted": [g["tiers"][t]["n_outgoing"] for t in range(2)],
            "index_keys": int(len(w["index_keys"])),
            "tier_us_p50": [float(np.median(x)) for x in per], "chain_us_p50": us,
            "chain_graph_us_p50": float(np.median(gtot)),
            "chain_call_us_p50": float(np.median(ctot)),
            "slots_scanned_per_s": slots / (us * 1e-6)}, w


def measure_step_only(cfg, stream, reps=100, warmup=10):
    """Parts 1-3 alone (cascade_step: budgets, actions, order, admission,
    preemption, move lists) on another workload, inputs resident in HBM:
    HIP events on the launch stream, median and p90.  No KV pool is needed."""
    import torch
    import paper_2608_06557_amd.synth as synth
    from paper_2608_06557_amd import device
    w = synth.make_workload(cfg)
    nb = w["params"]["num_blocks"]
    d = device.DeviceStep(w, slot_cap=nb, unpack_cap=nb, pack_cap=nb)
    for _ in range(warmup):
        assert d.run(stream) == 0
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * reps)]
    for k in range(reps):
        ev[2 * k].record(stream)
        assert d.run(stream) == 0
        ev[2 * k + 1].record(stream)
    torch.cuda.synchronize()
    t = np.array([ev[2 * k].elapsed_time(ev[2 * k + 1]) for k in range(reps)]) * 1e3
    res = d.fetch()
    assert res["status"] == 0
    n = len(w["id"])
    p50 = float(np.median(t))
    cb = step_compulsory_bytes(w, res)
    progress(f"step alone at {n} requests measured")
    return {"workload": WORKLOADS[cfg], "requests": n, "runs": reps,
            "sched_step_us_p50": p50, "sched_step_us_p90": float(np.percentile(t, 90)),
            "sched_req_per_s": n / (p50 * 1e-6), "compulsory_bytes": cb,
            "roofline_frac": cb / (p50 * 1e-6) / 1e9 / HBM_PEAK_GBPS}


def measure_host_tier(pl, d, st_in, st_out, n_unpack, n_pack, block_bytes, stream,
                      batch=64, reps=3):
    """The DRAM tier's side of the step's restores and spills: pinned host
    blocks (one 2-MiB-class block per move, at shuffled host places) over the
    host link, pipelined in batches with the on-GPU unpack / pack
    (cascade_restore_from_host / cascade_spill_to_host), against the link
    alone and the kernel alone.  Outside the step's timed region."""
    import torch
    from paper_2608_06557_amd import cascade, device
    out = {"batch_moves": batch}
    copy_s = torch.cuda.Stream()
    evs, handles = device.event_handles(4, stream)
    st = torch.zeros(1, dtype=torch.int32, device=stream.device)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    rng = np.random.default_rng(0)
    for name, n, fn, stage, n_ptr, moves in [
            ("restore", n_unpack, cascade.cascade_restore_from_host, st_in, d.n_unpack_ptr(),
             d.unpack_moves.data_ptr()),
            ("spill", n_pack, cascade.cascade_spill_to_host, st_out, d.n_pack_ptr(),
             d.pack_moves.data_ptr())]:
        if n == 0:
            continue
        host = torch.empty(n * block_bytes, dtype=torch.uint8, pin_memory=True)
        offs = rng.permutation(n).astype(np.int64) * block_bytes

        def run(bm):
            # the entry points order their copies after earlier work on the
            # compute stream themselves
            e0.record(stream)
            rc = fn(pl, stage.data_ptr(), n, host.data_ptr(), offs, moves, n_ptr, n, bm,
                    st.data_ptr(), copy_s.cuda_stream, stream.cuda_stream, handles)
            assert rc == 0
            # a restore ends with an unpack on the compute stream, a spill with
            # a host copy on the copy stream
            e1.record(stream if name == "restore" else copy_s)
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) * 1e3
        run(batch)
        piped = float(np.median([run(batch) for _ in range(reps)]))
        whole = float(np.median([run(n) for _ in range(reps)]))   # one batch: no overlap
        # the link alone: the same DMA copies with no kernel
        def dma_only():
            with torch.cuda.stream(copy_s):
                e0.record(copy_s)
                for m in range(n):
                    dev_b = stage[m * block_bytes:(m + 1) * block_bytes]
                    host_b = host[int(offs[m]):int(offs[m]) + block_bytes]
                    if name == "restore":
                        dev_b.copy_(host_b, non_blocking=True)
                    else:
                        host_b.copy_(dev_b, non_blocking=True)
                e1.record(copy_s)
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) * 1e3
        dma_only()
        link = float(np.median([dma_only() for _ in range(reps)]))
        nbytes = n * block_bytes
        out[name] = {"blocks": n, "bytes": nbytes, "pipelined_us": piped,
                     "pipelined_GBps": nbytes / (piped * 1e-6) / 1e9,
                     "unbatched_us": whole, "link_only_us": link,
                     "link_only_GBps": nbytes / (link * 1e-6) / 1e9}
        del host
    assert int(st.item()) == 0
    progress("host-tier restore and spill measured")
    return out


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--layout", default="layer_major", choices=["layer_major", "block_major"])
    ap.add_argument("--chunk-bytes", type=int, default=0,
                    help="KV chunk per (block, layer, K/V); default the model's bf16 chunk "
                         "(32768). 8192 = one GPU's share under 4-way tensor parallelism, "
                         "16384 = FP8 KV")
    ap.add_argument("--copy", default="fused", choices=["fused", "separate"],
                    help="one cascade_pack_unpack launch, or cascade_pack then cascade_unpack")
    ap.add_argument("--prefix-groups", action="store_true",
                    help="pass each request's shared-prefix family (config 3) as prefix_group, "
                         "so restores of a shared prefix are shared within the step")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="approximate CPU time spent on the oracle baseline")
    ap.add_argument("--no-prefix-probe", action="store_true",
                    help="skip the prefix-hit lookup measurement")
    ap.add_argument("--no-reclaim", action="store_true",
                    help="skip the per-tier LRU reclamation chain measurement")
    ap.add_argument("--no-host-tier", action="store_true",
                    help="skip the DRAM-tier (pinned host) restore/spill measurement")
    ap.add_argument("--no-scale-step", action="store_true",
                    help="skip timing the step alone on the 262144-request queue")
    ap.add_argument("--calib-copy-gb", type=float, default=0.0,
                    help="also run a plain torch copy of this size (counter calibration)")
    return ap.parse_args()


def cpu_baseline(w, res, geom, block_bytes, budget_s, tier_w=None):
    """The oracle as it stands, single thread, on this host's cores (plus, for
    context, its tier reclamation chain on the same tables as the GPU's)."""
    from oracle import ref
    ref.build(force=False)
    n = len(w["id"])
    t0 = time.perf_counter()
    reps = 0
    while True:
        ref.step(w)
        reps += 1
        el = time.perf_counter() - t0
        if el > 0.5 * budget_s or reps >= 200:
            break
    t_step = el / reps
    # KV copies: a sample of the step's own moves through the oracle's
    # per-chunk memcpy, on a compact host pool holding just those slots
    pm, um = res["pack_moves"], res["unpack_moves"]
    k = int(min(64, max(len(pm), 1)))
    L, cb = geom["num_layers"], geom["chunk_bytes"]
    g = dict(num_layers=L, chunk_bytes=cb, slot_stride=cb, kv_stride=k * cb,
             layer_stride=2 * k * cb)
    pool = np.ones(2 * L * k * cb, np.uint8)
    st = np.zeros(k * 2 * L * cb, np.uint8)
    mv = np.zeros(k, ref.MOVE_DTYPE)
    mv["pool_slot"] = np.random.default_rng(0).permutation(k)
    mv["staging_slot"] = np.arange(k)
    t0 = time.perf_counter()
    creps = 0
    while True:
        ref.pack(pool, g, st, mv)
        ref.unpack(pool, g, st, mv)
        creps += 1
        el = time.perf_counter() - t0
        if el > 0.5 * budget_s or creps >= 50:
            break
    t_copy_block = el / (creps * 2 * k)          # seconds per block per direction
    t_copy = t_copy_block * (len(pm) + len(um))
    total = t_step + t_copy
    extra = {}
    if tier_w is not None:
        t0 = time.perf_counter()
        inc, masks = None, tier_w["index_masks"]
        for t in range(3):
            tb = tier_w["tables"][t]
            o = ref.tier_reclaim(t, tb["block_hash"], tb["last_use_ns"], tb["held"],
                                 tier_w["needs"][t], incoming=inc,
                                 max_outgoing=0 if t == 2 else None,
                                 index_keys=tier_w["index_keys"], index_masks=masks)
            assert o["rc"] == 0
            inc, masks = o["outgoing"], o["index_masks"]
        extra["tier_reclaim_chain_ms"] = (time.perf_counter() - t0) * 1e3
    return {**extra,
        "value": n / total, "unit": "req/s", "cores": 1, "kind": "oracle",
        "host": host_cpu(),
        "step_ms": t_step * 1e3, "copy_ms_scaled": t_copy * 1e3,
        "sample": (f"full {n}-request step x{reps}; KV copies: {k} of the step's "
                   f"{len(pm) + len(um)} block moves x{creps} through the oracle memcpy, "
                   f"time scaled to all moves"),
    }


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py: runs on one GPU only; the step is independent per "
              "serving instance (no cross-GPU exchange), so --gpus must be 1", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2608_06557_amd.synth as synth
    from paper_2608_06557_amd import cascade, device

    assert torch.cuda.is_available(), "needs a ROCm GPU"
    cascade.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = args.config
    w = synth.make_workload(cfg, prefix_groups=args.prefix_groups)
    c = synth.CONFIGS[cfg]
    geom = (synth.kv_geometry(c["model"], c["pool"], args.layout, args.chunk_bytes)
            if args.chunk_bytes else synth.kv_geometry(c["model"], c["pool"], args.layout))
    n = len(w["id"])
    nb = geom["num_blocks"]
    d = device.DeviceStep(w, slot_cap=nb, unpack_cap=max(1, min(nb, c["max_move"])),
                          pack_cap=nb)
    stream = torch.cuda.current_stream()
    sh = device.stream_handle(stream)

    # first step: learn the move counts (deterministic for this input)
    assert d.run(stream) == 0
    res = d.fetch()
    assert res["status"] == 0, cascade.cascade_strerror(res["status"])
    n_pack, n_unpack = res["n_pack"], res["n_unpack"]
    block_bytes = 2 * geom["num_layers"] * geom["chunk_bytes"]

    progress(f"step done: {n} requests, {n_pack} spill / {n_unpack} restore blocks")
    pool = torch.empty(geom["pool_bytes"], dtype=torch.uint8, device=dev)
    device.fill_pattern_(pool, seed=1, progress=progress)
    st_out = torch.empty(max(n_pack, 1) * block_bytes, dtype=torch.uint8, device=dev)
    st_in = torch.empty(max(n_unpack, 1) * block_bytes, dtype=torch.uint8, device=dev)
    device.fill_pattern_(st_in, seed=2)
    cstat = torch.zeros(1, dtype=torch.int32, device=dev)
    pl = device.kv_pool_struct(pool.data_ptr(), geom)
    torch.cuda.synchronize()

    fused = args.copy == "fused"

    def one_step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        rc = d.run(stream)
        if ev is not None:
            ev[1].record(stream)
        if fused:
            rc |= cascade.cascade_pack_unpack(
                pl, st_out.data_ptr(), max(n_pack, 1), d.pack_moves.data_ptr(), d.n_pack_ptr(),
                d.caps[2], d.pack_hazard.data_ptr(), st_in.data_ptr(), max(n_unpack, 1),
                d.unpack_moves.data_ptr(), d.n_unpack_ptr(), d.caps[1],
                d.unpack_hazard.data_ptr(), cstat.data_ptr(), sh)
            if ev is not None:
                ev[2].record(stream)
        else:
            rc |= cascade.cascade_pack(pl, st_out.data_ptr(), max(n_pack, 1),
                                       d.pack_moves.data_ptr(), d.n_pack_ptr(), d.caps[2],
                                       cstat.data_ptr(), sh)
            if ev is not None:
                ev[2].record(stream)
            rc |= cascade.cascade_unpack(pl, st_in.data_ptr(), max(n_unpack, 1),
                                         d.unpack_moves.data_ptr(), d.n_unpack_ptr(), d.caps[1],
                                         cstat.data_ptr(), sh)
        if ev is not None:
            ev[3].record(stream)
        return rc

    progress("pool and staging filled")
    for _ in range(args.warmup):
        assert one_step() == 0
    torch.cuda.synchronize()
    progress(f"{args.warmup} warm-up steps done")
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        assert one_step(evs[k]) == 0
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    progress(f"{args.steps} timed steps done")
    res2 = d.fetch()
    assert res2["status"] == 0 and int(cstat.item()) == 0
    assert res2["n_pack"] == n_pack and res2["n_unpack"] == n_unpack

    t_step = np.array([e[0].elapsed_time(e[1]) for e in evs]) * 1e3      # us
    t_c1 = np.array([e[1].elapsed_time(e[2]) for e in evs]) * 1e3
    t_c2 = np.array([e[2].elapsed_time(e[3]) for e in evs]) * 1e3
    t_all = np.array([e[0].elapsed_time(e[3]) for e in evs]) * 1e3
    ms_per_step = wall * 1e3 / args.steps
    bytes_pack = 2.0 * n_pack * block_bytes
    bytes_unpack = 2.0 * n_unpack * block_bytes
    gbps = lambda b, us: b / (us * 1e-6) / 1e9 if us > 0 else 0.0
    copy_us = float(np.mean(t_c1) + np.mean(t_c2))          # all copy launches of a step
    launches = 1 if fused else 2
    achieved = gbps(bytes_pack + bytes_unpack, copy_us)
    extra = None
    if args.calib_copy_gb > 0:
        nbytes = int(args.calib_copy_gb * 1e9) // 16 * 16
        a = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        b.copy_(a)
        e1.record(stream)
        torch.cuda.synchronize()
        extra = {"bytes": nbytes, "us": e0.elapsed_time(e1) * 1e3,
                 "GBps": gbps(2.0 * nbytes, e0.elapsed_time(e1) * 1e3)}
        del a, b
    # outside the timed region: the step with a cold last-level cache (a 1 GB
    # write between runs evicts the 256 MB MALL), and a plain device-to-device
    # copy of the bytes one step moves (capped to what memory allows)
    flush = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    cold = []
    ce = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for k in range(20):
        flush.fill_(k & 255)
        ce[0].record(stream)
        assert d.run(stream) == 0
        ce[1].record(stream)
        torch.cuda.synchronize()
        cold.append(ce[0].elapsed_time(ce[1]) * 1e3)
    del flush
    moved = (n_pack + n_unpack) * block_bytes
    free_b = torch.cuda.mem_get_info(dev)[0]
    nb_copy = int(min(moved, (free_b - (2 << 30)) // 2)) // 16 * 16
    dtod = None
    if nb_copy >= (64 << 20):
        a = torch.empty(nb_copy, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        ce[0].record(stream)
        for _ in range(5):
            b.copy_(a)
        ce[1].record(stream)
        torch.cuda.synchronize()
        us = ce[0].elapsed_time(ce[1]) * 1e3 / 5
        dtod = {"bytes": nb_copy, "GBps": gbps(2.0 * nb_copy, us)}
        del a, b
    progress("cold-cache steps and device copy done")
    scale = (None if args.no_scale_step or cfg == 4
             else measure_step_only(4, stream))
    probe = None if args.no_prefix_probe else measure_prefix_probe(cfg, stream)
    reclaim, tier_w = (None, None) if args.no_reclaim else measure_reclaim(cfg, stream)
    host_tier = None if args.no_host_tier else measure_host_tier(
        pl, d, st_in, st_out, n_unpack, n_pack, block_bytes, stream)
    kernel = "kvmove_kernel" if fused else "kvcopy_kernel"
    step_bytes = step_compulsory_bytes(w, res)
    step_achieved = gbps(step_bytes, float(np.median(t_step)))
    copies = {"mode": args.copy, "pack_blocks": n_pack, "unpack_blocks": n_unpack,
              "paired_blocks": int((res["unpack_hazard"] >= 0).sum()),
              "copy_us_p50": float(np.median(t_c1 + t_c2)),
              "copy_GBps": gbps(bytes_pack + bytes_unpack, float(np.median(t_c1 + t_c2)))}
    if dtod:
        copies["device_copy_same_bytes_GBps"] = dtod["GBps"]
        copies["device_copy_bytes"] = dtod["bytes"]
    if not fused:
        copies["pack_GBps"] = gbps(bytes_pack, float(np.median(t_c1)))
        copies["unpack_GBps"] = gbps(bytes_unpack, float(np.median(t_c2)))
    out = {
        "metric": METRIC,
        "value": n * args.steps / wall,
        "unit": "req/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {"workload": WORKLOADS[cfg] + (", shared-prefix restores shared within "
                                                 "the step (prefix_group)"
                                                 if args.prefix_groups else ""),
                   "requests": n,
                   "kv_layout": args.layout, "pool_blocks": nb,
                   "chunk_bytes": geom["chunk_bytes"],
                   "block_bytes": block_bytes, "token_cap": c["token_cap"],
                   "move_cap_blocks": c["max_move"]},
        "sched_step_us_p50": float(np.median(t_step)),
        "sched_step_us_p90": float(np.percentile(t_step, 90)),
        "sched_step_us_cold_p50": float(np.median(cold)),
        "sched_req_per_s": n / (float(np.median(t_step)) * 1e-6),
        "roofline_step": {
            "bound": "hbm", "what": "cascade_step (parts 1-3), compulsory bytes / p50",
            "bytes_per_request": STEP_IN_BYTES_PER_REQUEST + STEP_OUT_BYTES_PER_REQUEST,
            "bytes": step_bytes, "achieved": step_achieved, "peak": HBM_PEAK_GBPS,
            "unit": "GB/s", "frac": step_achieved / HBM_PEAK_GBPS},
        "kv_copy": copies,
        "step_total_us_p50": float(np.median(t_all)),
        "roofline": {"bound": "hbm", "kernel": kernel + (" (one launch: pack and unpack)" if fused
                                                          else " (pack + unpack launches)"),
                     "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": (measured_traffic(cfg, args.layout, kernel, geom["chunk_bytes"])
                                 if fused else None),
                     "bytes_per_launch": (bytes_pack + bytes_unpack) / launches,
                     "us_per_launch": copy_us / launches},
    }
    if scale:
        out["step_262144"] = scale
    if probe:
        out["prefix_probe"] = probe
    if reclaim:
        out["tier_reclaim"] = reclaim
    if host_tier:
        out["host_tier"] = host_tier
    if extra:
        out["calib_copy"] = extra
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, res, geom, block_bytes, args.cpu_seconds, tier_w)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
