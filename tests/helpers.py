"""Test-only helpers: build workload dicts from fixtures and draw small
random workloads in the step's domain.  No scheduling arithmetic here."""
from __future__ import annotations

import json
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

QUEUED, RUNNING_PREFILL, DECODE = 0, 1, 2
KV_HBM, KV_DRAM, KV_NVME, KV_NONE = 0, 1, 2, 3


def load_golden(name: str) -> dict:
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def worked_example() -> tuple[dict, dict]:
    g = load_golden("worked_example.json")
    rq = g["requests"]
    w = {k: np.array(rq[k]) for k in ["id", "slo_class", "state", "queue_tier", "prefix_tier",
                                       "arrival_ns", "n_in", "n_out_pred", "n_prefix",
                                       "n_progress"]}
    w["id"] = w["id"].astype(np.uint64)
    lens = np.array(rq["row_lengths"])
    ro = np.zeros(len(lens) + 1, np.int32)
    ro[1:] = np.cumsum(lens)
    w["row_offsets"] = ro
    w["slots"] = np.concatenate([np.arange(900, 907), np.arange(800, 832)]).astype(np.int32)
    lo, hi = g["free_slots_range"]
    w["free_slots"] = np.arange(lo, hi, dtype=np.int32)
    w["params"] = g["params"]
    return w, g


def golden_workload(name: str) -> tuple[dict, dict]:
    """A hand-derived example whose block-table rows and free list are
    listed explicitly ("row_slots", "free_slots")."""
    g = load_golden(name)
    rq = g["requests"]
    w = {k: np.array(rq[k]) for k in ["id", "slo_class", "state", "queue_tier", "prefix_tier",
                                       "arrival_ns", "n_in", "n_out_pred", "n_prefix",
                                       "n_progress"]}
    w["id"] = w["id"].astype(np.uint64)
    rows = rq["row_slots"]
    ro = np.zeros(len(rows) + 1, np.int32)
    ro[1:] = np.cumsum([len(r) for r in rows])
    w["row_offsets"] = ro
    w["slots"] = np.array([s for r in rows for s in r], np.int32)
    w["free_slots"] = np.array(g["free_slots"], np.int32)
    if "prefix_group" in rq:
        w["prefix_group"] = np.array(rq["prefix_group"], np.int32)
    w["params"] = g["params"]
    return w, g


def base_params(**over) -> dict:
    """Small-number parameters under which every branch of the step is
    common: budgets of tens of microseconds, restores that are sometimes
    cheaper than recompute, partial grants, block deficits."""
    p = dict(t_now_ns=10 ** 9, num_classes=3, slo_ns=[20_000, 50_000, 200_000] + [0] * 13,
             block_tokens=4, chunk_tokens=16, load_decodes=2, max_batch=6, gamma_q16=81920,
             c_iter_ps=1_000_000, c_decode_ps=50_000, c_token_ps=100_000, c_attn_ps=30,
             link_delta_ns=[2_000, 6_000], link_blk_ns=[250, 100],
             token_cap=64, tier2_reserve_q16=8192, max_move_blocks=40, num_blocks=400)
    p.update(over)
    return p


def random_workload(rng: np.random.Generator, n: int, params: dict | None = None,
                    n_free: int | None = None, max_in: int = 120) -> dict:
    """A random valid workload with small numbers, so every branch of the
    step (restore, prefetch, recompute, victims, Tier-2 reserve, partial
    grants) is reachable with n <= 8."""
    p = dict(params or base_params())
    bt = p["block_tokens"]
    ncls = p["num_classes"]
    state = rng.integers(0, 3, n)
    n_in = rng.integers(1, max_in + 1, n)
    n_out = rng.integers(0, 60, n)
    tier = rng.integers(0, 4, n)
    n_prefix = bt * ((rng.random(n) * n_in) // bt).astype(np.int64)
    n_prefix = np.minimum(n_prefix, bt * ((n_in - 1) // bt))
    q = state == QUEUED
    none = (tier == KV_NONE) | (n_prefix == 0)
    tier = np.where(q & none, KV_NONE, tier)
    n_prefix = np.where(q & none, 0, n_prefix)
    prog = np.zeros(n, np.int64)
    rp = (state == RUNNING_PREFILL) & (n_in >= 2)
    state = np.where((state == RUNNING_PREFILL) & ~rp, QUEUED, state)
    # queued requests that became queued above need the prefix rule again
    q = state == QUEUED
    none = (tier == KV_NONE) | (n_prefix == 0)
    tier = np.where(q & none, KV_NONE, tier)
    n_prefix = np.where(q & none, 0, n_prefix)
    prog[rp] = 1 + (rng.random(rp.sum()) * (n_in[rp] - 1)).astype(np.int64)
    de = state == DECODE
    prog[de] = rng.integers(0, 70, de.sum())
    rows = np.zeros(n, np.int64)
    rows[rp] = -(-prog[rp] // bt)
    rows[de] = -(-(n_in[de] + prog[de]) // bt)
    nnz = int(rows.sum())
    nb = p["num_blocks"]
    if nnz > nb:
        p["num_blocks"] = nb = nnz + 64
    perm = rng.permutation(nb)
    slots = perm[:nnz].astype(np.int32)
    if n_free is None:
        n_free = int(rng.integers(0, min(48, nb - nnz) + 1))
    free = perm[nnz:nnz + n_free].astype(np.int32)
    ro = np.zeros(n + 1, np.int64)
    ro[1:] = np.cumsum(rows)
    cls = rng.integers(0, ncls, n)
    slo = np.array(p["slo_ns"][:ncls], np.int64)[cls]
    elapsed = (rng.random(n) * (slo + 1)).astype(np.int64)
    return dict(
        id=np.cumsum(rng.integers(1, 5, n)).astype(np.uint64),
        slo_class=cls.astype(np.uint8), state=state.astype(np.uint8),
        queue_tier=rng.integers(0, 3, n).astype(np.uint8), prefix_tier=tier.astype(np.uint8),
        arrival_ns=(p["t_now_ns"] - np.minimum(elapsed, p["t_now_ns"])).astype(np.int64),
        n_in=n_in.astype(np.int32), n_out_pred=n_out.astype(np.int32),
        n_prefix=n_prefix.astype(np.int32), n_progress=prog.astype(np.int32),
        row_offsets=ro.astype(np.int32), slots=slots, free_slots=free, params=p)
