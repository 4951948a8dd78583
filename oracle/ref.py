"""ctypes wrapper of the CPU oracle (``libcascade_ref.so``).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg may call this module; the product path never does.  It
imports nothing from the GPU package.

The oracle follows the Cascade paper (arXiv 2608.06557): Section 4.2
(estimator, eq:est_latency, eq:budget_eq, Tier-1/Tier-2), Section 4.3
(eq:rem_budget_eq, eq:restore_time, eq:max_restorable, Algorithm 1,
budget-aware preemption) and Section 4.4 (chunked prefill, final-hop HBM
allocation, preemption of the largest-budget prefill holder).
"""
from __future__ import annotations

import contextlib
import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcascade_ref.so")
SOURCES = [os.path.join(HERE, "cascade_ref.c")]

OK, EINVAL, ENOSPC = 0, -1, -2
QUEUED, RUNNING_PREFILL, DECODE = 0, 1, 2
QT_NEW, QT_TIER1, QT_TIER2 = 0, 1, 2
KV_HBM, KV_DRAM, KV_NVME, KV_NONE = 0, 1, 2, 3
ACT_RETAIN, ACT_RESTORE, ACT_PREFETCH, ACT_RECOMPUTE = 1, 2, 3, 4
ACT_PREEMPT_OFFLOAD, ACT_PREEMPT_DROP, ACT_SHARE = 5, 6, 7


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, single thread, no intrinsics)."""
    if force or not os.path.exists(LIB_PATH):
        tmp = LIB_PATH + ".tmp"
        cmd = ["gcc", "-std=gnu11", "-O2", "-fPIC", "-shared", "-Wall", "-Wextra",
               "-o", tmp] + SOURCES
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


class Params(C.Structure):
    _fields_ = [
        ("t_now_ns", C.c_int64), ("num_classes", C.c_int32), ("slo_ns", C.c_int64 * 16),
        ("block_tokens", C.c_int32), ("chunk_tokens", C.c_int32),
        ("load_decodes", C.c_int32), ("max_batch", C.c_int32), ("gamma_q16", C.c_int32),
        ("c_iter_ps", C.c_int64), ("c_decode_ps", C.c_int64),
        ("c_token_ps", C.c_int64), ("c_attn_ps", C.c_int64),
        ("link_delta_ns", C.c_int64 * 2), ("link_blk_ns", C.c_int64 * 2),
        ("token_cap", C.c_int32), ("tier2_reserve_q16", C.c_int32),
        ("max_move_blocks", C.c_int32), ("num_blocks", C.c_int32),
    ]


class Move(C.Structure):
    _fields_ = [("req", C.c_int32), ("blk", C.c_int32), ("pool_slot", C.c_int32),
                ("staging_slot", C.c_int32)]


class Outputs(C.Structure):
    _fields_ = [
        ("budget_ns", C.c_void_p), ("action", C.c_void_p), ("queue_tier_out", C.c_void_p),
        ("tokens_granted", C.c_void_p), ("restore_blocks", C.c_void_p), ("order", C.c_void_p),
        ("alloc_begin", C.c_void_p), ("alloc_count", C.c_void_p), ("admitted", C.c_void_p),
        ("n_admitted", C.c_int32),
        ("slot_list", C.c_void_p), ("slot_list_capacity", C.c_int32), ("n_slot_list", C.c_int32),
        ("unpack_moves", C.c_void_p), ("unpack_capacity", C.c_int32), ("n_unpack", C.c_int32),
        ("pack_moves", C.c_void_p), ("pack_capacity", C.c_int32), ("n_pack", C.c_int32),
        ("unpack_hazard", C.c_void_p), ("pack_hazard", C.c_void_p),
        ("share_leader", C.c_void_p),
    ]


class EvalOut(C.Structure):
    _fields_ = [("l_actual_ns", C.c_int64), ("l_max_ns", C.c_int64), ("l_ns", C.c_int64),
                ("budget0_ns", C.c_int64), ("budget_rem_ns", C.c_int64),
                ("tier_out", C.c_int32), ("group", C.c_int32), ("want_blocks", C.c_int32),
                ("key", C.c_uint64)]


class Pool(C.Structure):
    _fields_ = [("base", C.c_void_p), ("num_layers", C.c_int32), ("chunk_bytes", C.c_int64),
                ("layer_stride", C.c_int64), ("kv_stride", C.c_int64), ("slot_stride", C.c_int64)]


_lib = None


def _bind(L):
    """Declare the argument and result types of every oracle function."""
    L.cref_compute_ps.restype = C.c_int64
    L.cref_compute_ps.argtypes = [C.POINTER(Params), C.c_int64, C.c_int64, C.c_int64]
    L.cref_restore_time_ns.restype = C.c_int64
    L.cref_restore_time_ns.argtypes = [C.POINTER(Params), C.c_int32, C.c_int64]
    L.cref_check_params.restype = C.c_int32
    L.cref_check_params.argtypes = [C.POINTER(Params), C.c_int32, C.c_int32]
    L.cref_eval.restype = None
    L.cref_eval.argtypes = [C.POINTER(Params), C.c_uint8, C.c_uint8, C.c_uint8, C.c_uint8,
                            C.c_int64, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                            C.POINTER(EvalOut)]
    L.cref_step.restype = C.c_int32
    L.cref_step.argtypes = [C.c_int32] + [C.c_void_p] * 12 + [C.c_int32, C.c_void_p, C.c_void_p,
                                                               C.POINTER(Params),
                                                               C.POINTER(Outputs)]
    L.cref_pack.restype = None
    L.cref_pack.argtypes = [C.POINTER(Pool), C.c_void_p, C.c_void_p, C.c_int32]
    L.cref_unpack.restype = None
    L.cref_unpack.argtypes = [C.POINTER(Pool), C.c_void_p, C.c_void_p, C.c_int32]
    L.cref_prefix_probe.restype = C.c_int32
    L.cref_prefix_probe.argtypes = [C.c_int32, C.c_void_p, C.c_void_p, C.c_int32,
                                    C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32,
                                    C.c_void_p, C.c_void_p]
    L.cref_tier_reclaim.restype = C.c_int32
    L.cref_tier_reclaim.argtypes = [C.c_int32, C.c_int32, C.c_void_p, C.c_void_p,
                                    C.c_void_p, C.c_int32, C.c_int32, C.c_void_p,
                                    C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p,
                                    C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p]
    return L


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        _lib = _bind(C.CDLL(LIB_PATH))
    return _lib


@contextlib.contextmanager
def library(path: str):
    """Run the oracle functions of this module on another build of the
    oracle (the tests' planted-mistake copies) inside the block."""
    global _lib
    saved = _lib
    _lib = _bind(C.CDLL(path))
    try:
        yield
    finally:
        _lib = saved


PARAM_KEYS = ["t_now_ns", "num_classes", "block_tokens", "chunk_tokens", "load_decodes",
              "max_batch", "gamma_q16", "c_iter_ps", "c_decode_ps", "c_token_ps", "c_attn_ps",
              "token_cap", "tier2_reserve_q16", "max_move_blocks", "num_blocks"]


def make_params(p: dict) -> Params:
    s = Params()
    for k in PARAM_KEYS:
        setattr(s, k, int(p[k]))
    for c, v in enumerate(p["slo_ns"]):
        s.slo_ns[c] = int(v)
    for l in range(2):
        s.link_delta_ns[l] = int(p["link_delta_ns"][l])
        s.link_blk_ns[l] = int(p["link_blk_ns"][l])
    return s


def compute_ps(p: dict, n: int, s: int, dd: int) -> int:
    return lib().cref_compute_ps(C.byref(make_params(p)), n, s, dd)


def restore_time_ns(p: dict, tier: int, x: int) -> int:
    return lib().cref_restore_time_ns(C.byref(make_params(p)), tier, x)


def check_params(p: dict, n: int, n_free: int) -> int:
    return lib().cref_check_params(C.byref(make_params(p)), n, n_free)


def eval_one(p: dict, cls, state, queue_tier, prefix_tier, arrival_ns, n_in, n_out_pred,
             n_prefix, n_progress) -> dict:
    o = EvalOut()
    lib().cref_eval(C.byref(make_params(p)), cls, state, queue_tier, prefix_tier, arrival_ns,
                    n_in, n_out_pred, n_prefix, n_progress, C.byref(o))
    return {k: getattr(o, k) for k, _ in EvalOut._fields_}


REQ_FIELDS = [("id", np.uint64), ("slo_class", np.uint8), ("state", np.uint8),
              ("queue_tier", np.uint8), ("prefix_tier", np.uint8), ("arrival_ns", np.int64),
              ("n_in", np.int32), ("n_out_pred", np.int32), ("n_prefix", np.int32),
              ("n_progress", np.int32)]

MOVE_DTYPE = np.dtype([("req", np.int32), ("blk", np.int32), ("pool_slot", np.int32),
                       ("staging_slot", np.int32)])


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


def step(w: dict, slot_cap: int | None = None, unpack_cap: int | None = None,
         pack_cap: int | None = None) -> dict:
    """Run the oracle step on a workload dict (numpy arrays + params; an
    optional "prefix_group" array turns on shared-prefix restores).

    Returns every output array, the counts and the return code."""
    n = int(len(w["id"]))
    req = {k: np.ascontiguousarray(w[k], dtype=t) for k, t in REQ_FIELDS}
    ro = np.ascontiguousarray(w["row_offsets"], dtype=np.int32)
    slots = np.ascontiguousarray(w["slots"], dtype=np.int32)
    if slots.size == 0:
        slots = np.zeros(1, np.int32)
    free = np.ascontiguousarray(w["free_slots"], dtype=np.int32)
    n_free = int(free.size)
    if free.size == 0:
        free = np.zeros(1, np.int32)
    p = w["params"]
    nn = max(n, 1)
    o = {
        "budget_ns": np.zeros(nn, np.int64), "action": np.zeros(nn, np.uint8),
        "queue_tier_out": np.zeros(nn, np.uint8), "tokens_granted": np.zeros(nn, np.int32),
        "restore_blocks": np.zeros(nn, np.int32), "order": np.zeros(nn, np.int32),
        "alloc_begin": np.zeros(nn, np.int32), "alloc_count": np.zeros(nn, np.int32),
        "admitted": np.zeros(nn, np.int32),
    }
    if slot_cap is None:
        slot_cap = int(p["num_blocks"])
    if unpack_cap is None:
        unpack_cap = int(p["num_blocks"])
    if pack_cap is None:
        pack_cap = int(p["num_blocks"])
    sl = np.zeros(max(slot_cap, 1), np.int32)
    um = np.zeros(max(unpack_cap, 1), MOVE_DTYPE)
    pm = np.zeros(max(pack_cap, 1), MOVE_DTYPE)
    uh = np.full(max(unpack_cap, 1), -7, np.int32)
    ph = np.full(max(pack_cap, 1), -7, np.int32)
    out = Outputs()
    for k in o:
        setattr(out, k, _ptr(o[k]))
    out.slot_list, out.slot_list_capacity = _ptr(sl), slot_cap
    out.unpack_moves, out.unpack_capacity = _ptr(um), unpack_cap
    out.pack_moves, out.pack_capacity = _ptr(pm), pack_cap
    out.unpack_hazard, out.pack_hazard = _ptr(uh), _ptr(ph)
    pg = None
    if w.get("prefix_group") is not None:
        pg = np.ascontiguousarray(w["prefix_group"], dtype=np.int32)
        if pg.size == 0:
            pg = np.zeros(1, np.int32)
        o["share_leader"] = np.full(nn, -7, np.int32)
        out.share_leader = _ptr(o["share_leader"])
    args = [_ptr(req[k]) for k, _ in REQ_FIELDS] + [_ptr(ro), _ptr(slots)]
    rc = lib().cref_step(n, *args, n_free, _ptr(free), None if pg is None else _ptr(pg),
                         C.byref(make_params(p)), C.byref(out))
    res = {k: v[:n] for k, v in o.items()}
    res["rc"] = rc
    res["n_admitted"] = out.n_admitted
    res["admitted"] = res["admitted"][: out.n_admitted] if rc == OK else res["admitted"]
    res["n_slot_list"], res["n_unpack"], res["n_pack"] = out.n_slot_list, out.n_unpack, out.n_pack
    res["slot_list"] = sl[: min(out.n_slot_list, slot_cap)]
    res["unpack_moves"] = um[: min(out.n_unpack, unpack_cap)]
    res["pack_moves"] = pm[: min(out.n_pack, pack_cap)]
    if rc == OK:
        res["unpack_hazard"] = uh[: out.n_unpack]
        res["pack_hazard"] = ph[: out.n_pack]
    return res


def make_pool(base: np.ndarray, geom: dict) -> Pool:
    pl = Pool()
    pl.base = _ptr(base)
    pl.num_layers = geom["num_layers"]
    pl.chunk_bytes = geom["chunk_bytes"]
    pl.layer_stride = geom["layer_stride"]
    pl.kv_stride = geom["kv_stride"]
    pl.slot_stride = geom["slot_stride"]
    return pl


def pack(pool: np.ndarray, geom: dict, staging: np.ndarray, moves: np.ndarray) -> None:
    moves = np.ascontiguousarray(moves, dtype=MOVE_DTYPE)
    lib().cref_pack(C.byref(make_pool(pool, geom)), _ptr(staging), _ptr(moves), len(moves))


def unpack(pool: np.ndarray, geom: dict, staging: np.ndarray, moves: np.ndarray) -> None:
    moves = np.ascontiguousarray(moves, dtype=MOVE_DTYPE)
    lib().cref_unpack(C.byref(make_pool(pool, geom)), _ptr(staging), _ptr(moves), len(moves))


def prefix_probe(index_hashes: np.ndarray, index_tiers: np.ndarray, block_offsets: np.ndarray,
                 block_hashes: np.ndarray, n_in: np.ndarray, block_tokens: int) -> dict:
    """Matched prefix length (tokens) and tier of every request (Section 4.4,
    prefix hit detection), from the oracle."""
    ih = np.ascontiguousarray(index_hashes, dtype=np.uint64)
    it = np.ascontiguousarray(index_tiers, dtype=np.uint8)
    off = np.ascontiguousarray(block_offsets, dtype=np.int32)
    bh = np.ascontiguousarray(block_hashes, dtype=np.uint64)
    ni = np.ascontiguousarray(n_in, dtype=np.int32)
    n = len(off) - 1
    npre = np.zeros(max(n, 1), np.int32)
    tier = np.zeros(max(n, 1), np.uint8)
    keep = [ih, it, off, bh, ni]
    ptr = [_ptr(a if a.size else np.zeros(1, a.dtype)) for a in keep]
    rc = lib().cref_prefix_probe(len(ih), ptr[0], ptr[1], n, ptr[2], ptr[3], ptr[4],
                                 int(block_tokens), _ptr(npre), _ptr(tier))
    return {"rc": rc, "n_prefix": npre[:n], "prefix_tier": tier[:n]}


# one block demoted to the next tier: its hash, last use and source slot
DEMOTION_DTYPE = np.dtype([("hash", np.uint64), ("last_use_ns", np.int64),
                           ("src_slot", np.int32), ("pad", np.int32)])


def tier_reclaim(tier: int, block_hash: np.ndarray, last_use_ns: np.ndarray, held: np.ndarray,
                 need: int, incoming: np.ndarray | None = None, max_outgoing: int | None = None,
                 index_keys: np.ndarray | None = None, index_masks: np.ndarray | None = None
                 ) -> dict:
    """One tier's LRU reclamation (Section 4.4: free blocks reclaimed least
    recently used within each tier, cold ones spilled one tier deeper), from
    the oracle.  Inputs are not modified: the updated slot table and index
    come back as copies."""
    bh = np.array(block_hash, dtype=np.uint64, copy=True)
    lu = np.array(last_use_ns, dtype=np.int64, copy=True)
    hd = np.ascontiguousarray(held, dtype=np.uint8)
    inc = (np.zeros(0, DEMOTION_DTYPE) if incoming is None
           else np.ascontiguousarray(incoming, dtype=DEMOTION_DTYPE))
    n_inc = len(inc)
    if max_outgoing is None:
        max_outgoing = int(need) + n_inc
    keys = (np.zeros(0, np.uint64) if index_keys is None
            else np.ascontiguousarray(index_keys, dtype=np.uint64))
    masks = (np.zeros(0, np.uint8) if index_masks is None
             else np.array(index_masks, dtype=np.uint8, copy=True))
    n_tot = max(int(need) + n_inc, 0)
    out = np.zeros(max(int(max_outgoing), 1), DEMOTION_DTYPE)
    freed = np.zeros(max(int(need), 1), np.int32)
    placed = np.zeros(max(n_inc, 1), np.int32)
    n_out = np.zeros(1, np.int32)
    keep = [bh, lu, hd, inc, keys, masks]
    ptr = [_ptr(a if a.size else np.zeros(1, a.dtype)) for a in keep]
    rc = lib().cref_tier_reclaim(int(tier), len(bh), ptr[0], ptr[1], ptr[2], int(need), n_inc,
                                 ptr[3], int(max_outgoing), _ptr(out), _ptr(n_out), _ptr(freed),
                                 _ptr(placed), len(keys), ptr[4], ptr[5])
    no = int(n_out[0]) if rc == OK else 0
    return {"rc": rc, "freed": freed[:max(int(need), 0)] if rc == OK else freed[:0],
            "placed": placed[:n_inc] if rc == OK else placed[:0], "outgoing": out[:no],
            "n_outgoing": no, "block_hash": bh, "last_use_ns": lu, "index_keys": keys,
            "index_masks": masks, "n_reclaimed": n_tot if rc == OK else 0}
