"""ctypes binding of ``libcascade.so`` (see include/cascade.h).

Argument marshalling only: every step of the scheduling path runs in the
library's gfx950 kernels.  The library must be built (``build.py``); there is
no fallback, loading fails loudly if it is missing.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcascade.so")

OK, EINVAL, ENOSPC, EHIP, ETIMEOUT, EINTERNAL = 0, -1, -2, -3, -4, -5
QUEUED, RUNNING_PREFILL, DECODE = 0, 1, 2
QT_NEW, QT_TIER1, QT_TIER2 = 0, 1, 2
KV_HBM, KV_DRAM, KV_NVME, KV_NONE = 0, 1, 2, 3
ACT_RETAIN, ACT_RESTORE, ACT_PREFETCH, ACT_RECOMPUTE = 1, 2, 3, 4
ACT_PREEMPT_OFFLOAD, ACT_PREEMPT_DROP, ACT_SHARE = 5, 6, 7
INFO_STATUS, INFO_N_ADMITTED, INFO_N_SLOT_LIST, INFO_N_UNPACK, INFO_N_PACK = 0, 1, 2, 3, 4
INFO_LEN = 8

EXPORTED = ["cascade_step_workspace_bytes", "cascade_step", "cascade_step_noalloc",
            "cascade_pack", "cascade_unpack",
            "cascade_pack_unpack", "cascade_prefix_index_bytes", "cascade_prefix_index_clear",
            "cascade_prefix_index_insert", "cascade_prefix_probe", "cascade_restore_from_host",
            "cascade_spill_to_host", "cascade_reclaim_workspace_bytes", "cascade_tier_reclaim",
            "cascade_tier_chain_workspace_bytes", "cascade_tier_reclaim_chain",
            "cascade_strerror"]
INDEX_SLOT_BYTES = 16


class TierTable(C.Structure):
    _fields_ = [("n_slots", C.c_int32), ("block_hash", C.c_void_p), ("last_use_ns", C.c_void_p),
                ("held", C.c_void_p)]


# cascade_demotion_t: hash, last use, source slot (24 bytes)
DEMOTION_DTYPE = np.dtype([("hash", np.uint64), ("last_use_ns", np.int64),
                           ("src_slot", np.int32), ("pad", np.int32)])


class TierChain(C.Structure):
    _fields_ = [("table", TierTable * 3), ("need", C.c_int32 * 3),
                ("outgoing", C.c_void_p * 2), ("n_outgoing_dev", C.c_void_p * 2),
                ("max_outgoing", C.c_int32 * 2), ("freed", C.c_void_p * 3),
                ("placed", C.c_void_p * 3)]


class Requests(C.Structure):
    _fields_ = [("n", C.c_int32), ("id", C.c_void_p), ("slo_class", C.c_void_p),
                ("state", C.c_void_p), ("queue_tier", C.c_void_p), ("prefix_tier", C.c_void_p),
                ("arrival_ns", C.c_void_p), ("n_in", C.c_void_p), ("n_out_pred", C.c_void_p),
                ("n_prefix", C.c_void_p), ("n_progress", C.c_void_p),
                ("prefix_group", C.c_void_p)]


class BlockTable(C.Structure):
    _fields_ = [("row_offsets", C.c_void_p), ("slots", C.c_void_p)]


class TierState(C.Structure):
    _fields_ = [("num_blocks", C.c_int32), ("n_free", C.c_int32), ("free_slots", C.c_void_p)]


class Params(C.Structure):
    _fields_ = [
        ("t_now_ns", C.c_int64), ("num_classes", C.c_int32), ("slo_ns", C.c_int64 * 16),
        ("block_tokens", C.c_int32), ("chunk_tokens", C.c_int32),
        ("load_decodes", C.c_int32), ("max_batch", C.c_int32), ("gamma_q16", C.c_int32),
        ("c_iter_ps", C.c_int64), ("c_decode_ps", C.c_int64),
        ("c_token_ps", C.c_int64), ("c_attn_ps", C.c_int64),
        ("link_delta_ns", C.c_int64 * 2), ("link_blk_ns", C.c_int64 * 2),
        ("token_cap", C.c_int32), ("tier2_reserve_q16", C.c_int32),
        ("max_move_blocks", C.c_int32),
    ]


class Move(C.Structure):
    _fields_ = [("req", C.c_int32), ("blk", C.c_int32), ("pool_slot", C.c_int32),
                ("staging_slot", C.c_int32)]


class Outputs(C.Structure):
    _fields_ = [
        ("budget_ns", C.c_void_p), ("action", C.c_void_p), ("queue_tier_out", C.c_void_p),
        ("tokens_granted", C.c_void_p), ("restore_blocks", C.c_void_p), ("order", C.c_void_p),
        ("alloc_begin", C.c_void_p), ("alloc_count", C.c_void_p), ("admitted", C.c_void_p),
        ("slot_list", C.c_void_p), ("unpack_moves", C.c_void_p), ("pack_moves", C.c_void_p),
        ("slot_list_capacity", C.c_int32), ("unpack_capacity", C.c_int32),
        ("pack_capacity", C.c_int32), ("info", C.c_void_p),
        ("unpack_hazard", C.c_void_p), ("pack_hazard", C.c_void_p),
        ("share_leader", C.c_void_p),
    ]


class KvPool(C.Structure):
    _fields_ = [("base", C.c_void_p), ("num_layers", C.c_int32), ("num_slots", C.c_int32),
                ("chunk_bytes", C.c_int64), ("layer_stride", C.c_int64),
                ("kv_stride", C.c_int64), ("slot_stride", C.c_int64)]


_lib = None


def load() -> C.CDLL:
    """Load the library (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2608_06557_amd.build` (no CPU fallback exists)")
        L = C.CDLL(LIB_PATH)
        L.cascade_step_workspace_bytes.restype = C.c_size_t
        L.cascade_step_workspace_bytes.argtypes = [C.c_int32]
        L.cascade_step.restype = C.c_int
        L.cascade_step.argtypes = [C.POINTER(Requests), C.POINTER(BlockTable),
                                   C.POINTER(TierState), C.POINTER(Params), C.POINTER(Outputs),
                                   C.c_void_p, C.c_size_t, C.c_void_p]
        L.cascade_step_noalloc.restype = C.c_int
        L.cascade_step_noalloc.argtypes = [C.POINTER(Requests), C.POINTER(BlockTable),
                                           C.POINTER(TierState), C.POINTER(Params),
                                           C.POINTER(Outputs), C.c_void_p]
        for name in ("cascade_pack", "cascade_unpack"):
            f = getattr(L, name)
            f.restype = C.c_int
            f.argtypes = [C.POINTER(KvPool), C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p,
                          C.c_int32, C.c_void_p, C.c_void_p]
        L.cascade_pack_unpack.restype = C.c_int
        L.cascade_pack_unpack.argtypes = [C.POINTER(KvPool),
                                          C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p,
                                          C.c_int32, C.c_void_p,
                                          C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p,
                                          C.c_int32, C.c_void_p,
                                          C.c_void_p, C.c_void_p]
        L.cascade_prefix_index_bytes.restype = C.c_size_t
        L.cascade_prefix_index_bytes.argtypes = [C.c_int32]
        L.cascade_prefix_index_clear.restype = C.c_int
        L.cascade_prefix_index_clear.argtypes = [C.c_void_p, C.c_int32, C.c_void_p]
        L.cascade_prefix_index_insert.restype = C.c_int
        L.cascade_prefix_index_insert.argtypes = [C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p,
                                                  C.c_int32, C.c_void_p, C.c_void_p]
        L.cascade_prefix_probe.restype = C.c_int
        L.cascade_prefix_probe.argtypes = [C.c_void_p, C.c_int32, C.c_int32, C.c_void_p,
                                           C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p,
                                           C.c_void_p, C.c_void_p, C.c_void_p]
        for name in ("cascade_restore_from_host", "cascade_spill_to_host"):
            f = getattr(L, name)
            f.restype = C.c_int
            f.argtypes = [C.POINTER(KvPool), C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p,
                          C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_void_p,
                          C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32]
        L.cascade_reclaim_workspace_bytes.restype = C.c_size_t
        L.cascade_reclaim_workspace_bytes.argtypes = [C.c_int32]
        L.cascade_tier_reclaim.restype = C.c_int
        L.cascade_tier_reclaim.argtypes = [C.c_int32, C.POINTER(TierTable), C.c_int32,
                                           C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p,
                                           C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p,
                                           C.c_void_p, C.c_int32, C.c_void_p, C.c_size_t,
                                           C.c_void_p, C.c_void_p]
        L.cascade_tier_chain_workspace_bytes.restype = C.c_size_t
        L.cascade_tier_chain_workspace_bytes.argtypes = [C.POINTER(C.c_int32)]
        L.cascade_tier_reclaim_chain.restype = C.c_int
        L.cascade_tier_reclaim_chain.argtypes = [C.POINTER(TierChain), C.c_void_p, C.c_int32,
                                                 C.c_void_p, C.c_size_t, C.c_void_p,
                                                 C.c_void_p]
        L.cascade_strerror.restype = C.c_char_p
        L.cascade_strerror.argtypes = [C.c_int]
        _lib = L
    return _lib


def cascade_step_workspace_bytes(n: int) -> int:
    return int(load().cascade_step_workspace_bytes(n))


def cascade_step(requests: Requests, table: BlockTable, tier: TierState, params: Params,
                 outputs: Outputs, workspace: int, workspace_bytes: int, stream: int) -> int:
    return int(load().cascade_step(C.byref(requests), C.byref(table), C.byref(tier),
                                   C.byref(params), C.byref(outputs), C.c_void_p(workspace),
                                   workspace_bytes, C.c_void_p(stream)))


NOALLOC_MAX_REQUESTS = 262144


def cascade_step_noalloc(requests: Requests, table: BlockTable, tier: TierState, params: Params,
                         outputs: Outputs, stream: int) -> int:
    return int(load().cascade_step_noalloc(C.byref(requests), C.byref(table), C.byref(tier),
                                           C.byref(params), C.byref(outputs),
                                           C.c_void_p(stream)))


def cascade_pack(pool: KvPool, staging: int, staging_slots: int, moves: int, n_moves_dev: int,
                 max_moves: int, status_dev: int, stream: int) -> int:
    return int(load().cascade_pack(C.byref(pool), C.c_void_p(staging), staging_slots,
                                   C.c_void_p(moves), C.c_void_p(n_moves_dev), max_moves,
                                   C.c_void_p(status_dev), C.c_void_p(stream)))


def cascade_unpack(pool: KvPool, staging: int, staging_slots: int, moves: int, n_moves_dev: int,
                   max_moves: int, status_dev: int, stream: int) -> int:
    return int(load().cascade_unpack(C.byref(pool), C.c_void_p(staging), staging_slots,
                                     C.c_void_p(moves), C.c_void_p(n_moves_dev), max_moves,
                                     C.c_void_p(status_dev), C.c_void_p(stream)))


def cascade_pack_unpack(pool: KvPool, pack_staging: int, pack_staging_slots: int,
                        pack_moves: int, n_pack_dev: int, max_pack: int, pack_hazard: int,
                        unpack_staging: int, unpack_staging_slots: int, unpack_moves: int,
                        n_unpack_dev: int, max_unpack: int, unpack_hazard: int,
                        status_dev: int, stream: int) -> int:
    v = C.c_void_p
    return int(load().cascade_pack_unpack(
        C.byref(pool), v(pack_staging), pack_staging_slots, v(pack_moves), v(n_pack_dev),
        max_pack, v(pack_hazard), v(unpack_staging), unpack_staging_slots, v(unpack_moves),
        v(n_unpack_dev), max_unpack, v(unpack_hazard), v(status_dev), v(stream)))


def cascade_prefix_index_bytes(capacity: int) -> int:
    return int(load().cascade_prefix_index_bytes(capacity))


def cascade_prefix_index_clear(index: int, capacity: int, stream: int) -> int:
    return int(load().cascade_prefix_index_clear(C.c_void_p(index), capacity, C.c_void_p(stream)))


def cascade_prefix_index_insert(index: int, capacity: int, hashes: int, tiers: int, n: int,
                                status_dev: int, stream: int) -> int:
    v = C.c_void_p
    return int(load().cascade_prefix_index_insert(v(index), capacity, v(hashes), v(tiers), n,
                                                  v(status_dev), v(stream)))


def cascade_prefix_probe(index: int, capacity: int, n: int, block_offsets: int,
                         block_hashes: int, n_in: int, block_tokens: int, n_prefix_out: int,
                         prefix_tier_out: int, status_dev: int, stream: int) -> int:
    v = C.c_void_p
    return int(load().cascade_prefix_probe(v(index), capacity, n, v(block_offsets),
                                           v(block_hashes), v(n_in), block_tokens,
                                           v(n_prefix_out), v(prefix_tier_out), v(status_dev),
                                           v(stream)))


def _host_tier(fn, pool, staging, staging_slots, host_blocks, host_offsets, moves_dev,
               n_moves_dev, n_moves, batch_moves, status_dev, copy_stream, compute_stream,
               events):
    offs = np.ascontiguousarray(host_offsets, dtype=np.int64)
    ev = (C.c_void_p * max(len(events), 1))(*[C.c_void_p(e) for e in events])
    v = C.c_void_p
    return int(fn(C.byref(pool), v(staging), staging_slots, v(host_blocks),
                  offs.ctypes.data_as(v), v(moves_dev), v(n_moves_dev), n_moves, batch_moves,
                  v(status_dev), v(copy_stream), v(compute_stream), ev, len(events)))


def cascade_restore_from_host(pool: KvPool, staging: int, staging_slots: int, host_blocks: int,
                              host_offsets, moves_dev: int, n_moves_dev: int, n_moves: int,
                              batch_moves: int, status_dev: int, copy_stream: int,
                              compute_stream: int, events) -> int:
    return _host_tier(load().cascade_restore_from_host, pool, staging, staging_slots,
                      host_blocks, host_offsets, moves_dev, n_moves_dev, n_moves, batch_moves,
                      status_dev, copy_stream, compute_stream, events)


def cascade_spill_to_host(pool: KvPool, staging: int, staging_slots: int, host_blocks: int,
                          host_offsets, moves_dev: int, n_moves_dev: int, n_moves: int,
                          batch_moves: int, status_dev: int, copy_stream: int,
                          compute_stream: int, events) -> int:
    return _host_tier(load().cascade_spill_to_host, pool, staging, staging_slots, host_blocks,
                      host_offsets, moves_dev, n_moves_dev, n_moves, batch_moves, status_dev,
                      copy_stream, compute_stream, events)


def cascade_reclaim_workspace_bytes(n_slots: int) -> int:
    return int(load().cascade_reclaim_workspace_bytes(n_slots))


def cascade_tier_reclaim(tier: int, table: TierTable, need: int, incoming: int,
                         n_incoming_dev: int, max_incoming: int, outgoing: int,
                         n_outgoing_dev: int, max_outgoing: int, freed: int, placed: int,
                         index: int, index_capacity: int, workspace: int, workspace_bytes: int,
                         status_dev: int, stream: int) -> int:
    v = C.c_void_p
    return int(load().cascade_tier_reclaim(
        tier, C.byref(table), need, v(incoming), v(n_incoming_dev), max_incoming, v(outgoing),
        v(n_outgoing_dev), max_outgoing, v(freed), v(placed), v(index), index_capacity,
        v(workspace), workspace_bytes, v(status_dev), v(stream)))


def cascade_tier_chain_workspace_bytes(n_slots) -> int:
    arr = (C.c_int32 * 3)(*[int(x) for x in n_slots])
    return int(load().cascade_tier_chain_workspace_bytes(arr))


def cascade_tier_reclaim_chain(chain: TierChain, index: int, index_capacity: int,
                               workspace: int, workspace_bytes: int, status_dev: int,
                               stream: int) -> int:
    v = C.c_void_p
    return int(load().cascade_tier_reclaim_chain(C.byref(chain), v(index), index_capacity,
                                                 v(workspace), workspace_bytes, v(status_dev),
                                                 v(stream)))


def cascade_strerror(code: int) -> str:
    return load().cascade_strerror(code).decode()


PARAM_KEYS = ["t_now_ns", "num_classes", "block_tokens", "chunk_tokens", "load_decodes",
              "max_batch", "gamma_q16", "c_iter_ps", "c_decode_ps", "c_token_ps", "c_attn_ps",
              "token_cap", "tier2_reserve_q16", "max_move_blocks"]


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
