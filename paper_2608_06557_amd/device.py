"""Device-memory plumbing around the C ABI, using torch for allocation and
streams only.  Uploads a workload (numpy arrays from ``synth``), holds the
output and workspace buffers, enqueues ``cascade_step`` / ``cascade_pack`` /
``cascade_unpack`` and reads results back."""
from __future__ import annotations

import numpy as np

from . import cascade as cx

REQ_FIELDS = [("id", np.int64), ("slo_class", np.uint8), ("state", np.uint8),
              ("queue_tier", np.uint8), ("prefix_tier", np.uint8), ("arrival_ns", np.int64),
              ("n_in", np.int32), ("n_out_pred", np.int32), ("n_prefix", np.int32),
              ("n_progress", np.int32)]
MOVE_DTYPE = np.dtype([("req", np.int32), ("blk", np.int32), ("pool_slot", np.int32),
                       ("staging_slot", np.int32)])


def _torch():
    import torch
    return torch


def to_device(a: np.ndarray, device, dtype=None):
    """Upload an array; empty arrays become a 1-element buffer so that every
    pointer handed to the library is valid."""
    torch = _torch()
    a = np.ascontiguousarray(a if dtype is None else a.astype(dtype, copy=False))
    if a.dtype == np.uint64:
        a = a.view(np.int64)
    if a.size == 0:
        a = np.zeros(1, a.dtype)
    return torch.from_numpy(a.copy()).to(device)


def stream_handle(stream=None) -> int:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


class DeviceStep:
    """Buffers for one workload and its cascade_step outputs."""

    def __init__(self, w: dict, device="cuda:0", slot_cap: int | None = None,
                 unpack_cap: int | None = None, pack_cap: int | None = None):
        torch = _torch()
        self.device = torch.device(device)
        self.n = n = int(len(w["id"]))
        p = w["params"]
        self.params = cx.make_params(p)
        self.num_blocks = int(p["num_blocks"])
        self.inp = {k: to_device(np.asarray(w[k]), self.device, dt) for k, dt in REQ_FIELDS}
        self.ro = to_device(np.asarray(w["row_offsets"]), self.device, np.int32)
        self.slots = to_device(np.asarray(w["slots"]), self.device, np.int32)
        self.free = to_device(np.asarray(w["free_slots"]), self.device, np.int32)
        self.n_free = int(len(w["free_slots"]))
        # shared-prefix restores: a prefix_group array in the workload
        self.pg = (to_device(np.asarray(w["prefix_group"]), self.device, np.int32)
                   if w.get("prefix_group") is not None else None)
        nb = self.num_blocks
        self.caps = (nb if slot_cap is None else slot_cap, nb if unpack_cap is None else unpack_cap,
                     nb if pack_cap is None else pack_cap)
        nn = max(n, 1)
        z = lambda k, dt: torch.zeros(max(k, 1), dtype=dt, device=self.device)
        self.out = {"budget_ns": z(nn, torch.int64), "action": z(nn, torch.uint8),
                    "queue_tier_out": z(nn, torch.uint8), "tokens_granted": z(nn, torch.int32),
                    "restore_blocks": z(nn, torch.int32), "order": z(nn, torch.int32),
                    "alloc_begin": z(nn, torch.int32), "alloc_count": z(nn, torch.int32),
                    "admitted": z(nn, torch.int32)}
        self.slot_list = z(self.caps[0], torch.int32)
        self.unpack_moves = z(4 * max(self.caps[1], 1), torch.int32)
        self.pack_moves = z(4 * max(self.caps[2], 1), torch.int32)
        self.unpack_hazard = z(self.caps[1], torch.int32)
        self.pack_hazard = z(self.caps[2], torch.int32)
        self.info = z(cx.INFO_LEN, torch.int32)
        if self.pg is not None:
            self.out["share_leader"] = z(nn, torch.int32)
        self.ws_bytes = cx.cascade_step_workspace_bytes(n)
        self.ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=self.device)
        self.ws_ptr = (self.ws.data_ptr() + 255) & ~255

        self.c_req = cx.Requests(n, *[self.inp[k].data_ptr() for k, _ in REQ_FIELDS],
                                 self.pg.data_ptr() if self.pg is not None else None)
        self.c_table = cx.BlockTable(self.ro.data_ptr(), self.slots.data_ptr())
        self.c_tier = cx.TierState(self.num_blocks, self.n_free, self.free.data_ptr())
        o = self.out
        self.c_out = cx.Outputs(
            o["budget_ns"].data_ptr(), o["action"].data_ptr(), o["queue_tier_out"].data_ptr(),
            o["tokens_granted"].data_ptr(), o["restore_blocks"].data_ptr(), o["order"].data_ptr(),
            o["alloc_begin"].data_ptr(), o["alloc_count"].data_ptr(), o["admitted"].data_ptr(),
            self.slot_list.data_ptr(), self.unpack_moves.data_ptr(), self.pack_moves.data_ptr(),
            self.caps[0], self.caps[1], self.caps[2], self.info.data_ptr(),
            self.unpack_hazard.data_ptr(), self.pack_hazard.data_ptr(),
            o["share_leader"].data_ptr() if self.pg is not None else None)

    def run(self, stream=None) -> int:
        """Enqueue one step; returns the host-side return code."""
        return cx.cascade_step(self.c_req, self.c_table, self.c_tier, self.params, self.c_out,
                               self.ws_ptr, self.ws_bytes, stream_handle(stream))

    def run_noalloc(self, stream=None) -> int:
        """The same step through cascade_step_noalloc (no workspace)."""
        return cx.cascade_step_noalloc(self.c_req, self.c_table, self.c_tier, self.params,
                                       self.c_out, stream_handle(stream))

    def n_unpack_ptr(self) -> int:
        return self.info.data_ptr() + 4 * cx.INFO_N_UNPACK

    def n_pack_ptr(self) -> int:
        return self.info.data_ptr() + 4 * cx.INFO_N_PACK

    def fetch(self) -> dict:
        """Synchronise and return every output as numpy (trimmed to counts)."""
        torch = _torch()
        torch.cuda.synchronize(self.device)
        info = self.info.cpu().numpy()
        n = self.n
        res = {k: v.cpu().numpy()[:n] for k, v in self.out.items()}
        res["status"] = int(info[cx.INFO_STATUS])
        res["n_admitted"] = int(info[cx.INFO_N_ADMITTED])
        res["n_slot_list"] = int(info[cx.INFO_N_SLOT_LIST])
        res["n_unpack"] = int(info[cx.INFO_N_UNPACK])
        res["n_pack"] = int(info[cx.INFO_N_PACK])
        res["admitted"] = res["admitted"][:res["n_admitted"]]
        res["slot_list"] = self.slot_list.cpu().numpy()[:min(res["n_slot_list"], self.caps[0])]
        um = self.unpack_moves.cpu().numpy().view(MOVE_DTYPE)
        pm = self.pack_moves.cpu().numpy().view(MOVE_DTYPE)
        res["unpack_moves"] = um[:min(res["n_unpack"], self.caps[1])]
        res["pack_moves"] = pm[:min(res["n_pack"], self.caps[2])]
        res["unpack_hazard"] = self.unpack_hazard.cpu().numpy()[:len(res["unpack_moves"])]
        res["pack_hazard"] = self.pack_hazard.cpu().numpy()[:len(res["pack_moves"])]
        return res


def kv_pool_struct(base_ptr: int, geom: dict) -> cx.KvPool:
    return cx.KvPool(base_ptr, int(geom["num_layers"]), int(geom["num_blocks"]),
                     int(geom["chunk_bytes"]), int(geom["layer_stride"]),
                     int(geom["kv_stride"]), int(geom["slot_stride"]))


def fill_pattern_(t, seed: int, word_offset: int = 0, chunk_words: int = 1 << 26,
                  progress=None) -> None:
    """Fill a uint8 device tensor with the counter-based 32-bit pattern of
    ``synth.hash32_torch`` (word k holds hash32(word_offset + k, seed)).
    ``progress(msg)``, if given, is called about every 16 GB."""
    torch = _torch()
    from .synth import hash32_torch
    w = t.view(torch.int32)
    nw = w.numel()
    every = max(1, (4 << 30) // chunk_words)
    for k, s in enumerate(range(0, nw, chunk_words)):
        e = min(nw, s + chunk_words)
        idx = torch.arange(word_offset + s, word_offset + e, device=t.device, dtype=torch.int64)
        h = hash32_torch(idx, seed)
        w[s:e] = (h - ((h >> 31) << 32)).to(torch.int32)
        if progress is not None and (k + 1) % every == 0:
            torch.cuda.synchronize(t.device)
            progress(f"filled {4 * e / 1e9:.0f} of {4 * nw / 1e9:.0f} GB")


def index_capacity(n_entries: int) -> int:
    """Slots for an index of n_entries facts: a power of two, load <= 1/2."""
    cap = 64
    while cap < 2 * max(n_entries, 1):
        cap *= 2
    return cap


class DevicePrefix:
    """Device buffers of one prefix-hit lookup: the index built from
    (hash, tier) facts and the requests' block-hash CSR."""

    def __init__(self, pw: dict, device="cuda:0", capacity: int | None = None):
        torch = _torch()
        self.device = torch.device(device)
        self.n = int(len(pw["n_in"]))
        self.n_entries = int(len(pw["index_hashes"]))
        self.capacity = capacity or index_capacity(self.n_entries)
        self.bt = int(pw["block_tokens"])
        nbytes = cx.cascade_prefix_index_bytes(self.capacity)
        assert nbytes > 0, self.capacity
        self.index = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        self.ih = to_device(np.asarray(pw["index_hashes"]), self.device)
        self.it = to_device(np.asarray(pw["index_tiers"]), self.device, np.uint8)
        self.off = to_device(np.asarray(pw["block_offsets"]), self.device, np.int32)
        self.bh = to_device(np.asarray(pw["block_hashes"]), self.device)
        self.n_in = to_device(np.asarray(pw["n_in"]), self.device, np.int32)
        self.n_prefix = torch.zeros(max(self.n, 1), dtype=torch.int32, device=self.device)
        self.tier = torch.zeros(max(self.n, 1), dtype=torch.uint8, device=self.device)
        self.status = torch.zeros(1, dtype=torch.int32, device=self.device)

    def build(self, stream=None) -> int:
        s = stream_handle(stream)
        rc = cx.cascade_prefix_index_clear(self.index.data_ptr(), self.capacity, s)
        return rc or cx.cascade_prefix_index_insert(self.index.data_ptr(), self.capacity,
                                                    self.ih.data_ptr(), self.it.data_ptr(),
                                                    self.n_entries, self.status.data_ptr(), s)

    def probe(self, stream=None) -> int:
        return cx.cascade_prefix_probe(self.index.data_ptr(), self.capacity, self.n,
                                       self.off.data_ptr(), self.bh.data_ptr(),
                                       self.n_in.data_ptr(), self.bt, self.n_prefix.data_ptr(),
                                       self.tier.data_ptr(), self.status.data_ptr(),
                                       stream_handle(stream))

    def fetch(self) -> dict:
        torch = _torch()
        torch.cuda.synchronize(self.device)
        return {"status": int(self.status.item()),
                "n_prefix": self.n_prefix.cpu().numpy()[:self.n],
                "prefix_tier": self.tier.cpu().numpy()[:self.n]}


def event_handles(k: int, stream=None) -> list:
    """k HIP events (torch-owned), recorded once so that each has a handle."""
    torch = _torch()
    evs = [torch.cuda.Event() for _ in range(k)]
    s = stream if stream is not None else torch.cuda.current_stream()
    for e in evs:
        e.record(s)
    torch.cuda.synchronize()
    return evs, [int(e.cuda_event) for e in evs]


def index_facts(keys: np.ndarray, masks: np.ndarray):
    """(hash, tier) facts whose insertion gives each key its tier set."""
    keys = np.asarray(keys, np.uint64)
    masks = np.asarray(masks, np.uint8)
    hs, ts = [], []
    for t in range(3):
        sel = (masks >> t) & 1 == 1
        hs.append(keys[sel])
        ts.append(np.full(int(sel.sum()), t, np.uint8))
    return np.concatenate(hs), np.concatenate(ts)


def index_contents(index_bytes: np.ndarray):
    """Keys (ascending) and tier sets of the occupied slots of a device index
    read back."""
    slots = np.frombuffer(index_bytes.tobytes(), dtype=np.dtype(
        [("key", np.uint64), ("tiers", np.uint32), ("pad", np.uint32)]))
    occ = slots[slots["key"] != 0]
    order = np.argsort(occ["key"], kind="stable")
    return occ["key"][order], occ["tiers"][order]


class DeviceTiers:
    """Slot tables of the three tiers (HBM, DRAM, NVMe), the prefix index and
    the buffers of one reclamation chain HBM -> DRAM -> NVMe: each tier's
    demoted blocks are the next tier's incoming ones, one status word."""

    def __init__(self, tables: list, needs, index_keys=None, index_masks=None,
                 device="cuda:0", capacity: int | None = None):
        torch = _torch()
        self.device = torch.device(device)
        self.n = [int(len(t["block_hash"])) for t in tables]
        self.needs = [int(x) for x in needs]
        self.bh = [to_device(np.asarray(t["block_hash"], np.uint64), self.device)
                   for t in tables]
        self.lu = [to_device(np.asarray(t["last_use_ns"], np.int64), self.device)
                   for t in tables]
        self.held = [to_device(np.asarray(t["held"], np.uint8), self.device) for t in tables]
        self.tabs = [cx.TierTable(self.n[t], self.bh[t].data_ptr(), self.lu[t].data_ptr(),
                                  self.held[t].data_ptr()) for t in range(3)]
        # tier t takes at most the previous tier's outgoing capacity
        self.max_in = [0, 0, 0]
        self.max_out = [0, 0, 0]
        for t in range(3):
            self.max_in[t] = self.max_out[t - 1] if t > 0 else 0
            self.max_out[t] = self.needs[t] + self.max_in[t] if t < 2 else 0
        self.out = [torch.zeros(max(self.max_out[t], 1) * cx.DEMOTION_DTYPE.itemsize,
                                dtype=torch.uint8, device=self.device) for t in range(3)]
        self.n_out = torch.zeros(3, dtype=torch.int32, device=self.device)
        self.freed = [torch.full((max(self.needs[t], 1),), -1, dtype=torch.int32,
                                 device=self.device) for t in range(3)]
        self.placed = [torch.full((max(self.max_in[t], 1),), -1, dtype=torch.int32,
                                  device=self.device) for t in range(3)]
        self.ws_bytes = max(cx.cascade_reclaim_workspace_bytes(n) for n in self.n)
        self.ws = torch.zeros(self.ws_bytes, dtype=torch.uint8, device=self.device)
        self.status = torch.zeros(1, dtype=torch.int32, device=self.device)
        self.index = None
        self.capacity = 0
        if index_keys is not None:
            hs, ts = index_facts(index_keys, index_masks)
            self.capacity = capacity or index_capacity(len(index_keys))
            self.index = torch.empty(cx.cascade_prefix_index_bytes(self.capacity),
                                     dtype=torch.uint8, device=self.device)
            s = stream_handle()
            rc = cx.cascade_prefix_index_clear(self.index.data_ptr(), self.capacity, s)
            ih = to_device(hs, self.device)
            it = to_device(ts, self.device, np.uint8)
            rc = rc or cx.cascade_prefix_index_insert(self.index.data_ptr(), self.capacity,
                                                      ih.data_ptr(), it.data_ptr(), len(hs),
                                                      self.status.data_ptr(), s)
            assert rc == 0, rc
            torch.cuda.synchronize(self.device)
            assert int(self.status.item()) == 0

    def call(self, t: int, stream=None) -> int:
        """Enqueue tier t's reclamation (its incoming = tier t-1's outgoing)."""
        v = self
        inc = v.out[t - 1].data_ptr() if t > 0 else 0
        n_inc = v.n_out[t - 1:t].data_ptr() if t > 0 else 0
        return cx.cascade_tier_reclaim(
            t, v.tabs[t], v.needs[t], inc, n_inc, v.max_in[t],
            v.out[t].data_ptr() if t < 2 else 0, v.n_out[t:t + 1].data_ptr(), v.max_out[t],
            v.freed[t].data_ptr(), v.placed[t].data_ptr(),
            v.index.data_ptr() if v.index is not None else 0, v.capacity, v.ws.data_ptr(),
            v.ws_bytes, v.status.data_ptr(), stream_handle(stream))

    def run(self, stream=None, tiers=(0, 1, 2)) -> int:
        for t in tiers:
            rc = self.call(t, stream)
            if rc:
                return rc
        return 0

    def chain_args(self):
        """The chain call's arguments over the same buffers, with a workspace
        of its own (the three per-tier workspaces back to back)."""
        torch = _torch()
        if getattr(self, "ws_chain", None) is None:
            self.ws_chain_bytes = cx.cascade_tier_chain_workspace_bytes(self.n)
            self.ws_chain = torch.zeros(self.ws_chain_bytes, dtype=torch.uint8,
                                        device=self.device)
            c = cx.TierChain()
            for t in range(3):
                c.table[t] = self.tabs[t]
                c.need[t] = self.needs[t]
                c.freed[t] = self.freed[t].data_ptr()
                c.placed[t] = self.placed[t].data_ptr() if t > 0 else 0
            for t in range(2):
                c.outgoing[t] = self.out[t].data_ptr()
                c.n_outgoing_dev[t] = self.n_out[t:t + 1].data_ptr()
                c.max_outgoing[t] = self.max_out[t]
            self.chain = c
        return self.chain

    def run_chain(self, stream=None) -> int:
        """The whole chain in one cascade_tier_reclaim_chain call."""
        c = self.chain_args()
        return cx.cascade_tier_reclaim_chain(
            c, self.index.data_ptr() if self.index is not None else 0, self.capacity,
            self.ws_chain.data_ptr(), self.ws_chain_bytes, self.status.data_ptr(),
            stream_handle(stream))

    def fetch(self) -> dict:
        torch = _torch()
        torch.cuda.synchronize(self.device)
        n_out = self.n_out.cpu().numpy()
        res = {"status": int(self.status.item()), "tiers": []}
        for t in range(3):
            n_in = int(n_out[t - 1]) if t > 0 else 0
            no = int(n_out[t]) if t < 2 else 0
            out = np.frombuffer(self.out[t].cpu().numpy().tobytes(), cx.DEMOTION_DTYPE)[:no]
            res["tiers"].append({
                "freed": self.freed[t].cpu().numpy()[:self.needs[t]],
                "placed": self.placed[t].cpu().numpy()[:n_in],
                "outgoing": out, "n_outgoing": no,
                "block_hash": self.bh[t].cpu().numpy().view(np.uint64)[:self.n[t]],
                "last_use_ns": self.lu[t].cpu().numpy()[:self.n[t]]})
        if self.index is not None:
            res["index"] = index_contents(self.index.cpu().numpy())
        return res
