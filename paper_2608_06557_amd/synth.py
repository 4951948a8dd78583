"""Seeded synthetic request populations for the scheduling step.

This module only draws inputs: request fields, block tables, free lists,
parameters and KV payload bit patterns.  It holds none of the scheduling
method's arithmetic (no latency model, budget, order or admission), so
both the GPU library and the CPU oracle can be fed from it.

The Aliyun Bailian production traces used by the paper (Section 5,
"Workloads and Traces") are not available here; these populations stand in
for them.  Their shapes follow the paper's Table 2 (input/output lengths of
ChatBot / Tool&Agent / Coder / Reasoning), Table 3 (seconds-scale TTFT
targets) and Section 5's serving setup (chunk 512, max batch 128).

Five workloads (``make_workload(cfg)``):
  0  256 chat requests, 3 SLO classes, 8B-class KV, 4096-block pool
  1  8192 chat requests, 5 classes, 65536-block pool, token cap 16384
  2  65536 requests, 80% chat / 20% agentic, 200 GB pool
  3  reasoning-heavy, prefix-shared, high load, exact budget ties
  4  262144 requests, 70B-class KV, 250 GB pool, token cap 32768
"""
from __future__ import annotations

import numpy as np

QUEUED, RUNNING_PREFILL, DECODE = 0, 1, 2
QT_NEW, QT_TIER1, QT_TIER2 = 0, 1, 2
KV_HBM, KV_DRAM, KV_NVME, KV_NONE = 0, 1, 2, 3

T_NOW_NS = 10 ** 12
BLOCK_TOKENS = 16
CHUNK_TOKENS = 512           # Section 5: chunk size of 512 tokens
MAX_BATCH = 128              # Section 5: maximum batch size of 128
GAMMA_Q16 = 81920            # guardband 1.25 (the paper gives no value)
TIER2_RESERVE_Q16 = 4096     # 1/16 of the token cap reserved for Tier-2
SEC = 10 ** 9

# Synthetic MI355X-class per-iteration cost coefficients (picoseconds).
COSTS = {
    "8b": dict(c_iter_ps=2_000_000_000, c_decode_ps=33_000_000,
               c_token_ps=12_800_000, c_attn_ps=420),
    "70b": dict(c_iter_ps=17_500_000_000, c_decode_ps=80_000_000,
                c_token_ps=112_000_000, c_attn_ps=2_100),
}
# KV geometry: 8 KV heads x head_dim 128 x bf16 x 16 tokens = 32 KiB per
# (layer, K or V) chunk of one block.
GEOMETRY = {"8b": dict(num_layers=32), "70b": dict(num_layers=80)}
CHUNK_BYTES = 8 * 128 * 2 * BLOCK_TOKENS

# Links on the restore paths (Section 4.3): DRAM<->HBM and NVMe->DRAM,
# given as bandwidth (bytes/s) and a fixed per-transfer overhead (ns).
LINKS = {"dram_hbm": (55e9, 10_000), "nvme_dram": (14e9, 100_000)}


def block_bytes(model: str) -> int:
    return 2 * GEOMETRY[model]["num_layers"] * CHUNK_BYTES


def link_params(model: str) -> tuple[list[int], list[int]]:
    """Per-link fixed overhead (ns) and time per KV block (ns, rounded up).

    Unit conversion of the link specification only."""
    bb = block_bytes(model)
    delta, blk = [], []
    for name in ("dram_hbm", "nvme_dram"):
        bw, d = LINKS[name]
        blk.append(int(-(-bb * SEC // int(bw))))
        delta.append(d)
    return delta, blk


CONFIGS = {
    0: dict(n=256, model="8b", slo_s=[2, 10, 60], mix={"chat": 1.0},
            tiers=(0.50, 0.30, 0.00, 0.20), load_decodes=64, pool=4096,
            token_cap=8192, max_move=2 ** 31 - 1, elapsed_frac=1.0),
    # config 0's three targets plus two looser ones: with waits uniform over
    # the target, the least-budget head of a queue this long still has
    # budget to restore and spill
    1: dict(n=8192, model="8b", slo_s=[2, 10, 60, 120, 300], mix={"chat": 1.0},
            tiers=(0.35, 0.40, 0.10, 0.15), load_decodes=64, pool=65536,
            token_cap=16384, max_move=512, elapsed_frac=1.0),
    2: dict(n=65536, model="8b", slo_s=[1, 2, 10, 30, 60], mix={"chat": 0.8, "agentic": 0.2},
            classes={"chat": [0, 1, 2], "agentic": [2, 3, 4]},
            tiers=(0.35, 0.40, 0.10, 0.15), load_decodes=64, pool=95367,
            token_cap=16384, max_move=954, elapsed_frac=0.5),
    3: dict(n=65536, model="8b", slo_s=[1, 2, 10, 30, 60],
            mix={"reasoning": 0.5, "chat": 0.25, "agentic": 0.25},
            classes={"chat": [0, 1, 2], "agentic": [2, 3, 4], "reasoning": [3, 4]},
            tiers=(0.35, 0.40, 0.10, 0.15), load_decodes=MAX_BATCH - 1, pool=95367,
            token_cap=16384, max_move=954, elapsed_frac=None, shared_prefix=True,
            family_kind="reasoning", nominal_all_tokens=True, nominal_fixed_ms=20,
            nominal_tok_s=10_000, eps_ms=[-20, -10, 0, 10, 20]),
    # 70B-class targets are looser, as Table 3's grow with model size
    4: dict(n=262144, model="70b", slo_s=[2, 5, 10, 30, 60], mix={"chat": 0.8, "agentic": 0.2},
            classes={"chat": [0, 1, 2], "agentic": [4]},
            tiers=(0.40, 0.35, 0.15, 0.10), load_decodes=64, pool=47683,
            token_cap=32768, max_move=1526, elapsed_frac=0.5),
}

# Lognormal length laws (mu, sigma, clip) per request class.
LENGTHS = {
    "chat": dict(n_in=(6.0, 1.0, 16, 8192), n_out=(5.0, 1.0, 1, 65536)),
    "agentic": dict(n_in=(9.0, 0.7, 16, 131072), n_out=(7.0, 1.0, 1, 65536)),
    # fitted to Table 2's Reasoning row: input p50 3680, p95 16221
    "reasoning": dict(n_in=(8.21, 0.90, 16, 131072), n_out=(8.0, 1.0, 1, 131072)),
}


def _lognormal(rng, law, size):
    mu, sigma, lo, hi = law
    return np.clip(np.rint(rng.lognormal(mu, sigma, size)), lo, hi).astype(np.int64)


def make_params(cfg: int | dict, load_decodes=None) -> dict:
    c = CONFIGS[cfg] if isinstance(cfg, int) else cfg
    delta, blk = link_params(c["model"])
    slo = [int(s * SEC) for s in c["slo_s"]]
    p = dict(t_now_ns=T_NOW_NS, num_classes=len(slo), slo_ns=slo + [0] * (16 - len(slo)),
             block_tokens=BLOCK_TOKENS, chunk_tokens=CHUNK_TOKENS,
             load_decodes=c["load_decodes"] if load_decodes is None else load_decodes,
             max_batch=MAX_BATCH, gamma_q16=GAMMA_Q16, token_cap=c["token_cap"],
             tier2_reserve_q16=TIER2_RESERVE_Q16, max_move_blocks=c["max_move"],
             num_blocks=c["pool"], link_delta_ns=delta, link_blk_ns=blk)
    p.update(COSTS[c["model"]])
    return p


def kv_geometry(model: str, num_blocks: int, layout: str = "layer_major",
                chunk_bytes: int = CHUNK_BYTES) -> dict:
    """Strides (bytes) of a paged KV pool.

    layer_major: one K and one V cache per layer, each [num_blocks, chunk]
    (per-layer paged caches).  block_major: all layers of a block together."""
    L = GEOMETRY[model]["num_layers"]
    if layout == "layer_major":
        g = dict(slot_stride=chunk_bytes, kv_stride=num_blocks * chunk_bytes,
                 layer_stride=2 * num_blocks * chunk_bytes)
    elif layout == "block_major":
        g = dict(slot_stride=2 * L * chunk_bytes, kv_stride=chunk_bytes,
                 layer_stride=2 * chunk_bytes)
    else:
        raise ValueError(layout)
    g.update(num_layers=L, chunk_bytes=chunk_bytes, num_blocks=num_blocks,
             pool_bytes=2 * L * num_blocks * chunk_bytes)
    return g


def make_workload(cfg: int, seed: int | None = None, n: int | None = None,
                  prefix_groups: bool = False) -> dict:
    """Draw one synthetic scheduling-step input.

    Returns a dict of numpy arrays (request SoA, block table, free list) plus
    ``params`` (integers), ``geometry`` and ``config``.  With
    ``prefix_groups`` (workloads with shared prefixes), also a
    ``prefix_group`` array: the shared prefix each request extends, -1 for
    the others."""
    c = dict(CONFIGS[cfg])
    if n is not None:
        c["n"] = n
    n = c["n"]
    rng = np.random.Generator(np.random.PCG64(1000 + cfg if seed is None else seed))
    bt = BLOCK_TOKENS
    ncls = len(c["slo_s"])
    slo_ns = np.array([int(s * SEC) for s in c["slo_s"]], np.int64)

    # population class per request
    names = list(c["mix"])
    kind = rng.choice(len(names), size=n, p=[c["mix"][k] for k in names])
    n_in = np.zeros(n, np.int64)
    n_out = np.zeros(n, np.int64)
    for j, name in enumerate(names):
        m = kind == j
        n_in[m] = _lognormal(rng, LENGTHS[name]["n_in"], int(m.sum()))
        n_out[m] = _lognormal(rng, LENGTHS[name]["n_out"], int(m.sum()))
    # SLO targets are bound to the application class (Section 4.1, Table 3):
    # a class draws uniformly from its own subset of the SLO classes.
    slo_class = rng.integers(0, ncls, n).astype(np.int64)
    for j, name in enumerate(names):
        allowed = c.get("classes", {}).get(name)
        if allowed is not None:
            m = kind == j
            slo_class[m] = rng.choice(np.array(allowed), int(m.sum()))

    # prefix residency: tier drawn per request; the cached prefix is 50..100%
    # of the prompt (earlier turns of a conversation or agent loop)
    # A long prompt is long because of context accumulated in earlier turns,
    # so "no cached prefix" is drawn only for prompts shorter than the median
    # of their class (twice as often there); the tier marginals are kept.
    p_hbm, p_dram, p_nvme, p_none = c["tiers"]
    cached = np.array([p_hbm, p_dram, p_nvme]) / (1.0 - p_none)
    tier = rng.choice(3, size=n, p=cached)
    short = np.zeros(n, bool)
    for j in range(len(names)):
        m = kind == j
        if m.any():
            short[m] = n_in[m] < np.median(n_in[m])
    tier = np.where(short & (rng.random(n) < 2.0 * p_none), KV_NONE, tier)
    frac = rng.uniform(0.5, 1.0, n)
    n_prefix = bt * np.floor(frac * n_in / bt).astype(np.int64)
    n_prefix = np.minimum(n_prefix, bt * ((n_in - 1) // bt))
    arrival_jitter = None
    group = np.full(n, -1, np.int64)

    if c.get("shared_prefix"):
        # 30% of requests extend one of 512 shared prefixes of 1k..32k tokens;
        # they come in families of 4 parallel samples of one reasoning prompt
        # with the same suffix length, class and arrival time (exact ties in
        # every field).
        nfam_req = int(0.3 * n) // 4 * 4
        fam_ids = rng.permutation(n)[:nfam_req].reshape(-1, 4)
        pre_len = bt * (rng.integers(1024, 32769, 512) // bt)
        pre_tier = rng.choice(4, size=512, p=list(c["tiers"]))
        which = rng.integers(0, 512, fam_ids.shape[0])
        lead = fam_ids[:, 0]
        fam_kind = c.get("family_kind")
        if fam_kind is not None:
            # parallel samples of one prompt: the family takes that kind's
            # length law for its own suffix and one of that kind's classes
            kj = names.index(fam_kind)
            kind[lead] = kj
            n_in[lead] = _lognormal(rng, LENGTHS[fam_kind]["n_in"], len(lead))
            n_out[lead] = _lognormal(rng, LENGTHS[fam_kind]["n_out"], len(lead))
            slo_class[lead] = rng.choice(np.array(c["classes"][fam_kind]), len(lead))
        for col in range(4):
            members = fam_ids[:, col]
            group[members] = which
            n_in[members] = pre_len[which] + n_in[lead]
            n_out[members] = n_out[lead]
            slo_class[members] = slo_class[lead]
            kind[members] = kind[lead]
            tier[members] = pre_tier[which]
            n_prefix[members] = pre_len[which]
        n_in = np.minimum(n_in, 131072)
        n_prefix = np.minimum(n_prefix, bt * ((n_in - 1) // bt))
        # High load: every request has already waited about its SLO minus a
        # nominal service time (a fixed 20 ms plus its prompt at 10k tokens/s),
        # give or take up to 20 ms: a queueing-delay model, not the
        # scheduler's estimator.  Budgets end up small against the targets
        # (median about 0.5 s), a few of them already negative.
        uncached = np.where((tier == KV_NONE) | c.get("nominal_all_tokens", False),
                            n_in, n_in - n_prefix)
        nominal = (c.get("nominal_fixed_ms", 0) * 10 ** 6
                   + (uncached * SEC) // c.get("nominal_tok_s", 25_000))
        eps = rng.choice(np.array(c.get("eps_ms", [-20, -10, 0, 10, 20]), np.int64) * 10 ** 6, n)
        elapsed = slo_ns[slo_class] - nominal - eps
        fam_lead_elapsed = elapsed[lead]
        for col in range(4):
            elapsed[fam_ids[:, col]] = fam_lead_elapsed
        elapsed = np.clip(elapsed, 0, slo_ns[slo_class])
        arrival_jitter = elapsed
    no_prefix = (tier == KV_NONE) | (n_prefix <= 0)
    tier = np.where(no_prefix, KV_NONE, tier)
    n_prefix = np.where(no_prefix, 0, n_prefix)

    if arrival_jitter is None:
        hi = (slo_ns[slo_class] * c["elapsed_frac"]).astype(np.int64)
        elapsed = (rng.random(n) * (hi + 1)).astype(np.int64)
    arrival = T_NOW_NS - elapsed

    # state: QUEUED 90%, RUNNING_PREFILL 4%, DECODE 6%, while running rows fit
    # in 60% of the pool
    state = rng.choice(3, size=n, p=[0.90, 0.04, 0.06])
    u1 = rng.random(n)
    prog = np.zeros(n, np.int64)
    rp = state == RUNNING_PREFILL
    prog[rp] = 1 + np.floor(u1[rp] * (n_in[rp] - 1)).astype(np.int64)
    de = state == DECODE
    prog[de] = np.floor(u1[de] * n_out[de]).astype(np.int64)
    rows = np.zeros(n, np.int64)
    rows[rp] = -(-prog[rp] // bt)
    rows[de] = -(-(n_in[de] + prog[de]) // bt)
    budget = int(0.6 * c["pool"])
    cum = 0
    for i in np.flatnonzero(state != QUEUED):
        if cum + rows[i] <= budget:
            cum += int(rows[i])
        else:
            state[i] = QUEUED
            prog[i] = 0
            rows[i] = 0
    queued = state == QUEUED
    # a running request's cached prefix is already part of its computed tokens
    queue_tier = rng.choice(3, size=n, p=[0.25, 0.65, 0.10])
    queue_tier[de] = QT_TIER1

    nnz = int(rows.sum())
    perm = rng.permutation(c["pool"])
    slots = perm[:nnz].astype(np.int32)
    row_offsets = np.zeros(n + 1, np.int64)
    row_offsets[1:] = np.cumsum(rows)
    n_free = min(c["token_cap"] // bt, c["pool"] - nnz)
    free_slots = perm[nnz:nnz + n_free].astype(np.int32)

    ids = np.cumsum(rng.integers(1, 4, n)).astype(np.uint64) + np.uint64(10 ** 6)
    params = make_params(c)
    extra = {"prefix_group": group.astype(np.int32)} if prefix_groups else {}
    return dict(
        **extra, id=ids, slo_class=slo_class.astype(np.uint8), state=state.astype(np.uint8),
        queue_tier=queue_tier.astype(np.uint8), prefix_tier=tier.astype(np.uint8),
        arrival_ns=arrival.astype(np.int64), n_in=n_in.astype(np.int32),
        n_out_pred=n_out.astype(np.int32), n_prefix=n_prefix.astype(np.int32),
        n_progress=prog.astype(np.int32), row_offsets=row_offsets.astype(np.int32),
        slots=slots, free_slots=free_slots, params=params,
        geometry=kv_geometry(c["model"], c["pool"]), config=cfg, queued=queued,
    )


# ------------------------------------------------------ save and replay

def save_workload(w: dict, path: str) -> None:
    """One step's inputs (request arrays, block table, free list, optional
    prefix groups, parameters) to an .npz file (no pickled objects)."""
    import json
    arrays = {k: np.asarray(v) for k, v in w.items()
              if isinstance(v, np.ndarray) and k not in ("queued",)}
    arrays["params_json"] = np.frombuffer(json.dumps(w["params"]).encode(), np.uint8)
    np.savez_compressed(path, **arrays)


def load_workload(path: str) -> dict:
    """The inverse of save_workload (loads with allow_pickle=False)."""
    import json
    with np.load(path, allow_pickle=False) as z:
        w = {k: z[k] for k in z.files if k != "params_json"}
        w["params"] = json.loads(bytes(z["params_json"]).decode())
    return w


# ------------------------------------------------------------ KV payload

def hash32_np(word_index: np.ndarray, seed: int) -> np.ndarray:
    """Counter-based 32-bit pattern of a 4-byte word index (numpy)."""
    x = (word_index.astype(np.uint64) + np.uint64(seed * 0x9E3779B9 & 0xFFFFFFFF)) & np.uint64(0xFFFFFFFF)
    x = (x * np.uint64(0x7FEB352D)) & np.uint64(0xFFFFFFFF)
    x ^= x >> np.uint64(15)
    x = (x * np.uint64(0x346CA68B)) & np.uint64(0xFFFFFFFF)
    x ^= x >> np.uint64(16)
    return x.astype(np.uint32)


def hash32_torch(word_index, seed: int):
    """The same pattern with torch int64 ops (runs on any device)."""
    import torch
    m = 0xFFFFFFFF
    x = (word_index + (seed * 0x9E3779B9 & m)) & m
    x = (x * 0x7FEB352D) & m
    x = x ^ (x >> 15)
    x = (x * 0x346CA68B) & m
    x = x ^ (x >> 16)
    return x.to(torch.int64)


def block_hash64(req: np.ndarray, blk: np.ndarray, seed: int) -> np.ndarray:
    """Stand-in for a chained per-block prefix hash: a nonzero 64-bit value
    per (request or shared-prefix id, block index), two counter-based words."""
    key = (req.astype(np.int64) * np.int64(1 << 20) + blk.astype(np.int64)).astype(np.uint64)
    k_lo = (key & np.uint64(0xFFFFFFFF)).astype(np.int64)
    k_hi = (key >> np.uint64(32)).astype(np.int64)
    x1 = hash32_np(k_lo, seed).astype(np.int64)
    x2 = hash32_np(k_hi ^ x1, seed + 1).astype(np.uint64)
    x3 = hash32_np(k_lo ^ x2.astype(np.int64), seed + 2).astype(np.uint64)
    h = (x2 << np.uint64(32)) | x3
    return np.where(h == 0, np.uint64(1), h)


def make_prefix_workload(cfg: int, seed: int | None = None, n: int | None = None,
                         shared_frac: float = 0.0, dup_frac: float = 0.3,
                         gap_frac: float = 0.2, noise: int = 0) -> dict:
    """Inputs of the prefix-hit lookup: every request's prompt block hashes
    (its full blocks, CSR) and a cache index of (block hash, tier) facts.

    A request's cached run is the first n_prefix / bt blocks of the step
    workload, in its prefix tier.  Extras that a lookup must see through:
    shallower duplicates of cached blocks (dup_frac of the requests), a
    cached block past the first uncached one (gap_frac), unrelated entries
    (noise), and families of requests sharing leading blocks (shared_frac;
    members take their family head's cached run and tier)."""
    w = make_workload(cfg, seed=seed, n=n)
    rng = np.random.Generator(np.random.PCG64((7919 + cfg) if seed is None else seed + 7919))
    bt = BLOCK_TOKENS
    n = len(w["n_in"])
    n_in = np.asarray(w["n_in"], np.int64)
    full = n_in // bt
    pre_blocks = np.asarray(w["n_prefix"], np.int64) // bt
    tier = np.asarray(w["prefix_tier"], np.uint8).copy()
    owner = np.arange(n, dtype=np.int64)      # whose hash sequence a request's blocks use
    if shared_frac > 0 and n > 1:
        members = np.flatnonzero(rng.random(n) < shared_frac)
        heads = rng.integers(0, n, len(members))
        for m, hd in zip(members, heads):
            owner[m] = owner[hd]
            cap = (n_in[m] - 1) // bt
            pre_blocks[m] = min(pre_blocks[hd], cap, full[m])
            tier[m] = tier[hd]
    offsets = np.zeros(n + 1, np.int64)
    offsets[1:] = np.cumsum(full)
    req_of = np.repeat(np.arange(n), full)
    blk_of = np.arange(offsets[-1]) - offsets[req_of]
    hashes = block_hash64(owner[req_of], blk_of, 17 + cfg)
    cached = blk_of < pre_blocks[req_of]
    cached &= tier[req_of] <= 2
    ih = [hashes[cached]]
    it = [tier[req_of][cached]]
    dup = cached & (rng.random(len(hashes)) < dup_frac)
    ih.append(hashes[dup])
    it.append(rng.integers(0, 3, int(dup.sum())).astype(np.uint8) % (tier[req_of][dup] + 1))
    gap = (blk_of == pre_blocks[req_of] + 1) & (rng.random(len(hashes)) < gap_frac)
    ih.append(hashes[gap])
    it.append(rng.integers(0, 3, int(gap.sum())).astype(np.uint8))
    if noise:
        ih.append(block_hash64(np.full(noise, -1), np.arange(noise), 29 + cfg))
        it.append(rng.integers(0, 3, noise).astype(np.uint8))
    ih = np.concatenate(ih)
    it = np.concatenate(it)
    pre_blocks = np.where(tier <= 2, pre_blocks, 0)
    order = rng.permutation(len(ih))
    return {"n_in": w["n_in"].astype(np.int32), "block_offsets": offsets.astype(np.int32),
            "block_hashes": hashes, "index_hashes": ih[order], "index_tiers": it[order],
            "block_tokens": bt, "expect_blocks": pre_blocks, "expect_tier": tier}


# Capacities of the deeper tiers, in KV blocks: 1 TiB of host DRAM and 8 TiB
# of NVMe per instance, of the model's block size.
TIER_BYTES = (None, 1 << 40, 8 << 40)


def tier_sizes(cfg: int) -> tuple[int, int, int]:
    p = make_params(cfg)
    bb = block_bytes(CONFIGS[cfg]["model"])
    return int(p["num_blocks"]), TIER_BYTES[1] // bb, TIER_BYTES[2] // bb


def make_tier_workload(cfg: int = 2, seed: int | None = None, sizes=None, needs=None,
                       held=(0.6, 0.05, 0.01), empty=(0.002, 0.001, 0.0002),
                       overlap=(0.3, 0.2), index_frac: float = 1.0,
                       stamp_scale_s=(30.0, 600.0, 3600.0)) -> dict:
    """Slot tables of HBM, DRAM and NVMe for one reclamation chain.

    Every tier holds distinct block hashes; a share `overlap[k]` of tier k's
    blocks also sits one tier deeper (copies kept after a restore).  A share
    `held[k]` of the slots is in use and `empty[k]` holds nothing (near full:
    in steady state every tier reclaims cached blocks).  Last uses
    are nanosecond stamps before t_now, exponentially spread with a mean of
    stamp_scale_s[k] seconds for HBM and DRAM (recent blocks sit high) and
    uniform over that many seconds for NVMe.  The index holds the tier set of
    a share `index_frac` of the blocks.  Default needs are what one step can
    take: HBM the token cap's blocks plus the restore cap, DRAM the restore
    cap (spills of preempted prefills), NVMe nothing beyond the demotions;
    both at most half of HBM's free slots."""
    cfg_seed = (6007 + cfg) if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(cfg_seed + 7001))
    p = make_params(cfg)
    if sizes is None:
        sizes = tier_sizes(cfg)
    sizes = [int(x) for x in sizes]
    if needs is None:
        u = min(int(p["max_move_blocks"]), sizes[0])
        # at most half of HBM's free slots (a small pool is mostly held)
        room = int(sizes[0] * (1.0 - held[0]) / 2)
        needs = (min(int(p["token_cap"]) // int(p["block_tokens"]) + u, room), min(u, room), 0)
    t_now = np.int64(1_700_000_000_000_000_000)
    ids = []
    next_id = 1
    for k, n in enumerate(sizes):
        n_copy = int(round(overlap[k - 1] * len(ids[k - 1]))) if k > 0 else 0
        n_copy = min(n_copy, n)
        copy = rng.choice(ids[k - 1], n_copy, replace=False) if n_copy else np.zeros(0, np.int64)
        fresh = np.arange(next_id, next_id + (n - n_copy), dtype=np.int64)
        next_id += n - n_copy
        ids.append(rng.permutation(np.concatenate([copy, fresh])))
    tables = []
    for k, n in enumerate(sizes):
        bh = block_hash64(ids[k], np.zeros(n, np.int64), cfg_seed + 11)
        bh[rng.random(n) < empty[k]] = 0
        # one copy of a block per tier, even if two ids hashed alike
        _, first = np.unique(bh, return_index=True)
        dup = np.ones(n, bool)
        dup[first] = False
        bh[dup] = 0
        scale = stamp_scale_s[k] * 1e9
        age = rng.exponential(scale, n) if k < 2 else rng.uniform(0, scale, n)
        lu = (t_now - age.astype(np.int64)).astype(np.int64)
        lu[bh == 0] = rng.integers(0, 1 << 40, int((bh == 0).sum()))  # ignored for empty slots
        hd = (rng.random(n) < held[k]).astype(np.uint8)
        tables.append({"block_hash": bh, "last_use_ns": lu, "held": hd})
    # tier sets: each hash sits at most once per tier, so summing bits is OR
    hs = np.concatenate([t["block_hash"][t["block_hash"] != 0] for t in tables])
    bits = np.concatenate([np.full(int((t["block_hash"] != 0).sum()), 1 << k, np.uint8)
                           for k, t in enumerate(tables)])
    keys, inv = np.unique(hs, return_inverse=True)
    masks = np.zeros(len(keys), np.uint8)
    np.add.at(masks, inv, bits)
    if index_frac < 1.0:
        keep = rng.random(len(keys)) < index_frac
        keys, masks = keys[keep], masks[keep]
    return {"tables": tables, "index_keys": keys.astype(np.uint64), "index_masks": masks,
            "needs": tuple(int(x) for x in needs), "sizes": tuple(sizes)}
