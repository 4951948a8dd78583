"""GPU parity of the per-tier LRU reclamation chain (Section 4.4: free blocks
reclaimed least-recently-used within each tier, cold blocks demoted one tier
deeper) against the oracle, bit-exact: every tier's freed and placed slots,
demoted blocks, slot tables and the index's tier sets, over HBM -> DRAM ->
NVMe chains at full tier sizes and over small tables with tile tails, heavy
ties, extreme stamps, no index, partial indexes and every error path."""
import numpy as np
import pytest
import torch  # noqa: F401  (imported at collection: the first import is slow)

from oracle import ref
from paper_2608_06557_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    from paper_2608_06557_amd import cascade, device
    assert torch.cuda.is_available()
    cascade.load()
    return device


def oracle_chain(w, tiers=(0, 1, 2)):
    """The oracle over the chain; stops at the first failing tier like the
    device chain, which shares one status word."""
    keys = w.get("index_keys")
    masks = w.get("index_masks")
    outs, inc, rc = [], None, 0
    for t in tiers:
        tb = w["tables"][t]
        r = ref.tier_reclaim(t, tb["block_hash"], tb["last_use_ns"], tb["held"], w["needs"][t],
                             incoming=inc, max_outgoing=0 if t == 2 else None,
                             index_keys=keys, index_masks=masks)
        outs.append(r)
        if r["rc"] != 0:
            rc = r["rc"]
            break
        inc, masks = r["outgoing"], r["index_masks"]
    return rc, outs, masks


def assert_same_results(g, h, label=""):
    """Two device runs of a chain gave the same status, outputs and index."""
    assert g["status"] == h["status"], (label, g["status"], h["status"])
    for t in range(3):
        a, b = g["tiers"][t], h["tiers"][t]
        assert a["n_outgoing"] == b["n_outgoing"], (label, t)
        for k in ["freed", "placed", "block_hash", "last_use_ns"]:
            assert np.array_equal(a[k], b[k]), (label, t, k)
        assert np.array_equal(a["outgoing"].view(np.uint8), b["outgoing"].view(np.uint8)), \
            (label, t)
    assert ("index" in g) == ("index" in h)
    if "index" in g:
        for x, y in zip(g["index"], h["index"]):
            assert np.array_equal(x, y), label


def run_both(dev, w, index=True, capacity=None):
    """The chain as three per-tier calls and as one chain call (each on
    tables of its own), checked equal to each other; the per-tier results,
    the oracle's and the per-tier DeviceTiers are returned."""
    keys = w["index_keys"] if index else None
    masks = w["index_masks"] if index else None
    d = dev.DeviceTiers(w["tables"], w["needs"], keys, masks, capacity=capacity)
    assert d.run() == 0
    g = d.fetch()
    dc = dev.DeviceTiers(w["tables"], w["needs"], keys, masks, capacity=capacity)
    assert dc.run_chain() == 0
    assert_same_results(g, dc.fetch(), "one chain call")
    ow = dict(w)
    if not index:
        ow["index_keys"] = ow["index_masks"] = None
    rc, outs, masks = oracle_chain(ow)
    return g, rc, outs, masks, d


def assert_chain_same(w, g, rc, outs, masks, label=""):
    assert g["status"] == rc, (label, g["status"], rc)
    for t in range(3):
        gt = g["tiers"][t]
        tb = w["tables"][t]
        if t >= len(outs) or outs[t]["rc"] != 0:
            # a failed call and the calls after it write nothing
            assert np.array_equal(gt["block_hash"], tb["block_hash"]), (label, t)
            assert np.array_equal(gt["last_use_ns"], tb["last_use_ns"]), (label, t)
            continue
        o = outs[t]
        for k in ["freed", "placed", "block_hash", "last_use_ns"]:
            if not np.array_equal(gt[k], o[k]):
                bad = np.flatnonzero(np.asarray(gt[k]) != np.asarray(o[k]))
                raise AssertionError(f"{label} tier {t} {k}: {len(bad)} differ, first {bad[:5]}")
        assert gt["n_outgoing"] == o["n_outgoing"], (label, t)
        for f in ["hash", "last_use_ns", "src_slot"]:
            assert np.array_equal(gt["outgoing"][f], o["outgoing"][f]), (label, t, f)
    if rc == 0 and w.get("index_keys") is not None and "index" in g:
        gk, gm = g["index"]
        assert np.array_equal(gk, np.asarray(w["index_keys"], np.uint64)), label
        assert np.array_equal(gm, np.asarray(masks).astype(np.uint32)), label


@pytest.mark.parametrize("cfg", [0, 2, 4])
def test_full_size_chain_matches_oracle(dev, cfg):
    w = synth.make_tier_workload(cfg)
    print(f"tier chain cfg {cfg}: sizes {w['sizes']} needs {w['needs']}", flush=True)
    g, rc, outs, masks, _ = run_both(dev, w)
    assert rc == 0
    assert_chain_same(w, g, rc, outs, masks, f"cfg {cfg}")
    # the chain really demoted through every tier
    assert outs[0]["n_outgoing"] > 0 and outs[1]["n_outgoing"] > 0


def small(seed, sizes, needs, held=(0.3, 0.1, 0.05), empty=(0.05, 0.05, 0.05),
          index_frac=1.0, **kw):
    return synth.make_tier_workload(0, seed=seed, sizes=sizes, needs=needs, held=held,
                                    empty=empty, index_frac=index_frac, **kw)


CASES = [
    # sizes straddling tiles of 2048 slots and vectors of 8
    ((1, 7, 9), (0, 0, 0)),
    ((2047, 2048, 2049), (300, 200, 100)),
    ((2049, 4096, 6150), (900, 500, 0)),
    ((5000, 9000, 20011), (1500, 700, 300)),
    ((300, 301, 1999), (100, 37, 5)),
    # a tier with no slots at all: nothing to reclaim, or no room for the
    # demotions it receives (ENOSPC at DRAM)
    ((0, 3000, 2000), (0, 100, 10)),
    ((500, 0, 700), (50, 0, 0)),
]


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("seed", [1, 2])
def test_small_chains(dev, case, seed):
    sizes, needs = CASES[case]
    w = small(seed * 31 + case, sizes, needs)
    g, rc, outs, masks, _ = run_both(dev, w)
    assert_chain_same(w, g, rc, outs, masks, f"case {case} seed {seed}")


def test_nearly_full_index(dev):
    # an index at load 0.9: many blocks sit past their home slot, so the
    # compaction's gathered lookups (tiers 0 and 1) and the write kernel's
    # (tier 2) continue probing one lookup at a time
    w = small(41, (3500, 6000, 8200), (1000, 500, 100))
    keys = len(w["index_keys"])
    cap = 1 << int(np.ceil(np.log2(keys + 1)))
    assert keys / cap > 0.85, keys / cap
    g, rc, outs, masks, _ = run_both(dev, w, capacity=cap)
    assert rc == 0
    assert_chain_same(w, g, rc, outs, masks, "index at load 0.9")
    assert outs[0]["n_outgoing"] > 0 and outs[1]["n_outgoing"] > 0


@pytest.mark.parametrize("seed", range(12))
def test_random_chains(dev, seed):
    # seeded random chains: table sizes across tile boundaries, held and
    # empty shares, needs (some beyond the free slots: ENOSPC at some tier),
    # full or partial index; both call paths against the oracle
    rng = np.random.default_rng(900 + seed)
    sizes = tuple(int(x) for x in rng.integers(1, 9000, 3))
    held = tuple(float(x) for x in rng.uniform(0.0, 0.6, 3))
    empty = tuple(float(x) for x in rng.uniform(0.0, 0.3, 3))
    needs = tuple(int(rng.integers(0, max(1, int(sz * 0.5)) + 1)) for sz in sizes)
    w = small(900 + seed, sizes, needs, held=held, empty=empty,
              index_frac=float(rng.choice([1.0, 0.7])))
    print(f"random chain {seed}: sizes {sizes} needs {needs}", flush=True)
    g, rc, outs, masks, _ = run_both(dev, w)
    assert_chain_same(w, g, rc, outs, masks, f"random chain {seed}")


def test_empty_slots_alone_suffice_and_ties_split(dev):
    # plenty of empty slots: the threshold is the empty key, cut mid-way in
    # slot order; DRAM then takes exactly its empties
    w = small(5, (6000, 3000, 3000), (400, 10, 0), empty=(0.5, 0.2, 0.3))
    n_empty1 = int(((w["tables"][1]["block_hash"] == 0) & (w["tables"][1]["held"] == 0)).sum())
    w["needs"] = (400, 0, 0)
    g, rc, outs, masks, _ = run_both(dev, w)
    assert_chain_same(w, g, rc, outs, masks, "empties")
    assert outs[0]["n_outgoing"] == 0
    w2 = small(5, (6000, 3000, 3000), (0, n_empty1, 0), empty=(0.5, 0.2, 0.3))
    g, rc, outs, masks, _ = run_both(dev, w2)
    assert_chain_same(w2, g, rc, outs, masks, "exact empties")


def test_heavy_ties_and_extreme_stamps(dev):
    rng = np.random.default_rng(9)
    for stamps in ["ties", "extreme"]:
        w = small(17, (7000, 8000, 9000), (2500, 1200, 0))
        for t in w["tables"]:
            n = len(t["block_hash"])
            if stamps == "ties":
                t["last_use_ns"] = rng.integers(0, 3, n).astype(np.int64)
            else:
                t["last_use_ns"] = np.where(rng.random(n) < 0.5, 0,
                                            2**63 - 1 - rng.integers(0, 3, n)).astype(np.int64)
        g, rc, outs, masks, _ = run_both(dev, w)
        assert_chain_same(w, g, rc, outs, masks, stamps)


def test_threshold_prefix_shared_by_more_than_the_stage(dev):
    # NVMe: 80 % of the slots share one stamp, the oldest, and the rest lie
    # far above it, so the threshold's key and its first 20 bits are shared by
    # about 240 000 candidates: more than the select kernel stages, so it
    # resolves them from the whole list
    rng = np.random.default_rng(71)
    w = small(71, (3000, 4000, 300_000), (600, 300, 5000), empty=(0.05, 0.05, 0.0))
    t = w["tables"][2]
    n = len(t["block_hash"])
    t["last_use_ns"] = np.where(rng.random(n) < 0.8, 1_000_000,
                                rng.integers(2_000_000, 2 ** 40, n)).astype(np.int64)
    g, rc, outs, masks, _ = run_both(dev, w)
    assert rc == 0
    assert_chain_same(w, g, rc, outs, masks, "shared threshold prefix")


def test_more_tiles_than_the_select_kernel_keeps_in_lds(dev):
    # 2100 tiles of 2048 slots (above 2048): the select kernel keeps its
    # per-tile counts in memory instead of LDS
    w = small(73, (3000, 4000, 4_300_000), (600, 300, 3000), empty=(0.05, 0.05, 0.0))
    g, rc, outs, masks, _ = run_both(dev, w)
    assert rc == 0
    assert_chain_same(w, g, rc, outs, masks, "2100 tiles")


def test_hundreds_of_tiles_scanned_at_once(dev):
    # 489 tiles, a ragged last one: the select kernel's last workgroup scans
    # all chunks of 256 tiles in one block scan
    w = small(75, (3000, 4000, 1_000_001), (600, 300, 3000), empty=(0.05, 0.05, 0.0))
    g, rc, outs, masks, _ = run_both(dev, w)
    assert rc == 0
    assert_chain_same(w, g, rc, outs, masks, "489 tiles")


def test_every_free_slot_reclaimed(dev):
    w = small(21, (3000, 5000, 5000), (0, 0, 0))
    free0 = int((w["tables"][0]["held"] == 0).sum())
    w["needs"] = (free0, 0, 0)
    g, rc, outs, masks, _ = run_both(dev, w)
    assert rc == 0
    assert_chain_same(w, g, rc, outs, masks, "all free")


def test_without_index_and_with_partial_index(dev):
    w = small(23, (4000, 6000, 8000), (1200, 600, 100))
    g, rc, outs, masks, _ = run_both(dev, w, index=False)
    assert_chain_same(w, g, rc, outs, masks, "no index")
    w = small(24, (4000, 6000, 8000), (1200, 600, 100), index_frac=0.6)
    g, rc, outs, masks, _ = run_both(dev, w)
    assert_chain_same(w, g, rc, outs, masks, "partial index")


def test_enospc_stops_the_chain(dev):
    w = small(31, (3000, 4000, 4000), (0, 0, 0))
    free0 = int((w["tables"][0]["held"] == 0).sum())
    w["needs"] = (free0 + 1, 10, 0)
    g, rc, outs, masks, d = run_both(dev, w)
    assert rc == ref.ENOSPC
    assert_chain_same(w, g, rc, outs, masks, "enospc")
    gk, gm = g["index"]
    assert np.array_equal(gk, w["index_keys"])
    assert np.array_equal(gm, w["index_masks"].astype(np.uint32))
    # the deeper tiers find no room for the demotions: ENOSPC at DRAM
    w = small(32, (3000, 400, 400), (1000, 0, 0), held=(0.1, 0.9, 0.0))
    g, rc, outs, masks, _ = run_both(dev, w)
    assert rc == ref.ENOSPC and outs[0]["rc"] == 0 and outs[1]["rc"] == ref.ENOSPC
    assert_chain_same(w, g, rc, outs, masks, "enospc dram")


def test_einval_writes_nothing(dev):
    w = small(41, (3000, 3000, 3000), (500, 100, 0))
    w["tables"][1]["last_use_ns"][1234] = -5
    g, rc, outs, masks, _ = run_both(dev, w)
    assert rc == ref.EINVAL and outs[0]["rc"] == 0 and outs[1]["rc"] == ref.EINVAL
    assert_chain_same(w, g, rc, outs, masks, "negative stamp")


def test_incoming_zero_hash_is_einval(dev):
    import torch
    from paper_2608_06557_amd import cascade as cx
    w = small(43, (100, 3000, 100), (0, 10, 0))
    d = dev.DeviceTiers(w["tables"], w["needs"], w["index_keys"], w["index_masks"])
    inc = np.zeros(4, cx.DEMOTION_DTYPE)
    inc["hash"] = [5, 6, 0, 7]
    inc_d = torch.from_numpy(inc.view(np.uint8).copy()).cuda()
    n_inc = torch.tensor([4], dtype=torch.int32, device="cuda")
    out = torch.zeros(14 * cx.DEMOTION_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
    freed = torch.zeros(10, dtype=torch.int32, device="cuda")
    placed = torch.zeros(4, dtype=torch.int32, device="cuda")
    rc = cx.cascade_tier_reclaim(1, d.tabs[1], 10, inc_d.data_ptr(), n_inc.data_ptr(), 4,
                                 out.data_ptr(), d.n_out[1:2].data_ptr(), 14, freed.data_ptr(),
                                 placed.data_ptr(), d.index.data_ptr(), d.capacity,
                                 d.ws.data_ptr(), d.ws_bytes, d.status.data_ptr(),
                                 dev.stream_handle())
    assert rc == 0
    g = d.fetch()
    assert g["status"] == ref.EINVAL
    assert np.array_equal(g["tiers"][1]["block_hash"], w["tables"][1]["block_hash"])
    # n_incoming above max_incoming
    d.status.zero_()
    n_inc.fill_(5)
    rc = cx.cascade_tier_reclaim(1, d.tabs[1], 10, inc_d.data_ptr(), n_inc.data_ptr(), 4,
                                 out.data_ptr(), d.n_out[1:2].data_ptr(), 14, freed.data_ptr(),
                                 placed.data_ptr(), d.index.data_ptr(), d.capacity,
                                 d.ws.data_ptr(), d.ws_bytes, d.status.data_ptr(),
                                 dev.stream_handle())
    assert rc == 0
    assert d.fetch()["status"] == ref.EINVAL


def test_workspace_reused_across_calls(dev):
    # two chains in a row on one workspace, the second over smaller tables:
    # every counter the first left behind must be back at zero
    import torch
    w1 = small(51, (9000, 12000, 15000), (2000, 900, 50))
    d = dev.DeviceTiers(w1["tables"], w1["needs"], w1["index_keys"], w1["index_masks"])
    assert d.run() == 0
    g1 = d.fetch()
    rc, outs, masks = oracle_chain(w1)
    assert_chain_same(w1, g1, rc, outs, masks, "first")
    w2 = small(52, (3000, 2500, 2100), (700, 300, 20))
    d2 = dev.DeviceTiers(w2["tables"], w2["needs"], w2["index_keys"], w2["index_masks"])
    d2.ws = d.ws  # the first chain's workspace, as it left it
    d2.ws_bytes = d.ws_bytes
    assert d2.run() == 0
    g2 = d2.fetch()
    rc, outs, masks = oracle_chain(w2)
    assert_chain_same(w2, g2, rc, outs, masks, "second")
    torch.cuda.synchronize()


def test_chain_workspace_reused_across_calls(dev):
    # the same for one chain call per chain: a workspace sized for the first
    # chain's tables serves a second chain over smaller ones
    w1 = small(53, (9000, 12000, 15000), (2000, 900, 50))
    d = dev.DeviceTiers(w1["tables"], w1["needs"], w1["index_keys"], w1["index_masks"])
    assert d.run_chain() == 0
    g1 = d.fetch()
    rc, outs, masks = oracle_chain(w1)
    assert_chain_same(w1, g1, rc, outs, masks, "first chain call")
    w2 = small(54, (3000, 2500, 2100), (700, 300, 20))
    d2 = dev.DeviceTiers(w2["tables"], w2["needs"], w2["index_keys"], w2["index_masks"])
    d2.chain_args()
    d2.ws_chain = d.ws_chain  # the first call's workspace, as it left it
    d2.ws_chain_bytes = d.ws_chain_bytes
    assert d2.run_chain() == 0
    g2 = d2.fetch()
    rc, outs, masks = oracle_chain(w2)
    assert_chain_same(w2, g2, rc, outs, masks, "second chain call")


@pytest.mark.parametrize("one_call", [False, True], ids=["per_tier", "chain_call"])
def test_workspace_clean_after_a_failed_chain(dev, one_call):
    # a chain that stops at DRAM (ENOSPC) leaves its workspace as a good
    # chain needs it: the histograms its shared passes built for the tiers it
    # never reached are cleared too
    bad = small(55, (3000, 400, 400), (1000, 0, 0), held=(0.1, 0.9, 0.0))
    d = dev.DeviceTiers(bad["tables"], bad["needs"], bad["index_keys"], bad["index_masks"])
    assert (d.run_chain() if one_call else d.run()) == 0
    rc, _, _ = oracle_chain(bad)
    assert rc == ref.ENOSPC and d.fetch()["status"] == ref.ENOSPC
    good = small(56, (2500, 400, 400), (100, 20, 10))
    d2 = dev.DeviceTiers(good["tables"], good["needs"], good["index_keys"], good["index_masks"])
    if one_call:
        d2.chain_args()
        d2.ws_chain, d2.ws_chain_bytes = d.ws_chain, d.ws_chain_bytes
    else:
        d2.ws, d2.ws_bytes = d.ws, d.ws_bytes
    assert (d2.run_chain() if one_call else d2.run()) == 0
    g = d2.fetch()
    rc, outs, masks = oracle_chain(good)
    assert rc == 0
    assert_chain_same(good, g, rc, outs, masks, "after a failed chain")


def test_lookup_after_reclaim_reads_the_new_tiers(dev):
    # the prefix lookup on the updated index: a block whose every copy was
    # reclaimed is a miss; demoted blocks report their deeper tier
    w = small(61, (4000, 5000, 3000), (1500, 800, 0), held=(0.2, 0.05, 0.0))
    g, rc, outs, masks, d = run_both(dev, w)
    assert rc == 0
    assert_chain_same(w, g, rc, outs, masks, "chain")
    keys = w["index_keys"]
    rng = np.random.default_rng(3)
    n = 600
    per = rng.integers(1, 6, n)
    offs = np.concatenate([[0], np.cumsum(per)]).astype(np.int32)
    bh = keys[rng.integers(0, len(keys), int(offs[-1]))]
    n_in = (per * 16 + 1).astype(np.int32)
    facts_h, facts_t = dev.index_facts(keys, masks)
    o = ref.prefix_probe(facts_h, facts_t, offs, bh, n_in, 16)
    pw = {"n_in": n_in, "index_hashes": np.zeros(1, np.uint64),
          "index_tiers": np.zeros(1, np.uint8), "block_offsets": offs, "block_hashes": bh,
          "block_tokens": 16}
    p = dev.DevicePrefix(pw, capacity=d.capacity)
    p.index = d.index  # the reclaimed index, not rebuilt
    assert p.probe() == 0
    r = p.fetch()
    assert r["status"] == 0
    assert np.array_equal(r["n_prefix"], o["n_prefix"])
    assert np.array_equal(r["prefix_tier"], o["prefix_tier"])
    # some blocks became misses: dropped from NVMe with no copy left
    assert (masks == 0).any()
