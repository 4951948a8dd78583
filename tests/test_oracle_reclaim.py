"""Pins of the oracle's per-tier LRU reclamation (Section 4.4, prefix hit
detection: free blocks are reclaimed least-recently-used within each tier, so
hot prefixes stay in the fast tiers and cold ones spill one tier deeper).

What fixes the oracle here, other than itself:
  - a textbook LRU cache (collections.OrderedDict) driven by random access
    sequences evicts exactly the blocks the oracle reclaims;
  - a hand-derived three-tier example (HBM -> DRAM -> NVMe) with every
    decision worked out below;
  - the exchange property by brute force: every reclaimed slot precedes every
    free slot left behind (empty first, least recent use, lower slot);
  - a full cascade keeps the index equal to the tier sets recomputed from
    the slot tables, keeps every block somewhere unless NVMe dropped it, and
    lands every demoted block one tier deeper with its last use;
  - pinned slots are never reclaimed; every EINVAL / ENOSPC rule, with
    nothing written on error.
"""
from collections import OrderedDict

import numpy as np
import pytest

from oracle import ref

H = 0x9E3779B97F4A7C15  # spreads small block ids over 64-bit hashes


def hsh(i):
    return (int(i) * H) & 0xFFFFFFFFFFFFFFFF or 1


def demotions(rows):
    a = np.zeros(len(rows), ref.DEMOTION_DTYPE)
    for j, (h, lu, s) in enumerate(rows):
        a[j] = (h, lu, s, 0)
    return a


def test_reclaim_order_is_textbook_lru():
    rng = np.random.default_rng(11)
    for _ in range(60):
        cap = int(rng.integers(4, 48))
        lru, t = OrderedDict(), 0
        for _ in range(int(rng.integers(cap, 6 * cap))):
            b = int(rng.integers(1, 3 * cap))
            t += int(rng.integers(1, 4))
            if b in lru:
                lru.move_to_end(b)
            elif len(lru) == cap:
                lru.popitem(last=False)
            lru[b] = t
        blocks = list(lru.items())
        n = len(blocks)
        perm = rng.permutation(n)
        bh = np.zeros(n, np.uint64)
        lu = np.zeros(n, np.int64)
        for (b, tb), s in zip(blocks, perm):
            bh[s], lu[s] = hsh(b), tb
        need = int(rng.integers(0, n + 1))
        r = ref.tier_reclaim(0, bh, lu, np.zeros(n, np.uint8), need)
        assert r["rc"] == ref.OK
        # the textbook cache evicts from its least-recently-used end
        evict = set()
        for _ in range(need):
            evict.add(hsh(lru.popitem(last=False)[0]))
        assert {int(h) for h in bh[r["freed"]]} == evict
        assert np.all(np.diff(r["freed"]) > 0)
        # no index: every reclaimed block is demoted, in slot order
        assert list(r["outgoing"]["src_slot"]) == list(r["freed"])
        assert {int(h) for h in r["outgoing"]["hash"]} == evict


def test_equal_last_use_reclaims_the_lower_slots():
    n = 12
    bh = np.array([hsh(i + 1) for i in range(n)], np.uint64)
    lu = np.full(n, 77, np.int64)
    held = np.zeros(n, np.uint8)
    held[[2, 5]] = 1
    r = ref.tier_reclaim(1, bh, lu, held, 4)
    assert list(r["freed"]) == [0, 1, 3, 4]


def test_empty_slots_go_first_whatever_their_stamp():
    bh = np.array([hsh(1), 0, hsh(2), 0, hsh(3)], np.uint64)
    lu = np.array([1, 999, 2, 500, 3], np.int64)
    r = ref.tier_reclaim(0, bh, lu, np.zeros(5, np.uint8), 2)
    assert list(r["freed"]) == [1, 3]
    assert r["n_outgoing"] == 0
    r = ref.tier_reclaim(0, bh, lu, np.zeros(5, np.uint8), 3)
    assert list(r["freed"]) == [0, 1, 3]
    assert list(r["outgoing"]["src_slot"]) == [0]


def test_hand_example_three_tiers():
    A, B, C, D, E, F, G, I, Hh = (hsh(i) for i in range(1, 10))
    keys = np.array(sorted([A, B, C, D, E, F, G]), np.uint64)
    mask0 = {A: 1, B: 3, C: 1, D: 5, E: 1, F: 2, G: 4}
    masks = np.array([mask0[int(k)] for k in keys], np.uint8)

    # HBM: s1 empty; s2 (B) and s4 (D) share last use 10, slot order breaks
    # the tie; s3 is pinned; s0 (A, 50) is the most recent and survives
    bh0 = np.array([A, 0, B, C, D, E], np.uint64)
    lu0 = np.array([50, 0, 10, 5, 10, 40], np.int64)
    held0 = np.array([0, 0, 0, 1, 0, 0], np.uint8)
    r0 = ref.tier_reclaim(0, bh0, lu0, held0, 4, index_keys=keys, index_masks=masks)
    assert r0["rc"] == ref.OK
    assert list(r0["freed"]) == [1, 2, 4, 5]
    # B has a DRAM copy and D an NVMe copy: only E (HBM only) is demoted
    assert [(int(o["hash"]), int(o["last_use_ns"]), int(o["src_slot"]))
            for o in r0["outgoing"]] == [(E, 40, 5)]
    m = dict(zip(map(int, keys), map(int, r0["index_masks"])))
    assert m == {A: 1, B: 2, C: 1, D: 4, E: 2, F: 2, G: 4}
    assert list(r0["block_hash"]) == [A, 0, 0, C, 0, 0]
    assert list(r0["last_use_ns"]) == [50, 0, 0, 5, 0, 0]

    # DRAM: one slot for the caller plus E; t3 empty goes first, then F (3)
    bh1 = np.array([B, F, Hh, 0], np.uint64)
    lu1 = np.array([8, 3, 1, 0], np.int64)
    held1 = np.array([0, 0, 1, 0], np.uint8)
    r1 = ref.tier_reclaim(1, bh1, lu1, held1, 1, incoming=r0["outgoing"],
                          index_keys=keys, index_masks=r0["index_masks"])
    assert r1["rc"] == ref.OK
    assert list(r1["freed"]) == [1] and list(r1["placed"]) == [3]
    assert [(int(o["hash"]), int(o["last_use_ns"]), int(o["src_slot"]))
            for o in r1["outgoing"]] == [(F, 3, 1)]
    assert list(r1["block_hash"]) == [B, 0, Hh, E]
    assert list(r1["last_use_ns"]) == [8, 0, 1, 40]
    m = dict(zip(map(int, keys), map(int, r1["index_masks"])))
    assert m == {A: 1, B: 2, C: 1, D: 4, E: 2, F: 4, G: 4}

    # NVMe: F takes the least recent slot, I (stamp 0, not indexed) is dropped
    bh2 = np.array([D, G, I], np.uint64)
    lu2 = np.array([2, 7, 0], np.int64)
    r2 = ref.tier_reclaim(2, bh2, lu2, np.zeros(3, np.uint8), 0, incoming=r1["outgoing"],
                          max_outgoing=0, index_keys=keys, index_masks=r1["index_masks"])
    assert r2["rc"] == ref.OK
    assert list(r2["placed"]) == [2] and r2["n_outgoing"] == 0
    assert list(r2["block_hash"]) == [D, G, F]
    assert list(r2["last_use_ns"]) == [2, 7, 3]
    assert np.array_equal(r2["index_masks"], r1["index_masks"])
    # the probe reads the deepest tier: A 0, B 1, C 0, D 2, E 1, F 2, G 2
    deep = {int(k): int(mv).bit_length() - 1 for k, mv in zip(keys, r2["index_masks"])}
    assert deep == {A: 0, B: 1, C: 0, D: 2, E: 1, F: 2, G: 2}


def _lru_key(bh, lu, s):
    return (1, int(lu[s]), s) if bh[s] else (0, 0, s)


def test_exchange_property_brute_force():
    rng = np.random.default_rng(5)
    for _ in range(300):
        n = int(rng.integers(1, 40))
        bh = np.where(rng.random(n) < 0.3, 0,
                      rng.integers(1, 2**63, n, dtype=np.int64)).astype(np.uint64)
        lu = rng.integers(0, 6, n).astype(np.int64)  # many ties
        held = (rng.random(n) < 0.25).astype(np.uint8)
        free = [s for s in range(n) if not held[s]]
        total = int(rng.integers(0, len(free) + 1))
        n_inc = int(rng.integers(0, total + 1))
        need = total - n_inc
        inc = demotions([(hsh(1000 + j), int(rng.integers(0, 9)), j) for j in range(n_inc)])
        tier = int(rng.integers(0, 3))
        r = ref.tier_reclaim(tier, bh, lu, held, need, incoming=inc)
        assert r["rc"] == ref.OK
        rec = list(r["freed"]) + list(r["placed"])
        assert len(rec) == total and len(set(rec)) == total
        assert all(not held[s] for s in rec)
        assert rec == sorted(rec)
        kept = [s for s in free if s not in set(rec)]
        for a in rec:
            for b in kept:
                assert _lru_key(bh, lu, a) < _lru_key(bh, lu, b)
        # demoted: the reclaimed cached blocks above NVMe (no index given)
        want = [s for s in rec if bh[s] and tier < 2]
        assert list(r["outgoing"]["src_slot"]) == want
        assert list(r["outgoing"]["hash"]) == [bh[s] for s in want]
        assert list(r["outgoing"]["last_use_ns"]) == [lu[s] for s in want]
        # the table: caller's slots empty, incoming blocks placed in order
        for s in r["freed"]:
            assert r["block_hash"][s] == 0 and r["last_use_ns"][s] == 0
        for j, s in enumerate(r["placed"]):
            assert r["block_hash"][s] == inc[j]["hash"]
            assert r["last_use_ns"][s] == inc[j]["last_use_ns"]
        untouched = [s for s in range(n) if s not in set(rec)]
        assert np.array_equal(r["block_hash"][untouched], bh[untouched])
        assert np.array_equal(r["last_use_ns"][untouched], lu[untouched])


def make_tiers(rng, sizes, universe, held_frac=0.1, empty_frac=0.15):
    """Random slot tables, one hash at most once per tier, plus the index
    recomputed from them (bit k = tier k holds the block)."""
    tabs = []
    for n in sizes:
        pool = rng.permutation(universe)[:n]
        bh = np.array([hsh(b) for b in pool], np.uint64)
        bh[rng.random(n) < empty_frac] = 0
        lu = rng.integers(0, 4 * n, n).astype(np.int64)
        held = (rng.random(n) < held_frac).astype(np.uint8)
        tabs.append([bh, lu, held])
    return tabs


def index_from(tabs, keys):
    m = {int(k): 0 for k in keys}
    for t, (bh, _, _) in enumerate(tabs):
        for h in bh:
            if int(h) in m:
                m[int(h)] |= 1 << t
    return np.array([m[int(k)] for k in keys], np.uint8)


def run_cascade(tabs, needs, keys, masks):
    outs, inc = [], None
    for t in range(3):
        bh, lu, held = tabs[t]
        r = ref.tier_reclaim(t, bh, lu, held, needs[t], incoming=inc,
                             max_outgoing=0 if t == 2 else None,
                             index_keys=keys, index_masks=masks)
        assert r["rc"] == ref.OK, (t, r["rc"])
        outs.append(r)
        masks, inc = r["index_masks"], r["outgoing"]
        tabs[t] = [r["block_hash"], r["last_use_ns"], held]
    return outs, masks


@pytest.mark.parametrize("seed", range(8))
def test_cascade_keeps_index_and_blocks_consistent(seed):
    rng = np.random.default_rng(100 + seed)
    sizes = [int(rng.integers(20, 80)), int(rng.integers(60, 160)), int(rng.integers(150, 300))]
    universe = np.arange(1, 600)
    tabs = make_tiers(rng, sizes, universe)
    # the index knows every cached block, plus blocks cached nowhere (mask 0)
    keys = np.array(sorted({hsh(b) for b in universe if rng.random() < 0.8}
                           | {int(h) for t in tabs for h in t[0] if h}), np.uint64)
    masks = index_from(tabs, keys)
    old = [[a.copy() for a in t] for t in tabs]
    before = [set(int(h) for h in t[0] if h) for t in tabs]
    free = [int((t[2] == 0).sum()) for t in tabs]
    n0 = int(rng.integers(0, free[0] + 1))
    # size the deeper needs so that every tier can take its demotions
    n1 = int(rng.integers(0, max(free[1] - n0, 0) + 1))
    n2 = int(rng.integers(0, max(free[2] - n0 - n1, 0) + 1))
    outs, masks = run_cascade(tabs, [n0, n1, n2], keys, masks)
    after = [set(int(h) for h in t[0] if h) for t in tabs]
    # the index still says exactly which tiers hold each block
    assert np.array_equal(masks, index_from(tabs, keys))
    # at most one copy of a block per tier
    for t in tabs:
        nz = [int(h) for h in t[0] if h]
        assert len(nz) == len(set(nz))
    # a block held nowhere afterwards was in NVMe, the only tier that drops
    anywhere_after = after[0] | after[1] | after[2]
    for h in before[0] | before[1] | before[2]:
        if h not in anywhere_after:
            assert h in before[2], "a block vanished without passing through NVMe"
    # demoted blocks land one tier deeper with their last use
    for t in range(2):
        for o in outs[t]["outgoing"]:
            bh_next, lu_next, _ = tabs[t + 1]
            s = np.nonzero(bh_next == o["hash"])[0]
            assert len(s) == 1 and lu_next[s[0]] == o["last_use_ns"]
    # hot blocks stay: in every tier, no cached block left unpinned is less
    # recently used than a cached block the tier reclaimed
    for t in range(3):
        bh, lu, held = old[t]
        rec = set(int(s) for s in outs[t]["freed"]) | set(int(s) for s in outs[t]["placed"])
        gone = [int(lu[s]) for s in rec if bh[s]]
        stay = [int(lu[s]) for s in range(len(bh)) if bh[s] and not held[s] and s not in rec]
        if gone and stay:
            assert max(gone) <= min(stay)
        # and empty slots went before any cached one
        if gone:
            assert all(s in rec for s in range(len(bh)) if not bh[s] and not held[s])


def test_pinned_slots_never_reclaimed_and_enospc():
    bh = np.array([hsh(1), hsh(2), 0, hsh(3)], np.uint64)
    lu = np.array([1, 2, 0, 3], np.int64)
    held = np.array([1, 0, 1, 0], np.uint8)
    r = ref.tier_reclaim(0, bh, lu, held, 2)
    assert r["rc"] == ref.OK and list(r["freed"]) == [1, 3]
    r = ref.tier_reclaim(0, bh, lu, held, 3)
    assert r["rc"] == ref.ENOSPC
    assert np.array_equal(r["block_hash"], bh) and np.array_equal(r["last_use_ns"], lu)
    inc = demotions([(hsh(9), 5, 0)])
    r = ref.tier_reclaim(1, bh, lu, held, 2, incoming=inc)
    assert r["rc"] == ref.ENOSPC


def test_zero_work_is_a_no_op():
    bh = np.array([hsh(1), 0], np.uint64)
    lu = np.array([4, 0], np.int64)
    r = ref.tier_reclaim(0, bh, lu, np.zeros(2, np.uint8), 0)
    assert r["rc"] == ref.OK and r["n_outgoing"] == 0
    assert np.array_equal(r["block_hash"], bh)
    r = ref.tier_reclaim(2, np.zeros(0, np.uint64), np.zeros(0, np.int64),
                         np.zeros(0, np.uint8), 0, max_outgoing=0)
    assert r["rc"] == ref.OK


def test_einval_rules_write_nothing():
    bh = np.array([hsh(1), hsh(2), 0], np.uint64)
    lu = np.array([1, 2, 0], np.int64)
    held = np.zeros(3, np.uint8)
    keys = np.array(sorted([hsh(1), hsh(2)]), np.uint64)
    masks = np.array([1, 1], np.uint8)
    cases = [
        dict(tier=3),
        dict(tier=-1),
        dict(need=-1),
        dict(lu=np.array([1, -2, 0], np.int64)),
        dict(incoming=demotions([(0, 1, 0)])),
        dict(keys=keys[::-1].copy()),
        dict(keys=np.array([0, keys[1]], np.uint64)),
        dict(masks=np.array([8, 1], np.uint8)),
        dict(max_outgoing=1),  # need 2 on tier 0 needs room for 2 demotions
    ]
    for c in cases:
        r = ref.tier_reclaim(c.get("tier", 0), bh, c.get("lu", lu), held, c.get("need", 2),
                             incoming=c.get("incoming"), max_outgoing=c.get("max_outgoing"),
                             index_keys=c.get("keys", keys), index_masks=c.get("masks", masks))
        assert r["rc"] == ref.EINVAL, c
        assert np.array_equal(r["block_hash"], bh)
        assert np.array_equal(r["index_masks"], c.get("masks", masks))
    # NVMe demotes nothing, so it needs no outgoing room
    r = ref.tier_reclaim(2, bh, lu, held, 2, max_outgoing=0, index_keys=keys, index_masks=masks)
    assert r["rc"] == ref.OK
