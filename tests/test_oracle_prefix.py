"""Pins of the oracle's prefix-hit lookup (Section 4.4, prefix hit detection):
an index records the deepest tier holding each cached block; a request's
matched prefix is its longest run of leading blocks present in the index,
capped so that one prompt token is left to compute, in the deepest tier
over that run.  Checked against a hand example, special cases, a round
trip from known cached runs, and order and monotonicity properties."""
import numpy as np
import pytest

from oracle import ref
import paper_2608_06557_amd.synth as synth

HBM, DRAM, NVME, NONE = 0, 1, 2, 3


def probe(entries, reqs, bt=16):
    """entries: [(hash, tier)]; reqs: [(n_in, [hashes])]."""
    ih = np.array([e[0] for e in entries], np.uint64)
    it = np.array([e[1] for e in entries], np.uint8)
    off = np.cumsum([0] + [len(r[1]) for r in reqs]).astype(np.int32)
    bh = np.array([h for r in reqs for h in r[1]], np.uint64)
    ni = np.array([r[0] for r in reqs], np.int32)
    return ref.prefix_probe(ih, it, off, bh, ni, bt)


def test_hand_example():
    # request 0: blocks 11 (HBM), 12 (HBM and DRAM: deepest is DRAM), 13 not
    #   cached -> 2 blocks = 32 tokens, tier DRAM
    # request 1: block 21 (NVMe), 22 not cached -> 16 tokens, NVMe
    # request 2: block 31 not cached, 32 cached -> nothing matches
    # request 3: 40 prompt tokens allow at most 2 full blocks -> 32, HBM
    r = probe([(11, HBM), (12, HBM), (21, NVME), (12, DRAM), (32, DRAM), (41, HBM),
               (42, HBM), (43, HBM)],
              [(64, [11, 12, 13]), (40, [21, 22]), (64, [31, 32]), (40, [41, 42, 43])])
    assert r["rc"] == ref.OK
    assert list(r["n_prefix"]) == [32, 16, 0, 32]
    assert list(r["prefix_tier"]) == [DRAM, NVME, NONE, HBM]


def test_cap_leaves_one_prompt_token():
    for n_in in [1, 15, 16, 17, 32, 33, 48]:
        r = probe([(h, HBM) for h in range(1, 5)], [(n_in, [1, 2, 3, 4])])
        cap = min(4, (n_in - 1) // 16)
        assert r["n_prefix"][0] == 16 * cap
        assert r["prefix_tier"][0] == (HBM if cap > 0 else NONE)


def test_empty_index_and_empty_requests():
    r = probe([], [(100, [5, 6]), (3, [])])
    assert list(r["n_prefix"]) == [0, 0] and list(r["prefix_tier"]) == [NONE, NONE]
    r = probe([(1, DRAM)], [])
    assert r["rc"] == ref.OK and len(r["n_prefix"]) == 0


@pytest.mark.parametrize("cfg", [0, 1])
def test_round_trip_from_cached_runs(cfg):
    """An index built from each request's cached run (plus shallower
    duplicates, blocks past the first gap and unrelated entries) gives back
    exactly those runs and tiers."""
    pw = synth.make_prefix_workload(cfg, noise=2000)
    r = ref.prefix_probe(pw["index_hashes"], pw["index_tiers"], pw["block_offsets"],
                         pw["block_hashes"], pw["n_in"], pw["block_tokens"])
    assert r["rc"] == ref.OK
    exp_blocks = pw["expect_blocks"]
    assert np.array_equal(r["n_prefix"], exp_blocks * pw["block_tokens"])
    assert np.array_equal(r["prefix_tier"], np.where(exp_blocks > 0, pw["expect_tier"], NONE))
    assert (exp_blocks > 0).sum() > len(exp_blocks) // 3      # the pin is not vacuous


def test_index_order_does_not_matter():
    pw = synth.make_prefix_workload(0, shared_frac=0.3, noise=500)
    args = (pw["block_offsets"], pw["block_hashes"], pw["n_in"], pw["block_tokens"])
    a = ref.prefix_probe(pw["index_hashes"], pw["index_tiers"], *args)
    p = np.random.default_rng(1).permutation(len(pw["index_hashes"]))
    b = ref.prefix_probe(pw["index_hashes"][p], pw["index_tiers"][p], *args)
    assert np.array_equal(a["n_prefix"], b["n_prefix"])
    assert np.array_equal(a["prefix_tier"], b["prefix_tier"])


def test_more_entries_never_shorten_a_match():
    rng = np.random.default_rng(3)
    pw = synth.make_prefix_workload(0, noise=100)
    args = (pw["block_offsets"], pw["block_hashes"], pw["n_in"], pw["block_tokens"])
    a = ref.prefix_probe(pw["index_hashes"], pw["index_tiers"], *args)
    extra = rng.choice(pw["block_hashes"], 800, replace=False)
    et = rng.integers(0, 3, 800).astype(np.uint8)
    b = ref.prefix_probe(np.concatenate([pw["index_hashes"], extra]),
                         np.concatenate([pw["index_tiers"], et]), *args)
    assert np.all(b["n_prefix"] >= a["n_prefix"])
    same = b["n_prefix"] == a["n_prefix"]
    matched = a["n_prefix"] > 0
    # a deeper copy of a matched block can only deepen the tier
    assert np.all(b["prefix_tier"][same & matched] >= a["prefix_tier"][same & matched])


def test_shared_families_match_alike():
    """Requests whose leading hashes coincide get the same run, up to each
    one's own cap and block count."""
    pw = synth.make_prefix_workload(1, n=3000, shared_frac=0.4)
    r = ref.prefix_probe(pw["index_hashes"], pw["index_tiers"], pw["block_offsets"],
                         pw["block_hashes"], pw["n_in"], pw["block_tokens"])
    off, bh = pw["block_offsets"], pw["block_hashes"]
    first = {}
    for i in range(len(off) - 1):
        if off[i + 1] > off[i]:
            first.setdefault(int(bh[off[i]]), []).append(i)
    groups = [g for g in first.values() if len(g) > 1]
    assert len(groups) > 50
    for g in groups:
        a, b = g[0], g[1]
        la, lb = off[a + 1] - off[a], off[b + 1] - off[b]
        k = min(la, lb)
        if not np.array_equal(bh[off[a]:off[a] + k], bh[off[b]:off[b] + k]):
            continue
        ca = min(la, (pw["n_in"][a] - 1) // 16)
        cb = min(lb, (pw["n_in"][b] - 1) // 16)
        ma, mb = r["n_prefix"][a] // 16, r["n_prefix"][b] // 16
        # both runs agree on the common, uncapped part
        assert min(ma, cb, k) == min(mb, ca, k)


@pytest.mark.parametrize("case", ["hash0_request", "hash0_index", "tier3", "offsets", "n_in0"])
def test_einval(case):
    entries, reqs = [(7, HBM)], [(64, [7, 8])]
    if case == "hash0_request":
        reqs = [(64, [0, 8])]
    elif case == "hash0_index":
        entries = [(0, HBM)]
    elif case == "tier3":
        entries = [(7, NONE)]
    elif case == "n_in0":
        reqs = [(0, [7])]
    r = probe(entries, reqs)
    if case == "offsets":
        ih = np.array([7], np.uint64)
        r = ref.prefix_probe(ih, np.zeros(1, np.uint8), np.array([0, 2, 1], np.int32),
                             np.array([7, 8], np.uint64), np.array([64, 64], np.int32), 16)
    assert r["rc"] == ref.EINVAL
