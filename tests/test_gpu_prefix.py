"""GPU parity of the prefix-hit index and lookup (Section 4.4, prefix hit
detection) against the oracle, bit-exact: matched prefix length and tier of
every request, from seeded block-hash workloads with shared prefix families,
shallower duplicates, cached blocks past a gap and unrelated entries."""
import numpy as np
import pytest
import torch  # noqa: F401  (imported at collection: the first import is slow)

from oracle import ref

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    from paper_2608_06557_amd import cascade, device
    assert torch.cuda.is_available()
    cascade.load()
    return device


def run_both(dev, pw, capacity=None):
    d = dev.DevicePrefix(pw, capacity=capacity)
    assert d.build() == 0
    assert d.probe() == 0
    g = d.fetch()
    o = ref.prefix_probe(pw["index_hashes"], pw["index_tiers"], pw["block_offsets"],
                         pw["block_hashes"], pw["n_in"], pw["block_tokens"])
    return g, o, d


def assert_same(g, o, label=""):
    assert g["status"] == o["rc"], (label, g["status"], o["rc"])
    if o["rc"] != 0:
        return
    for k in ["n_prefix", "prefix_tier"]:
        if not np.array_equal(g[k], o[k]):
            bad = np.flatnonzero(g[k] != o[k])
            raise AssertionError(f"{label} {k}: {len(bad)} differ, first {bad[:5]}: "
                                 f"gpu {g[k][bad[:5]]} oracle {o[k][bad[:5]]}")


@pytest.mark.parametrize("cfg,shared", [(0, 0.0), (0, 0.3), (1, 0.3), (2, 0.3), (3, 0.5),
                                        (4, 0.2)])
def test_workloads(dev, cfg, shared):
    import paper_2608_06557_amd.synth as synth
    pw = synth.make_prefix_workload(cfg, shared_frac=shared, noise=5000)
    print(f"config {cfg}: {len(pw['n_in'])} requests, {len(pw['block_hashes'])} blocks, "
          f"{len(pw['index_hashes'])} index facts", flush=True)
    g, o, _ = run_both(dev, pw)
    assert_same(g, o, f"config {cfg}")
    assert (o["n_prefix"] > 0).sum() > len(o["n_prefix"]) // 4


def _pw(entries, reqs, bt=16):
    return {"index_hashes": np.array([e[0] for e in entries], np.uint64),
            "index_tiers": np.array([e[1] for e in entries], np.uint8),
            "block_offsets": np.cumsum([0] + [len(r[1]) for r in reqs]).astype(np.int32),
            "block_hashes": np.array([h for r in reqs for h in r[1]], np.uint64),
            "n_in": np.array([r[0] for r in reqs], np.int32), "block_tokens": bt}


def test_hand_example_and_long_runs(dev):
    # request 4 has 300 cached blocks (several 64-block rounds of one wave)
    # and request 5 misses at block 130
    long_run = list(range(1000, 1300))
    miss_130 = list(range(2000, 2200))
    entries = [(11, 0), (12, 0), (21, 2), (12, 1), (32, 1), (41, 0), (42, 0), (43, 0)]
    entries += [(h, h % 3) for h in long_run] + [(h, 1) for h in miss_130 if h != 2130]
    reqs = [(64, [11, 12, 13]), (40, [21, 22]), (64, [31, 32]), (40, [41, 42, 43]),
            (16 * 400, long_run), (16 * 400, miss_130)]
    g, o, _ = run_both(dev, _pw(entries, reqs))
    assert_same(g, o, "hand")
    assert list(g["n_prefix"][:4]) == [32, 16, 0, 32]
    assert g["n_prefix"][4] == 16 * 300 and g["n_prefix"][5] == 16 * 130


def test_duplicates_keep_the_deepest_tier(dev):
    rng = np.random.default_rng(4)
    hashes = np.arange(1, 201, dtype=np.uint64)
    entries = [(int(h), int(t)) for h in hashes for t in rng.integers(0, 3, 7)]
    rng.shuffle(entries)
    reqs = [(16 * 300, [int(h) for h in hashes])] + [(64, [int(h)]) for h in hashes]
    g, o, _ = run_both(dev, _pw(entries, reqs))
    assert_same(g, o, "duplicates")


def test_full_table_reports_enospc(dev):
    entries = [(h, 0) for h in range(1, 101)]      # 100 keys, 64 slots
    g, o, d = run_both(dev, _pw(entries, [(64, [1, 2])]), capacity=64)
    assert g["status"] == -2


@pytest.mark.parametrize("case", ["hash0_request", "hash0_index", "tier3", "n_in0", "offsets"])
def test_einval(dev, case):
    entries, reqs = [(7, 0)], [(64, [7, 8])]
    if case == "hash0_request":
        reqs = [(64, [0, 8])]
    elif case == "hash0_index":
        entries = [(0, 0)]
    elif case == "tier3":
        entries = [(7, 3)]
    elif case == "n_in0":
        reqs = [(0, [7])]
    pw = _pw(entries, reqs)
    if case == "offsets":
        pw = _pw(entries, [(64, [7]), (64, [8])])
        pw["block_offsets"] = np.array([0, 2, 1], np.int32)
    g, o, _ = run_both(dev, pw)
    assert o["rc"] == ref.EINVAL and g["status"] == ref.EINVAL


def test_clear_and_rebuild(dev):
    import paper_2608_06557_amd.synth as synth
    a = synth.make_prefix_workload(0, seed=11)
    b = synth.make_prefix_workload(0, seed=12)
    d = dev.DevicePrefix(a, capacity=1 << 16)
    assert d.build() == 0 and d.probe() == 0
    ga = d.fetch()
    db = dev.DevicePrefix(b, capacity=1 << 16)
    db.index = d.index                      # same index memory, cleared and refilled
    assert db.build() == 0 and db.probe() == 0
    gb = db.fetch()
    for pw, g in [(a, ga), (b, gb)]:
        o = ref.prefix_probe(pw["index_hashes"], pw["index_tiers"], pw["block_offsets"],
                             pw["block_hashes"], pw["n_in"], pw["block_tokens"])
        assert_same(g, o, "rebuild")


def test_empty(dev):
    g, o, _ = run_both(dev, _pw([], [(64, [5])]))
    assert_same(g, o, "empty index")
    g, o, _ = run_both(dev, _pw([(5, 1)], []))
    assert g["status"] == 0


def test_runs_ending_at_window_edges(dev):
    # A wave looks up 64, 128, 256, 256, ... blocks per window, so windows
    # start at blocks 0, 64, 192, 448, 704, 960, ...  Request j owns a
    # sequence whose first miss is at block m_j; the blocks past the miss are
    # cached in the deepest tier, and only the last block before the miss
    # reaches tier 1, so a window that let a block past the miss into the run
    # or its tier would show.
    edges = [0, 1, 2, 63, 64, 65, 127, 191, 192, 193, 447, 448, 449, 703, 704, 705, 959,
             960, 1215, 1216]
    entries, reqs = [], []
    for j, m in enumerate(edges):
        seq = [(j + 1) * 10_000 + b for b in range(1400)]
        entries += [(h, 0) for h in seq[:max(m - 1, 0)]]
        if m >= 1:
            entries.append((seq[m - 1], 1))
        entries += [(h, 2) for h in seq[m + 1:]]
        reqs.append((16 * 1400 + 5, seq))
    # runs capped by the prompt length at a window edge, with every block cached
    for j, lim in enumerate([64, 192, 448, 704]):
        seq = [900_000 + j * 10_000 + b for b in range(lim + 40)]
        entries += [(h, 1) for h in seq]
        reqs.append((16 * lim + 1, seq))
    g, o, _ = run_both(dev, _pw(entries, reqs))
    assert_same(g, o, "window edges")
    assert list(g["n_prefix"][:len(edges)] // 16) == edges
    assert list(g["n_prefix"][len(edges):] // 16) == [64, 192, 448, 704]


@pytest.mark.parametrize("seed", [1, 2])
def test_crowded_table(dev, seed):
    # 3700 keys in 4096 slots: long probe sequences, sequences that wrap past
    # the table's last slot, and keys one past a home slot at the end of a line
    rng = np.random.default_rng(seed)
    keys = np.unique(rng.integers(1, 1 << 40, 4000, dtype=np.uint64))[:3700]
    assert len(keys) == 3700
    tiers = rng.integers(0, 3, len(keys))
    entries = [(int(k), int(t)) for k, t in zip(keys, tiers)]
    absent = rng.integers(1 << 40, 1 << 41, 300, dtype=np.uint64)  # never a key
    reqs = []
    for _ in range(400):
        run = int(rng.integers(0, 600))
        seq = [int(k) for k in rng.choice(keys, run)] + [int(absent[rng.integers(0, 300)])]
        seq += [int(k) for k in rng.choice(keys, int(rng.integers(0, 50)))]
        reqs.append((16 * len(seq) + 1, seq))
    g, o, _ = run_both(dev, _pw(entries, reqs), capacity=4096)
    assert_same(g, o, f"crowded {seed}")


def test_null_status_and_a_single_long_request(dev):
    # status_dev may be NULL: the lookup then reports nothing, also on a zero
    # hash, and still writes every request's result.  One request in a
    # workgroup of four waves, its run of 700 blocks over five windows.
    import paper_2608_06557_amd.cascade as cx
    from paper_2608_06557_amd.device import stream_handle
    seq = [50_000 + b for b in range(900)]
    entries = [(h, 1) for h in seq[:700]]
    for reqs, want in [([(16 * 900 + 1, seq)], 700), ([(16 * 4 + 1, [7, 0, 8, 9])], None)]:
        pw = _pw(entries + [(7, 2)], reqs)
        d = dev.DevicePrefix(pw)
        assert d.build() == 0
        d.n_prefix.fill_(-1)
        assert cx.cascade_prefix_probe(d.index.data_ptr(), d.capacity, d.n, d.off.data_ptr(),
                                       d.bh.data_ptr(), d.n_in.data_ptr(), d.bt,
                                       d.n_prefix.data_ptr(), d.tier.data_ptr(), None,
                                       stream_handle(None)) == 0
        g = d.fetch()
        o = ref.prefix_probe(pw["index_hashes"], pw["index_tiers"], pw["block_offsets"],
                             pw["block_hashes"], pw["n_in"], pw["block_tokens"])
        assert g["status"] == 0  # the status word was left alone
        if want is None:  # invalid input (hash 0): the result is written, its value unspecified
            assert o["rc"] == ref.EINVAL and int(g["n_prefix"][0]) >= 0
        else:
            assert_same(g, o, "null status")
            assert int(g["n_prefix"][0]) == 16 * want
