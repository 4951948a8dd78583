"""GPU parity of shared-prefix restores within a step (prefix_group input):
the library against the oracle, element by element, bit for bit, on the
one-workgroup path (queues up to 1024) and the multi-launch path (leaders
and followers in different scan tiles, followers inside and outside the
batch), plus the results without groups left unchanged."""
import numpy as np
import pytest
import torch  # noqa: F401  (imported at collection: the first import is slow)

from oracle import ref
from tests import helpers
from tests.test_gpu_parity import assert_same

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    from paper_2608_06557_amd import cascade, device
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    cascade.load()
    return device


LAST_WORKLOAD = {}


def run_both(dev, w):
    LAST_WORKLOAD["w"] = w
    nb = int(w["params"]["num_blocks"])
    d = dev.DeviceStep(w, slot_cap=nb, unpack_cap=nb, pack_cap=nb)
    assert d.run() == 0
    g = d.fetch()
    o = ref.step(w, slot_cap=nb, unpack_cap=nb, pack_cap=nb)
    return g, o


def assert_same_sharing(g, o, label):
    assert_same(g, o, label)
    if o["rc"] == 0:
        assert np.array_equal(g["share_leader"], o["share_leader"]), label


def _groups(rng, n, k, frac=0.8):
    return np.where(rng.random(n) < frac, rng.integers(0, max(1, min(k, n)), n),
                    -1).astype(np.int32)


def test_worked_example(dev):
    w, gold = helpers.golden_workload("worked_example_shared_prefix.json")
    g, o = run_both(dev, w)
    assert_same_sharing(g, o, "shared-prefix example")
    exp = gold["expected_step"]
    for k in ["order", "action", "restore_blocks", "tokens_granted", "share_leader"]:
        assert [int(x) for x in g[k]] == exp[k], k


def test_random_small_queues(dev):
    rng = np.random.default_rng(321)
    shares = 0
    for t in range(200):
        p = helpers.base_params(token_cap=int(rng.integers(1, 600)),
                                max_move_blocks=int(rng.integers(0, 80)),
                                tier2_reserve_q16=int(rng.choice([0, 4096, 65536])),
                                block_tokens=int(rng.choice([1, 4, 16])))
        n = int(rng.integers(1, 1025))
        w = helpers.random_workload(rng, n, params=p)
        w["prefix_group"] = _groups(rng, n, int(rng.integers(1, 40)))
        g, o = run_both(dev, w)
        assert_same_sharing(g, o, f"case {t} n={n}")
        shares += int((o["action"] == ref.ACT_SHARE).sum())
    assert shares > 300


def _multi_launch_case(n, seed, k_groups):
    """A 65536-request-like queue cut to n requests, a few dozen prefix
    groups over all requests, a token cap that admits several hundred and a
    link cap leaders reach: followers inside and outside the batch."""
    import paper_2608_06557_amd.synth as synth
    w = synth.make_workload(2, seed=seed, n=n)
    rng = np.random.default_rng(seed)
    w["prefix_group"] = _groups(rng, n, k_groups, frac=0.6)
    w["params"] = dict(w["params"], token_cap=1 << 18, max_move_blocks=40000)
    return w


@pytest.mark.parametrize("n", [1025, 2049, 4097, 16385, 65536, 65537, 131073])
def test_multi_launch_sizes(dev, n):
    w = _multi_launch_case(n, 9100 + n, 48)
    print(f"shared prefixes n={n}", flush=True)
    g, o = run_both(dev, w)
    assert_same_sharing(g, o, f"n={n}")
    sh = np.flatnonzero(o["action"] == ref.ACT_SHARE)
    assert len(sh) > 20 and np.isin(sh, o["admitted"]).sum() >= 3   # not vacuous


def test_config3_full_size_unlimited_link(dev):
    """Config 3's 512 shared prefixes as groups, with the link cap lifted so
    that leaders restore: thousands of followers across the queue."""
    import paper_2608_06557_amd.synth as synth
    w = synth.make_workload(3, prefix_groups=True)
    w["params"] = dict(w["params"], max_move_blocks=2 ** 31 - 1)
    g, o = run_both(dev, w)
    assert_same_sharing(g, o, "config 3 groups")
    assert (o["action"] == ref.ACT_SHARE).sum() > 5000


def test_config3_full_size_with_groups(dev):
    import paper_2608_06557_amd.synth as synth
    w = synth.make_workload(3, prefix_groups=True)
    g, o = run_both(dev, w)
    assert_same_sharing(g, o, "config 3 groups, link cap 954")


@pytest.mark.parametrize("n", [3000, 9000])
def test_all_equal_keys(dev, n):
    """Every key equal: no radix pass moves data, the records are read in
    queue order; every member wants the same restore."""
    import paper_2608_06557_amd.synth as synth
    w = synth.make_workload(0, n=1)
    for k in ["slo_class", "state", "queue_tier", "prefix_tier", "arrival_ns", "n_in",
              "n_out_pred", "n_prefix", "n_progress"]:
        w[k] = np.repeat(w[k][:1], n)
    w["state"][:] = helpers.QUEUED
    w["n_progress"][:] = 0
    w["prefix_tier"][:] = helpers.KV_DRAM
    w["n_in"][:] = 400
    w["n_prefix"][:] = 320
    w["arrival_ns"][:] = w["params"]["t_now_ns"]
    w["id"] = np.arange(n, dtype=np.uint64) * 3 + 5
    w["row_offsets"] = np.zeros(n + 1, np.int32)
    w["slots"] = np.zeros(0, np.int32)
    w["prefix_group"] = (np.arange(n) % 5).astype(np.int32)
    w["params"] = dict(w["params"], max_move_blocks=200, token_cap=1 << 16)
    g, o = run_both(dev, w)
    assert list(g["order"]) == list(range(n))
    assert_same_sharing(g, o, "ties")
    assert (o["action"] == ref.ACT_SHARE).sum() == n - 5


@pytest.mark.parametrize("n", [700, 20000])
def test_groups_without_members_change_nothing(dev, n):
    """Groups on requests that cannot share (not queued in DRAM/NVMe) give
    the step without groups, on both paths."""
    import paper_2608_06557_amd.synth as synth
    w = synth.make_workload(2, seed=55 + n, n=n)
    g0, _ = run_both(dev, w)
    deep = (w["state"] == helpers.QUEUED) & np.isin(w["prefix_tier"],
                                                    [helpers.KV_DRAM, helpers.KV_NVME])
    w["prefix_group"] = np.where(deep, -1, np.arange(n) % 7).astype(np.int32)
    g1, o1 = run_both(dev, w)
    assert_same_sharing(g1, o1, "groups on non-members")
    for k in ["budget_ns", "action", "order", "tokens_granted", "restore_blocks", "alloc_begin",
              "alloc_count", "admitted", "slot_list"]:
        assert np.array_equal(g0[k], g1[k]), k
    assert np.all(g1["share_leader"] == -1)


@pytest.mark.parametrize("n", [100, 5000])
def test_group_id_out_of_range_is_einval(dev, n):
    import paper_2608_06557_amd.synth as synth
    w = synth.make_workload(2, seed=3, n=n)
    w["prefix_group"] = np.zeros(n, np.int32)
    w["prefix_group"][n // 2] = n
    g, o = run_both(dev, w)
    assert o["rc"] == ref.EINVAL and g["status"] == ref.EINVAL
