"""GPU parity: the gfx950 library against the CPU oracle, element by element.

Everything in the step is integer, so the bar is bit-exact equality of every
output array and count (tolerance 0).  Inputs come from the seeded generator
(all five workloads at full size, in the launch configuration the benchmark
times) and from random small queues that reach every branch."""
import numpy as np
import pytest
import torch  # noqa: F401  (imported at collection: the first import is slow)

from oracle import ref
from tests import helpers

pytestmark = pytest.mark.gpu

ARRAYS = ["budget_ns", "action", "queue_tier_out", "tokens_granted", "restore_blocks", "order",
          "alloc_begin", "alloc_count"]


@pytest.fixture(scope="module")
def dev():
    import torch
    from paper_2608_06557_amd import cascade, device
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    cascade.load()   # fails loudly when the library is missing
    return device


# the workload of the running test, saved to .npz if the test fails (see
# conftest.py; replay with `python -m tests.replay_step FILE`)
LAST_WORKLOAD = {}


def run_both(dev, w, caps=(None, None, None)):
    LAST_WORKLOAD["w"] = w
    d = dev.DeviceStep(w, slot_cap=caps[0], unpack_cap=caps[1], pack_cap=caps[2])
    rc = d.run()
    assert rc == 0, rc
    g = d.fetch()
    o = ref.step(w, slot_cap=d.caps[0], unpack_cap=d.caps[1], pack_cap=d.caps[2])
    return g, o


def assert_same(g, o, label=""):
    assert g["status"] == o["rc"], (label, g["status"], o["rc"])
    if o["rc"] not in (0, -2):
        return
    for k in ["n_admitted", "n_slot_list", "n_unpack", "n_pack"]:
        assert g[k] == o[k], (label, k, g[k], o[k])
    if o["rc"] != 0:
        return
    for k in ARRAYS:
        if not np.array_equal(g[k], o[k]):
            bad = np.flatnonzero(g[k] != o[k])
            raise AssertionError(f"{label} {k}: {len(bad)} differ, first at {bad[:5]}: "
                                 f"gpu {g[k][bad[:5]]} oracle {o[k][bad[:5]]}")
    assert np.array_equal(g["admitted"], o["admitted"]), label
    assert np.array_equal(g["slot_list"], o["slot_list"]), label
    for k in ["unpack_moves", "pack_moves"]:
        assert np.array_equal(g[k].view(np.int32), o[k].view(np.int32)), (label, k)
    for k in ["unpack_hazard", "pack_hazard"]:
        assert np.array_equal(g[k], o[k]), (label, k)


@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_configs_full_size(dev, cfg):
    import paper_2608_06557_amd.synth as synth
    w = synth.make_workload(cfg)
    print(f"config {cfg} n={len(w['id'])}", flush=True)
    g, o = run_both(dev, w)
    assert_same(g, o, f"config {cfg}")


@pytest.mark.parametrize("n", [1, 2, 63, 64, 65, 255, 256, 257, 511, 512, 513, 1023, 1024, 1025,
                               2047, 2048,
                               2049, 4095, 4096, 4097, 8193, 12289, 16385, 65535, 65537, 69633,
                               131073])
def test_fuzz_sizes(dev, n):
    import paper_2608_06557_amd.synth as synth
    w = synth.make_workload(2, seed=7000 + n, n=n)
    g, o = run_both(dev, w)
    assert_same(g, o, f"n={n}")


def test_random_small_queues(dev):
    rng = np.random.default_rng(123)
    for t in range(200):
        p = helpers.base_params(token_cap=int(rng.integers(1, 300)),
                                max_move_blocks=int(rng.integers(0, 60)),
                                tier2_reserve_q16=int(rng.choice([0, 4096, 65536])),
                                block_tokens=int(rng.choice([1, 4, 16])))
        w = helpers.random_workload(rng, int(rng.integers(1, 300)), params=p)
        g, o = run_both(dev, w)
        assert_same(g, o, f"case {t}")


@pytest.mark.parametrize("n", [3000, 9000])
def test_all_equal_keys_large(dev, n):
    """Every key equal: no radix pass moves data, so the order is the queue
    order (queues of two and of five sort tiles)."""
    import paper_2608_06557_amd.synth as synth
    w = synth.make_workload(0, n=1)
    for k in ["slo_class", "state", "queue_tier", "prefix_tier", "arrival_ns", "n_in",
              "n_out_pred", "n_prefix", "n_progress"]:
        w[k] = np.repeat(w[k][:1], n)
    w["state"][:] = helpers.QUEUED
    w["n_progress"][:] = 0
    w["id"] = np.arange(n, dtype=np.uint64) * 3 + 5
    w["row_offsets"] = np.zeros(n + 1, np.int32)
    w["slots"] = np.zeros(0, np.int32)
    g, o = run_both(dev, w)
    assert list(g["order"]) == list(range(n))
    assert_same(g, o, "ties")


def test_config3_ties_are_stable(dev):
    import paper_2608_06557_amd.synth as synth
    w = synth.make_workload(3)
    g, o = run_both(dev, w)
    b = g["budget_ns"][g["order"]]
    ties = np.flatnonzero(np.diff(b) == 0)
    assert len(ties) > 1000
    assert_same(g, o, "config 3")


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_many_victims_every_restore_in_a_spilled_slot(dev, seed):
    """No free slots, zero elapsed time: hundreds of running prefills are
    preempted (more than the finishing workgroup stages in LDS) and every
    restore lands in a spilled slot, so every unpack move has a hazard."""
    rng = np.random.default_rng(seed)
    p = helpers.base_params(token_cap=20000, max_move_blocks=5000, tier2_reserve_q16=0)
    w = helpers.random_workload(rng, 3000, params=p, n_free=0)
    w["arrival_ns"] = np.full(3000, p["t_now_ns"], np.int64)
    g, o = run_both(dev, w)
    assert_same(g, o, f"victims seed {seed}")
    victims = np.isin(o["action"], [ref.ACT_PREEMPT_OFFLOAD, ref.ACT_PREEMPT_DROP]).sum()
    assert victims > 256 and o["n_unpack"] > 300
    assert np.all(o["unpack_hazard"] >= 0)


@pytest.mark.parametrize("seed", [0, 1])
def test_finish_more_victims_than_staged(dev, seed):
    """Thousands of preempted running prefills: more victims than the parallel
    finish stages, so one workgroup finishes the step sequentially."""
    rng = np.random.default_rng(seed)
    n = 12000
    p = helpers.base_params(token_cap=200000, max_move_blocks=60000, tier2_reserve_q16=0,
                            num_blocks=100000)
    w = helpers.random_workload(rng, n, params=p, n_free=0)
    w["arrival_ns"] = np.full(n, p["t_now_ns"], np.int64)
    g, o = run_both(dev, w)
    assert_same(g, o, f"victims {seed}")
    victims = np.isin(o["action"], [ref.ACT_PREEMPT_OFFLOAD, ref.ACT_PREEMPT_DROP]).sum()
    assert victims > 1024


@pytest.mark.parametrize("seed", [0, 1])
def test_finish_long_restore_list(dev, seed):
    """More restoring requests than the restore list's LDS copy holds."""
    rng = np.random.default_rng(seed)
    n = 12000
    p = helpers.base_params(token_cap=1_000_000, max_move_blocks=200000, tier2_reserve_q16=0,
                            num_blocks=400000, slo_ns=[10 ** 9] * 3 + [0] * 13,
                            link_blk_ns=[1, 1], link_delta_ns=[1, 1])
    w = helpers.random_workload(rng, n, params=p, n_free=300000)
    w["arrival_ns"] = np.full(n, p["t_now_ns"], np.int64)
    g, o = run_both(dev, w)
    assert_same(g, o, f"restores {seed}")
    assert (o["restore_blocks"][o["admitted"]] > 0).sum() > 1024


def _key_width(w, o):
    """Bits of the sort key over (group, budget) that the step orders by."""
    b = np.clip(o["budget_ns"].astype(np.int64), -(1 << 61), (1 << 61) - 1)
    st = np.asarray(w["state"])
    grp = np.where(st == ref.DECODE, 0,
                   np.where(o["queue_tier_out"] == 1, 1, 2)).astype(np.int64)
    span = int(b.max()) - int(b.min()) + 1
    return int((grp * span + (b - b.min())).max()).bit_length()


@pytest.mark.parametrize("seed", [0, 1])
def test_wide_keys_nine_bit_digits(dev, seed):
    """Requests that arrived long ago widen the key beyond what 8-bit digits
    cover in the passes the parameters allow for, so the sort runs on 9-bit
    digits."""
    import paper_2608_06557_amd.synth as synth
    rng = np.random.default_rng(seed)
    n = 20000
    w = synth.make_workload(2, seed=11 + seed, n=n)
    idx = rng.choice(n, 300, replace=False)
    w["arrival_ns"] = w["arrival_ns"].copy()
    w["arrival_ns"][idx] = rng.integers(0, 1000, 300)
    g, o = run_both(dev, w)
    assert_same(g, o, f"wide keys {seed}")
    assert _key_width(w, o) > 40


@pytest.mark.parametrize("n", [37, 300, 512, 700, 3000, 8192])
def test_small_queue_keys_over_54_bits(dev, n):
    """Requests that arrived at time zero under a clock near 2^61 ns clamp their
    budgets far below the others: keys wider than 54 bits leave no room for
    the request index below them, so short queues sort by digits instead of
    counting ranks; longer queues take seven radix passes of 9-bit digits."""
    rng = np.random.default_rng(n)
    p = helpers.base_params(t_now_ns=(1 << 61) + 12345)
    w = helpers.random_workload(rng, n, params=p)
    old = rng.random(n) < 0.3
    w["arrival_ns"] = np.where(old, 0, w["arrival_ns"]).astype(np.int64)
    g, o = run_both(dev, w)
    assert_same(g, o, f"wide small {n}")
    assert _key_width(w, o) > 54


def test_empty_queue(dev):
    w = helpers.random_workload(np.random.default_rng(0), 1)
    for k in [f for f, _ in ref.REQ_FIELDS]:
        w[k] = w[k][:0]
    w["row_offsets"] = np.zeros(1, np.int32)
    w["slots"] = np.zeros(0, np.int32)
    g, o = run_both(dev, w)
    assert_same(g, o, "empty")
    assert g["n_slot_list"] == len(w["free_slots"])


def test_worked_example(dev):
    w, gold = helpers.worked_example()
    g, o = run_both(dev, w)
    assert_same(g, o, "worked example")
    assert list(g["order"]) == gold["expected_step"]["order"]


def test_second_worked_example(dev):
    """PREFETCH, HBM-prefix RETAIN inside and outside the batch, three
    victims spilled and dropped from the back of the order."""
    w, gold = helpers.golden_workload("worked_example_2.json")
    g, o = run_both(dev, w)
    assert_same(g, o, "second worked example")
    exp = gold["expected_step"]
    for k in ["order", "action", "restore_blocks", "tokens_granted"]:
        assert [int(x) for x in g[k]] == exp[k], k
    assert [list(map(int, m)) for m in g["pack_moves"].view(np.int32).reshape(-1, 4)] \
        == exp["pack_moves"]


def test_scarce_resources(dev):
    rng = np.random.default_rng(99)
    for t in range(150):
        p = helpers.base_params(token_cap=int(rng.integers(1, 40)),
                                max_move_blocks=int(rng.integers(0, 12)),
                                tier2_reserve_q16=int(rng.choice([0, 4096, 65536])))
        w = helpers.random_workload(rng, int(rng.integers(1, 40)), params=p,
                                    n_free=int(rng.integers(0, 6)))
        g, o = run_both(dev, w)
        assert_same(g, o, f"scarce {t}")


from tests.test_oracle_invariants import MUTATIONS  # noqa: E402


@pytest.mark.parametrize("name,mutate", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_einval_matches(dev, name, mutate):
    w, _ = helpers.worked_example()
    mutate(w)
    assert ref.step(w)["rc"] == ref.EINVAL
    d = dev.DeviceStep(w)
    rc = d.run()
    status = rc if rc != 0 else d.fetch()["status"]
    assert status == ref.EINVAL, name


@pytest.mark.parametrize("n", [6000, 20000])
@pytest.mark.parametrize("field", ["state", "slot", "row"])
def test_einval_on_the_multi_launch_path(dev, field, n):
    """Bad request data in a queue of 6000 or 20000 requests: the radix
    passes and the scan tiles stop at the failed status without waiting on
    each other (a wait would run to its poll limit and report a timeout
    instead)."""
    import time
    import torch
    import paper_2608_06557_amd.synth as synth
    w = synth.make_workload(2, seed=5, n=n)
    if field == "state":
        w["state"] = w["state"].copy()
        w["state"][n // 2 + 345] = 7
    elif field == "slot":
        w["slots"] = w["slots"].copy()
        w["slots"][len(w["slots"]) // 2] = w["params"]["num_blocks"]
    else:
        w["row_offsets"] = w["row_offsets"].copy()
        w["row_offsets"][n // 2:] += 1
    assert ref.step(w)["rc"] == ref.EINVAL
    d = dev.DeviceStep(w)
    assert d.run() == 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    assert d.run() == 0
    status = d.fetch()["status"]
    elapsed = time.perf_counter() - t0
    assert status == ref.EINVAL, (field, status)
    assert elapsed < 0.05, elapsed


@pytest.mark.parametrize("which", ["slot", "free_slot", "none"])
def test_small_queue_large_pool_list_checks(dev, which):
    """A queue of at most 1024 requests runs as one workgroup; over a pool
    larger than it checks itself, a separate grid checks the free list and
    the block table.  Out-of-range entries must still give EINVAL."""
    w, _ = helpers.worked_example()
    w["params"] = dict(w["params"], num_blocks=100_000)
    if which == "slot":
        assert len(w["slots"]) > 0
        w["slots"] = w["slots"].copy()
        w["slots"][-1] = 100_000
    elif which == "free_slot":
        w["free_slots"] = w["free_slots"].copy()
        w["free_slots"][0] = 100_000
    o = ref.step(w)
    assert o["rc"] == (ref.OK if which == "none" else ref.EINVAL)
    g, o = run_both(dev, w)
    assert_same(g, o, which)


def test_enospc_matches(dev):
    w, _ = helpers.worked_example()
    for caps in [(71, 100, 100), (100, 19, 100), (100, 100, 31), (0, 0, 0), (72, 20, 32)]:
        g, o = run_both(dev, w, caps)
        assert_same(g, o, f"caps {caps}")


def test_workspace_too_small(dev):
    from paper_2608_06557_amd import cascade
    w, _ = helpers.worked_example()
    d = dev.DeviceStep(w)
    rc = cascade.cascade_step(d.c_req, d.c_table, d.c_tier, d.params, d.c_out, d.ws_ptr,
                              d.ws_bytes - 1, dev.stream_handle())
    assert rc == cascade.ENOSPC


def test_repeatable(dev):
    import paper_2608_06557_amd.synth as synth
    w = synth.make_workload(2, seed=31)
    d = dev.DeviceStep(w)
    outs = []
    for _ in range(3):
        assert d.run() == 0
        outs.append(d.fetch())
    for k in ARRAYS + ["admitted", "slot_list"]:
        assert np.array_equal(outs[0][k], outs[1][k]) and np.array_equal(outs[0][k], outs[2][k])


# ------------------------------------------------------ domain corners

CORNERS = {
    # every cost at its bound: c_iter + B_max * c_dec = 2^36, c_tok = 2^28,
    # c_attn = 2^16, gamma = 16, one-token blocks, links at 2^40 / 2^32 per
    # block, targets of 2^50 ns, a clock just under 2^62, the largest caps
    "max": dict(c_iter_ps=(1 << 36) - 4096 * (1 << 23), c_decode_ps=1 << 23, max_batch=4096,
                load_decodes=4095, c_token_ps=1 << 28, c_attn_ps=1 << 16, gamma_q16=1 << 20,
                block_tokens=1, chunk_tokens=16, link_delta_ns=[1 << 40, 1 << 40],
                link_blk_ns=[1 << 32, 1 << 32], slo_ns=[1 << 50] * 16, num_classes=16,
                t_now_ns=(1 << 62) - 1, token_cap=1 << 24, tier2_reserve_q16=65536,
                max_move_blocks=2 ** 31 - 1),
    # every cost and cap at its floor, a clock at zero, 65536-token blocks
    "min": dict(c_iter_ps=0, c_decode_ps=0, c_token_ps=0, c_attn_ps=0, gamma_q16=65536,
                max_batch=1, load_decodes=0, block_tokens=1 << 16, chunk_tokens=1 << 20,
                link_delta_ns=[0, 0], link_blk_ns=[1, 1], slo_ns=[0] * 16, num_classes=1,
                t_now_ns=0, token_cap=1, tier2_reserve_q16=0, max_move_blocks=0),
    # the cost bound reached at batch 128 with 16-token blocks, full guardband
    "mid": dict(c_iter_ps=(1 << 36) - 128 * (1 << 28), c_decode_ps=1 << 28, max_batch=128,
                load_decodes=64, c_token_ps=1 << 28, c_attn_ps=1 << 16, gamma_q16=1 << 20,
                block_tokens=16, chunk_tokens=512, slo_ns=[1 << 50, 1 << 40, 1 << 30] + [0] * 13,
                num_classes=3, t_now_ns=(1 << 62) - 1, token_cap=1 << 20,
                tier2_reserve_q16=4096, max_move_blocks=100000),
}


@pytest.mark.parametrize("corner", sorted(CORNERS))
@pytest.mark.parametrize("n,max_in", [(300, 1 << 17), (3000, 1 << 12)])
def test_parameter_domain_corners(dev, corner, n, max_in):
    """Parameters at the edges of the domain (the gamma product needs more
    than 64 bits before its shift at the "max" corner), prompts up to 2^17
    tokens, and a fifth of the queue arriving at time zero (budgets clamped
    in the key); the one-workgroup and the multi-launch path."""
    rng = np.random.default_rng(n + len(corner))
    p = helpers.base_params(**CORNERS[corner])
    w = helpers.random_workload(rng, n, params=p, max_in=max_in)
    old = rng.random(n) < 0.2
    w["arrival_ns"] = np.where(old, 0, w["arrival_ns"]).astype(np.int64)
    print(f"corner {corner} n={n} max_in={max_in} pool={w['params']['num_blocks']}", flush=True)
    g, o = run_both(dev, w)
    assert o["rc"] == ref.OK
    assert_same(g, o, f"corner {corner} n={n}")


def test_largest_queue(dev):
    """2^20 requests, the most a step takes."""
    import paper_2608_06557_amd.synth as synth
    w = synth.make_workload(2, seed=2024, n=1 << 20)
    print(f"n={len(w['id'])}", flush=True)
    g, o = run_both(dev, w)
    assert_same(g, o, "n=2^20")
