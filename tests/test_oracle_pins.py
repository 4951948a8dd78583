"""Pins of the CPU oracle against values fixed by the paper's equations and by
plain mathematics (no GPU).

* The hand-derived five-request worked example (tests/golden/worked_example.json).
* Closed forms and special cases of the cost model, eq:est_latency,
  eq:budget_eq, eq:rem_budget_eq, eq:restore_time and eq:max_restorable.
"""
import itertools

import numpy as np
import pytest

from oracle import ref
from tests import helpers

EVAL_KEYS = ["l_actual_ns", "l_max_ns", "l_ns", "budget0_ns", "budget_rem_ns", "tier_out",
             "want_blocks"]


def _eval_req(p, w, i):
    return ref.eval_one(p, int(w["slo_class"][i]), int(w["state"][i]), int(w["queue_tier"][i]),
                        int(w["prefix_tier"][i]), int(w["arrival_ns"][i]), int(w["n_in"][i]),
                        int(w["n_out_pred"][i]), int(w["n_prefix"][i]), int(w["n_progress"][i]))


def test_worked_example_per_request_values():
    w, g = helpers.worked_example()
    exp = g["expected_eval"]
    for i in range(5):
        e = _eval_req(w["params"], w, i)
        for k in EVAL_KEYS:
            assert e[k] == exp[k][i], (i, k, e[k], exp[k][i])


def test_worked_example_step():
    w, g = helpers.worked_example()
    r = ref.step(w)
    exp = g["expected_step"]
    assert r["rc"] == ref.OK
    for k in ["order", "restore_blocks", "tokens_granted", "action", "alloc_begin",
              "alloc_count"]:
        assert list(r[k]) == exp[k], k
    assert list(r["admitted"]) == exp["admitted"]
    assert r["n_slot_list"] == exp["n_slot_list"]
    assert r["n_unpack"] == exp["n_unpack"] and r["n_pack"] == exp["n_pack"]
    # slot list = free list then the victim's row
    assert list(r["slot_list"]) == list(range(40)) + list(range(800, 832))
    um = r["unpack_moves"]
    assert list(um["req"]) == [0] * 20 and list(um["blk"]) == list(range(20))
    assert list(um["pool_slot"]) == list(range(20, 40))
    assert list(um["staging_slot"]) == list(range(20))
    pm = r["pack_moves"]
    assert list(pm["req"]) == [4] * 32 and list(pm["pool_slot"]) == list(range(800, 832))
    assert list(pm["staging_slot"]) == list(range(32)) and list(pm["blk"]) == list(range(32))


def test_second_example_per_request_values():
    w, g = helpers.golden_workload("worked_example_2.json")
    exp = g["expected_eval"]
    for i in range(len(w["id"])):
        e = _eval_req(w["params"], w, i)
        for k in EVAL_KEYS:
            assert e[k] == exp[k][i], (i, k, e[k], exp[k][i])


def _moves(a):
    return [[int(m["req"]), int(m["blk"]), int(m["pool_slot"]), int(m["staging_slot"])]
            for m in a]


def test_second_example_step():
    """PREFETCH of a capped restore outside the batch, RETAIN of HBM-prefix
    requests inside and outside the batch, three victims taken from the back
    of the order (Tier-2 first) with their spill moves in that order."""
    w, g = helpers.golden_workload("worked_example_2.json")
    r = ref.step(w)
    exp = g["expected_step"]
    assert r["rc"] == ref.OK
    for k in ["order", "restore_blocks", "tokens_granted", "action", "alloc_begin",
              "alloc_count", "admitted", "slot_list", "unpack_hazard", "pack_hazard"]:
        assert [int(x) for x in r[k]] == exp[k], (k, list(r[k]), exp[k])
    assert _moves(r["unpack_moves"]) == exp["unpack_moves"]
    assert _moves(r["pack_moves"]) == exp["pack_moves"]
    assert r["n_slot_list"] == len(exp["slot_list"])
    assert r["n_unpack"] == len(exp["unpack_moves"]) and r["n_pack"] == len(exp["pack_moves"])


# ---------------------------------------------------------------- cost model

def _zero_cost(**kw):
    p = helpers.base_params(c_iter_ps=0, c_decode_ps=0, c_token_ps=0, c_attn_ps=0)
    p.update(kw)
    return p


@pytest.mark.parametrize("n,s", [(1, 0), (1, 7), (5, 0), (5, 9), (16, 3), (37, 100), (200, 0)])
def test_attention_pairs_brute_force(n, s):
    # Each of the n new tokens at positions s..s+n-1 attends to every position
    # up to its own: count the pairs one by one.
    p = _zero_cost(c_attn_ps=1)
    pairs = sum(t + 1 for t in range(s, s + n))
    assert ref.compute_ps(p, n, s, 0) == pairs


@pytest.mark.parametrize("chunk", [16, 17, 64, 512])
def test_iteration_count_brute_force(chunk):
    p = _zero_cost(c_iter_ps=1, chunk_tokens=chunk)
    for n in range(0, 3 * chunk + 2, 7):
        iters, done = 0, 0
        while done < n:        # chunked prefill: at most `chunk` tokens per iteration
            done += chunk
            iters += 1
        assert ref.compute_ps(p, n, 0, 0) == iters


def test_decode_share_per_iteration():
    # each co-scheduled decode adds its cost to every iteration
    p = _zero_cost(c_decode_ps=5, chunk_tokens=16)
    assert ref.compute_ps(p, 40, 0, 3) == 3 * 5 * 3
    assert ref.compute_ps(p, 0, 0, 3) == 0


def test_single_iteration_linear_closed_form():
    p = helpers.base_params(c_attn_ps=0, chunk_tokens=64)
    for n in [1, 10, 64]:
        for d in [0, 2, 5]:
            assert ref.compute_ps(p, n, 11, d) == (p["c_iter_ps"] + d * p["c_decode_ps"]
                                                   + n * p["c_token_ps"])


def _queued_none(p, n_in, cls=1, elapsed=0):
    return ref.eval_one(p, cls, ref.QUEUED, ref.QT_NEW, ref.KV_NONE, p["t_now_ns"] - elapsed,
                        n_in, 5, 0, 0)


def test_gamma_one_is_plain_average():
    p = helpers.base_params(gamma_q16=65536)
    for n_in in [1, 17, 50, 120]:
        e = _queued_none(p, n_in)
        assert e["l_ns"] == (e["l_actual_ns"] + e["l_max_ns"]) // 2


def test_full_load_scales_single_estimate():
    # actual load = maximum load: L = gamma * L_actual, floored
    for gq in [65536, 81920, 99999, 1 << 20]:
        p = helpers.base_params(load_decodes=5, max_batch=6, gamma_q16=gq)
        for n_in in [3, 40, 119]:
            e = _queued_none(p, n_in)
            assert e["l_actual_ns"] == e["l_max_ns"]
            assert e["l_ns"] == (e["l_actual_ns"] * gq) // 65536


def test_gamma_product_exact_at_domain_edge():
    # the largest estimates in the domain need more than 64 bits before the
    # shift; the floor must still be exact
    p = helpers.base_params(c_iter_ps=(1 << 36) - 4096 * (1 << 23), c_decode_ps=1 << 23,
                            max_batch=4096, load_decodes=4095, c_token_ps=1 << 28,
                            c_attn_ps=1 << 16, chunk_tokens=16, block_tokens=1,
                            gamma_q16=1 << 20, link_delta_ns=[1 << 40, 1 << 40],
                            link_blk_ns=[1 << 32, 1 << 32])
    n_in, n_pre = 1 << 17, (1 << 17) - 1
    e = ref.eval_one(p, 0, ref.QUEUED, ref.QT_NEW, ref.KV_NVME, p["t_now_ns"], n_in, 0, n_pre, 0)
    s = e["l_actual_ns"] + e["l_max_ns"]
    assert s * (1 << 20) > (1 << 63)
    assert e["l_ns"] == (s * (1 << 20)) >> 17


def test_budget_is_slo_minus_elapsed_without_cost():
    p = _zero_cost()
    for cls in range(3):
        for elapsed in [0, 1, 19_999, 20_000, 123_456]:
            e = _queued_none(p, 30, cls=cls, elapsed=elapsed)
            assert e["l_ns"] == 0
            assert e["budget0_ns"] == p["slo_ns"][cls]
            assert e["budget_rem_ns"] == p["slo_ns"][cls] - elapsed


def test_budget_subtracts_estimate_and_elapsed():
    # a single-iteration queued request with only per-token cost: L_act =
    # L_max = n * c_token (ns), L = 1.25 * that
    p = _zero_cost(c_token_ps=8_000, gamma_q16=81920)
    e = _queued_none(p, 10, cls=2, elapsed=1_000)
    assert e["l_ns"] == 100
    assert e["budget0_ns"] == 200_000 - 100
    assert e["budget_rem_ns"] == 200_000 - 100 - 1_000


def test_decode_without_remaining_tokens_has_no_service_time():
    p = helpers.base_params()
    e = ref.eval_one(p, 0, ref.DECODE, ref.QT_TIER1, ref.KV_NONE, p["t_now_ns"] - 7, 10, 5, 0, 9)
    assert e["l_ns"] == 0 and e["budget_rem_ns"] == 20_000 - 7


@pytest.mark.parametrize("state,qt,positive,expect", [
    (ref.QUEUED, ref.QT_NEW, True, ref.QT_TIER1), (ref.QUEUED, ref.QT_NEW, False, ref.QT_TIER2),
    (ref.QUEUED, ref.QT_TIER1, False, ref.QT_TIER1), (ref.QUEUED, ref.QT_TIER2, True, ref.QT_TIER1),
    (ref.QUEUED, ref.QT_TIER2, False, ref.QT_TIER2),
    (ref.RUNNING_PREFILL, ref.QT_NEW, False, ref.QT_TIER2),
    (ref.DECODE, ref.QT_TIER2, True, ref.QT_TIER2), (ref.DECODE, ref.QT_NEW, True, ref.QT_NEW),
])
def test_tier_transitions(state, qt, positive, expect):
    # zero cost model: B = SLO exactly; SLO 0 gives B = 0, which is not > 0
    p = _zero_cost(slo_ns=[0, 50_000, 200_000] + [0] * 13)
    cls = 1 if positive else 0
    prog = 1 if state == ref.RUNNING_PREFILL else 0
    e = ref.eval_one(p, cls, state, qt, ref.KV_NONE, p["t_now_ns"], 30, 5, 0, prog)
    assert e["tier_out"] == expect
    assert e["group"] == (0 if state == ref.DECODE else (1 if expect == ref.QT_TIER1 else 2))


# ------------------------------------------------- eq:restore_time / eq:max_restorable

def test_restore_time_paths():
    p = helpers.base_params(link_delta_ns=[3, 40], link_blk_ns=[5, 600])
    assert ref.restore_time_ns(p, ref.KV_DRAM, 0) == 0
    assert ref.restore_time_ns(p, ref.KV_NVME, 0) == 0
    # DRAM -> HBM is one link; NVMe -> DRAM -> HBM charges both links
    assert ref.restore_time_ns(p, ref.KV_DRAM, 7) == 3 + 7 * 5
    assert ref.restore_time_ns(p, ref.KV_NVME, 7) == (3 + 40) + 7 * (5 + 600)


def _cheap_restore_params(**kw):
    # recomputing a block (16 tokens at 10 us each) always costs more than
    # moving it, so eq:max_restorable alone decides the restore volume
    p = helpers.base_params(c_token_ps=10_000_000, c_attn_ps=0, block_tokens=16,
                            chunk_tokens=4096, link_delta_ns=[2_000, 3_000],
                            link_blk_ns=[700, 900])
    p.update(kw)
    return p


def test_max_restorable_brute_force():
    rng = np.random.default_rng(5)
    p = _cheap_restore_params(slo_ns=[10 ** 6] * 16, num_classes=16)
    for _ in range(300):
        tier = int(rng.choice([ref.KV_DRAM, ref.KV_NVME]))
        n_in = int(rng.integers(17, 4000))
        n_pre = 16 * int(rng.integers(1, (n_in - 1) // 16 + 1))
        elapsed = int(rng.integers(0, 10 ** 6))
        e = ref.eval_one(p, 0, ref.QUEUED, ref.QT_TIER1, tier, p["t_now_ns"] - elapsed, n_in, 1,
                         n_pre, 0)
        b = e["budget_rem_ns"]
        # largest x in [0, prefix blocks] whose restore fits the remaining budget
        best = 0
        for x in range(0, n_pre // 16 + 1):
            if x == 0 or ref.restore_time_ns(p, tier, x) <= b:
                best = x
        assert e["want_blocks"] == best, (b, tier, n_pre)


def test_max_restorable_unit_link_special_case():
    # delta = 0 and one ns per block: x = min(prefix blocks, B_rem)
    p = _cheap_restore_params(link_delta_ns=[0, 0], link_blk_ns=[1, 1], slo_ns=[10 ** 6] * 16,
                              num_classes=16)
    for elapsed in [10 ** 6 - 50, 10 ** 6 - 3, 10 ** 6 - 10_000, 0]:
        e = ref.eval_one(p, 0, ref.QUEUED, ref.QT_TIER1, ref.KV_DRAM, p["t_now_ns"] - elapsed,
                         4000, 1, 3200, 0)
        assert e["want_blocks"] == max(0, min(200, e["budget_rem_ns"]))


def test_inverse_consistency():
    # T_k(x) <= B_rem < T_k(x + 1) whenever 0 < x < prefix blocks
    p = _cheap_restore_params(slo_ns=[2_500_000] * 16, num_classes=16)
    rng = np.random.default_rng(11)
    hits = 0
    for _ in range(300):
        tier = int(rng.choice([ref.KV_DRAM, ref.KV_NVME]))
        e = ref.eval_one(p, 0, ref.QUEUED, ref.QT_TIER1, tier,
                         p["t_now_ns"] - int(rng.integers(0, 2_500_000)), 20000, 1, 19984, 0)
        x, b = e["want_blocks"], e["budget_rem_ns"]
        if 0 < x < 19984 // 16:
            hits += 1
            assert ref.restore_time_ns(p, tier, x) <= b < ref.restore_time_ns(p, tier, x + 1)
        if x == 0:
            assert b <= ref.restore_time_ns(p, tier, 1)
    assert hits > 50


def test_restore_dearer_than_recompute_is_refused():
    # moving one block costs far more than computing its 16 tokens
    p = helpers.base_params(block_tokens=16, c_token_ps=1, c_attn_ps=0, c_iter_ps=1,
                            link_delta_ns=[0, 0], link_blk_ns=[10 ** 6, 10 ** 6],
                            slo_ns=[10 ** 12] * 16, num_classes=16)
    e = ref.eval_one(p, 0, ref.QUEUED, ref.QT_TIER1, ref.KV_DRAM, p["t_now_ns"], 4000, 1, 3200, 0)
    assert e["budget_rem_ns"] > 10 ** 9 and e["want_blocks"] == 0


def test_restore_equal_to_recompute_is_refused():
    # restore time equal to the compute it saves: not strictly cheaper -> 0
    # one iteration, no per-iteration cost: recompute saving of x blocks is
    # x * 16 tokens * 1000 ps = 16 x ns; restore costs 16 x ns with delta 0
    p = helpers.base_params(block_tokens=16, c_token_ps=1000, c_attn_ps=0, c_iter_ps=0,
                            c_decode_ps=0, chunk_tokens=1 << 20, link_delta_ns=[0, 0],
                            link_blk_ns=[16, 16], slo_ns=[10 ** 9] * 16, num_classes=16)
    e = ref.eval_one(p, 0, ref.QUEUED, ref.QT_TIER1, ref.KV_DRAM, p["t_now_ns"], 400, 1, 320, 0)
    assert e["want_blocks"] == 0
    p["link_blk_ns"] = [15, 15]
    e = ref.eval_one(p, 0, ref.QUEUED, ref.QT_TIER1, ref.KV_DRAM, p["t_now_ns"], 400, 1, 320, 0)
    assert e["want_blocks"] == 20


def test_hbm_prefix_is_reused_without_transfer():
    p = helpers.base_params()
    a = ref.eval_one(p, 2, ref.QUEUED, ref.QT_NEW, ref.KV_HBM, p["t_now_ns"], 100, 1, 80, 0)
    b = ref.eval_one(p, 2, ref.QUEUED, ref.QT_NEW, ref.KV_NONE, p["t_now_ns"], 20, 1, 0, 0)
    # an HBM hit only leaves the suffix to compute (attending to the prefix)
    assert a["l_actual_ns"] == ref.compute_ps(p, 20, 80, p["load_decodes"]) // 1000
    assert b["l_actual_ns"] == ref.compute_ps(p, 20, 0, p["load_decodes"]) // 1000
    assert a["want_blocks"] == 0


def test_key_orders_groups_then_budget():
    p = helpers.base_params()
    keys = []
    for state, qt, cls, el in itertools.product([ref.QUEUED, ref.DECODE], [ref.QT_TIER1,
                                                                          ref.QT_TIER2],
                                                [0, 2], [0, 15_000]):
        prog = 3 if state == ref.DECODE else 0
        e = ref.eval_one(p, cls, state, qt, ref.KV_NONE, p["t_now_ns"] - el, 12, 9, 0, prog)
        keys.append((e["key"], e["group"], e["budget_rem_ns"]))
    ks = sorted(keys)
    assert [k[1:] for k in ks] == sorted(k[1:] for k in keys)


# ------------------------------------------------------ shared-prefix restores

def test_shared_prefix_example_per_request_values():
    w, g = helpers.golden_workload("worked_example_shared_prefix.json")
    exp = g["expected_eval"]
    for i in range(len(w["id"])):
        e = _eval_req(w["params"], w, i)
        for k in EVAL_KEYS:
            assert e[k] == exp[k][i], (i, k, e[k], exp[k][i])


def test_shared_prefix_example_step():
    """A leader restoring for its followers inside and outside the batch, a
    follower with a shorter prefix, a member ahead of its leader, a second
    leader capped by the link, and a Tier-2 member that shares nothing."""
    w, g = helpers.golden_workload("worked_example_shared_prefix.json")
    r = ref.step(w)
    exp = g["expected_step"]
    assert r["rc"] == ref.OK
    for k in ["order", "restore_blocks", "tokens_granted", "action", "share_leader",
              "alloc_begin", "alloc_count", "admitted"]:
        assert [int(x) for x in r[k]] == exp[k], (k, list(r[k]), exp[k])
    assert _moves(r["unpack_moves"]) == exp["unpack_moves"]
    assert r["n_slot_list"] == exp["n_slot_list"] and r["n_pack"] == exp["n_pack"]
