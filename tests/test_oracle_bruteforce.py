"""Brute-force checks of the oracle's step on tiny queues (n <= 8).

Each part of the step is checked against its definition evaluated by
exhaustion or unit-by-unit simulation, not against a retyped formula:

* order: the unique permutation sorted by (group, remaining budget), ties by
  input position, found among all n! permutations (Algorithm 1's
  least-remaining-budget-first sort; decodes first, Section 4.4);
* restore cap and token grants: handed out one block / one token at a time in
  priority order (eq:opt_goal_compact link constraint; chunked prefill cap
  with the Tier-2 reserve);
* admission: the longest prefix of the granted requests whose blocks fit;
* victims: among all subsets of preemptible holders, the smallest set taken
  from the back of the order that covers the deficit (Algorithm 1 preempts
  the largest remaining budget first; Section 4.4 never preempts decodes).
"""
import itertools
import math

import numpy as np
import pytest

from oracle import ref
from tests import helpers


def _evals(w):
    p = w["params"]
    return [ref.eval_one(p, int(w["slo_class"][i]), int(w["state"][i]), int(w["queue_tier"][i]),
                         int(w["prefix_tier"][i]), int(w["arrival_ns"][i]), int(w["n_in"][i]),
                         int(w["n_out_pred"][i]), int(w["n_prefix"][i]), int(w["n_progress"][i]))
            for i in range(len(w["id"]))]


def _clamp(b):
    return max(-(1 << 61), min((1 << 61) - 1, b))


def _cases(count, nmax, seed):
    rng = np.random.default_rng(seed)
    for _ in range(count):
        n = int(rng.integers(1, nmax + 1))
        yield helpers.random_workload(rng, n)


@pytest.mark.parametrize("seed", [1, 2])
def test_order_is_unique_sorted_permutation(seed):
    for w in _cases(150, 6, seed):
        ev = _evals(w)
        n = len(ev)
        rank = [(e["group"], _clamp(e["budget_rem_ns"])) for e in ev]
        sorted_perms = [perm for perm in itertools.permutations(range(n))
                        if all(rank[perm[k]] < rank[perm[k + 1]] or
                               (rank[perm[k]] == rank[perm[k + 1]] and perm[k] < perm[k + 1])
                               for k in range(n - 1))]
        assert len(sorted_perms) == 1
        r = ref.step(w)
        assert r["rc"] == ref.OK
        assert tuple(r["order"]) == sorted_perms[0]


def test_all_equal_keys_give_identity_order():
    rng = np.random.default_rng(3)
    w = helpers.random_workload(rng, 8)
    for k in ["slo_class", "state", "queue_tier", "prefix_tier", "arrival_ns", "n_in",
              "n_out_pred", "n_prefix", "n_progress"]:
        w[k] = np.repeat(w[k][:1], 8)
    w["state"][:] = helpers.QUEUED
    w["n_progress"][:] = 0
    w["prefix_tier"][:] = helpers.KV_DRAM
    w["n_prefix"][:] = w["params"]["block_tokens"] * ((w["n_in"][0] - 1) // w["params"]["block_tokens"])
    if w["n_prefix"][0] == 0:
        w["prefix_tier"][:] = helpers.KV_NONE
    w["row_offsets"] = np.zeros(9, np.int32)
    w["slots"] = np.zeros(0, np.int32)
    r = ref.step(w)
    assert r["rc"] == ref.OK and list(r["order"]) == list(range(8))


def _sharing(w, ev, order):
    """Leaders and followers of shared prefixes, by walking the order: in
    each (prefix group, priority group) the first queued DRAM/NVMe member
    with a positive want leads; every later such member follows it."""
    pg = w.get("prefix_group")
    follows = {}
    if pg is None:
        return follows
    leader = {}
    for i in order:
        deep = (int(pg[i]) >= 0 and w["state"][i] == helpers.QUEUED
                and w["prefix_tier"][i] in (helpers.KV_DRAM, helpers.KV_NVME))
        if not deep:
            continue
        key = (int(pg[i]), ev[i]["group"])
        if key in leader:
            follows[i] = leader[key]
        elif ev[i]["want_blocks"] > 0:
            leader[key] = i
    return follows


def _blocks_needed(w, i, g, r, shared=None):
    """New HBM blocks so request i holds its reused/restored prefix and g new
    tokens (the tokens it will have after this step, minus what is already in
    HBM for it: its own row, a shared HBM prefix, or blocks another request
    restores for it)."""
    bt = w["params"]["block_tokens"]
    st, pt = int(w["state"][i]), int(w["prefix_tier"][i])
    row = int(w["row_offsets"][i + 1] - w["row_offsets"][i])
    if shared is not None:
        return math.ceil((bt * shared + g) / bt) - shared
    if st == helpers.DECODE:
        tokens_after = int(w["n_in"][i]) + int(w["n_progress"][i]) + 1
        return math.ceil(tokens_after / bt) - row
    if st == helpers.RUNNING_PREFILL:
        return math.ceil((int(w["n_progress"][i]) + g) / bt) - row
    if pt == helpers.KV_HBM:
        shared = int(w["n_prefix"][i])
        return math.ceil((shared + g) / bt) - shared // bt
    return math.ceil((bt * r + g) / bt)


def _check_against_definitions(w):
    p = w["params"]
    ev = _evals(w)
    res = ref.step(w)
    assert res["rc"] == ref.OK
    n = len(ev)
    order = list(res["order"])
    st = w["state"].astype(int)
    bt = p["block_tokens"]
    row = np.diff(w["row_offsets"]).astype(int)

    # restore / prefetch blocks: one block at a time to the first request in
    # priority order that still wants one, until U blocks are out; followers
    # of a shared prefix want none themselves and take min(leader's blocks,
    # own prefix blocks) of the leader's restore
    follows = _sharing(w, ev, order)
    got = [0] * n
    for _ in range(min(p["max_move_blocks"], 10 ** 6)):
        nxt = next((i for i in order if i not in follows and got[i] < ev[i]["want_blocks"]),
                   None)
        if nxt is None:
            break
        got[nxt] += 1
    share = {i: min(got[l], int(w["n_prefix"][i]) // bt) for i, l in follows.items()}
    assert list(res["restore_blocks"]) == [share.get(i, got[i]) for i in range(n)]
    if "prefix_group" in w:
        assert list(res["share_leader"]) == [follows[i] if share.get(i, 0) > 0 else -1
                                            for i in range(n)]

    # tokens: one at a time; decodes and Tier-1 share cap - reserve (the
    # reserve exists only if Tier-2 is non-empty), Tier-2 gets what is left
    def need(i):
        if st[i] == helpers.DECODE:
            return 1
        if st[i] == helpers.RUNNING_PREFILL:
            return int(w["n_in"][i] - w["n_progress"][i])
        if w["prefix_tier"][i] == helpers.KV_HBM:
            return int(w["n_in"][i] - w["n_prefix"][i])
        if i in share:
            return int(w["n_in"][i]) - bt * share[i]
        return int(w["n_in"][i]) - bt * got[i]
    has2 = any(e["group"] == 2 for e in ev)
    reserve = (p["token_cap"] * p["tier2_reserve_q16"]) // 65536 if has2 else 0
    g = [0] * n
    first = [i for i in order if ev[i]["group"] <= 1]
    second = [i for i in order if ev[i]["group"] == 2]
    used1 = 0
    while used1 < p["token_cap"] - reserve:
        nxt = next((i for i in first if g[i] < need(i)), None)
        if nxt is None:
            break
        g[nxt] += 1
        used1 += 1
    total = used1
    while total < p["token_cap"]:
        nxt = next((i for i in second if g[i] < need(i)), None)
        if nxt is None:
            break
        g[nxt] += 1
        total += 1
    assert sum(g) <= p["token_cap"]

    # admission: the longest prefix of the granted requests (in order) whose
    # new blocks plus the blocks they already hold fit in free + held blocks
    granted = [i for i in order if g[i] > 0]
    held_total = int(sum(row[i] for i in range(n) if st[i] == helpers.RUNNING_PREFILL))
    avail = len(w["free_slots"]) + held_total
    nbk = lambda i: _blocks_needed(w, i, g[i], got[i], share.get(i))
    cost = {i: nbk(i) + (row[i] if st[i] == helpers.RUNNING_PREFILL else 0) for i in granted}
    best = 0
    for j in range(len(granted) + 1):
        if sum(cost[i] for i in granted[:j]) <= avail:
            best = j
    admitted = granted[:best]
    assert list(res["admitted"]) == admitted
    for i in range(n):
        assert res["tokens_granted"][i] == (g[i] if i in admitted else 0)
        if i in admitted:
            assert res["alloc_count"][i] == nbk(i)

    # victims: smallest set of non-admitted prefill holders, taken from the
    # back of the order, whose blocks cover the deficit
    deficit = sum(nbk(i) for i in admitted) - len(w["free_slots"])
    holders = [i for i in order if st[i] == helpers.RUNNING_PREFILL and i not in admitted
               and row[i] > 0]
    victims = set()
    if deficit > 0:
        best_set = None
        for mask in range(1 << len(holders)):
            s = [holders[k] for k in range(len(holders)) if mask >> k & 1]
            pos = sorted(order.index(i) for i in s)
            back = sorted(order.index(i) for i in holders)[len(holders) - len(s):]
            if pos != back or sum(row[i] for i in s) < deficit:
                continue
            if best_set is None or len(s) < len(best_set):
                best_set = s
        assert best_set is not None      # covering is always possible
        victims = set(best_set)
    spilled = set()
    for i in range(n):
        a = res["action"][i]
        if i in victims:
            spill = ref.restore_time_ns(p, ref.KV_DRAM, int(row[i])) <= ev[i]["budget_rem_ns"]
            assert a == (ref.ACT_PREEMPT_OFFLOAD if spill else ref.ACT_PREEMPT_DROP)
            if spill:
                spilled.add(i)
            continue
        # Section 4.4: KV already in HBM (a running request's rows, a shared
        # HBM prefix) is kept whether or not the request is in the batch; a
        # deeper prefix with blocks under the link cap is restored when the
        # request is in the batch (HBM is allocated at the final hop) and only
        # prefetched otherwise; anything else is recomputed
        if st[i] != helpers.QUEUED or w["prefix_tier"][i] == helpers.KV_HBM:
            assert a == ref.ACT_RETAIN, (i, a)
        elif i in share:
            assert a == (ref.ACT_SHARE if share[i] > 0 else ref.ACT_RECOMPUTE), (i, a)
        elif got[i] > 0:
            assert a == (ref.ACT_RESTORE if i in admitted else ref.ACT_PREFETCH), (i, a)
        else:
            assert a == ref.ACT_RECOMPUTE, (i, a)

    # slot list: the free list, then every victim's row, victims in the order
    # they were preempted (from the back), each row in row order; a spill
    # moves each block of a spilled victim, in that same order
    rows = [list(w["slots"][w["row_offsets"][i]:w["row_offsets"][i + 1]]) for i in range(n)]
    by_back = [i for i in reversed(order) if i in victims]
    assert list(res["slot_list"]) == list(w["free_slots"]) + [s for i in by_back for s in rows[i]]
    want_pack = [(i, b, s) for i in by_back if i in spilled for b, s in enumerate(rows[i])]
    assert [(int(m["req"]), int(m["blk"]), int(m["pool_slot"])) for m in res["pack_moves"]] \
        == want_pack
    assert list(res["pack_moves"]["staging_slot"]) == list(range(len(want_pack)))
    # restores: the first restore_blocks blocks of each admitted restoring
    # request's allocation, in admitted order
    sl = list(res["slot_list"])
    want_unpack = [(i, b, sl[res["alloc_begin"][i] + b]) for i in admitted
                   for b in range(got[i]) if res["action"][i] == ref.ACT_RESTORE]
    assert [(int(m["req"]), int(m["blk"]), int(m["pool_slot"])) for m in res["unpack_moves"]] \
        == want_unpack
    return res


@pytest.mark.parametrize("seed", range(6))
def test_step_matches_definitions(seed):
    for w in _cases(120, 8, 100 + seed):
        _check_against_definitions(w)


def test_definitions_under_scarce_resources():
    rng = np.random.default_rng(77)
    for _ in range(300):
        p = helpers.base_params(token_cap=int(rng.integers(1, 40)),
                                max_move_blocks=int(rng.integers(0, 12)),
                                tier2_reserve_q16=int(rng.choice([0, 4096, 65536])))
        w = helpers.random_workload(rng, int(rng.integers(1, 9)), params=p,
                                    n_free=int(rng.integers(0, 6)))
        _check_against_definitions(w)


def _with_groups(rng, w, k):
    """Random prefix groups (ids below k, -1 for none) on every request;
    the step uses them only for queued DRAM/NVMe requests."""
    n = len(w["id"])
    w["prefix_group"] = np.where(rng.random(n) < 0.75, rng.integers(0, max(1, min(k, n)), n),
                                 -1).astype(np.int32)
    return w


@pytest.mark.parametrize("seed", range(6))
def test_shared_prefix_step_matches_definitions(seed):
    rng = np.random.default_rng(500 + seed)
    for _ in range(150):
        p = helpers.base_params(token_cap=int(rng.integers(1, 400)),
                                max_move_blocks=int(rng.integers(0, 60)),
                                tier2_reserve_q16=int(rng.choice([0, 4096, 65536])))
        w = helpers.random_workload(rng, int(rng.integers(1, 9)), params=p)
        _check_against_definitions(_with_groups(rng, w, int(rng.integers(1, 4))))


def test_shared_prefix_without_members_changes_nothing():
    """Groups on requests that are not queued DRAM/NVMe, or one member per
    group, give exactly the step without groups."""
    rng = np.random.default_rng(9)
    for _ in range(200):
        w = helpers.random_workload(rng, int(rng.integers(1, 9)))
        n = len(w["id"])
        base = ref.step(w)
        w["prefix_group"] = np.arange(n, dtype=np.int32)      # every request alone
        alone = ref.step(w)
        deep = (w["state"] == helpers.QUEUED) & np.isin(w["prefix_tier"],
                                                        [helpers.KV_DRAM, helpers.KV_NVME])
        w["prefix_group"] = np.where(deep, -1, 0).astype(np.int32)  # only non-members grouped
        others = ref.step(w)
        for r in (alone, others):
            assert r["rc"] == base["rc"] == ref.OK
            for k in ["order", "action", "restore_blocks", "tokens_granted", "alloc_begin",
                      "alloc_count", "admitted", "slot_list"]:
                assert np.array_equal(r[k], base[k]), k
            assert np.all(r["share_leader"] == -1)
