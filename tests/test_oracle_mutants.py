"""Planted mistakes: each one is a plausible misreading of the paper written
into a copy of the oracle's C source, compiled on the CPU, and run through
the oracle's pins (the hand-derived examples, the brute-force definitions,
the closed forms, the textbook LRU).  Every mutant must fail at least one of
them; a mutant that passes everything would mark a branch of the oracle that
nothing pins.  No GPU is involved.
"""
import os
import subprocess

import numpy as np
import pytest

from oracle import ref
from tests import helpers
from tests import test_oracle_bruteforce as bf
from tests import test_oracle_pins as pins
from tests import test_oracle_reclaim as rc
from tests import test_oracle_prefix as pf

SRC = os.path.join(os.path.dirname(ref.LIB_PATH), "cascade_ref.c")


def _step_pins():
    """The step's pins, as zero-argument checks."""
    yield pins.test_worked_example_per_request_values
    yield pins.test_worked_example_step
    yield pins.test_second_example_per_request_values
    yield pins.test_second_example_step
    yield pins.test_restore_equal_to_recompute_is_refused
    yield pins.test_max_restorable_brute_force
    yield pins.test_inverse_consistency
    yield pins.test_gamma_one_is_plain_average
    yield pins.test_budget_subtracts_estimate_and_elapsed
    for args in [(ref.QUEUED, ref.QT_NEW, False, ref.QT_TIER2),
                 (ref.QUEUED, ref.QT_TIER1, False, ref.QT_TIER1),
                 (ref.QUEUED, ref.QT_TIER2, True, ref.QT_TIER1)]:
        yield lambda a=args: pins.test_tier_transitions(*a)
    yield lambda: bf.test_order_is_unique_sorted_permutation(1)
    yield bf.test_all_equal_keys_give_identity_order
    yield lambda: [bf._check_against_definitions(w) for w in bf._cases(150, 8, 101)]
    yield bf.test_definitions_under_scarce_resources
    yield pins.test_shared_prefix_example_step
    yield lambda: bf.test_shared_prefix_step_matches_definitions(0)


def _other_pins():
    yield rc.test_reclaim_order_is_textbook_lru
    yield rc.test_equal_last_use_reclaims_the_lower_slots
    yield rc.test_empty_slots_go_first_whatever_their_stamp
    yield rc.test_hand_example_three_tiers
    for seed in (0, 1):
        yield lambda s=seed: rc.test_cascade_keeps_index_and_blocks_consistent(s)
    yield pf.test_hand_example
    for cfg in (0, 1):
        yield lambda c=cfg: pf.test_round_trip_from_cached_runs(c)
    yield pf.test_more_entries_never_shorten_a_match


# (name, exact fragment of the oracle source, its mutated text)
MUTANTS = [
    # Section 4.4: a restore outside the batch is prefetched (HBM only at
    # the final hop), not dropped to recompute
    ("prefetch becomes recompute",
     "adm[i] ? CREF_ACT_RESTORE : CREF_ACT_PREFETCH;",
     "adm[i] ? CREF_ACT_RESTORE : CREF_ACT_RECOMPUTE;"),
    # a shared HBM prefix is referenced in place
    ("hbm prefix not retained",
     "} else if (st[i] != CREF_QUEUED || pt[i] == CREF_KV_HBM) {",
     "} else if (st[i] != CREF_QUEUED) {"),
    # spills in the order victims are preempted, from the back of the order
    ("pack moves from the front",
     "int64_t npk = 0;\n  for (int32_t q = n - 1; q >= 0; q--) {",
     "int64_t npk = 0;\n  for (int32_t q = 0; q < n; q++) {"),
    ("victims' rows enter the slot list from the front",
     "for (int32_t q = n - 1; q >= 0; q--) {\n    int32_t i = pq[q].idx;\n    if (!victim[i]) continue;",
     "for (int32_t q = 0; q < n; q++) {\n    int32_t i = pq[q].idx;\n    if (!victim[i]) continue;"),
    # Algorithm 1 preempts the largest remaining budget first
    ("victims from the front of the order",
     "for (int32_t q = n - 1; q >= 0 && deficit > 0; q--) {",
     "for (int32_t q = 0; q < n && deficit > 0; q++) {"),
    # the spill crosses the DRAM link only
    ("spill priced on the NVMe path",
     "cref_restore_time_ns(p, CREF_KV_DRAM, held) <= ev[i].budget_rem_ns",
     "cref_restore_time_ns(p, CREF_KV_NVME, held) <= ev[i].budget_rem_ns"),
    # eq:opt_goal_compact's link constraint
    ("restore cap ignored",
     "int64_t take = min64(ev[i].want_blocks, move_left);",
     "int64_t take = ev[i].want_blocks;"),
    # Tier-2 gets every token decode and Tier-1 leave, not just the reserve
    ("tier-2 limited to its reserve",
     "if (q == e1) left = p->token_cap - used_first;",
     "if (q == e1) left = reserve2;"),
    ("ties broken by descending position",
     "return x->idx < y->idx ? -1 : (x->idx > y->idx ? 1 : 0);",
     "return x->idx > y->idx ? -1 : (x->idx < y->idx ? 1 : 0);"),
    # admission stops at the first request that does not fit
    ("first fit instead of a prefix",
     "if (cost > avail) { stopped = 1; continue; }",
     "if (cost > avail) { continue; }"),
    ("hbm prefix blocks allocated again",
     "nb[i] = ceil_div(reuse + g[i], bt) - (pt[i] == CREF_KV_HBM ? npre[i] / bt : 0);",
     "nb[i] = ceil_div(reuse + g[i], bt);"),
    ("restore lands at the end of the allocation",
     "int64_t s = next + b;",
     "int64_t s = next + nb[i] - r[i] + b;"),
    # restore only if strictly cheaper than recompute
    ("restore kept on a tie with recompute",
     "if (cref_restore_time_ns(p, ptier, x) >= recompute_all - with_restore) x = 0;",
     "if (cref_restore_time_ns(p, ptier, x) > recompute_all - with_restore) x = 0;"),
    # Tier-1 iff B > 0
    ("tier-1 at zero budget",
     "else tier_out = (b0 > 0) ? CREF_QT_TIER1 : CREF_QT_TIER2;",
     "else tier_out = (b0 >= 0) ? CREF_QT_TIER1 : CREF_QT_TIER2;"),
    ("decode load used for the maximum estimate",
     "const int64_t dmax = p->max_batch - 1;",
     "const int64_t dmax = p->load_decodes;"),
    # shared prefixes: a follower references at most its own prefix
    ("follower takes the leader's whole restore",
     "shared[i] = r[lead] < pb ? r[lead] : pb;",
     "shared[i] = r[lead];"),
    ("leader chosen without a restore want",
     "if (deep && ev[i].want_blocks > 0) leader_of[slot] = i;",
     "if (deep) leader_of[slot] = i;"),
    ("sharing across priority groups",
     "int32_t slot = deep ? 2 * pg[i] + (ev[i].group == 2 ? 1 : 0) : -1;",
     "int32_t slot = deep ? 2 * pg[i] : -1;"),
    ("shared blocks allocated again",
     "nb[i] = ceil_div(bt * shared[i] + g[i], bt) - shared[i];",
     "nb[i] = ceil_div(bt * shared[i] + g[i], bt);"),
    ("follower still charged to the link",
     "      r[i] = 0;\n      continue;",
     "      r[i] = 0;\n      move_left -= min64(ev[i].want_blocks, move_left);\n      continue;"),
    # Section 4.4: least recently used first
    ("reclaim most recent first",
     "if (x->last_use != y->last_use) return x->last_use < y->last_use ? -1 : 1;",
     "if (x->last_use != y->last_use) return x->last_use > y->last_use ? -1 : 1;"),
    ("reclaim ties by the higher slot",
     "return x->slot < y->slot ? -1 : (x->slot > y->slot ? 1 : 0);\n}\nstatic int cmp_i32",
     "return x->slot > y->slot ? -1 : (x->slot < y->slot ? 1 : 0);\n}\nstatic int cmp_i32"),
    ("demotion sets the wrong tier bit",
     "if (demote[i]) *m = (uint8_t)(*m | (1u << (tier + 1)));",
     "if (demote[i]) *m = (uint8_t)(*m | (1u << tier));"),
    ("empty slots ranked by their stamp",
     "cand[n_free].last_use = block_hash[s] != 0 ? last_use_ns[s] : 0;\n    cand[n_free].slot = s;",
     "cand[n_free].last_use = last_use_ns[s];\n    cand[n_free].cached = 1;\n    cand[n_free].slot = s;"),
    # the prefix run stops at the first uncached block
    ("prefix run skips a gap",
     "if (!hit) break;",
     "if (!hit) { matched++; continue; }"),
    ("prefix tier is the shallowest",
     "if (hit->tier > tier) tier = hit->tier;",
     "if (matched == 0 || hit->tier < tier) tier = hit->tier;"),
]


def _build_mutant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, f"fragment of '{name}' not found once in the oracle"
    d = tmp_path / name.replace(" ", "_").replace("'", "")
    d.mkdir()
    for f in ("cascade_ref.h",):
        (d / f).write_text(open(os.path.join(os.path.dirname(SRC), f)).read())
    (d / "cascade_ref.c").write_text(src.replace(old, new))
    so = d / "libmutant.so"
    subprocess.run(["gcc", "-std=gnu11", "-O1", "-fPIC", "-shared", "-o", str(so),
                    str(d / "cascade_ref.c")], check=True)
    return str(so)


def _caught(checks):
    """Name of the first check the loaded oracle fails, else None."""
    for chk in checks:
        try:
            chk()
        except (AssertionError, KeyError, IndexError, ValueError) as e:
            return f"{getattr(chk, '__name__', 'check')}: {type(e).__name__}"
    return None


def test_unmutated_oracle_passes_the_checks(tmp_path):
    """The harness itself: a copy built the same way passes everything."""
    so = _build_mutant(tmp_path, "identity", "int32_t cref_step(", "int32_t cref_step(")
    with ref.library(so):
        assert _caught(list(_step_pins()) + list(_other_pins())) is None


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(tmp_path, name, old, new):
    so = _build_mutant(tmp_path, name, old, new)
    with ref.library(so):
        hit = _caught(list(_step_pins()) + list(_other_pins()))
    assert hit is not None, f"planted mistake '{name}' passes every pin"
