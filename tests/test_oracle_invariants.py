"""Invariants of the oracle's step over random queues (no GPU), its error
codes, and the byte-exact KV pack/unpack."""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import ref
from tests import helpers


def _check_invariants(w, r):
    _check_invariants_base(w, r)


def _check_invariants_base(w, r, skip_restore_fit=None):
    p = w["params"]
    n = len(w["id"])
    assert r["rc"] == ref.OK
    order = np.asarray(r["order"])
    assert sorted(order.tolist()) == list(range(n))          # a permutation
    ev = [ref.eval_one(p, int(w["slo_class"][i]), int(w["state"][i]), int(w["queue_tier"][i]),
                       int(w["prefix_tier"][i]), int(w["arrival_ns"][i]), int(w["n_in"][i]),
                       int(w["n_out_pred"][i]), int(w["n_prefix"][i]), int(w["n_progress"][i]))
          for i in range(n)]
    keys = [ev[i]["key"] for i in order]
    for a, b, ia, ib in zip(keys, keys[1:], order, order[1:]):
        assert a < b or (a == b and ia < ib)                  # sorted, stable
    assert np.array_equal(r["budget_ns"], [e["budget_rem_ns"] for e in ev])
    st_ = w["state"]
    # decodes come first and are never preempted
    nd = int((st_ == helpers.DECODE).sum())
    assert all(st_[i] == helpers.DECODE for i in order[:nd])
    assert not np.any((st_ == helpers.DECODE) &
                      np.isin(r["action"], [ref.ACT_PREEMPT_OFFLOAD, ref.ACT_PREEMPT_DROP]))
    g = r["tokens_granted"]
    assert g.sum() <= p["token_cap"]
    adm = set(r["admitted"].tolist())
    assert adm == set(np.flatnonzero(g > 0).tolist())         # admitted <=> granted
    # a decode without tokens means the cap ran out before any prefill
    if np.any((st_ == helpers.DECODE) & (g == 0)):
        assert not np.any((st_ != helpers.DECODE) & (g > 0) &
                          (r["queue_tier_out"] == ref.QT_TIER1))
    # restores fit the remaining budget (eq:max_restorable) and the step cap
    rb = r["restore_blocks"]
    if skip_restore_fit is not None:
        rb = np.where(skip_restore_fit, 0, rb)   # a follower's blocks cross no link
    assert rb.sum() <= p["max_move_blocks"]
    for i in np.flatnonzero(rb > 0):
        assert ref.restore_time_ns(p, int(w["prefix_tier"][i]), int(rb[i])) <= r["budget_ns"][i]
        assert rb[i] <= ev[i]["want_blocks"]
    # blocks: new blocks never exceed free + freed
    victims = np.isin(r["action"], [ref.ACT_PREEMPT_OFFLOAD, ref.ACT_PREEMPT_DROP])
    rows = np.diff(w["row_offsets"])
    assert r["alloc_count"].sum() <= len(w["free_slots"]) + rows[victims].sum()
    assert r["n_slot_list"] == len(w["free_slots"]) + rows[victims].sum()
    sl = r["slot_list"]
    assert list(sl[:len(w["free_slots"])]) == list(w["free_slots"])
    vic_order = [i for i in order[::-1] if victims[i]]
    tail = np.concatenate([w["slots"][w["row_offsets"][i]:w["row_offsets"][i + 1]]
                           for i in vic_order]) if vic_order else np.zeros(0)
    assert list(sl[len(w["free_slots"]):]) == list(tail)
    # every allocated slot is distinct
    alloc = np.concatenate([sl[r["alloc_begin"][i]:r["alloc_begin"][i] + r["alloc_count"][i]]
                            for i in r["admitted"]]) if len(r["admitted"]) else np.zeros(0)
    assert len(set(alloc.tolist())) == len(alloc)
    # moves: distinct slots, staging indices 0..k-1
    for mv in (r["unpack_moves"], r["pack_moves"]):
        assert list(mv["staging_slot"]) == list(range(len(mv)))
        assert len(set(mv["pool_slot"].tolist())) == len(mv)
    assert r["n_unpack"] == int(rb[r["action"] == ref.ACT_RESTORE].sum())
    assert r["n_pack"] == int(rows[r["action"] == ref.ACT_PREEMPT_OFFLOAD].sum())
    # every request gets an action; Tier-2 requests are never dropped
    assert np.all((r["action"] >= 1) & (r["action"] <= 6))
    _check_hazards(r)


def _check_hazards(r):
    """Copy-order hazards by brute force over the two move lists: the pack
    move reading the slot an unpack move writes, and back; -1 if none."""
    um, pm = r["unpack_moves"], r["pack_moves"]
    uh, ph = r["unpack_hazard"], r["pack_hazard"]
    assert len(uh) == len(um) and len(ph) == len(pm)
    for m in range(len(um)):
        js = [j for j in range(len(pm)) if pm["pool_slot"][j] == um["pool_slot"][m]]
        assert uh[m] == (js[0] if js else -1)
    for j in range(len(pm)):
        ms = [m for m in range(len(um)) if um["pool_slot"][m] == pm["pool_slot"][j]]
        assert ph[j] == (ms[0] if ms else -1)
    # pairs are mutual
    for m in np.flatnonzero(uh >= 0):
        assert ph[uh[m]] == m


@settings(max_examples=300, deadline=None)
@given(seed=st.integers(0, 2 ** 32 - 1), n=st.integers(1, 64),
       cap=st.integers(1, 400), moves=st.integers(0, 80), rho=st.sampled_from([0, 4096, 65536]),
       nfree=st.integers(0, 80), bt=st.sampled_from([1, 4, 16]))
def test_invariants_property(seed, n, cap, moves, rho, nfree, bt):
    rng = np.random.default_rng(seed)
    p = helpers.base_params(token_cap=cap, max_move_blocks=moves, tier2_reserve_q16=rho,
                            block_tokens=bt)
    w = helpers.random_workload(rng, n, params=p, n_free=None)
    w["free_slots"] = w["free_slots"][:nfree]
    _check_invariants(w, ref.step(w))


def _check_sharing(w, r):
    """Shared-prefix restores: a follower (SHARE) sits behind its leader in
    the same priority group, uses no more blocks than the leader restores or
    its own prefix holds, and is in the batch only if its leader restores in
    the batch; the link carries at most U blocks."""
    p = w["params"]
    order = list(r["order"])
    pos = {i: k for k, i in enumerate(order)}
    adm = set(r["admitted"].tolist())
    link = r["restore_blocks"][np.isin(r["action"], [ref.ACT_RESTORE, ref.ACT_PREFETCH])].sum()
    assert link <= p["max_move_blocks"]
    for i in np.flatnonzero(r["action"] == ref.ACT_SHARE):
        lead = int(r["share_leader"][i])
        assert lead >= 0 and pos[lead] < pos[i]
        assert w["prefix_group"][lead] == w["prefix_group"][i] >= 0
        assert r["queue_tier_out"][lead] == r["queue_tier_out"][i]
        assert r["action"][lead] in (ref.ACT_RESTORE, ref.ACT_PREFETCH)
        u = int(r["restore_blocks"][i])
        assert 0 < u <= min(int(r["restore_blocks"][lead]),
                            int(w["n_prefix"][i]) // p["block_tokens"])
        if i in adm:
            assert lead in adm and r["action"][lead] == ref.ACT_RESTORE
    assert np.all((r["share_leader"] >= 0) == (r["action"] == ref.ACT_SHARE))


@settings(max_examples=300, deadline=None)
@given(seed=st.integers(0, 2 ** 32 - 1), n=st.integers(1, 64),
       cap=st.integers(1, 400), moves=st.integers(0, 80), rho=st.sampled_from([0, 4096, 65536]),
       groups=st.integers(1, 6))
def test_shared_prefix_invariants(seed, n, cap, moves, rho, groups):
    rng = np.random.default_rng(seed)
    p = helpers.base_params(token_cap=cap, max_move_blocks=moves, tier2_reserve_q16=rho)
    w = helpers.random_workload(rng, n, params=p)
    w["prefix_group"] = np.where(rng.random(n) < 0.8, rng.integers(0, min(groups, n), n),
                                 -1).astype(np.int32)
    r = ref.step(w)
    sharing = r["action"] == ref.ACT_SHARE
    r2 = dict(r)
    r2["action"] = np.where(sharing, ref.ACT_RECOMPUTE, r["action"])  # the rest as before
    _check_invariants_base(w, r2, skip_restore_fit=sharing)
    _check_sharing(w, r)


def test_shared_prefix_group_ids_in_range():
    w = helpers.random_workload(np.random.default_rng(1), 5)
    for bad in ([-2, 0, 0, 0, 0], [0, 0, 5, 0, 0]):
        w["prefix_group"] = np.array(bad, np.int32)
        assert ref.step(w)["rc"] == ref.EINVAL


def test_invariants_on_synthetic_configs():
    import paper_2608_06557_amd.synth as synth
    for cfg in range(4):
        w = synth.make_workload(cfg, n=2048)
        _check_invariants(w, ref.step(w))


def test_hazards_present_on_tiny_config():
    """The tiny workload hands preempted requests' slots to restores, so the
    copy order matters there: every such slot is a victim's slot that the
    step spills (Section 4.4) and a restore then receives."""
    import paper_2608_06557_amd.synth as synth
    w = synth.make_workload(0)
    r = ref.step(w)
    _check_hazards(r)
    uh = r["unpack_hazard"]
    assert (uh >= 0).sum() > 10
    nf = len(w["free_slots"])
    sl = r["slot_list"]
    victims_region = set(sl[nf:].tolist())
    for m in np.flatnonzero(uh >= 0):
        assert int(r["unpack_moves"]["pool_slot"][m]) in victims_region
    for m in np.flatnonzero(uh < 0):
        s = int(r["unpack_moves"]["pool_slot"][m])
        assert s in set(sl[:nf].tolist()) or s not in set(r["pack_moves"]["pool_slot"].tolist())


def test_empty_queue():
    w = helpers.random_workload(np.random.default_rng(0), 1)
    for k in ["id", "slo_class", "state", "queue_tier", "prefix_tier", "arrival_ns", "n_in",
              "n_out_pred", "n_prefix", "n_progress"]:
        w[k] = w[k][:0]
    w["row_offsets"] = np.zeros(1, np.int32)
    w["slots"] = np.zeros(0, np.int32)
    r = ref.step(w)
    assert r["rc"] == ref.OK and r["n_admitted"] == 0 and r["n_unpack"] == 0 and r["n_pack"] == 0
    assert r["n_slot_list"] == len(w["free_slots"])


# ---------------------------------------------------------------- error codes

def _mutations():
    """(name, function) pairs that each break exactly one domain rule."""
    def setf(field, idx, val):
        def f(w):
            w[field] = w[field].copy()
            w[field][idx] = val
        return f

    def setp(key, val):
        def f(w):
            w["params"] = dict(w["params"])
            w["params"][key] = val
        return f
    return [
        ("ids not increasing", setf("id", 1, 10)),
        ("class out of range", setf("slo_class", 0, 2)),
        ("bad state", setf("state", 2, 3)),
        ("bad queue tier", setf("queue_tier", 2, 3)),
        ("bad prefix tier", setf("prefix_tier", 2, 4)),
        ("n_in zero", setf("n_in", 2, 0)),
        ("n_in too big", setf("n_in", 2, (1 << 17) + 1)),
        ("n_out negative", setf("n_out_pred", 2, -1)),
        ("prefix not block aligned", setf("n_prefix", 0, 321)),
        ("prefix covers prompt", setf("n_prefix", 0, 400)),
        ("queued prefix without tier", setf("prefix_tier", 0, 3)),
        ("queued tier without prefix", setf("prefix_tier", 2, 1)),
        ("queued with progress", setf("n_progress", 2, 1)),
        ("arrival in the future", setf("arrival_ns", 2, 100001)),
        ("arrival negative", setf("arrival_ns", 2, -1)),
        ("prefill progress zero", setf("n_progress", 4, 0)),
        ("prefill progress complete", setf("n_progress", 4, 1000)),
        ("prefill row length", setf("n_progress", 4, 520)),
        ("decode row length", setf("n_progress", 3, 20)),
        ("row offsets start", setf("row_offsets", 0, 1)),
        ("slot out of range", setf("slots", 3, 1000)),
        ("slot negative", setf("slots", 3, -1)),
        ("free slot out of range", setf("free_slots", 5, 1000)),
        ("block_tokens 0", setp("block_tokens", 0)),
        ("chunk too small", setp("chunk_tokens", 15)),
        ("gamma below 1", setp("gamma_q16", 65535)),
        ("load above max", setp("load_decodes", 5)),
        ("max_batch 0", setp("max_batch", 0)),
        ("num_classes 0", setp("num_classes", 0)),
        ("num_classes 17", setp("num_classes", 17)),
        ("token cap 0", setp("token_cap", 0)),
        ("reserve above 1", setp("tier2_reserve_q16", 65537)),
        ("negative move cap", setp("max_move_blocks", -1)),
        ("c_token too big", setp("c_token_ps", (1 << 28) + 1)),
        ("c_attn too big", setp("c_attn_ps", (1 << 16) + 1)),
        ("iteration cost too big", setp("c_iter_ps", 1 << 36)),
        ("link blk zero", setp("link_blk_ns", [0, 1800])),
        ("link delta too big", setp("link_delta_ns", [1000, (1 << 40) + 1])),
        ("t_now negative", setp("t_now_ns", -1)),
        ("slo too big", setp("slo_ns", [60000, (1 << 50) + 1] + [0] * 14)),
        ("free list larger than pool", setp("num_blocks", 39)),
    ]


MUTATIONS = _mutations()


def test_worked_example_is_valid():
    w, _ = helpers.worked_example()
    assert ref.step(w)["rc"] == ref.OK


@pytest.mark.parametrize("name,mutate", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_einval(name, mutate):
    w, _ = helpers.worked_example()
    mutate(w)
    assert ref.step(w)["rc"] == ref.EINVAL


def test_enospc_reports_required_sizes():
    w, g = helpers.worked_example()
    exp = g["expected_step"]
    for caps in [(71, 100, 100), (100, 19, 100), (100, 100, 31), (0, 0, 0)]:
        r = ref.step(w, slot_cap=caps[0], unpack_cap=caps[1], pack_cap=caps[2])
        assert r["rc"] == ref.ENOSPC
        assert r["n_slot_list"] == exp["n_slot_list"]
        assert r["n_unpack"] == exp["n_unpack"] and r["n_pack"] == exp["n_pack"]
        assert list(r["order"]) == exp["order"]
    r = ref.step(w, slot_cap=72, unpack_cap=20, pack_cap=32)
    assert r["rc"] == ref.OK


# ------------------------------------------------------------ pack / unpack

def _geom(layout, num_blocks, L=3, chunk=64):
    if layout == "layer_major":
        return dict(num_layers=L, chunk_bytes=chunk, slot_stride=chunk,
                    kv_stride=num_blocks * chunk, layer_stride=2 * num_blocks * chunk)
    return dict(num_layers=L, chunk_bytes=chunk, slot_stride=2 * L * chunk, kv_stride=chunk,
                layer_stride=2 * chunk)


@pytest.mark.parametrize("layout", ["layer_major", "block_major"])
def test_pack_unpack_identity_and_bytes(layout):
    rng = np.random.default_rng(9)
    nb, L, chunk = 50, 3, 64
    g = _geom(layout, nb, L, chunk)
    pool = rng.integers(0, 256, 2 * L * nb * chunk, dtype=np.uint8)
    slots = rng.permutation(nb)[:17].astype(np.int32)
    moves = np.zeros(17, ref.MOVE_DTYPE)
    moves["pool_slot"] = slots
    moves["staging_slot"] = np.arange(17)
    staging = np.zeros(17 * 2 * L * chunk, np.uint8)
    ref.pack(pool, g, staging, moves)
    # staging slot j holds (layer, K/V) chunks of pool slot j back to back
    for j, s in enumerate(slots):
        for l in range(L):
            for kv in range(2):
                off = l * g["layer_stride"] + kv * g["kv_stride"] + s * g["slot_stride"]
                soff = ((j * L + l) * 2 + kv) * chunk
                assert np.array_equal(staging[soff:soff + chunk], pool[off:off + chunk])
    pool2 = rng.integers(0, 256, pool.size, dtype=np.uint8)
    before = pool2.copy()
    ref.unpack(pool2, g, staging, moves)
    touched = np.zeros(pool.size, bool)
    for s in slots:
        for l in range(L):
            for kv in range(2):
                off = l * g["layer_stride"] + kv * g["kv_stride"] + s * g["slot_stride"]
                touched[off:off + chunk] = True
    assert np.array_equal(pool2[touched], pool[touched])       # pack then unpack = identity
    assert np.array_equal(pool2[~touched], before[~touched])   # nothing else written
