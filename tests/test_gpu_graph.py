"""The library under HIP graph capture: the scheduling step with its KV copies,
and a tier reclamation chain, captured once and replayed several times with
eager work and synchronizations between replays.  Every replay must give the
eager result: nothing the library enqueues may depend on host state at
capture time or on a memset node (none is used: buffers are cleared by
kernels)."""
import numpy as np
import pytest
import torch  # noqa: F401  (imported at collection: the first import is slow)

from paper_2608_06557_amd import synth

pytestmark = pytest.mark.gpu

STEP_KEYS = ["budget_ns", "action", "queue_tier_out", "tokens_granted", "restore_blocks",
             "order", "alloc_begin", "alloc_count", "admitted", "slot_list", "unpack_moves",
             "pack_moves", "unpack_hazard", "pack_hazard"]


@pytest.fixture(scope="module")
def dev():
    import torch
    from paper_2608_06557_amd import cascade, device
    assert torch.cuda.is_available()
    cascade.load()
    return device


@pytest.mark.parametrize("cfg", [0, 2])
def test_step_and_copies_replay_like_eager(dev, cfg):
    import torch
    from paper_2608_06557_amd import cascade
    w = synth.make_workload(cfg)
    d = dev.DeviceStep(w)
    s = torch.cuda.Stream()
    assert d.run(s) == 0
    torch.cuda.synchronize()
    ref = d.fetch()
    # a small pool of 256-byte chunks so the copies run for real
    nb = int(w["params"]["num_blocks"])
    geom = synth.kv_geometry("8b", nb, chunk_bytes=256)
    blk = 2 * geom["num_layers"] * geom["chunk_bytes"]
    npk, nup = ref["n_pack"], ref["n_unpack"]
    rng = np.random.default_rng(cfg)
    pool0 = torch.from_numpy(rng.integers(0, 256, geom["pool_bytes"], dtype=np.uint8)).cuda()
    pool = pool0.clone()
    pst = torch.zeros(max(npk, 1) * blk, dtype=torch.uint8, device="cuda")
    ust = torch.from_numpy(rng.integers(0, 256, max(nup, 1) * blk, dtype=np.uint8)).cuda()
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    pl = dev.kv_pool_struct(pool.data_ptr(), geom)

    def enqueue():
        rc = d.run(s)
        return rc | cascade.cascade_pack_unpack(
            pl, pst.data_ptr(), max(npk, 1), d.pack_moves.data_ptr(), d.n_pack_ptr(),
            d.caps[2], d.pack_hazard.data_ptr(), ust.data_ptr(), max(nup, 1),
            d.unpack_moves.data_ptr(), d.n_unpack_ptr(), d.caps[1], d.unpack_hazard.data_ptr(),
            st.data_ptr(), int(s.cuda_stream))

    with torch.cuda.stream(s):
        assert enqueue() == 0
    torch.cuda.synchronize()
    want_pool, want_pst = pool.clone(), pst.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        assert enqueue() == 0
    for r in range(4):
        # eager work between replays: scramble every output, restore the pool
        for k in ["order", "action", "budget_ns"]:
            d.out[k].fill_(7)
        d.slot_list.fill_(-3)
        d.unpack_hazard.fill_(99)
        pool.copy_(pool0)
        pst.zero_()
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            g.replay()
        torch.cuda.synchronize()
        got = d.fetch()
        assert got["status"] == 0 and int(st.item()) == 0
        for k in STEP_KEYS:
            assert np.array_equal(np.asarray(got[k]), np.asarray(ref[k])), (cfg, r, k)
        assert torch.equal(pool, want_pool), (cfg, r)
        assert torch.equal(pst, want_pst), (cfg, r)


@pytest.mark.parametrize("one_call", [False, True], ids=["per_tier", "chain_call"])
def test_tier_chain_replays_like_eager(dev, one_call):
    import torch
    w = synth.make_tier_workload(0, seed=77, sizes=(6000, 9000, 20000), needs=(1200, 500, 30),
                                 held=(0.3, 0.1, 0.05), empty=(0.01, 0.01, 0.01))
    d = dev.DeviceTiers(w["tables"], w["needs"], w["index_keys"], w["index_masks"])
    keep = ([b.clone() for b in d.bh], [x.clone() for x in d.lu], d.index.clone())
    s = torch.cuda.Stream()

    def restore():
        for t in range(3):
            d.bh[t].copy_(keep[0][t])
            d.lu[t].copy_(keep[1][t])
        d.index.copy_(keep[2])
        d.status.zero_()
        d.n_out.fill_(-1)
        for t in range(3):
            d.freed[t].fill_(-1)
            d.placed[t].fill_(-1)
        torch.cuda.synchronize()

    run = d.run_chain if one_call else d.run
    d.chain_args()  # the chain call's workspace, allocated outside the capture
    restore()
    assert run(s) == 0
    ref = d.fetch()
    assert ref["status"] == 0
    restore()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        assert run(s) == 0
    for r in range(4):
        restore()
        with torch.cuda.stream(s):
            g.replay()
        got = d.fetch()
        assert got["status"] == 0
        for t in range(3):
            for k in ["freed", "placed", "block_hash", "last_use_ns"]:
                assert np.array_equal(got["tiers"][t][k], ref["tiers"][t][k]), (r, t, k)
            assert got["tiers"][t]["n_outgoing"] == ref["tiers"][t]["n_outgoing"]
        assert np.array_equal(got["index"][0], ref["index"][0])
        assert np.array_equal(got["index"][1], ref["index"][1])
