"""GPU parity of the paged-KV pack / unpack kernels against the oracle's
per-chunk memcpy (byte-exact).  Small pools are compared in full; the
65536-request workload's 200 GB pool is checked on sampled chunks, whose expected
bytes the CPU regenerates from the counter-based fill."""
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


def _geom(layout, nb, L, chunk):
    if layout == "layer_major":
        g = dict(slot_stride=chunk, kv_stride=nb * chunk, layer_stride=2 * nb * chunk)
    else:
        g = dict(slot_stride=2 * L * chunk, kv_stride=chunk, layer_stride=2 * chunk)
    g.update(num_layers=L, chunk_bytes=chunk, num_blocks=nb)
    return g


def _moves(slots, staging=None):
    m = np.zeros(len(slots), ref.MOVE_DTYPE)
    m["pool_slot"] = slots
    m["staging_slot"] = np.arange(len(slots)) if staging is None else staging
    return m


@pytest.mark.parametrize("layout", ["layer_major", "block_major"])
@pytest.mark.parametrize("chunk", [16, 48, 4096, 8192, 16384, 32768, 65536])
def test_pack_unpack_small(dev, layout, chunk):
    import torch
    from paper_2608_06557_amd import cascade
    rng = np.random.default_rng(chunk)
    nb, L = 40, 3
    g = _geom(layout, nb, L, chunk)
    pool_h = rng.integers(0, 256, 2 * L * nb * chunk, dtype=np.uint8)
    nm = 23
    slots = rng.permutation(nb)[:nm].astype(np.int32)
    stage_ids = rng.permutation(nm + 5)[:nm].astype(np.int32)
    mv = _moves(slots, stage_ids)
    # oracle
    st_h = np.zeros((nm + 5) * 2 * L * chunk, np.uint8)
    ref.pack(pool_h, g, st_h, mv)
    # gpu
    pool = torch.from_numpy(pool_h.copy()).cuda()
    st = torch.zeros(st_h.size, dtype=torch.uint8, device="cuda")
    mv_d = torch.from_numpy(mv.view(np.int32).copy()).cuda()
    n_d = torch.tensor([nm], dtype=torch.int32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    pl = dev.kv_pool_struct(pool.data_ptr(), g)
    s = dev.stream_handle()
    assert cascade.cascade_pack(pl, st.data_ptr(), nm + 5, mv_d.data_ptr(), n_d.data_ptr(), nm,
                                status.data_ptr(), s) == 0
    torch.cuda.synchronize()
    assert np.array_equal(st.cpu().numpy(), st_h)
    # unpack into a different pool: identity on the moved chunks, rest untouched
    pool2_h = rng.integers(0, 256, pool_h.size, dtype=np.uint8)
    exp = pool2_h.copy()
    ref.unpack(exp, g, st_h, mv)
    pool2 = torch.from_numpy(pool2_h.copy()).cuda()
    pl2 = dev.kv_pool_struct(pool2.data_ptr(), g)
    assert cascade.cascade_unpack(pl2, st.data_ptr(), nm + 5, mv_d.data_ptr(), n_d.data_ptr(),
                                  nm, status.data_ptr(), s) == 0
    torch.cuda.synchronize()
    assert np.array_equal(pool2.cpu().numpy(), exp)
    assert int(status.item()) == 0


def test_count_read_on_device_and_bad_moves_skipped(dev):
    import torch
    from paper_2608_06557_amd import cascade
    nb, L, chunk = 8, 2, 64
    g = _geom("layer_major", nb, L, chunk)
    pool = torch.arange(2 * L * nb * chunk, dtype=torch.int32).to(torch.uint8).cuda()
    before = pool.clone()
    mv = _moves(np.array([1, -1, 9, 3], np.int32), np.array([0, 1, 2, 7], np.int32))
    mv_d = torch.from_numpy(mv.view(np.int32).copy()).cuda()
    st = torch.zeros(4 * 2 * L * chunk, dtype=torch.uint8, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    n_d = torch.tensor([4], dtype=torch.int32, device="cuda")
    pl = dev.kv_pool_struct(pool.data_ptr(), g)
    assert cascade.cascade_pack(pl, st.data_ptr(), 4, mv_d.data_ptr(), n_d.data_ptr(), 4,
                                status.data_ptr(), dev.stream_handle()) == 0
    torch.cuda.synchronize()
    assert int(status.item()) == cascade.EINVAL       # slots -1, 9 and staging 7 rejected
    h = st.cpu().numpy().reshape(4, 2 * L, chunk)
    ph = before.cpu().numpy()
    for l in range(L):
        for kv in range(2):
            off = l * g["layer_stride"] + kv * g["kv_stride"] + 1 * chunk
            assert np.array_equal(h[0, 2 * l + kv], ph[off:off + chunk])
    assert not h[1:].any()
    # device count of 0 copies nothing
    n_d.zero_()
    st.zero_()
    assert cascade.cascade_pack(pl, st.data_ptr(), 4, mv_d.data_ptr(), n_d.data_ptr(), 4,
                                status.data_ptr(), dev.stream_handle()) == 0
    torch.cuda.synchronize()
    assert not st.cpu().numpy().any()
    # host-side checks
    bad = dev.kv_pool_struct(pool.data_ptr() + 1, g)
    assert cascade.cascade_pack(bad, st.data_ptr(), 4, mv_d.data_ptr(), n_d.data_ptr(), 4, 0,
                                dev.stream_handle()) == cascade.EINVAL


def _chunk_words(geom, slot, l, kv):
    off = l * geom["layer_stride"] + kv * geom["kv_stride"] + slot * geom["slot_stride"]
    return np.arange(off // 4, (off + geom["chunk_bytes"]) // 4, dtype=np.int64)


def _block_words(geom, slot):
    """Word indices (4-byte words of the pool) of every (layer, K/V) chunk of
    pool slot `slot`, in the chunk order of one staging slot."""
    import torch
    L, cw = geom["num_layers"], geom["chunk_bytes"] // 4
    base = torch.tensor([(l * geom["layer_stride"] + kv * geom["kv_stride"]
                          + slot * geom["slot_stride"]) // 4
                         for l in range(L) for kv in range(2)], dtype=torch.int64,
                        device="cuda")
    return (base[:, None] + torch.arange(cw, device="cuda")[None, :]).reshape(-1)


def _u32(t):
    import torch
    return t.view(torch.int32).to(torch.int64) & 0xFFFFFFFF


def _check_packed_block(st_out, geom, staging_slot, pool_slot, seed):
    """Staging slot `staging_slot` holds all 2L chunks of pool slot
    `pool_slot` as filled with pattern `seed` (checked on the GPU)."""
    import paper_2608_06557_amd.synth as synth
    blk = 2 * geom["num_layers"] * geom["chunk_bytes"]
    got = _u32(st_out[staging_slot * blk:(staging_slot + 1) * blk])
    exp = synth.hash32_torch(_block_words(geom, pool_slot), seed)
    bad = (got != exp).nonzero()
    assert bad.numel() == 0, (staging_slot, pool_slot, int(bad[0]) if bad.numel() else None)


def _check_unpacked_block(pool, geom, pool_slot, staging_slot, seed):
    """Every chunk of pool slot `pool_slot` holds staging slot `staging_slot`
    as filled with pattern `seed`."""
    import torch
    import paper_2608_06557_amd.synth as synth
    blk4 = 2 * geom["num_layers"] * geom["chunk_bytes"] // 4
    got = pool.view(torch.int32)[_block_words(geom, pool_slot)].to(torch.int64) & 0xFFFFFFFF
    exp = synth.hash32_torch(torch.arange(staging_slot * blk4, (staging_slot + 1) * blk4,
                                          device="cuda"), seed)
    bad = (got != exp).nonzero()
    assert bad.numel() == 0, (pool_slot, staging_slot, int(bad[0]) if bad.numel() else None)


def test_65536_request_step_moves_full_size(dev):
    """Config 2 at full size: 200 GB pool, the step's own move lists, pack
    then unpack as the benchmark runs them; sampled chunks checked."""
    import torch
    import paper_2608_06557_amd.synth as synth
    from paper_2608_06557_amd import cascade
    w = synth.make_workload(2)
    geom = w["geometry"]
    d = dev.DeviceStep(w, unpack_cap=geom["num_blocks"], pack_cap=geom["num_blocks"])
    assert d.run() == 0
    res = d.fetch()
    assert res["status"] == 0
    o = ref.step(w)
    assert np.array_equal(res["unpack_moves"].view(np.int32), o["unpack_moves"].view(np.int32))
    assert np.array_equal(res["pack_moves"].view(np.int32), o["pack_moves"].view(np.int32))
    npk, nup = res["n_pack"], res["n_unpack"]
    assert npk > 500 and nup > 500
    print(f"pool {geom['pool_bytes'] / 1e9:.1f} GB, pack {npk}, unpack {nup}", flush=True)
    pool = torch.empty(geom["pool_bytes"], dtype=torch.uint8, device="cuda")
    dev.fill_pattern_(pool, seed=1)
    blk = 2 * geom["num_layers"] * geom["chunk_bytes"]
    st_out = torch.zeros(npk * blk, dtype=torch.uint8, device="cuda")
    st_in = torch.empty(nup * blk, dtype=torch.uint8, device="cuda")
    dev.fill_pattern_(st_in, seed=2)
    pl = dev.kv_pool_struct(pool.data_ptr(), geom)
    s = dev.stream_handle()
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    assert cascade.cascade_pack(pl, st_out.data_ptr(), npk, d.pack_moves.data_ptr(),
                                d.n_pack_ptr(), d.caps[2], status.data_ptr(), s) == 0
    assert cascade.cascade_unpack(pl, st_in.data_ptr(), nup, d.unpack_moves.data_ptr(),
                                  d.n_unpack_ptr(), d.caps[1], status.data_ptr(), s) == 0
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    rng = np.random.default_rng(5)
    L = geom["num_layers"]
    pm, um = res["pack_moves"], res["unpack_moves"]
    unpacked = set(um["pool_slot"].tolist())
    # every (layer, K/V) chunk of each sampled block
    for k in rng.choice(npk, 48, replace=False):
        _check_packed_block(st_out, geom, int(pm[k]["staging_slot"]), int(pm[k]["pool_slot"]), 1)
    for k in rng.choice(nup, 48, replace=False):
        _check_unpacked_block(pool, geom, int(um[k]["pool_slot"]), int(um[k]["staging_slot"]), 2)
    # slots nobody wrote keep their bytes
    for slot in rng.choice(geom["num_blocks"], 64, replace=False):
        if int(slot) in unpacked:
            continue
        words = _chunk_words(geom, int(slot), int(rng.integers(L)), int(rng.integers(2)))
        got = pool[4 * words[0]:4 * (words[-1] + 1)].view(torch.int32).cpu().numpy()
        assert np.array_equal(got.view(np.uint32), synth.hash32_np(words, 1))
    del pool, st_in, st_out
    torch.cuda.empty_cache()


# ------------------------------------------------- pack and unpack in one launch

def _hazards(pm, um):
    """Copy-order pairs by pool slot, the way the step defines them."""
    ph = np.full(len(pm), -1, np.int32)
    uh = np.full(len(um), -1, np.int32)
    for j in range(len(pm)):
        for m in range(len(um)):
            if pm["pool_slot"][j] == um["pool_slot"][m]:
                ph[j], uh[m] = m, j
    return ph, uh


def _fused(dev, pool_t, geom, pst, np_slots, pm, ph, ust, nu_slots, um, uh, caps=None):
    import torch
    from paper_2608_06557_amd import cascade
    cp = len(pm) if caps is None else caps[0]
    cu = len(um) if caps is None else caps[1]
    dv = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int32).copy()
                                    if a.size else np.zeros(4, np.int32)).cuda()
    pm_d, um_d, ph_d, uh_d = dv(pm), dv(um), dv(ph), dv(uh)
    np_d = torch.tensor([len(pm)], dtype=torch.int32, device="cuda")
    nu_d = torch.tensor([len(um)], dtype=torch.int32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    pl = dev.kv_pool_struct(pool_t.data_ptr(), geom)
    rc = cascade.cascade_pack_unpack(pl, pst.data_ptr(), np_slots, pm_d.data_ptr(),
                                     np_d.data_ptr(), cp, ph_d.data_ptr(), ust.data_ptr(),
                                     nu_slots, um_d.data_ptr(), nu_d.data_ptr(), cu,
                                     uh_d.data_ptr(), status.data_ptr(), dev.stream_handle())
    torch.cuda.synchronize()
    return rc, int(status.item())


@pytest.mark.parametrize("layout", ["layer_major", "block_major"])
@pytest.mark.parametrize("chunk", [16, 48, 4096, 8192, 16384])
@pytest.mark.parametrize("n_pack,n_unpack,shared", [(23, 17, 9), (5, 31, 5), (31, 0, 0),
                                                    (0, 12, 0), (40, 40, 40), (1, 1, 1)])
def test_fused_equals_pack_then_unpack(dev, layout, chunk, n_pack, n_unpack, shared):
    """One launch gives the bytes of cascade_pack followed by cascade_unpack,
    also where unpack destinations are pack sources (the shared slots)."""
    import torch
    rng = np.random.default_rng(chunk + 7 * n_pack + n_unpack)
    nb, L = 90, 3
    g = _geom(layout, nb, L, chunk)
    perm = rng.permutation(nb).astype(np.int32)
    p_slots = perm[:n_pack]
    u_slots = np.concatenate([rng.permutation(p_slots)[:shared],
                              perm[n_pack:n_pack + n_unpack - shared]]).astype(np.int32)
    rng.shuffle(u_slots)
    pm = _moves(p_slots, rng.permutation(n_pack + 3)[:n_pack].astype(np.int32))
    um = _moves(u_slots, rng.permutation(n_unpack + 2)[:n_unpack].astype(np.int32))
    ph, uh = _hazards(pm, um)
    assert (uh >= 0).sum() == shared
    pool_h = rng.integers(0, 256, 2 * L * nb * chunk, dtype=np.uint8)
    pst_h = np.zeros((n_pack + 3) * 2 * L * chunk, np.uint8)
    ust_h = rng.integers(0, 256, (n_unpack + 2) * 2 * L * chunk, dtype=np.uint8)
    exp_pool, exp_pst = pool_h.copy(), pst_h.copy()
    ref.pack(exp_pool, g, exp_pst, pm)
    ref.unpack(exp_pool, g, ust_h, um)
    pool = torch.from_numpy(pool_h.copy()).cuda()
    pst = torch.from_numpy(pst_h.copy()).cuda()
    ust = torch.from_numpy(ust_h.copy()).cuda()
    rc, status = _fused(dev, pool, g, pst, n_pack + 3, pm, ph, ust, n_unpack + 2, um, uh)
    assert rc == 0 and status == 0
    assert np.array_equal(pst.cpu().numpy(), exp_pst)
    assert np.array_equal(pool.cpu().numpy(), exp_pool)


def test_fused_any_hazard_arrays_copy_every_move_once(dev):
    """Hazard arrays that declare no real pair (garbage, out of range, or
    one-sided) still leave every move copied exactly once."""
    import torch
    rng = np.random.default_rng(3)
    nb, L, chunk = 60, 2, 64
    g = _geom("layer_major", nb, L, chunk)
    perm = rng.permutation(nb).astype(np.int32)
    pm, um = _moves(perm[:20]), _moves(perm[20:45])
    pool_h = rng.integers(0, 256, 2 * L * nb * chunk, dtype=np.uint8)
    ust_h = rng.integers(0, 256, 25 * 2 * L * chunk, dtype=np.uint8)
    exp_pool, exp_pst = pool_h.copy(), np.zeros(20 * 2 * L * chunk, np.uint8)
    ref.pack(exp_pool, g, exp_pst, pm)
    ref.unpack(exp_pool, g, ust_h, um)
    cases = [(rng.integers(-5, 40, 20), rng.integers(-5, 40, 25)),
             (np.arange(20), np.full(25, -1)),            # pack side only
             (np.full(20, -1), np.arange(25) % 20),       # unpack side only
             (np.full(20, 1 << 30), np.full(25, -(1 << 30)))]
    for ph, uh in cases:
        pool = torch.from_numpy(pool_h.copy()).cuda()
        pst = torch.zeros(exp_pst.size, dtype=torch.uint8, device="cuda")
        ust = torch.from_numpy(ust_h.copy()).cuda()
        rc, status = _fused(dev, pool, g, pst, 20, pm, ph.astype(np.int32), ust, 25, um,
                            uh.astype(np.int32))
        assert rc == 0 and status == 0
        assert np.array_equal(pst.cpu().numpy(), exp_pst)
        assert np.array_equal(pool.cpu().numpy(), exp_pool)


def test_fused_bad_moves_skipped(dev):
    import torch
    from paper_2608_06557_amd import cascade
    nb, L, chunk = 8, 2, 64
    g = _geom("layer_major", nb, L, chunk)
    pool_h = (np.arange(2 * L * nb * chunk) % 251).astype(np.uint8)
    pm = _moves(np.array([1, 9, 3], np.int32), np.array([0, 1, 5], np.int32))   # 9, 5 bad
    um = _moves(np.array([3, -2, 6], np.int32), np.array([0, 1, 2], np.int32))  # -2 bad
    ph, uh = _hazards(pm, um)            # pack 2 (bad staging) pairs with unpack 0
    ust_h = np.full(3 * 2 * L * chunk, 77, np.uint8)
    pool = torch.from_numpy(pool_h.copy()).cuda()
    pst = torch.zeros(3 * 2 * L * chunk, dtype=torch.uint8, device="cuda")
    ust = torch.from_numpy(ust_h.copy()).cuda()
    rc, status = _fused(dev, pool, g, pst, 3, pm, ph, ust, 3, um, uh)
    assert rc == 0 and status == cascade.EINVAL
    exp_pool, exp_pst = pool_h.copy(), np.zeros(pst.numel(), np.uint8)
    ref.pack(exp_pool, g, exp_pst, pm[:1])
    ref.unpack(exp_pool, g, ust_h, um[[0, 2]])  # the pair's unpack still happens
    assert np.array_equal(pst.cpu().numpy(), exp_pst)
    assert np.array_equal(pool.cpu().numpy(), exp_pool)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_fused_step_moves_full_size(dev, cfg):
    """The step's own lists at full size (200 GB / 250 GB pools), hazards
    included: every spilled block that a restore overwrites is checked to
    hold the old bytes in staging, plus samples of the rest."""
    import torch
    import paper_2608_06557_amd.synth as synth
    w = synth.make_workload(cfg)
    geom = w["geometry"]
    d = dev.DeviceStep(w, unpack_cap=geom["num_blocks"], pack_cap=geom["num_blocks"])
    assert d.run() == 0
    res = d.fetch()
    assert res["status"] == 0
    npk, nup = res["n_pack"], res["n_unpack"]
    paired = np.flatnonzero(res["pack_hazard"] >= 0)
    assert npk > 50 and nup > 50
    assert len(paired) > (50 if cfg != 1 else -1)
    print(f"config {cfg}: pool {geom['pool_bytes'] / 1e9:.1f} GB, pack {npk}, unpack {nup}, "
          f"paired {len(paired)}", flush=True)
    pool = torch.empty(geom["pool_bytes"], dtype=torch.uint8, device="cuda")
    dev.fill_pattern_(pool, seed=1)
    blk = 2 * geom["num_layers"] * geom["chunk_bytes"]
    st_out = torch.zeros(npk * blk, dtype=torch.uint8, device="cuda")
    st_in = torch.empty(nup * blk, dtype=torch.uint8, device="cuda")
    dev.fill_pattern_(st_in, seed=2)
    from paper_2608_06557_amd import cascade
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    pl = dev.kv_pool_struct(pool.data_ptr(), geom)
    assert cascade.cascade_pack_unpack(
        pl, st_out.data_ptr(), npk, d.pack_moves.data_ptr(), d.n_pack_ptr(), d.caps[2],
        d.pack_hazard.data_ptr(), st_in.data_ptr(), nup, d.unpack_moves.data_ptr(),
        d.n_unpack_ptr(), d.caps[1], d.unpack_hazard.data_ptr(), status.data_ptr(),
        dev.stream_handle()) == 0
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    rng = np.random.default_rng(11)
    pm, um = res["pack_moves"], res["unpack_moves"]
    # every paired block and a sample of the rest, each with all its chunks
    sample_p = np.unique(np.concatenate([paired, rng.choice(npk, 32, replace=False)]))
    for k in sample_p:
        _check_packed_block(st_out, geom, int(pm[k]["staging_slot"]), int(pm[k]["pool_slot"]), 1)
    sample_u = np.unique(np.concatenate([res["pack_hazard"][paired],
                                         rng.choice(nup, 32, replace=False)]))
    for k in sample_u:
        _check_unpacked_block(pool, geom, int(um[k]["pool_slot"]), int(um[k]["staging_slot"]), 2)
    del pool, st_in, st_out
    torch.cuda.empty_cache()
