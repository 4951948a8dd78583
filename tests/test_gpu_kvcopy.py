"""GPU parity of the paged-KV pack / unpack kernels against the oracle's
per-chunk memcpy (byte-exact).  Small pools are compared in full; the
headline workload's 200 GB pool is checked on sampled chunks, whose expected
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
@pytest.mark.parametrize("chunk", [16, 48, 8192, 32768])
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


def test_headline_step_moves_full_size(dev):
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
    cw = geom["chunk_bytes"] // 4
    pm, um = res["pack_moves"], res["unpack_moves"]
    unpacked = set(um["pool_slot"].tolist())
    for k in rng.choice(npk, 24, replace=False):
        m = pm[k]
        for l, kv in [(0, 0), (L - 1, 1), (int(rng.integers(L)), int(rng.integers(2)))]:
            soff = ((int(m["staging_slot"]) * L + l) * 2 + kv) * cw
            got = st_out[4 * soff:4 * (soff + cw)].view(torch.int32).cpu().numpy()
            exp = synth.hash32_np(_chunk_words(geom, int(m["pool_slot"]), l, kv), 1)
            assert np.array_equal(got.view(np.uint32), exp)
    for k in rng.choice(nup, 24, replace=False):
        m = um[k]
        for l, kv in [(0, 1), (L - 1, 0), (int(rng.integers(L)), int(rng.integers(2)))]:
            words = _chunk_words(geom, int(m["pool_slot"]), l, kv)
            got = pool[4 * words[0]:4 * (words[-1] + 1)].view(torch.int32).cpu().numpy()
            soff = ((int(m["staging_slot"]) * L + l) * 2 + kv) * cw
            exp = synth.hash32_np(np.arange(soff, soff + cw, dtype=np.int64), 2)
            assert np.array_equal(got.view(np.uint32), exp)
    # slots nobody wrote keep their bytes
    for slot in rng.choice(geom["num_blocks"], 64, replace=False):
        if int(slot) in unpacked:
            continue
        words = _chunk_words(geom, int(slot), int(rng.integers(L)), int(rng.integers(2)))
        got = pool[4 * words[0]:4 * (words[-1] + 1)].view(torch.int32).cpu().numpy()
        assert np.array_equal(got.view(np.uint32), synth.hash32_np(words, 1))
    del pool, st_in, st_out
    torch.cuda.empty_cache()
