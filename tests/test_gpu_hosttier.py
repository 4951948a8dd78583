"""GPU tests of the DRAM-tier side of restores and spills: pinned host blocks
-> staging -> pool (restore) and pool -> staging -> host (spill), pipelined
in batches over two streams, byte-exact against the oracle's per-chunk
memcpy."""
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


def _case(seed, layout, chunk, nm, nb=70, L=3):
    rng = np.random.default_rng(seed)
    g = _geom(layout, nb, L, chunk)
    blk = 2 * L * chunk
    mv = np.zeros(nm, ref.MOVE_DTYPE)
    mv["pool_slot"] = rng.permutation(nb)[:nm]
    mv["staging_slot"] = np.arange(nm)
    # distinct host places in [0, 3*nm] (the buffer holds 3*nm + 1 blocks),
    # about 40 % of them right after the
    # previous move's place (runs that travel as one copy)
    host_off = np.zeros(nm, np.int64)
    used = set()
    for m in range(nm):
        p = int(rng.integers(0, 3 * nm))
        nxt = int(host_off[m - 1] // blk + 1) if m > 0 else -1
        if m > 0 and rng.random() < 0.4 and nxt <= 3 * nm and nxt not in used:
            p = nxt
        while p in used:
            p = (p + 1) % (3 * nm + 1)
        used.add(p)
        host_off[m] = p * blk
    host_len = (3 * nm + 1) * blk
    return rng, g, blk, mv, host_off, host_len


def _restore_spill(dev, layout, chunk, batch, nm=25, nb=70, L=3, n_dev=None, seed=0):
    """Restore nm moves from pinned host blocks into the pool and spill the
    same slots back out, checked byte for byte against the oracle.  Only
    the first n_dev moves (the device count) are unpacked and packed; the
    host link carries all nm.  Every buffer is written on the compute stream
    just before the call, so the copies rely on the entry points' own
    ordering against earlier compute-stream work."""
    import torch
    from paper_2608_06557_amd import cascade
    n_dev = nm if n_dev is None else n_dev
    rng, g, blk, mv, host_off, host_len = _case(seed, layout, chunk, nm, nb=nb, L=L)
    pool_h = rng.integers(0, 256, 2 * g["num_layers"] * g["num_blocks"] * chunk, dtype=np.uint8)
    host = torch.from_numpy(rng.integers(0, 256, host_len, dtype=np.uint8)).pin_memory()
    host_h = host.numpy().copy()
    # restore: staging slot m gets host block host_off[m], then the oracle
    # unpacks the moves the device count covers
    st_h = np.concatenate([host_h[o:o + blk] for o in host_off])
    exp_pool = pool_h.copy()
    ref.unpack(exp_pool, g, st_h, mv[:n_dev])
    comp_s = torch.cuda.current_stream()
    pool = torch.from_numpy(pool_h.copy()).cuda()
    st = torch.full((nm * blk,), 7, dtype=torch.uint8, device="cuda")
    mv_d = torch.from_numpy(mv.view(np.int32).copy()).cuda()
    n_d = torch.tensor([n_dev], dtype=torch.int32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    copy_s = torch.cuda.Stream()
    evs, handles = dev.event_handles(2)
    pl = dev.kv_pool_struct(pool.data_ptr(), g)
    rc = cascade.cascade_restore_from_host(pl, st.data_ptr(), nm, host.data_ptr(), host_off,
                                           mv_d.data_ptr(), n_d.data_ptr(), nm, batch,
                                           status.data_ptr(), copy_s.cuda_stream,
                                           comp_s.cuda_stream, handles)
    assert rc == 0
    comp_s.synchronize()
    assert int(status.item()) == 0
    assert np.array_equal(pool.cpu().numpy(), exp_pool)
    # spill the same slots back out to other host places: the oracle packs
    # the moves the device count covers; the staging slots past it keep
    # their old bytes, which the host link still carries
    host2 = torch.zeros(host_len, dtype=torch.uint8).pin_memory()
    st2 = torch.full((nm * blk,), 9, dtype=torch.uint8, device="cuda")
    exp_st = np.full(nm * blk, 9, np.uint8)
    ref.pack(exp_pool, g, exp_st, mv[:n_dev])
    exp_host = np.zeros(host_len, np.uint8)
    for m in range(nm):
        exp_host[host_off[m]:host_off[m] + blk] = exp_st[m * blk:(m + 1) * blk]
    rc = cascade.cascade_spill_to_host(pl, st2.data_ptr(), nm, host2.data_ptr(), host_off,
                                       mv_d.data_ptr(), n_d.data_ptr(), nm, batch,
                                       status.data_ptr(), copy_s.cuda_stream,
                                       comp_s.cuda_stream, handles)
    assert rc == 0
    copy_s.synchronize()
    assert np.array_equal(host2.numpy(), exp_host)
    torch.cuda.synchronize()


@pytest.mark.parametrize("layout", ["layer_major", "block_major"])
@pytest.mark.parametrize("chunk", [64, 4096])
@pytest.mark.parametrize("batch", [1, 3, 7, 100])
def test_restore_and_spill(dev, layout, chunk, batch):
    _restore_spill(dev, layout, chunk, batch, seed=batch * 7 + chunk)


@pytest.mark.parametrize("n_dev", [0, 1, 13, 24])
def test_device_count_short_of_the_host_count(dev, n_dev):
    """Batches past the device count copy nothing on the GPU."""
    _restore_spill(dev, "layer_major", 256, 4, nm=25, n_dev=n_dev, seed=40 + n_dev)


@pytest.mark.parametrize("layout", ["layer_major", "block_major"])
def test_real_2mib_blocks(dev, layout):
    """Blocks of the 8B-class geometry: 32 layers x K/V x 32 KiB = 2 MiB."""
    print(f"host tier 2 MiB blocks {layout}", flush=True)
    _restore_spill(dev, layout, 32768, 5, nm=24, nb=48, L=32, seed=3)


def test_host_checks(dev):
    import torch
    from paper_2608_06557_amd import cascade
    g = _geom("layer_major", 8, 2, 64)
    pl = dev.kv_pool_struct(4096, g)
    _, handles = dev.event_handles(1)
    args = dict(staging=4096, staging_slots=4, host_blocks=4096, host_offsets=np.zeros(4),
                moves_dev=4096, n_moves_dev=4096, n_moves=4, batch_moves=2, status_dev=0,
                copy_stream=0, compute_stream=0, events=handles)
    f = cascade.cascade_restore_from_host
    assert f(pl, **dict(args, batch_moves=0)) == cascade.EINVAL
    assert f(pl, **dict(args, n_moves=5)) == cascade.ENOSPC
    assert f(pl, **dict(args, events=[])) == cascade.EINVAL
    assert f(pl, **dict(args, n_moves=0, events=[])) == cascade.OK
