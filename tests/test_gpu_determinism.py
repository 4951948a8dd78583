"""Repeatability of the kernels that hand results between workgroups
(decoupled look-backs, last-workgroup tickets): the 65536- and
262144-request steps and a full HBM -> DRAM -> NVMe reclamation chain, each
run 1000 times on the same inputs, every output compared bit for bit with
the first run's.  The loop stops at the first difference."""
import numpy as np
import pytest
import torch  # noqa: F401  (imported at collection: the first import is slow)

pytestmark = pytest.mark.gpu
REPS = 1000


@pytest.fixture(scope="module")
def dev():
    import torch
    from paper_2608_06557_amd import cascade, device
    assert torch.cuda.is_available()
    cascade.load()
    return device


def _snapshot(tensors):
    return [t.clone() for t in tensors]


def _same(a, b):
    import torch
    return all(torch.equal(x, y) for x, y in zip(a, b))


@pytest.mark.parametrize("cfg", [2, 4])
def test_step_repeats_bit_for_bit(dev, cfg):
    import torch
    import paper_2608_06557_amd.synth as synth
    w = synth.make_workload(cfg)
    nb = int(w["params"]["num_blocks"])
    d = dev.DeviceStep(w, slot_cap=nb, unpack_cap=nb, pack_cap=nb)
    outs = list(d.out.values()) + [d.slot_list, d.unpack_moves, d.pack_moves, d.unpack_hazard,
                                   d.pack_hazard, d.info]

    def poison():
        # stale results cannot pass, and whole buffers are compared, so a
        # write past a list's count would show too
        for t in outs:
            t.fill_(0x5A if t.dtype == torch.uint8 else -7)

    poison()
    assert d.run() == 0
    first = _snapshot(outs)
    assert int(d.info[0].item()) == 0
    print(f"config {cfg}: {len(w['id'])} requests x {REPS}", flush=True)
    for k in range(REPS):
        poison()
        assert d.run() == 0
        assert _same(outs, first), f"config {cfg}: run {k + 1} differs from the first"


@pytest.mark.parametrize("one_call", [False, True], ids=["per_tier", "chain_call"])
def test_tier_chain_repeats_bit_for_bit(dev, one_call):
    import paper_2608_06557_amd.synth as synth
    w = synth.make_tier_workload(2)
    d = dev.DeviceTiers(w["tables"], w["needs"], w["index_keys"], w["index_masks"])
    run = d.run_chain if one_call else d.run
    keep = _snapshot(d.bh + d.lu + [d.index])
    outs = d.bh + d.lu + [d.index] + d.out + [d.n_out] + d.freed + d.placed

    import torch

    def reset():
        for t, s in zip(d.bh + d.lu + [d.index], keep):
            t.copy_(s)
        for t in d.out + d.freed + d.placed + [d.n_out]:
            t.fill_(0xA5 if t.dtype == torch.uint8 else -3)
        d.status.zero_()

    reset()
    assert run() == 0
    assert int(d.status.item()) == 0
    first = _snapshot(outs)
    print(f"tier chain {w['sizes']} x {REPS} ({'one call' if one_call else 'per tier'})",
          flush=True)
    for k in range(REPS):
        reset()
        assert run() == 0
        assert _same(outs, first), f"tier chain: run {k + 1} differs from the first"
    assert int(d.status.item()) == 0
