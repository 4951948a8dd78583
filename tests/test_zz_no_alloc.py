"""cascade_step_noalloc, the step for callers that cannot allocate: its
results equal cascade_step's (with a caller workspace) bit for bit, on
consecutive calls of different sizes that share the library's fixed array,
and a queue over its limit is refused before anything is enqueued."""
import numpy as np
import pytest

from tests import helpers

ARRAYS = ["budget_ns", "action", "queue_tier_out", "tokens_granted", "restore_blocks", "order",
          "alloc_begin", "alloc_count", "admitted", "slot_list", "unpack_moves", "pack_moves",
          "unpack_hazard", "pack_hazard"]


def _same(a, b, label):
    assert a["status"] == b["status"] == 0, (label, a["status"], b["status"])
    for k in ["n_admitted", "n_slot_list", "n_unpack", "n_pack"]:
        assert a[k] == b[k], (label, k)
    for k in ARRAYS:
        x, y = np.asarray(a[k]), np.asarray(b[k])
        assert x.shape == y.shape and np.array_equal(x.view(np.uint8), y.view(np.uint8)), \
            (label, k)


@pytest.mark.gpu
def test_noalloc_equals_workspace_step_on_consecutive_calls():
    import torch
    import paper_2608_06557_amd.synth as synth
    from paper_2608_06557_amd import cascade, device
    assert torch.cuda.is_available()
    cascade.load()
    # the largest queue the array holds, then smaller ones on the same array:
    # multi-launch paths of two tile sizes and the one-workgroup path
    cases = [("config 4, 262144 requests", synth.make_workload(4)),
             ("config 2, 6000 requests", synth.make_workload(2, seed=77, n=6000)),
             ("small, 300 requests", helpers.random_workload(np.random.default_rng(5), 300,
                                                             params=helpers.base_params(
                                                                 token_cap=200)))]
    for label, w in cases:
        print(f"no-alloc step: {label}", flush=True)
        nb = int(w["params"]["num_blocks"])
        a = device.DeviceStep(w, slot_cap=nb, unpack_cap=nb, pack_cap=nb)
        b = device.DeviceStep(w, slot_cap=nb, unpack_cap=nb, pack_cap=nb)
        assert b.run() == 0
        ref_out = b.fetch()
        assert a.run_noalloc() == 0
        got = a.fetch()
        _same(got, ref_out, label)
        # a second call on the same array after other work gives the same
        assert a.run_noalloc() == 0
        _same(a.fetch(), ref_out, label + " (again)")
        del a, b
        torch.cuda.synchronize()


def test_noalloc_refuses_a_queue_over_its_limit():
    """Host-side check, no GPU needed: nothing is enqueued."""
    from paper_2608_06557_amd import cascade
    lib = cascade.load()
    assert cascade.NOALLOC_MAX_REQUESTS == 262144
    rq = cascade.Requests(cascade.NOALLOC_MAX_REQUESTS + 1, *([0] * 10))
    rc = cascade.cascade_step_noalloc(rq, cascade.BlockTable(0, 0), cascade.TierState(0, 0, 0),
                                      cascade.Params(), cascade.Outputs(), 0)
    assert rc == cascade.ENOSPC
    assert lib.cascade_step_noalloc(None, None, None, None, None, None) == cascade.EINVAL
