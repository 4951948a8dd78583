"""Saving a step input to .npz and loading it back gives the same oracle
step (no GPU); the replay tool's CLI refuses a missing argument."""
import numpy as np

from oracle import ref
from tests import helpers


def test_save_load_round_trip(tmp_path):
    import paper_2608_06557_amd.synth as synth
    for w in [synth.make_workload(0), synth.make_workload(3, n=3000, prefix_groups=True),
              helpers.random_workload(np.random.default_rng(4), 37)]:
        path = str(tmp_path / "step.npz")
        synth.save_workload(w, path)
        v = synth.load_workload(path)
        assert v["params"] == w["params"]
        for k in ["id", "arrival_ns", "n_in", "row_offsets", "slots", "free_slots"]:
            assert np.array_equal(v[k], w[k]) and v[k].dtype == np.asarray(w[k]).dtype
        a, b = ref.step(w), ref.step(v)
        for k in ["order", "action", "budget_ns", "admitted", "slot_list"]:
            assert np.array_equal(a[k], b[k]), k
        assert ("prefix_group" in v) == ("prefix_group" in w)


def test_replay_cli_usage():
    from tests import replay_step
    assert replay_step.main(["replay_step"]) == 2
