"""Replay one saved scheduling-step input (an .npz written by
``synth.save_workload``, e.g. by a failing GPU parity test) through the GPU
library and the CPU oracle and report where they differ.

    python -m tests.replay_step path/to/step.npz

Test infrastructure: it runs the oracle next to the library."""
from __future__ import annotations

import sys

import numpy as np


def compare(w: dict) -> list[str]:
    """Names of the outputs on which the GPU step and the oracle differ."""
    import torch
    from oracle import ref
    from paper_2608_06557_amd import cascade, device
    assert torch.cuda.is_available(), "replay needs a ROCm GPU"
    cascade.load()
    nb = int(w["params"]["num_blocks"])
    d = device.DeviceStep(w, slot_cap=nb, unpack_cap=nb, pack_cap=nb)
    rc = d.run()
    if rc != 0:
        return [f"host return code {rc}"]
    g = d.fetch()
    o = ref.step(w, slot_cap=nb, unpack_cap=nb, pack_cap=nb)
    diff = []
    if g["status"] != o["rc"]:
        diff.append(f"status gpu {g['status']} oracle {o['rc']}")
        return diff
    for k in ["n_admitted", "n_slot_list", "n_unpack", "n_pack"]:
        if g[k] != o[k]:
            diff.append(f"{k} gpu {g[k]} oracle {o[k]}")
    if o["rc"] != 0:
        return diff
    keys = ["budget_ns", "action", "queue_tier_out", "tokens_granted", "restore_blocks", "order",
            "alloc_begin", "alloc_count", "admitted", "slot_list", "unpack_moves", "pack_moves",
            "unpack_hazard", "pack_hazard"] + (["share_leader"] if "share_leader" in o else [])
    for k in keys:
        a, b = np.asarray(g[k]), np.asarray(o[k])
        if a.shape != b.shape or not np.array_equal(a.view(np.uint8), b.view(np.uint8)):
            diff.append(k)
    return diff


def main(argv: list[str]) -> int:
    import paper_2608_06557_amd.synth as synth
    if len(argv) != 2:
        print(__doc__, file=sys.stderr)
        return 2
    w = synth.load_workload(argv[1])
    diff = compare(w)
    print(f"{argv[1]}: {len(w['id'])} requests, " +
          ("GPU and oracle agree" if not diff else "differ in " + ", ".join(diff)))
    return 1 if diff else 0


if __name__ == "__main__":
    sys.exit(main(sys.argv))
