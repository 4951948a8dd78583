"""Resource use of the library's kernels (no GPU), read from the compiler's
resource-usage remarks of a gfx950 build: the HBM-bound copy kernels must
keep the full 8 waves per SIMD, since every wave in flight holds part of the
bytes the copy needs to cover HBM latency; the latency-bound kernels must not
use scratch memory."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2608_06557_amd", "csrc", "cascade_kvcopy.hip")


@pytest.mark.skipif(shutil.which("hipcc") is None, reason="hipcc not installed")
def test_copy_kernels_keep_full_occupancy(tmp_path):
    cmd = ["hipcc", "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), "-c", SRC, "-o", str(tmp_path / "k.o"),
           "-Rpass-analysis=kernel-resource-usage"]
    out = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert out.returncode == 0, out.stderr[-2000:]
    occ = {}
    name = None
    for line in out.stderr.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
        m = re.search(r"Occupancy \[waves/SIMD\]: (\d+)", line)
        if m and name:
            occ[name] = int(m.group(1))
    kernels = {k: v for k, v in occ.items() if "kvcopy_kernel" in k or "kvmove_kernel" in k}
    # pack and unpack (kvcopy) and the fused launch (kvmove), each in four
    # unit shapes: whole chunks, and groups of 8, 4 or 2 chunks
    assert len(kernels) == 12, occ
    assert all(v == 8 for v in kernels.values()), kernels


def _resource_remarks(src, tmp_path):
    cmd = ["hipcc", "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.dirname(src), "-c", src,
           "-o", str(tmp_path / "k.o"), "-Rpass-analysis=kernel-resource-usage"]
    out = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert out.returncode == 0, out.stderr[-2000:]
    scratch = {}
    name = None
    for line in out.stderr.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and name:
            scratch[name] = int(m.group(1))
    return scratch


@pytest.mark.skipif(shutil.which("hipcc") is None, reason="hipcc not installed")
@pytest.mark.parametrize("src", ["cascade_step.hip", "cascade_reclaim.hip", "cascade_prefix.hip"])
def test_latency_bound_kernels_use_no_scratch(src, tmp_path):
    """The step's kernels run on dependent round trips: a private array or
    a spill placed in scratch memory adds a round trip of its own (as a
    non-inlined device function or an array of HIP vector types can)."""
    scratch = _resource_remarks(os.path.join(ROOT, "paper_2608_06557_amd", "csrc", src), tmp_path)
    assert scratch, "no resource remarks"
    assert all(v == 0 for v in scratch.values()), {k: v for k, v in scratch.items() if v}
