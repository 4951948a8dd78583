"""AddressSanitizer + UndefinedBehaviorSanitizer builds of host code (no
GPU): the CPU oracle, run through its pins, and the host side of the GPU
library, run through its host-side argument checks.  Each runs in a child
process with the sanitizer runtime preloaded; any report fails the test.
Device code is built as usual and not instrumented; no kernel is launched."""
import glob
import os
import shutil
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_06557_amd", "csrc")
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _run_child(preload, script, *args):
    env = dict(os.environ, LD_PRELOAD=preload, **SAN_ENV)
    env.pop("PYTHONSTARTUP", None)
    out = subprocess.run([sys.executable, "-c", textwrap.dedent(script), ROOT, *args],
                         capture_output=True, text=True, timeout=600, env=env)
    text = out.stdout + out.stderr
    assert out.returncode == 0, text[-4000:]
    assert "AddressSanitizer" not in text and "runtime error" not in text, text[-4000:]
    return text


def test_oracle_under_asan_and_ubsan(tmp_path):
    libasan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                             text=True).stdout.strip()
    if not os.path.isabs(libasan):
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    so = str(tmp_path / "liboracle_san.so")
    subprocess.run(["gcc", "-std=gnu11", "-O1", "-g", "-fPIC", "-shared",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    "-fno-omit-frame-pointer", "-o", so,
                    os.path.join(ROOT, "oracle", "cascade_ref.c")], check=True)
    text = _run_child(libasan, """
        import sys
        sys.path.insert(0, sys.argv[1])
        import numpy as np
        from oracle import ref
        from tests import test_oracle_pins as pins, test_oracle_bruteforce as bf
        from tests import test_oracle_invariants as inv, test_oracle_prefix as pf
        from tests import test_oracle_reclaim as rc
        checks = [pins.test_worked_example_step, pins.test_second_example_step,
                  pins.test_shared_prefix_example_step, pins.test_max_restorable_brute_force,
                  pins.test_gamma_product_exact_at_domain_edge,
                  lambda: [bf._check_against_definitions(w) for w in bf._cases(100, 8, 7)],
                  lambda: bf.test_shared_prefix_step_matches_definitions(1),
                  inv.test_invariants_on_synthetic_configs, inv.test_empty_queue,
                  inv.test_enospc_reports_required_sizes,
                  lambda: [inv.test_einval(name, m) for name, m in inv.MUTATIONS],
                  pf.test_hand_example, pf.test_empty_index_and_empty_requests,
                  lambda: pf.test_round_trip_from_cached_runs(0),
                  rc.test_hand_example_three_tiers, rc.test_einval_rules_write_nothing,
                  lambda: rc.test_cascade_keeps_index_and_blocks_consistent(0)]
        with ref.library(sys.argv[2]):
            for c in checks:
                c()
        print("sanitized oracle: all checks ran")
        """, so)
    assert "all checks ran" in text


def test_library_host_code_under_asan_and_ubsan(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    rt = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not os.path.exists(hipcc) or not rt:
        pytest.skip("hipcc or clang's AddressSanitizer runtime is not installed")
    from concurrent.futures import ThreadPoolExecutor

    def compile_one(src):
        obj = str(tmp_path / src.replace(".hip", ".o"))
        subprocess.run([hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
                        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                        "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                        "-Xarch_host", "-fno-sanitize-recover=undefined", "-shared-libsan",
                        "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-c",
                        os.path.join(CSRC, src), "-o", obj], check=True, capture_output=True)
        return obj

    with ThreadPoolExecutor(4) as ex:
        objs = list(ex.map(compile_one, ["cascade_step.hip", "cascade_kvcopy.hip",
                                         "cascade_prefix.hip", "cascade_reclaim.hip",
                                         "cascade_hosttier.hip"]))
    so = str(tmp_path / "libcascade_san.so")
    subprocess.run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-shared-libsan",
                    "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                    "-o", so, *objs], check=True, capture_output=True)
    text = _run_child(rt[-1], """
        import sys
        sys.path.insert(0, sys.argv[1])
        from paper_2608_06557_amd import cascade
        cascade.LIB_PATH = sys.argv[2]
        cascade._lib = None
        lib = cascade.load()
        from tests import test_abi as t
        from tests import test_zz_no_alloc as z
        for c in [t.test_workspace_size, t.test_host_checks_return_einval_without_launch,
                  t.test_copy_host_checks, t.test_fused_copy_host_checks,
                  t.test_reclaim_workspace_size, t.test_reclaim_host_checks,
                  t.test_reclaim_chain_host_checks]:
            c(lib)
        z.test_noalloc_refuses_a_queue_over_its_limit()
        for code in range(-6, 2):
            assert cascade.cascade_strerror(code)
        print("sanitized library: all host checks ran")
        """, so)
    assert "all host checks ran" in text
