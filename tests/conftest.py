import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_runtest_setup(item):
    mod = getattr(item, "module", None)
    last = getattr(mod, "LAST_WORKLOAD", None)
    if isinstance(last, dict):
        last.clear()


def pytest_runtest_makereport(item, call):
    """A failing parity test leaves its step input behind as an .npz (under
    $CASCADE_FAILED_STEPS, default failed_steps/ at the repository root) for
    replay."""
    if call.when != "call" or call.excinfo is None:
        return
    last = getattr(getattr(item, "module", None), "LAST_WORKLOAD", None)
    if not isinstance(last, dict) or "w" not in last:
        return
    import re
    import paper_2608_06557_amd.synth as synth
    out = os.environ.get("CASCADE_FAILED_STEPS", os.path.join(ROOT, "failed_steps"))
    try:
        os.makedirs(out, exist_ok=True)
        path = os.path.join(out, re.sub(r"[^\w.-]+", "_", item.nodeid) + ".npz")
        synth.save_workload(last["w"], path)
        print(f"\nfailing step input saved to {path}", flush=True)
    except OSError:
        pass
