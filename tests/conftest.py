import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


# Worst errors and exact/tie tallies that the GPU parity tests record
# (tests.parity.record); written to gpurun_out/parity_summary.json when any
# test recorded something.
def pytest_sessionfinish(session, exitstatus):
    from tests import parity
    if parity.SUMMARY:
        import json
        out = os.path.join(ROOT, "gpurun_out")
        os.makedirs(out, exist_ok=True)
        with open(os.path.join(out, "parity_summary.json"), "w") as f:
            json.dump(parity.SUMMARY, f, indent=1, sort_keys=True)
