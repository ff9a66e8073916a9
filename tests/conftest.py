import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# Where the GPU parity tests write every error and near-tie count they measured.
PARITY_RECORD = os.environ.get("MOE_PARITY_RECORD", os.path.join(ROOT, "gpurun_out", "parity_record.json"))


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long CPU test")


def pytest_sessionfinish(session, exitstatus):
    parity = sys.modules.get("tests.parity")
    if parity is not None:
        parity.write_record(PARITY_RECORD)
