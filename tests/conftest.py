import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_sessionfinish(session, exitstatus):
    # Per-case parity margins (tests/parity_util.py) as a Markdown table, when
    # NORMPRE_PARITY_LOG names the output file.
    path = os.environ.get("NORMPRE_PARITY_LOG")
    mod = sys.modules.get("parity_util")
    if path and mod is not None and mod.RECORDS:
        mod.write_markdown(path)
