import os
import sys
import time

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# Progress of GPU test runs also goes to a file under gpurun_out/, so that a
# long test (an oracle replay of a whole full-size trace) keeps showing signs
# of life while pytest holds its output.
PROGRESS = os.path.join(ROOT, "gpurun_out", "test_progress.log")


def progress(msg: str) -> None:
    print(msg, flush=True)
    try:
        os.makedirs(os.path.dirname(PROGRESS), exist_ok=True)
        with open(PROGRESS, "a") as f:
            f.write(f"{time.strftime('%H:%M:%S')} {msg}\n")
    except OSError:
        pass


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def pytest_runtest_logstart(nodeid, location):
    if "gpu" in nodeid or "test_gpu" in nodeid:
        progress(f"start {nodeid}")


def pytest_runtest_logreport(report):
    if report.when == "call" and "test_gpu" in report.nodeid:
        progress(f"{report.outcome} {report.nodeid} {report.duration:.1f} s")
