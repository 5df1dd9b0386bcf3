import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
TESTS = os.path.dirname(os.path.abspath(__file__))
if TESTS not in sys.path:
    sys.path.insert(0, TESTS)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs a real MI355X (gfx950) GPU")


_PROGRESS = os.environ.get("MK_PROGRESS_FILE")


def pytest_runtest_logstart(nodeid, location):
    # On GPU runs, name each test in a file before it starts, so a run that
    # takes the box down still says which case was running.
    if _PROGRESS:
        with open(_PROGRESS, "a") as fh:
            fh.write(f"start {nodeid}\n")
            fh.flush()
            os.fsync(fh.fileno())


def pytest_runtest_logfinish(nodeid, location):
    if _PROGRESS:
        with open(_PROGRESS, "a") as fh:
            fh.write(f"end   {nodeid}\n")
            fh.flush()
