import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def pytest_runtest_logstart(nodeid, location):
    # Name each test on the real stderr before it runs, so a GPU run that dies
    # mid-test still shows which case it was in.
    sys.__stderr__.write(f"[start] {nodeid}\n")
    sys.__stderr__.flush()
