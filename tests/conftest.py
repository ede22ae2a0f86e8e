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


def pytest_runtest_logfinish(nodeid, location):
    # every parity test reports its worst element-wise and normwise errors
    # (outside pytest's output capture, like the [start] line)
    from tests import common
    if common.WORST:
        e, ew = common.WORST.get("elem", (0.0, ""))
        n, nw = common.WORST.get("norm", (0.0, ""))
        sys.__stderr__.write(f"[parity] {nodeid}: worst element-wise {e:.3g} ({ew}), "
                             f"normwise {n:.3g} ({nw})\n")
        sys.__stderr__.flush()
        common.WORST.clear()
