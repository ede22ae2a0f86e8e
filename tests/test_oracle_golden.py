"""The oracle still reproduces its stored regression fixture."""
import json
import os

import numpy as np

from tests.golden.make_golden import build

HERE = os.path.dirname(os.path.abspath(__file__))


def test_oracle_reproduces_golden_fixture():
    with open(os.path.join(HERE, "golden", "tiny_layer.json")) as f:
        stored = json.load(f)
    now = build()
    assert now["ranges"] == stored["ranges"]
    for k, v in stored["outputs"].items():
        assert np.max(np.abs(np.array(now["outputs"][k]) - np.array(v))) < 1e-13, k
