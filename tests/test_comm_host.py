"""Host side of the partial-sum transmission scaling (paper Sec. 4.3.2):
the library's planner (vt_qplan, C) against the oracle's plan, bit-exact,
and argument validation of the encode/decode entry points (errors are
returned before anything is launched, so no GPU is needed).
"""
import numpy as np
import pytest

from oracle import comm as C
from paper_2607_07046_amd import voltron as vt


@pytest.fixture(scope="module")
def lib():
    return vt.load_library()


@pytest.mark.parametrize("seed", range(12))
def test_plan_matches_oracle(lib, seed):
    rng = np.random.default_rng(100 + seed)
    nb = int(rng.integers(1, 300))
    imp = (rng.integers(0, 9, nb) * rng.choice([1.0, 0.37])).astype(np.float32)  # ties
    budget = int(rng.integers(-10, 64 * nb + 40))
    prec, offs, tot = vt.vt_qplan(imp, budget)
    p0, o0, t0 = C.plan(imp, budget)
    assert np.array_equal(prec, p0.astype(np.uint8))
    assert np.array_equal(offs, o0.astype(np.int32))
    assert tot == t0


def test_plan_validation(lib):
    with pytest.raises(vt.VoltronError) as e:
        vt.vt_qplan(np.array([1.0, np.nan], np.float32), 10)
    assert e.value.status == vt.VT_ERR_ARG
    with pytest.raises(vt.VoltronError) as e:
        vt.vt_qplan(np.zeros(0, np.float32), 10)
    assert e.value.status == vt.VT_ERR_ARG


def test_encode_decode_validation(lib):
    A = 1 << 20
    for n in (0, 31, 48):
        with pytest.raises(vt.VoltronError) as e:
            vt.vt_partial_encode(A, n, A, A, A, 64)
        assert e.value.status == vt.VT_ERR_ARG
    with pytest.raises(vt.VoltronError) as e:
        vt.vt_partial_encode(A + 2, 32, A, A, A, 64)
    assert e.value.status == vt.VT_ERR_ALIGN
    with pytest.raises(vt.VoltronError) as e:
        vt.vt_partial_decode_add(None, 64, 32, A, A, None, A)
    assert e.value.status == vt.VT_ERR_ARG
    with pytest.raises(vt.VoltronError) as e:
        vt.vt_partial_decode_add(A, 1 << 31, 32, A, A, None, A)
    assert e.value.status == vt.VT_ERR_UNSUPPORTED
