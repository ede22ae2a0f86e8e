"""Pins of oracle.comm (transmission-precision scaling of partial sums,
paper Sec. 4.3.2 with the importance-ordered lowering of Sec. 4.2.2).

The plan is checked against what the paper fixes (least lowering that fits
the budget, in ascending importance, FP16 -> INT8 -> INT4 -> pruned) with
hand-worked cases and properties; the quantiser against closed forms of the
block-absmax reading (exact grids, extremes, zero blocks, symmetry, the
half-step error bound, ties to even) and a hand-packed INT4 layout.
"""
import numpy as np
import pytest

from oracle import comm as C


def test_plan_hand_worked():
    imp = [3.0, 1.0, 2.0, 0.0]
    # 4 FP16 blocks = 256 B; budget 200: lower block 3 (228 B) then block 1 (200 B)
    prec, off, tot = C.plan(imp, 200)
    assert list(prec) == [C.FP16, C.INT8, C.FP16, C.INT8]
    assert list(off) == [0, 64, 100, 164] and tot == 200
    # budget 100: all INT8 is 144 B; then blocks 3, 1, 2 to INT4 -> 96 B
    prec, off, tot = C.plan(imp, 100)
    assert list(prec) == [C.INT8, C.INT4, C.INT4, C.INT4]
    assert list(off) == [0, 36, 56, 76] and tot == 96
    # budget 50: all INT4 is 80 B; prune block 3 (60 B) then block 1 (40 B)
    prec, off, tot = C.plan(imp, 50)
    assert list(prec) == [C.INT4, C.PRUNED, C.INT4, C.PRUNED]
    assert list(off) == [0, 20, 20, 40] and tot == 40


def test_plan_extremes_and_ties():
    prec, off, tot = C.plan(np.ones(5), 10 ** 9)
    assert list(prec) == [C.FP16] * 5 and list(off) == [0, 64, 128, 192, 256] and tot == 320
    prec, off, tot = C.plan(np.ones(5), 0)
    assert list(prec) == [C.PRUNED] * 5 and tot == 0
    # equal importance: the lower block index is lowered first
    prec, _, tot = C.plan(np.ones(3), 3 * 64 - 28)
    assert list(prec) == [C.INT8, C.FP16, C.FP16] and tot == 164


@pytest.mark.parametrize("seed", range(8))
def test_plan_properties(seed):
    rng = np.random.default_rng(seed)
    nb = int(rng.integers(1, 40))
    imp = rng.integers(0, 6, nb).astype(np.float32)   # many ties
    budget = int(rng.integers(0, 64 * nb + 10))
    prec, off, tot = C.plan(imp, budget)
    size = np.array([C.BLOCK_BYTES[int(p)] for p in prec])
    assert tot == size.sum() and tot <= max(budget, 0)
    assert np.array_equal(off, np.concatenate([[0], np.cumsum(size)[:-1]]))
    # monotone in importance order: a less important block is never at a
    # higher precision than a more important one
    order = sorted(range(nb), key=lambda b: (imp[b], b))
    lv = [int(prec[b]) for b in order]
    assert all(lv[i] >= lv[i + 1] for i in range(nb - 1))
    # least lowering: undoing the last step (the most important block among
    # those at the deepest level reached) would overflow the budget
    if tot < 64 * nb:
        deepest = max(lv)
        last = max((i for i in range(nb) if lv[i] == deepest))
        b = order[last]
        undone = tot + C.BLOCK_BYTES[deepest - 1] - C.BLOCK_BYTES[deepest]
        assert undone > budget, (b, undone, budget)


def test_quantize_exact_grid_and_extremes():
    k = np.arange(-127, 128, 8)[:32].astype(np.float32)
    k[-1] = 127.0
    x = k / np.float32(8.0)                       # absmax 127/8 -> scale exactly 1/8
    s, c = C.quantize_block(x, C.INT8)
    assert s == np.float32(0.125) and np.array_equal(c, k.astype(np.int64))
    x = np.linspace(-3.0, 5.0, 32).astype(np.float32)
    s, c = C.quantize_block(x, C.INT4)
    assert c.max() == 7 and s == np.float32(np.float32(5.0) / np.float32(7.0))
    s0, c0 = C.quantize_block(np.zeros(32, np.float32), C.INT8)
    assert s0 == 0 and not c0.any()
    s2, c2 = C.quantize_block(-x, C.INT4)
    assert s2 == s and np.array_equal(c2, -c)


def test_quantize_ties_round_to_even():
    x = np.zeros(32, np.float32)
    x[0] = 127.0                                   # scale 1 exactly
    x[1:7] = [2.5, 3.5, -2.5, -3.5, 0.5, 1.5]
    s, c = C.quantize_block(x, C.INT8)
    assert s == 1.0 and list(c[:7]) == [127, 2, 4, -2, -4, 0, 2]


@pytest.mark.parametrize("level", [C.INT8, C.INT4])
def test_quantize_error_bound(level):
    rng = np.random.default_rng(level)
    for _ in range(50):
        x = (rng.standard_normal(32) * 10 ** rng.uniform(-3, 3)).astype(np.float16).astype(np.float32)
        s, c = C.quantize_block(x, level)
        err = np.abs(x.astype(np.float64) - c * np.float64(s))
        assert np.all(err <= np.float64(s) * (0.5 + 1e-6)), err.max() / s
        assert np.all(np.abs(c) <= C.QMAX[level])


def test_encode_layout_by_hand():
    p = np.zeros(64, np.float16)
    p[32:36] = [7.0, -7.0, 1.0, -1.0]              # block 1: absmax 7 -> INT4 scale 1
    prec, off = np.array([C.FP16, C.INT4]), np.array([0, 64])
    msg = C.encode(p, prec, off, 84)
    assert msg[:64].tobytes() == p[:32].tobytes()
    assert np.frombuffer(msg[64:68].tobytes(), np.float32)[0] == 1.0
    # codes 7, -7 -> nibbles 0x7, 0x9 ; 1, -1 -> 0x1, 0xF
    assert msg[68] == 0x97 and msg[69] == 0xF1 and not msg[70:84].any()
    back = C.decode(msg, prec, off, 64)
    assert np.array_equal(back, p.astype(np.float64))


def test_round_trip_fp16_and_pruned():
    rng = np.random.default_rng(3)
    p = rng.standard_normal(96).astype(np.float16)
    prec = np.array([C.FP16, C.PRUNED, C.INT8])
    off = np.array([0, 64, 64])
    back = C.decode(C.encode(p, prec, off, 100), prec, off, 96)
    assert np.array_equal(back[:32], p[:32].astype(np.float64))
    assert not back[32:64].any()
    x = p[64:].astype(np.float32)
    s, _ = C.quantize_block(x, C.INT8)
    assert np.all(np.abs(back[64:] - x) <= s * 0.5 + 1e-7)
