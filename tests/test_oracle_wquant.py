"""Pins of the oracle's block quantisation of weight shards (oracle.wquant),
against what the definition and the arithmetic fix rather than a re-typing
of it: weights already on a quantisation grid come back exactly with their
grid step as the scale, the reconstruction error of any weight is at most
half a step, the largest magnitude of a block maps to +-Q, the map is odd
and scale-equivariant, exact ties round to the even code, zero and
underflowing blocks give zero, and packing is a bijection with the stated
nibble order.
"""
import numpy as np
import pytest

from oracle import wquant as W

LEVELS = [W.INT8, W.INT4]


def grid_matrix(rng, rows, cols, level, exps):
    """Weights k * 2^-e with integer |k| <= Q and a +-Q in every block."""
    Q = W.QMAX[level]
    k = rng.integers(-Q, Q + 1, size=(rows, cols))
    nb = W.n_blocks(cols)
    for r in range(rows):
        for b in range(nb):
            c = b * W.BLOCK + rng.integers(0, min(W.BLOCK, cols - b * W.BLOCK))
            k[r, c] = Q if rng.random() < 0.5 else -Q
    e = np.repeat(exps[:, :, None], W.BLOCK, axis=2).reshape(rows, nb * W.BLOCK)[:, :cols]
    return (k * np.exp2(-e.astype(np.float64))).astype(np.float16), k, exps


@pytest.mark.parametrize("level", LEVELS)
@pytest.mark.parametrize("cols", [32, 100, 256, 7])
def test_grid_weights_are_exact(level, cols):
    rng = np.random.default_rng(11 + cols + level)
    rows = 5
    exps = rng.integers(2, 9, size=(rows, W.n_blocks(cols)))
    w, k, _ = grid_matrix(rng, rows, cols, level, exps)
    assert np.array_equal(w.astype(np.float64) / np.exp2(-np.repeat(exps, W.BLOCK, 1)[:, :cols]), k)
    codes, scales = W.quantize_rows(w, level)
    assert np.array_equal(scales.astype(np.float64), np.exp2(-exps.astype(np.float64)))
    assert np.array_equal(codes[:, :cols], k)
    assert not codes[:, cols:].any()                      # padded tail
    assert np.array_equal(W.dequantize(codes, scales, cols), w.astype(np.float64))


@pytest.mark.parametrize("level", LEVELS)
def test_error_at_most_half_a_step(level):
    rng = np.random.default_rng(3 + level)
    w = (rng.standard_normal((64, 333)) * 0.02).astype(np.float16)
    codes, scales = W.quantize_rows(w, level)
    deq = W.dequantize(codes, scales, 333)
    step = np.repeat(scales.astype(np.float64), W.BLOCK, axis=1)[:, :333]
    assert np.all(np.abs(deq - w.astype(np.float64)) <= step * (0.5 + 1e-4))
    # the block's largest magnitude lands on +-Q
    Q = W.QMAX[level]
    assert np.all(np.max(np.abs(codes.reshape(64, -1, W.BLOCK)), axis=2) == Q)
    assert np.all(np.abs(codes) <= Q)


@pytest.mark.parametrize("level", LEVELS)
def test_odd_and_scale_equivariant(level):
    rng = np.random.default_rng(17 + level)
    w = (rng.standard_normal((8, 96)) * 0.05).astype(np.float16)
    c, s = W.quantize_rows(w, level)
    cn, sn = W.quantize_rows(-w, level)
    assert np.array_equal(cn, -c) and np.array_equal(sn, s)
    for m in (-3, 4):
        c2, s2 = W.quantize_rows((w.astype(np.float64) * 2.0 ** m).astype(np.float16), level)
        assert np.array_equal(c2, c)
        assert np.array_equal(s2.astype(np.float64), s.astype(np.float64) * 2.0 ** m)


@pytest.mark.parametrize("level", LEVELS)
def test_ties_round_to_even(level):
    Q = W.QMAX[level]
    step = 2.0 ** -6
    row = np.zeros(32)
    row[0] = Q * step                      # sets the scale to exactly step
    ties = [0.5, 1.5, 2.5, -0.5, -1.5, -2.5, 3.5, -3.5]
    row[1:1 + len(ties)] = np.array(ties) * step
    codes, scales = W.quantize_rows(row[None].astype(np.float16), level)
    assert scales[0, 0] == np.float16(step)
    assert list(codes[0, 1:1 + len(ties)]) == [0, 2, 2, 0, -2, -2, 4, -4]


@pytest.mark.parametrize("level", LEVELS)
def test_zero_and_underflowing_blocks(level):
    w = np.zeros((2, 64), np.float16)
    w[1, 32:] = np.float16(6e-8)             # the smallest subnormal: absmax / Q underflows
    codes, scales = W.quantize_rows(w, level)
    assert not codes.any() and not scales.astype(np.float64).any()
    assert not W.dequantize(codes, scales, 64).any()


@pytest.mark.parametrize("level", LEVELS)
def test_packing(level):
    rng = np.random.default_rng(5 + level)
    Q = W.QMAX[level]
    codes = rng.integers(-Q, Q + 1, size=(6, 96))
    packed = W.pack_codes(codes, level)
    assert packed.shape == (6, W.code_bytes_per_row(96, level))
    assert np.array_equal(W.unpack_codes(packed, level), codes)
    # one non-zero code per row: it lands in byte j (INT8), or (INT4) column
    # 8g + i in the low nibble of byte 4g + i and column 8g + 4 + i in its
    # high nibble; every other nibble is the zero code
    one = np.zeros((2, 64), np.int64)
    one[0, 10], one[1, 13] = -3, 5          # 10 = 8 + 2 (low of byte 6), 13 = 8 + 4 + 1 (high of byte 5)
    p = W.pack_codes(one, level)
    if level == W.INT8:
        assert p[0, 10] == 253 and p[1, 13] == 5 and np.count_nonzero(p) == 2
    else:
        assert p[0, 6] == 0x80 | 5 and p[1, 5] == (13 << 4) | 8
        assert np.all(np.delete(p[0], 6) == 0x88) and np.all(np.delete(p[1], 5) == 0x88)
