"""GPU parity of the block-quantised weight shards (paper Sec. 2.2, 4.2.2,
4.3.1 precision heterogeneity and scaling) through the C ABI:

* vt_quantize_rows writes the same code bytes and fp16 scales as the
  oracle's quantiser, bit for bit, on seeded weights and on rows built to hit
  the edges (zero and underflowing blocks, fp16 extremes, exact ties,
  partial last blocks);
* vt_layer_decode_q matches the fp64 oracle run with the dequantised shard
  weights (the values the codes stand for) to the decode bar of
  tests/common.py, fused and staged, on the tiny, 7B and 70B GQA shards and
  on a shard whose column count is not a multiple of the block.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import wquant as W
from paper_2607_07046_amd import voltron as vt
from synth import get
from synth.gen import LayerInputs
from tests.common import assert_close, ffn_at_h16, oracle_qshard_weights, oracle_ranges, tiny_workload
from tests.gpu_common import GpuShard
from tests.test_gpu_decode import RAGGED_H, RAGGED_IDS
from tests.test_gpu_random_shapes import IDS as RANDOM_IDS, SHAPES as RANDOM_SHAPES

pytestmark = pytest.mark.gpu

LEVELS = {"int8": vt.VT_W_INT8, "int4": vt.VT_W_INT4}
BOTH = vt.VT_ATTN | vt.VT_FFN


def gpu_quantize(w16, level):
    rows, cols = w16.shape
    ld = ((cols + 7) // 8) * 8
    src = np.zeros((rows, ld), np.float16)
    src[:, :cols] = w16
    nb = W.n_blocks(cols)
    cb = W.code_bytes_per_row(cols, level)
    ld_codes = cb + 16                       # a spare 16 bytes per row must stay untouched
    t = torch.from_numpy(src.view(np.int16)).cuda()
    codes = torch.full((rows, ld_codes), 0xA5, dtype=torch.uint8, device="cuda")
    scales = torch.full((rows, nb + 1), 0x7E00, dtype=torch.int16, device="cuda")
    vt.vt_quantize_rows(t.data_ptr(), ld, rows, cols, level, codes.data_ptr(), ld_codes,
                        scales.data_ptr(), nb + 1)
    torch.cuda.synchronize()
    c, s = codes.cpu().numpy(), scales.cpu().numpy()
    assert np.all(c[:, cb:] == 0xA5) and np.all(s[:, nb:] == 0x7E00)   # nothing past the blocks
    return c[:, :cb], s[:, :nb].view(np.float16)


def edge_rows(cols, level):
    rng = np.random.default_rng(cols + level)
    Q = W.QMAX[level]
    rows = [np.zeros(cols)]                                        # all zero
    rows.append(np.full(cols, 6e-8))                               # underflowing scale
    rows.append(np.where(np.arange(cols) % 2, 65504.0, -65504.0))  # fp16 extremes
    tie = np.zeros(cols)
    step = 2.0 ** -5
    for b in range(0, cols, 32):                                   # exact ties per block
        tie[b] = Q * step
        tie[b + 1:min(b + 9, cols)] = (np.array([0.5, 1.5, 2.5, -0.5, -1.5, -2.5, 3.5, -3.5])
                                       * step)[:max(0, min(b + 9, cols) - b - 1)]
    rows.append(tie)
    rows.append(rng.standard_normal(cols) * np.exp2(rng.integers(-20, 8, cols)))  # wide range
    return np.array(rows).astype(np.float16)


@pytest.mark.parametrize("level", LEVELS)
@pytest.mark.parametrize("cols", [7, 32, 100, 688, 3302])
def test_quantize_rows_bit_exact(level, cols):
    lv = LEVELS[level]
    rng = np.random.default_rng(40 + cols)
    w = np.concatenate([(rng.standard_normal((61, cols)) * 0.02).astype(np.float16),
                        edge_rows(cols, lv)])
    codes, scales = gpu_quantize(w, lv)
    wc, ws = W.quantize_rows(w, lv)
    assert np.array_equal(scales.view(np.int16), ws.view(np.int16))
    want = W.pack_codes(wc, lv)
    bad = np.argwhere(codes != want)
    assert not len(bad), (bad[:5], codes[tuple(bad[0])], want[tuple(bad[0])])


_cache = {}


def case(wl, level):
    key = (repr(wl), level)  # the whole workload: shapes, partition, context
    if key not in _cache:
        li = LayerInputs(wl)
        r = oracle_ranges(wl)
        w = oracle_qshard_weights(li, r, level)
        kc, vc = li.kv_context_heads(r.kv_head_begin, r.kv_head_begin + r.n_kv_heads)
        d = wl.dims
        x = li.x(0)
        ref = oracle.decode(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, x,
                            kc, vc, wl.ctx, window=d.window)
        ref = ffn_at_h16(w, d.rms_eps, ref)
        _cache[key] = (li, x, ref)
    return _cache[key]


def run(wl, level, phases=BOTH):
    li, x, ref = case(wl, LEVELS[level])
    gs = GpuShard(wl, li=li, prec=LEVELS[level])
    got = gs.decode(x, wl.ctx, phases)
    for k in ("p_attn", "h", "p_ffn", "y"):
        assert_close(got[k], ref[k], f"{wl.key} {level} {k}")
    kc, vc = gs.cache()
    assert gs.kv.len == wl.ctx + 1
    for g in range(kc.shape[0]):
        assert_close(kc[g, wl.ctx].view(np.float16).astype(np.float64), ref["k_new"][g], "key")
        assert_close(vc[g, wl.ctx].view(np.float16).astype(np.float64), ref["v_new"][g], "value")
    return got, ref


@pytest.mark.parametrize("level", LEVELS)
@pytest.mark.parametrize("key", ["tiny", "7b", "70b_gqa"])
def test_decode_q_matches_oracle(key, level):
    run(get(key), level)


@pytest.mark.parametrize("level", LEVELS)
def test_decode_q_staged(level):
    run(get("tiny"), level, BOTH | vt.VT_STAGED)


@pytest.mark.parametrize("level", LEVELS)
def test_decode_q_ragged_columns(level):
    # 1000 FFN columns over 3 devices: 333 on device 1, not a multiple of 32;
    # GQA groups of 2
    wl = tiny_workload(411, 512, 8, 4, 64, 1000, (0.33, 0.34, 0.33), 1, 40)
    run(wl, level)


@pytest.mark.parametrize("level", LEVELS)
@pytest.mark.parametrize("case", RAGGED_H[:2], ids=RAGGED_IDS[:2])
def test_decode_q_ragged_hidden(case, level):
    # hidden a multiple of 8 but not of 32: the last 32-column block of every
    # K = hidden row is partial
    run(tiny_workload(*case, sigma=0.03), level)


@pytest.mark.parametrize("level", LEVELS)
@pytest.mark.parametrize("wl", RANDOM_SHAPES[:4], ids=RANDOM_IDS[:4])
def test_decode_q_random_shapes(wl, level):
    run(wl, level)


@pytest.mark.parametrize("level", LEVELS)
def test_decode_q_sub_layers(level):
    # attention alone, then the FFN alone from the h it wrote
    wl = get("tiny")
    li, x, ref = case(wl, LEVELS[level])
    gs = GpuShard(wl, li=li, prec=LEVELS[level])
    a = gs.decode(x, wl.ctx, vt.VT_ATTN, want_y=False)
    for k in ("p_attn", "h"):
        assert_close(a[k], ref[k], k)
    f = gs.decode(None, None, vt.VT_FFN, h_in=a["h"])
    assert_close(f["p_ffn"], ref["p_ffn"], "p_ffn")
