"""GPU parity of the prefill chunk (vt_layer_prefill_chunk, MFMA path)
against the fp64 oracle, through the C ABI.

Same bar as decode (per-row element-wise relative error <= 2e-2 with the
denominator floored at 0.2 of the row's RMS, normwise <= 1.5e-3; the FFN
outputs against the oracle's FFN at fp16(h)); the appended K/V of every chunk token lands in
its slot and every other cache byte is unchanged.
"""
import numpy as np
import pytest

import oracle
from paper_2607_07046_amd import voltron as vt
from synth import get
from synth.gen import LayerInputs
from tests.common import (assert_close, ffn_at_h16, max_rel_err, norm_rel_err, oracle_ranges,
                          oracle_shard_weights, tiny_workload)
from tests.gpu_common import GpuShard

pytestmark = pytest.mark.gpu
BOTH = vt.VT_ATTN | vt.VT_FFN


def run_case(wl, T, li=None, check_kv=True):
    li = li or LayerInputs(wl)
    d = wl.dims
    r = oracle_ranges(wl)
    w = oracle_shard_weights(li, r)
    kc, vc = li.kv_context_heads(r.kv_head_begin, r.kv_head_begin + r.n_kv_heads)
    X = li.x_chunk(T)
    pa, pf = li.peer("attn", rows=T), li.peer("ffn", rows=T)
    ref = oracle.prefill(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, X, kc,
                         vc, wl.ctx, pa, pf)
    ref = ffn_at_h16(w, d.rms_eps, ref, pf)
    gs = GpuShard(wl, li=li, capacity=wl.ctx + T + 3, max_tokens=T)
    k0, v0 = gs.cache()
    got = gs.prefill(X, wl.ctx, BOTH, peer_attn=pa, peer_ffn=pf)
    errs = {k: (max_rel_err(got[k], ref[k]), norm_rel_err(got[k], ref[k]))
            for k in ("p_attn", "h", "p_ffn", "y")}
    print(wl.key, T, errs)
    for k in ("p_attn", "h", "p_ffn", "y"):
        assert_close(got[k], ref[k], k)
    # the decode kernel's synchronisation words share the workspace
    assert not gs.sync_words().any()
    if check_kv:
        kc1, vc1 = gs.cache()
        assert gs.kv.len == wl.ctx + T
        rng = slice(wl.ctx, wl.ctx + T)
        mask = np.ones(kc1.shape[1], bool)
        mask[rng] = False
        assert np.array_equal(kc1[:, mask], k0[:, mask])
        assert np.array_equal(vc1[:, mask], v0[:, mask])
        kn = kc1[:, rng].view(np.float16).astype(np.float64)     # [nkv, T, d]
        vn = vc1[:, rng].view(np.float16).astype(np.float64)
        assert_close(np.transpose(kn, (1, 0, 2)).reshape(T, -1), ref["k_new"].reshape(T, -1),
                     "appended keys")
        assert_close(np.transpose(vn, (1, 0, 2)).reshape(T, -1), ref["v_new"].reshape(T, -1),
                     "appended values")
    return gs, li


def test_prefill_7b_chunk_full_size():
    """256 tokens at positions 768..1023 through the 50% shard of the 7B layer."""
    wl = get("7b_prefill")
    run_case(wl, wl.chunk)


CASES = [
    # seed, hidden, heads, kv, d, ffn, fracs, device, ctx, T
    (301, 512, 8, 8, 64, 1000, (0.5, 0.5), 0, 0, 1),        # empty cache, one token
    (302, 512, 8, 2, 64, 1000, (0.5, 0.5), 1, 7, 5),        # GQA group 4, ragged everything
    (303, 1024, 8, 4, 128, 1501, (0.6, 0.4), 0, 40, 70),    # d 128, odd FFN width, 3 query blocks
    (304, 768, 12, 12, 64, 2000, (0.3, 0.7), 1, 100, 129),  # M > one 128-row tile, 5 query blocks
]


@pytest.mark.parametrize("case", CASES, ids=[str(c[0]) for c in CASES])
def test_prefill_ragged_shapes(case):
    seed, H, nh, nkv, d, F, fr, dev, ctx, T = case
    wl = tiny_workload(seed, H, nh, nkv, d, F, fr, dev, ctx, sigma=0.03, chunk=T)
    run_case(wl, T)


def test_prefill_then_decode_continues_the_cache():
    wl = tiny_workload(305, 512, 8, 4, 64, 800, (0.5, 0.5), 0, 20, sigma=0.03, chunk=9)
    li = LayerInputs(wl)
    gs, _ = run_case(wl, 9, li)
    d = wl.dims
    r = oracle_ranges(wl)
    w = oracle_shard_weights(li, r)
    kc, vc = li.kv_context_heads(r.kv_head_begin, r.kv_head_begin + r.n_kv_heads)
    X = li.x_chunk(9)
    pre = oracle.prefill(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, X, kc,
                         vc, wl.ctx)
    kc2, vc2 = oracle.append_kv(kc, vc, pre["k_new"], pre["v_new"], wl.ctx)
    x = li.x(77)
    ref = oracle.decode(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, x, kc2,
                        vc2, wl.ctx + 9)
    ref = ffn_at_h16(w, d.rms_eps, ref)
    got = gs.decode(x, wl.ctx + 9, BOTH)
    for k in ("p_attn", "h", "p_ffn", "y"):
        assert_close(got[k], ref[k], k)


def test_prefill_rejects_bad_positions():
    wl = tiny_workload(306, 512, 8, 8, 64, 600, (0.5, 0.5), 0, 4, chunk=3)
    li = LayerInputs(wl)
    gs = GpuShard(wl, li=li, capacity=8, max_tokens=8)
    X = li.x_chunk(3)
    with pytest.raises(vt.VoltronError) as e:
        gs.prefill(X, 3)
    assert e.value.status == vt.VT_ERR_POS
    with pytest.raises(vt.VoltronError) as e:
        gs.prefill(li.x_chunk(5), 4)
    assert e.value.status == vt.VT_ERR_KV_FULL
    assert gs.kv.len == 4
