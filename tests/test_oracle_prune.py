"""Pins of the pruned-layer oracle (oracle.prune, paper Sec. 4.3.1 Pruning):
keeping everything changes nothing, a pruned layer and its complement add up
to the full layer, dropping everything leaves the residual stream alone, and
the partial sums of the kept shards of a partition equal the pruned layer
(fp64, 1e-9) -- the sharding and the pruning are independent computations.
"""
import numpy as np
import pytest

import oracle
from oracle.prune import pruned_weights
from tests.common import full_weights, oracle_shard_weights, tiny_workload
from synth.gen import LayerInputs


def setup(seed=901, fracs=(0.25, 0.25, 0.25, 0.25)):
    wl = tiny_workload(seed, 128, 8, 4, 64, 200, fracs, 0, 6, sigma=0.1)
    li = LayerInputs(wl)
    return wl, li


def run(wl, li, w):
    d = wl.dims
    kc, vc = li.kv_context_heads(0, d.n_kv_heads)
    return oracle.decode(w, d.n_heads, d.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base,
                         li.x(0), kc, vc, wl.ctx)


def rel(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


def test_keep_all_is_identity():
    wl, li = setup()
    d = wl.dims
    w = full_weights(li)
    p = pruned_weights(w, d.head_dim, d.n_heads // d.n_kv_heads, np.ones(d.n_kv_heads, bool),
                       np.ones(d.ffn, bool))
    a, b = run(wl, li, w), run(wl, li, p)
    for k in ("p_attn", "p_ffn", "h", "y"):
        assert np.array_equal(a[k], b[k])


def test_complements_add_up():
    wl, li = setup()
    d = wl.dims
    G = d.n_heads // d.n_kv_heads
    w = full_weights(li)
    rng = np.random.default_rng(3)
    kg = rng.random(d.n_kv_heads) < 0.5
    kc = rng.random(d.ffn) < 0.5
    full = run(wl, li, w)
    a = run(wl, li, pruned_weights(w, d.head_dim, G, kg, kc))
    b = run(wl, li, pruned_weights(w, d.head_dim, G, ~kg, ~kc))
    assert rel(a["p_attn"] + b["p_attn"], full["p_attn"]) < 1e-9
    # the FFN input h differs between the three runs (it holds the pruned
    # attention), so the FFN is compared on the full layer's h
    fa, _ = oracle.ffn_sublayer(pruned_weights(w, d.head_dim, G, kg, kc), d.rms_eps, full["h"])
    fb, _ = oracle.ffn_sublayer(pruned_weights(w, d.head_dim, G, ~kg, ~kc), d.rms_eps, full["h"])
    assert rel(fa + fb, full["p_ffn"]) < 1e-9


def test_drop_everything():
    wl, li = setup()
    d = wl.dims
    w = pruned_weights(full_weights(li), d.head_dim, d.n_heads // d.n_kv_heads,
                       np.zeros(d.n_kv_heads, bool), np.zeros(d.ffn, bool))
    r = run(wl, li, w)
    assert not r["p_attn"].any() and not r["p_ffn"].any()
    assert np.array_equal(r["h"], li.x(0).astype(np.float64))
    assert np.array_equal(r["y"], r["h"])


@pytest.mark.parametrize("dropped", [(1,), (0, 3), (2,)])
def test_kept_shards_sum_to_pruned_layer(dropped):
    wl, li = setup()
    d = wl.dims
    G = d.n_heads // d.n_kv_heads
    kg = np.ones(d.n_kv_heads, bool)
    kc = np.ones(d.ffn, bool)
    parts_a, parts_f = [], []
    x = li.x(0)
    kc_all, vc_all = li.kv_context_heads(0, d.n_kv_heads)
    ref_full = run(wl, li, full_weights(li))
    for dev in range(len(wl.fracs)):
        r = oracle.shard_ranges(d.n_heads, d.n_kv_heads, d.ffn, wl.fracs, wl.fracs, dev)
        if dev in dropped:
            kg[r.kv_head_begin:r.kv_head_begin + r.n_kv_heads] = False
            kc[r.col_begin:r.col_begin + r.n_cols] = False
            continue
        sw = oracle_shard_weights(li, r)
        g0, g1 = r.kv_head_begin, r.kv_head_begin + r.n_kv_heads
        o = oracle.decode(sw, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, x,
                          kc_all[g0:g1], vc_all[g0:g1], wl.ctx)
        parts_a.append(o["p_attn"])
        f, _ = oracle.ffn_sublayer(sw, d.rms_eps, ref_full["h"])
        parts_f.append(f)
    pw = pruned_weights(full_weights(li), d.head_dim, G, kg, kc)
    pr = run(wl, li, pw)
    assert rel(np.sum(parts_a, axis=0), pr["p_attn"]) < 1e-9
    fp, _ = oracle.ffn_sublayer(pw, d.rms_eps, ref_full["h"])
    assert rel(np.sum(parts_f, axis=0), fp) < 1e-9
