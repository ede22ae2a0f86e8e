"""Pins of sliding-window attention in the oracle (window > 0: a token
attends to the last ``window`` positions; the local layers of the gemma
models in the paper's Table 3): a window at least the context long changes
nothing, a window of one gives each head its own token's value exactly,
keys outside the window have no effect at all, and the vectorised oracle
equals the independent scalar brute force for windows shorter than the
context (decode and a prefill chunk).
"""
import numpy as np
import pytest

import oracle
from oracle.brute import brute_layer
from tests.common import full_weights, tiny_workload
from synth.gen import LayerInputs


def setup(ctx=12):
    wl = tiny_workload(951, 32, 4, 2, 64, 48, (1.0,), 0, ctx, sigma=0.2)
    return wl, LayerInputs(wl)


def dec(wl, li, window, kc=None, vc=None, x=None):
    d = wl.dims
    k0, v0 = li.kv_context_heads(0, d.n_kv_heads)
    return oracle.decode(full_weights(li), d.n_heads, d.n_kv_heads, d.head_dim, d.rms_eps,
                         d.rope_base, li.x(0) if x is None else x, k0 if kc is None else kc,
                         v0 if vc is None else vc, wl.ctx, window=window)


def test_long_window_is_full_attention():
    wl, li = setup()
    a, b = dec(wl, li, 0), dec(wl, li, wl.ctx + 1)
    for k in ("p_attn", "h", "p_ffn", "y"):
        assert np.array_equal(a[k], b[k])


def test_window_of_one_is_own_value():
    wl, li = setup()
    d = wl.dims
    r = dec(wl, li, 1)
    G = d.n_heads // d.n_kv_heads
    o = np.concatenate([r["v_new"][j // G] for j in range(d.n_heads)])
    want = o @ np.asarray(full_weights(li).wo, np.float64).T
    assert np.max(np.abs(r["p_attn"] - want)) <= 1e-12 * np.max(np.abs(want))


def test_keys_outside_window_do_not_matter():
    wl, li = setup()
    d = wl.dims
    k0, v0 = li.kv_context_heads(0, d.n_kv_heads)
    W = 5
    k1, v1 = k0.copy(), v0.copy()
    k1[:, :wl.ctx - W + 1] *= -3          # positions before ctx - W + 1 are outside
    v1[:, :wl.ctx - W + 1] += 1
    a, b = dec(wl, li, W, k0, v0), dec(wl, li, W, k1, v1)
    assert np.array_equal(a["p_attn"], b["p_attn"])
    c = dec(wl, li, W + 1, k1, v1)        # one more position: it now matters
    assert not np.array_equal(a["p_attn"], c["p_attn"])


@pytest.mark.parametrize("window", [2, 5, 9])
def test_matches_brute_force(window):
    wl, li = setup(ctx=10)
    d = wl.dims
    k0, v0 = li.kv_context_heads(0, d.n_kv_heads)
    w = full_weights(li)
    X = np.stack([li.x(t) for t in range(3)])
    ref = brute_layer(w, d.n_heads, d.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, X,
                      k0, v0, wl.ctx, window=window)
    got = oracle.prefill(w, d.n_heads, d.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, X,
                         k0, v0, wl.ctx, window=window)
    for k in ("p_attn", "h", "p_ffn", "y"):
        r = np.asarray(ref[k])
        assert np.max(np.abs(got[k] - r)) <= 1e-12 * max(1.0, np.max(np.abs(r))), k
