"""Planted mistakes in the oracle must be caught by its pins.

Each case rewrites one line of the oracle's source on the CPU (a flipped
sign, a wrong index, a dropped term, a wrong scale), re-executes the module
into a private namespace, and checks that the brute-force or torch-library
pin then fails. This shows the pins are sensitive to the plausible slips.
"""
import inspect
import types

import numpy as np
import pytest

import oracle.layer as layer_mod
from oracle.brute import brute_layer
from synth.gen import LayerInputs
from tests.common import oracle_ranges, oracle_shard_weights, tiny_workload
from tests.test_oracle_pins import torch_layer

MUTATIONS = [
    ("rope sign", "out[..., 0::2] = a * c - b * s", "out[..., 0::2] = a * c + b * s"),
    ("rope pairing", "a, b = z[..., 0::2], z[..., 1::2]",
     "a, b = z[..., :z.shape[-1] // 2], z[..., z.shape[-1] // 2:]"),
    ("rope frequency", "theta = np.power(float(base), -2.0 * i / d)",
     "theta = np.power(float(base), -1.0 * i / d)"),
    ("gqa index", "g = j // G", "g = j % n_kv"),
    ("score scale", "a = softmax(K @ q / np.sqrt(q.shape[-1]))",
     "a = softmax(K @ q / q.shape[-1])"),
    ("residual", "h = X + p_attn + (0.0 if peer is None else _f64(peer))",
     "h = p_attn + (0.0 if peer is None else _f64(peer))"),
    ("rmsnorm eps", "return x / np.sqrt(ms + eps) * _f64(g)",
     "return x / np.sqrt(ms + 1.0) * _f64(g)"),
    ("silu", "return z / (1.0 + np.exp(-z))", "return 1.0 / (1.0 + np.exp(-z))"),
    ("swiglu operands", "m = silu(Wn @ _f64(w.wg).T) * (Wn @ _f64(w.wu).T)",
     "m = silu(Wn @ _f64(w.wu).T) * (Wn @ _f64(w.wg).T)"),
    ("causal length", "L = pos0 + t + 1", "L = pos0 + t"),
    ("cache append", "return np.concatenate([kc, kn], axis=1), np.concatenate([vc, vn], axis=1)",
     "return np.concatenate([kc, kn], axis=1), np.concatenate([vc, kn], axis=1)"),
]


def _mutant(old, new):
    src = inspect.getsource(layer_mod)
    assert src.count(old) == 1, f"mutation anchor not found exactly once: {old!r}"
    mod = types.ModuleType("oracle_layer_mutant")
    exec(compile(src.replace(old, new), "<mutant>", "exec"), mod.__dict__)
    return mod


def _caught(mod, wl, use_torch):
    li = LayerInputs(wl)
    r = oracle_ranges(wl)
    w = oracle_shard_weights(li, r)
    d = wl.dims
    kc, vc = li.kv_context_heads(r.kv_head_begin, r.kv_head_begin + r.n_kv_heads)
    T = wl.chunk or 1
    X = li.x_chunk(T) if wl.chunk else li.x(0)[None]
    try:
        o = mod.prefill(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, X,
                        kc, vc, wl.ctx)
    except Exception:
        return True
    if use_torch:
        ref = torch_layer(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base,
                          X, kc, vc, wl.ctx)
    else:
        ref = brute_layer(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base,
                          X, kc, vc, wl.ctx)
    for k in ("p_attn", "y"):
        a, b = np.asarray(o[k]), np.asarray(ref[k])
        if a.shape != b.shape or np.max(np.abs(a - b)) > 1e-9 * (1 + np.max(np.abs(b))):
            return True
    return False


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_is_caught(name, old, new):
    mod = _mutant(old, new)
    # GQA (group 2), a 3-token chunk after 4 cached positions, full layer.
    wl = tiny_workload(130, 32, 4, 2, 8, 20, (1.0,), 0, 4, chunk=3)
    assert _caught(mod, wl, use_torch=False), f"brute force missed: {name}"
    assert _caught(mod, wl, use_torch=True), f"torch cross-check missed: {name}"


def test_unmutated_oracle_passes_both():
    mod = _mutant("L = pos0 + t + 1", "L = pos0 + t + 1")
    wl = tiny_workload(130, 32, 4, 2, 8, 20, (1.0,), 0, 4, chunk=3)
    assert not _caught(mod, wl, use_torch=False)
    assert not _caught(mod, wl, use_torch=True)
