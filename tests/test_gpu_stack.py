"""GPU parity of decode through the 40-layer 13B-shaped stack (40% shard:
16 of 40 heads, 5530 of 13824 FFN columns, cache starting at 2048
positions), against the fp64 oracle.

Chain: layer l's input for token t is layer l-1's output y of token t, with
the other devices' partial sums taken as zero. The chain's inputs at every
layer come from the oracle's own fp64 chain (tests/golden/make_stack_golden.py,
which calls only ``oracle/``), rounded to fp16, the precision of the layer
interface.

* Every layer, teacher-forced: each of the 40 layers is fed the chain's
  inputs of the first four tokens (positions 2048..2051) and must match the
  oracle, evaluated here on exactly those inputs, to the single-layer bar
  (tests/common.py) on full vectors: p_attn, h, p_ffn, y and the appended
  keys and values.
* Layers 20 and 39, teacher-forced over all 64 tokens (positions
  2048..2111): full vectors of every token at the same bar.
* Free-running (the whole stack, 2560 vt_layer_decode calls, each layer's y
  fed to the next): properties bind (finite outputs, h = x + p_attn and
  y = h + p_ffn within fp16 rounding, each layer's cache advanced by exactly
  64 tokens); the drift from the exact chain is printed next to the drift
  that fp16 rounding alone produces in the stored model. A 40-layer chain of
  random layers amplifies the rounding of every fp16 interface, so no
  implementation with fp16 layer outputs can hold its deep layers to 2e-2;
  parity is bound by the teacher-forced tests above.
"""
import os
import time

import numpy as np
import pytest

import oracle
from synth import get
from synth.gen import LayerInputs
from tests.common import assert_close, ffn_at_h16, oracle_ranges, oracle_shard_weights
from tests.golden.make_stack_golden import KEYS, sample_index
from tests.gpu_common import GpuShard

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "stack_13b.npz")
GROUPS = 5  # the 40 layers in groups of 8, one test each


def check_residuals(x, out):
    assert np.all(np.isfinite(np.stack([out[k] for k in KEYS])))
    assert np.max(np.abs(out["h"] - (x + out["p_attn"]))) <= 1e-3 * (np.max(np.abs(out["h"])) + 1)
    assert np.max(np.abs(out["y"] - (out["h"] + out["p_ffn"]))) <= \
        1e-3 * (np.max(np.abs(out["y"])) + 1)


def teacher_forced(wl, layer, X):
    """Decode the fp16 rows X (tokens 0.. at positions ctx..) through a fresh
    shard of ``layer`` and compare every output with the oracle on X."""
    d = wl.dims
    T = X.shape[0]
    li = LayerInputs(wl, layer)
    li.full("wo")  # drawn once, kept for the packing and the oracle's slices
    li.full("wd")
    r = oracle_ranges(wl)
    w = oracle_shard_weights(li, r)
    kc, vc = li.kv_context_heads(r.kv_head_begin, r.kv_head_begin + r.n_kv_heads)
    gs = GpuShard(wl, layer=layer, li=li, capacity=wl.ctx + T)
    outs = []
    for t in range(T):
        x = X[t].astype(np.float64)
        out = gs.decode(x, wl.ctx + t)
        check_residuals(x, out)
        outs.append(out)
    assert gs.kv.len == wl.ctx + T
    kc1, vc1 = gs.cache()
    del gs
    ref = oracle.prefill(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base,
                         X.astype(np.float64), kc, vc, wl.ctx)
    ref = ffn_at_h16(w, d.rms_eps, ref)
    worst = {}
    for k in KEYS:
        got = np.stack([o[k] for o in outs])
        worst[k] = assert_close(got, ref[k], f"layer {layer} {k}")
    kn = kc1[:, wl.ctx:wl.ctx + T].view(np.float16).astype(np.float64)   # [nkv, T, d]
    vn = vc1[:, wl.ctx:wl.ctx + T].view(np.float16).astype(np.float64)
    worst["k_new"] = assert_close(np.transpose(kn, (1, 0, 2)).reshape(T, -1),
                                  ref["k_new"].reshape(T, -1), f"layer {layer} appended keys")
    worst["v_new"] = assert_close(np.transpose(vn, (1, 0, 2)).reshape(T, -1),
                                  ref["v_new"].reshape(T, -1), f"layer {layer} appended values")
    print(f"layer {layer}, {T} tokens: " + ", ".join(f"{k} {e:.2e}/{n:.2e}"
                                                      for k, (e, n) in worst.items()), flush=True)


@pytest.mark.parametrize("group", range(GROUPS))
def test_13b_stack_every_layer_teacher_forced(group):
    wl = get("13b_stack")
    g = np.load(GOLDEN)
    per = wl.n_layers // GROUPS
    for layer in range(group * per, (group + 1) * per):
        teacher_forced(wl, layer, g["tf4_x"][layer])


@pytest.mark.parametrize("which", [0, 1])
def test_13b_stack_layer_all_64_tokens_teacher_forced(which):
    wl = get("13b_stack")
    g = np.load(GOLDEN)
    teacher_forced(wl, int(g["tf_layers"][which]), g["tf_x"][which])


def test_13b_stack_64_tokens_free_running():
    wl = get("13b_stack")
    g = np.load(GOLDEN)
    H, T, NL = wl.dims.hidden, wl.n_tokens, wl.n_layers
    t0 = time.time()
    shards = []
    for layer in range(NL):
        shards.append(GpuShard(wl, layer=layer, li=LayerInputs(wl, layer),
                               capacity=wl.ctx + T))
        if layer % 8 == 7:
            print(f"packed layers 0..{layer} in {time.time() - t0:.0f} s", flush=True)
    li0 = LayerInputs(wl, 0)
    drift = np.zeros((NL, len(KEYS)))
    for t in range(T):
        x = li0.x(t).astype(np.float64)
        for layer in range(NL):
            out = shards[layer].decode(x, wl.ctx + t)
            check_residuals(x, out)
            idx = sample_index(H, layer, t)
            for ki, k in enumerate(KEYS):
                ref = g["samples"][layer, t, ki].astype(np.float64)
                e = np.max(np.abs(out[k][idx] - ref) / np.maximum(np.abs(ref),
                                                                   g["rms"][layer, t, ki]))
                drift[layer, ki] = max(drift[layer, ki], e)
            x = out["y"]
        if t % 16 == 15:
            print(f"tokens 0..{t} through {NL} layers", flush=True)
    for s in shards:
        assert s.kv.len == wl.ctx + T
    # diagnostics: drift from the exact chain (40 sampled elements per vector,
    # denominator floored at the RMS) next to the fp16 rounding model's drift
    for layer in list(range(0, NL, 8)) + [NL - 1]:
        print(f"free-running layer {layer}: drift "
              + ", ".join(f"{k} {drift[layer, i]:.2e} (rounding model {g['model_err'][layer, i]:.2e})"
                          for i, k in enumerate(KEYS)), flush=True)
