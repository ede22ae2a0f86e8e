"""Writes tests/golden/stack_13b.npz: the fp64 oracle's free-running chain of
64 consecutive decode tokens through the 40-layer 13B-shaped stack (40%
shard: 16 of 40 heads, 5530 of 13824 FFN columns, cached positions
0..2047 per layer).

Chain (the single-device stand-in for the stack): layer l's input for token
t is layer l-1's output y of token t; the other devices' partial sums are
taken as zero, so y = h + p_ffn. Token inputs of layer 0 come from the seeded
generator. The oracle computes each layer for all 64 tokens at once as a
causal chunk at positions 2048..2111: token t of layer l depends only on
tokens 0..t of that layer, so this equals 64 decode steps in a row.

Stored per (layer, token, output) with outputs ordered p_attn, h, p_ffn, y:
the vector's RMS (the tolerance floor) and its values at 40 sampled indices
(``sample_index``); full vectors of the first and last token at the first
and last layer.

Teacher forcing: at every layer, the chain's inputs of the first TF4
tokens (``tf4_x``); at layers TF_LAYERS, the chain's inputs of all 64
tokens (``tf_x``) and the oracle's outputs for exactly those inputs (RMS,
samples, full vectors of tokens TF_FULL_TOKENS). Inputs are rounded to fp16,
the precision of the layer interface. A device run fed these inputs is held
to the single-layer bar (the GPU test evaluates the oracle on them again),
free of the drift a 40-layer chain accumulates.

Drift model: the same chain computed with fp16 rounding at the points where
the device rounds (the normalised inputs of the projections, q, the cached
keys and values, the SiLU-gate product, every layer output), compared with
the exact chain by the element-wise metric; ``model_err[layer, output]`` is
the largest error over the 64 tokens. It is the expected size of fp16
compounding, used to bound the free-running chain below the first layer.

No value comes from the GPU path: only ``oracle/``, numpy rounding and the
seeded generator are called. Run: python tests/golden/make_stack_golden.py
(about twelve minutes of host time).
"""
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
from oracle import layer as OL  # noqa: E402
from synth import get  # noqa: E402
from synth.gen import LayerInputs  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "stack_13b.npz")
KEYS = ("p_attn", "h", "p_ffn", "y")
N_SAMPLES = 40
FULL_LAYERS = (0, 39)
FULL_TOKENS = (0, 63)
TF_LAYERS = (20, 39)
TF_FULL_TOKENS = (0, 31, 63)
TF4 = 4  # leading tokens teacher-forced at every layer


def sample_index(hidden, layer, token):
    """Indices compared for (layer, token): one per stretch of hidden/40
    elements, at an offset that moves with the layer and the token."""
    stride = hidden // N_SAMPLES
    return np.arange(N_SAMPLES) * stride + (layer * 37 + token * 11) % stride


def shard_weights(li, r, d):
    q0, q1 = r.q_head_begin * d, (r.q_head_begin + r.n_q_heads) * d
    k0, k1 = r.kv_head_begin * d, (r.kv_head_begin + r.n_kv_heads) * d
    c0, c1 = r.col_begin, r.col_begin + r.n_cols
    return oracle.ShardWeights(g_attn=li.g_attn(), wq=li.rows("wq", q0, q1),
                               wk=li.rows("wk", k0, k1), wv=li.rows("wv", k0, k1),
                               wo=li.cols("wo", q0, q1), g_ffn=li.g_ffn(),
                               wg=li.rows("wg", c0, c1), wu=li.rows("wu", c0, c1),
                               wd=li.cols("wd", c0, c1))


def h16(a):
    return np.asarray(a, np.float16).astype(np.float64)


def rounded_layer(w, r, dm, X, kc, vc, pos0):
    """The layer with fp16 rounding where the device rounds (drift model)."""
    d = dm.head_dim
    T = X.shape[0]
    U = h16(OL.rmsnorm(X, w.g_attn, dm.rms_eps))
    pos = pos0 + np.arange(T)
    Q = OL.rope((U @ np.float64(w.wq).T).reshape(T, r.n_q_heads, d), pos[:, None], dm.rope_base)
    K = h16(OL.rope((U @ np.float64(w.wk).T).reshape(T, r.n_kv_heads, d), pos[:, None],
                    dm.rope_base))
    V = h16((U @ np.float64(w.wv).T).reshape(T, r.n_kv_heads, d))
    Q = h16(Q)
    Kall, Vall = OL.append_kv(kc, vc, K, V, pos0)
    G = r.n_q_heads // r.n_kv_heads
    O = np.zeros((T, r.n_q_heads, d))
    for t in range(T):
        n = pos0 + t + 1
        for j in range(r.n_q_heads):
            O[t, j] = OL.attention(Q[t, j], Kall[j // G, :n], Vall[j // G, :n])
    pa = h16(O.reshape(T, -1) @ np.float64(w.wo).T)
    h = h16(X + pa)
    Wn = h16(OL.rmsnorm(h, w.g_ffn, dm.rms_eps))
    m = h16(OL.silu(Wn @ np.float64(w.wg).T) * (Wn @ np.float64(w.wu).T))
    pf = h16(m @ np.float64(w.wd).T)
    return dict(p_attn=pa, h=h, p_ffn=pf, y=h16(h + pf))


def elementwise_err(got, ref):
    rms = np.sqrt(np.mean(ref * ref, axis=1, keepdims=True))
    return float(np.max(np.abs(got - ref) / np.maximum(np.abs(ref), rms)))


def summarize(ref, layer, H, T):
    rms = np.zeros((T, len(KEYS)))
    samples = np.zeros((T, len(KEYS), N_SAMPLES))
    for ki, k in enumerate(KEYS):
        v = ref[k]
        rms[:, ki] = np.sqrt(np.mean(v * v, axis=1))
        for t in range(T):
            samples[t, ki] = v[t, sample_index(H, layer, t)]
    return rms, samples


def build():
    wl = get("13b_stack")
    dm = wl.dims
    H, d, T = dm.hidden, dm.head_dim, wl.n_tokens
    r = oracle.shard_ranges(dm.n_heads, dm.n_kv_heads, dm.ffn, wl.fracs, wl.fracs, wl.device)
    li0 = LayerInputs(wl, 0)
    X = np.stack([li0.x(t) for t in range(T)]).astype(np.float64)
    rms = np.zeros((wl.n_layers, T, len(KEYS)))
    samples = np.zeros((wl.n_layers, T, len(KEYS), N_SAMPLES))
    full = np.zeros((len(FULL_LAYERS), len(FULL_TOKENS), len(KEYS), H))
    tf_x = np.zeros((len(TF_LAYERS), T, H), np.float16)
    tf4_x = np.zeros((wl.n_layers, TF4, H), np.float16)
    tf_rms = np.zeros((len(TF_LAYERS), T, len(KEYS)))
    tf_samples = np.zeros((len(TF_LAYERS), T, len(KEYS), N_SAMPLES))
    tf_full = np.zeros((len(TF_LAYERS), len(TF_FULL_TOKENS), len(KEYS), H))
    model_err = np.zeros((wl.n_layers, len(KEYS)))
    XC = X.copy()
    for layer in range(wl.n_layers):
        t0 = time.time()
        li = li0 if layer == 0 else LayerInputs(wl, layer)
        w = shard_weights(li, r, d)
        kc, vc = li.kv_context_heads(r.kv_head_begin, r.kv_head_begin + r.n_kv_heads)
        tf4_x[layer] = X[:TF4].astype(np.float16)
        ref = oracle.prefill(w, r.n_q_heads, r.n_kv_heads, d, dm.rms_eps, dm.rope_base, X, kc,
                             vc, wl.ctx)
        rms[layer], samples[layer] = summarize(ref, layer, H, T)
        if layer in FULL_LAYERS:
            for ti, t in enumerate(FULL_TOKENS):
                for ki, k in enumerate(KEYS):
                    full[FULL_LAYERS.index(layer), ti, ki] = ref[k][t]
        if layer in TF_LAYERS:
            i = TF_LAYERS.index(layer)
            tf_x[i] = X.astype(np.float16)
            tf = oracle.prefill(w, r.n_q_heads, r.n_kv_heads, d, dm.rms_eps, dm.rope_base,
                                tf_x[i].astype(np.float64), kc, vc, wl.ctx)
            tf_rms[i], tf_samples[i] = summarize(tf, layer, H, T)
            for ti, t in enumerate(TF_FULL_TOKENS):
                for ki, k in enumerate(KEYS):
                    tf_full[i, ti, ki] = tf[k][t]
        C = rounded_layer(w, r, dm, XC, kc, vc, wl.ctx)
        for ki, k in enumerate(KEYS):
            model_err[layer, ki] = elementwise_err(C[k], ref[k])
        X = ref["y"]
        XC = C["y"]
        print(f"layer {layer}: {time.time() - t0:.1f} s, rms(y) {rms[layer, :, 3].mean():.3f}, "
              f"model drift " + " ".join(f"{model_err[layer, ki]:.2e}" for ki in range(4)),
              flush=True)
    np.savez_compressed(OUT, rms=rms, samples=samples.astype(np.float32),
                        full=full.astype(np.float32),
                        full_layers=np.array(FULL_LAYERS), full_tokens=np.array(FULL_TOKENS),
                        n_samples=np.array(N_SAMPLES), tf_layers=np.array(TF_LAYERS),
                        tf_x=tf_x, tf_rms=tf_rms, tf_samples=tf_samples.astype(np.float32),
                        tf_full=tf_full.astype(np.float32), tf_full_tokens=np.array(TF_FULL_TOKENS),
                        tf4_x=tf4_x, model_err=model_err)
    print("wrote", OUT, os.path.getsize(OUT), "bytes")


if __name__ == "__main__":
    build()
