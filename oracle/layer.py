"""fp64 definition of a decoder layer and of one device's tensor-parallel share.

All arithmetic is float64 on fp16-valued inputs with no intermediate
rounding; library matrix products serve as steps, nothing is blocked,
fused or reordered.

Layer (paper Sec. 2.1, Fig. Background1(a)), with the Llama readings for
what the paper leaves open:
    u  = RMSNorm(x) * g_attn                      pre-norm, eps from the layer
    q, k, v = Wq u, Wk u, Wv u                     split into heads
    q, k  <- RoPE at the token's absolute position  adjacent pairs (2i, 2i+1)
    K, V cache <- append k, v at that position      Sec. 2.1 (LLM Inference)
    o_j = softmax(q_j K_g^T / sqrt(d)) V_g,  g = j // (n_heads / n_kv_heads)
    attn = Wo concat(o_j)                          output linear O
    h  = x + attn
    w  = RMSNorm(h) * g_ffn
    ffn = Wd (silu(Wg w) * (Wu w))                 SwiGLU, no biases
    y  = h + ffn

Tensor parallelism (Sec. 3.2.1, Fig. Motivation1(b)): every device receives
the same broadcast input, computes the rows of Wq/Wk/Wv (its heads) and of
Wg/Wu (its FFN columns), and the matching columns of Wo and Wd. Its outputs
are the partial sums p_attn = Wo[:, heads] o and p_ffn = Wd[:, cols] m,
which the main device aggregates; the sum over a partition's shards is the
unsharded attn / ffn. ``peer_attn`` / ``peer_ffn`` stand for the sum of the
other devices' partials, so ``h = x + p_attn + peer_attn`` and
``y = h + p_ffn + peer_ffn`` are the aggregated sub-layer outputs.
"""
from dataclasses import dataclass
from typing import Optional

import numpy as np


@dataclass
class ShardWeights:
    """One shard's weights, canonical out x in, any float dtype.

    wq: [n_q*d, H]  wk, wv: [n_kv*d, H]  wo: [H, n_q*d]
    wg, wu: [n_cols, H]  wd: [H, n_cols]  g_attn, g_ffn: [H]
    """
    g_attn: np.ndarray
    wq: np.ndarray
    wk: np.ndarray
    wv: np.ndarray
    wo: np.ndarray
    g_ffn: np.ndarray
    wg: np.ndarray
    wu: np.ndarray
    wd: np.ndarray


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def rmsnorm(x, g, eps):
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    x = _f64(x)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * _f64(g)


def rope(z, pos, base):
    """Rotate adjacent pairs (z[2i], z[2i+1]) by angle pos * base^(-2i/d).

    ``z`` is [..., d]; ``pos`` broadcasts against z.shape[:-1].
    """
    z = _f64(z)
    d = z.shape[-1]
    i = np.arange(d // 2, dtype=np.float64)
    theta = np.power(float(base), -2.0 * i / d)
    phi = _f64(pos)[..., None] * theta
    c, s = np.cos(phi), np.sin(phi)
    a, b = z[..., 0::2], z[..., 1::2]
    out = np.empty_like(z)
    out[..., 0::2] = a * c - b * s
    out[..., 1::2] = a * s + b * c
    return out


def softmax(s):
    """Max-subtracted softmax over the last axis (-inf entries get weight 0)."""
    s = _f64(s)
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def silu(z):
    z = _f64(z)
    return z / (1.0 + np.exp(-z))


def attention(q, K, V):
    """Scaled dot-product attention of one query over keys K and values V."""
    q, K, V = _f64(q), _f64(K), _f64(V)
    a = softmax(K @ q / np.sqrt(q.shape[-1]))
    return a @ V


def append_kv(k_cache, v_cache, k_new, v_new, pos):
    """Cache after writing the new tokens' keys/values at positions pos.. .

    k_cache: [n_kv, n_pos, d] holding positions 0..pos-1 (extra slots ignored);
    k_new: [T, n_kv, d]. Returns [n_kv, pos+T, d] float64 arrays.
    """
    kc, vc = _f64(k_cache)[:, :pos], _f64(v_cache)[:, :pos]
    kn, vn = np.transpose(_f64(k_new), (1, 0, 2)), np.transpose(_f64(v_new), (1, 0, 2))
    return np.concatenate([kc, kn], axis=1), np.concatenate([vc, vn], axis=1)


def attn_sublayer(w: ShardWeights, n_q: int, n_kv: int, d: int, eps: float, base: float,
                  X, k_cache, v_cache, pos0: int, peer=None, window: int = 0):
    """ATTN sub-layer of a shard for T tokens at positions pos0..pos0+T-1.

    X: [T, H] input rows; k_cache/v_cache: [n_kv, >=pos0, d] the shard's
    cached (already rotated) keys and values. Token t attends to positions
    0..pos0+t, or with ``window`` > 0 (sliding-window attention, the local
    layers of Table 3's gemma models) to the last ``window`` of them.
    Returns p_attn [T, H], h [T, H], k_new, v_new [T, n_kv, d].
    """
    X = _f64(X)
    T, H = X.shape
    G = n_q // n_kv if n_kv else 1
    pos = pos0 + np.arange(T)
    U = rmsnorm(X, w.g_attn, eps)
    Q = (U @ _f64(w.wq).T).reshape(T, n_q, d)
    K = (U @ _f64(w.wk).T).reshape(T, n_kv, d)
    V = (U @ _f64(w.wv).T).reshape(T, n_kv, d)
    Q = rope(Q, pos[:, None], base)
    K = rope(K, pos[:, None], base)
    Kall, Vall = append_kv(k_cache, v_cache, K, V, pos0)       # [n_kv, pos0+T, d]
    O = np.zeros((T, n_q, d))
    for t in range(T):
        L = pos0 + t + 1
        lo = max(0, L - window) if window > 0 else 0
        for j in range(n_q):
            g = j // G
            O[t, j] = attention(Q[t, j], Kall[g, lo:L], Vall[g, lo:L])
    p_attn = O.reshape(T, n_q * d) @ _f64(w.wo).T
    h = X + p_attn + (0.0 if peer is None else _f64(peer))
    return p_attn, h, K, V


def ffn_sublayer(w: ShardWeights, eps: float, Hin, peer=None):
    """FFN sub-layer of a shard. Hin: [T, H]. Returns p_ffn [T, H], y [T, H]."""
    Hin = _f64(Hin)
    Wn = rmsnorm(Hin, w.g_ffn, eps)
    m = silu(Wn @ _f64(w.wg).T) * (Wn @ _f64(w.wu).T)
    p_ffn = m @ _f64(w.wd).T
    y = Hin + p_ffn + (0.0 if peer is None else _f64(peer))
    return p_ffn, y


def decode(w: ShardWeights, n_q, n_kv, d, eps, base, x, k_cache, v_cache, pos,
           peer_attn=None, peer_ffn=None, window=0) -> dict:
    """One batch-1 decode step of a shard at position ``pos``.

    x: [H]. Returns p_attn, h, p_ffn, y ([H] each) and the appended
    k_new, v_new ([n_kv, d]).
    """
    p_attn, h, K, V = attn_sublayer(w, n_q, n_kv, d, eps, base, _f64(x)[None], k_cache,
                                    v_cache, pos, None if peer_attn is None else
                                    _f64(peer_attn)[None], window)
    p_ffn, y = ffn_sublayer(w, eps, h, None if peer_ffn is None else _f64(peer_ffn)[None])
    return dict(p_attn=p_attn[0], h=h[0], p_ffn=p_ffn[0], y=y[0], k_new=K[0], v_new=V[0])


def prefill(w: ShardWeights, n_q, n_kv, d, eps, base, X, k_cache, v_cache, pos0,
            peer_attn=None, peer_ffn=None, window=0) -> dict:
    """A prefill chunk of T tokens of a shard at positions pos0..pos0+T-1."""
    p_attn, h, K, V = attn_sublayer(w, n_q, n_kv, d, eps, base, X, k_cache, v_cache, pos0,
                                    peer_attn, window)
    p_ffn, y = ffn_sublayer(w, eps, h, peer_ffn)
    return dict(p_attn=p_attn, h=h, p_ffn=p_ffn, y=y, k_new=K, v_new=V)
