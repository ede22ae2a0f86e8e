"""Pins of the fp64 oracle against facts it does not define itself.

* apportionment: the shard sizes each workload's definition states;
* brute force: an independent scalar-loop layer on tiny shapes;
* library: the unsharded layer through torch float64 ops (rms_norm,
  complex-number rotation, scaled_dot_product_attention with an explicit
  causal mask and repeat_interleave for GQA, silu);
* closed forms and invariants: softmax rows sum to 1, RoPE preserves pair
  norms, is the identity at position 0 and depends only on relative
  position in dot products; an empty cache attends to the token's own
  value; equal keys average the values; zero query/key weights give uniform
  attention; silu(0) = 0; RMSNorm output has unit RMS;
* linearity: the partials of all shards of a partition sum to the
  unsharded sub-layer outputs (1e-9), for MHA and GQA layers.
"""
import math

import numpy as np
import pytest

import oracle
from oracle.brute import brute_layer
from synth import get
from synth.gen import LayerInputs
from tests.common import (full_weights, oracle_ranges, oracle_shard_weights, tiny_workload)


# --------------------------------------------------------------------------
# apportionment
# --------------------------------------------------------------------------
# (workload, q heads, kv heads, FFN columns) of the benchmarked shard, as the
# workload definitions state them.
STATED = [("tiny", 4, 4, 688), ("7b", 10, 10, 3302), ("13b_stack", 16, 16, 5530),
          ("70b_gqa", 16, 2, 7168), ("7b_prefill", 16, 16, 5504)]


@pytest.mark.parametrize("key,nq,nkv,ncols", STATED)
def test_apportion_stated_shard_sizes(key, nq, nkv, ncols):
    r = oracle_ranges(get(key))
    assert (r.n_q_heads, r.n_kv_heads, r.n_cols) == (nq, nkv, ncols)


def test_apportion_properties():
    rng = np.random.default_rng(1)
    for _ in range(2000):
        n = int(rng.integers(1, 9))
        total = int(rng.integers(0, 40000))
        f = rng.random(n)
        f[rng.random(n) < 0.2] = 0.0
        if f.sum() == 0:
            f[0] = 1.0
        f = list(f / f.sum())
        if abs(math.fsum(f) - 1.0) > 1e-9:
            continue
        c = oracle.apportion(total, f)
        assert sum(c) == total
        for ci, fi in zip(c, f):
            q = fi * total
            assert math.floor(q) <= ci <= math.floor(q) + 1
            if fi == 0.0:
                assert ci == 0


def test_apportion_ties_and_errors():
    assert oracle.apportion(3, [0.5, 0.5]) == [2, 1]
    assert oracle.apportion(5, [0.2] * 5) == [1] * 5
    assert oracle.apportion(1, [1 / 3] * 3) == [1, 0, 0]
    for bad in ([0.5, 0.4], [1.2, -0.2], [float("nan"), 1.0], []):
        with pytest.raises(ValueError):
            oracle.apportion(10, bad)


def test_shard_ranges_cover_layer_contiguously():
    wl = get("70b_gqa")
    d = wl.dims
    prev_kv = prev_c = 0
    for dev in range(len(wl.fracs)):
        r = oracle_ranges(wl, dev)
        assert r.kv_head_begin == prev_kv and r.col_begin == prev_c
        assert r.q_head_begin == r.kv_head_begin * d.group
        assert r.n_q_heads == r.n_kv_heads * d.group
        prev_kv += r.n_kv_heads
        prev_c += r.n_cols
    assert (prev_kv, prev_c) == (d.n_kv_heads, d.ffn)


# --------------------------------------------------------------------------
# building blocks: closed forms and invariants
# --------------------------------------------------------------------------
def test_softmax_rows_sum_to_one():
    rng = np.random.default_rng(2)
    s = rng.normal(0, 30, size=(64, 257))
    a = oracle.softmax(s)
    assert np.all(a >= 0)
    assert np.max(np.abs(a.sum(-1) - 1)) < 1e-12
    # invariance to a per-row shift, and the two-point closed form
    assert np.allclose(oracle.softmax(s + 1234.5), a, rtol=0, atol=1e-12)
    assert abs(oracle.softmax(np.array([0.0, math.log(3.0)]))[1] - 0.75) < 1e-15


def test_rope_norms_identity_relativity():
    rng = np.random.default_rng(3)
    d = 128
    z = rng.normal(size=(5, d))
    for pos in (0, 1, 17, 1023, 4096):
        r = oracle.rope(z, pos, 10000.0)
        n0 = z[:, 0::2] ** 2 + z[:, 1::2] ** 2
        n1 = r[:, 0::2] ** 2 + r[:, 1::2] ** 2
        assert np.max(np.abs(n0 - n1)) < 1e-12
    assert np.array_equal(oracle.rope(z, 0, 10000.0), z)
    q, k = rng.normal(size=d), rng.normal(size=d)
    for m, n in ((9, 4), (300, 7), (2050, 2047)):
        lhs = oracle.rope(q, m, 10000.0) @ oracle.rope(k, n, 10000.0)
        rhs = oracle.rope(q, m - n, 10000.0) @ k
        assert abs(lhs - rhs) < 1e-10 * (1 + abs(lhs))
    # closed form for the first pair (frequency 1): angle = position
    e = np.zeros(d)
    e[0] = 1.0
    r = oracle.rope(e, 2.0, 10000.0)
    assert abs(r[0] - math.cos(2.0)) < 1e-15 and abs(r[1] - math.sin(2.0)) < 1e-15
    # last pair rotates by pos * base^(-(d-2)/d)
    e = np.zeros(d)
    e[d - 2] = 1.0
    ang = 100.0 * 10000.0 ** (-(d - 2) / d)
    r = oracle.rope(e, 100.0, 10000.0)
    assert abs(r[d - 2] - math.cos(ang)) < 1e-14 and abs(r[d - 1] - math.sin(ang)) < 1e-14


def test_rmsnorm_and_silu_closed_forms():
    rng = np.random.default_rng(4)
    x = rng.normal(size=(3, 4096)) * 7
    u = oracle.rmsnorm(x, np.ones(4096), 0.0)
    assert np.max(np.abs(np.sqrt(np.mean(u * u, -1)) - 1)) < 1e-12
    assert np.allclose(oracle.rmsnorm(2 * x, np.ones(4096), 0.0), u, atol=1e-13)
    assert oracle.silu(0.0) == 0.0
    assert abs(oracle.silu(1.0) - 1 / (1 + math.exp(-1))) < 1e-16
    assert abs(oracle.silu(-50.0)) < 1e-19


def test_attention_special_cases():
    rng = np.random.default_rng(5)
    q = rng.normal(size=64)
    K = rng.normal(size=(1, 64))
    V = rng.normal(size=(1, 64))
    assert np.array_equal(oracle.attention(q, K, V), V[0])       # one key: its value
    K = np.repeat(rng.normal(size=(1, 64)), 9, 0)                 # equal keys: mean of V
    V = rng.normal(size=(9, 64))
    assert np.allclose(oracle.attention(q, K, V), V.mean(0), atol=1e-14)


# --------------------------------------------------------------------------
# layer: brute force and library cross-checks
# --------------------------------------------------------------------------
TINY = [
    # seed, hidden, heads, kv, d, ffn, fracs, device, ctx, chunk
    (101, 16, 4, 4, 4, 24, (0.5, 0.5), 1, 5, 0),        # MHA decode
    (102, 32, 4, 2, 8, 20, (0.6, 0.4), 0, 3, 0),        # GQA group 2
    (103, 24, 6, 2, 4, 18, (1.0,), 0, 4, 3),            # GQA group 3, prefill chunk 3
    (104, 16, 2, 1, 8, 12, (1.0,), 0, 0, 2),            # MQA, empty cache, prefill
    (105, 16, 4, 4, 4, 30, (0.3, 0.3, 0.4), 2, 2, 0),   # 3-device uneven split
]


def _tiny_inputs(wl):
    li = LayerInputs(wl)
    r = oracle_ranges(wl)
    w = oracle_shard_weights(li, r)
    kc, vc = li.kv_context_heads(r.kv_head_begin, r.kv_head_begin + r.n_kv_heads)
    T = wl.chunk or 1
    X = li.x_chunk(T) if wl.chunk else li.x(0)[None]
    return li, r, w, kc, vc, X


@pytest.mark.parametrize("case", TINY)
def test_oracle_matches_brute_force(case):
    seed, H, nh, nkv, d, F, fr, dev, ctx, chunk = case
    wl = tiny_workload(seed, H, nh, nkv, d, F, fr, dev, ctx, chunk=chunk)
    li, r, w, kc, vc, X = _tiny_inputs(wl)
    peer_a = li.peer("attn", rows=X.shape[0])
    peer_f = li.peer("ffn", rows=X.shape[0])
    o = oracle.prefill(w, r.n_q_heads, r.n_kv_heads, d, 1e-5, 10000.0, X, kc, vc, ctx,
                       peer_a, peer_f)
    b = brute_layer(w, r.n_q_heads, r.n_kv_heads, d, 1e-5, 10000.0, X, kc, vc, ctx,
                    peer_a, peer_f)
    for key in ("p_attn", "h", "p_ffn", "y"):
        ref = np.array(b[key])
        assert np.max(np.abs(o[key] - ref)) <= 1e-12 * (1 + np.max(np.abs(ref))), key


def torch_layer(w, n_q, n_kv, d, eps, base, X, kc, vc, pos0):
    """The unsharded layer through torch float64 library routines."""
    import torch
    import torch.nn.functional as F
    t = lambda a: torch.as_tensor(np.asarray(a, np.float64))
    X = t(X)
    T, H = X.shape
    U = F.rms_norm(X, (H,), weight=t(w.g_attn), eps=eps)
    Q = (U @ t(w.wq).T).view(T, n_q, d)
    K = (U @ t(w.wk).T).view(T, n_kv, d)
    V = (U @ t(w.wv).T).view(T, n_kv, d)
    pos = torch.arange(pos0, pos0 + T, dtype=torch.float64)
    inv = 1.0 / (base ** (torch.arange(0, d, 2, dtype=torch.float64) / d))
    rot = torch.polar(torch.ones(T, d // 2, dtype=torch.float64), torch.outer(pos, inv))

    def rotate(Z):
        c = torch.view_as_complex(Z.reshape(T, Z.shape[1], d // 2, 2).contiguous())
        return torch.view_as_real(c * rot[:, None, :]).reshape(T, Z.shape[1], d)

    Q, K = rotate(Q), rotate(K)
    Kall = torch.cat([t(kc)[:, :pos0], K.transpose(0, 1)], 1)
    Vall = torch.cat([t(vc)[:, :pos0], V.transpose(0, 1)], 1)
    G = n_q // n_kv
    Kx = Kall.repeat_interleave(G, 0)
    Vx = Vall.repeat_interleave(G, 0)
    S = pos0 + T
    mask = torch.arange(S)[None, :] <= (pos0 + torch.arange(T))[:, None]
    O = F.scaled_dot_product_attention(Q.transpose(0, 1), Kx, Vx, attn_mask=mask)
    p_attn = O.transpose(0, 1).reshape(T, n_q * d) @ t(w.wo).T
    h = X + p_attn
    Wn = F.rms_norm(h, (H,), weight=t(w.g_ffn), eps=eps)
    p_ffn = (F.silu(Wn @ t(w.wg).T) * (Wn @ t(w.wu).T)) @ t(w.wd).T
    return dict(p_attn=p_attn.numpy(), h=h.numpy(), p_ffn=p_ffn.numpy(),
                y=(h + p_ffn).numpy(), k_new=K.numpy(), v_new=V.numpy())


def _torch_case(wl, T=None):
    li = LayerInputs(wl)
    d = wl.dims
    w = full_weights(li)
    kc, vc = li.kv_context_heads(0, d.n_kv_heads)
    T = T or wl.chunk or 1
    X = li.x_chunk(T) if (wl.chunk or T > 1) else li.x(0)[None]
    return li, w, kc, vc, X


@pytest.mark.parametrize("key,T", [("tiny", 1), ("tiny", 5)])
def test_oracle_matches_torch_library(key, T):
    wl = get(key)
    d = wl.dims
    li, w, kc, vc, X = _torch_case(wl, T)
    o = oracle.prefill(w, d.n_heads, d.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, X,
                       kc, vc, wl.ctx)
    ref = torch_layer(w, d.n_heads, d.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, X,
                      kc, vc, wl.ctx)
    for k in ("p_attn", "h", "p_ffn", "y", "k_new", "v_new"):
        err = np.max(np.abs(o[k] - ref[k])) / (1 + np.max(np.abs(ref[k])))
        assert err < 1e-11, (k, err)


def test_oracle_matches_torch_library_gqa():
    wl = tiny_workload(110, 64, 8, 2, 16, 96, (1.0,), 0, 37, chunk=4)
    d = wl.dims
    li, w, kc, vc, X = _torch_case(wl)
    o = oracle.prefill(w, 8, 2, 16, d.rms_eps, d.rope_base, X, kc, vc, wl.ctx)
    ref = torch_layer(w, 8, 2, 16, d.rms_eps, d.rope_base, X, kc, vc, wl.ctx)
    for k in ("p_attn", "h", "p_ffn", "y"):
        assert np.max(np.abs(o[k] - ref[k])) < 1e-11 * (1 + np.max(np.abs(ref[k]))), k


def test_zero_qk_weights_give_uniform_attention():
    """Closed form: with Wq = Wk = 0 every score is 0, so each head's output
    is the plain mean of its values over positions 0..pos."""
    wl = tiny_workload(111, 16, 4, 2, 4, 8, (1.0,), 0, 6)
    li, r, w, kc, vc, X = _tiny_inputs(wl)
    w.wq = np.zeros_like(w.wq)
    w.wk = np.zeros_like(w.wk)
    o = oracle.decode(w, 4, 2, 4, 1e-5, 10000.0, X[0], kc, vc, 6)
    u = oracle.rmsnorm(X[0], w.g_attn, 1e-5)
    v_new = (np.asarray(w.wv, np.float64) @ u).reshape(2, 4)
    heads = []
    for j in range(4):
        g = j // 2
        heads.append((np.asarray(vc[g], np.float64).sum(0) + v_new[g]) / 7.0)
    expect = np.asarray(w.wo, np.float64) @ np.concatenate(heads)
    assert np.max(np.abs(o["p_attn"] - expect)) < 1e-13


def test_empty_cache_attends_to_own_value():
    wl = tiny_workload(112, 32, 4, 4, 8, 16, (1.0,), 0, 0)
    li, r, w, kc, vc, X = _tiny_inputs(wl)
    o = oracle.decode(w, 4, 4, 8, 1e-5, 10000.0, X[0], kc, vc, 0)
    u = oracle.rmsnorm(X[0], w.g_attn, 1e-5)
    v = np.asarray(w.wv, np.float64) @ u
    assert np.max(np.abs(o["p_attn"] - np.asarray(w.wo, np.float64) @ v)) < 1e-13


# --------------------------------------------------------------------------
# linearity: shards of a partition sum to the unsharded layer
# --------------------------------------------------------------------------
def _check_shard_sum(wl, T=1):
    d = wl.dims
    li = LayerInputs(wl)
    kc_all, vc_all = li.kv_context_heads(0, d.n_kv_heads)
    X = li.x_chunk(T) if T > 1 else li.x(0)[None]
    full = oracle.attn_sublayer(full_weights(li), d.n_heads, d.n_kv_heads, d.head_dim,
                                d.rms_eps, d.rope_base, X, kc_all, vc_all, wl.ctx)
    h_full = full[1]
    ffn_full, _ = oracle.ffn_sublayer(full_weights(li), d.rms_eps, h_full)
    sum_attn = np.zeros_like(h_full)
    sum_ffn = np.zeros_like(h_full)
    for dev in range(len(wl.fracs)):
        r = oracle_ranges(wl, dev)
        w = oracle_shard_weights(li, r)
        g0, g1 = r.kv_head_begin, r.kv_head_begin + r.n_kv_heads
        pa, _, _, _ = oracle.attn_sublayer(w, r.n_q_heads, r.n_kv_heads, d.head_dim,
                                           d.rms_eps, d.rope_base, X, kc_all[g0:g1],
                                           vc_all[g0:g1], wl.ctx)
        pf, _ = oracle.ffn_sublayer(w, d.rms_eps, h_full)
        sum_attn += pa
        sum_ffn += pf
    assert np.max(np.abs(sum_attn + X - h_full)) <= 1e-9 * np.max(np.abs(full[0]))
    assert np.max(np.abs(sum_ffn - ffn_full)) <= 1e-9 * np.max(np.abs(ffn_full))


def test_shard_sum_tiny_mha():
    _check_shard_sum(get("tiny"))


def test_shard_sum_gqa_uneven():
    _check_shard_sum(tiny_workload(120, 128, 16, 4, 16, 200, (0.5, 0.25, 0.25), 0, 33), T=3)


@pytest.mark.slow
def test_shard_sum_7b_three_devices():
    _check_shard_sum(get("7b"))
