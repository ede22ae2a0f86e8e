"""GPU parity of the prefill chunk (vt_layer_prefill_chunk, MFMA path)
against the fp64 oracle, through the C ABI.

Same bar as decode (per-row element-wise relative error <= 2e-2 with the
denominator floored at 0.2 of the row's RMS, normwise <= 1.5e-3; the FFN
outputs against the oracle's FFN at fp16(h)); the appended K/V of every chunk token lands in
its slot and every other cache byte is unchanged. Also: the sub-layers as
separate calls, NaN in the weight rows' padding, and bit-identical repeats
(the split-K reduction's order does not depend on arrival order).
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from paper_2607_07046_amd import voltron as vt
from synth import get
from synth.gen import LayerInputs
from tests.common import (FLOOR, NORM_TOL, REL_TOL, assert_close, ffn_at_h16, max_rel_err,
                          norm_rel_err, oracle_ranges, oracle_shard_weights, tiny_workload)
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


def _sample_rows(T, seed, n_random=24):
    """Rows at both edges of every 128-row GEMM tile plus seeded random ones."""
    rows = {0, 1, T - 2, T - 1}
    for e in range(128, T, 128):
        rows |= {e - 1, e}
    rng = np.random.default_rng(seed)
    rows |= set(int(r) for r in rng.integers(0, T, n_random))
    return sorted(r for r in rows if 0 <= r < T)


@pytest.mark.parametrize("T", [1024, 4096])
def test_prefill_long_chunks(T):
    """The 7B 50% shard with 1024 and 4096 tokens at positions 768.. : the
    split-K choice goes from 4 slices down to 3, 2 and 1 (no reduction), and
    the attention runs over up to 4864 keys. Every appended key and value is
    checked; the layer outputs on rows at both edges of every 128-row tile
    and seeded random rows, each against the oracle's decode step of that
    token over the context and the chunk's earlier keys and values (the
    oracle's attention sub-layer with a one-position window gives the
    chunk's keys and values: they do not depend on the window)."""
    wl = get("7b_prefill")
    li = LayerInputs(wl)
    d = wl.dims
    r = oracle_ranges(wl)
    w = oracle_shard_weights(li, r)
    # the same values held as float64 once, so the per-row oracle calls below
    # do not widen the shard's weights again each time
    w = oracle.ShardWeights(**{f.name: np.asarray(getattr(w, f.name), np.float64)
                               for f in dataclasses.fields(w)})
    kc, vc = li.kv_context_heads(r.kv_head_begin, r.kv_head_begin + r.n_kv_heads)
    X = li.x_chunk(T)
    pa, pf = li.peer("attn", rows=T), li.peer("ffn", rows=T)
    # the workspace is sized for the longest chunk, 4096 tokens, and must
    # serve the shorter one too (whose GEMMs take more split-K slices)
    gs = GpuShard(wl, li=li, capacity=wl.ctx + T, max_tokens=4096)
    k0, v0 = gs.cache()
    got = gs.prefill(X, wl.ctx, BOTH, peer_attn=pa, peer_ffn=pf)
    assert not gs.sync_words().any()
    _, _, K, V = oracle.attn_sublayer(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps,
                                      d.rope_base, X, kc, vc, wl.ctx, window=1)
    kc1, vc1 = gs.cache()
    assert gs.kv.len == wl.ctx + T
    assert np.array_equal(kc1[:, :wl.ctx], k0[:, :wl.ctx])
    assert np.array_equal(vc1[:, :wl.ctx], v0[:, :wl.ctx])
    rng = slice(wl.ctx, wl.ctx + T)
    kn = kc1[:, rng].view(np.float16).astype(np.float64)
    vn = vc1[:, rng].view(np.float16).astype(np.float64)
    assert_close(np.transpose(kn, (1, 0, 2)).reshape(T, -1), K.reshape(T, -1), "appended keys")
    assert_close(np.transpose(vn, (1, 0, 2)).reshape(T, -1), V.reshape(T, -1), "appended values")
    rows = _sample_rows(T, 7000 + T)
    ref = {k: [] for k in ("p_attn", "h", "p_ffn", "y")}
    for t in rows:
        kt, vt_ = oracle.append_kv(kc, vc, K[:t], V[:t], wl.ctx)
        o = oracle.decode(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, X[t],
                          kt, vt_, wl.ctx + t, pa[t], pf[t])
        o = ffn_at_h16(w, d.rms_eps, o, pf[t])
        for k in ref:
            ref[k].append(o[k])
    for k in ref:
        assert_close(got[k][rows], np.stack(ref[k]), f"{k} on {len(rows)} sampled rows")


def _close_dev(got, ref, what):
    """The parity bar (element-wise with the row-RMS floor, and normwise) of
    two fp16 [rows, H] device tensors, evaluated on the device."""
    g, r = got.double(), ref.double()
    assert bool(torch.isfinite(g).all()), what
    floor = FLOOR * torch.sqrt((r * r).mean(dim=1, keepdim=True))
    e = float(((g - r).abs() / torch.maximum(r.abs(), floor)).max())
    n = float(torch.linalg.norm(g - r) / torch.linalg.norm(r))
    print(f"{what}: element-wise {e:.3g}, normwise {n:.3g}")
    assert e <= REL_TOL and n <= NORM_TOL, f"{what}: element-wise {e:.3g}, normwise {n:.3g}"


def test_prefill_max_chunk():
    """The largest chunk the entry point takes: 65536 tokens at positions
    768.. of the 7B 50% shard in one call (GEMM grids of 512 row tiles, 2048
    query blocks per head, keys up to 66303). The first 1024 tokens' keys,
    values and sampled output rows against the oracle (those rows attend to
    the context and the first 1024 tokens only); every output row and every
    appended key and value against the same tokens prefilled as sixteen
    4096-token chunks, at the same bar; the context's cache bytes unchanged."""
    T, C, R = 65536, 4096, 1024
    wl = get("7b_prefill")
    li = LayerInputs(wl)
    d = wl.dims
    X = li.x_chunk(T)
    one = GpuShard(wl, li=li, capacity=wl.ctx + T, max_tokens=T)
    k0, v0 = one.cache()
    big = one.prefill(X, wl.ctx, BOTH, on_device=True)
    assert not one.sync_words().any()
    assert one.kv.len == wl.ctx + T
    split = GpuShard(wl, li=li, capacity=wl.ctx + T, max_tokens=C)
    parts = [split.prefill(X[i:i + C], wl.ctx + i, BOTH, on_device=True) for i in range(0, T, C)]
    assert not split.sync_words().any()
    for k in ("p_attn", "h", "p_ffn", "y"):
        _close_dev(big[k], torch.cat([pt[k] for pt in parts]), f"{k}, one chunk vs 16")
    del parts
    new = slice(wl.ctx, wl.ctx + T)
    for a, b, name in ((one.kc, split.kc, "keys"), (one.vc, split.vc, "values")):
        _close_dev(a[:, new].reshape(-1, a.shape[-1] * 16), b[:, new].reshape(-1, a.shape[-1] * 16),
                   f"appended {name}, one chunk vs 16")
    kc1, vc1 = one.cache()
    assert np.array_equal(kc1[:, :wl.ctx], k0[:, :wl.ctx])
    assert np.array_equal(vc1[:, :wl.ctx], v0[:, :wl.ctx])

    # the oracle on the first R tokens
    r = oracle_ranges(wl)
    w = oracle_shard_weights(li, r)
    w = oracle.ShardWeights(**{f.name: np.asarray(getattr(w, f.name), np.float64)
                               for f in dataclasses.fields(w)})
    kc, vc = li.kv_context_heads(r.kv_head_begin, r.kv_head_begin + r.n_kv_heads)
    _, _, K, V = oracle.attn_sublayer(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps,
                                      d.rope_base, X[:R], kc, vc, wl.ctx, window=1)
    first = slice(wl.ctx, wl.ctx + R)
    kn = kc1[:, first].view(np.float16).astype(np.float64)
    vn = vc1[:, first].view(np.float16).astype(np.float64)
    assert_close(np.transpose(kn, (1, 0, 2)).reshape(R, -1), K.reshape(R, -1), "appended keys")
    assert_close(np.transpose(vn, (1, 0, 2)).reshape(R, -1), V.reshape(R, -1), "appended values")
    rows = _sample_rows(R, 7100, n_random=8)
    got = {k: big[k][rows].float().cpu().numpy().astype(np.float64) for k in big}
    ref = {k: [] for k in ("p_attn", "h", "p_ffn", "y")}
    for t in rows:
        kt, vt_ = oracle.append_kv(kc, vc, K[:t], V[:t], wl.ctx)
        o = oracle.decode(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, X[t],
                          kt, vt_, wl.ctx + t, None, None)
        o = ffn_at_h16(w, d.rms_eps, o)
        for k in ref:
            ref[k].append(o[k])
    for k in ref:
        assert_close(got[k], np.stack(ref[k]), f"{k} on {len(rows)} sampled rows")


CASES = [
    # seed, hidden, heads, kv, d, ffn, fracs, device, ctx, T
    (301, 512, 8, 8, 64, 1000, (0.5, 0.5), 0, 0, 1),        # empty cache, one token
    (302, 512, 8, 2, 64, 1000, (0.5, 0.5), 1, 7, 5),        # GQA group 4, ragged everything
    (303, 1024, 8, 4, 128, 1501, (0.6, 0.4), 0, 40, 70),    # d 128, odd FFN width, 3 query blocks
    (304, 768, 12, 12, 64, 2000, (0.3, 0.7), 1, 100, 129),  # M > one 128-row tile, 5 query blocks
    (310, 1536, 12, 4, 128, 1000, (0.5, 0.5), 1, 90, 77),   # GQA group 3
    (311, 1792, 28, 4, 64, 1200, (0.5, 0.5), 0, 45, 140),   # GQA group 7
    (312, 1024, 16, 4, 128, 1000, (0.5, 0.5), 1, 30000, 64),  # a 64-token chunk after 30000 positions
    (313, 1024, 16, 4, 64, 1000, (0.5, 0.5), 0, 20000, 200),  # head size 64 after 20000 positions
]


@pytest.mark.parametrize("case", CASES, ids=[str(c[0]) for c in CASES])
def test_prefill_ragged_shapes(case):
    seed, H, nh, nkv, d, F, fr, dev, ctx, T = case
    wl = tiny_workload(seed, H, nh, nkv, d, F, fr, dev, ctx, sigma=0.03, chunk=T)
    run_case(wl, T)


# Seeded shapes around the GEMM tiles' edges (128 tokens, 128 features,
# 64 k-columns, 16-column k-steps): tokens one either side of a tile, hidden
# sizes that are multiples of 8 but not of 16 or 128, odd FFN shares, both
# head sizes, GQA groups; drawn once from a fixed seed.
def _edge_cases():
    rng = np.random.default_rng(20261202)
    out = []
    for i, T in enumerate((127, 128, 129, 255, 257)):
        d = (64, 128)[i % 2]
        nkv = int(rng.choice([1, 2, 4]))
        nh = nkv * int(rng.choice([1, 2, 4]))
        while nh < 2:
            nh *= 2
        H = int(rng.choice([520, 776, 1032, 1288]))
        F = int(rng.integers(300, 1500))
        fr = (0.5, 0.5) if nh % 2 == 0 and nkv % 2 == 0 else (1.0,)
        dev = int(rng.integers(0, len(fr)))
        ctx = int(rng.integers(0, 60))
        out.append((400 + i, H, nh, nkv, d, F, fr, dev, ctx, T))
    return out


EDGE = _edge_cases()


@pytest.mark.parametrize("case", EDGE, ids=[f"T{c[9]}-H{c[1]}-d{c[4]}" for c in EDGE])
def test_prefill_tile_edges(case):
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


@pytest.mark.parametrize("shape", [
    # seed, hidden, heads, kv, d, ffn, fracs, device, ctx, T
    (307, 512, 8, 4, 64, 700, (0.5, 0.5), 1, 30, 37),
    (309, 1032, 4, 2, 128, 900, (0.5, 0.5), 0, 11, 130),   # hidden a multiple of 8, not 16
], ids=["h512", "h1032"])
def test_prefill_attention_then_ffn_calls(shape):
    """The two sub-layers as separate calls: VT_ATTN alone (the O GEMM's
    epilogue without the FFN input), then VT_FFN alone from the device's h
    (the RMSNorm before the gate/up GEMM computed on its own); the FFN is
    checked against the oracle's FFN sub-layer at exactly that h."""
    seed, H, nh, nkv, hd, F, fr, dev, ctx, T = shape
    wl = tiny_workload(seed, H, nh, nkv, hd, F, fr, dev, ctx, sigma=0.03, chunk=T)
    li = LayerInputs(wl)
    d = wl.dims
    r = oracle_ranges(wl)
    w = oracle_shard_weights(li, r)
    kc, vc = li.kv_context_heads(r.kv_head_begin, r.kv_head_begin + r.n_kv_heads)
    X = li.x_chunk(T)
    pa, pf = li.peer("attn", rows=T), li.peer("ffn", rows=T)
    ref = oracle.prefill(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, X, kc,
                         vc, wl.ctx, pa, pf)
    gs = GpuShard(wl, li=li, capacity=wl.ctx + T + 3, max_tokens=T)
    a = gs.prefill(X, wl.ctx, vt.VT_ATTN, peer_attn=pa)
    for k in ("p_attn", "h"):
        assert_close(a[k], ref[k], k)
    assert np.isnan(a["p_ffn"]).all() and np.isnan(a["y"]).all()  # not written
    assert gs.kv.len == wl.ctx + T
    f = gs.prefill(None, wl.ctx, vt.VT_FFN, peer_ffn=pf, h_in=a["h"])
    fr = ffn_at_h16(w, d.rms_eps, {"h": a["h"]}, pf)
    for k in ("p_ffn", "y"):
        assert_close(f[k], fr[k], k)
    assert gs.kv.len == wl.ctx + T


def test_prefill_ignores_row_padding():
    """Down-projection rows padded past the shard's columns (not a multiple
    of 8 here) with NaN: the k-chunk that straddles the column count is
    masked, so the outputs match the oracle."""
    wl = tiny_workload(308, 1024, 8, 4, 128, 1501, (0.6, 0.4), 0, 40, sigma=0.03, chunk=70)
    li = LayerInputs(wl)
    r = oracle_ranges(wl)
    assert r.n_cols % 8 != 0
    gs_probe = GpuShard(wl, li=li, capacity=wl.ctx + 73, max_tokens=70)
    wd = gs_probe.w.tensors["wd"]
    assert wd.shape[1] > r.n_cols
    wd[:, r.n_cols:] = float("nan")
    torch.cuda.synchronize()
    # the same case as run_case, on the shard whose padding now holds NaN
    d = wl.dims
    w = oracle_shard_weights(li, r)
    kc, vc = li.kv_context_heads(r.kv_head_begin, r.kv_head_begin + r.n_kv_heads)
    X = li.x_chunk(70)
    ref = ffn_at_h16(w, d.rms_eps, oracle.prefill(w, r.n_q_heads, r.n_kv_heads, d.head_dim,
                                                  d.rms_eps, d.rope_base, X, kc, vc, wl.ctx))
    got = gs_probe.prefill(X, wl.ctx, BOTH)
    for k in ("p_attn", "h", "p_ffn", "y"):
        assert np.isfinite(got[k]).all(), k
        assert_close(got[k], ref[k], k)


def test_prefill_repeat_is_bitwise():
    """The split-K slices of an output tile are added in slice order by
    whichever arrives last: the same chunk twice gives the same bits."""
    wl = get("7b_prefill")
    li = LayerInputs(wl)
    gs = GpuShard(wl, li=li, capacity=wl.ctx + wl.chunk, max_tokens=wl.chunk)
    X = li.x_chunk(wl.chunk)
    outs, caches = [], []
    for _ in range(2):
        outs.append(gs.prefill(X, wl.ctx, BOTH))
        caches.append(gs.cache())
        gs.kv.len = wl.ctx
    for k in ("p_attn", "h", "p_ffn", "y"):
        assert np.array_equal(outs[0][k], outs[1][k]), k
    assert np.array_equal(caches[0][0], caches[1][0]) and np.array_equal(caches[0][1], caches[1][1])
    assert not gs.sync_words().any()


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
