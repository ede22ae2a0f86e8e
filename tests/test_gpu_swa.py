"""GPU parity of sliding-window decode attention (vt_layer_dims.window > 0:
a token attends to the last ``window`` positions; the local layers of the
gemma models of the paper's Table 3) against the fp64 oracle, through the C
ABI: the 7B-shaped 30% shard with window 1024 at position 4096, a tiny
GQA layer with windows shorter than the context, fused and staged; a window
covering the whole context gives bit for bit the output of full attention;
a window of one attends to the new token only.
"""
import dataclasses

import numpy as np
import pytest

import oracle
from paper_2607_07046_amd import voltron as vt
from synth import get
from synth.configs import LayerDims, Workload
from synth.gen import LayerInputs
from tests.common import assert_close, ffn_at_h16, oracle_decode, oracle_ranges, oracle_shard_weights
from tests.gpu_common import GpuShard

pytestmark = pytest.mark.gpu

BOTH = vt.VT_ATTN | vt.VT_FFN


def tiny_swa(window, ctx=300, seed=961):
    return Workload(key=f"tiny_swa{window}", seed_id=seed, title="tiny sliding-window layer",
                    dims=LayerDims(hidden=512, n_heads=8, n_kv_heads=4, head_dim=64, ffn=1376,
                                   window=window),
                    fracs=(0.5, 0.5), device=1, weight_sigma=0.03, ctx=ctx)


def check(wl, phases=BOTH):
    li = LayerInputs(wl)
    gs = GpuShard(wl, li=li)
    x = li.x(0)
    got = gs.decode(x, wl.ctx, phases)
    kc, vc = gs.context()
    ref = oracle_decode(wl, li, oracle_ranges(wl), x, kc, vc, wl.ctx)
    for k in ("p_attn", "h", "p_ffn", "y"):
        assert_close(got[k], ref[k], f"{wl.key} {k}")
    return got


def test_7b_window_1024_at_4096():
    check(get("7b_swa"))


@pytest.mark.parametrize("mode", [0, vt.VT_STAGED])
@pytest.mark.parametrize("window", [1, 37, 64, 129])
def test_tiny_windows(window, mode):
    check(tiny_swa(window), BOTH | mode)


@pytest.mark.parametrize("mode", [0, vt.VT_STAGED])
def test_window_after_a_million_positions(mode):
    """A window of 4096 at position 1,000,000: the attended range starts
    far into the cache (the first 995,905 positions are never read)."""
    check(tiny_swa(4096, ctx=1_000_000, seed=962), BOTH | mode)


def test_window_covering_context_is_full_attention():
    a = check(tiny_swa(301))                       # positions 0..300: all of them
    b = check(dataclasses.replace(tiny_swa(301), dims=dataclasses.replace(tiny_swa(301).dims,
                                                                             window=0)))
    for k in ("p_attn", "h", "p_ffn", "y"):
        assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("window", [1, 40, 100, 1000])
def test_prefill_chunk_window(window):
    """A 128-token prefill chunk at positions 200..327 of a sliding-window
    layer (windows shorter than a query block, than the chunk, than the
    context, and longer than everything)."""
    wl = tiny_swa(window, ctx=200)
    d = wl.dims
    li = LayerInputs(wl)
    gs = GpuShard(wl, li=li, capacity=wl.ctx + 128, max_tokens=128)
    X = np.stack([li.x(t) for t in range(128)])
    got = gs.prefill(X, wl.ctx)
    r = oracle_ranges(wl)
    kc, vc = gs.context()
    w = oracle_shard_weights(li, r)
    ref = oracle.prefill(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, X, kc,
                         vc, wl.ctx, window=window)
    ref = ffn_at_h16(w, d.rms_eps, ref)
    for k in ("p_attn", "h", "p_ffn", "y"):   # every row of the chunk
        assert_close(got[k], ref[k], f"window {window} {k}")


@pytest.mark.parametrize("window,T", [(33, 77), (200, 161)])
def test_prefill_window_ragged_gqa(window, T):
    """A ragged chunk (77 / 161 tokens: a partial last query block) of a GQA
    layer with head size 128, hidden 1032 and a window that ends inside a key
    block, at positions 150.. ."""
    wl = Workload(key=f"swa_ragged{window}", seed_id=962, title="ragged sliding-window GQA layer",
                  dims=LayerDims(hidden=1032, n_heads=12, n_kv_heads=4, head_dim=128, ffn=900,
                                 window=window),
                  fracs=(0.5, 0.5), device=0, weight_sigma=0.03, ctx=150)
    d = wl.dims
    li = LayerInputs(wl)
    gs = GpuShard(wl, li=li, capacity=wl.ctx + T, max_tokens=T)
    X = np.stack([li.x(t) for t in range(T)])
    got = gs.prefill(X, wl.ctx)
    r = oracle_ranges(wl)
    kc, vc = gs.context()
    w = oracle_shard_weights(li, r)
    ref = oracle.prefill(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, X, kc,
                         vc, wl.ctx, window=window)
    ref = ffn_at_h16(w, d.rms_eps, ref)
    for k in ("p_attn", "h", "p_ffn", "y"):
        assert_close(got[k], ref[k], f"window {window} T {T} {k}")
