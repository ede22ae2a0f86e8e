"""GPU parity on seeded random layer shapes (decode step and prefill chunk
against the fp64 oracle, through the C ABI).

Shapes drawn once from a fixed seed: hidden any multiple of 8 from 128 to
3200, 1-8 KV heads with 1-8 query heads each, head size 64 or 128, 64-4000
FFN columns, 1-4 devices with random fractions, contexts of 0-700
positions, chunks of 1-300 tokens, sometimes a sliding window; the bar is
the derived one of tests/common.py. Weights are drawn with standard
deviation 1/sqrt(hidden), as a trained layer's are scaled with its fan-in,
so that queries, keys and attention logits keep the spread of the paper's
workloads at every hidden size (the bar's error model assumes that spread:
at a fixed 0.03 and hidden 3144 the logits are three times wider, and the
prefill p_attn error grows past it by rounding alone, as an fp16 model of
the kernel's rounding points reproduces). The drawn shard must hold at
least one head and one FFN column (prefill needs both).
"""
import numpy as np
import pytest

import oracle
from paper_2607_07046_amd import voltron as vt
from synth.configs import LayerDims, Workload
from synth.gen import LayerInputs
from tests.common import assert_close, ffn_at_h16, oracle_decode, oracle_ranges, oracle_shard_weights
from tests.gpu_common import GpuShard

pytestmark = pytest.mark.gpu
KEYS = ("p_attn", "h", "p_ffn", "y")


def _draw(n=12, seed=20261204, small=False):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        nkv = int(rng.integers(1, 9)) if not small else int(rng.integers(1, 3))
        G = int(rng.integers(1, 9)) if not small else int(rng.integers(1, 4))
        d = int(rng.choice([64, 128]))
        H = 8 * int(rng.integers(16, 401)) if not small else 8 * int(rng.integers(2, 65))
        F = int(rng.integers(64, 4001)) if not small else int(rng.integers(1, 200))
        ndev = int(rng.integers(1, 5))
        fr = rng.dirichlet(np.ones(ndev))
        fr = tuple(float(round(f, 3)) for f in fr)
        fr = fr[:-1] + (round(1.0 - sum(fr[:-1]), 3),)
        dev = int(rng.integers(0, ndev))
        ctx = int(rng.integers(0, 701)) if not small else int(rng.integers(0, 40))
        T = int(rng.integers(1, 301)) if not small else int(rng.integers(1, 41))
        window = int(rng.choice([0, 0, 0, int(rng.integers(1, 400))]))
        wl = Workload(key=f"rand{'s' if small else ''}{len(out)}", seed_id=(760 if small else 700) + len(out),
                      title="random test layer",
                      dims=LayerDims(hidden=H, n_heads=nkv * G, n_kv_heads=nkv, head_dim=d, ffn=F,
                                     window=window),
                      fracs=fr, device=dev, weight_sigma=float(1.0 / np.sqrt(H)), ctx=ctx, chunk=T)
        try:
            r = oracle_ranges(wl)
        except Exception:
            continue
        if r.n_q_heads == 0 or r.n_cols == 0 or min(fr) <= 0:
            continue
        out.append(wl)
    return out


# the main draw, then small layers (hidden 16-512, 1-2 KV heads, FFN shares
# down to a single column, contexts and chunks under 40 positions)
SHAPES = _draw() + _draw(n=8, seed=20261206, small=True)
IDS = [f"{w.key}-H{w.dims.hidden}-kv{w.dims.n_kv_heads}x{w.dims.n_heads // w.dims.n_kv_heads}-"
       f"d{w.dims.head_dim}-F{w.dims.ffn}-n{len(w.fracs)}-c{w.ctx}-T{w.chunk}-w{w.dims.window}"
       for w in SHAPES]


@pytest.mark.parametrize("wl", SHAPES, ids=IDS)
def test_random_shape_decode_and_prefill(wl):
    d = wl.dims
    li = LayerInputs(wl)
    r = oracle_ranges(wl)
    w = oracle_shard_weights(li, r)
    # decode at position ctx, with the other devices' partials; the staged
    # and the cooperative launches give the same bits as the fused one
    x = li.x(0)
    pa, pf = li.peer("attn"), li.peer("ffn")
    runs = []
    for flags in (0, vt.VT_STAGED, vt.VT_COOPERATIVE):
        gs = GpuShard(wl, li=li)
        runs.append(gs.decode(x, wl.ctx, vt.VT_ATTN | vt.VT_FFN | flags, peer_attn=pa, peer_ffn=pf))
        assert not gs.sync_words().any()
    got = runs[0]
    for other in runs[1:]:
        for k in KEYS:
            assert np.array_equal(other[k], got[k]), k
    kc, vc = gs.context()
    ref = oracle_decode(wl, li, r, x, kc, vc, wl.ctx, peer_attn=pa, peer_ffn=pf, w=w)
    for k in KEYS:
        assert_close(got[k], ref[k], f"decode {k}")
    # a prefill chunk of T tokens at positions ctx.. on a fresh cache
    T = wl.chunk
    gp = GpuShard(wl, li=li, capacity=wl.ctx + T, max_tokens=T)
    X = li.x_chunk(T)
    qa, qf = li.peer("attn", rows=T), li.peer("ffn", rows=T)
    got = gp.prefill(X, wl.ctx, peer_attn=qa, peer_ffn=qf)
    refp = oracle.prefill(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, X, kc,
                          vc, wl.ctx, qa, qf, window=d.window)
    refp = ffn_at_h16(w, d.rms_eps, refp, qf)
    for k in KEYS:
        assert_close(got[k], refp[k], f"prefill {k}")
    kc1, vc1 = gp.cache()
    rng_ = slice(wl.ctx, wl.ctx + T)
    kn = np.transpose(kc1[:, rng_].view(np.float16).astype(np.float64), (1, 0, 2)).reshape(T, -1)
    vn = np.transpose(vc1[:, rng_].view(np.float16).astype(np.float64), (1, 0, 2)).reshape(T, -1)
    assert_close(kn, refp["k_new"].reshape(T, -1), "appended keys")
    assert_close(vn, refp["v_new"].reshape(T, -1), "appended values")
