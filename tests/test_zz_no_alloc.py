"""vt_layer_decode_noalloc (the decode step with its workspace in the
library's own scratch array, for callers that cannot allocate) against
vt_layer_decode with a caller workspace: the same kernels, so outputs and
caches must agree bit for bit. Two calls in a row on one GPU share the
scratch array: the 7B-shaped 30% shard at position 1024, then a smaller
input (the tiny shard at position 128, fewer heads and a shorter context),
then the large one again; every call's barrier error word is zero.
"""
import numpy as np
import pytest
import torch

from paper_2607_07046_amd import voltron as vt
from synth import get
from synth.gen import LayerInputs
from tests.gpu_common import GpuShard, h16, ptr

pytestmark = pytest.mark.gpu
BOTH = vt.VT_ATTN | vt.VT_FFN


def decode_noalloc(gs, x):
    """gs.decode's outputs, computed by vt_layer_decode_noalloc."""
    H = gs.dims.hidden
    xt = h16(x)
    out = {k: torch.full((H,), float("nan"), dtype=torch.float16, device="cuda")
           for k in ("p_attn", "h", "p_ffn", "y")}
    err = torch.full((1,), 0x7777, dtype=torch.int32, device="cuda")
    io = vt.vt_layer_io(x=ptr(xt), peer_attn=None, peer_ffn=None,
                        attn_partial=ptr(out["p_attn"]), h=ptr(out["h"]),
                        ffn_partial=ptr(out["p_ffn"]), y=ptr(out["y"]))
    vt.vt_layer_decode_noalloc(gs.spec, gs.w.struct, gs.kv, io, gs.kv.len, BOTH, err.data_ptr(),
                               None)
    torch.cuda.synchronize()
    assert int(err.item()) == 0, "a barrier wait expired"
    return {k: v.float().cpu().numpy().astype(np.float64) for k, v in out.items()}


def test_noalloc_matches_workspace_decode_on_consecutive_calls():
    cases = []
    for key in ("7b", "tiny", "7b"):   # the second call's input is smaller than the first's
        wl = get(key)
        li = LayerInputs(wl)
        x = li.x(3)
        a = GpuShard(wl, li=li)            # with its own workspace
        b = GpuShard(wl, li=li)            # the same shard and cache, for the scratch path
        ga = a.decode(x, wl.ctx, BOTH)
        gb = decode_noalloc(b, x)
        cases.append((key, ga, gb, a.cache(), b.cache(), a.kv.len, b.kv.len))
    for key, ga, gb, ca, cb, la, lb in cases:
        for k in ("p_attn", "h", "p_ffn", "y"):
            assert np.all(np.isfinite(gb[k])), (key, k)
            assert np.array_equal(ga[k], gb[k]), (key, k)
        assert np.array_equal(ca[0], cb[0]) and np.array_equal(ca[1], cb[1]), key
        assert la == lb == get(key).ctx + 1, key


def test_noalloc_on_random_shapes():
    """Seeded random layer shapes (hidden sizes that are multiples of 8 only,
    GQA groups up to 8, sliding windows) in a row through the scratch array:
    each equals the decode with a caller workspace bit for bit."""
    from tests.test_gpu_random_shapes import SHAPES
    for wl in SHAPES[:6] + SHAPES[12:15]:
        li = LayerInputs(wl)
        x = li.x(5)
        a = GpuShard(wl, li=li)
        b = GpuShard(wl, li=li)
        ga = a.decode(x, wl.ctx, BOTH)
        gb = decode_noalloc(b, x)
        for k in ("p_attn", "h", "p_ffn", "y"):
            assert np.array_equal(ga[k], gb[k]), (wl.key, k)
        ca, cb = a.cache(), b.cache()
        assert np.array_equal(ca[0], cb[0]) and np.array_equal(ca[1], cb[1]), wl.key
