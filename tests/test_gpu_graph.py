"""HIP-graph replays of the library's persistent kernels (the way the bench
runs them): each entry point is captured once, then the graph is replayed
several times with unrelated eager work and synchronisations in between;
every replay must reproduce the eager call bit for bit, and the
workspace's synchronisation words must be zero after each replay (the
kernels clear them with ordinary stores; nothing in a graph is a memset).
"""
import numpy as np
import pytest
import torch

from paper_2607_07046_amd import voltron as vt
from synth import get
from tests.gpu_common import GpuShard, h16, ptr
from tests.test_gpu_moe import GpuMoE, small, CachedInputs

pytestmark = pytest.mark.gpu

REPLAYS = 3


def replay_matches_eager(enqueue, outputs, sync_words, before=lambda: None, kept=()):
    """enqueue(stream) issues the call; outputs: device tensors it writes
    (poisoned before each replay); kept: tensors it updates in place (a KV
    cache: the replay rewrites the same slots), compared but not poisoned."""
    before()
    enqueue(torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    want = [o.clone() for o in outputs]
    want_kept = [o.clone() for o in kept]
    assert np.all(sync_words() == 0)
    before()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        enqueue(torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    a = torch.randn(512, 512, device="cuda")
    for r in range(REPLAYS):
        for o in outputs:
            o.view(torch.int16).fill_(0x7E00)          # NaN pattern, eager
        b = (a @ a).sum()                              # unrelated eager work
        torch.cuda.synchronize()
        assert torch.isfinite(b)
        g.replay()
        torch.cuda.synchronize()
        for i, (o, w) in enumerate(zip(list(outputs) + list(kept), want + want_kept)):
            assert torch.equal(o.view(torch.int16), w.view(torch.int16)), (r, i)
        assert np.all(sync_words() == 0), r


def io_for(H, T=1):
    shape = (T, H) if T > 1 else (H,)
    return {k: torch.empty(shape, dtype=torch.float16, device="cuda")
            for k in ("p_attn", "h", "p_ffn", "y")}


@pytest.mark.parametrize("prec", [None, vt.VT_W_INT8, vt.VT_W_INT4])
def test_decode_graph_replays(prec):
    wl = get("7b")
    gs = GpuShard(wl, capacity=wl.ctx + 1, prec=prec)
    x = h16(gs.li.x(0))
    out = io_for(gs.dims.hidden)
    io = vt.vt_layer_io(x=ptr(x), peer_attn=None, peer_ffn=None, attn_partial=ptr(out["p_attn"]),
                        h=ptr(out["h"]), ffn_partial=ptr(out["p_ffn"]), y=ptr(out["y"]))
    pos = wl.ctx

    def reset():
        gs.kv.len = pos

    def enqueue(stream):
        if prec is None:
            vt.vt_layer_decode(gs.spec, gs.w.struct, gs.kv, io, pos, vt.VT_ATTN | vt.VT_FFN,
                               ptr(gs.ws), gs.ws_bytes, stream)
        else:
            vt.vt_layer_decode_q(gs.spec, gs.qw.struct, gs.kv, io, pos, vt.VT_ATTN | vt.VT_FFN,
                                 ptr(gs.ws), gs.ws_bytes, stream)

    replay_matches_eager(enqueue, list(out.values()), gs.sync_words, reset, kept=(gs.kc, gs.vc))


def test_prefill_graph_replays():
    wl = get("tiny")
    T = 48
    gs = GpuShard(wl, capacity=wl.ctx + T, max_tokens=T)
    X = h16(np.stack([gs.li.x(t) for t in range(T)]))
    out = io_for(gs.dims.hidden, T)
    io = vt.vt_layer_io(x=ptr(X), peer_attn=None, peer_ffn=None, attn_partial=ptr(out["p_attn"]),
                        h=ptr(out["h"]), ffn_partial=ptr(out["p_ffn"]), y=ptr(out["y"]))
    pos0 = wl.ctx

    def reset():
        gs.kv.len = pos0

    def enqueue(stream):
        vt.vt_layer_prefill_chunk(gs.spec, gs.w.struct, gs.kv, io, T, pos0, vt.VT_ATTN | vt.VT_FFN,
                                  ptr(gs.ws), gs.ws_bytes, stream)

    replay_matches_eager(enqueue, list(out.values()), gs.sync_words, reset, kept=(gs.kc, gs.vc))


def test_moe_graph_replays():
    wl = small(971, 512, 16, 700, 4, (0.4, 0.6))
    mi = CachedInputs(wl)
    g = GpuMoE(mi, 1)
    H = wl.hidden
    h = h16(mi.h(0))
    p = torch.empty(H, dtype=torch.float16, device="cuda")
    y = torch.empty(H, dtype=torch.float16, device="cuda")
    sel = torch.empty(wl.top_k, dtype=torch.int32, device="cuda")
    io = vt.vt_layer_io(x=None, peer_attn=None, peer_ffn=None, attn_partial=None, h=ptr(h),
                        ffn_partial=ptr(p), y=ptr(y))

    def enqueue(stream):
        vt.vt_moe_ffn_decode(g.spec, g.w.struct, wl.n_experts, wl.top_k, io, ptr(sel), None,
                             ptr(g.ws), g.ws_bytes, stream)

    def sync_words():
        return g.ws[:4 * 3104].view(torch.int32).cpu().numpy()

    replay_matches_eager(enqueue, [p, y, sel], sync_words)
