"""GPU checks of vt_stack_decode: several layers of one shard shape decoded
for one token in a single persistent launch (layer l's y is layer l+1's x).

* Bit for bit equal to the same layers run one vt_layer_decode call each,
  every call fed the previous call's y (outputs of every layer and both
  caches), over consecutive tokens: a tiny GQA stack, a stack of one layer,
  and four layers of the 13B-shaped 40% shard at positions 2048...
* The first layer (whose input is the caller's x) matches the oracle at the
  single-layer bar; deeper layers inherit the per-layer kernels' parity,
  which the teacher-forced stack tests check on all 40 13B-shaped layers.
* The KV stack's len advances once per token; the workspace's
  synchronisation words are left zero.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_07046_amd import pack
from paper_2607_07046_amd import voltron as vt
from synth import get
from synth.gen import LayerInputs
from tests.common import assert_close, ffn_at_h16, oracle_ranges, oracle_shard_weights, \
    tiny_workload
from tests.gpu_common import lib_dims
from tests.test_gpu_random_shapes import IDS as RANDOM_IDS, SHAPES as RANDOM_SHAPES

pytestmark = pytest.mark.gpu
KEYS = ("p_attn", "h", "p_ffn", "y")


class Stack:
    def __init__(self, wl, n_layers, cap):
        self.wl = wl
        self.spec = vt.vt_shard_spec_create(lib_dims(wl.dims), wl.fracs, wl.fracs, wl.device)
        self.dims, self.info = vt.vt_shard_spec_query(self.spec)
        self.L = n_layers
        self.lis = [LayerInputs(wl, l) for l in range(n_layers)]
        self.w = pack.pack_stack(self.lis, self.dims, self.info)
        nkv, d = self.info.n_kv_heads, self.dims.head_dim
        self.cap = cap
        self.ctx = [li.kv_context_heads(self.info.kv_head_begin, self.info.kv_head_begin + nkv)
                    for li in self.lis]
        self.ws_bytes = vt.vt_workspace_size(self.spec, 1, cap)

    def caches(self):
        nkv, d = self.info.n_kv_heads, self.dims.head_dim
        kc = torch.zeros((self.L, nkv, self.cap, d), dtype=torch.float16, device="cuda")
        vc = torch.zeros_like(kc)
        for l, (k, v) in enumerate(self.ctx):
            kc[l, :, :self.wl.ctx] = torch.from_numpy(k).cuda()
            vc[l, :, :self.wl.ctx] = torch.from_numpy(v).cuda()
        return kc, vc

    def run_stack(self, xs):
        """vt_stack_decode of each token x in xs; outputs [T][L][H]."""
        H = self.dims.hidden
        kc, vc = self.caches()
        kv = vt.vt_kv_stack(k=kc.data_ptr(), v=vc.data_ptr(), n_layers=self.L, capacity=self.cap,
                            n_kv_heads=self.info.n_kv_heads, head_dim=self.dims.head_dim,
                            len=self.wl.ctx)
        ws = torch.zeros(self.ws_bytes, dtype=torch.uint8, device="cuda")
        outs = []
        for t, x in enumerate(xs):
            xt = torch.from_numpy(x).cuda()
            o = {k: torch.full((self.L, H), float("nan"), dtype=torch.float16, device="cuda")
                 for k in KEYS}
            io = vt.vt_layer_io(x=xt.data_ptr(), peer_attn=None, peer_ffn=None,
                                attn_partial=o["p_attn"].data_ptr(), h=o["h"].data_ptr(),
                                ffn_partial=o["p_ffn"].data_ptr(), y=o["y"].data_ptr())
            vt.vt_stack_decode(self.spec, self.w.struct, kv, io, self.wl.ctx + t, ws.data_ptr(),
                               self.ws_bytes, None)
            torch.cuda.synchronize()
            outs.append({k: v.cpu().numpy() for k, v in o.items()})
        assert kv.len == self.wl.ctx + len(xs)
        sync = ws[:4 * (3072 + 32 * (self.info.n_q_heads + 1))].view(torch.int32).cpu().numpy()
        assert not sync.any(), "synchronisation or error words left set"
        return outs, kc.cpu().numpy(), vc.cpu().numpy()

    def run_chain(self, xs):
        """The same layers, one vt_layer_decode per layer and token."""
        H = self.dims.hidden
        kc, vc = self.caches()
        kvs = [vt.vt_kv_view(k=kc[l].data_ptr(), v=vc[l].data_ptr(), capacity=self.cap,
                             n_kv_heads=self.info.n_kv_heads, head_dim=self.dims.head_dim,
                             len=self.wl.ctx) for l in range(self.L)]
        ws = torch.zeros(self.ws_bytes, dtype=torch.uint8, device="cuda")
        outs = []
        for t, x in enumerate(xs):
            o = {k: torch.full((self.L, H), float("nan"), dtype=torch.float16, device="cuda")
                 for k in KEYS}
            xin = torch.from_numpy(x).cuda()
            for l in range(self.L):
                io = vt.vt_layer_io(x=xin.data_ptr(), peer_attn=None, peer_ffn=None,
                                    attn_partial=o["p_attn"][l].data_ptr(),
                                    h=o["h"][l].data_ptr(), ffn_partial=o["p_ffn"][l].data_ptr(),
                                    y=o["y"][l].data_ptr())
                vt.vt_layer_decode(self.spec, self.w.layer(l), kvs[l], io, self.wl.ctx + t,
                                   vt.VT_ATTN | vt.VT_FFN, ws.data_ptr(), self.ws_bytes, None)
                xin = o["y"][l]
            torch.cuda.synchronize()
            outs.append({k: v.cpu().numpy() for k, v in o.items()})
        return outs, kc.cpu().numpy(), vc.cpu().numpy()


def check_equal(stack, n_tok):
    xs = [stack.lis[0].x(t) for t in range(n_tok)]
    a, ka, va = stack.run_stack(xs)
    b, kb, vb = stack.run_chain(xs)
    for t in range(n_tok):
        for k in KEYS:
            assert np.all(np.isfinite(a[t][k].astype(np.float32))), (t, k)
            assert np.array_equal(a[t][k].view(np.int16), b[t][k].view(np.int16)), (t, k)
    assert np.array_equal(ka.view(np.int16), kb.view(np.int16))
    assert np.array_equal(va.view(np.int16), vb.view(np.int16))
    return a


def check_first_layer(stack, outs, n_tok):
    """Layer 0 against the oracle (its inputs are the caller's exact x)."""
    wl, d = stack.wl, stack.wl.dims
    li = stack.lis[0]
    r = oracle_ranges(wl)
    w = oracle_shard_weights(li, r)
    kc, vc = stack.ctx[0]
    X = np.stack([li.x(t) for t in range(n_tok)]).astype(np.float64)
    ref = oracle.prefill(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, X, kc,
                         vc, wl.ctx, window=d.window)
    ref = ffn_at_h16(w, d.rms_eps, ref)
    for k in KEYS:
        got = np.stack([o[k][0] for o in outs]).astype(np.float64)
        assert_close(got, ref[k], f"stack layer 0 {k}")


def test_tiny_gqa_stack_equals_layer_chain():
    wl = tiny_workload(501, 512, 8, 2, 64, 1000, (0.6, 0.4), 0, 40, sigma=0.03)
    st = Stack(wl, 3, wl.ctx + 4)
    outs = check_equal(st, 4)
    check_first_layer(st, outs, 4)


def test_one_layer_stack_equals_layer_decode():
    wl = tiny_workload(502, 1024, 16, 4, 64, 3000, (0.37, 0.33, 0.30), 2, 150, sigma=0.03)
    st = Stack(wl, 1, wl.ctx + 2)
    outs = check_equal(st, 2)
    check_first_layer(st, outs, 2)


def test_ragged_hidden_stack_equals_layer_chain():
    # hidden a multiple of 8 but not of 16 (the last weight piece of every
    # K = hidden row and the next layer's x staging are ragged)
    wl = tiny_workload(504, 1032, 4, 2, 128, 900, (0.5, 0.5), 1, 20, sigma=0.03)
    st = Stack(wl, 3, wl.ctx + 3)
    outs = check_equal(st, 3)
    check_first_layer(st, outs, 3)


@pytest.mark.parametrize("wl", RANDOM_SHAPES[:4], ids=RANDOM_IDS[:4])
def test_random_shape_stack_equals_layer_chain(wl):
    # the first two shapes have sliding windows (1 and 160 positions)
    st = Stack(wl, 3, wl.ctx + 3)
    outs = check_equal(st, 3)
    check_first_layer(st, outs, 3)


def test_13b_four_layers_equal_layer_chain():
    wl = get("13b_stack")
    st = Stack(wl, 4, wl.ctx + 3)
    outs = check_equal(st, 3)
    check_first_layer(st, outs, 3)


def test_stack_rejects_bad_arguments():
    wl = tiny_workload(503, 512, 8, 8, 64, 600, (0.5, 0.5), 0, 4)
    st = Stack(wl, 2, 6)
    kc, vc = st.caches()
    H = st.dims.hidden
    x = torch.zeros(H, dtype=torch.float16, device="cuda")
    o = torch.zeros((2, H), dtype=torch.float16, device="cuda")
    ws = torch.zeros(st.ws_bytes, dtype=torch.uint8, device="cuda")
    io = vt.vt_layer_io(x=x.data_ptr(), peer_attn=None, peer_ffn=None, attn_partial=o.data_ptr(),
                        h=o.data_ptr(), ffn_partial=o.data_ptr(), y=o.data_ptr())
    bad_layers = vt.vt_kv_stack(k=kc.data_ptr(), v=vc.data_ptr(), n_layers=3, capacity=6,
                                n_kv_heads=st.info.n_kv_heads, head_dim=64, len=4)
    with pytest.raises(vt.VoltronError) as e:
        vt.vt_stack_decode(st.spec, st.w.struct, bad_layers, io, 4, ws.data_ptr(), st.ws_bytes)
    assert e.value.status == vt.VT_ERR_ARG
    kv = vt.vt_kv_stack(k=kc.data_ptr(), v=vc.data_ptr(), n_layers=2, capacity=6,
                        n_kv_heads=st.info.n_kv_heads, head_dim=64, len=4)
    with pytest.raises(vt.VoltronError) as e:
        vt.vt_stack_decode(st.spec, st.w.struct, kv, io, 3, ws.data_ptr(), st.ws_bytes)
    assert e.value.status == vt.VT_ERR_POS
    io.y = None
    with pytest.raises(vt.VoltronError) as e:
        vt.vt_stack_decode(st.spec, st.w.struct, kv, io, 4, ws.data_ptr(), st.ws_bytes)
    assert e.value.status == vt.VT_ERR_ARG
    assert kv.len == 4
