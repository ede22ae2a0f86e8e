"""GPU-side test harness: one shard of a workload on the device, driven
through the C ABI. The shard's ranges come from the library's spec; the
weights and cache contents come from the seeded generator (never from the
oracle or vice versa).
"""
import numpy as np
import torch

from paper_2607_07046_amd import pack
from paper_2607_07046_amd import voltron as vt
from synth.gen import LayerInputs

SENTINEL = 0x3C01  # fp16 bit pattern left in unused cache slots


def lib_dims(wd) -> vt.vt_layer_dims:
    return vt.vt_layer_dims(hidden=wd.hidden, n_heads=wd.n_heads, n_kv_heads=wd.n_kv_heads,
                            head_dim=wd.head_dim, ffn=wd.ffn, rms_eps=wd.rms_eps,
                            rope_base=wd.rope_base, window=wd.window)


def h16(a):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, np.float16))).cuda()


def ptr(t):
    return None if t is None else t.data_ptr()


class GpuShard:
    """Device ``device`` of workload ``wl``: packed weights, KV cache, workspace."""

    def __init__(self, wl, device=None, layer=0, li=None, capacity=None, fill_ctx=True,
                 max_tokens=1, fracs=None, prec=None):
        self.wl = wl
        self.li = li or LayerInputs(wl, layer)
        fr = fracs or wl.fracs
        self.spec = vt.vt_shard_spec_create(lib_dims(wl.dims), fr, fr,
                                            wl.device if device is None else device)
        self.dims, self.info = vt.vt_shard_spec_query(self.spec)
        self.w = pack.pack_shard(self.li, self.dims, self.info)
        # prec (VT_W_INT8 / VT_W_INT4): decode through the block-quantised
        # weights the library's quantiser makes from the fp16 shard
        self.prec = prec
        self.qw = pack.quantize_shard(self.w, self.dims, self.info, prec) if prec else None
        d, nkv = self.dims.head_dim, self.info.n_kv_heads
        self.cap = capacity or wl.capacity
        sent = torch.full((nkv, self.cap, d), SENTINEL, dtype=torch.int16, device="cuda")
        self.kc = sent.view(torch.float16).clone()
        self.vc = sent.view(torch.float16).clone()
        self.kv = vt.vt_kv_view(k=ptr(self.kc) if self.kc.numel() else None,
                                v=ptr(self.vc) if self.vc.numel() else None, capacity=self.cap,
                                n_kv_heads=nkv, head_dim=d, len=0)
        self.ws_bytes = vt.vt_workspace_size(self.spec, max_tokens, self.cap)
        self.ws = torch.zeros(self.ws_bytes, dtype=torch.uint8, device="cuda")
        if fill_ctx and wl.ctx > 0:
            k, v = self.context()
            self.append(np.transpose(k, (1, 0, 2)), np.transpose(v, (1, 0, 2)))

    def context(self):
        g0 = self.info.kv_head_begin
        return self.li.kv_context_heads(g0, g0 + self.info.n_kv_heads)

    def append(self, k_tnd, v_tnd):
        """vt_kv_append of [n_tok][n_kv][d] host arrays at the current length."""
        n = k_tnd.shape[0]
        kt, vt_ = h16(k_tnd), h16(v_tnd)
        vt.vt_kv_append(self.kv, ptr(kt) if kt.numel() else None,
                        ptr(vt_) if vt_.numel() else None, n, self.kv.len, None)
        torch.cuda.synchronize()

    def decode(self, x, pos=None, phases=vt.VT_ATTN | vt.VT_FFN, peer_attn=None, peer_ffn=None,
               h_in=None, want_y=True):
        H = self.dims.hidden
        pos = self.kv.len if pos is None else pos
        xt = h16(x) if x is not None else torch.zeros(H, dtype=torch.float16, device="cuda")
        pa = h16(peer_attn) if peer_attn is not None else None
        pf = h16(peer_ffn) if peer_ffn is not None else None
        out = {k: torch.full((H,), float("nan"), dtype=torch.float16, device="cuda")
               for k in ("p_attn", "h", "p_ffn", "y")}
        if h_in is not None:
            out["h"] = h16(h_in)
        io = vt.vt_layer_io(x=ptr(xt), peer_attn=ptr(pa), peer_ffn=ptr(pf),
                            attn_partial=ptr(out["p_attn"]), h=ptr(out["h"]),
                            ffn_partial=ptr(out["p_ffn"]), y=ptr(out["y"]) if want_y else None)
        if self.qw is not None:
            vt.vt_layer_decode_q(self.spec, self.qw.struct, self.kv, io, pos, phases,
                                 ptr(self.ws), self.ws_bytes, None)
        else:
            vt.vt_layer_decode(self.spec, self.w.struct, self.kv, io, pos, phases, ptr(self.ws),
                               self.ws_bytes, None)
        torch.cuda.synchronize()
        return {k: v.float().cpu().numpy().astype(np.float64) for k, v in out.items()}

    def prefill(self, X, pos0=None, phases=vt.VT_ATTN | vt.VT_FFN, peer_attn=None,
                peer_ffn=None, h_in=None, on_device=False):
        """vt_layer_prefill_chunk of the [T][H] fp16 rows X at positions pos0.. .
        The outputs as float64 host arrays, or (on_device) as the fp16 device
        tensors the call wrote."""
        H = self.dims.hidden
        T = X.shape[0] if X is not None else h_in.shape[0]
        pos0 = self.kv.len if pos0 is None else pos0
        xt = h16(X) if X is not None else torch.zeros((T, H), dtype=torch.float16, device="cuda")
        pa = h16(peer_attn) if peer_attn is not None else None
        pf = h16(peer_ffn) if peer_ffn is not None else None
        out = {k: torch.full((T, H), float("nan"), dtype=torch.float16, device="cuda")
               for k in ("p_attn", "h", "p_ffn", "y")}
        if h_in is not None:
            out["h"] = h16(h_in)
        io = vt.vt_layer_io(x=ptr(xt), peer_attn=ptr(pa), peer_ffn=ptr(pf),
                            attn_partial=ptr(out["p_attn"]), h=ptr(out["h"]),
                            ffn_partial=ptr(out["p_ffn"]), y=ptr(out["y"]))
        vt.vt_layer_prefill_chunk(self.spec, self.w.struct, self.kv, io, T, pos0, phases,
                                  ptr(self.ws), self.ws_bytes, None)
        torch.cuda.synchronize()
        if on_device:
            return out
        return {k: v.float().cpu().numpy().astype(np.float64) for k, v in out.items()}

    def sync_words(self):
        """The workspace's synchronisation words (must be zero between calls):
        barrier, exit and error words and one counter per query head."""
        n = 3072 + 32 * (self.info.n_q_heads + 1)
        return self.ws[:4 * n].view(torch.int32).cpu().numpy()

    def cache(self):
        return (self.kc.view(torch.int16).cpu().numpy(), self.vc.view(torch.int16).cpu().numpy())
