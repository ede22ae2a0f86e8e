"""Shard-wise weight allocation on the device.

Paper Sec. 4.3.1 (Pruning) allocates each shard's weights separately so a
shard can be dropped or loaded on its own. ``pack_shard`` slices a shard out
of a layer's canonical tensors (rows of Wq/Wk/Wv/Wg/Wu, columns of Wo/Wd)
and uploads each slice as its own device tensor. Pure data movement: no
value is computed. ``src`` is any object with ``rows(name, r0, r1)``,
``cols(name, c0, c1)``, ``g_attn()`` and ``g_ffn()`` returning fp16 host
arrays of the canonical out x in tensors.
"""
from dataclasses import dataclass

import numpy as np
import torch

from . import voltron as vt


def _dev(a, device):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


@dataclass
class ShardWeightsDev:
    tensors: dict
    struct: vt.vt_layer_weights


def round_up(v, m):
    return (v + m - 1) // m * m


def pack_shard(src, dims: vt.vt_layer_dims, info: vt.vt_shard_info, device="cuda") \
        -> ShardWeightsDev:
    d = dims.head_dim
    q0, q1 = info.q_head_begin * d, (info.q_head_begin + info.n_q_heads) * d
    k0, k1 = info.kv_head_begin * d, (info.kv_head_begin + info.n_kv_heads) * d
    c0, c1 = info.col_begin, info.col_begin + info.n_cols
    t = {
        "g_attn": _dev(src.g_attn(), device),
        "g_ffn": _dev(src.g_ffn(), device),
        "wq": _dev(src.rows("wq", q0, q1), device),
        "wk": _dev(src.rows("wk", k0, k1), device),
        "wv": _dev(src.rows("wv", k0, k1), device),
        "wo": _dev(src.cols("wo", q0, q1), device),
        "wg": _dev(src.rows("wg", c0, c1), device),
        "wu": _dev(src.rows("wu", c0, c1), device),
    }
    # Wd rows are padded to a multiple of 8 elements (16-byte aligned rows).
    ld_d = max(8, round_up(info.n_cols, 8))
    wd = np.zeros((dims.hidden, ld_d), np.float16)
    wd[:, :info.n_cols] = src.cols("wd", c0, c1)
    t["wd"] = _dev(wd, device)
    return ShardWeightsDev(t, struct_of(t, dims, info, ld_d))


def struct_of(t, dims, info, ld_d):
    H = dims.hidden
    p = lambda x: x.data_ptr() if x.numel() else None
    return vt.vt_layer_weights(
        g_attn=p(t["g_attn"]), wq=p(t["wq"]), ld_q=H, wk=p(t["wk"]), ld_k=H, wv=p(t["wv"]),
        ld_v=H, wo=p(t["wo"]), ld_o=max(8, info.n_q_heads * dims.head_dim),
        g_ffn=p(t["g_ffn"]), wg=p(t["wg"]), ld_g=H, wu=p(t["wu"]), ld_u=H, wd=p(t["wd"]),
        ld_d=ld_d)
