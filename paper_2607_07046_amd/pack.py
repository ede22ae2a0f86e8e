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


@dataclass
class QShardWeightsDev:
    tensors: dict
    struct: vt.vt_layer_qweights
    layout: dict = None   # name -> (code bytes of a row, row stride in bytes)
    prec: int = 0


def quantize_shard(sw: ShardWeightsDev, dims: vt.vt_layer_dims, info: vt.vt_shard_info, prec,
                   stream=None) -> QShardWeightsDev:
    """The shard's seven matrices in the library's INT8 / INT4 block format,
    quantised on the device by vt_quantize_rows (allocation and the calls
    only; the gains stay fp16). Each row holds its codes followed by its
    block scales (one buffer per matrix, rows padded to 16 bytes), so a
    row's scales share its codes' pages."""
    H, d = dims.hidden, dims.head_dim
    qd, kd, nc = info.n_q_heads * d, info.n_kv_heads * d, info.n_cols
    shapes = {"wq": (qd, H), "wk": (kd, H), "wv": (kd, H), "wo": (H, qd), "wg": (nc, H),
              "wu": (nc, H), "wd": (H, nc)}
    per_block = 32 if prec == vt.VT_W_INT8 else 16
    t = {"g_attn": sw.tensors["g_attn"], "g_ffn": sw.tensors["g_ffn"]}
    layout = {}
    for name, (rows, cols) in shapes.items():
        src = sw.tensors[name]
        nb = max(1, (cols + 31) // 32)
        code_bytes = nb * per_block
        ld = round_up(code_bytes + 2 * nb, 16)
        buf = torch.zeros((rows, ld), dtype=torch.uint8, device=src.device)
        if rows > 0 and cols > 0:
            vt.vt_quantize_rows(src.data_ptr(), src.shape[1], rows, cols, prec, buf.data_ptr(), ld,
                                buf.data_ptr() + code_bytes, ld // 2, stream)
        t[name] = buf
        layout[name] = (code_bytes, ld)
    return QShardWeightsDev(t, _qstruct(t, layout, prec), layout, prec)


def _qstruct(t, layout, prec):
    p = lambda x: x.data_ptr() if x.numel() else None
    mats = {}
    for name, (code_bytes, ld) in layout.items():
        b = t[name]
        mats[name] = vt.vt_qmat(codes=p(b), ld_codes=ld,
                                scales=(b.data_ptr() + code_bytes) if b.numel() else None,
                                ld_scales=ld // 2)
    return vt.vt_layer_qweights(prec=prec, g_attn=p(t["g_attn"]), g_ffn=p(t["g_ffn"]), **mats)


def clone_qshard(q: QShardWeightsDev) -> QShardWeightsDev:
    """A copy of the quantised shard in new device buffers (same layout)."""
    t = {n: x.clone() for n, x in q.tensors.items()}
    return QShardWeightsDev(t, _qstruct(t, q.layout, q.prec), q.layout, q.prec)


def upload_full(src, dims: vt.vt_layer_dims, device="cuda") -> ShardWeightsDev:
    """The whole layer's weights on the device (canonical out x in, each
    matrix contiguous; the rows of Wd padded with zeros to a multiple of 8
    columns, the row alignment the library requires): the source
    vt_shard_pack gathers shards from."""
    t = {"g_attn": _dev(src.g_attn(), device), "g_ffn": _dev(src.g_ffn(), device)}
    for name in ("wq", "wk", "wv", "wo", "wg", "wu", "wd"):
        t[name] = _dev(src.full(name), device)
    wd = t["wd"]
    if wd.shape[1] % 8:
        t["wd"] = torch.zeros((wd.shape[0], round_up(wd.shape[1], 8)), dtype=wd.dtype, device=wd.device)
        t["wd"][:, :wd.shape[1]] = wd
    p = lambda x: x.data_ptr() if x.numel() else None
    st = vt.vt_layer_weights(g_attn=p(t["g_attn"]), wq=p(t["wq"]), ld_q=t["wq"].shape[1],
                             wk=p(t["wk"]), ld_k=t["wk"].shape[1], wv=p(t["wv"]),
                             ld_v=t["wv"].shape[1], wo=p(t["wo"]), ld_o=t["wo"].shape[1],
                             g_ffn=p(t["g_ffn"]), wg=p(t["wg"]), ld_g=t["wg"].shape[1],
                             wu=p(t["wu"]), ld_u=t["wu"].shape[1], wd=p(t["wd"]),
                             ld_d=t["wd"].shape[1])
    return ShardWeightsDev(t, st)


def alloc_shard(dims: vt.vt_layer_dims, info: vt.vt_shard_info, device="cuda") -> ShardWeightsDev:
    """Separately allocated (uninitialised) buffers for one shard, laid out
    as pack_shard lays them out: the target of vt_shard_pack."""
    H, d = dims.hidden, dims.head_dim
    qd, kd, nc = info.n_q_heads * d, info.n_kv_heads * d, info.n_cols
    ld_d = max(8, round_up(nc, 8))
    e = lambda *shape: torch.empty(shape, dtype=torch.float16, device=device)
    t = {"g_attn": e(H), "g_ffn": e(H), "wq": e(qd, H), "wk": e(kd, H), "wv": e(kd, H),
         "wo": e(H, qd), "wg": e(nc, H), "wu": e(nc, H), "wd": e(H, ld_d)}
    return ShardWeightsDev(t, struct_of(t, dims, info, ld_d))


@dataclass
class MoEShardDev:
    tensors: dict
    struct: vt.vt_moe_weights


def pack_moe_shard(mi, c0, n_cols, device="cuda", ld_pad=0) -> MoEShardDev:
    """One device's share of an MoE FFN (columns [c0, c0 + n_cols) of every
    expert) laid out as vt_moe_ffn_decode takes it: wr [E][H], wg / wu
    [E][n_cols][H + ld_pad], wd [E][H][round_up(n_cols, 8) + ld_pad]. ``mi``
    is any object with ``g_ffn()``, ``router()`` and ``expert(name, e)``
    returning fp16 host arrays (canonical out x in). Row padding is left as
    zero; a caller may fill it to check that it is never used."""
    wl = mi.wl
    H, E = wl.hidden, wl.n_experts
    ldg = H + ld_pad
    ldd = max(8, round_up(n_cols, 8)) + ld_pad
    wg = np.zeros((E, n_cols, ldg), np.float16)
    wu = np.zeros((E, n_cols, ldg), np.float16)
    wd = np.zeros((E, H, ldd), np.float16)
    for e in range(E):
        wg[e, :, :H] = mi.expert("wg", e)[c0:c0 + n_cols]
        wu[e, :, :H] = mi.expert("wu", e)[c0:c0 + n_cols]
        wd[e, :, :n_cols] = mi.expert("wd", e)[:, c0:c0 + n_cols]
    t = {"g_ffn": _dev(mi.g_ffn(), device), "wr": _dev(mi.router(), device),
         "wg": _dev(wg, device), "wu": _dev(wu, device), "wd": _dev(wd, device)}
    p = lambda x: x.data_ptr() if x.numel() else None
    st = vt.vt_moe_weights(g_ffn=p(t["g_ffn"]), wr=p(t["wr"]), ld_r=H, wg=p(t["wg"]), ld_g=ldg,
                           wu=p(t["wu"]), ld_u=ldg, wd=p(t["wd"]), ld_d=ldd)
    return MoEShardDev(t, st)


@dataclass
class StackWeightsDev:
    """A stack of layers' shards, each matrix of every layer in one tensor
    [n_layers, rows, ld] (gains [n_layers, hidden]): the layout
    vt_stack_decode takes."""
    tensors: dict
    struct: vt.vt_stack_weights
    dims: vt.vt_layer_dims
    info: vt.vt_shard_info
    ld_d: int

    def layer(self, l) -> vt.vt_layer_weights:
        """Layer l's weights (views into the stacked tensors), as
        vt_layer_decode takes them."""
        return struct_of({n: t[l] for n, t in self.tensors.items()}, self.dims, self.info, self.ld_d)


def alloc_stack(dims: vt.vt_layer_dims, info: vt.vt_shard_info, n_layers, device="cuda",
                fill=None) -> StackWeightsDev:
    """Stacked buffers of n_layers shards (zero-filled, or filled by
    ``fill(name, shape)`` returning a device fp16 tensor of that shape; the
    padding columns of wd stay zero)."""
    H, d = dims.hidden, dims.head_dim
    qd, kd, nc = info.n_q_heads * d, info.n_kv_heads * d, info.n_cols
    ld_d = max(8, round_up(nc, 8))
    shapes = {"g_attn": (H,), "g_ffn": (H,), "wq": (qd, H), "wk": (kd, H), "wv": (kd, H),
              "wo": (H, qd), "wg": (nc, H), "wu": (nc, H), "wd": (H, ld_d)}
    t = {}
    for name, shape in shapes.items():
        buf = torch.zeros((n_layers, *shape), dtype=torch.float16, device=device)
        if fill is not None and buf.numel():
            if name == "wd":
                buf[:, :, :nc] = fill(name, (n_layers, H, nc))
            else:
                buf.copy_(fill(name, (n_layers, *shape)))
        t[name] = buf
    return _stack(t, dims, info, n_layers, ld_d)


def pack_stack(sources, dims: vt.vt_layer_dims, info: vt.vt_shard_info,
               device="cuda") -> StackWeightsDev:
    """The shards of len(sources) layers (each source as for pack_shard)
    copied into stacked buffers."""
    st = alloc_stack(dims, info, len(sources), device)
    for l, src in enumerate(sources):
        one = pack_shard(src, dims, info, device)
        for name, t in one.tensors.items():
            if t.numel():
                st.tensors[name][l].copy_(t)
        del one
    return st


def _stack(t, dims, info, n_layers, ld_d):
    first = struct_of({n: x[0] for n, x in t.items()}, dims, info, ld_d)
    return StackWeightsDev(t, vt.vt_stack_weights(n_layers=n_layers, w=first), dims, info, ld_d)
