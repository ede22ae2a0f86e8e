"""Seeded generator of the canonical fp16 tensors of a synthetic decoder layer.

Every tensor is drawn in its canonical out x in, row-major order, in blocks of
``BLOCK_ROWS`` rows. Block ``b`` of tensor ``t`` of layer ``l`` of workload
``w`` comes from ``PCG64(SeedSequence([7046, w.seed_id, l, t, b]))``: standard
normal float32 values, times the tensor's scale in float32, rounded to fp16.
So any row range can be drawn without drawing the rest, and a shard and the
unsharded layer always see identical numbers.

Scales: projection weights N(0, sigma) with sigma the workload's weight scale;
RMSNorm gains 1 + N(0, 0.1); input activations, cached keys and cached values
N(0, 1). The cached keys stand for keys that were already rotated when they
were appended.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .configs import Workload

BLOCK_ROWS = 256
ROOT_SEED = 7046

# tensor ids (part of the seed)
T_G_ATTN, T_WQ, T_WK, T_WV, T_WO, T_G_FFN, T_WG, T_WU, T_WD = range(9)
T_X, T_XCHUNK, T_KCTX, T_VCTX, T_PEER_ATTN, T_PEER_FFN = range(9, 15)

_NAMES = {"wq": T_WQ, "wk": T_WK, "wv": T_WV, "wo": T_WO,
          "wg": T_WG, "wu": T_WU, "wd": T_WD}

_POOL = None


def _pool():
    global _POOL
    if _POOL is None:
        n = max(1, min(16, len(os.sched_getaffinity(0))))
        _POOL = ThreadPoolExecutor(n)
    return _POOL


def _normal(seed, shape, scale, offset=0.0):
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
    v = rng.standard_normal(shape, dtype=np.float32)
    if scale != 1.0:
        v *= np.float32(scale)
    if offset != 0.0:
        v += np.float32(offset)
    return v.astype(np.float16)


def canonical_shape(wl: Workload, name: str):
    d = wl.dims
    qd, kvd = d.n_heads * d.head_dim, d.n_kv_heads * d.head_dim
    return {"wq": (qd, d.hidden), "wk": (kvd, d.hidden), "wv": (kvd, d.hidden),
            "wo": (d.hidden, qd), "wg": (d.ffn, d.hidden), "wu": (d.ffn, d.hidden),
            "wd": (d.hidden, d.ffn)}[name]


class LayerInputs:
    """Draws (and caches) the fp16 tensors of layer ``layer`` of a workload."""

    def __init__(self, wl: Workload, layer: int = 0):
        self.wl = wl
        self.layer = layer
        self._cache = {}

    def _seed(self, tensor, block):
        return [ROOT_SEED, self.wl.seed_id, self.layer, tensor, block]

    # ---- projection weights -------------------------------------------------
    def rows(self, name: str, r0: int, r1: int) -> np.ndarray:
        """Rows [r0, r1) of canonical tensor ``name`` (fp16, [r1-r0, cols])."""
        R, C = canonical_shape(self.wl, name)
        if not (0 <= r0 <= r1 <= R):
            raise ValueError(f"row range [{r0},{r1}) outside {name} with {R} rows")
        if (name, "full") in self._cache:
            return self._cache[(name, "full")][r0:r1]
        out = np.empty((r1 - r0, C), np.float16)
        if r1 == r0:
            return out
        b0, b1 = r0 // BLOCK_ROWS, (r1 - 1) // BLOCK_ROWS
        tid = _NAMES[name]

        def draw(b):
            lo, hi = b * BLOCK_ROWS, min(R, (b + 1) * BLOCK_ROWS)
            blk = _normal(self._seed(tid, b), (hi - lo, C), self.wl.weight_sigma)
            a, z = max(lo, r0), min(hi, r1)
            out[a - r0:z - r0] = blk[a - lo:z - lo]

        list(_pool().map(draw, range(b0, b1 + 1)))
        return out

    def full(self, name: str, keep: bool = True) -> np.ndarray:
        key = (name, "full")
        if key in self._cache:
            return self._cache[key]
        R, _ = canonical_shape(self.wl, name)
        t = self.rows(name, 0, R)
        if keep:
            self._cache[key] = t
        return t

    def cols(self, name: str, c0: int, c1: int) -> np.ndarray:
        """Columns [c0, c1) of canonical tensor ``name`` (draws whole rows)."""
        return np.ascontiguousarray(self.full(name, keep=False)[:, c0:c1]) \
            if (name, "full") not in self._cache else \
            np.ascontiguousarray(self._cache[(name, "full")][:, c0:c1])

    # ---- gains --------------------------------------------------------------
    def g_attn(self) -> np.ndarray:
        return _normal(self._seed(T_G_ATTN, 0), (self.wl.dims.hidden,), 0.1, 1.0)

    def g_ffn(self) -> np.ndarray:
        return _normal(self._seed(T_G_FFN, 0), (self.wl.dims.hidden,), 0.1, 1.0)

    # ---- activations and cache ----------------------------------------------
    def x(self, token: int = 0) -> np.ndarray:
        """Decode input activation of token ``token`` ([hidden] fp16)."""
        return _normal(self._seed(T_X, token), (self.wl.dims.hidden,), 1.0)

    def x_chunk(self, n_tok: int) -> np.ndarray:
        """Prefill chunk of input activations ([n_tok, hidden] fp16)."""
        return _normal(self._seed(T_XCHUNK, 0), (n_tok, self.wl.dims.hidden), 1.0)

    def peer(self, which: str, token: int = 0, rows: int = 0) -> np.ndarray:
        """Stand-in for the other devices' partial sum ("attn" or "ffn")."""
        tid = T_PEER_ATTN if which == "attn" else T_PEER_FFN
        shape = (rows, self.wl.dims.hidden) if rows else (self.wl.dims.hidden,)
        return _normal(self._seed(tid, token), shape, 0.5)

    def kv_context(self, kv_head: int, n_pos: int = -1):
        """Cached keys and values of KV head ``kv_head`` at positions 0..n_pos-1."""
        n = self.wl.ctx if n_pos < 0 else n_pos
        d = self.wl.dims.head_dim
        k = _normal(self._seed(T_KCTX, kv_head), (n, d), 1.0)
        v = _normal(self._seed(T_VCTX, kv_head), (n, d), 1.0)
        return k, v

    def kv_context_heads(self, g0: int, g1: int, n_pos: int = -1):
        """Stacked [g1-g0, n_pos, d] keys and values of KV heads g0..g1-1."""
        ks, vs = zip(*_pool().map(lambda g: self.kv_context(g, n_pos), range(g0, g1))) \
            if g1 > g0 else ((), ())
        d = self.wl.dims.head_dim
        n = self.wl.ctx if n_pos < 0 else n_pos
        if g1 == g0:
            return np.empty((0, n, d), np.float16), np.empty((0, n, d), np.float16)
        return np.stack(ks), np.stack(vs)


def layer_inputs(wl: Workload, layer: int = 0) -> LayerInputs:
    return LayerInputs(wl, layer)


def vector(tag: int, n: int, scale: float = 1.0, seed_id: int = 99) -> np.ndarray:
    """A seeded fp16 vector N(0, scale) of length n, for tests of the
    partial-sum transmission (``tag`` distinguishes vectors)."""
    return _normal([ROOT_SEED, seed_id, 0, 1000 + tag, 0], (n,), scale)


# MoE tensors (ids past the dense layer's): router [E, H], per expert e the
# gate and up [F_e, H] and down [H, F_e] matrices, the FFN gain and input h
T_MOE_G, T_MOE_WR, T_MOE_H = 20, 21, 22
T_MOE_WG, T_MOE_WU, T_MOE_WD = 23, 24, 25


class MoEInputs:
    """Draws the fp16 tensors of an MoE FFN workload (same seeding scheme:
    expert e's tensor t from PCG64(SeedSequence([7046, seed_id, e, t, 0])))."""

    def __init__(self, wl):
        self.wl = wl

    def _seed(self, e, tensor, block=0):
        return [ROOT_SEED, self.wl.seed_id, e, tensor, block]

    def g_ffn(self) -> np.ndarray:
        return _normal(self._seed(0, T_MOE_G), (self.wl.hidden,), 0.1, 1.0)

    def router(self) -> np.ndarray:
        return _normal(self._seed(0, T_MOE_WR), (self.wl.n_experts, self.wl.hidden),
                       self.wl.router_sigma)

    def h(self, token: int = 0) -> np.ndarray:
        return _normal(self._seed(token, T_MOE_H), (self.wl.hidden,), 1.0)

    def expert(self, name: str, e: int) -> np.ndarray:
        """Expert e's canonical "wg" / "wu" [F_e, H] or "wd" [H, F_e]."""
        w = self.wl
        tid, shape = {"wg": (T_MOE_WG, (w.expert_ffn, w.hidden)),
                      "wu": (T_MOE_WU, (w.expert_ffn, w.hidden)),
                      "wd": (T_MOE_WD, (w.hidden, w.expert_ffn))}[name]
        return _normal(self._seed(e, tid), shape, w.weight_sigma)
