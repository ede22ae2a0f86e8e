"""Test helpers: oracle-side shard slicing and the parity tolerance.

The oracle side slices the canonical tensors with the oracle's own
apportionment; the HIP side (in ``gpu_common``) slices with the ranges the
C library reports. Both draw from the same seeded generator.
"""
import numpy as np

import oracle
from synth import LayerDims, Workload
from synth.gen import LayerInputs

# Parity bar on fp16 outputs (max relative error 2e-2). Element-wise relative
# error, with each denominator floored at the root-mean-square of the
# reference vector: |got_i - ref_i| / max(|ref_i|, rms(ref)). The floor is
# needed because the error that fp16 activations at the sub-layer boundaries
# (x, h, the partial sums) carry into a projection scales with the vector's
# norm, not with each element, so elements near zero by cancellation would
# otherwise dominate. A normwise bound ||got - ref|| / ||ref|| <= NORM_TOL
# (an order of magnitude above fp16 rounding noise) also catches small
# systematic slips such as one wrong column of a wide projection.
REL_TOL = 2e-2
NORM_TOL = 4e-3


def max_rel_err(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if got.size == 0:
        return 0.0
    if not np.all(np.isfinite(got)):
        return float("inf")
    rms = np.sqrt(np.mean(ref * ref, axis=-1, keepdims=True))
    if np.any(rms == 0):
        # an all-zero reference vector must be reproduced exactly
        zero_rows = (rms == 0)[..., 0]
        if np.any(got[zero_rows] != 0):
            return float("inf")
        rms = np.where(rms == 0, 1.0, rms)
    denom = np.maximum(np.abs(ref), rms)
    return float(np.max(np.abs(got - ref) / denom))


def norm_rel_err(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if not np.all(np.isfinite(got)):
        return float("inf")
    n = np.linalg.norm(ref)
    e = np.linalg.norm(got - ref)
    return float(e / n) if n > 0 else (0.0 if e == 0 else float("inf"))


def assert_close(got, ref, what=""):
    e, n = max_rel_err(got, ref), norm_rel_err(got, ref)
    assert e <= REL_TOL and n <= NORM_TOL, f"{what}: element-wise {e:.3g}, normwise {n:.3g}"
    return e, n


def oracle_ranges(wl: Workload, device=None):
    d = wl.dims
    return oracle.shard_ranges(d.n_heads, d.n_kv_heads, d.ffn, wl.fracs, wl.fracs,
                               wl.device if device is None else device)


def oracle_shard_weights(li: LayerInputs, r) -> oracle.ShardWeights:
    d = li.wl.dims.head_dim
    q0, q1 = r.q_head_begin * d, (r.q_head_begin + r.n_q_heads) * d
    k0, k1 = r.kv_head_begin * d, (r.kv_head_begin + r.n_kv_heads) * d
    c0, c1 = r.col_begin, r.col_begin + r.n_cols
    return oracle.ShardWeights(
        g_attn=li.g_attn(), wq=li.rows("wq", q0, q1), wk=li.rows("wk", k0, k1),
        wv=li.rows("wv", k0, k1), wo=li.cols("wo", q0, q1), g_ffn=li.g_ffn(),
        wg=li.rows("wg", c0, c1), wu=li.rows("wu", c0, c1), wd=li.cols("wd", c0, c1))


def full_weights(li: LayerInputs) -> oracle.ShardWeights:
    """The unsharded layer as a single shard."""
    return oracle.ShardWeights(
        g_attn=li.g_attn(), wq=li.full("wq"), wk=li.full("wk"), wv=li.full("wv"),
        wo=li.full("wo"), g_ffn=li.g_ffn(), wg=li.full("wg"), wu=li.full("wu"),
        wd=li.full("wd"))


def oracle_decode(wl: Workload, li: LayerInputs, r, x, kc, vc, pos, peer_attn=None,
                  peer_ffn=None, w=None):
    d = wl.dims
    w = w if w is not None else oracle_shard_weights(li, r)
    return oracle.decode(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base,
                         x, kc, vc, pos, peer_attn, peer_ffn, window=d.window)


def tiny_workload(seed_id, hidden, n_heads, n_kv, head_dim, ffn, fracs, device, ctx,
                  sigma=0.25, chunk=0):
    return Workload(key=f"tiny{seed_id}", seed_id=seed_id, title="tiny test layer",
                    dims=LayerDims(hidden=hidden, n_heads=n_heads, n_kv_heads=n_kv,
                                   head_dim=head_dim, ffn=ffn),
                    fracs=tuple(fracs), device=device, weight_sigma=sigma, ctx=ctx,
                    chunk=chunk)


def oracle_qshard_weights(li: LayerInputs, r, level) -> oracle.ShardWeights:
    """The shard's weights as its INT8 / INT4 blocks stand for them: each
    sliced matrix quantised and dequantised by the oracle (fp64); the gains
    stay fp16."""
    from oracle import wquant
    w = oracle_shard_weights(li, r)
    q = lambda m: wquant.dequantized(m, level) if m.size else np.asarray(m, np.float64)
    return oracle.ShardWeights(g_attn=w.g_attn, wq=q(w.wq), wk=q(w.wk), wv=q(w.wv), wo=q(w.wo),
                               g_ffn=w.g_ffn, wg=q(w.wg), wu=q(w.wu), wd=q(w.wd))
