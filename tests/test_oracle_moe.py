"""Pins of the MoE FFN oracle (oracle.moe): one expert selected out of one is
the dense FFN oracle exactly; selecting every expert is the probability-
weighted sum of every expert's FFN; relabelling the experts (router rows
and expert tensors together) changes nothing; the column shards of a
partition add up to the unsharded sub-layer (fp64, 1e-9) under the same
routing; the selection takes the largest logits with ties to the lower
index.
"""
import numpy as np

import oracle
from oracle.moe import moe_ffn, route
from oracle.layer import ShardWeights, rmsnorm, silu
from synth.configs import MoEWorkload
from synth.gen import MoEInputs


def small(E=6, F=40, H=32, k=2, seed=971):
    wl = MoEWorkload(key="moe_t", seed_id=seed, title="", hidden=H, n_experts=E, expert_ffn=F,
                     top_k=k, fracs=(1.0,), device=0, weight_sigma=0.1, router_sigma=0.2)
    mi = MoEInputs(wl)
    wg = np.stack([mi.expert("wg", e) for e in range(E)])
    wu = np.stack([mi.expert("wu", e) for e in range(E)])
    wd = np.stack([mi.expert("wd", e) for e in range(E)])
    return wl, mi, wg, wu, wd


def test_single_expert_is_dense_ffn():
    wl, mi, wg, wu, wd = small(E=1, k=1)
    h = mi.h()
    r = moe_ffn(mi.g_ffn(), mi.router(), wg, wu, wd, wl.rms_eps, h, 1)
    dense = ShardWeights(g_attn=None, wq=None, wk=None, wv=None, wo=None, g_ffn=mi.g_ffn(),
                         wg=wg[0], wu=wu[0], wd=wd[0])
    p, y = oracle.ffn_sublayer(dense, wl.rms_eps, h[None].astype(np.float64))
    assert np.array_equal(r["p_ffn"], p[0]) and np.array_equal(r["y"], y[0])


def test_all_experts_is_weighted_sum():
    wl, mi, wg, wu, wd = small(E=5, k=5)
    h = mi.h()
    r = moe_ffn(mi.g_ffn(), mi.router(), wg, wu, wd, wl.rms_eps, h, 5)
    w = rmsnorm(h.astype(np.float64), mi.g_ffn(), wl.rms_eps)
    logits = mi.router().astype(np.float64) @ w
    p = np.exp(logits - logits.max())
    p /= p.sum()
    want = sum(p[e] * (wd[e].astype(np.float64) @ (silu(wg[e].astype(np.float64) @ w) *
                                                      (wu[e].astype(np.float64) @ w)))
               for e in range(5))
    assert np.max(np.abs(r["p_ffn"] - want)) <= 1e-12 * np.max(np.abs(want))
    assert abs(np.sum(r["probs"]) - 1.0) < 1e-12


def test_relabelling_experts():
    wl, mi, wg, wu, wd = small()
    h = mi.h()
    perm = np.array([3, 0, 5, 1, 4, 2])
    a = moe_ffn(mi.g_ffn(), mi.router(), wg, wu, wd, wl.rms_eps, h, wl.top_k)
    b = moe_ffn(mi.g_ffn(), mi.router()[perm], wg[perm], wu[perm], wd[perm], wl.rms_eps, h,
                wl.top_k)
    assert np.max(np.abs(a["p_ffn"] - b["p_ffn"])) <= 1e-12 * np.max(np.abs(a["p_ffn"]))
    assert sorted(perm[b["sel"]]) == sorted(a["sel"])


def test_column_shards_add_up():
    wl, mi, wg, wu, wd = small(F=41)
    h = mi.h()
    full = moe_ffn(mi.g_ffn(), mi.router(), wg, wu, wd, wl.rms_eps, h, wl.top_k)
    fr = (0.3, 0.45, 0.25)
    parts = []
    for dev in range(3):
        c = oracle.apportion(41, fr)
        c0 = sum(c[:dev])
        c1 = c0 + c[dev]
        parts.append(moe_ffn(mi.g_ffn(), mi.router(), wg[:, c0:c1], wu[:, c0:c1], wd[:, :, c0:c1],
                             wl.rms_eps, h, wl.top_k)["p_ffn"])
    s = np.sum(parts, axis=0)
    assert np.max(np.abs(s - full["p_ffn"])) <= 1e-9 * np.max(np.abs(full["p_ffn"]))


def test_selection_order_and_ties():
    w = np.array([1.0, 0.0])
    wr = np.array([[1.0, 0], [3.0, 0], [3.0, 0], [2.0, 0], [-1.0, 0]])
    sel, probs, logits = route(w, wr, 3)
    assert list(sel) == [1, 2, 3]                 # 3, 3 (lower index first), 2
    assert np.allclose(probs, np.exp(logits[[1, 2, 3]]) / np.exp(logits).sum(), rtol=0, atol=1e-15)
