"""Test infrastructure only: the fp64 definition of a mixture-of-experts FFN
sub-layer and of one device's share of it (paper Sec. 2.1: MoE FFNs
activate a subset of expert networks per token; Table 3's MoE model).
Nothing in the product imports this module.

Readings where the paper is silent (the routed part of Qwen1.5-MoE, the MoE
model of Table 3; its shared expert is a dense FFN, the dense path):
* w = RMSNorm(h) * g_ffn, as for the dense FFN;
* router logits r = Wr w over all E experts; probabilities p = softmax(r);
* the k experts with the largest logits are selected (ties: lower index);
* output = sum over the selected experts e of p_e * Wd_e (silu(Wg_e w) *
  (Wu_e w)), with p_e the softmax probability over all E (not
  renormalised over the k);
* tensor parallelism shards every expert by its FFN columns, as the dense
  FFN: a device holds columns [c0, c1) of each expert's Wg / Wu rows and
  Wd columns, computes the routing itself (the router is small and every
  device has w), and its partial sum is the same sum over its columns. The
  partial sums of a partition add up to the unsharded output.
The selection is an integer decision taken from floating-point logits; a
test that compares it with a device's selection checks that the margin
between the k-th and (k+1)-th logit is far above rounding.
"""
import numpy as np

from .layer import rmsnorm, silu, softmax


def route(w, wr, top_k):
    """(selected experts [k], their probabilities [k], logits [E])."""
    logits = np.asarray(wr, np.float64) @ np.asarray(w, np.float64)
    p = softmax(logits)
    sel = np.argsort(-logits, kind="stable")[:top_k]
    return sel, p[sel], logits


def moe_ffn(g_ffn, wr, wg, wu, wd, eps, h, top_k, peer=None):
    """MoE FFN of a shard for one token.

    wr: [E, H] router; wg, wu: [E, n_cols, H] the shard's columns of every
    expert; wd: [E, H, n_cols]; h: [H]. Returns dict p_ffn, y, sel, probs,
    logits.
    """
    h = np.asarray(h, np.float64)
    w = rmsnorm(h, g_ffn, eps)
    sel, probs, logits = route(w, wr, top_k)
    p_ffn = np.zeros_like(h)
    for e, pe in zip(sel, probs):
        m = silu(np.asarray(wg[e], np.float64) @ w) * (np.asarray(wu[e], np.float64) @ w)
        p_ffn = p_ffn + pe * (np.asarray(wd[e], np.float64) @ m)
    y = h + p_ffn + (0.0 if peer is None else np.asarray(peer, np.float64))
    return dict(p_ffn=p_ffn, y=y, sel=sel, probs=probs, logits=logits)
