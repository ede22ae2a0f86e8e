"""Writes tests/golden/tiny_layer.json from the fp64 oracle.

Regression fixture only: the paper prints no worked numeric example, so the
stored values come from the oracle (pinned separately by brute force, the
torch library path and closed forms). A change to the oracle's arithmetic
that moves these values must name the passage of the paper, or the reading
of it, that justifies it. Run: python tests/golden/make_golden.py
"""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
from synth import LayerDims, Workload  # noqa: E402
from synth.gen import LayerInputs  # noqa: E402

CASE = dict(seed_id=140, hidden=32, n_heads=4, n_kv_heads=2, head_dim=8, ffn=20,
            fracs=[0.6, 0.4], device=0, ctx=4, chunk=3, sigma=0.25)


def build():
    c = CASE
    wl = Workload(key="golden", seed_id=c["seed_id"], title="golden tiny layer",
                  dims=LayerDims(c["hidden"], c["n_heads"], c["n_kv_heads"], c["head_dim"],
                                 c["ffn"]),
                  fracs=tuple(c["fracs"]), device=c["device"], weight_sigma=c["sigma"],
                  ctx=c["ctx"], chunk=c["chunk"])
    li = LayerInputs(wl)
    r = oracle.shard_ranges(c["n_heads"], c["n_kv_heads"], c["ffn"], c["fracs"], c["fracs"],
                            c["device"])
    d = c["head_dim"]
    w = oracle.ShardWeights(
        g_attn=li.g_attn(), wq=li.rows("wq", r.q_head_begin * d,
                                       (r.q_head_begin + r.n_q_heads) * d),
        wk=li.rows("wk", r.kv_head_begin * d, (r.kv_head_begin + r.n_kv_heads) * d),
        wv=li.rows("wv", r.kv_head_begin * d, (r.kv_head_begin + r.n_kv_heads) * d),
        wo=li.cols("wo", r.q_head_begin * d, (r.q_head_begin + r.n_q_heads) * d),
        g_ffn=li.g_ffn(), wg=li.rows("wg", r.col_begin, r.col_begin + r.n_cols),
        wu=li.rows("wu", r.col_begin, r.col_begin + r.n_cols),
        wd=li.cols("wd", r.col_begin, r.col_begin + r.n_cols))
    kc, vc = li.kv_context_heads(r.kv_head_begin, r.kv_head_begin + r.n_kv_heads)
    X = li.x_chunk(c["chunk"])
    o = oracle.prefill(w, r.n_q_heads, r.n_kv_heads, d, 1e-5, 10000.0, X, kc, vc, c["ctx"])
    return {"case": c, "ranges": r.__dict__,
            "outputs": {k: np.asarray(o[k]).tolist() for k in ("p_attn", "h", "p_ffn", "y")}}


if __name__ == "__main__":
    out = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tiny_layer.json")
    with open(out, "w") as f:
        json.dump(build(), f, indent=1)
    print("wrote", out)
