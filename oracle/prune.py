"""Test infrastructure only: the layer that shard-wise pruning leaves
(paper Sec. 4.3.1, Pruning; shards allocated separately, Sec. 4.3.1
Overhead Mitigation). Nothing in the product imports this module.

What the paper fixes: pruning drops whole shards of a layer, in ascending
order of importance, the same number in every layer; a dropped shard's
weights are simply released, and the layer runs on the shards kept.

Reading: a shard is a range of KV groups (a KV head and the query heads
sharing it) and a range of FFN columns. The kept shards' partial sums add up
to the layer in which the dropped query heads and FFN columns contribute
nothing: their columns of Wo and of Wd are zero (the projections into them
may be computed, but nothing reads them). The KV cache of a dropped group is
not kept up to date.
"""
from dataclasses import replace

import numpy as np

from .layer import ShardWeights


def pruned_weights(w: ShardWeights, head_dim: int, group: int, keep_groups, keep_cols) -> ShardWeights:
    """The full layer's weights with dropped heads and columns silenced.

    keep_groups: bool [n_kv_heads]; keep_cols: bool [ffn].
    """
    keep_groups = np.asarray(keep_groups, dtype=bool)
    keep_cols = np.asarray(keep_cols, dtype=bool)
    heads = np.repeat(keep_groups, group)                 # query head j -> group j // G
    head_cols = np.repeat(heads, head_dim)                 # columns of Wo
    wo = np.asarray(w.wo, dtype=np.float64) * head_cols[None, :]
    wd = np.asarray(w.wd, dtype=np.float64) * keep_cols[None, :]
    return replace(w, wo=wo, wd=wd)
