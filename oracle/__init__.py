"""fp64 CPU oracle of one device's share of a tensor-parallel decoder layer.

TEST INFRASTRUCTURE ONLY. Nothing in the product imports, calls or links
this package: only the tests, the smoke check and the bench's CPU-baseline
leg use it. It shares no code with the HIP path; both receive their inputs
from the seeded generator in ``synth``, which holds none of the layer's
arithmetic.

What it follows (paper: Voltron, arXiv 2607.07046):
  * Sec. 2.1 (LLM Architecture, Fig. Background1): per-head scaled
    dot-product attention over Q, K, V; an output linear O; a feed-forward
    network; GQA shares K and V across query heads.
  * Sec. 2.1 (LLM Inference): prefill processes the prompt tokens in
    parallel; decode produces one token per step; the K and V of each new
    token are accumulated into the KV cache.
  * Sec. 3.2.1 (Fig. Motivation1(b)): tensor parallelism broadcasts a
    layer's input to every device, each device computes its shard, and the
    results are aggregated on the main device.
  * Sec. 4.2.1: shards are assigned to devices greedily by performance,
    i.e. unevenly; ``apportion`` is the reading of that used here.
  * Sec. 4.3.2 with Sec. 4.2.2 (Communication Scaling, importance-ordered
    lowering): ``comm`` plans and encodes the transmission precision of a
    shard's partial sums (FP16 / INT8 / INT4 / pruned blocks).
  * Sec. 2.2, 4.2.2, 4.3.1 (mixed precision, precision scaling):
    ``wquant`` quantises a shard's weight rows to INT8 / INT4 blocks and
    gives the values the quantised shard stands for.
  * Sec. 4.3.1 (Pruning): ``prune`` gives the layer that the kept shards of
    a pruned partition add up to.
  * Sec. 2.1 (FFN variants) and Table 3: ``moe`` is a mixture-of-experts
    FFN sub-layer (top-k routing) and a device's column share of it.

The paper does not define the decoder's internals (normalisation, rotary
embedding, FFN form); the readings used here are the Llama layer:
pre-norm RMSNorm, adjacent-pair RoPE, SwiGLU FFN, no biases. Every reading
is listed with the module that implements it.

Parity status: every function here is pinned by tests that do not re-type
its formula (brute force on tiny layers, the torch float64 library path,
closed forms and invariants, and the shard sizes stated in the workload
definitions). No function is "parity unpinned".
"""
from .apportion import apportion, shard_ranges, ShardRanges
from .layer import (ShardWeights, rmsnorm, rope, softmax, silu, attention,
                    attn_sublayer, ffn_sublayer, decode, prefill, append_kv)

__all__ = ["apportion", "shard_ranges", "ShardRanges", "ShardWeights", "rmsnorm",
           "rope", "softmax", "silu", "attention", "attn_sublayer", "ffn_sublayer",
           "decode", "prefill", "append_kv"]
