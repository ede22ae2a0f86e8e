"""The five synthetic workloads of the decoder-layer shard.

Each workload is a Llama-shaped decoder layer (or stack of layers), a
partition of its heads and FFN columns over a number of devices given as
fractions, the device whose share is run, and the decode position(s).
Nothing here is derived from the method: the fractions, shapes, value
scales and context lengths are the workload's definition.
"""
from dataclasses import dataclass, field
from typing import Tuple


@dataclass(frozen=True)
class LayerDims:
    hidden: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    rms_eps: float = 1e-5
    rope_base: float = 10000.0
    window: int = 0          # sliding-window attention span (0: full causal)

    @property
    def group(self) -> int:
        return self.n_heads // self.n_kv_heads


@dataclass(frozen=True)
class Workload:
    key: str            # short name used in tests and the bench
    seed_id: int        # distinct per workload; part of every seed
    title: str
    dims: LayerDims
    fracs: Tuple[float, ...]   # head fraction == column fraction per device
    device: int         # the device whose share is run
    weight_sigma: float
    ctx: int            # cached positions before the first new token
    n_layers: int = 1
    n_tokens: int = 1   # consecutive decode tokens (decode workloads)
    chunk: int = 0      # prefill chunk length (0: decode workload)

    @property
    def pos(self) -> int:
        return self.ctx

    @property
    def capacity(self) -> int:
        return self.ctx + max(self.n_tokens, self.chunk)


_LLAMA7B = LayerDims(hidden=4096, n_heads=32, n_kv_heads=32, head_dim=128, ffn=11008)

WORKLOADS = {
    "tiny": Workload(
        key="tiny", seed_id=1,
        title="tiny layer: hidden 512, 8x64 heads, FFN 1376, 2 devices 50/50, decode at 128",
        dims=LayerDims(hidden=512, n_heads=8, n_kv_heads=8, head_dim=64, ffn=1376),
        fracs=(0.5, 0.5), device=0, weight_sigma=0.02, ctx=128),
    "7b": Workload(
        key="7b", seed_id=2,
        title="7B-shaped layer: hidden 4096, 32x128 MHA, FFN 11008, 3 devices 50/30/20, "
              "30% shard, decode at 1024",
        dims=_LLAMA7B, fracs=(0.5, 0.3, 0.2), device=1, weight_sigma=0.02, ctx=1024),
    "13b_stack": Workload(
        key="13b_stack", seed_id=3,
        title="13B-shaped 40-layer stack: hidden 5120, 40x128 MHA, FFN 13824, 40% shard, "
              "64 consecutive tokens from 2048",
        dims=LayerDims(hidden=5120, n_heads=40, n_kv_heads=40, head_dim=128, ffn=13824),
        fracs=(0.4, 0.6), device=0, weight_sigma=0.02, ctx=2048, n_layers=40, n_tokens=64),
    "70b_gqa": Workload(
        key="70b_gqa", seed_id=4,
        title="70B-shaped GQA layer: hidden 8192, 64x128 heads, 8 KV heads, FFN 28672, "
              "4 devices 25% each, decode at 4096",
        dims=LayerDims(hidden=8192, n_heads=64, n_kv_heads=8, head_dim=128, ffn=28672),
        fracs=(0.25, 0.25, 0.25, 0.25), device=0, weight_sigma=0.015, ctx=4096),
    "7b_swa": Workload(
        key="7b_swa", seed_id=6,
        title="7B-shaped layer with sliding-window attention (window 1024): 30% shard, "
              "decode at 4096",
        dims=LayerDims(hidden=4096, n_heads=32, n_kv_heads=32, head_dim=128, ffn=11008,
                       window=1024),
        fracs=(0.5, 0.3, 0.2), device=1, weight_sigma=0.02, ctx=4096),
    "7b_prefill": Workload(
        key="7b_prefill", seed_id=5,
        title="prefill chunk on the 7B-shaped layer: 50% shard, 256 tokens at positions 768..1023",
        dims=_LLAMA7B, fracs=(0.5, 0.5), device=0, weight_sigma=0.02, ctx=768, chunk=256),
}


def get(key: str) -> Workload:
    return WORKLOADS[key]


@dataclass(frozen=True)
class MoEWorkload:
    """An MoE FFN sub-layer (routed experts, SwiGLU each) and one device's
    share of every expert's columns."""
    key: str
    seed_id: int
    title: str
    hidden: int
    n_experts: int
    expert_ffn: int
    top_k: int
    fracs: tuple
    device: int
    weight_sigma: float = 0.02
    router_sigma: float = 0.02
    rms_eps: float = 1e-5


MOE_WORKLOADS = {
    "moe": MoEWorkload(
        key="moe", seed_id=7,
        title="MoE FFN shaped like Qwen1.5-MoE-A2.7B's routed experts: hidden 2048, 60 experts "
              "of 1408 columns, top-4, 4 devices 25% (352 columns of every expert)",
        hidden=2048, n_experts=60, expert_ffn=1408, top_k=4, fracs=(0.25, 0.25, 0.25, 0.25),
        device=0),
}
