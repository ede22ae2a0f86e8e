"""Uneven split of a layer's heads and FFN columns over devices.

Paper Sec. 4.2.1 (TP allocation): shards, i.e. partitions of a layer, are
assigned to devices greedily according to their performance so that every
device finishes at about the same time; Sec. 3.2.2 shows why an even split
fails on heterogeneous devices. The paper gives no rounding rule. Reading
used here: each device's share is a fraction; whole units are dealt by the
largest-remainder rule (floor of fraction x units, then one extra unit to
the devices with the largest fractional parts, lower device index first on
ties); devices take contiguous unit ranges in device order. Attention is
split in whole KV groups (a KV head and the query heads sharing it, Sec.
2.1, GQA), so a group never straddles devices; FFN columns are split
independently of heads.

The arithmetic (fraction times units in IEEE double, floor, remainder) is
stated so that any implementation of this rule yields identical integers.
"""
import math
from dataclasses import dataclass
from typing import Sequence


def apportion(total: int, fracs: Sequence[float]) -> list:
    """Largest-remainder split of ``total`` units by ``fracs`` (sum 1 +- 1e-9)."""
    n = len(fracs)
    if n < 1:
        raise ValueError("need at least one device")
    if total < 0:
        raise ValueError("negative unit count")
    for f in fracs:
        if not math.isfinite(f) or f < 0.0:
            raise ValueError(f"bad fraction {f!r}")
    if abs(math.fsum(fracs) - 1.0) > 1e-9:
        raise ValueError(f"fractions sum to {math.fsum(fracs)!r}, not 1")
    quota = [float(f) * float(total) for f in fracs]
    base = [int(math.floor(q)) for q in quota]
    rem = [q - b for q, b in zip(quota, base)]
    left = total - sum(base)
    # Remainders sum to ``left`` up to the 1e-9 slack, so 0 <= left <= n.
    order = sorted(range(n), key=lambda i: (-rem[i], i))
    for i in order[:left]:
        base[i] += 1
    return base


@dataclass(frozen=True)
class ShardRanges:
    q_head_begin: int
    n_q_heads: int
    kv_head_begin: int
    n_kv_heads: int
    col_begin: int
    n_cols: int


def shard_ranges(n_heads: int, n_kv_heads: int, ffn: int, head_fracs, col_fracs,
                 device: int) -> ShardRanges:
    """Head and column ranges of ``device``'s shard (see module docstring)."""
    if n_kv_heads < 1 or n_heads % n_kv_heads:
        raise ValueError("n_heads must be a positive multiple of n_kv_heads")
    if len(head_fracs) != len(col_fracs):
        raise ValueError("head and column fractions must cover the same devices")
    if not 0 <= device < len(head_fracs):
        raise ValueError("device index out of range")
    group = n_heads // n_kv_heads
    kv = apportion(n_kv_heads, head_fracs)
    cols = apportion(ffn, col_fracs)
    kv0 = sum(kv[:device])
    c0 = sum(cols[:device])
    return ShardRanges(q_head_begin=kv0 * group, n_q_heads=kv[device] * group,
                       kv_head_begin=kv0, n_kv_heads=kv[device],
                       col_begin=c0, n_cols=cols[device])
