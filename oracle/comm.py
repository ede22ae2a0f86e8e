"""Test infrastructure only: the fp32 reference of the transmission-precision
scaling of a shard's partial sums (paper Sec. 4.3.2, Communication Scaling),
with the importance-ordered lowering of Sec. 4.2.2. Nothing in the product
imports this module.

What the paper fixes: to cut the bytes sent between devices, the precision
of the transmitted activations is lowered (FP16 -> INT8 -> INT4) in
ascending order of importance, and if every activation at INT4 is still too
much, transmitted activations are pruned in the same order; the lowering
starts from full precision and goes no further than the budget needs.

Readings where the paper is silent (stated once here and in the design
notes):
* granularity: blocks of 32 consecutive activations, one precision each;
  a block's importance is supplied by the caller (the sum over its
  activations of the importance of the weight shards that produce them);
* quantisation: symmetric absmax per block; scale s = absmax / Q in fp32
  (Q = 127 for INT8, 7 for INT4); code = clamp(rint(x / s), -Q, Q), the
  division in fp32 and rint rounding half to even; an all-zero block has
  s = 0 and codes 0; value = code * s;
* wire format of one block: FP16 = the 32 fp16 values (64 B); INT8 = fp32
  scale + 32 int8 codes (36 B); INT4 = fp32 scale + 16 bytes holding two
  4-bit two's-complement codes each, element 2k in the low nibble of byte k
  (20 B); PRUNED = nothing (reads as 0). Blocks are stored in order, each at
  the sum of the sizes before it;
* plan: all blocks start at FP16; in ascending importance (ties: lower
  block index first) blocks go FP16 -> INT8 one at a time until the message
  fits the byte budget; then, in the same order, INT8 -> INT4; then INT4 ->
  PRUNED. Each step is the least lowering that meets the budget.

Floating-point steps that decide an integer (the codes) are taken in fp32,
the precision the device kernels use.
"""
import numpy as np

FP16, INT8, INT4, PRUNED = 0, 1, 2, 3
BLOCK = 32
BLOCK_BYTES = {FP16: 64, INT8: 36, INT4: 20, PRUNED: 0}
QMAX = {INT8: 127, INT4: 7}


def plan(importance, budget_bytes):
    """Per-block precisions, byte offsets and total message size.

    importance: [n_blocks] scores (higher = more important).
    Returns (prec [n_blocks] int, offsets [n_blocks] int, total bytes).
    """
    imp = np.asarray(importance, dtype=np.float32)
    nb = imp.shape[0]
    prec = np.full(nb, FP16, dtype=np.int64)
    total = nb * BLOCK_BYTES[FP16]
    # ascending importance, ties to the lower index (stable sort)
    order = np.argsort(imp, kind="stable")
    for frm, to in ((FP16, INT8), (INT8, INT4), (INT4, PRUNED)):
        for b in order:
            if total <= budget_bytes:
                break
            if prec[b] == frm:
                total -= BLOCK_BYTES[frm] - BLOCK_BYTES[to]
                prec[b] = to
    offsets = np.zeros(nb, dtype=np.int64)
    acc = 0
    for b in range(nb):
        offsets[b] = acc
        acc += BLOCK_BYTES[int(prec[b])]
    return prec, offsets, acc


def quantize_block(x, level):
    """(scale, codes) of one block of fp32 values at INT8 or INT4."""
    x = np.asarray(x, dtype=np.float32)
    q = np.float32(QMAX[level])
    a = np.max(np.abs(x))
    if a == 0:
        return np.float32(0), np.zeros(x.shape, dtype=np.int64)
    s = np.float32(a / q)                       # fp32 division
    c = np.rint(np.float32(x / s))              # fp32 division, half to even
    return s, np.clip(c, -QMAX[level], QMAX[level]).astype(np.int64)


def encode(p16, prec, offsets, total):
    """The message (uint8 [total]) for the fp16 partial vector p16 [n]."""
    p16 = np.asarray(p16, dtype=np.float16)
    msg = np.zeros(total, dtype=np.uint8)
    for b, level in enumerate(prec):
        level = int(level)
        blk = p16[b * BLOCK:(b + 1) * BLOCK]
        o = int(offsets[b])
        if level == FP16:
            msg[o:o + 64] = np.frombuffer(blk.tobytes(), dtype=np.uint8)
        elif level in (INT8, INT4):
            s, c = quantize_block(blk.astype(np.float32), level)
            msg[o:o + 4] = np.frombuffer(np.float32(s).tobytes(), dtype=np.uint8)
            if level == INT8:
                msg[o + 4:o + 36] = (c & 0xFF).astype(np.uint8)
            else:
                nib = (c & 0xF).astype(np.uint8)
                msg[o + 4:o + 20] = nib[0::2] | (nib[1::2] << 4)
    return msg


def decode(msg, prec, offsets, n):
    """Values (float64 [n]) a receiver reconstructs from the message."""
    msg = np.asarray(msg, dtype=np.uint8)
    out = np.zeros(n)
    for b, level in enumerate(prec):
        level = int(level)
        o = int(offsets[b])
        sl = slice(b * BLOCK, (b + 1) * BLOCK)
        if level == FP16:
            out[sl] = np.frombuffer(msg[o:o + 64].tobytes(), dtype=np.float16).astype(np.float64)
        elif level in (INT8, INT4):
            s = np.frombuffer(msg[o:o + 4].tobytes(), dtype=np.float32)[0]
            if level == INT8:
                c = msg[o + 4:o + 36].astype(np.int64)
                c = np.where(c > 127, c - 256, c)
            else:
                by = msg[o + 4:o + 20].astype(np.int64)
                c = np.empty(BLOCK, dtype=np.int64)
                c[0::2], c[1::2] = by & 0xF, by >> 4
                c = np.where(c > 7, c - 16, c)
            out[sl] = (c.astype(np.float32) * np.float32(s)).astype(np.float64)
    return out
