"""Test infrastructure only: the reference of the block-quantised weight
shards used by precision scaling (paper Sec. 2.2 precision heterogeneity,
Sec. 4.2.2 importance-aware mixed precision, Sec. 4.3.1 precision scaling).
Nothing in the product imports this module.

What the paper fixes: a layer's weights may be held at FP16, INT8 or INT4,
a precision per layer chosen by importance; the system uses an existing
family of block quantisation formats (Sec. 5.1) whose definition is not
part of the paper.

Readings where the paper is silent (a format of this build's own, stated
once here and in the design notes):
* blocks of 32 consecutive input columns of one row (the last block of a
  row may be partial; its missing columns count as zero);
* symmetric absmax scale per block, stored as fp16: s = fp16(absmax / Q)
  with the division in fp32 and round-to-nearest-even conversion, Q = 127
  (INT8) or 7 (INT4);
* code = clamp(rint(w / s), -Q, Q), w and s as fp32, the division in fp32,
  rint rounding half to even; a block whose s is zero (all zero, or so
  small that absmax / Q underflows fp16) has all codes 0;
* value = code * s;
* storage of a row: INT8 codes as two's-complement bytes, byte k = column
  k; INT4 codes as offset-binary nibbles u = code + 8 (1..15), in groups of
  8 columns per 4 bytes: column 8g + i (i < 4) in the low nibble of byte
  4g + i, column 8g + 4 + i in its high nibble (so the low nibbles of a
  32-bit word are 4 consecutive columns, and so are the high ones); the
  codes of a row's padded tail are 0. Scales: one fp16 per block, in column
  order.

Floating-point steps that decide an integer (the codes) are taken in fp32,
the precision the device kernels use.
"""
import numpy as np

INT8, INT4 = 1, 2
BLOCK = 32
QMAX = {INT8: 127, INT4: 7}


def n_blocks(cols):
    return (cols + BLOCK - 1) // BLOCK


def quantize_rows(w, level):
    """Codes and scales of the fp16 matrix w [rows, cols].

    Returns (codes int64 [rows, n_blocks * 32], scales float16 [rows, n_blocks]).
    """
    w = np.asarray(w, dtype=np.float16)
    rows, cols = w.shape
    nb = n_blocks(cols)
    q = np.float32(QMAX[level])
    padded = np.zeros((rows, nb * BLOCK), dtype=np.float32)
    padded[:, :cols] = w.astype(np.float32)
    blocks = padded.reshape(rows, nb, BLOCK)
    absmax = np.max(np.abs(blocks), axis=2)
    scales = (absmax / q).astype(np.float32).astype(np.float16)   # fp32 division, then fp16
    s32 = scales.astype(np.float32)[:, :, None]
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(s32 > 0, blocks / np.where(s32 > 0, s32, np.float32(1)), np.float32(0))
    codes = np.clip(np.rint(ratio.astype(np.float32)), -QMAX[level], QMAX[level]).astype(np.int64)
    return codes.reshape(rows, nb * BLOCK), scales


def dequantize(codes, scales, cols):
    """The values (float64 [rows, cols]) the codes and scales stand for."""
    codes = np.asarray(codes, dtype=np.int64)
    rows = codes.shape[0]
    nb = scales.shape[1]
    s = np.asarray(scales, dtype=np.float16).astype(np.float64)
    v = codes.reshape(rows, nb, BLOCK).astype(np.float64) * s[:, :, None]
    return v.reshape(rows, nb * BLOCK)[:, :cols]


def pack_codes(codes, level):
    """Row bytes of the codes (uint8 [rows, n_blocks * 32 or * 16])."""
    codes = np.asarray(codes, dtype=np.int64)
    if level == INT8:
        return (codes & 0xFF).astype(np.uint8)
    u = (codes + 8).astype(np.uint8)
    rows, n = u.shape
    g = u.reshape(rows, n // 8, 2, 4)            # [group][low half / high half][i]
    return (g[:, :, 0, :] | (g[:, :, 1, :] << 4)).reshape(rows, n // 2).astype(np.uint8)


def unpack_codes(packed, level):
    """Inverse of pack_codes."""
    b = np.asarray(packed, dtype=np.uint8).astype(np.int64)
    if level == INT8:
        return np.where(b > 127, b - 256, b)
    rows, nb = b.shape
    g = b.reshape(rows, nb // 4, 1, 4)
    out = np.concatenate([(g & 0xF) - 8, (g >> 4) - 8], axis=2)   # [group][half][i]
    return out.reshape(rows, nb * 2)


def dequantized(w, level):
    """w [rows, cols] as the quantised shard holds it (float64)."""
    codes, scales = quantize_rows(w, level)
    return dequantize(codes, scales, np.asarray(w).shape[1])


def code_bytes_per_row(cols, level):
    return n_blocks(cols) * (BLOCK if level == INT8 else BLOCK // 2)
