"""Oracle: blockwise symmetric INT8 quantization (test infrastructure only).

Follows Section 3.2 and Appendix C ("Blockwise INT8 Quantization",
"Quantization Granularity"):

  * one scale per block and per attention head, where a query block is 128
    consecutive tokens by d and a key block is 64 consecutive tokens by d;
  * the scale is the block absmax divided by 127 and is computed in FP32;
  * codes are the nearest integers to x / scale, within [-127, 127];
  * the scale is stored in the operand dtype (FP16).

Readings where the paper is silent:
  * nearest-integer conversion rounds half to even;
  * x / scale is an IEEE FP32 division (not a reciprocal multiply);
  * codes are clamped to [-127, 127] after rounding;
  * a block whose absmax is 0 gets codes 0 and scale 0;
  * the codes come from the FP32 scale, the score rescale uses the FP16-stored
    scale;
  * the last block of a sequence holds only the rows that exist.

Pins: tests/test_oracle_quantize.py (hand-worked golden block with rounding
ties, code range, per-block extreme code 127, reconstruction bound delta/2,
zero block, scale round trip).
"""

from __future__ import annotations

import math

import numpy as np

QUANT_BLOCK_Q = 128  # query block rows (Appendix C, BLK_Q)
QUANT_BLOCK_K = 64   # key block rows (Appendix C, BLK_K)


def quantize_one_block(block_fp16: np.ndarray) -> tuple[np.ndarray, np.float16]:
    """Quantize one block (any shape) of FP16 values.

    Returns (codes as int8 array of the same shape, scale as float16).
    """
    x32 = np.asarray(block_fp16, dtype=np.float16).astype(np.float32)
    absmax = np.float32(np.max(np.abs(x32))) if x32.size else np.float32(0.0)
    if absmax == np.float32(0.0):
        return np.zeros(x32.shape, dtype=np.int8), np.float16(0.0)
    delta32 = np.float32(absmax / np.float32(127.0))          # FP32 scale
    ratio = (x32 / delta32).astype(np.float32)                 # IEEE FP32 divide
    codes = np.clip(np.rint(ratio), -127.0, 127.0)             # round half to even
    return codes.astype(np.int8), np.float16(delta32)          # scale stored FP16


def quantize_blocks(x: np.ndarray, block_rows: int, heads=None) -> tuple[np.ndarray, np.ndarray]:
    """Quantize X of shape [B, L, H, d] in blocks of ``block_rows`` tokens per head.

    ``heads`` optionally restricts the work to a list of (b, h) pairs; other
    entries of the outputs are left at zero.

    Returns:
      codes: int8 [B, L, H, d]
      delta: float16 [B, ceil(L / block_rows), H]
    """
    x = np.asarray(x)
    if x.ndim != 4:
        raise ValueError("expected [B, L, H, d]")
    B, L, H, d = x.shape
    nblk = math.ceil(L / block_rows) if L else 0
    codes = np.zeros((B, L, H, d), dtype=np.int8)
    delta = np.zeros((B, nblk, H), dtype=np.float16)
    pairs = [(b, h) for b in range(B) for h in range(H)] if heads is None else list(heads)
    for b, h in pairs:
        for r in range(nblk):
            lo = r * block_rows
            hi = min(L, lo + block_rows)
            c, s = quantize_one_block(x[b, lo:hi, h, :])
            codes[b, lo:hi, h, :] = c
            delta[b, r, h] = s
    return codes, delta
