"""Oracle: routed decode over an INT8 key/value cache (test infrastructure only).

Follows Appendix C, "Additional Execution Interfaces": the cache holds K8 and V8 with
per-block scales; during decode the cached K8 feeds the routed INT8 score path and the
cached V8 enters P.V dequantized by its block scale (folding the scale into P, as the paper
does, is the same number in exact arithmetic).  Scores and routing follow Sections 4.2, 4.3
and Appendix C exactly as in oracle/attention.py; the decode query is the newest token and
sees every cached key.

Readings: V is quantized like K, in 64-token blocks per KV head (the paper says
"per-block scales" without the block shape); the single decode query row forms its own
128-row quantization block.

Pins: tests/test_oracle_decode.py (equals the prefill oracle's last row when V is exactly
representable by its codes; the V-quantization error bound; the all-FP16 route against
exact attention).
"""

from __future__ import annotations

import numpy as np

from .quantize import quantize_blocks, QUANT_BLOCK_Q, QUANT_BLOCK_K


def kv_cache(K: np.ndarray, V: np.ndarray):
    """(K8, dK, V8, dV): the cache of FP16 K, V [B, L_k, H_k, d]."""
    k8, dk = quantize_blocks(K, QUANT_BLOCK_K)
    v8, dv = quantize_blocks(V, QUANT_BLOCK_K)
    return k8, dk, v8, dv


def routed_decode(Q, K, k8, dk, v8, dv, words, group_size: int, scale: float,
                  seqlens=None) -> np.ndarray:
    """O [B, 1, H_q, d] in float64 for one decode token per sequence.

    Q: FP16 [B, 1, H_q, d]; K: FP16 key cache [B, L_k, H_k, d] (FP16 route);
    k8/dk, v8/dv: the INT8 cache; words: uint64 [B_r, H_k, 1, W].
    seqlens: optional per-sequence cache lengths [B]: sequence b attends to its first
    seqlens[b] cached keys only (clamped to [0, L_k]); a sequence with none gets O = 0.
    """
    Q = np.asarray(Q)
    B, _, Hq, d = Q.shape
    Lk, Hk = K.shape[1], K.shape[2]
    q8, dq = quantize_blocks(Q, QUANT_BLOCK_Q)
    words = np.asarray(words, dtype=np.uint64)
    out = np.zeros((B, 1, Hq, d), dtype=np.float64)
    j = np.arange(Lk)
    blk = j // QUANT_BLOCK_K
    gj = (j // 64) // group_size
    for b in range(B):
        br = b if words.shape[0] > 1 else 0
        for hq in range(Hq):
            hk = hq // (Hq // Hk)
            bits = ((words[br, hk, 0, gj // 64] >> (gj % 64).astype(np.uint64)) & np.uint64(1)).astype(bool)
            s16 = scale * (K[b, :, hk, :].astype(np.float64) @ Q[b, 0, hq, :].astype(np.float64))
            c = k8[b, :, hk, :].astype(np.int64) @ q8[b, 0, hq, :].astype(np.int64)
            s8 = scale * float(dq[b, 0, hq]) * dk[b, blk, hk].astype(np.float64) * c.astype(np.float64)
            s = np.where(bits, s8, s16)
            vdeq = dv[b, blk, hk].astype(np.float64)[:, None] * v8[b, :, hk, :].astype(np.float64)
            n = Lk if seqlens is None else min(max(int(seqlens[b]), 0), Lk)
            if n == 0:
                continue
            s, vdeq = s[:n], vdeq[:n]
            p = np.exp(s - s.max())
            out[b, 0, hq] = (p[:, None] * vdeq).sum(axis=0) / p.sum()
    return out
