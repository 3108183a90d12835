"""Oracle: routed causal prefill attention, row by row (test infrastructure only).

What is computed, and where the paper states it:

  * Section 3.1: S = Q K^T / sqrt(d) (the scale is passed in), P = softmax(S)
    over the legal keys of each query row, O = P V.  The online-softmax
    recurrence of Section 3.1 reaches exactly this result (up to rounding
    order); oracle/streaming.py restates the recurrence itself and the tests
    check that the two agree.
  * Section 4.1: query head h_q reads KV head h_k = floor(h_q / (H_q / H_k)).
  * Sections 4.2 and 4.3: the routing bit of the tile group holding key j in
    query-tile row m selects the score of the pair (i, j):
      bit 0 (FP16 path):  s = scale * sum_c Q[i, c] K[j, c]
      bit 1 (INT8 path):  s = scale * dQ[r] * dK[s] * C,
                          C = sum_c Q8[i, c] K8[j, c]  (exact integer),
    where r = floor(i / 128) and s = floor(j / 64) are the quantization
    blocks of Appendix C and dQ, dK are the FP16-stored block scales.
  * Legality (Section 4.1, Appendix B): causal and boundary masks decide which
    (i, j) exist, independent of routing.  Key j is legal for query i iff
    j < L_k and, when causal, j <= i + (L_k - L_q) (bottom-right alignment,
    which is plain j <= i when L_q == L_k).

All floating point here is float64; the integer products are int64.  The
INT8 operands come from oracle/quantize.py, never from the HIP path.

Pins: tests/test_oracle_attention.py -- pure-Python brute force on tiny
shapes, torch CPU scaled_dot_product_attention (float64) for the all-FP16
mask, V == 1 gives O == 1, O[0] == V[0], causal perturbation, the
integer-valued special case where both routes coincide, the closed-form INT8
score error bound, and agreement with the streaming recurrence.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .quantize import quantize_blocks, QUANT_BLOCK_Q, QUANT_BLOCK_K
from .routing import route_bits_for_keys


@dataclass
class OracleOperands:
    """The oracle's own INT8 forms of Q and K with their FP16 block scales."""
    q8: np.ndarray   # int8 [B, Lq, Hq, d]
    dq: np.ndarray   # float16 [B, ceil(Lq/128), Hq]
    k8: np.ndarray   # int8 [B, Lk, Hk, d]
    dk: np.ndarray   # float16 [B, ceil(Lk/64), Hk]

    @staticmethod
    def from_inputs(Q: np.ndarray, K: np.ndarray, q_heads=None, k_heads=None) -> "OracleOperands":
        q8, dq = quantize_blocks(Q, QUANT_BLOCK_Q, heads=q_heads)
        k8, dk = quantize_blocks(K, QUANT_BLOCK_K, heads=k_heads)
        return OracleOperands(q8, dq, k8, dk)


def _legal_keys(i: int, Lq: int, Lk: int, causal: bool) -> np.ndarray:
    if causal:
        last = min(Lk - 1, i + (Lk - Lq))
        return np.arange(0, last + 1, dtype=np.int64) if last >= 0 else np.zeros(0, np.int64)
    return np.arange(0, Lk, dtype=np.int64)


def _softmax_output(s: np.ndarray, v: np.ndarray, d: int) -> np.ndarray:
    """O = softmax(s) @ v for one row, float64; an empty row gives zeros."""
    if s.size == 0:
        return np.zeros(d, dtype=np.float64)
    p = np.exp(s - np.max(s))
    return (p @ v) / np.sum(p)


def _head_map(Hq: int, Hk: int, h_q: int) -> int:
    if Hq % Hk:
        raise ValueError("H_q must be a multiple of H_k")
    return h_q // (Hq // Hk)


def _normalize_rows(rows):
    out = []
    for b, h_q, idx in rows:
        out.append((int(b), int(h_q), np.atleast_1d(np.asarray(idx, dtype=np.int64))))
    return out


def routed_attention_rows(Q, K, V, route_bits, *, block_m: int, block_n: int, group_size: int,
                          causal: bool, scale: float, rows, operands: OracleOperands | None = None,
                          want_scores: bool = False):
    """Routed attention output for selected rows.

    Q: fp16 [B, Lq, Hq, d]; K, V: fp16 [B, Lk, Hk, d];
    route_bits: uint64 [B_r, Hk, T_m, W];
    rows: list of (b, h_q, query indices).

    Returns a list of float64 arrays [len(indices), d] (and, if
    ``want_scores``, a parallel list of per-row (keys, bits, scores) tuples).
    """
    Q = np.asarray(Q); K = np.asarray(K); V = np.asarray(V)
    B, Lq, Hq, d = Q.shape
    _, Lk, Hk, _ = K.shape
    rows = _normalize_rows(rows)
    if operands is None:
        q_heads = sorted({(b, h) for b, h, _ in rows})
        k_heads = sorted({(b, _head_map(Hq, Hk, h)) for b, h, _ in rows})
        operands = OracleOperands.from_inputs(Q, K, q_heads, k_heads)
    outs, scores = [], []
    cache = {}
    for b, h_q, idx in rows:
        h_k = _head_map(Hq, Hk, h_q)
        if (b, h_k) not in cache:
            cache = {(b, h_k): (K[b, :, h_k, :].astype(np.float64),
                                V[b, :, h_k, :].astype(np.float64),
                                operands.k8[b, :, h_k, :].astype(np.int64),
                                operands.dk[b, :, h_k].astype(np.float64))}
        k64, v64, k8, dk = cache[(b, h_k)]
        o = np.zeros((idx.size, d), dtype=np.float64)
        row_scores = []
        for t, i in enumerate(idx):
            keys = _legal_keys(int(i), Lq, Lk, causal)
            if keys.size == 0:
                row_scores.append((keys, keys, np.zeros(0)))
                continue
            bits = route_bits_for_keys(route_bits, b, h_k, int(i), keys, block_m, block_n, group_size)
            sel = slice(int(keys[0]), int(keys[-1]) + 1)      # legal keys are one contiguous run
            q64 = Q[b, i, h_q, :].astype(np.float64)
            s_fp16_path = scale * (k64[sel] @ q64)
            c_int = k8[sel] @ operands.q8[b, i, h_q, :].astype(np.int64)         # exact int64
            dq = np.float64(operands.dq[b, i // QUANT_BLOCK_Q, h_q])
            s_int8_path = scale * dq * dk[keys // QUANT_BLOCK_K] * c_int.astype(np.float64)
            s = np.where(bits == 1, s_int8_path, s_fp16_path)
            o[t] = _softmax_output(s, v64[sel], d)
            if want_scores:
                row_scores.append((keys, bits, s))
        outs.append(o)
        scores.append(row_scores)
    return (outs, scores) if want_scores else outs


def exact_attention_rows(Q, K, V, *, causal: bool, scale: float, rows):
    """Textbook softmax attention (Section 3.1) on the FP16 inputs, float64.

    This is the definition the all-FP16 routing reduces to (the "Zero" layout
    of Appendix B routes every legal group to FP16).
    """
    Q = np.asarray(Q); K = np.asarray(K); V = np.asarray(V)
    B, Lq, Hq, d = Q.shape
    _, Lk, Hk, _ = K.shape
    outs = []
    for b, h_q, idx in _normalize_rows(rows):
        h_k = _head_map(Hq, Hk, h_q)
        k64 = K[b, :, h_k, :].astype(np.float64)
        v64 = V[b, :, h_k, :].astype(np.float64)
        o = np.zeros((idx.size, d), dtype=np.float64)
        for t, i in enumerate(idx):
            keys = _legal_keys(int(i), Lq, Lk, causal)
            s = scale * (k64[keys] @ Q[b, i, h_q, :].astype(np.float64))
            o[t] = _softmax_output(s, v64[keys], d)
        outs.append(o)
    return outs


def int8_tile_product(operands: OracleOperands, b: int, h_q: int, h_k: int, m: int, n: int,
                      block_m: int, block_n: int) -> np.ndarray:
    """Exact INT32-path tile C = Q8_m K8_n^T as int64 [BLOCK_M, BLOCK_N].

    Appendix C, INT8 score computation.  Entries whose query or key index lies
    beyond the sequence are 0.
    """
    Lq = operands.q8.shape[1]
    Lk = operands.k8.shape[1]
    out = np.zeros((block_m, block_n), dtype=np.int64)
    q_lo, k_lo = m * block_m, n * block_n
    q_hi, k_hi = min(Lq, q_lo + block_m), min(Lk, k_lo + block_n)
    if q_hi <= q_lo or k_hi <= k_lo:
        return out
    a = operands.q8[b, q_lo:q_hi, h_q, :].astype(np.int64)
    c = operands.k8[b, k_lo:k_hi, h_k, :].astype(np.int64)
    out[: q_hi - q_lo, : k_hi - k_lo] = a @ c.T
    return out
