"""Oracle: the tile-streaming form of routed attention (test infrastructure only).

Restates, for one query row, the algorithm in the paper's own order:

  * Section 3.1: key/value tiles n = 0 .. T_n - 1 of BLOCK_N tokens are
    streamed; the state (m~, z~, O~) starts at (-inf, 0, 0) and after each
    tile becomes
        m~' = max(m~, rowmax S^n)
        z~' = exp(m~ - m~') z~ + rowsum exp(S^n - m~')
        O~' = exp(m~ - m~') O~ + exp(S^n - m~') V_n
    and the output is O~ / z~ after the last tile.
  * Section 4.3: the score tile S^n is built by the path that the routing bit
    of group g_j = floor(n / g) selects (looked up once per tile here, not per
    key as in oracle/attention.py).

Float64 throughout; used only to pin oracle/attention.py (the two must agree
to rounding), never as a reference for the GPU on its own.
"""

from __future__ import annotations

import math

import numpy as np

from .quantize import QUANT_BLOCK_Q, QUANT_BLOCK_K
from .routing import route_bit


def streaming_attention_row(Q, K, V, route_bits, operands, *, b: int, h_q: int, i: int,
                            block_m: int, block_n: int, group_size: int, causal: bool,
                            scale: float) -> np.ndarray:
    B, Lq, Hq, d = Q.shape
    Lk, Hk = K.shape[1], K.shape[2]
    h_k = h_q // (Hq // Hk)
    m = i // block_m
    m_run, z_run, o_run = -math.inf, 0.0, np.zeros(d, dtype=np.float64)
    q64 = Q[b, i, h_q, :].astype(np.float64)
    q8 = operands.q8[b, i, h_q, :].astype(np.int64)
    dq = float(operands.dq[b, i // QUANT_BLOCK_Q, h_q])
    for n in range(math.ceil(Lk / block_n)):
        lo, hi = n * block_n, min(Lk, (n + 1) * block_n)
        keys = np.arange(lo, hi)
        if causal:
            keys = keys[keys <= i + (Lk - Lq)]
        if keys.size == 0:
            continue
        if route_bit(route_bits, b, h_k, m, n // group_size) == 1:
            c = operands.k8[b, keys, h_k, :].astype(np.int64) @ q8
            dk = operands.dk[b, keys // QUANT_BLOCK_K, h_k].astype(np.float64)
            s = scale * dq * dk * c.astype(np.float64)
        else:
            s = scale * (K[b, keys, h_k, :].astype(np.float64) @ q64)
        m_new = max(m_run, float(np.max(s)))
        alpha = math.exp(m_run - m_new) if m_run != -math.inf else 0.0
        p = np.exp(s - m_new)
        z_run = alpha * z_run + float(np.sum(p))
        o_run = alpha * o_run + p @ V[b, keys, h_k, :].astype(np.float64)
        m_run = m_new
    if z_run == 0.0:
        return np.zeros(d, dtype=np.float64)
    return o_run / z_run
