"""Oracle: routing-word lookup (test infrastructure only).

Follows Section 4.2 ("Why grouping is needed", "Bitmask packing",
"Constant-time lookup") and Section 4.3 ("Tile-group dispatch"):

  * key tile n = floor(j / BLOCK_N) belongs to routing group g_j = floor(n / g);
  * the decisions of one (h_k, m) row are packed little-endian into 64-bit
    words, bit g_j of the row selects the path, 1 = INT8 and 0 = FP16;
  * the decision is (word >> g_j) & 1.

Reading beyond the paper: the paper keeps one word per row (at most 64 groups
per row).  Rows with more groups continue into further words: group g_j lives
in word floor(g_j / 64) at bit g_j mod 64.  With one word per row this is the
paper's layout bit for bit.  The route array carries a leading batch axis of
size 1 (one map shared by every sequence, as in the paper) or B.

Pins: tests/test_oracle_routing.py (hand-packed words, multi-word rows,
group/tile mapping against a brute-force table).
"""

from __future__ import annotations

import numpy as np


def route_bit(route_bits: np.ndarray, b: int, h_k: int, m: int, g_j: int) -> int:
    """Return R[h_k, m, g_j] (1 = INT8, 0 = FP16) for sequence ``b``.

    ``route_bits``: uint64 array [B_r, H_k, T_m, W], B_r in {1, B}.
    """
    rb = np.asarray(route_bits, dtype=np.uint64)
    b_r = b if rb.shape[0] > 1 else 0
    word = int(rb[b_r, h_k, m, g_j // 64])
    return (word >> (g_j % 64)) & 1


def route_bits_for_keys(route_bits: np.ndarray, b: int, h_k: int, i: int, keys: np.ndarray,
                        block_m: int, block_n: int, group_size: int) -> np.ndarray:
    """Route bit for query token ``i`` against each key token in ``keys``.

    Query token i lies in query tile m = floor(i / BLOCK_M); key token j lies in
    key tile n = floor(j / BLOCK_N) and routing group g_j = floor(n / g).
    """
    rb = np.asarray(route_bits, dtype=np.uint64)
    b_r = b if rb.shape[0] > 1 else 0
    m = i // block_m
    keys = np.asarray(keys, dtype=np.int64)
    n = keys // block_n
    g_j = n // group_size
    words = rb[b_r, h_k, m, (g_j // 64)].astype(np.uint64)
    shifts = (g_j % 64).astype(np.uint64)
    return ((words >> shifts) & np.uint64(1)).astype(np.int64)
