"""CPU oracle for TileMix routed prefill attention -- TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, obviously-correct NumPy restatement of what the
routed attention path computes, in float64 for floating point and int64 for the
INT8 score products.  It exists to check the HIP implementation; it is not a
fallback.  Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline``
leg of ``bench.py`` may import or call it.  It shares no code with the HIP path
(``paper_2608_17336_amd``) and imports nothing from it.

Passages followed (TileMix, arXiv 2608.17336):
  * Section 3.1  -- tiled attention and the online-softmax recurrence.
  * Section 3.2 and Appendix C -- blockwise symmetric INT8 quantization,
    quantization granularity (128-row query blocks, 64-row key blocks), the
    INT8 score computation with INT32 accumulation and scale restoration.
  * Section 4.1  -- GQA head mapping h_k = floor(h_q / (H_q / H_k)).
  * Section 4.2  -- grouping factor g, packed routing words, shift-and-mask lookup.
  * Section 4.3  -- tile-group dispatch equation (INT8 vs FP16 score tile).

Every function is pinned by ``tests/test_oracle_*.py`` against closed forms,
invariants, brute force on tiny inputs and a library routine (torch CPU SDPA);
see the module docstrings for which pin covers what.
"""

from .quantize import quantize_blocks, QUANT_BLOCK_Q, QUANT_BLOCK_K
from .routing import route_bit, route_bits_for_keys
from .attention import (
    routed_attention_rows,
    exact_attention_rows,
    int8_tile_product,
    OracleOperands,
)
from .streaming import streaming_attention_row

__all__ = [
    "quantize_blocks",
    "QUANT_BLOCK_Q",
    "QUANT_BLOCK_K",
    "route_bit",
    "route_bits_for_keys",
    "routed_attention_rows",
    "exact_attention_rows",
    "int8_tile_product",
    "OracleOperands",
    "streaming_attention_row",
]
