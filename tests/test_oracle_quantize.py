"""Pins for oracle/quantize.py (Appendix C, blockwise symmetric INT8 quantization)."""

import numpy as np
import pytest

from conftest import read_golden
from oracle.quantize import quantize_one_block, quantize_blocks, QUANT_BLOCK_Q, QUANT_BLOCK_K


@pytest.mark.parametrize("name", ["quant_block_ties.txt", "quant_block_scale2.txt"])
def test_golden_blocks(name):
    rows = read_golden(name)
    scale = float(rows[0][1])
    x = np.array([float(r[0]) for r in rows[1:]], dtype=np.float16)
    want = np.array([int(r[1]) for r in rows[1:]], dtype=np.int8)
    codes, delta = quantize_one_block(x)
    assert float(delta) == scale
    np.testing.assert_array_equal(codes, want)


def _blocks(seed):
    rng = np.random.default_rng(seed)
    out = []
    for scale in [1e-3, 0.5, 1.0, 3.0, 40.0]:
        x = (rng.standard_normal((128, 64)) * scale).astype(np.float16)
        out.append(x)
    x = rng.standard_normal((64, 128)).astype(np.float16)
    x[:, 7] = (x[:, 7].astype(np.float32) * 8).astype(np.float16)  # outlier channel
    out.append(x)
    out.append(np.full((3, 5), -2.0, dtype=np.float16))  # constant block
    return out


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_code_range_extreme_and_reconstruction(seed):
    for x in _blocks(seed):
        codes, d16 = quantize_one_block(x)
        x32 = x.astype(np.float32)
        absmax = np.max(np.abs(x32))
        d32 = np.float32(absmax / np.float32(127))
        assert codes.dtype == np.int8
        assert np.max(np.abs(codes.astype(np.int32))) == 127      # the absmax element maps to +-127
        assert np.all(np.abs(codes.astype(np.int32)) <= 127)
        # the element attaining the absmax gets the extreme code with the right sign
        k = np.argmax(np.abs(x32))
        assert codes.flat[k] == (127 if x32.flat[k] > 0 else -127)
        # nearest integer: |x - d32 * code| <= d32 / 2 (+ one fp32 rounding of x / d32)
        err = np.abs(x32.astype(np.float64) - np.float64(d32) * codes.astype(np.float64))
        assert np.all(err <= np.float64(d32) * (0.5 + 2.0 ** -17))
        # the stored scale is the FP16 (round-to-nearest-even) image of the FP32 scale
        assert d16 == np.float16(d32)


def test_zero_block():
    codes, d16 = quantize_one_block(np.zeros((64, 128), dtype=np.float16))
    assert float(d16) == 0.0
    assert not codes.any()


def test_sign_symmetry():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((64, 32)).astype(np.float16)
    c1, d1 = quantize_one_block(x)
    c2, d2 = quantize_one_block(-x)
    assert d1 == d2
    np.testing.assert_array_equal(c1, -c2)


def test_block_partition_and_heads():
    rng = np.random.default_rng(7)
    B, L, H, d = 2, 300, 3, 16
    x = rng.standard_normal((B, L, H, d)).astype(np.float16)
    codes, delta = quantize_blocks(x, QUANT_BLOCK_Q)
    assert delta.shape == (B, 3, H)          # ceil(300 / 128) blocks, last holds 44 rows
    # each block is the single-block quantizer applied to exactly those rows of one head
    for b in range(B):
        for h in range(H):
            for r, (lo, hi) in enumerate([(0, 128), (128, 256), (256, 300)]):
                c, s = quantize_one_block(x[b, lo:hi, h, :])
                assert delta[b, r, h] == s
                np.testing.assert_array_equal(codes[b, lo:hi, h, :], c)
    # a large value in row 128 of head 1 changes block 1 of head 1 only
    y = x.copy()
    y[0, 128, 1, 0] = np.float16(100.0)
    _, delta2 = quantize_blocks(y, QUANT_BLOCK_Q)
    changed = np.argwhere(delta2 != delta)
    assert [tuple(c) for c in changed] == [(0, 1, 1)]
    # key blocks are 64 rows
    _, dk = quantize_blocks(x, QUANT_BLOCK_K)
    assert dk.shape == (B, 5, H)


def test_heads_subset_matches_full():
    rng = np.random.default_rng(9)
    x = rng.standard_normal((2, 130, 4, 8)).astype(np.float16)
    full_c, full_d = quantize_blocks(x, QUANT_BLOCK_K)
    sub_c, sub_d = quantize_blocks(x, QUANT_BLOCK_K, heads=[(1, 2)])
    np.testing.assert_array_equal(sub_c[1, :, 2], full_c[1, :, 2])
    np.testing.assert_array_equal(sub_d[1, :, 2], full_d[1, :, 2])
    assert not sub_c[0].any()
