"""Pins for oracle/attention.py and oracle/streaming.py.

Sections 3.1 (softmax attention, online recurrence), 4.1 (GQA head map),
4.2-4.3 (routing lookup and tile-group dispatch), Appendix C (INT8 score path).
"""

import math

import numpy as np
import pytest

from conftest import read_golden
from oracle import (OracleOperands, exact_attention_rows, routed_attention_rows,
                    streaming_attention_row, int8_tile_product)
from synth import pack_route_bits


# ----------------------------------------------------------------------------- helpers

def _rand_inputs(seed, B, Lq, Lk, Hq, Hk, d, kscale=1.0):
    rng = np.random.default_rng(seed)
    Q = rng.standard_normal((B, Lq, Hq, d)).astype(np.float16)
    K = (rng.standard_normal((B, Lk, Hk, d)) * kscale).astype(np.float16)
    V = rng.standard_normal((B, Lk, Hk, d)).astype(np.float16)
    return Q, K, V


def _rand_route(seed, Hk, T_m, T_mask, p=0.5, B_r=1):
    rng = np.random.default_rng(seed + 1000)
    R = (rng.random((B_r, Hk, T_m, T_mask)) < p).astype(np.uint8)
    return np.concatenate([pack_route_bits(R[b]) for b in range(B_r)], axis=0), R


def _all_rows(B, Hq, Lq):
    return [(b, h, np.arange(Lq)) for b in range(B) for h in range(Hq)]


# --------------------------------------------------------------- pure-Python brute force

def _bf_quant_block(vals):
    """Scalar restatement of Appendix C for one block (list of python floats)."""
    absmax = max((abs(v) for v in vals), default=0.0)
    if absmax == 0.0:
        return [0] * len(vals), 0.0
    d32 = np.float32(np.float32(absmax) / np.float32(127.0))
    codes = []
    for v in vals:
        r = float(np.float32(np.float32(v) / d32))
        codes.append(max(-127, min(127, round(r))))     # python round(): half to even
    return codes, float(np.float16(d32))


def _bf_attention(Q, K, V, R, *, bm, bn, g, causal, scale):
    """Pure-Python loops with math.fsum; R is the unpacked 0/1 map [B_r, Hk, T_m, T_mask]."""
    B, Lq, Hq, d = Q.shape
    Lk, Hk = K.shape[1], K.shape[2]
    q = Q.astype(np.float64).tolist()
    k = K.astype(np.float64).tolist()
    v = V.astype(np.float64).tolist()
    # quantize: query blocks of 128 rows, key blocks of 64 rows, per (b, head)
    q8 = [[[None] * Lq for _ in range(Hq)] for _ in range(B)]
    dq = {}
    for b in range(B):
        for h in range(Hq):
            for r0 in range(0, Lq, 128):
                rows = range(r0, min(Lq, r0 + 128))
                codes, s = _bf_quant_block([q[b][i][h][c] for i in rows for c in range(d)])
                dq[(b, r0 // 128, h)] = s
                for t, i in enumerate(rows):
                    q8[b][h][i] = codes[t * d:(t + 1) * d]
    k8 = [[[None] * Lk for _ in range(Hk)] for _ in range(B)]
    dk = {}
    for b in range(B):
        for h in range(Hk):
            for r0 in range(0, Lk, 64):
                rows = range(r0, min(Lk, r0 + 64))
                codes, s = _bf_quant_block([k[b][j][h][c] for j in rows for c in range(d)])
                dk[(b, r0 // 64, h)] = s
                for t, j in enumerate(rows):
                    k8[b][h][j] = codes[t * d:(t + 1) * d]
    out = np.zeros((B, Lq, Hq, d))
    for b in range(B):
        for hq in range(Hq):
            hk = (hq * Hk) // Hq
            for i in range(Lq):
                keys = [j for j in range(Lk) if (not causal) or j <= i + (Lk - Lq)]
                if not keys:
                    continue
                s = []
                for j in keys:
                    bit = int(R[b if R.shape[0] > 1 else 0, hk, i // bm, (j // bn) // g])
                    if bit:
                        cint = sum(q8[b][hq][i][c] * k8[b][hk][j][c] for c in range(d))
                        s.append(scale * dq[(b, i // 128, hq)] * dk[(b, j // 64, hk)] * cint)
                    else:
                        s.append(scale * math.fsum(q[b][i][hq][c] * k[b][j][hk][c] for c in range(d)))
                mx = max(s)
                p = [math.exp(x - mx) for x in s]
                z = math.fsum(p)
                for c in range(d):
                    out[b, i, hq, c] = math.fsum(p[t] * v[b][keys[t]][hk][c] for t in range(len(keys))) / z
    return out


BRUTE_CASES = [
    # B, Lq, Lk, Hq, Hk, d, bm, bn, g, causal, p
    (1, 1, 1, 1, 1, 4, 2, 2, 1, True, 0.5),
    (1, 37, 37, 2, 1, 8, 5, 3, 2, True, 0.5),
    (2, 23, 23, 4, 2, 4, 4, 4, 3, True, 0.7),
    (1, 19, 33, 2, 2, 8, 8, 5, 1, False, 0.5),
    (1, 12, 30, 2, 1, 4, 4, 4, 1, True, 0.5),      # L_q < L_k: bottom-right causal
    (1, 70, 70, 1, 1, 4, 7, 1, 1, True, 0.5),      # 70 groups per row: two words
    (1, 140, 140, 1, 1, 4, 64, 8, 1, True, 0.5),   # crosses a 128-row query block and 64-row key blocks
]


@pytest.mark.parametrize("case", BRUTE_CASES)
def test_bruteforce_agrees(case):
    B, Lq, Lk, Hq, Hk, d, bm, bn, g, causal, p = case
    Q, K, V = _rand_inputs(hash(case) % 1000, B, Lq, Lk, Hq, Hk, d, kscale=2.0)
    T_m, T_n = -(-Lq // bm), -(-Lk // bn)
    words, R = _rand_route(7, Hk, T_m, -(-T_n // g), p)
    got = routed_attention_rows(Q, K, V, words, block_m=bm, block_n=bn, group_size=g,
                                causal=causal, scale=0.3, rows=_all_rows(B, Hq, Lq))
    want = _bf_attention(Q, K, V, R, bm=bm, bn=bn, g=g, causal=causal, scale=0.3)
    for (b, h, idx), o in zip(_all_rows(B, Hq, Lq), got):
        np.testing.assert_allclose(o, want[b, idx, h, :], rtol=1e-12, atol=1e-12)


def test_bruteforce_per_sequence_route_maps():
    B, L, H, d, bm, bn = 2, 20, 1, 4, 4, 4
    Q, K, V = _rand_inputs(11, B, L, L, H, H, d)
    words, R = _rand_route(3, H, 5, 5, 0.5, B_r=2)
    got = routed_attention_rows(Q, K, V, words, block_m=bm, block_n=bn, group_size=1,
                                causal=True, scale=0.5, rows=_all_rows(B, H, L))
    want = _bf_attention(Q, K, V, R, bm=bm, bn=bn, g=1, causal=True, scale=0.5)
    for (b, h, idx), o in zip(_all_rows(B, H, L), got):
        np.testing.assert_allclose(o, want[b, idx, h, :], rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------------ worked example

def test_worked_example_l2_d2():
    rows = read_golden("worked_example_l2_d2.txt")
    Q = np.array([[[[127, 0]], [[0, 127]]]], dtype=np.float16)     # [1, 2, 1, 2]
    K = np.array([[[[254, 1]], [[3, 254]]]], dtype=np.float16)
    V = np.array([[[[0, 1]], [[1, 0]]]], dtype=np.float16)
    scale = 1.0 / 32258.0
    ops = OracleOperands.from_inputs(Q, K)
    assert float(ops.dq[0, 0, 0]) == 1.0 and float(ops.dk[0, 0, 0]) == 2.0
    assert ops.k8[0, :, 0, :].tolist() == [[127, 0], [2, 127]]
    s_fp16 = [127 * scale, 1.0]
    s_int8 = [0.0, 1.0]
    for _, word, name in rows:
        word = int(word)
        words = np.array([[[[1], [word]]]], dtype=np.uint64)           # [1, 1, T_m=2, W=1]
        o = routed_attention_rows(Q, K, V, words, block_m=1, block_n=1, group_size=1, causal=True,
                                  scale=scale, rows=[(0, 0, [0, 1])], operands=ops)[0]
        s0 = s_int8[0] if word & 1 else s_fp16[0]
        s1 = s_int8[1] if word & 2 else s_fp16[1]
        w0 = 1.0 / (1.0 + math.exp(s1 - s0))
        np.testing.assert_allclose(o[0], [0.0, 1.0], atol=0, rtol=0)
        np.testing.assert_allclose(o[1], [1.0 - w0, w0], rtol=1e-14, atol=1e-15), name
    # the two routes really differ here (key 0's small K component is lost in INT8)
    assert abs(1.0 / (1.0 + math.exp(1.0 - s_fp16[0])) - 1.0 / (1.0 + math.exp(1.0))) > 5e-4


# ------------------------------------------------------------- library routine / invariants

@pytest.mark.parametrize("causal", [True, False])
def test_all_fp16_equals_torch_sdpa(causal):
    torch = pytest.importorskip("torch")
    B, L, Hq, Hk, d = 2, 150, 4, 2, 16
    Q, K, V = _rand_inputs(21, B, L, L, Hq, Hk, d)
    words = np.zeros((1, Hk, 2, 1), dtype=np.uint64)                  # all FP16
    scale = 1.0 / math.sqrt(d)
    got = routed_attention_rows(Q, K, V, words, block_m=128, block_n=64, group_size=1, causal=causal,
                                scale=scale, rows=_all_rows(B, Hq, L))
    q = torch.from_numpy(Q.astype(np.float64)).permute(0, 2, 1, 3)
    k = torch.from_numpy(K.astype(np.float64)).permute(0, 2, 1, 3).repeat_interleave(Hq // Hk, dim=1)
    v = torch.from_numpy(V.astype(np.float64)).permute(0, 2, 1, 3).repeat_interleave(Hq // Hk, dim=1)
    ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=causal, scale=scale)
    ref = ref.permute(0, 2, 1, 3).numpy()
    for (b, h, idx), o in zip(_all_rows(B, Hq, L), got):
        np.testing.assert_allclose(o, ref[b, idx, h, :], rtol=1e-11, atol=1e-12)
    ex = exact_attention_rows(Q, K, V, causal=causal, scale=scale, rows=_all_rows(B, Hq, L))
    for a, e in zip(got, ex):
        np.testing.assert_array_equal(a, e)


@pytest.mark.parametrize("p", [0.0, 0.5, 1.0])
def test_value_ones_gives_ones_and_first_row(p):
    B, L, Hq, Hk, d = 1, 200, 2, 1, 8
    Q, K, _ = _rand_inputs(4, B, L, L, Hq, Hk, d, kscale=3.0)
    words, _ = _rand_route(5, Hk, 2, 4, p)
    ones = np.ones((B, L, Hk, d), dtype=np.float16)
    o = routed_attention_rows(Q, K, ones, words, block_m=128, block_n=64, group_size=1, causal=True,
                              scale=0.25, rows=_all_rows(B, Hq, L))
    for x in o:
        np.testing.assert_allclose(x, 1.0, rtol=1e-13)
    _, _, V = _rand_inputs(6, B, L, L, Hq, Hk, d)
    o = routed_attention_rows(Q, K, V, words, block_m=128, block_n=64, group_size=1, causal=True,
                              scale=0.25, rows=[(0, h, [0]) for h in range(Hq)])
    for h in range(Hq):
        np.testing.assert_array_equal(o[h][0], V[0, 0, 0].astype(np.float64))


def test_causal_perturbation():
    B, L, Hq, Hk, d = 1, 300, 2, 1, 16
    Q, K, V = _rand_inputs(8, B, L, L, Hq, Hk, d)
    words, _ = _rand_route(9, Hk, 3, 5, 0.5)
    kw = dict(block_m=128, block_n=64, group_size=1, causal=True, scale=0.25)
    rows = [(0, h, [0, 50, 100, 127]) for h in range(Hq)]
    base = routed_attention_rows(Q, K, V, words, rows=rows, **kw)
    V2, K2 = V.copy(), K.copy()
    V2[0, 128:] = np.float16(7.0)            # every value after row 127
    K2[0, 128:] = np.float16(-9.0)           # key blocks 2.. lie wholly after row 127
    got = routed_attention_rows(Q, K2, V2, words, rows=rows, **kw)
    for a, b in zip(base, got):
        np.testing.assert_array_equal(a, b)
    # Reading: quantize-once sees the whole 64-row key block, so a future key in the same
    # block changes the INT8 scores of earlier queries through the block scale.
    words_all_int8 = np.full((1, Hk, 3, 1), np.uint64(2 ** 5 - 1), dtype=np.uint64)
    K3 = K.copy()
    K3[0, 60, 0, 0] = np.float16(60.0)       # row 60 is in key block 0, after query 50
    a = routed_attention_rows(Q, K, V, words_all_int8, rows=[(0, 0, [50])], **kw)[0]
    b = routed_attention_rows(Q, K3, V, words_all_int8, rows=[(0, 0, [50])], **kw)[0]
    assert not np.array_equal(a, b)


def test_integer_inputs_routes_coincide():
    # Every 128-row Q block and 64-row K block holds integers with absmax exactly 127,
    # so every scale is 1, Q8 = Q, K8 = K, and both score paths give the same numbers.
    rng = np.random.default_rng(12)
    B, L, Hq, Hk, d = 1, 256, 2, 1, 16
    Q = rng.integers(-127, 128, size=(B, L, Hq, d)).astype(np.float16)
    K = rng.integers(-127, 128, size=(B, L, Hk, d)).astype(np.float16)
    Q[:, ::128, :, 0] = 127.0
    K[:, ::64, :, 0] = -127.0
    V = rng.standard_normal((B, L, Hk, d)).astype(np.float16)
    kw = dict(block_m=128, block_n=64, group_size=1, causal=True, scale=1.0 / 4000.0)
    z = routed_attention_rows(Q, K, V, np.zeros((1, Hk, 2, 1), np.uint64), rows=_all_rows(B, Hq, L), **kw)
    o = routed_attention_rows(Q, K, V, np.full((1, Hk, 2, 1), 15, np.uint64), rows=_all_rows(B, Hq, L), **kw)
    for a, b in zip(z, o):
        np.testing.assert_array_equal(a, b)


def test_int8_score_error_bound():
    B, L, Hq, Hk, d = 1, 256, 2, 1, 64
    Q, K, V = _rand_inputs(13, B, L, L, Hq, Hk, d, kscale=1.0)
    K[..., 3] = (K[..., 3].astype(np.float32) * 8).astype(np.float16)
    ops = OracleOperands.from_inputs(Q, K)
    ones = np.full((1, Hk, 2, 1), 15, np.uint64)
    zeros = np.zeros((1, Hk, 2, 1), np.uint64)
    kw = dict(block_m=128, block_n=64, group_size=1, causal=True, scale=1.0, operands=ops, want_scores=True)
    rows = [(0, 0, [5, 130, 255]), (0, 1, [77])]
    _, s8 = routed_attention_rows(Q, K, V, ones, rows=rows, **kw)
    _, s16 = routed_attention_rows(Q, K, V, zeros, rows=rows, **kw)
    for (b, h, idx), r8, r16 in zip(rows, s8, s16):
        for i, (keys, bits8, a), (_, bits16, e) in zip(idx, r8, r16):
            assert bits8.all() and not bits16.any()
            q = Q[b, i, h].astype(np.float64)
            dq16 = float(ops.dq[b, i // 128, h])
            dq32 = float(np.float32(np.max(np.abs(Q[b, (i // 128) * 128:(i // 128) * 128 + 128, h]).astype(np.float32)) / np.float32(127)))
            Eq = dq32 * (0.5 + 2 ** -17) + 127 * abs(dq16 - dq32)
            for t, j in enumerate(keys):
                k = K[b, j, 0].astype(np.float64)
                blk = K[b, (j // 64) * 64:(j // 64) * 64 + 64, 0].astype(np.float32)
                dk32 = float(np.float32(np.max(np.abs(blk)) / np.float32(127)))
                dk16 = float(ops.dk[b, j // 64, 0])
                Ek = dk32 * (0.5 + 2 ** -17) + 127 * abs(dk16 - dk32)
                bound = np.sum(np.abs(q) * Ek + np.abs(k) * Eq + Eq * Ek)
                assert abs(a[t] - e[t]) <= bound * (1 + 1e-9)


@pytest.mark.parametrize("g", [1, 2, 3])
def test_streaming_recurrence_agrees(g):
    B, L, Hq, Hk, d = 1, 333, 4, 2, 8
    Q, K, V = _rand_inputs(15, B, L, L, Hq, Hk, d, kscale=2.0)
    bm, bn = 128, 64
    T_mask = -(-(-(-L // bn)) // g)
    words, _ = _rand_route(16, Hk, 3, T_mask, 0.5)
    ops = OracleOperands.from_inputs(Q, K)
    idx = [0, 1, 63, 64, 127, 128, 200, 255, 256, 332]
    direct = routed_attention_rows(Q, K, V, words, block_m=bm, block_n=bn, group_size=g, causal=True,
                                   scale=0.35, rows=[(0, h, idx) for h in range(Hq)], operands=ops)
    for h in range(Hq):
        for t, i in enumerate(idx):
            s = streaming_attention_row(Q, K, V, words, ops, b=0, h_q=h, i=i, block_m=bm, block_n=bn,
                                        group_size=g, causal=True, scale=0.35)
            np.testing.assert_allclose(s, direct[h][t], rtol=1e-12, atol=1e-13)


def test_gqa_heads_share_kv_and_route():
    B, L, Hq, Hk, d = 1, 130, 4, 2, 8
    Q, K, V = _rand_inputs(17, B, L, L, Hq, Hk, d)
    Q[:, :, 1] = Q[:, :, 0]        # heads 0 and 1 -> KV head 0
    Q[:, :, 3] = Q[:, :, 0]        # head 3 -> KV head 1
    words, _ = _rand_route(18, Hk, 2, 3, 0.5)
    o = routed_attention_rows(Q, K, V, words, block_m=128, block_n=64, group_size=1, causal=True,
                              scale=0.3, rows=[(0, h, np.arange(L)) for h in range(Hq)])
    np.testing.assert_array_equal(o[0], o[1])
    assert not np.array_equal(o[0], o[3])


def test_int8_tile_product_exact_and_ragged():
    B, L, Hq, Hk, d = 1, 150, 2, 1, 32
    Q, K, _ = _rand_inputs(19, B, L, L, Hq, Hk, d)
    ops = OracleOperands.from_inputs(Q, K)
    t = int8_tile_product(ops, 0, 1, 0, 1, 2, 128, 64)      # rows 128..149, keys 128..149
    assert t.shape == (128, 64)
    assert not t[22:].any() and not t[:, 22:].any()
    for i in range(22):
        for j in range(22):
            assert t[i, j] == sum(int(a) * int(b) for a, b in zip(ops.q8[0, 128 + i, 1], ops.k8[0, 128 + j, 0]))
