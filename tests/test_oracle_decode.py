"""Pins of the INT8 key/value cache decode oracle.  CPU only."""

import numpy as np

from oracle import routed_attention_rows
from oracle.decode import kv_cache, routed_decode
from synth import make_qkv, pack_route_bits, small_workload


def _words(Hk, T_mask, rng, p):
    R = (rng.random((Hk, 1, T_mask)) < p).astype(np.uint8)
    return pack_route_bits(R)


def test_equals_prefill_last_row_when_v_is_exact():
    # V integer-valued with absmax 127 in every 64-key block of every head: dV = 1, V8 = V,
    # so decoding must reproduce the prefill oracle's row for one query that sees all keys.
    rng = np.random.default_rng(3)
    cfg = small_workload("dec", B=2, Hq=4, Hk=2, d=64, L=300, group_size=2, index=900)
    Q, K, _ = make_qkv(cfg)
    V = rng.integers(-127, 128, size=K.shape).astype(np.float16)
    V[:, ::64, :, 0] = 127.0
    Q1 = Q[:, -1:]
    k8, dk, v8, dv = kv_cache(K, V)
    assert np.all(dv == np.float16(1.0)) and np.array_equal(v8.astype(np.float16), V)
    T_mask = -(-(-(-300 // 64)) // 2)
    for p in (0.0, 0.5, 1.0):
        words = _words(2, T_mask, rng, p)
        got = routed_decode(Q1, K, k8, dk, v8, dv, words, 2, cfg.scale)
        rows = [(b, h, np.array([0])) for b in range(2) for h in range(4)]
        ref = routed_attention_rows(Q1, K, V, words, block_m=128, block_n=64, group_size=2,
                                    causal=True, scale=cfg.scale, rows=rows)
        for (b, h, _), r in zip(rows, ref):
            np.testing.assert_allclose(got[b, 0, h], r[0], rtol=0, atol=1e-12)


def test_value_quantization_error_bound():
    # |O_decode - O_exact| <= max_j dV_j / 2 elementwise: every dequantized value is within
    # half a step of V and the softmax weights are a convex combination.
    cfg = small_workload("dec2", B=1, Hq=2, Hk=1, d=128, L=700, group_size=1, index=901)
    Q, K, V = make_qkv(cfg)
    Q1 = Q[:, -1:]
    k8, dk, v8, dv = kv_cache(K, V)
    words = pack_route_bits(np.zeros((1, 1, 11), np.uint8))    # all FP16 scores
    got = routed_decode(Q1, K, k8, dk, v8, dv, words, 1, cfg.scale)
    rows = [(0, h, np.array([0])) for h in range(2)]
    ref = routed_attention_rows(Q1, K, V, words, block_m=128, block_n=64, group_size=1,
                                causal=True, scale=cfg.scale, rows=rows)
    bound = float(dv.astype(np.float64).max()) / 2
    for (_, h, _), r in zip(rows, ref):
        err = np.abs(got[0, 0, h] - r[0]).max()
        assert 0 < err <= bound * (1 + 1e-6)


def test_per_sequence_lengths():
    # Sequence b attends to its first L_b cached keys.  With the cache entries past L_b set to
    # zero, the cache's blocks that hold keys below L_b have the codes and scales of each
    # sequence's own shorter cache, so the result must equal decoding each slice on its own;
    # all-full lengths equal the plain call, and a length of 0 gives zeros.
    cfg = small_workload("decvl", B=4, Hq=4, Hk=2, d=64, L=300, group_size=2, k_outliers=True,
                         index=902)
    Q, K, V = make_qkv(cfg)
    Q1 = Q[:, -1:]
    lens = [300, 1, 0, 130]
    for b, n in enumerate(lens):
        K[b, n:] = 0.0
        V[b, n:] = 0.0
    rng = np.random.default_rng(9)
    T_mask = -(-(-(-300 // 64)) // 2)
    words = _words(2, T_mask, rng, 0.5)
    cache = kv_cache(K, V)
    got = routed_decode(Q1, K, *cache, words, 2, cfg.scale, seqlens=lens)
    for b, n in enumerate(lens):
        if n == 0:
            assert np.all(got[b] == 0.0)
            continue
        Kb, Vb = K[b:b + 1, :n], V[b:b + 1, :n]
        ref = routed_decode(Q1[b:b + 1], Kb, *kv_cache(Kb, Vb), words, 2, cfg.scale)
        np.testing.assert_allclose(got[b], ref[0], rtol=0, atol=1e-12)
    full = routed_decode(Q1, K, *cache, words, 2, cfg.scale, seqlens=[300] * 4)
    np.testing.assert_array_equal(full, routed_decode(Q1, K, *cache, words, 2, cfg.scale))
