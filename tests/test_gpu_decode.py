"""GPU parity of the INT8 key/value cache decode path against the decode oracle."""

import numpy as np
import pytest

from gpu_util import MAX_ABS, REL_L2, log, to_dev
from oracle.decode import kv_cache, routed_decode
from synth import make_qkv, pack_route_bits, small_workload

pytestmark = pytest.mark.gpu


def test_quantize_kv_bitexact():
    import paper_2608_17336_amd as tm
    cfg = small_workload("kvq", B=2, Hq=2, Hk=2, d=128, L=333, k_outliers=True, index=910)
    _, K, V = make_qkv(cfg)
    V[1, 64:128, 0, :] = 0.0   # a zero block
    k8, dk, v8, dv = [t.cpu().numpy() for t in tm.tilemix_quantize_kv(to_dev(K), to_dev(V))]
    ok8, odk, ov8, odv = kv_cache(K, V)
    np.testing.assert_array_equal(k8, ok8)
    # V8 is stored per 64-key block channel-major: [B, H_k, blocks, d, 64], padding keys 0
    B, L, Hk, d = V.shape
    nb = -(-L // 64)
    pad = np.zeros((B, nb * 64, Hk, d), np.int8)
    pad[:, :L] = ov8
    want = pad.reshape(B, nb, 64, Hk, d).transpose(0, 3, 1, 4, 2)
    np.testing.assert_array_equal(v8, want)
    np.testing.assert_array_equal(dk.view(np.uint16), odk.view(np.uint16))
    np.testing.assert_array_equal(dv.view(np.uint16), odv.view(np.uint16))


CASES = [
    # B, Hq, Hk, d, L_k, g, route_per_batch
    (2, 8, 2, 128, 5000, 4, False),
    (1, 4, 4, 128, 1, 1, False),
    (2, 4, 2, 128, 63, 1, True),
    (1, 16, 1, 128, 700, 2, False),
    (3, 6, 2, 64, 300, 1, False),
    (1, 2, 1, 64, 257, 3, True),
    # MHA (one head per group, 15 padding columns), 20032 key tiles: each wave streams 10 tiles
    (8, 8, 8, 64, 20000, 2, False),
]


@pytest.mark.parametrize("B,Hq,Hk,d,Lk,g,rpb", CASES, ids=[str(c) for c in CASES])
def test_decode_parity(B, Hq, Hk, d, Lk, g, rpb):
    import torch
    import paper_2608_17336_amd as tm
    cfg = small_workload("dec", B=B, Hq=Hq, Hk=Hk, d=d, L=Lk, group_size=g, k_outliers=True,
                         index=920 + Lk)
    Q, K, V = make_qkv(cfg)
    Q1 = np.ascontiguousarray(Q[:, -1:])
    k, v = to_dev(K), to_dev(V)
    K8, dK, V8, dV = tm.tilemix_quantize_kv(k, v)
    ck = kv_cache(K, V)   # the oracle's own cache (bit-identical: test_quantize_kv_bitexact)
    T_mask = -(-(-(-Lk // 64)) // g)
    rng = np.random.default_rng(Lk)
    for p in (0.5, 0.0, 1.0):
        R = (rng.random((B if rpb else 1, Hk, 1, T_mask)) < p).astype(np.uint8)
        words = np.concatenate([pack_route_bits(R[i]) for i in range(R.shape[0])], axis=0)
        log(f"decode B={B} Hq={Hq} Hk={Hk} d={d} Lk={Lk} g={g} rpb={rpb} p={p}")
        O = tm.tilemix_decode(to_dev(Q1), k, K8, dK, V8, dV, to_dev(words), g, cfg.scale,
                              route_per_batch=rpb, route_hint=0 if p == 0.0 else -1)
        torch.cuda.synchronize()
        got = O.float().cpu().numpy().astype(np.float64)
        ref = routed_decode(Q1, K, *ck, words, g, cfg.scale)
        diff = got - ref
        mx = float(np.abs(diff).max())
        rel = float(np.sqrt((diff ** 2).sum() / (ref ** 2).sum()))
        log(f"  max_abs={mx:.3e} rel_l2={rel:.3e}")
        assert mx <= MAX_ABS and rel <= REL_L2, (p, mx, rel)


def _check(got, ref, what):
    diff = got - ref
    mx = float(np.abs(diff).max())
    rel = float(np.sqrt((diff ** 2).sum() / (ref ** 2).sum()))
    log(f"  {what}: max_abs={mx:.3e} rel_l2={rel:.3e}")
    assert mx <= MAX_ABS and rel <= REL_L2, (what, mx, rel)


@pytest.mark.timeout(600)
def test_decode_full_workload_sampled():
    """The 64K-key, B = 4, 64/8-head decode step bench.py times, with its three routing maps:
    every query head of sampled (sequence, KV head) groups against the oracle."""
    import torch
    import paper_2608_17336_amd as tm
    from synth import WORKLOADS, decode_route_bits
    cfg = WORKLOADS["64k-b4-gqa"]
    log(f"decode {cfg.name}: generating inputs")
    Q, K, V = make_qkv(cfg)
    Q1 = np.ascontiguousarray(Q[:, -1:])
    del Q
    k, v = to_dev(K), to_dev(V)
    K8, dK, V8, dV = tm.tilemix_quantize_kv(k, v)
    G = cfg.Hq // cfg.Hk
    picks = [(0, 0), (cfg.B - 1, cfg.Hk - 1), (cfg.B // 2, 3)]
    # the oracle's cache of each picked (sequence, KV head) slice (quantization is per slice)
    caches = {(b, hk): kv_cache(K[b:b + 1, :, hk:hk + 1], V[b:b + 1, :, hk:hk + 1]) for b, hk in picks}
    q1 = to_dev(Q1)
    for mask in cfg.masks:
        words, _ = decode_route_bits(cfg, mask)
        hint = 0 if mask.kind == "all_fp16" else -1
        log(f"  mask={mask.label}: GPU")
        O = tm.tilemix_decode(q1, k, K8, dK, V8, dV, to_dev(words), cfg.group_size, cfg.scale,
                              route_hint=hint)
        torch.cuda.synchronize()
        got = O.float().cpu().numpy().astype(np.float64)
        for b, hk in picks:
            ref = routed_decode(Q1[b:b + 1, :, hk * G:(hk + 1) * G], K[b:b + 1, :, hk:hk + 1],
                                *caches[(b, hk)], words[:, hk:hk + 1], cfg.group_size, cfg.scale)
            _check(got[b:b + 1, :, hk * G:(hk + 1) * G], ref, f"{mask.label} b={b} hk={hk}")


@pytest.mark.timeout(300)
def test_decode_longest_cache_full_group():
    """L_k = 262144 (the longest cache the build supports: each wave streams two tiles, 256
    chunks to merge) with a 16-head GQA group (every matrix-core column used), g = 16 (four
    routing words)."""
    import torch
    import paper_2608_17336_amd as tm
    Lk, g = 262144, 16
    cfg = small_workload("declong", B=1, Hq=16, Hk=1, d=128, L=Lk, group_size=g, k_outliers=True,
                         index=977)
    log(f"decode L_k={Lk} G=16 g={g}: generating inputs")
    Q, K, V = make_qkv(cfg)
    Q1 = np.ascontiguousarray(Q[:, -1:])
    del Q
    k, v = to_dev(K), to_dev(V)
    K8, dK, V8, dV = tm.tilemix_quantize_kv(k, v)
    ck = kv_cache(K, V)
    T_mask = -(-(-(-Lk // 64)) // g)
    R = (np.random.default_rng(977).random((1, 1, T_mask)) < 0.5).astype(np.uint8)
    words = pack_route_bits(R)
    assert words.shape[-1] == 4
    O = tm.tilemix_decode(to_dev(Q1), k, K8, dK, V8, dV, to_dev(words), g, cfg.scale)
    torch.cuda.synchronize()
    got = O.float().cpu().numpy().astype(np.float64)
    _check(got, routed_decode(Q1, K, *ck, words, g, cfg.scale), "L_k=262144")


RAGGED = [
    # B, Hq, Hk, d, capacity, g, lengths
    (4, 8, 2, 128, 700, 2, [700, 1, 0, 333]),
    (3, 16, 1, 128, 5000, 4, [4999, 512, 513]),
    (2, 4, 4, 64, 300, 1, [64, 299]),
    # 10016 key tiles in the batch: each wave streams 5 tiles, a chunk holds 40
    (4, 32, 8, 128, 20000, 4, [20000, 1, 0, 7777]),
]


@pytest.mark.parametrize("B,Hq,Hk,d,cap,g,lens", RAGGED, ids=[str(c[-1]) for c in RAGGED])
def test_decode_ragged_lengths(B, Hq, Hk, d, cap, g, lens):
    """tilemix_decode_varlen: each sequence attends to the first L_b keys of a padded cache
    (the entries past L_b hold unrelated keys and values and must not count)."""
    import torch
    import paper_2608_17336_amd as tm
    cfg = small_workload("decrag", B=B, Hq=Hq, Hk=Hk, d=d, L=cap, group_size=g, k_outliers=True,
                         index=940 + cap)
    Q, K, V = make_qkv(cfg)
    Q1 = np.ascontiguousarray(Q[:, -1:])
    k, v = to_dev(K), to_dev(V)
    K8, dK, V8, dV = tm.tilemix_quantize_kv(k, v)
    ck = kv_cache(K, V)
    T_mask = -(-(-(-cap // 64)) // g)
    rng = np.random.default_rng(cap)
    sl = torch.tensor(lens, dtype=torch.int32, device="cuda:0")
    for p in (0.5, 0.0, 1.0):
        words = pack_route_bits((rng.random((Hk, 1, T_mask)) < p).astype(np.uint8))
        log(f"ragged decode lens={lens} d={d} g={g} p={p}")
        O = tm.tilemix_decode(to_dev(Q1), k, K8, dK, V8, dV, to_dev(words), g, cfg.scale,
                              seqlens_k=sl, route_hint=0 if p == 0.0 else -1)
        torch.cuda.synchronize()
        got = O.float().cpu().numpy().astype(np.float64)
        ref = routed_decode(Q1, K, *ck, words, g, cfg.scale, seqlens=lens)
        for b, n in enumerate(lens):
            if n == 0:
                assert np.all(got[b] == 0.0), b
        nz = [b for b, n in enumerate(lens) if n > 0]
        _check(got[nz], ref[nz], f"lens={lens} p={p}")
