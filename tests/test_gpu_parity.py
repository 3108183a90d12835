"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bars: quantization codes/scales and INT32 tile products bit-exact; O within max-abs 2e-3
and rel-L2 1e-3 (fp16 output vs float64 oracle); invariants bitwise.
"""

import math

import numpy as np
import pytest

from gpu_util import MAX_ABS, REL_L2, compare_rows, log, prefill, to_dev
from oracle import (OracleOperands, quantize_blocks, routed_attention_rows, int8_tile_product,
                    QUANT_BLOCK_Q, QUANT_BLOCK_K)
from synth import (MaskSpec, WORKLOADS, make_qkv, make_route_bits, pack_route_bits, sample_rows,
                   small_workload)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2608_17336_amd as tm
    tm.load_library()


def _oracle(cfg, Q, K, V, words, rows, operands=None):
    return routed_attention_rows(Q, K, V, words, block_m=cfg.block_m, block_n=cfg.block_n,
                                 group_size=cfg.group_size, causal=cfg.causal, scale=cfg.scale,
                                 rows=rows, operands=operands)


# ------------------------------------------------------------------------- quantization

QUANT_SHAPES = [(1, 300, 4, 2, 128), (2, 64, 2, 2, 64), (1, 129, 3, 1, 64), (1, 1, 2, 1, 128),
                (1, 8192, 32, 8, 128)]


@pytest.mark.parametrize("shape", QUANT_SHAPES)
def test_quantize_bitexact(shape):
    import paper_2608_17336_amd as tm
    B, L, Hq, Hk, d = shape
    log(f"quantize shape={shape}")
    cfg = small_workload("q", B=B, Hq=Hq, Hk=Hk, d=d, L=L, k_outliers=True, index=200 + L)
    Q, K, _ = make_qkv(cfg)
    Q[0, 0, 0, :] = 0.0                         # a zero row inside a non-zero block
    if L >= 128:
        K[0, 64:128, 0, :] = 0.0                # an all-zero key block -> scale 0, codes 0
    q8, dq, k8, dk = [t.cpu().numpy() for t in tm.tilemix_quantize(to_dev(Q), to_dev(K))]
    oq8, odq = quantize_blocks(Q, QUANT_BLOCK_Q)
    ok8, odk = quantize_blocks(K, QUANT_BLOCK_K)
    np.testing.assert_array_equal(q8, oq8)
    np.testing.assert_array_equal(k8, ok8)
    np.testing.assert_array_equal(dq.view(np.uint16), odq.view(np.uint16))
    np.testing.assert_array_equal(dk.view(np.uint16), odk.view(np.uint16))


# ------------------------------------------------------------------- INT32 tile products

@pytest.mark.parametrize("d,bm,L", [(128, 128, 300), (64, 64, 1024), (128, 64, 200), (64, 128, 257)])
def test_int32_tiles_bitexact(d, bm, L):
    import torch
    import paper_2608_17336_amd as tm
    log(f"int32 tiles d={d} bm={bm} L={L}")
    cfg = small_workload("t", B=2, Hq=4, Hk=2, d=d, L=L, block_m=bm, k_outliers=True, index=300 + d)
    Q, K, _ = make_qkv(cfg)
    q8, _, k8, _ = tm.tilemix_quantize(to_dev(Q), to_dev(K), tile=(bm, 64))
    ops = OracleOperands.from_inputs(Q, K)
    rng = np.random.default_rng(1)
    T_m, T_n = cfg.T_m, cfg.T_n
    tiles = [(b, h, T_m - 1, T_n - 1) for b in range(2) for h in range(4)]          # ragged corner
    tiles += [(1, 3, m, min(T_n - 1, (m * bm) // 64)) for m in range(T_m)]         # diagonal
    tiles += [(int(rng.integers(2)), int(rng.integers(4)), int(rng.integers(T_m)), int(rng.integers(T_n)))
              for _ in range(40)]
    t = torch.tensor(tiles, dtype=torch.int32, device="cuda:0")
    out = tm.tilemix_debug_qk_int32(q8, k8, t, heads_q=4, heads_kv=2, tile=(bm, 64)).cpu().numpy()
    for e, (b, h, m, n) in enumerate(tiles):
        want = int8_tile_product(ops, b, h, h // 2, m, n, bm, 64)
        np.testing.assert_array_equal(out[e].astype(np.int64), want, err_msg=str((b, h, m, n)))


# --------------------------------------------------------------------- small full parity

SMALL = [
    # name, kwargs
    ("ragged-d128-bm128-g1", dict(B=1, Hq=4, Hk=2, d=128, L=333, block_m=128, group_size=1)),
    ("ragged-d128-bm128-g3", dict(B=2, Hq=2, Hk=1, d=128, L=517, block_m=128, group_size=3,
                                  k_outliers=True)),
    ("d64-bm64-g1", dict(B=1, Hq=2, Hk=2, d=64, L=1024, block_m=64, group_size=1)),
    ("d64-bm64-ragged", dict(B=2, Hq=4, Hk=1, d=64, L=190, block_m=64, group_size=2)),
    ("d128-bm64", dict(B=1, Hq=2, Hk=1, d=128, L=400, block_m=64, group_size=1)),
    ("d64-bm128", dict(B=1, Hq=2, Hk=2, d=64, L=300, block_m=128, group_size=1)),
    ("tiny-L1", dict(B=1, Hq=1, Hk=1, d=128, L=1, block_m=128, group_size=1)),
    ("tiny-L33", dict(B=1, Hq=2, Hk=1, d=64, L=33, block_m=64, group_size=1)),
    ("noncausal", dict(B=1, Hq=2, Hk=1, d=128, L=300, block_m=128, group_size=1, causal=False)),
    ("gqa3", dict(B=1, Hq=6, Hk=2, d=128, L=260, block_m=128, group_size=2)),
    ("multiword-g1", dict(B=1, Hq=2, Hk=1, d=128, L=4500, block_m=128, group_size=1)),
]
MASKS = [MaskSpec("bernoulli", 0.5), MaskSpec("all_fp16"), MaskSpec("all_int8")]


@pytest.mark.parametrize("name,kw", SMALL, ids=[s[0] for s in SMALL])
def test_small_parity(name, kw):
    for mi, mask in enumerate(MASKS):
        cfg = small_workload(name, mask=mask, index=400 + len(name), **kw)
        log(f"small {name} mask={mask.label}")
        Q, K, V = make_qkv(cfg)
        words, _ = make_route_bits(cfg, mask, mi)
        O = prefill(cfg, Q, K, V, words)
        rows = [(b, h, np.arange(cfg.L)) for b in range(cfg.B) for h in range(cfg.Hq)]
        ref = _oracle(cfg, Q, K, V, words, rows)
        mx, rel = compare_rows(O, rows, ref)
        log(f"  max_abs={mx:.3e} rel_l2={rel:.3e}")
        assert mx <= MAX_ABS and rel <= REL_L2, (name, mask.label, mx, rel)


def test_unequal_lengths_bottom_right_causal():
    import paper_2608_17336_amd as tm
    import torch
    rng = np.random.default_rng(3)
    for Lq, Lk in [(100, 300), (300, 100)]:
        log(f"Lq={Lq} Lk={Lk}")
        Q = rng.standard_normal((1, Lq, 2, 128)).astype(np.float16)
        K = rng.standard_normal((1, Lk, 1, 128)).astype(np.float16)
        V = rng.standard_normal((1, Lk, 1, 128)).astype(np.float16)
        T_m, T_n = -(-Lq // 128), -(-Lk // 64)
        R = (rng.random((1, T_m, T_n)) < 0.5).astype(np.uint8)
        words = pack_route_bits(R)
        O = tm.tilemix_prefill(to_dev(Q), to_dev(K), to_dev(V), to_dev(words), 1, (128, 64), True,
                               1 / math.sqrt(128))
        torch.cuda.synchronize()
        rows = [(0, h, np.arange(Lq)) for h in range(2)]
        ref = routed_attention_rows(Q, K, V, words, block_m=128, block_n=64, group_size=1,
                                    causal=True, scale=1 / math.sqrt(128), rows=rows)
        mx, rel = compare_rows(O, rows, ref)
        log(f"  max_abs={mx:.3e} rel_l2={rel:.3e}")
        assert mx <= MAX_ABS and rel <= REL_L2


@pytest.mark.timeout(600)
def test_longest_key_sequence_64_routing_words():
    """L_k = 262144, the longest key sequence the build takes: with g = 1 a routing row is 64
    words, the most the kernel holds (one per lane).  A ragged L_q = 200 query block at the end
    of the sequence (bottom-right causal) and the non-causal case, against the oracle on
    sampled rows."""
    import paper_2608_17336_amd as tm
    import torch
    rng = np.random.default_rng(262144)
    Lq, Lk, d = 200, 262144, 128
    Q = rng.standard_normal((1, Lq, 2, d)).astype(np.float16)
    K = rng.standard_normal((1, Lk, 1, d)).astype(np.float16)
    V = rng.standard_normal((1, Lk, 1, d)).astype(np.float16)
    T_m, T_n = -(-Lq // 128), -(-Lk // 64)
    R = (rng.random((1, T_m, T_n)) < 0.5).astype(np.uint8)
    words = pack_route_bits(R)
    assert words.shape[-1] == 64
    q, k, v, w = to_dev(Q), to_dev(K), to_dev(V), to_dev(words)
    idx = np.unique(np.concatenate([np.arange(8), np.arange(Lq - 8, Lq), [127, 128],
                                    rng.choice(Lq, 16, replace=False)]))
    rows = [(0, h, idx) for h in range(2)]
    ops = OracleOperands.from_inputs(Q, K, q_heads=[(0, 0), (0, 1)], k_heads=[(0, 0)])
    for causal in (True, False):
        log(f"Lq={Lq} Lk={Lk} causal={causal}")
        O = tm.tilemix_prefill(q, k, v, w, 1, (128, 64), causal, 1 / math.sqrt(d))
        torch.cuda.synchronize()
        ref = routed_attention_rows(Q, K, V, words, block_m=128, block_n=64, group_size=1,
                                    causal=causal, scale=1 / math.sqrt(d), rows=rows, operands=ops)
        mx, rel = compare_rows(O, rows, ref)
        log(f"  max_abs={mx:.3e} rel_l2={rel:.3e}")
        assert mx <= MAX_ABS and rel <= REL_L2, (causal, mx, rel)


# --------------------------------------------------------------------- full-size workloads

WL = [(name, mi) for name, cfg in WORKLOADS.items() for mi in range(len(cfg.masks))]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", list(WORKLOADS))
def test_workload_parity_sampled(name):
    cfg = WORKLOADS[name]
    log(f"workload {name}: generating inputs")
    Q, K, V = make_qkv(cfg)
    import torch
    dev = (to_dev(Q), to_dev(K), to_dev(V))
    rows = sample_rows(cfg) if name != "1k-mha-d64" else \
        [(0, h, np.arange(cfg.L)) for h in range(cfg.Hq)]
    ops = OracleOperands.from_inputs(Q, K, q_heads=sorted({(b, h) for b, h, _ in rows}),
                                     k_heads=sorted({(b, h // (cfg.Hq // cfg.Hk)) for b, h, _ in rows}))
    for mi, mask in enumerate(cfg.masks):
        words, _ = make_route_bits(cfg, mask, mi)
        hint = 0 if mask.kind == "all_fp16" else -1
        log(f"  mask={mask.label} hint={hint}: GPU")
        O = prefill(cfg, Q, K, V, words, route_hint=hint, dev_inputs=dev)
        log(f"  mask={mask.label}: oracle on {sum(len(r[2]) for r in rows)} rows")
        ref = _oracle(cfg, Q, K, V, words, rows, operands=ops)
        mx, rel = compare_rows(O, rows, ref)
        log(f"  max_abs={mx:.3e} rel_l2={rel:.3e}")
        assert mx <= MAX_ABS and rel <= REL_L2, (name, mask.label, mx, rel)
        del O
        torch.cuda.empty_cache()


def test_deviation_from_fp16_matches_oracle():
    """The routed output's deviation from exact attention (every tile FP16), measured on the GPU,
    agrees with the oracle's on sampled rows (the figure bench.py reports)."""
    cfg = WORKLOADS["8k-gqa"]
    Q, K, V = make_qkv(cfg)
    dev = (to_dev(Q), to_dev(K), to_dev(V))
    words, _ = make_route_bits(cfg, cfg.masks[0], 0)
    zeros = np.zeros_like(words)
    O_r = prefill(cfg, Q, K, V, words, dev_inputs=dev).float().cpu().numpy()
    O_f = prefill(cfg, Q, K, V, zeros, route_hint=0, dev_inputs=dev).float().cpu().numpy()
    rows = sample_rows(cfg)[:2]
    ops = OracleOperands.from_inputs(Q, K, q_heads=sorted({(b, h) for b, h, _ in rows}),
                                     k_heads=sorted({(b, h // (cfg.Hq // cfg.Hk)) for b, h, _ in rows}))
    ref_r = _oracle(cfg, Q, K, V, words, rows, operands=ops)
    ref_f = _oracle(cfg, Q, K, V, zeros, rows, operands=ops)
    for (b, h, idx), rr, rf in zip(rows, ref_r, ref_f):
        gpu_dev = O_r[b, idx, h].astype(np.float64) - O_f[b, idx, h].astype(np.float64)
        ora_dev = rr - rf
        log(f"deviation b={b} h={h}: gpu mean_abs {np.abs(gpu_dev).mean():.3e} "
            f"oracle mean_abs {np.abs(ora_dev).mean():.3e}")
        assert 1e-6 < np.abs(ora_dev).mean() < 1e-2
        assert np.abs(gpu_dev - ora_dev).max() <= 2 * MAX_ABS


# ------------------------------------------------------------------------ invariants

def _inv_cfg(**kw):
    base = dict(B=1, Hq=4, Hk=2, d=128, L=400, block_m=128, group_size=1, k_outliers=True)
    base.update(kw)
    return small_workload("inv", index=500, **base)


def _integer_inputs(L=512):
    rng = np.random.default_rng(9)
    Q = rng.integers(-127, 128, size=(1, L, 4, 128)).astype(np.float16)
    K = rng.integers(-127, 128, size=(1, L, 2, 128)).astype(np.float16)
    Q[:, ::128, :, 0] = 127.0     # every 128-row query block and 64-row key block has
    K[:, ::64, :, 0] = -127.0     # absmax 127, so its scale is 1 and its codes are the inputs
    V = rng.standard_normal((1, L, 2, 128)).astype(np.float16)
    return Q, K, V


def _both_routes(cfg, Q, K, V, scale):
    import paper_2608_17336_amd as tm
    import torch
    w16, _ = make_route_bits(cfg, MaskSpec("all_fp16"))
    w8, _ = make_route_bits(cfg, MaskSpec("all_int8"))
    outs = []
    for w in (w16, w8):
        O = tm.tilemix_prefill(to_dev(Q), to_dev(K), to_dev(V), to_dev(w), 1, (128, 64), True, scale)
        torch.cuda.synchronize()
        outs.append(O)
    return outs, w16


def test_integer_inputs_int8_equals_fp16_bitwise():
    # With scale 1 blocks the INT8 route computes exactly the FP16 route's products.  At this
    # softmax scale (1.5 * 2^23 * scale * log2(e) >= 2^14) the kernel converts the INT32
    # products exactly instead of folding the accumulator bias, so the two routes must agree
    # bit for bit (integer scores reach thousands of log2 units: this also drives the running-
    # max refresh many times per row).
    L = 512
    Q, K, V = _integer_inputs(L)
    cfg = _inv_cfg(L=L)
    scale = 1.0 / 512.0
    outs, _ = _both_routes(cfg, Q, K, V, scale)
    a, b = (o.cpu().numpy() for o in outs)
    np.testing.assert_array_equal(a.view(np.uint16), b.view(np.uint16))


def test_integer_inputs_folded_bias_within_bound():
    # At a smaller scale the INT8 tiles fold the accumulator bias into the exp subtrahend, which
    # rounds the exp argument by at most 2^-11 (log2 units): the routes then agree within the
    # parity bar, and both match the oracle (where the routes coincide exactly).
    L = 512
    Q, K, V = _integer_inputs(L)
    cfg = _inv_cfg(L=L)
    scale = 1.0 / 4000.0
    outs, w16 = _both_routes(cfg, Q, K, V, scale)
    rows = [(0, h, np.arange(L)) for h in range(4)]
    ref = routed_attention_rows(Q, K, V, w16, block_m=128, block_n=64, group_size=1, causal=True,
                                scale=scale, rows=rows)
    for O in outs:
        mx, rel = compare_rows(O, rows, ref)
        log(f"  max_abs={mx:.3e} rel_l2={rel:.3e}")
        assert mx <= MAX_ABS and rel <= REL_L2, (mx, rel)
    a, b = (o.float().cpu().numpy() for o in outs)
    assert float(np.max(np.abs(a - b))) <= MAX_ABS


def test_running_max_refresh():
    # Keys whose norm grows along the sequence make every later tile's scores exceed the
    # running max taken from the first tile by far more than FP16 P can hold, so the kernel
    # must refresh the max (and rescale its accumulators) many times per row.
    cfg = _inv_cfg(L=1024, group_size=1)
    Q, K, V = make_qkv(cfg)
    grow = (1.0 + np.arange(cfg.L, dtype=np.float32) / 48.0)[None, :, None, None]
    K = (K.astype(np.float32) * grow).astype(np.float16)
    for mi, mask in enumerate(MASKS):
        words, _ = make_route_bits(cfg, mask, mi)
        O = prefill(cfg, Q, K, V, words)
        rows = [(0, h, np.arange(cfg.L)) for h in range(cfg.Hq)]
        ref = _oracle(cfg, Q, K, V, words, rows)
        mx, rel = compare_rows(O, rows, ref)
        log(f"  refresh mask={mask.label} max_abs={mx:.3e} rel_l2={rel:.3e}")
        assert mx <= MAX_ABS and rel <= REL_L2, (mask.label, mx, rel)


def test_first_row_equals_v0_and_route_hint():
    cfg = _inv_cfg()
    Q, K, V = make_qkv(cfg)
    for mi, mask in enumerate(MASKS):
        words, _ = make_route_bits(cfg, mask, mi)
        O = prefill(cfg, Q, K, V, words).cpu().numpy()
        for h in range(cfg.Hq):
            np.testing.assert_array_equal(O[0, 0, h], V[0, 0, h // 2])
    zero, _ = make_route_bits(cfg, MaskSpec("all_fp16"))
    a = prefill(cfg, Q, K, V, zero).cpu().numpy()
    b = prefill(cfg, Q, K, V, zero, route_hint=0).cpu().numpy()
    np.testing.assert_array_equal(a.view(np.uint16), b.view(np.uint16))


def test_causal_perturbation_bitwise():
    cfg = _inv_cfg(L=512)
    Q, K, V = make_qkv(cfg)
    words, _ = make_route_bits(cfg, MaskSpec("bernoulli", 0.5))
    base = prefill(cfg, Q, K, V, words).cpu().numpy()
    V2, K2 = V.copy(), K.copy()
    V2[0, 256:] = np.float16(5.0)
    K2[0, 256:] = np.float16(-3.0)     # key blocks 4.. lie wholly after row 255
    got = prefill(cfg, Q, K2, V2, words).cpu().numpy()
    np.testing.assert_array_equal(base[0, :256].view(np.uint16), got[0, :256].view(np.uint16))
    assert not np.array_equal(base[0, 256:], got[0, 256:])


def test_gqa_identical_heads_bitwise():
    cfg = _inv_cfg()
    Q, K, V = make_qkv(cfg)
    Q[:, :, 1] = Q[:, :, 0]
    words, _ = make_route_bits(cfg, MaskSpec("bernoulli", 0.5))
    O = prefill(cfg, Q, K, V, words).cpu().numpy()
    np.testing.assert_array_equal(O[0, :, 0].view(np.uint16), O[0, :, 1].view(np.uint16))


def test_illegal_and_padding_bits_ignored_bitwise():
    cfg = _inv_cfg(L=700, group_size=3)
    Q, K, V = make_qkv(cfg)
    words, R = make_route_bits(cfg, MaskSpec("bernoulli", 0.5))
    from synth import legal_group_table
    legal = legal_group_table(cfg)
    R2 = R.copy()
    R2[:, ~legal] = 1                                     # set every illegal group's bit
    w2 = pack_route_bits(R2)
    w2[..., -1] |= np.uint64(1) << np.uint64(63)         # and a bit past T_mask
    a = prefill(cfg, Q, K, V, words).cpu().numpy()
    b = prefill(cfg, Q, K, V, w2).cpu().numpy()
    np.testing.assert_array_equal(a.view(np.uint16), b.view(np.uint16))


def test_per_sequence_route_maps():
    cfg = _inv_cfg(B=2, L=300)
    Q, K, V = make_qkv(cfg)
    rng = np.random.default_rng(4)
    R = (rng.random((2, cfg.Hk, cfg.T_m, cfg.T_mask)) < 0.5).astype(np.uint8)
    words = np.concatenate([pack_route_bits(R[b]) for b in range(2)], axis=0)
    O = prefill(cfg, Q, K, V, words, route_per_batch=True)
    rows = [(b, h, np.arange(cfg.L)) for b in range(2) for h in range(cfg.Hq)]
    ref = _oracle(cfg, Q, K, V, words, rows)
    mx, rel = compare_rows(O, rows, ref)
    assert mx <= MAX_ABS and rel <= REL_L2


@pytest.mark.parametrize("kind", ["band", "global", "rowrand", "aligned", "bigbird", "sptrans"])
def test_template_routes_parity(kind):
    # routing words from the library's Appendix B templates (fitted to 50% INT8 coverage)
    import paper_2608_17336_amd as tm
    cfg = small_workload("tmpl", B=1, Hq=4, Hk=2, d=128, L=1300, block_m=128, group_size=2,
                         k_outliers=True, index=700)
    p = tm.Params(cfg.B, cfg.Hq, cfg.Hk, cfg.L, cfg.L, cfg.d, cfg.block_m, cfg.block_n,
                  cfg.group_size, True, cfg.scale)
    t = tm.tilemix_fit_template(p, tm.Template(kind, sp_stride=256, seed=5), 0.5)
    words = tm.tilemix_route_template(p, t)
    log(f"template {t} coverage {tm.tilemix_route_coverage(p, words)}")
    Q, K, V = make_qkv(cfg)
    O = prefill(cfg, Q, K, V, words)
    rows = [(0, h, np.arange(cfg.L)) for h in range(cfg.Hq)]
    ref = _oracle(cfg, Q, K, V, words, rows)
    mx, rel = compare_rows(O, rows, ref)
    log(f"  max_abs={mx:.3e} rel_l2={rel:.3e}")
    assert mx <= MAX_ABS and rel <= REL_L2, (kind, mx, rel)
