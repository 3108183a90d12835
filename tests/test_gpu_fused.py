"""GPU checks of the fused on-the-fly operand mode (tilemix_prefill_fused): its on-chip codes
and scales equal those of the quantize-once pass, so its output equals tilemix_prefill's bit
for bit; and against the oracle at the parity bar."""

import numpy as np
import pytest

from gpu_util import MAX_ABS, REL_L2, compare_rows, log, prefill, to_dev
from oracle import routed_attention_rows
from synth import MaskSpec, WORKLOADS, make_qkv, make_route_bits, small_workload

pytestmark = pytest.mark.gpu


def fused(cfg, Q, K, V, words, *, route_hint=-1, dev_inputs=None):
    import paper_2608_17336_amd as tm
    import torch
    q, k, v = dev_inputs if dev_inputs is not None else (to_dev(Q), to_dev(K), to_dev(V))
    O = tm.tilemix_prefill_fused(q, k, v, to_dev(words), cfg.group_size, (cfg.block_m, cfg.block_n),
                                 cfg.causal, cfg.scale, route_hint=route_hint)
    torch.cuda.synchronize()
    return O


def same_bits(a, b):
    import torch
    return bool(torch.equal(a.view(torch.int16), b.view(torch.int16)))


CASES = [
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
    ("zero-blocks", dict(B=1, Hq=2, Hk=1, d=128, L=700, block_m=128, group_size=1)),
    ("zero-blocks-bm64", dict(B=1, Hq=2, Hk=2, d=128, L=700, block_m=64, group_size=1)),
]
MASKS = [MaskSpec("bernoulli", 0.5), MaskSpec("all_fp16"), MaskSpec("all_int8")]


def _inputs(name, cfg):
    Q, K, V = make_qkv(cfg)
    if name.startswith("zero-blocks"):
        Q[0, 128:256, 0, :] = 0.0      # a whole 128-row query block: scale 0, codes 0
        K[0, 64:128, 0, :] = 0.0       # a whole 64-key block
        Q[0, 300:301, 1, :] = 0.0      # one zero row inside a block
    return Q, K, V


@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_fused_equals_quantize_once_bitwise(name, kw):
    for mi, mask in enumerate(MASKS):
        cfg = small_workload(name, mask=mask, index=600 + len(name), **kw)
        log(f"fused {name} mask={mask.label}")
        Q, K, V = _inputs(name, cfg)
        words, _ = make_route_bits(cfg, mask, mi)
        dev = (to_dev(Q), to_dev(K), to_dev(V))
        hint = 0 if mask.kind == "all_fp16" else -1
        O1 = prefill(cfg, Q, K, V, words, dev_inputs=dev, route_hint=hint)
        O2 = fused(cfg, Q, K, V, words, dev_inputs=dev, route_hint=hint)
        assert same_bits(O1, O2), (name, mask.label)
        # the all-FP16 map given without the hint takes the same path
        if mask.kind == "all_fp16":
            assert same_bits(O1, fused(cfg, Q, K, V, words, dev_inputs=dev)), name


@pytest.mark.parametrize("name", ["ragged-d128-bm128-g3", "d128-bm64", "zero-blocks"])
def test_fused_parity_vs_oracle(name):
    kw = dict(CASES)[name]
    mask = MaskSpec("bernoulli", 0.5)
    cfg = small_workload(name, mask=mask, index=650 + len(name), **kw)
    Q, K, V = _inputs(name, cfg)
    words, _ = make_route_bits(cfg, mask, 0)
    O = fused(cfg, Q, K, V, words)
    rows = [(b, h, np.arange(cfg.L)) for b in range(cfg.B) for h in range(cfg.Hq)]
    ref = routed_attention_rows(Q, K, V, words, block_m=cfg.block_m, block_n=cfg.block_n,
                                group_size=cfg.group_size, causal=cfg.causal, scale=cfg.scale,
                                rows=rows)
    mx, rel = compare_rows(O, rows, ref)
    log(f"fused {name}: max_abs={mx:.3e} rel_l2={rel:.3e}")
    assert mx <= MAX_ABS and rel <= REL_L2, (name, mx, rel)


def test_fused_unequal_lengths_bitwise():
    import paper_2608_17336_amd as tm
    import torch
    cfg = small_workload("uneq", B=2, Hq=4, Hk=2, d=128, L=900, block_m=128, group_size=2, index=661)
    Q, K, V = make_qkv(cfg)
    Lq = 333
    q = to_dev(np.ascontiguousarray(Q[:, -Lq:]))
    k, v = to_dev(K), to_dev(V)
    p = tm.Params(cfg.B, cfg.Hq, cfg.Hk, Lq, cfg.L, cfg.d, cfg.block_m, cfg.block_n, cfg.group_size)
    W = tm.tilemix_route_words_per_row(p)
    words = np.random.default_rng(661).integers(0, 2 ** 63, size=(1, cfg.Hk, p.T_m, W), dtype=np.int64)
    w = to_dev(words)
    for causal in (True, False):
        O1 = tm.tilemix_prefill(q, k, v, w, cfg.group_size, (cfg.block_m, 64), causal, cfg.scale)
        O2 = tm.tilemix_prefill_fused(q, k, v, w, cfg.group_size, (cfg.block_m, 64), causal, cfg.scale)
        torch.cuda.synchronize()
        assert same_bits(O1, O2), causal


def test_fused_per_sequence_routes_bitwise():
    """route_per_batch: each sequence reads its own routing map (B_r = B)."""
    import paper_2608_17336_amd as tm
    import torch
    cfg = small_workload("rpb", B=3, Hq=4, Hk=2, d=128, L=700, block_m=128, group_size=2, index=671)
    Q, K, V = make_qkv(cfg)
    q, k, v = to_dev(Q), to_dev(K), to_dev(V)
    p = tm.Params(cfg.B, cfg.Hq, cfg.Hk, cfg.L, cfg.L, cfg.d, cfg.block_m, cfg.block_n, cfg.group_size)
    W = tm.tilemix_route_words_per_row(p)
    words = np.random.default_rng(671).integers(0, 2 ** 63, size=(cfg.B, cfg.Hk, p.T_m, W), dtype=np.int64)
    w = to_dev(words)
    O1 = tm.tilemix_prefill(q, k, v, w, cfg.group_size, (128, 64), True, cfg.scale, route_per_batch=True)
    O2 = tm.tilemix_prefill_fused(q, k, v, w, cfg.group_size, (128, 64), True, cfg.scale,
                                  route_per_batch=True)
    torch.cuda.synchronize()
    assert same_bits(O1, O2)


def test_fused_longest_key_sequence_bitwise():
    """L_k = 262144 with g = 1 (64 routing words per row), L_q = 200: fused equals quantize-once."""
    import paper_2608_17336_amd as tm
    import torch
    rng = np.random.default_rng(262145)
    Lq, Lk, d = 200, 262144, 128
    q = to_dev(rng.standard_normal((1, Lq, 2, d)).astype(np.float16))
    k = to_dev(rng.standard_normal((1, Lk, 1, d)).astype(np.float16))
    v = to_dev(rng.standard_normal((1, Lk, 1, d)).astype(np.float16))
    words = rng.integers(0, 2 ** 63, size=(1, 1, 2, 64), dtype=np.int64)
    w = to_dev(words)
    for causal in (True, False):
        O1 = tm.tilemix_prefill(q, k, v, w, 1, (128, 64), causal, 1 / np.sqrt(d))
        O2 = tm.tilemix_prefill_fused(q, k, v, w, 1, (128, 64), causal, 1 / np.sqrt(d))
        torch.cuda.synchronize()
        assert same_bits(O1, O2), causal


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", ["8k-gqa", "32k-gqa"])
def test_fused_full_workload_bitwise(name):
    """The benchmark workloads in the launch configuration bench.py times: every output element
    of the fused mode equals the quantize-once path's."""
    import torch
    cfg = WORKLOADS[name]
    log(f"fused {name}: generating inputs")
    Q, K, V = make_qkv(cfg)
    dev = (to_dev(Q), to_dev(K), to_dev(V))
    words, _ = make_route_bits(cfg, cfg.masks[0], 0)
    O1 = prefill(cfg, Q, K, V, words, dev_inputs=dev)
    O2 = fused(cfg, Q, K, V, words, dev_inputs=dev)
    ok = same_bits(O1, O2)
    if not ok:
        d = (O1.float() - O2.float()).abs()
        log(f"  differing elements: {int((d > 0).sum())}, max diff {d.max().item():.3e}")
    assert ok
    del O1, O2
    torch.cuda.empty_cache()
