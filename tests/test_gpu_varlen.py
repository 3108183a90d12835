"""GPU parity of the variable-length batch entry point (tilemix_prefill_varlen) against the
oracle applied to each sequence on its own (Section 4.1 varlen batching, Appendix C varlen
scale layout)."""

import numpy as np
import pytest

from gpu_util import MAX_ABS, REL_L2, log, to_dev
from oracle import routed_attention_rows
from synth import make_qkv, pack_route_bits, small_workload

pytestmark = pytest.mark.gpu


def _legal_groups(lq, lk, bm, span, causal=True):
    """bool [T_m, T_mask] legal groups of one sequence (prefix of each row)."""
    T_m, T_mask = -(-lq // bm), -(-(-(-lk // 64)) // (span // 64))
    out = np.zeros((T_m, T_mask), bool)
    for m in range(T_m):
        last = min(lk - 1, min(lq, (m + 1) * bm) - 1 + lk - lq) if causal else lk - 1
        if last >= 0:
            out[m, :last // span + 1] = True
    return out


def _pack(lens_q, lens_k, Hk, bm, g, W, rng, p_int8):
    """Random Bernoulli routing rows for each sequence: [sum T_m, H_k, W] and per-sequence maps."""
    rows, per_seq = [], []
    for lq, lk in zip(lens_q, lens_k):
        legal = _legal_groups(lq, lk, bm, 64 * g)
        R = (rng.random((Hk,) + legal.shape) < p_int8) & legal[None]
        w = pack_route_bits(R.astype(np.uint8))[0]                    # [H_k, T_m, W_b]
        full = np.zeros((Hk, legal.shape[0], W), np.uint64)
        full[..., :w.shape[-1]] = w
        per_seq.append(full[None])                                    # [1, H_k, T_m, W]
        rows.append(full.transpose(1, 0, 2))
    return np.concatenate(rows, axis=0) if rows else np.zeros((0, Hk, W), np.uint64), per_seq


CASES = [
    # name, lens_q, lens_k, d, block_m, g
    ("mixed-d128", [333, 1, 1024, 517, 64], None, 128, 128, 1),
    ("empty-and-tiny", [70, 0, 5, 257], None, 128, 128, 2),
    ("d64-bm64", [190, 1100, 33], None, 64, 64, 1),
    ("q-shorter-than-k", [100, 300, 17], [200, 300, 64], 128, 128, 1),
]


@pytest.mark.parametrize("name,lens_q,lens_k,d,bm,g", CASES, ids=[c[0] for c in CASES])
def test_varlen_parity(name, lens_q, lens_k, d, bm, g):
    import torch
    import paper_2608_17336_amd as tm
    lens_k = lens_k or lens_q
    Hq, Hk = 4, 2
    B = len(lens_q)
    total_q, total_k = sum(lens_q), sum(lens_k)
    Lq, Lk = max(lens_q), max(lens_k)
    cfg = small_workload("vl", B=1, Hq=Hq, Hk=Hk, d=d, L=max(total_q, total_k), block_m=bm,
                         group_size=g, k_outliers=True, index=800 + len(name))
    Q, K, V = make_qkv(cfg)
    Q, K, V = Q[0, :total_q], K[0, :total_k], V[0, :total_k]
    p = tm.Params(B, Hq, Hk, Lq, Lk, d, bm, 64, g, True, cfg.scale)
    W = tm.tilemix_route_words_per_row(p)
    rng = np.random.default_rng(len(name))
    for p_int8 in (0.5, 0.0, 1.0):
        words, per_seq = _pack(lens_q, lens_k, Hk, bm, g, W, rng, p_int8)
        cu_q = torch.tensor(np.concatenate([[0], np.cumsum(lens_q)]), dtype=torch.int32, device="cuda:0")
        cu_k = torch.tensor(np.concatenate([[0], np.cumsum(lens_k)]), dtype=torch.int32, device="cuda:0")
        log(f"varlen {name} p_int8={p_int8} lens_q={lens_q} lens_k={lens_k}")
        O = tm.tilemix_prefill_varlen(to_dev(Q), to_dev(K), to_dev(V), cu_q, cu_k, Lq, Lk,
                                      to_dev(words), g, (bm, 64), True, cfg.scale,
                                      route_hint=0 if p_int8 == 0.0 else -1)
        torch.cuda.synchronize()
        got = O.float().cpu().numpy().astype(np.float64)
        num = den = mx = 0.0
        q0 = k0 = 0
        for b, (lq, lk) in enumerate(zip(lens_q, lens_k)):
            if lq:
                Qb, Kb, Vb = Q[None, q0:q0 + lq], K[None, k0:k0 + lk], V[None, k0:k0 + lk]
                rows = [(0, h, np.arange(lq)) for h in range(Hq)]
                ref = routed_attention_rows(Qb, Kb, Vb, per_seq[b], block_m=bm, block_n=64,
                                            group_size=g, causal=True, scale=cfg.scale, rows=rows)
                for (_, h, idx), r in zip(rows, ref):
                    diff = got[q0 + idx, h, :] - r
                    mx = max(mx, float(np.abs(diff).max()))
                    num += float((diff ** 2).sum())
                    den += float((r ** 2).sum())
            q0 += lq
            k0 += lk
        rel = (num / den) ** 0.5
        log(f"  max_abs={mx:.3e} rel_l2={rel:.3e}")
        assert mx <= MAX_ABS and rel <= REL_L2, (name, p_int8, mx, rel)


def test_varlen_equal_lengths_matches_fixed_bitwise():
    import torch
    import paper_2608_17336_amd as tm
    from gpu_util import prefill
    from synth import make_route_bits, MaskSpec
    cfg = small_workload("vleq", B=3, Hq=4, Hk=2, d=128, L=777, block_m=128, group_size=2,
                         k_outliers=True, index=850, mask=MaskSpec("bernoulli", 0.5))
    Q, K, V = make_qkv(cfg)
    words, _ = make_route_bits(cfg)                      # one map for all three sequences
    O_fixed = prefill(cfg, Q, K, V, words).cpu().numpy()
    rows = np.concatenate([words[0].transpose(1, 0, 2)] * cfg.B, axis=0)
    cu = torch.tensor([0, 777, 1554, 2331], dtype=torch.int32, device="cuda:0")
    O = tm.tilemix_prefill_varlen(to_dev(Q.reshape(-1, 4, 128)), to_dev(K.reshape(-1, 2, 128)),
                                  to_dev(V.reshape(-1, 2, 128)), cu, cu, 777, 777, to_dev(rows), 2,
                                  (128, 64), True, cfg.scale)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(O.cpu().numpy().reshape(O_fixed.shape).view(np.uint16),
                                  O_fixed.view(np.uint16))


@pytest.mark.parametrize("name,lens_q,lens_k,d,bm,g", CASES, ids=[c[0] for c in CASES])
def test_varlen_fused_equals_quantize_once_bitwise(name, lens_q, lens_k, d, bm, g):
    """The fused on-the-fly operand mode over the same packed batch (Appendix D; Section 4.1
    prefix sums): codes and scales made on chip equal the quantize-once ones, so the output is
    bitwise that of tilemix_prefill_varlen (checked against the oracle above); one mask is also
    checked against the oracle directly."""
    import torch
    import paper_2608_17336_amd as tm
    lens_k = lens_k or lens_q
    Hq, Hk = 4, 2
    B = len(lens_q)
    total_q, total_k = sum(lens_q), sum(lens_k)
    Lq, Lk = max(lens_q), max(lens_k)
    cfg = small_workload("vlf", B=1, Hq=Hq, Hk=Hk, d=d, L=max(total_q, total_k), block_m=bm,
                         group_size=g, k_outliers=True, index=900 + len(name))
    Q, K, V = make_qkv(cfg)
    Q, K, V = Q[0, :total_q], K[0, :total_k], V[0, :total_k]
    p = tm.Params(B, Hq, Hk, Lq, Lk, d, bm, 64, g, True, cfg.scale)
    W = tm.tilemix_route_words_per_row(p)
    rng = np.random.default_rng(len(name) + 50)
    cu_q = torch.tensor(np.concatenate([[0], np.cumsum(lens_q)]), dtype=torch.int32, device="cuda:0")
    cu_k = torch.tensor(np.concatenate([[0], np.cumsum(lens_k)]), dtype=torch.int32, device="cuda:0")
    q, k, v = to_dev(Q), to_dev(K), to_dev(V)
    for p_int8 in (0.5, 1.0, 0.0):
        words, per_seq = _pack(lens_q, lens_k, Hk, bm, g, W, rng, p_int8)
        w = to_dev(words)
        hint = 0 if p_int8 == 0.0 else -1
        log(f"varlen fused {name} p_int8={p_int8}")
        O_once = tm.tilemix_prefill_varlen(q, k, v, cu_q, cu_k, Lq, Lk, w, g, (bm, 64), True,
                                           cfg.scale, route_hint=hint)
        O_fused = tm.tilemix_prefill_varlen_fused(q, k, v, cu_q, cu_k, Lq, Lk, w, g, (bm, 64), True,
                                                  cfg.scale, route_hint=hint)
        torch.cuda.synchronize()
        assert torch.equal(O_once.view(torch.int16), O_fused.view(torch.int16)), (name, p_int8)
        if p_int8 == 0.5:
            got = O_fused.float().cpu().numpy().astype(np.float64)
            num = den = mx = 0.0
            q0 = k0 = 0
            for b, (lq, lk) in enumerate(zip(lens_q, lens_k)):
                if lq:
                    rows = [(0, h, np.arange(lq)) for h in range(Hq)]
                    ref = routed_attention_rows(Q[None, q0:q0 + lq], K[None, k0:k0 + lk],
                                                V[None, k0:k0 + lk], per_seq[b], block_m=bm,
                                                block_n=64, group_size=g, causal=True,
                                                scale=cfg.scale, rows=rows)
                    for (_, h, idx), r in zip(rows, ref):
                        diff = got[q0 + idx, h, :] - r
                        mx = max(mx, float(np.abs(diff).max()))
                        num += float((diff ** 2).sum())
                        den += float((r ** 2).sum())
                q0 += lq
                k0 += lk
            rel = (num / den) ** 0.5
            log(f"  max_abs={mx:.3e} rel_l2={rel:.3e}")
            assert mx <= MAX_ABS and rel <= REL_L2, (name, mx, rel)
