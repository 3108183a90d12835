"""GPU: the INT8 operands the attention kernel itself makes and multiplies, bit for bit.

The attention kernel quantizes every 128-row query block in the prologue of the workgroup
that owns it (Appendix C, "Quantization Granularity": one scale per 128 query tokens and
head) and multiplies the codes on the INT8 matrix cores with either a zero or a
1.5 * 2^23-biased accumulator start (Appendix C, "INT8 Score Computation").
tilemix_debug_prefill runs that same kernel in an instantiation that also writes out:
  * each row's query codes and its workgroup's query-block scale, compared with
    oracle.quantize_blocks (128-row blocks restarting at each sequence's first row);
  * the INT32 product C of every INT8-routed tile each wave computes, with the bias taken
    off, compared with the oracle's exact integer products;
  * how each wave formed each tile (biased start, zero start, or the masked per-tile path),
    compared with the geometry: which tiles every row sees in full and which waves see a
    tile that crosses the diagonal or the sequence end.
Its output O must equal the ordinary call's bit for bit.
"""

import math

import numpy as np
import pytest

from gpu_util import MAX_ABS, REL_L2, log, to_dev
from oracle import QUANT_BLOCK_Q, OracleOperands, int8_tile_product, quantize_blocks
from oracle import routed_attention_rows
from synth import MaskSpec, WORKLOADS, make_qkv, make_route_bits, pack_route_bits, small_workload

pytestmark = pytest.mark.gpu

FOLDED, EXACT, MASKED = 1, 2, 3


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2608_17336_amd as tm
    tm.load_library()


def _route_bit(words_row, gj):
    return int((int(words_row[gj >> 6]) >> (gj & 63)) & 1)


def check_sequence(Q, K, words, exports, *, bm, g, causal, label):
    """Check the exports of one sequence.  Q [1, Lq, Hq, d], K [1, Lk, Hk, d], words
    [1, Hk, T_m, W]; exports = (q8 [Lq, Hq, d], dq [T_m, Hq] int16 bits, tiles
    [T_m, Hq, T_n, bm, 64], kinds [T_m, Hq, T_n, bm // 32]) as NumPy arrays, the slices of
    this sequence.  Returns a count of the kinds seen."""
    q8, dq, tiles, kinds = exports
    _, Lq, Hq, d = Q.shape
    _, Lk, Hk, _ = K.shape
    T_m = -(-Lq // bm)
    ops = OracleOperands.from_inputs(Q, K)
    off = (Lk - Lq) if causal else Lk
    seen = {FOLDED: 0, EXACT: 0, MASKED: 0}
    for m in range(T_m):
        wg_last_key = min(Lk - 1, min(Lq - 1, m * bm + bm - 1) + off)
        rows = slice(m * bm, min(Lq, (m + 1) * bm))
        if wg_last_key < 0:
            continue
        n_end = wg_last_key // 64
        n_split = max(0, min(n_end + 1, (min(Lk - 1, m * bm + off) + 1) // 64))
        for hq in range(Hq):
            hk = hq // (Hq // Hk)
            wrow = words[0, hk, m]
            need_int8 = any(_route_bit(wrow, gj) for gj in range(n_end // g + 1))
            where = f"{label} m={m} hq={hq}"
            if need_int8:
                np.testing.assert_array_equal(q8[rows, hq], ops.q8[0, rows, hq], err_msg=where)
                want = ops.dq[0, (m * bm) // QUANT_BLOCK_Q, hq].view(np.int16)
                assert dq[m, hq] == want, (where, dq[m, hq], want)
            else:
                assert np.all(q8[rows, hq] == -128), where
                assert dq[m, hq] == -1, where
            for n in range(n_end + 1):
                int8 = _route_bit(wrow, n // g) == 1
                full = int8_tile_product(ops, 0, hq, hk, m, n, bm, 64) if int8 else None
                for w in range(bm // 32):
                    q0 = m * bm + 32 * w
                    kind = int(kinds[m, hq, n, w])
                    if not int8 or q0 >= Lq:
                        assert kind == 0, (where, n, w, kind)
                        continue
                    wave_last_key = min(Lk - 1, min(Lq - 1, q0 + 31) + off)
                    if n < n_split:
                        assert kind in (FOLDED, EXACT), (where, n, w, kind)
                    elif n * 64 <= wave_last_key:
                        assert kind == MASKED, (where, n, w, kind)
                    else:
                        assert kind == 0, (where, n, w, kind)
                        continue
                    seen[kind] += 1
                    nq = min(32, Lq - q0)
                    nk = min(64, Lk - n * 64)
                    got = tiles[m, hq, n, 32 * w:32 * w + nq, :nk].astype(np.int64)
                    np.testing.assert_array_equal(got, full[32 * w:32 * w + nq, :nk],
                                                  err_msg=f"{where} n={n} w={w} kind={kind}")
    return seen


def _debug_and_plain(Q, K, V, words, *, bm, g, causal, scale, fused, **kw):
    import torch
    import paper_2608_17336_amd as tm
    q, k, v, w = to_dev(Q), to_dev(K), to_dev(V), to_dev(words)
    O, q8, dq, tiles, kinds = tm.tilemix_debug_prefill(q, k, v, w, g, (bm, 64), causal, scale,
                                                       fused=fused, **kw)
    run = tm.tilemix_prefill_fused if fused else tm.tilemix_prefill
    O_plain = run(q, k, v, w, g, (bm, 64), causal, scale, **kw)
    torch.cuda.synchronize()
    assert torch.equal(O.view(torch.int16), O_plain.view(torch.int16)), "debug kernel output differs"
    return O, (q8.cpu().numpy(), dq.cpu().numpy(), tiles.cpu().numpy(), kinds.cpu().numpy())


def _check_batch(Q, K, words, exports, *, bm, g, causal, label, route_per_batch=False):
    q8, dq, tiles, kinds = exports
    B, Lq = Q.shape[0], Q.shape[1]
    T_m = -(-Lq // bm)
    seen = {FOLDED: 0, EXACT: 0, MASKED: 0}
    for b in range(B):
        r = slice(b * T_m, (b + 1) * T_m)
        wb = words[b:b + 1] if route_per_batch else words
        s = check_sequence(Q[b:b + 1], K[b:b + 1], wb, (q8[b], dq[r], tiles[r], kinds[r]),
                           bm=bm, g=g, causal=causal, label=f"{label} b={b}")
        for k2 in seen:
            seen[k2] += s[k2]
    return seen


CASES = [
    # name, small_workload kwargs
    ("d128-bm128-ragged", dict(B=2, Hq=4, Hk=2, d=128, L=333, block_m=128, group_size=1,
                               k_outliers=True)),
    ("d128-bm64", dict(B=1, Hq=2, Hk=1, d=128, L=300, block_m=64, group_size=1)),
    ("d64-bm64-ragged", dict(B=2, Hq=4, Hk=1, d=64, L=190, block_m=64, group_size=2)),
    ("d64-bm128", dict(B=1, Hq=2, Hk=2, d=64, L=257, block_m=128, group_size=1)),
    ("zero-blocks", dict(B=1, Hq=2, Hk=1, d=128, L=700, block_m=128, group_size=1)),
    ("zero-blocks-bm64", dict(B=1, Hq=2, Hk=2, d=128, L=700, block_m=64, group_size=3)),
    ("noncausal", dict(B=1, Hq=2, Hk=1, d=128, L=300, block_m=128, group_size=1, causal=False)),
    ("large-scores", dict(B=1, Hq=2, Hk=1, d=128, L=400, block_m=128, group_size=1)),
]


def _case_inputs(name, cfg):
    Q, K, V = make_qkv(cfg)
    if name.startswith("zero-blocks"):
        Q[0, 128:256, 0, :] = 0.0      # a whole 128-row query block: scale 0, codes 0
        Q[0, 300:301, 1, :] = 0.0      # one zero row inside a block
        K[0, 64:128, 0, :] = 0.0       # a whole 64-key block
    if name == "large-scores":
        # query values 16 times larger: the INT8 score factor then exceeds the biased start's
        # bound, so the pipelined INT8 tiles start their accumulators at 0
        Q = (Q.astype(np.float32) * 16.0).astype(np.float16)
    return Q, K, V


@pytest.mark.parametrize("fused", [False, True], ids=["quantize-once", "fused"])
@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_kernel_operands_bitexact(name, kw, fused):
    totals = {FOLDED: 0, EXACT: 0, MASKED: 0}
    for mi, mask in enumerate([MaskSpec("bernoulli", 0.5), MaskSpec("all_int8")]):
        cfg = small_workload(name, mask=mask, index=1200 + len(name), **kw)
        log(f"operands {name} fused={fused} mask={mask.label}")
        Q, K, V = _case_inputs(name, cfg)
        words, _ = make_route_bits(cfg, mask, mi)
        _, ex = _debug_and_plain(Q, K, V, words, bm=cfg.block_m, g=cfg.group_size,
                                 causal=cfg.causal, scale=cfg.scale, fused=fused)
        seen = _check_batch(Q, K, words, ex, bm=cfg.block_m, g=cfg.group_size, causal=cfg.causal,
                            label=name)
        log(f"  tiles by kind: {seen}")
        for k2 in totals:
            totals[k2] += seen[k2]
    if name == "large-scores":
        assert totals[EXACT] > 0 and totals[FOLDED] == 0, totals
    else:
        assert totals[FOLDED] > 0, totals
    if cfg.causal:
        assert totals[MASKED] > 0, totals


def test_kernel_operands_outlier_workload():
    """The 32K workload's heads, group size, Bernoulli 0.75 map and K outlier channels, on a
    shorter sequence."""
    cfg = WORKLOADS["32k-gqa"].with_(L=640)
    mask = cfg.masks[0]
    Q, K, V = make_qkv(cfg)
    words, _ = make_route_bits(cfg, mask, 0)
    for fused in (False, True):
        log(f"operands 32k-gqa shape at L=640 fused={fused}")
        _, ex = _debug_and_plain(Q, K, V, words, bm=cfg.block_m, g=cfg.group_size,
                                 causal=cfg.causal, scale=cfg.scale, fused=fused)
        seen = _check_batch(Q, K, words, ex, bm=cfg.block_m, g=cfg.group_size, causal=True,
                            label="32k-gqa@640")
        log(f"  tiles by kind: {seen}")
        assert seen[FOLDED] > 0 and seen[MASKED] > 0


def test_kernel_operands_per_sequence_maps():
    cfg = small_workload("per-seq", B=3, Hq=4, Hk=2, d=128, L=260, block_m=128, group_size=2,
                         k_outliers=True, index=1290)
    Q, K, V = make_qkv(cfg)
    rng = np.random.default_rng(5)
    R = (rng.random((3, cfg.Hk, cfg.T_m, cfg.T_mask)) < 0.5).astype(np.uint8)
    words = pack_route_bits(R.reshape(3 * cfg.Hk, cfg.T_m, cfg.T_mask)).reshape(3, cfg.Hk, cfg.T_m, -1)
    _, ex = _debug_and_plain(Q, K, V, words, bm=128, g=2, causal=True, scale=cfg.scale, fused=False,
                             route_per_batch=True)
    seen = _check_batch(Q, K, words, ex, bm=128, g=2, causal=True, label="per-seq",
                        route_per_batch=True)
    assert seen[FOLDED] > 0


VARLEN = [
    # name, lens, d, block_m, g
    ("bm128", [300, 1, 0, 129, 64, 200], 128, 128, 1),
    ("bm64", [300, 1, 0, 129, 64, 200], 128, 64, 2),
    ("d64-bm64", [190, 33, 257], 64, 64, 1),
]


def _varlen_inputs(name, lens, d, bm, g, p_int8=0.6):
    import paper_2608_17336_amd as tm
    Hq, Hk = 4, 2
    total = sum(lens)
    cfg = small_workload("vlops", B=1, Hq=Hq, Hk=Hk, d=d, L=total, block_m=bm, group_size=g,
                         k_outliers=True, index=1300 + len(name))
    Q, K, V = make_qkv(cfg)
    Q, K, V = Q[0], K[0], V[0]
    Lmax = max(lens)
    p = tm.Params(len(lens), Hq, Hk, Lmax, Lmax, d, bm, 64, g, True, cfg.scale)
    W = tm.tilemix_route_words_per_row(p)
    rng = np.random.default_rng(len(name) + 7)
    rows, per_seq = [], []
    for L in lens:
        T_m, T_mask = -(-L // bm), -(-(-(-L // 64)) // g)
        legal = np.zeros((T_m, T_mask), bool)
        for m in range(T_m):
            legal[m, :(min(L, (m + 1) * bm) - 1) // (64 * g) + 1] = True
        Rb = (rng.random((Hk, T_m, T_mask)) < p_int8) & legal[None]
        full = np.zeros((Hk, T_m, W), np.uint64)
        if T_m:
            wb = pack_route_bits(Rb.astype(np.uint8))[0]             # [H_k, T_m, W_b]
            full[..., :wb.shape[-1]] = wb
        per_seq.append(full[None])
        rows.append(full.transpose(1, 0, 2))
    words = np.concatenate(rows, axis=0)
    return cfg, Q, K, V, words, per_seq, Hq


@pytest.mark.parametrize("fused", [False, True], ids=["quantize-once", "fused"])
@pytest.mark.parametrize("name,lens,d,bm,g", VARLEN, ids=[c[0] for c in VARLEN])
def test_kernel_operands_varlen(name, lens, d, bm, g, fused):
    """Query blocks restart at each sequence's first row (Appendix C, varlen scale layout)."""
    import torch
    import paper_2608_17336_amd as tm
    cfg, Q, K, V, words, per_seq, Hq = _varlen_inputs(name, lens, d, bm, g)
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32, device="cuda:0")
    Lmax = max(lens)
    log(f"operands varlen {name} fused={fused} lens={lens}")
    q, k, v, w = to_dev(Q), to_dev(K), to_dev(V), to_dev(words)
    O, q8, dq, tiles, kinds = tm.tilemix_debug_prefill(q, k, v, w, g, (bm, 64), True, cfg.scale,
                                                       fused=fused, cu_seqlens_q=cu, cu_seqlens_k=cu,
                                                       max_len_q=Lmax, max_len_k=Lmax)
    run = tm.tilemix_prefill_varlen_fused if fused else tm.tilemix_prefill_varlen
    O_plain = run(q, k, v, cu, cu, Lmax, Lmax, w, g, (bm, 64), True, cfg.scale)
    torch.cuda.synchronize()
    assert torch.equal(O.view(torch.int16), O_plain.view(torch.int16))
    q8, dq, tiles, kinds = q8.cpu().numpy(), dq.cpu().numpy(), tiles.cpu().numpy(), kinds.cpu().numpy()
    seen = {FOLDED: 0, EXACT: 0, MASKED: 0}
    q0 = r0 = 0
    for b, L in enumerate(lens):
        T_m = -(-L // bm)
        if L:
            Qb, Kb = Q[None, q0:q0 + L], K[None, q0:q0 + L]
            s = check_sequence(Qb, Kb, per_seq[b], (q8[q0:q0 + L], dq[r0:r0 + T_m],
                                                   tiles[r0:r0 + T_m], kinds[r0:r0 + T_m]),
                               bm=bm, g=g, causal=True, label=f"{name} seq={b}")
            for k2 in seen:
                seen[k2] += s[k2]
        q0 += L
        r0 += T_m
    log(f"  tiles by kind: {seen}")
    assert seen[FOLDED] > 0 and seen[MASKED] > 0


def test_fold_bound_after_running_max_jump():
    """INT8 tiles whose biased start is admitted against the running max as it stands, followed by
    a score jump that moves the running max past the fold's bound: the kernel drops the bias
    from the affected tiles and the output stays within the bar against the oracle.
    Query and keys are multiples of one sign pattern, so every INT8 product is 128 * 127^2 and
    the scores grow with the key block's magnitude."""
    import torch
    import paper_2608_17336_amd as tm
    rng = np.random.default_rng(11)
    d, L = 128, 1024
    u = np.where(rng.random(d) < 0.5, -1.0, 1.0).astype(np.float32)
    s_q = 4.0
    # key block magnitudes: scale * log2(e) * s_q * s_k * 128 is the log2 score; the jump at
    # block 9 takes it from about 1630 to about 2365 while 1.5 * 2^23 * c is about 14430
    s_k = np.where(np.arange(L // 64) < 9, 25.0, 36.25)
    Q = (s_q * np.tile(u, (L, 1)))[None, :, None, :].astype(np.float16)
    K = (np.repeat(s_k, 64)[:, None] * u[None, :])[None, :, None, :].astype(np.float16)
    V = rng.standard_normal((1, L, 1, d), dtype=np.float32).astype(np.float16)
    R = np.ones((1, L // 128, L // 64), np.uint8)
    words = pack_route_bits(R)
    scale = 1.0 / math.sqrt(d)
    O = tm.tilemix_prefill(to_dev(Q), to_dev(K), to_dev(V), to_dev(words), 1, (128, 64), True, scale)
    torch.cuda.synchronize()
    rows = [(0, 0, np.arange(L))]
    ref = routed_attention_rows(Q, K, V, words, block_m=128, block_n=64, group_size=1, causal=True,
                                scale=scale, rows=rows)[0]
    got = O[0, :, 0, :].float().cpu().numpy().astype(np.float64)
    mx = float(np.abs(got - ref).max())
    rel = float(np.sqrt(((got - ref) ** 2).sum() / (ref ** 2).sum()))
    log(f"fold bound: max_abs={mx:.3e} rel_l2={rel:.3e}")
    assert mx <= MAX_ABS and rel <= REL_L2


def test_varlen_route_rows_bound():
    """A routing tensor with fewer rows than the batch's query tiles: the sequences that fit
    are attended as usual, the rest are empty and their output rows are not written."""
    import torch
    import paper_2608_17336_amd as tm
    lens = [200, 300, 100]             # 2 + 3 + 1 query-tile rows at BLOCK_M = 128
    cfg, Q, K, V, words, per_seq, Hq = _varlen_inputs("rows", lens, 128, 128, 1)
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32, device="cuda:0")
    sentinel = torch.full((sum(lens), Hq, 128), 7.0, dtype=torch.float16, device="cuda:0")
    O = sentinel.clone()
    tm.tilemix_prefill_varlen(to_dev(Q), to_dev(K), to_dev(V), cu, cu, 300, 300, to_dev(words[:4]),
                              1, (128, 64), True, cfg.scale, O=O)
    torch.cuda.synchronize()
    got = O.float().cpu().numpy()
    assert np.all(got[200:] == 7.0)    # sequences 1 and 2 do not fit in 4 rows
    ref = routed_attention_rows(Q[None, :200], K[None, :200], V[None, :200], per_seq[0],
                                block_m=128, block_n=64, group_size=1, causal=True, scale=cfg.scale,
                                rows=[(0, h, np.arange(200)) for h in range(Hq)])
    for h, r in enumerate(ref):
        diff = got[:200, h].astype(np.float64) - r
        assert float(np.abs(diff).max()) <= MAX_ABS
