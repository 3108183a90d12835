"""Seeded generators: Q/K/V tensors, routing maps, packed routing words, row samples.

Random streams (NumPy PCG64) are keyed by (workload seed, stream id, chunk)
so that the tensors do not depend on the number of threads used to draw them:
stream 0 = Q, 1 = K, 2 = V, 3 = outlier channels, 4 + mask index = routing map,
9 = row sample.

Layout: Q, O are [B, L, H_q, d]; K, V are [B, L, H_k, d] (token-major,
head-interleaved, contiguous).  Routing words are uint64 [1, H_k, T_m, W]
(one map for all sequences of the batch), bit g of a row in word g // 64 at
position g % 64, 1 = INT8 and 0 = FP16.  Bits of groups that no legal
(query, key) pair touches are left at 0.
"""

from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .configs import MaskSpec, WorkloadConfig

_STREAM_Q, _STREAM_K, _STREAM_V, _STREAM_OUTLIER, _STREAM_MASK, _STREAM_ROWS = 0, 1, 2, 3, 4, 9
_CHUNK_ROWS = 2048


def _workers() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _normal_fp16(seed: int, stream: int, shape) -> np.ndarray:
    """N(0,1) drawn in float32, rounded to float16, drawn chunk by chunk in parallel."""
    B, L, H, d = shape
    out = np.empty(shape, dtype=np.float16)
    jobs = [(b, c) for b in range(B) for c in range(math.ceil(L / _CHUNK_ROWS))]

    def fill(job):
        b, c = job
        lo, hi = c * _CHUNK_ROWS, min(L, (c + 1) * _CHUNK_ROWS)
        ss = np.random.SeedSequence(seed, spawn_key=(stream, b, c))
        rng = np.random.Generator(np.random.PCG64(ss))
        out[b, lo:hi] = rng.standard_normal((hi - lo, H, d), dtype=np.float32).astype(np.float16)

    if len(jobs) == 1:
        fill(jobs[0])
    else:
        with ThreadPoolExecutor(_workers()) as ex:
            list(ex.map(fill, jobs))
    return out


def outlier_channels(cfg: WorkloadConfig) -> np.ndarray:
    """[H_k, n_out] channel indices scaled x8 in K (ceil(1% of d) per KV head)."""
    n_out = math.ceil(0.01 * cfg.d)
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(cfg.seed, spawn_key=(_STREAM_OUTLIER,))))
    return np.stack([rng.choice(cfg.d, size=n_out, replace=False) for _ in range(cfg.Hk)])


def make_qkv(cfg: WorkloadConfig):
    """Return (Q, K, V) as float16 NumPy arrays for the workload."""
    Q = _normal_fp16(cfg.seed, _STREAM_Q, (cfg.B, cfg.Lq, cfg.Hq, cfg.d))
    K = _normal_fp16(cfg.seed, _STREAM_K, (cfg.B, cfg.Lk, cfg.Hk, cfg.d))
    V = _normal_fp16(cfg.seed, _STREAM_V, (cfg.B, cfg.Lk, cfg.Hk, cfg.d))
    if cfg.k_outliers:
        ch = outlier_channels(cfg)
        for h in range(cfg.Hk):
            for c in ch[h]:
                K[:, :, h, c] = (K[:, :, h, c].astype(np.float32) * 8.0).astype(np.float16)
    return Q, K, V


def _group_bounds(cfg: WorkloadConfig):
    """Per query-tile row m: [q_lo, q_hi]; per group g: [k_lo, k_hi] (inclusive)."""
    m = np.arange(cfg.T_m, dtype=np.int64)
    q_lo = m * cfg.block_m
    q_hi = np.minimum(cfg.Lq, (m + 1) * cfg.block_m) - 1
    g = np.arange(cfg.T_mask, dtype=np.int64)
    span = cfg.group_size * cfg.block_n
    k_lo = g * span
    k_hi = np.minimum(cfg.Lk, (g + 1) * span) - 1
    return q_lo, q_hi, k_lo, k_hi


def legal_group_table(cfg: WorkloadConfig) -> np.ndarray:
    """bool [T_m, T_mask]: does any legal (i, j) pair fall in row m, group g?"""
    q_lo, q_hi, k_lo, k_hi = _group_bounds(cfg)
    legal = (k_lo[None, :] <= k_hi[None, :]) & np.ones((cfg.T_m, 1), bool)
    if cfg.causal:
        off = cfg.Lk - cfg.Lq
        legal &= k_lo[None, :] <= (q_hi[:, None] + off)
    return legal


def _pairs_in_groups(cfg: WorkloadConfig) -> np.ndarray:
    """int64 [T_m, T_mask]: number of legal (i, j) pairs in each row/group rectangle."""
    q_lo, q_hi, k_lo, k_hi = _group_bounds(cfg)
    out = np.zeros((cfg.T_m, cfg.T_mask), dtype=np.int64)
    off = cfg.Lk - cfg.Lq
    for m in range(cfg.T_m):
        i = np.arange(q_lo[m], q_hi[m] + 1, dtype=np.int64)
        last = np.minimum(cfg.Lk - 1, i + off) if cfg.causal else np.full(i.shape, cfg.Lk - 1)
        # per i: count of j in [k_lo, min(k_hi, last_i)]
        hi = np.minimum(k_hi[None, :], last[:, None])
        out[m] = np.clip(hi - k_lo[None, :] + 1, 0, None).sum(axis=0)
    return out


def pack_route_bits(R: np.ndarray) -> np.ndarray:
    """Pack a 0/1 map [H_k, T_m, T_mask] into uint64 words [1, H_k, T_m, W]."""
    R = np.asarray(R).astype(np.uint64)
    Hk, T_m, T_mask = R.shape
    W = max(1, math.ceil(T_mask / 64))
    padded = np.zeros((Hk, T_m, W * 64), dtype=np.uint64)
    padded[..., :T_mask] = R
    padded = padded.reshape(Hk, T_m, W, 64)
    weights = np.left_shift(np.uint64(1), np.arange(64, dtype=np.uint64))
    words = np.bitwise_or.reduce(padded * weights, axis=-1)
    return words.reshape(1, Hk, T_m, W).astype(np.uint64)


def route_map(cfg: WorkloadConfig, mask: MaskSpec, mask_index: int = 0) -> np.ndarray:
    """The 0/1 routing map [H_k, T_m, T_mask] (illegal groups are 0)."""
    legal = legal_group_table(cfg)
    shape = (cfg.Hk, cfg.T_m, cfg.T_mask)
    if mask.kind == "all_fp16":
        R = np.zeros(shape, dtype=bool)
    elif mask.kind == "all_int8":
        R = np.broadcast_to(legal, shape).copy()
    elif mask.kind == "bernoulli":
        ss = np.random.SeedSequence(cfg.seed, spawn_key=(_STREAM_MASK + mask_index,))
        draws = np.random.Generator(np.random.PCG64(ss)).random(shape)
        R = (draws < mask.p_int8) & legal[None]
    elif mask.kind == "sink_band":
        q_lo, q_hi, k_lo, k_hi = _group_bounds(cfg)
        sink = (k_lo < mask.sink_keys)[None, :]
        # smallest (i - j) over legal pairs of the rectangle; 0 when it meets the diagonal
        gap = np.maximum(0, q_lo[:, None] - k_hi[None, :])
        near = gap < mask.band_tokens
        fp16 = sink | near
        R = np.broadcast_to(legal & ~fp16, shape).copy()
    else:
        raise ValueError(f"unknown mask kind {mask.kind!r}")
    return R.astype(np.uint8)


def make_route_bits(cfg: WorkloadConfig, mask: MaskSpec | None = None, mask_index: int = 0):
    """Return (packed uint64 words [1, H_k, T_m, W], 0/1 map [H_k, T_m, T_mask])."""
    if mask is None:
        mask = cfg.masks[mask_index]
    R = route_map(cfg, mask, mask_index)
    return pack_route_bits(R), R


def decode_route_bits(cfg: WorkloadConfig, mask: MaskSpec):
    """Routing map of one decode step over the workload's L keys: one query-tile row per KV
    head, all FP16 / all INT8 / Bernoulli(p_int8, default 0.5) per key group, broadcast over
    sequences.  Return (packed words [1, H_k, 1, W], 0/1 map [H_k, 1, T_mask])."""
    T_mask = -(-(-(-cfg.L // cfg.block_n)) // cfg.group_size)
    if mask.kind == "all_fp16":
        R = np.zeros((cfg.Hk, 1, T_mask), np.uint8)
    elif mask.kind == "all_int8":
        R = np.ones((cfg.Hk, 1, T_mask), np.uint8)
    else:
        rng = np.random.default_rng(cfg.seed)
        R = (rng.random((cfg.Hk, 1, T_mask)) < (mask.p_int8 or 0.5)).astype(np.uint8)
    return pack_route_bits(R), R


def route_stats(cfg: WorkloadConfig, R: np.ndarray) -> dict:
    """Realized INT8 coverage: over legal groups (rho_hat) and over legal pairs (rho_p)."""
    legal = legal_group_table(cfg)
    pairs = _pairs_in_groups(cfg)
    n_groups = int(legal.sum()) * cfg.Hk
    int8_groups = int((R.astype(bool) & legal[None]).sum())
    # pairs are counted per query head: each KV head serves H_q / H_k query heads
    tot_pairs = int(pairs.sum()) * cfg.Hk
    int8_pairs = int((R.astype(np.int64) * pairs[None]).sum())
    return {
        "legal_groups": n_groups,
        "int8_groups": int8_groups,
        "rho_hat": int8_groups / n_groups if n_groups else 0.0,
        "rho_pairs": int8_pairs / tot_pairs if tot_pairs else 0.0,
        "legal_pairs_total": cfg.legal_pairs(),
    }


def sample_rows(cfg: WorkloadConfig, n_random: int = 64, n_pairs: int = 4, max_boundaries: int = 8):
    """Rows for sampled checks: list of (b, h_q, sorted query indices).

    (b, h_q) pairs cover two query heads of one KV group and more than one KV
    head; rows are the first 8, the last 8, pairs of rows on each side of a few
    query-tile boundaries, and uniform random rows.
    """
    ss = np.random.SeedSequence(cfg.seed, spawn_key=(_STREAM_ROWS,))
    rng = np.random.Generator(np.random.PCG64(ss))
    grp = cfg.Hq // cfg.Hk
    cand = [(0, 0)]
    if grp > 1:
        cand.append((0, 1))
    cand.append((cfg.B - 1, cfg.Hq - 1))
    cand.append((cfg.B // 2, min(cfg.Hq - 1, (cfg.Hq // 2) + 1)))
    pairs = []
    for p in cand:
        if p not in pairs:
            pairs.append(p)
    pairs = pairs[:max(n_pairs, 1)]
    L = cfg.Lq
    out = []
    for b, h in pairs:
        rows = set(range(min(8, L))) | set(range(max(0, L - 8), L))
        ms = rng.choice(np.arange(1, max(2, cfg.T_m)), size=min(max_boundaries, max(1, cfg.T_m - 1)),
                        replace=False) if cfg.T_m > 1 else []
        for m in ms:
            rows.add(int(m) * cfg.block_m - 1)
            rows.add(int(m) * cfg.block_m)
        rows |= set(int(x) for x in rng.integers(0, L, size=n_random))
        out.append((b, h, np.array(sorted(r for r in rows if 0 <= r < L), dtype=np.int64)))
    return out
