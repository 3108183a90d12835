"""Oracle: routing templates and coverage accounting (test infrastructure only).

Follows Appendix B ("Policy Construction and Sharing", "Coverage Accounting", and the
layouts One, Zero, Band, Global, Row-Random, Aligned Sparse, BigBird, SpTrans), written
from the set definitions with plain loops over tokens:

  * a routing group (m, g_j) is legal iff the rectangle I_m x J_{g_j} holds a legal
    (query, key) pair -- the garbled definition of the legal set is read this way;
  * each layout defines the FP16 set F_m inside the legal groups G_m of row m; every
    other legal group is INT8 (bit 1), illegal groups keep bit 0;
  * the 2-D map is broadcast over KV heads and packed little-endian into 64-bit words;
  * rho_hat = INT8 legal groups / legal groups.

Readings where Appendix B leaves details open (the library states the same ones):
  * "round" in k_m = round((1 - rho) |G_m|) rounds half up: floor(x + 1/2);
  * Row-Random's "uniform subset without replacement with a fixed seed": groups are taken in
    ascending order of the SplitMix64 output for seed XOR (m << 32 | g_j), ties by g_j;
  * SpTrans positions are key coordinates: query i sits at i' = i + L_k - L_q;
  * the paper's automatic group size formula is reproduced as printed.

Pins: tests/test_oracle_templates.py.
"""

from __future__ import annotations

import math

import numpy as np

MASK64 = (1 << 64) - 1


def splitmix64(x: int) -> int:
    """Output of the SplitMix64 generator (Steele, Lea, Flood 2014) for state ``x``."""
    z = (x + 0x9E3779B97F4A7C15) & MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def auto_group_size(len_k: int, block_n: int) -> int:
    """b_64 = ceil(L_k/64); BLOCK_N^mask = BLOCK_N ceil(max(b_64, BLOCK_N)/BLOCK_N); g = ratio."""
    b64 = math.ceil(len_k / 64)
    block_mask = block_n * math.ceil(max(b64, block_n) / block_n)
    return block_mask // block_n


class Geometry:
    def __init__(self, len_q, len_k, block_m, block_n, group_size, causal=True):
        self.Lq, self.Lk = len_q, len_k
        self.BM, self.BN, self.g = block_m, block_n, group_size
        self.causal = causal
        self.T_m = math.ceil(len_q / block_m)
        self.T_mask = math.ceil(math.ceil(len_k / block_n) / group_size)
        self.W = max(1, math.ceil(self.T_mask / 64))

    def queries(self, m):
        return np.arange(m * self.BM, min(self.Lq, (m + 1) * self.BM), dtype=np.int64)

    def keys(self, gj):
        span = self.g * self.BN
        return np.arange(gj * span, min(self.Lk, (gj + 1) * span), dtype=np.int64)

    def legal(self, i, j):
        """Elementwise legality of query positions i and key positions j (broadcasting)."""
        i, j = np.broadcast_arrays(i, j)
        ok = (j >= 0) & (j < self.Lk)
        if self.causal:
            ok = ok & (j <= i + (self.Lk - self.Lq))
        return ok

    def rect(self, m, gj):
        """Boolean [|I_m|, |J_g|]: legality of every pair of the row/group rectangle."""
        return self.legal(self.queries(m)[:, None], self.keys(gj)[None, :])

    def legal_groups(self, m):
        """G_m: groups whose rectangle with row m holds a legal pair (brute force, memoized)."""
        cache = self.__dict__.setdefault("_legal", {})
        if m not in cache:
            cache[m] = [gj for gj in range(self.T_mask) if self.rect(m, gj).any()]
        return list(cache[m])

    def pairs(self, m, gj):
        return int(self.rect(m, gj).sum())


def fp16_set(geo: Geometry, kind: str, m: int, *, band_w=0, global_groups=0, rand_fp16=0.0,
             align_alpha=0.0, align_beta=0.0, sp_stride=1, sp_tail=0, seed=0):
    """F_m of the named layout, as a Python set of group indices."""
    G = geo.legal_groups(m)
    Gs = set(G)
    if not G:
        return set()
    if kind == "one":
        return set()
    if kind == "zero":
        return set(G)
    if kind == "band":
        gamma = (m * geo.BM) // (geo.g * geo.BN)
        return {gj for gj in G if abs(gj - gamma) <= band_w}
    if kind == "global":
        return set(range(global_groups)) & Gs
    if kind == "rowrand":
        k = math.floor(rand_fp16 * len(G) + 0.5)
        order = sorted(G, key=lambda gj: (splitmix64(seed ^ ((m << 32) | gj)), gj))
        return set(order[:k])
    if kind == "aligned":
        a = min(len(G), max(0, math.ceil(align_alpha + align_beta * m)))
        gmax = max(G)
        return {gj for gj in G if gj >= gmax - a + 1}
    if kind == "bigbird":
        out = fp16_set(geo, "global", m, global_groups=global_groups)
        out |= fp16_set(geo, "rowrand", m, rand_fp16=rand_fp16, seed=seed)
        if band_w >= 0:
            out |= fp16_set(geo, "band", m, band_w=band_w)
        return out
    if kind == "sptrans":
        # K_i = [u s, i'] U (for r < u) [max(r s, (r+1) s - c), (r+1) s - 1], u = floor(i'/s),
        # as a boolean [query, key] table over every key position.
        s, c = sp_stride, sp_tail
        ip = geo.queries(m) + (geo.Lk - geo.Lq)
        ip = ip[ip >= 0]
        if ip.size == 0:
            return set()
        u = (ip // s)[:, None]
        k = np.arange(geo.Lk, dtype=np.int64)[None, :]
        r = k // s
        local = (k >= u * s) & (k <= ip[:, None])
        tail = (r < u) & (k >= np.maximum(r * s, (r + 1) * s - c)) & (k <= (r + 1) * s - 1)
        selected = (local | tail).any(axis=0)
        return {gj for gj in G if selected[geo.keys(gj)].any()}
    raise ValueError(kind)


def template_map(geo: Geometry, kind: str, **kw) -> np.ndarray:
    """0/1 map [T_m, T_mask]: 1 = INT8 on legal groups outside F_m, 0 elsewhere."""
    R = np.zeros((geo.T_m, geo.T_mask), dtype=np.uint8)
    for m in range(geo.T_m):
        f = fp16_set(geo, kind, m, **kw)
        for gj in geo.legal_groups(m):
            if gj not in f:
                R[m, gj] = 1
    return R


def pack_words(R: np.ndarray, heads_kv: int, planes: int = 1) -> np.ndarray:
    """b_{h_k,m} = sum_j R[m, j] 2^j, continued into further words past 64 groups; the map is
    broadcast over KV heads (and ``planes`` sequences): uint64 [planes, H_k, T_m, W]."""
    T_m, T_mask = R.shape
    W = max(1, math.ceil(T_mask / 64))
    out = np.zeros((planes, heads_kv, T_m, W), dtype=np.uint64)
    for m in range(T_m):
        for w in range(W):
            word = 0
            for j in range(64 * w, min(T_mask, 64 * (w + 1))):
                word |= int(R[m, j]) << (j - 64 * w)
            out[:, :, m, w] = np.uint64(word)
    return out


def coverage(geo: Geometry, R: np.ndarray):
    """(rho_hat over legal groups, INT8 share of legal pairs) of a 2-D map."""
    n_g = n_int8 = 0
    p_all = p_int8 = 0
    # (each KV head carries the same map, so the shares are those of one plane)
    for m in range(geo.T_m):
        for gj in geo.legal_groups(m):
            n_g += 1
            n_int8 += int(R[m, gj])
            p = geo.pairs(m, gj)
            p_all += p
            p_int8 += p * int(R[m, gj])
    return (n_int8 / n_g if n_g else 0.0), (p_int8 / p_all if p_all else 0.0)
