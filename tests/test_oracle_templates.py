"""Pins of the routing-template oracle (Appendix B) against closed forms, published values
and hand-worked cases.  CPU only."""

import math

import numpy as np
import pytest

from oracle.templates import (Geometry, auto_group_size, coverage, fp16_set, pack_words,
                              splitmix64, template_map)
from synth import pack_route_bits


def test_splitmix64_published_vector():
    # first outputs of SplitMix64 started from state 0 (reference implementation by Vigna)
    assert splitmix64(0) == 0xE220A8397B1DCDAF
    assert splitmix64(0x9E3779B97F4A7C15) == 0x6E789E6AA1B965F4


@pytest.mark.parametrize("L,g", [(1024, 1), (4096, 1), (8192, 2), (32768, 8), (65536, 16),
                                 (131072, 32), (262144, 64)])
def test_auto_group_size_values(L, g):
    # b_64 = ceil(L/64), BLOCK_N = 64: g = ceil(max(b_64, 64) / 64)
    assert auto_group_size(L, 64) == g


def test_auto_group_size_keeps_one_word():
    for L in list(range(1, 5000, 37)) + [2 ** k for k in range(6, 19)] + [262143, 262144]:
        g = auto_group_size(L, 64)
        assert math.ceil(math.ceil(L / 64) / g) <= 64, L


GEOS = [Geometry(1000, 1000, 128, 64, 2, True), Geometry(333, 333, 64, 64, 1, True),
        Geometry(300, 500, 128, 64, 3, True), Geometry(260, 260, 128, 64, 1, False)]


@pytest.mark.parametrize("geo", GEOS, ids=range(len(GEOS)))
def test_legal_groups_are_the_closed_form_prefix(geo):
    span = geo.g * geo.BN
    for m in range(geo.T_m):
        q_hi = min(geo.Lq, (m + 1) * geo.BM) - 1
        last = min(geo.Lk - 1, q_hi + geo.Lk - geo.Lq) if geo.causal else geo.Lk - 1
        want = list(range(last // span + 1)) if last >= 0 else []
        assert geo.legal_groups(m) == want


@pytest.mark.parametrize("geo", GEOS, ids=range(len(GEOS)))
def test_one_zero_and_limits(geo):
    legal = np.zeros((geo.T_m, geo.T_mask), np.uint8)
    for m in range(geo.T_m):
        legal[m, geo.legal_groups(m)] = 1
    one = template_map(geo, "one")
    zero = template_map(geo, "zero")
    np.testing.assert_array_equal(one, legal)
    assert not zero.any()
    np.testing.assert_array_equal(template_map(geo, "band", band_w=geo.T_mask), zero)
    np.testing.assert_array_equal(template_map(geo, "global", global_groups=0), one)
    np.testing.assert_array_equal(template_map(geo, "global", global_groups=geo.T_mask), zero)
    np.testing.assert_array_equal(template_map(geo, "rowrand", rand_fp16=0.0, seed=3), one)
    np.testing.assert_array_equal(template_map(geo, "rowrand", rand_fp16=1.0, seed=3), zero)
    np.testing.assert_array_equal(template_map(geo, "aligned", align_alpha=0, align_beta=0), one)
    assert coverage(geo, one) == (1.0, 1.0)
    assert coverage(geo, zero) == (0.0, 0.0)


def test_band_is_the_diagonal_group_at_width_zero():
    geo = GEOS[0]
    for m in range(geo.T_m):
        gamma = (m * geo.BM) // (geo.g * geo.BN)
        assert fp16_set(geo, "band", m, band_w=0) == ({gamma} & set(geo.legal_groups(m)))


def test_rowrand_row_sizes_and_determinism():
    geo = GEOS[0]
    for f in (0.1, 0.25, 0.5, 0.9):
        for m in range(geo.T_m):
            n = len(geo.legal_groups(m))
            a = fp16_set(geo, "rowrand", m, rand_fp16=f, seed=11)
            assert len(a) == math.floor(f * n + 0.5)
            assert a == fp16_set(geo, "rowrand", m, rand_fp16=f, seed=11)
    assert (template_map(geo, "rowrand", rand_fp16=0.5, seed=1) !=
            template_map(geo, "rowrand", rand_fp16=0.5, seed=2)).any()


def test_aligned_is_a_right_aligned_run():
    geo = GEOS[0]
    for m in range(geo.T_m):
        G = geo.legal_groups(m)
        a = min(len(G), math.ceil(1.0 + 0.75 * m))
        assert fp16_set(geo, "aligned", m, align_alpha=1.0, align_beta=0.75) == set(G[len(G) - a:])


def test_bigbird_is_the_union_of_its_components():
    geo = GEOS[2]
    kw = dict(band_w=1, global_groups=1, rand_fp16=0.3, seed=5)
    bb = template_map(geo, "bigbird", **kw)
    parts = [template_map(geo, "band", band_w=1), template_map(geo, "global", global_groups=1),
             template_map(geo, "rowrand", rand_fp16=0.3, seed=5)]
    np.testing.assert_array_equal(bb, parts[0] & parts[1] & parts[2])


def test_sptrans_hand_worked():
    # L = 8 tokens, one token per key group (BLOCK_N = 1 would be the paper's token-level
    # definition): BLOCK_M = 2, stride s = 4, tail c = 1.  Query rows {0,1}, {2,3}, {4,5}, {6,7}.
    # Row 2 (queries 4, 5): local [4, 4] and [4, 5]; tails of stride 0: key 3 -> F = {3, 4, 5}.
    # Row 3 (queries 6, 7): local [4, 6], [4, 7]; tail key 3 -> F = {3, 4, 5, 6, 7}.
    geo = Geometry(8, 8, 2, 1, 1, True)
    want = [{0, 1}, {0, 1, 2, 3}, {3, 4, 5}, {3, 4, 5, 6, 7}]
    for m in range(4):
        assert fp16_set(geo, "sptrans", m, sp_stride=4, sp_tail=1) == want[m]


def test_sptrans_limits():
    geo = GEOS[0]
    zero = template_map(geo, "zero")
    # one stride covering the whole sequence: every key up to i is local -> all FP16
    np.testing.assert_array_equal(template_map(geo, "sptrans", sp_stride=4096, sp_tail=0), zero)
    # tails as long as the stride: every earlier stride is kept whole -> all FP16
    np.testing.assert_array_equal(template_map(geo, "sptrans", sp_stride=200, sp_tail=200), zero)


def test_coverage_hand_count():
    # L = 4, BLOCK_M = BLOCK_N = 2, g = 1, causal: row 0 has group 0 (3 pairs); row 1 has
    # groups 0 (4 pairs) and 1 (3 pairs).  INT8 on (1, 0) only: groups 1/3, pairs 4/10.
    geo = Geometry(4, 4, 2, 2, 1, True)
    R = np.array([[0, 0], [1, 0]], np.uint8)
    assert coverage(geo, R) == (1 / 3, 4 / 10)


def test_pack_words_matches_the_generator_packing():
    rng = np.random.default_rng(0)
    R = rng.integers(0, 2, size=(5, 130)).astype(np.uint8)
    np.testing.assert_array_equal(pack_words(R, 3), pack_route_bits(np.broadcast_to(R, (3, 5, 130))))


def test_coverage_hand_count_full_attention():
    # L = 260, BLOCK_M = 128, BLOCK_N = 64, g = 1, no causal mask: 3 x 5 groups, all legal.
    # Band w = 0 keeps (0,0), (1,2), (2,4) in FP16: 8192 + 8192 + 16 of the 260^2 pairs.
    geo = Geometry(260, 260, 128, 64, 1, False)
    R = template_map(geo, "band", band_w=0)
    g, p = coverage(geo, R)
    assert g == 12 / 15
    assert p == (260 * 260 - 16400) / (260 * 260)
