"""The work model behind bench.py's effective TFLOP/s and roofline fraction, pinned to closed
forms and to brute force (no GPU): legal (query, key) pairs of the causal triangle, the
precision-weighted time at peak, and the share of legal pairs the route map sends to INT8."""

import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from synth import WORKLOADS, MaskSpec, small_workload  # noqa: E402
from synth.generate import route_map, route_stats  # noqa: E402


def test_legal_pairs_closed_form():
    for cfg in WORKLOADS.values():
        L = cfg.L
        per_head = L * (L + 1) // 2 if cfg.causal else L * L
        assert cfg.legal_pairs() == cfg.B * cfg.Hq * per_head, cfg.name


def test_weighted_peak_32k():
    cfg = WORKLOADS["32k-gqa"]
    pairs = 32 * 32768 * 32769 // 2
    F = 2.0 * 128 * pairs   # each of the two products, Q K^T and P V
    fm = bench.flop_model(cfg, 0.75)
    assert fm["pairs"] == pairs
    assert fm["flops"] == 2 * F
    t = 0.25 * F / 2.5e15 + 0.75 * F / 5.0e15 + F / 2.5e15
    assert fm["t_star_s"] == pytest.approx(t, rel=1e-12)
    assert fm["t_star_s"] == pytest.approx(2.8588e-3, rel=1e-4)
    assert fm["weighted_peak"] == pytest.approx(2 * F / t, rel=1e-12)
    # the uniform masks bracket it: all FP16 prices everything at 2.5, all INT8 halves Q K^T
    assert bench.flop_model(cfg, 0.0)["weighted_peak"] == pytest.approx(2.5e15, rel=1e-12)
    assert bench.flop_model(cfg, 1.0)["weighted_peak"] == pytest.approx(2 / (1 / 5.0e15 + 1 / 2.5e15),
                                                                        rel=1e-12)


@pytest.mark.parametrize("L,bm,bn,g", [(300, 128, 64, 1), (257, 64, 64, 3), (1000, 128, 64, 2),
                                       (1024, 64, 64, 4)])
def test_route_coverage_brute_force(L, bm, bn, g):
    cfg = small_workload("coverage", Hq=4, Hk=2, d=64, L=L, block_m=bm, block_n=bn, group_size=g,
                         mask=MaskSpec("bernoulli", 0.5))
    R = route_map(cfg, cfg.masks[0])
    st = route_stats(cfg, R)
    i = np.arange(L)[:, None]
    j = np.arange(L)[None, :]
    legal = j <= i
    m, grp = np.broadcast_arrays(i // bm, (j // bn) // g)   # query tile, key tile group
    int8_pairs = sum(int((R[hk][m, grp].astype(bool) & legal).sum()) for hk in range(cfg.Hk))
    assert st["rho_pairs"] == pytest.approx(int8_pairs / (int(legal.sum()) * cfg.Hk), rel=1e-12)
    # groups: legal when some pair in them is legal
    gl = np.zeros((cfg.T_m, cfg.T_mask), dtype=bool)
    gl[m[legal], grp[legal]] = True
    int8_groups = sum(int((R[hk].astype(bool) & gl).sum()) for hk in range(cfg.Hk))
    assert st["rho_hat"] == pytest.approx(int8_groups / (int(gl.sum()) * cfg.Hk), rel=1e-12)
    assert not (R.astype(bool) & ~gl[None]).any()   # illegal groups are never routed
    for kind, want in (("all_fp16", 0.0), ("all_int8", 1.0)):
        assert route_stats(cfg, route_map(cfg, MaskSpec(kind)))["rho_pairs"] == want
