"""Pins for oracle/routing.py (Section 4.2: grouping, packed words, shift-and-mask lookup)
and for the packing done by the input generator."""

import numpy as np

from oracle.routing import route_bit, route_bits_for_keys
from synth import pack_route_bits, legal_group_table, small_workload, WORKLOADS


def test_hand_packed_single_word():
    # R = [1, 1, 0, 1] -> b = 1 + 2 + 8 = 11 (Section 4.2, bitmask packing)
    words = np.array([[[[11]]]], dtype=np.uint64)
    assert [route_bit(words, 0, 0, 0, g) for g in range(6)] == [1, 1, 0, 1, 0, 0]
    R = np.array([[[1, 1, 0, 1]]], dtype=np.uint8)
    assert int(pack_route_bits(R)[0, 0, 0, 0]) == 11


def test_multi_word_rows():
    # 130 groups: group 64 -> word 1 bit 0, group 127 -> word 1 bit 63, group 129 -> word 2 bit 1
    R = np.zeros((1, 1, 130), dtype=np.uint8)
    for g in (0, 63, 64, 127, 129):
        R[0, 0, g] = 1
    w = pack_route_bits(R)
    assert w.shape == (1, 1, 1, 3)
    assert int(w[0, 0, 0, 0]) == (1 << 0) | (1 << 63)
    assert int(w[0, 0, 0, 1]) == (1 << 0) | (1 << 63)
    assert int(w[0, 0, 0, 2]) == (1 << 1)
    got = [g for g in range(130) if route_bit(w, 0, 0, 0, g)]
    assert got == [0, 63, 64, 127, 129]


def test_batch_axis_broadcast_and_per_sequence():
    w = np.zeros((2, 1, 1, 1), dtype=np.uint64)
    w[0, 0, 0, 0] = 1
    w[1, 0, 0, 0] = 2
    assert route_bit(w, 0, 0, 0, 0) == 1 and route_bit(w, 1, 0, 0, 0) == 0
    assert route_bit(w, 1, 0, 0, 1) == 1
    shared = w[:1]
    assert route_bit(shared, 1, 0, 0, 0) == 1     # one map for the whole batch


def test_key_to_group_mapping_bruteforce():
    rng = np.random.default_rng(3)
    block_m, block_n, g = 3, 5, 3
    Lk = 97
    T_n = -(-Lk // block_n)
    T_mask = -(-T_n // g)
    R = rng.integers(0, 2, size=(2, 4, T_mask)).astype(np.uint8)
    words = pack_route_bits(R)
    keys = np.arange(Lk)
    for h_k in range(2):
        for i in range(12):
            m = i // block_m
            got = route_bits_for_keys(words, 0, h_k, i, keys, block_m, block_n, g)
            want = [int(R[h_k, m, (j // block_n) // g]) for j in keys]
            assert list(got) == want


def test_legal_group_counts_closed_form():
    # causal, L_q = L_k: row m (BLOCK_M rows) reaches key (m+1)*BLOCK_M - 1, so with
    # group span S = g * BLOCK_N the legal groups of row m number ceil((m+1)*BLOCK_M / S)
    expect = {"1k-mha-d64": 136, "8k-gqa": 4160, "32k-gqa": 16512, "128k-gqa": 66048,
              "64k-b4-gqa": 33024}
    for name, want in expect.items():
        cfg = WORKLOADS[name]
        S = cfg.group_size * cfg.block_n
        closed = sum(-(-min(cfg.L, (m + 1) * cfg.block_m) // S) for m in range(cfg.T_m))
        assert closed == want
        assert int(legal_group_table(cfg).sum()) == want


def test_legal_groups_ragged_noncausal():
    cfg = small_workload("t", L=300, block_m=128, block_n=64, group_size=2, causal=False)
    tab = legal_group_table(cfg)
    assert tab.shape == (3, 3) and tab.all()
    cfg = small_workload("t", L=300, block_m=128, block_n=64, group_size=2, causal=True)
    tab = legal_group_table(cfg)
    # row 0 (queries 0..127): groups of 128 keys: only group 0; row 2 (256..299): all 3
    assert tab.tolist() == [[True, False, False], [True, True, False], [True, True, True]]
