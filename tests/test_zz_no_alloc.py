"""GPU: tilemix_prefill_noalloc, the entry point for callers that cannot allocate, against
tilemix_prefill on the same inputs (bitwise), on consecutive calls of decreasing size that
share the library's per-GPU scratch array."""

import numpy as np
import pytest

from gpu_util import log, to_dev
from synth import MaskSpec, WORKLOADS, make_qkv, make_route_bits, small_workload

pytestmark = pytest.mark.gpu


def _case(cfg, mask_index=0):
    import torch
    import paper_2608_17336_amd as tm
    mask = cfg.masks[mask_index]
    Q, K, V = make_qkv(cfg)
    words, _ = make_route_bits(cfg, mask, mask_index)
    q, k, v, w = to_dev(Q), to_dev(K), to_dev(V), to_dev(words)
    kw = dict(group_size=cfg.group_size, tile=(cfg.block_m, cfg.block_n), causal=cfg.causal,
              scale=cfg.scale)
    O_ref = tm.tilemix_prefill(q, k, v, w, **kw)
    O = torch.full_like(O_ref, float("nan"))
    tm.tilemix_prefill_noalloc(q, k, v, w, O=O, **kw)
    torch.cuda.synchronize()
    return bool(torch.equal(O.view(torch.int16), O_ref.view(torch.int16)))


def test_prefill_noalloc_matches_prefill():
    import paper_2608_17336_amd as tm
    big = WORKLOADS["32k-gqa"]                   # the benchmark workload: 101 MB of workspace
    p = tm.Params(big.B, big.Hq, big.Hk, big.L, big.L, big.d, big.block_m, big.block_n,
                  big.group_size, True, big.scale)
    assert tm.tilemix_workspace_size(p) <= tm.NOALLOC_SCRATCH_BYTES
    cases = [("32k-gqa", big),
             ("L=1000 g=2", small_workload("na1", B=2, Hq=8, Hk=2, d=128, L=1000, group_size=2,
                                           k_outliers=True, mask=MaskSpec("bernoulli", 0.5),
                                           index=1400)),
             ("L=333 d=64 bm=64", small_workload("na2", B=1, Hq=4, Hk=4, d=64, L=333, block_m=64,
                                                 mask=MaskSpec("all_int8"), index=1401))]
    for name, cfg in cases:
        log(f"noalloc {name}")
        assert _case(cfg), name
