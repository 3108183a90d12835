"""Helpers for the GPU tests: device transfer, one routed prefill call, parity metrics."""

from __future__ import annotations

import sys

import numpy as np

MAX_ABS = 2e-3     # fp16 output vs float64 oracle
REL_L2 = 1e-3


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(a: np.ndarray):
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint64:
        a = a.view(np.int64)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to("cuda:0")


def prefill(cfg, Q, K, V, words, *, route_hint=-1, dev_inputs=None, route_per_batch=False):
    import paper_2608_17336_amd as tm
    import torch
    q, k, v = dev_inputs if dev_inputs is not None else (to_dev(Q), to_dev(K), to_dev(V))
    O = tm.tilemix_prefill(q, k, v, to_dev(words), cfg.group_size, (cfg.block_m, cfg.block_n),
                           cfg.causal, cfg.scale, route_hint=route_hint,
                           route_per_batch=route_per_batch)
    torch.cuda.synchronize()
    return O


def compare_rows(O_dev, rows, ref):
    """max-abs and rel-L2 of the GPU output against oracle rows [(b, h, idx)] -> arrays."""
    import torch
    num = den = 0.0
    mx = 0.0
    for (b, h, idx), r in zip(rows, ref):
        g = O_dev[b, torch.as_tensor(idx, device=O_dev.device), h, :].float().cpu().numpy().astype(np.float64)
        diff = g - r
        mx = max(mx, float(np.max(np.abs(diff))) if diff.size else 0.0)
        num += float(np.sum(diff * diff))
        den += float(np.sum(r * r))
    rel = (num / den) ** 0.5 if den > 0 else (0.0 if num == 0 else float("inf"))
    return mx, rel
