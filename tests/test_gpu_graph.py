"""GPU: the library's calls captured in a HIP graph (torch.cuda.CUDAGraph on ROCm) and replayed.

A call validates on the host and then only enqueues kernels on the caller's stream: it
allocates nothing, clears nothing with a memset and never synchronizes.  A graph captured
from a call must therefore reproduce the eager result bit for bit on every replay, with the
program's own eager work and synchronizations between the replays (the output is overwritten
with NaN before each replay, so a replay that wrote nothing would show).
"""

import numpy as np
import pytest

from gpu_util import log, to_dev
from synth import MaskSpec, make_qkv, make_route_bits, small_workload, decode_route_bits

pytestmark = pytest.mark.gpu

REPLAYS = 3


def _check_graph(name, call, O, O_ref):
    """Capture call() (which writes O) once, replay it REPLAYS times against O_ref."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # warm-up off the default stream, as capture requires
        call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    assert torch.equal(O.view(torch.int16), O_ref.view(torch.int16)), f"{name}: eager on a side stream"
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    torch.cuda.synchronize()
    for r in range(REPLAYS):
        O.fill_(float("nan"))
        noise = torch.randn(1 << 20, device=O.device)   # unrelated eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        del noise
        ok = torch.equal(O.view(torch.int16), O_ref.view(torch.int16))
        log(f"graph {name}: replay {r} bitwise equal to eager: {ok}")
        assert ok, (name, r)


def _prefill_inputs(cfg):
    mask = cfg.masks[0]
    Q, K, V = make_qkv(cfg)
    words, _ = make_route_bits(cfg, mask, 0)
    kw = dict(group_size=cfg.group_size, tile=(cfg.block_m, cfg.block_n), causal=cfg.causal,
              scale=cfg.scale)
    return to_dev(Q), to_dev(K), to_dev(V), to_dev(words), kw


CFG = dict(B=2, Hq=8, Hk=2, d=128, L=1000, group_size=2, k_outliers=True,
           mask=MaskSpec("bernoulli", 0.5))


def test_prefill_graph_replays():
    """tilemix_prefill (quantize-once), its fused mode and the no-allocation entry point."""
    import torch
    import paper_2608_17336_amd as tm
    cfg = small_workload("graph", index=1500, **CFG)
    q, k, v, w, kw = _prefill_inputs(cfg)
    p = tm.Params(cfg.B, cfg.Hq, cfg.Hk, cfg.L, cfg.L, cfg.d, cfg.block_m, cfg.block_n,
                  cfg.group_size, True, cfg.scale)
    O_ref = tm.tilemix_prefill(q, k, v, w, **kw)
    torch.cuda.synchronize()

    ws = torch.empty(tm.tilemix_workspace_size(p), dtype=torch.uint8, device=q.device)
    O = torch.empty_like(O_ref)
    _check_graph("prefill", lambda: tm.tilemix_prefill(
        q, k, v, w, O=O, workspace=ws, stream=torch.cuda.current_stream(), **kw), O, O_ref)

    wsf = torch.empty(tm.tilemix_fused_workspace_size(p), dtype=torch.uint8, device=q.device)
    Of = torch.empty_like(O_ref)
    _check_graph("prefill_fused", lambda: tm.tilemix_prefill_fused(
        q, k, v, w, O=Of, workspace=wsf, stream=torch.cuda.current_stream(), **kw), Of, O_ref)

    On = torch.empty_like(O_ref)
    _check_graph("prefill_noalloc", lambda: tm.tilemix_prefill_noalloc(
        q, k, v, w, O=On, stream=torch.cuda.current_stream(), **kw), On, O_ref)


def test_varlen_graph_replays():
    """tilemix_prefill_varlen: the sequence table is built on the device inside the call."""
    import torch
    import paper_2608_17336_amd as tm
    lens = [700, 1, 0, 333]
    cfg = small_workload("graphvl", B=1, Hq=4, Hk=2, d=128, L=max(lens), group_size=1,
                         mask=MaskSpec("bernoulli", 0.5), index=1501)
    qs, ks, vs, rows = [], [], [], []
    Lmax = max(lens)
    p = tm.Params(len(lens), cfg.Hq, cfg.Hk, Lmax, Lmax, cfg.d, cfg.block_m, cfg.block_n,
                  cfg.group_size, True, cfg.scale)
    W = tm.tilemix_route_words_per_row(p)
    for i, L in enumerate(lens):
        c = cfg.with_(L=max(L, 1), index=cfg.index * 100 + i)
        Q, K, V = make_qkv(c)
        Q, K, V = Q[:, :L], K[:, :L], V[:, :L]
        words, _ = make_route_bits(c, c.masks[0], 0)
        T_m = -(-L // cfg.block_m)
        full = np.zeros((cfg.Hk, T_m, W), np.uint64)
        full[..., :words.shape[-1]] = words[0][:, :T_m]
        qs.append(Q[0]); ks.append(K[0]); vs.append(V[0]); rows.append(full.transpose(1, 0, 2))
    q, k, v = to_dev(np.concatenate(qs)), to_dev(np.concatenate(ks)), to_dev(np.concatenate(vs))
    w = to_dev(np.concatenate(rows))
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32, device=q.device)
    args = (q, k, v, cu, cu, Lmax, Lmax, w, cfg.group_size, (cfg.block_m, cfg.block_n), True,
            cfg.scale)
    O_ref = tm.tilemix_prefill_varlen(*args)
    torch.cuda.synchronize()
    ws = torch.empty(tm.tilemix_varlen_workspace_size(p, sum(lens), sum(lens)), dtype=torch.uint8,
                     device=q.device)
    O = torch.empty_like(O_ref)
    _check_graph("prefill_varlen", lambda: tm.tilemix_prefill_varlen(
        *args, O=O, workspace=ws, stream=torch.cuda.current_stream()), O, O_ref)


def test_decode_graph_replays():
    """tilemix_decode: the split-K partial kernel and the combine kernel in one graph."""
    import torch
    import paper_2608_17336_amd as tm
    cfg = small_workload("graphdec", B=2, Hq=16, Hk=2, d=128, L=5000, group_size=4,
                         k_outliers=True, mask=MaskSpec("bernoulli", 0.5), index=1502)
    Q, K, V = make_qkv(cfg)
    q1, k, v = to_dev(np.ascontiguousarray(Q[:, -1:])), to_dev(K), to_dev(V)
    K8, dK, V8, dV = tm.tilemix_quantize_kv(k, v)
    words, _ = decode_route_bits(cfg, cfg.masks[0])
    w = to_dev(words)
    O_ref = tm.tilemix_decode(q1, k, K8, dK, V8, dV, w, cfg.group_size, cfg.scale)
    torch.cuda.synchronize()
    p = tm.Params(cfg.B, cfg.Hq, cfg.Hk, 1, cfg.L, cfg.d, cfg.block_m, cfg.block_n,
                  cfg.group_size, True, cfg.scale)
    ws = torch.empty(tm.tilemix_decode_workspace_size(p), dtype=torch.uint8, device=q1.device)
    O = torch.empty_like(O_ref)
    _check_graph("decode", lambda: tm.tilemix_decode(
        q1, k, K8, dK, V8, dV, w, cfg.group_size, cfg.scale, O=O, workspace=ws,
        stream=torch.cuda.current_stream()), O, O_ref)
