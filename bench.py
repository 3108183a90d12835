"""Benchmark: TileMix routed prefill attention on one MI355X.

One step = one whole pass of the hot path on one batch of synthetic input: the operand
preparation (the quantize-once pass over the keys + the V tile layout) followed by the fused
routed attention kernel, which quantizes each 128-row query block in its prologue; exactly what
tilemix_prefill enqueues.  Inputs are resident in HBM before the timed region starts.

Prints one JSON line (rank 0).  Extra per-run detail goes to stderr.

Default workload: 32k-gqa (B=1, 32/8 heads, d=128, L=32768, causal, tile 128x64, g=4,
Bernoulli(0.75) INT8 routing, K outlier channels).
"""

from __future__ import annotations

import argparse
import hashlib
import statistics
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "prefill attention ms + effective TFLOP/s at 32K ctx; % of MFMA roofline"
P16 = 2.5e15   # MI355X dense FP16 matrix peak, FLOP/s (published)
P8 = 5.0e15    # MI355X dense INT8 matrix peak, OP/s (published)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def flop_model(cfg, rho_pairs):
    """Algorithmic work of one pass: legal pairs only (causal triangle)."""
    pairs = cfg.legal_pairs()
    d = cfg.d
    qk = 2.0 * d * pairs
    pv = 2.0 * d * pairs
    qk8 = qk * rho_pairs
    qk16 = qk - qk8
    t_star = qk16 / P16 + qk8 / P8 + pv / P16
    total = qk + pv
    return {"pairs": pairs, "flops": total, "flops_fp16": qk16 + pv, "flops_int8": qk8,
            "t_star_s": t_star, "weighted_peak": total / t_star}


def kernel_source_digest(source="attn_fwd.hip"):
    """SHA-256 of a kernel source file: HBM traffic counters belong to one build."""
    path = os.path.join(ROOT, "paper_2608_17336_amd", "csrc", source)
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def recorded_traffic(profile, mask_label, source="attn_fwd.hip"):
    """HBM bytes per launch (per step for decode) from the committed counter summary
    profiles/<profile>_hbm_traffic.md, or None when there is none, or it was taken with another
    routing mask or on a different kernel source."""
    path = os.path.join(ROOT, "profiles", f"{profile}_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            m = re.match(r"^- (\w+): `([^`]*)`", line.strip())
            if m:
                fields[m.group(1)] = m.group(2)
    if fields.get("mask") != mask_label:
        return None
    if fields.get("kernel_source_sha256") != kernel_source_digest(source):
        return None
    try:
        return int(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def copy_calibration(dev):
    """One plain 256 MiB device-to-device copy: HBM counters on it give the scale factors."""
    import torch

    a = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()
    del a, b


def host_cpu():
    """(logical cores of the host, CPU model name)."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    return os.cpu_count() or 1, model


def cpu_baseline(cfg, Q, K, V, words, budget_rows=None):
    """Time the CPU oracle on a bounded, strided sample of query rows of one head."""
    import numpy as np
    from oracle import routed_attention_rows
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    n_cpu, model = host_cpu()
    stride = 3   # about 11k rows of one head: 10-20 s of oracle work on a server host
    idx = np.arange(stride // 2, cfg.L, stride, dtype=np.int64)
    if budget_rows:
        idx = idx[:budget_rows]
    rows = [(0, 0, idx)]
    pairs = int(np.sum(np.minimum(idx + 1, cfg.L))) if cfg.causal else idx.size * cfg.L
    t0 = time.perf_counter()
    routed_attention_rows(Q, K, V, words, block_m=cfg.block_m, block_n=cfg.block_n,
                          group_size=cfg.group_size, causal=cfg.causal, scale=cfg.scale, rows=rows)
    dt = time.perf_counter() - t0
    flops = 4.0 * cfg.d * pairs
    full = dt * cfg.legal_pairs() / pairs
    return {
        "value": flops / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "host_cores": int(n_cpu),
        "cpu_model": model,
        "kind": "oracle",
        "sample": (f"{idx.size} query rows (one in {stride}) of head 0 of {cfg.name}, "
                   f"{pairs} legal pairs incl. the oracle's own quantization of that head, "
                   f"{dt:.1f} s on {threads} BLAS threads of a {n_cpu}-core host ({model}); "
                   f"full pass extrapolates to {full / 3600:.1f} h"),
        "seconds": dt,
    }


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="32k-gqa")
    ap.add_argument("--mask", type=int, default=0, help="index into the workload's masks")
    ap.add_argument("--template", default="",
                    help="route with a routing template of the library instead of the workload's "
                         "mask: KIND[:RHO] (KIND one of one, zero, band, global, rowrand, aligned, "
                         "bigbird, sptrans; RHO the INT8 coverage to fit, default 0.75)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=0, help="cap on oracle rows (0 = default sample)")
    ap.add_argument("--varlen", default="",
                    help="time a packed variable-length batch instead: comma-separated sequence "
                         "lengths (the workload's heads, d, tile, g, mask kind and seed)")
    ap.add_argument("--decode", action="store_true",
                    help="time one decode step over an INT8 key/value cache of the workload's "
                         "shape (L_k = L, one query token per sequence)")
    ap.add_argument("--fused", action="store_true",
                    help="time the fused on-the-fly operand mode (tilemix_prefill_fused: no Q8/K8 "
                         "scratch, quantization on chip) instead of quantize-once")
    ap.add_argument("--no-deviation", action="store_true",
                    help="skip the untimed all-FP16 launch behind deviation_vs_fp16, so that a kernel "
                         "trace holds the timed launches only")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one plain 256 MiB device copy (HBM counter calibration)")
    args = ap.parse_args(argv)

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "bench.py runs on exactly one GPU; the routed attention "
                                   "path shards by (batch, KV head) with no communication, "
                                   "but multi-GPU runs are not part of it", "n_gpus": args.gpus}))
        return 2

    import numpy as np
    import torch

    import paper_2608_17336_amd as tm
    from synth import WORKLOADS, make_qkv, make_route_bits, route_stats

    cfg = WORKLOADS[args.config]
    mask = cfg.masks[args.mask]
    dev = torch.device("cuda:0")
    tm.load_library()
    if args.varlen:
        return bench_varlen(args, cfg, mask)
    if args.decode:
        return bench_decode(args, cfg, mask)

    t0 = time.perf_counter()
    Q, K, V = make_qkv(cfg)
    mask_label = mask.label
    mask_kind = mask.kind
    if args.template:
        kind, _, rho = args.template.partition(":")
        rho = float(rho) if rho else 0.75
        tp = tm.Params(cfg.B, cfg.Hq, cfg.Hk, cfg.L, cfg.L, cfg.d, cfg.block_m, cfg.block_n,
                       cfg.group_size, cfg.causal, cfg.scale)
        # SpTrans: a stride of about sqrt(T_mask) whole key groups
        span = cfg.group_size * cfg.block_n
        stride = span * max(1, int(round(math.sqrt(cfg.T_mask))))
        tmpl = tm.tilemix_fit_template(tp, tm.Template(kind, sp_stride=stride, seed=cfg.seed), rho)
        words = tm.tilemix_route_template(tp, tmpl)
        rho_g, rho_p = tm.tilemix_route_coverage(tp, words)
        stats = {"rho_hat": rho_g, "rho_pairs": rho_p}
        mask_label = f"template:{kind}@{rho:g}"
        mask_kind = "all_fp16" if kind == "zero" else kind
        log(f"[bench] template {tmpl}")
    else:
        words, R = make_route_bits(cfg, mask, args.mask)
        stats = route_stats(cfg, R)
    log(f"[bench] inputs for {cfg.name} mask={mask_label} generated in {time.perf_counter() - t0:.1f}s; "
        f"rho_hat={stats['rho_hat']:.4f} rho_pairs={stats['rho_pairs']:.4f}")
    to = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    q, k, v = to(Q), to(K), to(V)
    w = to(words.view(np.int64))
    hint = 0 if mask_kind == "all_fp16" else -1
    kw = dict(group_size=cfg.group_size, tile=(cfg.block_m, cfg.block_n), causal=cfg.causal,
              scale=cfg.scale, route_hint=hint)
    p = tm.Params(cfg.B, cfg.Hq, cfg.Hk, cfg.L, cfg.L, cfg.d, cfg.block_m, cfg.block_n,
                  cfg.group_size, cfg.causal, cfg.scale, False, hint)
    ws_bytes = tm.tilemix_fused_workspace_size(p) if args.fused else tm.tilemix_workspace_size(p)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    O = torch.empty((cfg.B, cfg.L, cfg.Hq, cfg.d), dtype=torch.float16, device=dev)
    stream = torch.cuda.current_stream()

    def step(e0=None, e1=None, e2=None):
        if e0 is not None:
            e0.record(stream)
        if args.fused:   # one call: V tiles, then the kernel that quantizes on chip
            if e1 is not None:
                e1.record(stream)
            tm.tilemix_prefill_fused(q, k, v, w, workspace=ws, O=O, stream=stream, **kw)
        else:
            tm.tilemix_prepare(q, k, v, workspace=ws, stream=stream, **kw)
            if e1 is not None:
                e1.record(stream)
            tm.tilemix_attend(q, k, w, ws, O=O, stream=stream, **kw)
        if e2 is not None:
            e2.record(stream)

    if args.copy_calibration:
        copy_calibration(dev)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"[bench] warmup done ({args.warmup} steps)")

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        step(*evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    step_ms = [e0.elapsed_time(e2) for e0, _, e2 in evs]
    prep_ms = [e0.elapsed_time(e1) for e0, e1, _ in evs]
    attn_ms = [e1.elapsed_time(e2) for _, e1, e2 in evs]
    ms_per_step = wall * 1e3 / args.steps
    attn_avg = sum(attn_ms) / len(attn_ms)
    prep_avg = sum(prep_ms) / len(prep_ms)
    log(f"[bench] {args.steps} steps: wall {ms_per_step:.3f} ms/step, events step {sum(step_ms)/len(step_ms):.3f} "
        f"(prep {prep_avg:.3f}, attention {attn_avg:.3f}; attention min {min(attn_ms):.3f} max {max(attn_ms):.3f})")

    # Deviation of the routed output from exact attention: the same kernel with every tile on
    # the FP16 route (untimed).
    deviation = None if args.no_deviation else deviation_vs_fp16(args, cfg, tm, q, k, v, w, ws, O,
                                                                 kw, stream)
    fm = flop_model(cfg, stats["rho_pairs"])
    eff = fm["flops"] / (ms_per_step * 1e-3) / 1e12
    achieved = fm["flops"] / (attn_avg * 1e-3) / 1e12
    peak = fm["weighted_peak"] / 1e12
    line = {
        "metric": METRIC,
        "value": round(eff, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16+i8",
        "data": "synthetic",
        "config": {"workload": cfg.name, "B": cfg.B, "Hq": cfg.Hq, "Hk": cfg.Hk, "d": cfg.d,
                   "L": cfg.L, "causal": cfg.causal, "tile": f"{cfg.block_m}x{cfg.block_n}",
                   "group_size": cfg.group_size, "mask": mask_label,
                   "operands": "fused on-the-fly" if args.fused else "quantize-once",
                   "rho_hat": round(stats["rho_hat"], 4), "rho_pairs": round(stats["rho_pairs"], 4)},
        "pct_of_weighted_roofline": round(100.0 * fm["t_star_s"] / (ms_per_step * 1e-3), 2),
        "attention_ms": round(attn_avg, 4),
        "deviation_vs_fp16": (None if deviation is None else
                              {k2: float(f"{v2:.4e}") for k2, v2 in deviation.items()}),
        "prepare_ms": round(prep_avg, 4),
        "timing_ms": {"step_median": round(statistics.median(step_ms), 4),
                      "step_min": round(min(step_ms), 4),
                      "attention_median": round(statistics.median(attn_ms), 4),
                      "attention_min": round(min(attn_ms), 4)},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": round(peak, 2),
                     "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                     "traffic": None if args.fused else recorded_traffic(f"routed_attn_fwd_{cfg.name}", mask_label),
                     "kernel": (f"v_tiles_kernel + routed_attn_fwd_kernel<{cfg.d}, {cfg.block_m}, 1, true>"
                                if args.fused else f"routed_attn_fwd_kernel<{cfg.d}, {cfg.block_m}, 1>"),
                     "peak_note": "precision-weighted: QK^T FP16 share at 2.5 PFLOP/s, INT8 share at "
                                  "5.0 POP/s, P.V at 2.5 PFLOP/s"},
    }
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample")
        cb = cpu_baseline(cfg, Q, K, V, words, args.cpu_rows or None)
        cb.pop("seconds")
        line["cpu_baseline"] = cb
    print(json.dumps(line), flush=True)
    return 0


def deviation_vs_fp16(args, cfg, tm, q, k, v, w, ws, O, kw, stream):
    """max-abs, mean-abs and rel-L2 of the routed O against the same kernel with every tile on
    the FP16 route, i.e. exact attention (one untimed launch)."""
    import math
    import torch
    O16 = torch.empty_like(O)
    kw16 = dict(kw, route_hint=0)
    if args.fused:
        tm.tilemix_prefill_fused(q, k, v, w, workspace=ws, O=O16, stream=stream, **kw16)
    else:
        tm.tilemix_prepare(q, k, v, workspace=ws, stream=stream, **kw16)
        tm.tilemix_attend(q, k, w, ws, O=O16, stream=stream, **kw16)
    torch.cuda.synchronize()
    ss = sa = ref = 0.0
    mx = 0.0
    for b0 in range(cfg.B):                      # per sequence, to bound the float copies
        d = O[b0].float() - O16[b0].float()
        mx = max(mx, d.abs().max().item())
        sa += d.abs().sum().item()
        ss += (d * d).sum().item()
        ref += (O16[b0].float() ** 2).sum().item()
    deviation = {"max_abs": mx, "mean_abs": sa / O.numel(),
                 "rel_l2": math.sqrt(ss / ref) if ref > 0 else 0.0}
    log(f"[bench] routed vs all-FP16 output: max_abs {mx:.3e} mean_abs {deviation['mean_abs']:.3e} "
        f"rel_l2 {deviation['rel_l2']:.3e}")
    return deviation


def bench_decode(args, cfg, mask):
    """One step = tilemix_decode: each sequence's newest token against an INT8 key/value cache
    of L keys (K8 + V8 + scales, and the FP16 key cache for FP16-routed groups).  HBM-bound:
    the roofline is algorithmic bytes (cache bytes each routed key needs) per launch time."""
    import numpy as np
    import torch

    import paper_2608_17336_amd as tm
    from synth import make_qkv

    dev = torch.device("cuda:0")
    Q, K, V = make_qkv(cfg)
    to = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    q1, k, v = to(Q[:, -1:]), to(K), to(V)
    del Q
    K8, dK, V8, dV = tm.tilemix_quantize_kv(k, v)
    from synth import decode_route_bits
    words, R = decode_route_bits(cfg, mask)
    w = to(words.view(np.int64))
    hint = 0 if mask.kind == "all_fp16" else -1
    p = tm.Params(cfg.B, cfg.Hq, cfg.Hk, 1, cfg.L, cfg.d, cfg.block_m, cfg.block_n,
                  cfg.group_size, True, cfg.scale, False, hint)
    ws = torch.empty(tm.tilemix_decode_workspace_size(p), dtype=torch.uint8, device=dev)
    O = torch.empty_like(q1)
    stream = torch.cuda.current_stream()
    run = lambda: tm.tilemix_decode(q1, k, K8, dK, V8, dV, w, cfg.group_size, cfg.scale, O=O,
                                    workspace=ws, stream=stream, route_hint=hint)
    if args.copy_calibration:
        copy_calibration(dev)
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / args.steps
    ms = e0.elapsed_time(e1) / args.steps
    # algorithmic bytes: per KV head and key, d (K8) or 2d (FP16 K) by route, plus d (V8)
    keys = np.arange(cfg.L)
    bits = R[:, 0, (keys // cfg.block_n) // cfg.group_size].astype(np.int64)   # [Hk, L]
    kbytes = float(np.where(bits == 1, cfg.d, 2 * cfg.d).sum()) * cfg.B
    vbytes = float(cfg.d) * cfg.L * cfg.Hk * cfg.B
    nkb = -(-cfg.L // 64)
    sbytes = 2.0 * 2 * nkb * cfg.Hk * cfg.B
    qo = 2.0 * 2 * cfg.B * cfg.Hq * cfg.d
    nbytes = kbytes + vbytes + sbytes + qo
    gbs = nbytes / (ms * 1e-3) / 1e9
    line = {
        "metric": "decode step ms over an INT8 key/value cache; % of HBM roofline",
        "value": round(ms, 4), "unit": "ms", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(wall, 4), "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None, "dtype": "i8+f16", "data": "synthetic",
        "config": {"workload": f"decode-{cfg.name}", "B": cfg.B, "Hq": cfg.Hq, "Hk": cfg.Hk,
                   "d": cfg.d, "L_k": cfg.L, "group_size": cfg.group_size, "mask": mask.label,
                   "int8_key_share": round(float(bits.mean()), 4)},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": 8000.0, "unit": "GB/s",
                     "frac": round(gbs / 8000.0, 4),
                     "traffic": recorded_traffic(f"decode_{cfg.name}", mask.label, "decode.hip"),
                     "kernel": "decode_partial_kernel + decode_combine_kernel (event-timed step)"},
    }
    print(json.dumps(line), flush=True)
    return 0


def bench_varlen(args, cfg, mask):
    """One step = tilemix_prefill_varlen over a packed batch of the given sequence lengths
    (sequence table, key quantization, V tiles and the attention kernel), causal, with the
    workload's heads, head size, tile, group size and routing mask kind drawn per sequence.
    With --fused: tilemix_prefill_varlen_fused (no key quantization pass; codes made on chip)."""
    import numpy as np
    import torch

    import paper_2608_17336_amd as tm
    from synth import make_qkv, make_route_bits, route_stats

    lens = [int(x) for x in args.varlen.split(",") if x]
    dev = torch.device("cuda:0")
    qs, ks, vs, rows, pairs, int8_pairs = [], [], [], [], 0, 0.0
    Lmax = max(lens)
    p = tm.Params(len(lens), cfg.Hq, cfg.Hk, Lmax, Lmax, cfg.d, cfg.block_m, cfg.block_n,
                  cfg.group_size, True, cfg.scale)
    W = tm.tilemix_route_words_per_row(p)
    for i, L in enumerate(lens):
        c = cfg.with_(B=1, L=L, index=cfg.index * 1000 + i)
        Q, K, V = make_qkv(c)
        words, R = make_route_bits(c, mask, args.mask)
        st = route_stats(c, R)
        pairs += c.legal_pairs()
        int8_pairs += c.legal_pairs() * st["rho_pairs"]
        full = np.zeros((c.Hk, c.T_m, W), np.uint64)
        full[..., :words.shape[-1]] = words[0]
        qs.append(Q[0]); ks.append(K[0]); vs.append(V[0]); rows.append(full.transpose(1, 0, 2))
    to = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    q, k, v = to(np.concatenate(qs)), to(np.concatenate(ks)), to(np.concatenate(vs))
    w = to(np.concatenate(rows).view(np.int64))
    cu = to(np.concatenate([[0], np.cumsum(lens)]).astype(np.int32))
    hint = 0 if mask.kind == "all_fp16" else -1
    size = tm.tilemix_varlen_fused_workspace_size if args.fused else tm.tilemix_varlen_workspace_size
    ws = torch.empty(size(p, sum(lens), sum(lens)), dtype=torch.uint8, device=dev)
    O = torch.empty_like(q)
    stream = torch.cuda.current_stream()
    entry = tm.tilemix_prefill_varlen_fused if args.fused else tm.tilemix_prefill_varlen
    run = lambda: entry(q, k, v, cu, cu, Lmax, Lmax, w, cfg.group_size, (cfg.block_m, cfg.block_n),
                        True, cfg.scale, O=O, workspace=ws, stream=stream, route_hint=hint)
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / args.steps
    ms = e0.elapsed_time(e1) / args.steps
    rho = int8_pairs / pairs
    flops = 4.0 * cfg.d * pairs
    t_star = (2.0 * cfg.d * pairs * (1 - rho)) / P16 + (2.0 * cfg.d * pairs * rho) / P8 + 2.0 * cfg.d * pairs / P16
    line = {
        "metric": METRIC + " (variable-length batch)",
        "value": round(flops / (wall * 1e-3) / 1e12, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(wall, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f16+i8",
        "data": "synthetic",
        "config": {"workload": f"varlen-{cfg.name}", "lens": lens, "Hq": cfg.Hq, "Hk": cfg.Hk,
                   "d": cfg.d, "tile": f"{cfg.block_m}x{cfg.block_n}", "group_size": cfg.group_size,
                   "mask": mask.label, "rho_pairs": round(rho, 4),
                   "operands": "fused on-the-fly" if args.fused else "quantize-once"},
        "step_ms_events": round(ms, 4),
        "pct_of_weighted_roofline": round(100.0 * t_star / (wall * 1e-3), 2),
        # one call enqueues the sequence table, the key quantization, the V tiles and the kernel,
        # so the achieved rate is over the whole event-timed call
        "roofline": {"bound": "mfma", "achieved": round(flops / (ms * 1e-3) / 1e12, 2),
                     "peak": round(flops / t_star / 1e12, 2), "unit": "TFLOP/s",
                     "frac": round(t_star / (ms * 1e-3), 4), "traffic": None,
                     "kernel": (f"tilemix_prefill_varlen_fused (seq table, V tiles, "
                                f"routed_attn_fwd_kernel<{cfg.d}, {cfg.block_m}, 1, true>)" if args.fused else
                                f"tilemix_prefill_varlen (seq table, K quantization, V tiles, "
                                f"routed_attn_fwd_kernel<{cfg.d}, {cfg.block_m}, 1>)")},
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
