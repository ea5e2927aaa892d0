#!/usr/bin/env python3
"""Decode benchmark of the offloaded-MoE hot path on one MI355X.

A step is one decode token of batch 1 through the whole hot path of every
layer of the workload: router (softmax, top-K), adapter priorities for the
next layer, window-aware prefetch of the next layer's experts, on-demand loads
of missing experts, and the routed-expert SwiGLU FFN over the HBM slot cache.
Expert weights live in pinned host memory (the offload tier); the layer-0
hidden states of all steps are resident in HBM before the timed region.

Prints one JSON line (rank 0, N = 1).  Multi-GPU runs are not part of this
build: the path runs on one GPU.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decode tokens/s with offloaded experts; next-layer coverage; exposed-transfer %"
HBM_PEAK_GBS = 8000.0


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


def measured_traffic(profile: str, kernel_source: str):
    """HBM bytes per launch from the committed counter summary, or None when the
    kernel source changed since the counters were taken."""
    import hashlib
    try:
        fields = dict(line.split(": ", 1) for line in open(profile).read().splitlines() if ": " in line)
        digest = hashlib.sha256(open(kernel_source, "rb").read()).hexdigest()[:16]
        if fields.get("kernel_source_sha256_16", "").strip() != digest:
            return None
        return int(fields["traffic_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def step_hbm_bytes(cfg, distinct_per_layer=None) -> int:
    """Algorithmic HBM bytes of one decode step (all layers, the batch): every
    layer's router and stand-in projection, the adapters of layers 0..L-2, and
    each expert the step routes to (K per layer at batch 1; the measured
    distinct count of a batched step) plus the shared experts, read once."""
    e = cfg.elem_bytes
    per_expert = cfg.blob_bytes
    experts = cfg.K if cfg.batch == 1 or distinct_per_layer is None else distinct_per_layer
    total = 0.0
    for l in range(cfg.L):
        total += cfg.n * cfg.D * e                                   # router
        if cfg.has_proj:
            total += cfg.D * cfg.D * e                               # stand-in projection
        if l < cfg.L - 1 and cfg.r > 0:
            total += (cfg.r * cfg.D + cfg.n * cfg.r) * e             # adapter A, B
        total += (experts + cfg.n_shared) * per_expert
    return int(round(total))


def _ffn_stats(rs):
    n = max(rs.ffn_launches, 1)
    return rs.ffn_us / n


def run_mode(stack, dev_h, row_bytes, warmup, steps, M_max, naive=False):
    """One timed run; naive: Naive Prefetch (the preceding step's experts) instead of the adapter."""
    import torch
    from paper_2607_24787_amd import spp

    cfg = stack.cfg
    base = dev_h.data_ptr()
    spp.spp_set_prefetch_source(stack.ctx, spp.PREFETCH_PREV_TOKEN if naive else spp.PREFETCH_ADAPTER)
    stack.reset()
    spp.spp_set_timing(stack.ctx, 0)
    for t in range(warmup):
        stack.decode_step_from(base + t * row_bytes, M_max)
    # pass 1, uninstrumented: the throughput (and the host timers, which cost nothing)
    torch.cuda.synchronize()
    spp.spp_reset_run_stats(stack.ctx)
    t0 = time.perf_counter()
    for t in range(warmup, warmup + steps):
        stack.decode_step_from(base + t * row_bytes, M_max)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    rs1 = spp.spp_get_run_stats(stack.ctx)
    # pass 2, the next `steps` tokens with HIP events on: coverage, exposed share, windows, kernel times
    spp.spp_reset_run_stats(stack.ctx)
    spp.spp_set_timing(stack.ctx, 1)
    hits_target = 0
    hits_first = 0
    distinct = 0
    t1 = time.perf_counter()
    for t in range(warmup + steps, warmup + 2 * steps):
        out = stack.decode_step_from(base + t * row_bytes, M_max)
        hits_first += out[0][2].token_hits
        for l in range(1, cfg.L):
            hits_target += out[l][2].token_hits
        for l in range(cfg.L):
            distinct += out[l][2].hits + out[l][2].misses
    torch.cuda.synchronize()
    wall_timed = time.perf_counter() - t1
    rs = spp.spp_get_run_stats(stack.ctx)
    lt = spp.spp_get_layer_times(stack.ctx, cfg.L)
    spp.spp_set_timing(stack.ctx, 0)
    spp.spp_set_prefetch_source(stack.ctx, spp.PREFETCH_ADAPTER)
    demand = cfg.K * cfg.batch * steps
    return {
        "M_max": M_max,
        "policy": "naive" if naive else ("off" if M_max < 0 else "adapter"),
        "tokens_per_s": cfg.batch * steps / wall,
        "ms_per_step": 1e3 * wall / steps,
        "wall_s": wall,
        "tokens_per_s_instrumented": cfg.batch * steps / wall_timed,
        "next_layer_coverage": hits_target / (demand * max(cfg.L - 1, 1)),
        "first_layer_hit_rate": hits_first / demand,
        "exposed_transfer_pct": 100.0 * rs.exposed_us / rs.span_us if rs.span_us > 0 else None,
        "span_us": rs.span_us,
        "exposed_us": rs.exposed_us,
        "router_us_per_layer": rs.router_us / max(rs.layer_calls, 1),
        # host time per layer call in the uninstrumented pass: router launch ->
        # routing seen, routing seen -> FFN enqueued
        "host_route_us_per_layer": rs1.host_route_us / max(rs1.layer_calls, 1),
        "host_decide_us_per_layer": rs1.host_decide_us / max(rs1.layer_calls, 1),
        "ffn_kernel_us": _ffn_stats(rs),
        "ffn_launches": rs.ffn_launches,
        "misses_per_step": rs.misses / steps,
        "prefetched_per_step": rs.prefetched / steps,
        # m_l: prefetch copies issued per prediction, as fractions of the predictions
        "prefetch_count_hist": ({str(m): rs.prefetch_hist[m] / sum(rs.prefetch_hist)
                                 for m in range(17) if rs.prefetch_hist[m]} if sum(rs.prefetch_hist) else None),
        "prefetch_used_per_step": rs.prefetch_used / steps,
        "ready_on_time_frac": rs.ready_on_time / max(rs.hits + rs.misses, 1),
        "copy_bytes": rs.copy_bytes,
        "h2d_gbs_during_run": rs.copy_bytes / (rs.span_us * 1e3) if rs.span_us > 0 else None,
        "distinct_experts_per_layer": distinct / (steps * cfg.L),
        "window_us": rs.window_us / rs.window_samples if rs.window_samples else None,
        "compute_window_us": rs.compute_window_us / rs.window_samples if rs.window_samples else None,
        "combine_us_per_layer": rs.tail_us / max(rs.layer_calls, 1),
        "exposed_breakdown_pct": {
            "on_demand_loads": 100.0 * rs.exposed_load_us / rs.span_us if rs.span_us > 0 else None,
            "on_demand_loads_sharing_link_with_prefetch":
                100.0 * rs.exposed_shared_us / rs.span_us if rs.span_us > 0 else None,
            "copy_stream_waits": 100.0 * rs.exposed_wait_us / rs.span_us if rs.span_us > 0 else None},
        "layer_calls_sharing_link": rs.shared_calls,
        # per layer: exposed time / the layer's latency (its start to the next layer's start)
        "per_layer": [{"layer": l,
                       "exposed_us_per_call": float(lt["exposed_us"][l] / max(lt["calls"][l], 1)),
                       "latency_us_per_call": (float(lt["latency_us"][l] / lt["latency_calls"][l])
                                               if lt["latency_calls"][l] else None),
                       "exposed_pct": (100.0 * float(lt["exposed_us"][l] / max(lt["calls"][l], 1))
                                       / float(lt["latency_us"][l] / lt["latency_calls"][l])
                                       if lt["latency_calls"][l] and lt["latency_us"][l] > 0 else None)}
                      for l in range(cfg.L)] if cfg.L <= 4 else None,
        "ready_plus_waited_per_step": (rs.ready_on_time + rs.waited) / steps,
        "expert_recall": ({f"@{M}": rs.recall_hits[j] / (cfg.K * rs.recall_tokens)
                           for j, M in enumerate((max(cfg.K // 2, 1), cfg.K, cfg.K + 2))}
                          if rs.recall_tokens else None),
        "demand_exceeds_budget": ({f"top{M}": rs.demand_exceeds[j] / rs.pred_events
                                   for j, M in enumerate((max(cfg.K // 2, 1), cfg.K, cfg.K + 2))}
                                  if rs.pred_events else None),
        # predictions whose missing top-M experts exceed the configured window
        # (in experts), the quantity of the paper's motivating measurement
        "demand_exceeds_window": ({f"top{M}": sum(rs.demand_hist[j][cfg.window + 1:]) / rs.pred_events
                                   for j, M in enumerate((max(cfg.K // 2, 1), cfg.K, cfg.K + 2))}
                                  if rs.pred_events else None),
    }


def distill_adapters(stack, cfg, seqs: int, length: int):
    """Train every adapter by KL distillation on traces of `seqs` fresh AR(1)
    sequences of `length` tokens (same weights, other sequence streams), score
    ExpertRecall on 4 held-out sequences, and return a stack bound to the
    distilled adapters with the report."""
    import numpy as np
    from paper_2607_24787_amd import distill
    from paper_2607_24787_amd.model import OffloadedMoEStack
    from workload import gen

    t0 = time.perf_counter()
    B = cfg.batch
    pool = gen.hidden_states(cfg.with_(batch=B * (1 + seqs + 4)), tokens=length)   # [T, B*(1+seqs+4), D]
    def seq_block(first, count):   # sequences first..first+count-1 in groups of B, laid end to end in time
        blk = pool[:, B * first: B * (first + count)].reshape(length, count, B, cfg.D)
        return np.ascontiguousarray(blk.transpose(1, 0, 2, 3).reshape(count * length, B, cfg.D))
    X, Z = distill.collect_traces(stack, seq_block(1, seqs))
    Xe, Ze = distill.collect_traces(stack, seq_block(1 + seqs, 4))

    def values(a):
        a = np.asarray(a)
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32) if a.dtype == np.uint16 else a.astype(np.float32)
    adapters, report = {}, []
    for l in range(cfg.L - 1):
        A0, B0 = (values(m) for m in gen.adapter_weights(cfg, l))
        A, Bm, (k0, k1) = distill.distill_adapter(X[l], Z[l + 1], A0, B0, seed=l)
        adapters[l] = (A, Bm)
        row = {"layer": l, "kl_start": k0, "kl_end": k1}
        for M in sorted({max(1, cfg.K // 2), cfg.K, cfg.K + 2}):
            row[f"recall@{M}_svd"] = distill.expert_recall(A0, B0, Xe[l], Ze[l + 1], cfg.K, M)
            row[f"recall@{M}_distilled"] = distill.expert_recall(A, Bm, Xe[l], Ze[l + 1], cfg.K, M)
        report.append(row)
        _log(f"[bench] distill layer {l}: KL {k0:.4f} -> {k1:.4f}, held-out recall@{cfg.K} "
             f"{row[f'recall@{cfg.K}_svd']:.3f} -> {row[f'recall@{cfg.K}_distilled']:.3f}")
    stack.close()
    new = OffloadedMoEStack(cfg, adapter_values=lambda l: adapters[l])
    info = {"sequences": seqs, "tokens_per_sequence": length, "held_out_sequences": 4,
            "train_pairs_per_layer": int(X[0].shape[0]), "seconds": time.perf_counter() - t0, "layers": report}
    return new, info


def cpu_baseline(cfg, tokens: int, target_s: float = 15.0):
    """The oracle, untuned, on the host cores: decode of the first steps of the
    workload through all layers (expert weights decoded before the timed
    region).  A first pass over `tokens` steps sizes the sample: while a pass
    takes less than a third of `target_s`, the next one decodes as many steps
    as the last pass's rate puts at about `target_s` seconds (at most 20,000,
    and at most three more passes); the last pass is the sample."""
    from concurrent.futures import ThreadPoolExecutor

    import threadpoolctl

    import oracle as o
    from workload import gen

    W = o.OracleWeights(cfg, cache_experts=cfg.L * cfg.n + 8)
    with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
        list(ex.map(lambda le: W.expert(*le), [(l, e) for l in range(cfg.L) for e in range(cfg.n)]))
    for l in range(cfg.L):
        W.router(l)
        if l < cfg.L - 1:
            W.adapter(l)
    avail = len(os.sched_getaffinity(0))

    def timed(n):
        h0 = gen.hidden_states(cfg, tokens=n)
        t0 = time.perf_counter()
        o.run_decode(cfg, W, h0, M_max=cfg.window)
        return time.perf_counter() - t0

    with threadpoolctl.threadpool_limits(limits=avail, user_api="blas"):
        blas = [p.get("num_threads") for p in threadpoolctl.threadpool_info() if p.get("user_api") == "blas"]
        n = tokens
        dt = timed(n)
        for _ in range(3):
            if dt >= target_s / 3 or n >= 20000:
                break
            n = min(20000, max(n + 1, int(n * target_s / max(dt, 1e-3))))
            dt = timed(n)
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next(l.split(":", 1)[1].strip() for l in f if l.startswith("model name"))
    except (OSError, StopIteration):
        pass
    used = min(int(blas[0]), avail) if blas else 1
    return {"value": n * cfg.batch / dt, "unit": "tokens/s", "cores": used,
            "kind": "oracle", "blas_threads": int(blas[0]) if blas else None, "host_cores_available": avail,
            "cpu_model": cpu_model,
            "sample": f"first {n} decode steps of the same workload (batch {cfg.batch}, all {cfg.L} layers, "
                      f"M_max={cfg.window}), fp64 numpy with BLAS on {used} threads, expert weights decoded "
                      f"before the timed region, {dt:.1f} s"}


def stack_record(args, key: str, tie: int):
    """A whole decode stack (the 48-layer Qwen-shaped one by default; stand-in
    projection per layer, 25% of experts resident, configured window 1): decode
    tokens/s at the configured window and with prediction off, next-layer
    coverage, exposure, and the step's algorithmic HBM bytes against the 8 TB/s
    roofline.  tie > 0: the offload tier holds tie distinct expert layers,
    shared round-robin by the 48 (bounds pinned host memory and set-up time;
    routers, adapters, projections and slot pools stay per layer)."""
    import numpy as np
    import torch

    import workload
    from paper_2607_24787_amd.model import OffloadedMoEStack
    from workload import gen

    cfg = workload.get(key)
    if tie:
        cfg = cfg.with_(expert_layers=tie)
    t0 = time.perf_counter()
    h_all = gen.hidden_states(cfg, tokens=args.warmup + 2 * args.steps)
    stack = OffloadedMoEStack(cfg)
    row_bytes = cfg.batch * cfg.D * cfg.elem_bytes
    dev_h = torch.from_numpy(np.ascontiguousarray(h_all).reshape(-1).view(np.uint8).copy()).to(stack.device)
    torch.cuda.synchronize()
    _log(f"[bench] stack setup {time.perf_counter() - t0:.1f}s workload={cfg.name} (offload tier tied over {tie})")
    try:
        on = run_mode(stack, dev_h, row_bytes, args.warmup, args.steps, cfg.window)
        _log(f"[bench] stack ON  {on['tokens_per_s']:.1f} tok/s coverage={on['next_layer_coverage']:.3f} "
             f"exposed={on['exposed_transfer_pct']:.1f}%")
        off = run_mode(stack, dev_h, row_bytes, args.warmup, args.steps, -1)
        _log(f"[bench] stack OFF {off['tokens_per_s']:.1f} tok/s coverage={off['next_layer_coverage']:.3f}")
    finally:
        stack.close()
    per_token = step_hbm_bytes(cfg) / cfg.batch
    ceiling = HBM_PEAK_GBS * 1e9 / per_token
    rec = {"workload": cfg.name + (f"+expert_layers={tie}" if tie else ""), "layers": cfg.L,
           "window_experts": cfg.window, "hbm_slots_per_layer": cfg.S, "steps": args.steps, "warmup": args.warmup,
           "tokens_per_s": on["tokens_per_s"], "ms_per_step": on["ms_per_step"],
           "next_layer_coverage": on["next_layer_coverage"], "exposed_transfer_pct": on["exposed_transfer_pct"],
           "exposed_breakdown_pct": on["exposed_breakdown_pct"],
           "hbm_bytes_per_token": int(per_token), "hbm_roofline_tokens_per_s": ceiling,
           "hbm_roofline_frac": on["tokens_per_s"] / ceiling,
           "h2d_gbs_during_run": on["h2d_gbs_during_run"],
           "modes": {"on": on, "off": off}}
    if args.stack_cpu_tokens > 0:
        _log(f"[bench] stack cpu baseline: oracle, probe of {args.stack_cpu_tokens} tokens")
        rec["cpu_baseline"] = cpu_baseline(cfg, args.stack_cpu_tokens)
    return rec


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=240)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--workload", default="c1", help="configuration key in workload.configs")
    ap.add_argument("--cpu-tokens", type=int, default=192,
                    help="oracle probe size in decode steps (0 disables); the timed sample grows from it to about 15 s")
    ap.add_argument("--ablation", type=int, default=1, help="also time OFF, PRED0 and Naive Prefetch modes")
    ap.add_argument("--ffn-wgs", type=int, default=0, help="FFN workgroups (0: library default)")
    ap.add_argument("--ffn-overlap", type=int, default=0,
                    help="1: split the batch-1 FFN, resident experts beside the on-demand copies")
    ap.add_argument("--prefetch-parallel", type=int, default=0,
                    help="1: a layer's whole prefetch copies alternate the two copy streams")
    ap.add_argument("--batch", type=int, default=0, help="override the workload's batch (0: keep)")
    ap.add_argument("--slots", type=int, default=0, help="override HBM slots per layer (0: keep)")
    ap.add_argument("--layers", type=int, default=0, help="override the layer count (0: keep)")
    ap.add_argument("--tie-layers", type=int, default=0,
                    help="offload tier of k distinct expert layers shared round-robin (0: one per layer)")
    ap.add_argument("--sweep", type=lambda v: [int(x) for x in v.split(",") if x != ""], default=[],
                    help="extra modes at these M_max values, e.g. 0,1,2,4,8,16")
    ap.add_argument("--distill", type=int, default=0,
                    help="train the adapters by KL distillation on traces of this many fresh sequences first")
    ap.add_argument("--distill-len", type=int, default=64, help="tokens per distillation sequence")
    ap.add_argument("--tier-gbps", type=lambda v: [float(x) for x in v.split(",") if x != ""], default=[],
                    help="storage emulation: for each offload-tier bandwidth (GB/s, below the link's), "
                         "time OFF and M_max 1, 2 with every expert copy slowed to it")
    ap.add_argument("--copy-engine", choices=("split", "kernel", "sdma"), default="split",
                    help="expert copies: on-demand by the copy kernel and prefetches by the DMA engines "
                         "(split, default), all by the copy kernel, or all by the DMA engines")
    ap.add_argument("--stack", default="c2",
                    help="workload key of the whole-stack record run after the headline pair ('' disables)")
    ap.add_argument("--stack-tie", type=int, default=4,
                    help="distinct expert layers of the stack record's offload tier (0: one per layer)")
    ap.add_argument("--stack-cpu-tokens", type=int, default=1, help="oracle probe of the stack record in steps (0 disables); the sample grows to about 15 s")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a 256 MiB device-to-device copy three times (counter calibration)")
    args = ap.parse_args()

    if args.copy_probe:
        import torch
        src = torch.ones(256 << 20, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": src.numel()}), flush=True)
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "the offloaded-MoE hot path runs on one GPU only; "
                                   "run with --gpus 1"}), flush=True)
        sys.exit(2)

    import numpy as np
    import torch

    import workload
    from paper_2607_24787_amd import spp
    from paper_2607_24787_amd.model import OffloadedMoEStack
    from workload import gen

    cfg = workload.get(args.workload)
    over = {k: v for k, v in (("batch", args.batch), ("S", args.slots), ("L", args.layers),
                              ("expert_layers", args.tie_layers)) if v > 0}
    if over:
        cfg = cfg.with_(**over)
    total = args.warmup + 2 * args.steps   # warm-up, the timed pass, the instrumented pass
    t_setup = time.perf_counter()
    h_all = gen.hidden_states(cfg, tokens=total)                      # [T, B, D] storage
    stack = OffloadedMoEStack(cfg)
    if args.ffn_wgs:
        spp.spp_set_ffn_workgroups(stack.ctx, args.ffn_wgs)
    if args.ffn_overlap:
        spp.spp_set_ffn_overlap(stack.ctx, 1)
    if args.prefetch_parallel:
        spp.spp_set_prefetch_parallel(stack.ctx, 1)
    row_bytes = cfg.batch * cfg.D * cfg.elem_bytes
    dev_h = torch.from_numpy(np.ascontiguousarray(h_all).reshape(-1).view(np.uint8).copy()).to(stack.device)
    torch.cuda.synchronize()
    _log(f"[bench] setup {time.perf_counter() - t_setup:.1f}s workload={cfg.name}")

    distilled = None
    if args.distill > 0:
        stack, distilled = distill_adapters(stack, cfg, args.distill, args.distill_len)
        if args.ffn_wgs:
            spp.spp_set_ffn_workgroups(stack.ctx, args.ffn_wgs)
        if args.ffn_overlap:
            spp.spp_set_ffn_overlap(stack.ctx, 1)
        if args.prefetch_parallel:
            spp.spp_set_prefetch_parallel(stack.ctx, 1)

    engines = {"split": spp.COPY_SPLIT, "kernel": spp.COPY_KERNEL, "sdma": spp.COPY_SDMA}
    engine = engines[args.copy_engine]
    # per-expert cost on each engine (the budget uses the one of on-demand loads)
    engine_us = {}
    for name in ("kernel", "sdma"):
        spp.spp_set_copy_engine(stack.ctx, engines[name])
        engine_us[name] = spp.spp_profile_expert_copy(stack.ctx, 0, 32)
    spp.spp_set_copy_engine(stack.ctx, engine)
    per_expert_us = spp.spp_profile_expert_copy(stack.ctx, 0, 32)   # the prefetch engine: the budget's cost c
    link_gbs = cfg.blob_bytes / (min(engine_us.values()) * 1e3)       # the link's peak: the faster engine
    _log(f"[bench] pinned H2D per expert: copy kernel {engine_us['kernel']:.1f} us "
         f"({cfg.blob_bytes / (engine_us['kernel'] * 1e3):.2f} GB/s), DMA {engine_us['sdma']:.1f} us "
         f"({cfg.blob_bytes / (engine_us['sdma'] * 1e3):.2f} GB/s); engine {args.copy_engine}")

    # what the batch-1 FFN's own access pattern streams without its arithmetic
    read_probe = None
    if spp.spp_blob_layout(stack.desc) in (spp.LAYOUT_UNITS, spp.LAYOUT_Q4_UNITS) and cfg.dtype == "bf16":
        probe_us, probe_gbs = spp.spp_probe_read_ceiling(stack.ctx, 40)
        read_probe = {"us_per_launch": probe_us, "gbs": probe_gbs, "frac_of_peak": probe_gbs / HBM_PEAK_GBS}
        _log(f"[bench] read probe (FFN loads, no arithmetic): {probe_us:.2f} us per launch, {probe_gbs:.0f} GB/s")
    # the same byte count read as one contiguous stream: the chip's ceiling for it in one launch
    stream_probe = None
    if cfg.S >= cfg.K:
        s_us, s_gbs = spp.spp_probe_stream_read(stack.ctx, 40)
        stream_probe = {"us_per_launch": s_us, "gbs": s_gbs, "frac_of_peak": s_gbs / HBM_PEAK_GBS}
        _log(f"[bench] stream probe (the same bytes, one contiguous read): {s_us:.2f} us per launch, {s_gbs:.0f} GB/s")

    on = run_mode(stack, dev_h, row_bytes, args.warmup, args.steps, cfg.window)
    _log(f"[bench] ON  {on['tokens_per_s']:.1f} tok/s coverage={on['next_layer_coverage']:.3f} "
         f"exposed={on['exposed_transfer_pct']:.1f}% ffn={on['ffn_kernel_us']:.2f}us")
    if on["expert_recall"]:
        _log("[bench] ON  expert recall " + " ".join(f"{k}={v:.3f}" for k, v in on["expert_recall"].items())
             + "; predictions with more missing than M_max: "
             + " ".join(f"{k}={v:.2f}" for k, v in on["demand_exceeds_budget"].items())
             + "; exposed = on-demand loads {on_demand_loads:.1f}% + copy-stream waits {copy_stream_waits:.1f}%"
             .format(**on["exposed_breakdown_pct"]))
    modes = {"on": on}
    if args.ablation:
        for name, M, naive in (("pred0", 0, False), ("off", -1, False), ("naive", cfg.window, True)):
            modes[name] = run_mode(stack, dev_h, row_bytes, args.warmup, args.steps, M, naive)
            _log(f"[bench] {name} {modes[name]['tokens_per_s']:.1f} tok/s "
                 f"coverage={modes[name]['next_layer_coverage']:.3f}")
            if name == "pred0" and modes[name]["demand_exceeds_window"]:
                _log(f"[bench] pred0 predictions with more than {cfg.window} of the top-M missing: "
                     + " ".join(f"{k}={v:.2f}" for k, v in modes[name]["demand_exceeds_window"].items()))
        # the same SpecPrefetch run with the other copy engines
        for ename in engines:
            if ename == args.copy_engine:
                continue
            spp.spp_set_copy_engine(stack.ctx, engines[ename])
            name = f"on_copy_{ename}"
            modes[name] = run_mode(stack, dev_h, row_bytes, args.warmup, args.steps, cfg.window)
            _log(f"[bench] {name} {modes[name]['tokens_per_s']:.1f} tok/s "
                 f"exposed={modes[name]['exposed_transfer_pct']:.1f}% ffn={modes[name]['ffn_kernel_us']:.2f}us")
        spp.spp_set_copy_engine(stack.ctx, engine)
        # SpecPrefetch at the budget the window-aware rule derives from the
        # compute window measured in the run above (section "Window-Aware
        # Prefetch Budgeting"); 0 is PRED0, and the configured window is "on"
        if on["compute_window_us"] is not None:
            rule_M = spp.select_prefetch_budget(on["compute_window_us"], per_expert_us, cfg.n)
            if rule_M == 0:
                modes["rule"] = dict(modes["pred0"], rule_budget=0)
            elif rule_M == cfg.window:
                modes["rule"] = dict(on, rule_budget=rule_M)
            else:
                modes["rule"] = dict(run_mode(stack, dev_h, row_bytes, args.warmup, args.steps, rule_M),
                                     rule_budget=rule_M)
            _log(f"[bench] rule (M_max={rule_M} = floor(W/c)) {modes['rule']['tokens_per_s']:.1f} tok/s "
                 f"coverage={modes['rule']['next_layer_coverage']:.3f}")
    for M in args.sweep:
        modes[f"M{M}"] = run_mode(stack, dev_h, row_bytes, args.warmup, args.steps, M)
        _log(f"[bench] sweep M_max={M} {modes[f'M{M}']['tokens_per_s']:.1f} tok/s "
             f"coverage={modes[f'M{M}']['next_layer_coverage']:.3f} "
             f"exposed={modes[f'M{M}']['exposed_transfer_pct']:.1f}%")

    for gbps in args.tier_gbps:
        # one expert then takes blob / gbps: a busy wait of the difference before each copy
        delay = max(0, int(round(cfg.blob_bytes / (gbps * 1e3) - min(engine_us.values()))))
        spp.spp_set_tier_delay(stack.ctx, min(delay, 100000))
        for name, M in (("off", -1), ("M1", 1), ("M2", 2)):
            r = run_mode(stack, dev_h, row_bytes, args.warmup, args.steps, M)
            r["tier_gbps"], r["tier_delay_us"] = gbps, delay
            modes[f"tier{gbps:g}_{name}"] = r
            _log(f"[bench] tier {gbps:g} GB/s (+{delay} us per expert) {name} {r['tokens_per_s']:.1f} tok/s "
                 f"coverage={r['next_layer_coverage']:.3f}")
        spp.spp_set_tier_delay(stack.ctx, 0)
    window_us = on["compute_window_us"]
    implied_budget = (spp.select_prefetch_budget(window_us, per_expert_us, cfg.n)
                      if window_us is not None else None)
    # algorithmic bytes per FFN launch: every distinct expert the batch routes to, streamed once
    distinct = on["distinct_experts_per_layer"] if cfg.batch > 1 else cfg.K
    ffn_bytes = int(round((distinct + cfg.n_shared) * cfg.blob_bytes))
    achieved = ffn_bytes / (on["ffn_kernel_us"] * 1e3)                   # GB/s
    # the FFN kernel this context runs: grouped MFMA over the tiled layout, or the unit-stream kernel
    layout = spp.spp_blob_layout(stack.desc)
    kernel = {spp.LAYOUT_TILED: "ffn_grouped_kernel", spp.LAYOUT_Q4_UNITS: "ffn_q4_kernel"}.get(
        layout, "ffn_units_kernel" if args.ffn_overlap else "ffn_slices_kernel")
    step_bytes = step_hbm_bytes(cfg, on["distinct_experts_per_layer"])
    hbm_ceiling = HBM_PEAK_GBS * 1e9 * cfg.batch / step_bytes          # tokens/s at 8 TB/s
    workload = cfg.name + ("" if not over else "+" + ",".join(f"{k}={v}" for k, v in over.items()))
    slug = workload.replace("+", "__").replace("=", "").replace(",", "_")
    traffic = measured_traffic(os.path.join(ROOT, "profiles", f"{kernel}__{slug}.md"),
                               os.path.join(ROOT, "paper_2607_24787_amd", "csrc", "spp_kernels.hip"))
    line = {
        "metric": METRIC,
        "value": on["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": on["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": ("synthetic (seeded AR(1) hidden states, N(0,{w:g}) weights{rr}{us}{q4}, SVD-built adapters)"
                 .format(w=cfg.w_std,
                         rr=f", rank-{cfg.router_rank} routers" if cfg.router_rank > 0 else "",
                         us=f", expert updates x{cfg.update_scale:g}" if cfg.update_scale != 1.0 else "",
                         q4=", 4-bit experts" if cfg.codec == "q4" else "")),
        "config": {"workload": workload,
                   "layers": cfg.L, "hidden": cfg.D, "experts": cfg.n, "top_k": cfg.K,
                   "intermediate": cfg.I, "adapter_rank": cfg.r, "hbm_slots_per_layer": cfg.S,
                   "window_experts": cfg.window, "batch": cfg.batch, "shared_experts": cfg.n_shared,
                   "offload_tier": "pinned host DRAM", "expert_bytes": cfg.blob_bytes,
                   "ffn_split": bool(args.ffn_overlap), "prefetch_parallel": bool(args.prefetch_parallel)},
        "next_layer_coverage": on["next_layer_coverage"],
        "exposed_transfer_pct": on["exposed_transfer_pct"],
        # the headline layer of a pair is its prefetch target, layer 1
        "exposed_transfer_pct_layer1": (on["per_layer"][1]["exposed_pct"]
                                        if on["per_layer"] and cfg.L >= 2 else None),
        "hbm_bytes_per_token": int(step_bytes / cfg.batch),
        "hbm_roofline_tokens_per_s": hbm_ceiling,
        "hbm_roofline_frac": on["tokens_per_s"] / hbm_ceiling,
        "exposed_breakdown_pct": on["exposed_breakdown_pct"],
        "expert_recall": on["expert_recall"],
        "demand_exceeds_budget": on["demand_exceeds_budget"],
        # without transfers (PRED0), how often the missing top-M experts exceed the window
        "demand_exceeds_window_pred0": modes["pred0"]["demand_exceeds_window"] if "pred0" in modes else None,
        "roofline": {"kernel": kernel + " (routed-expert SwiGLU FFN)", "bound": "hbm",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": traffic, "bytes_per_launch": ffn_bytes, "avg_launch_us": on["ffn_kernel_us"],
                     "read_probe": read_probe,
                     "frac_of_read_probe": achieved / read_probe["gbs"] if read_probe else None,
                     "stream_probe": stream_probe,
                     "frac_of_stream_probe": achieved / stream_probe["gbs"] if stream_probe else None},
        "link": {"bound": "host link (pinned H2D)", "copy_engine": args.copy_engine,
                 "per_expert_us_prefetch_engine": per_expert_us, "peak_gbs_measured": link_gbs,
                 "per_expert_us_by_engine": engine_us,
                 "achieved_gbs_during_run": on["h2d_gbs_during_run"],
                 "frac": (on["h2d_gbs_during_run"] / link_gbs) if on["h2d_gbs_during_run"] else None},
        "window": {"compute_window_us": window_us, "live_window_us": on["window_us"],
                   "per_expert_transfer_us": per_expert_us,
                   "implied_budget": implied_budget, "configured_budget": cfg.window,
                   "tokens_per_s_at_implied_budget": modes["rule"]["tokens_per_s"] if "rule" in modes else None},
        "modes": modes,
    }
    if distilled is not None:
        line["config"]["adapters"] = "KL-distilled on synthetic traces"
        line["distill"] = distilled
    stack.close()
    if args.cpu_tokens > 0:
        _log(f"[bench] cpu baseline: oracle, probe of {args.cpu_tokens} tokens")
        line["cpu_baseline"] = cpu_baseline(cfg, args.cpu_tokens)
    if args.stack:
        line["stack48" if args.stack == "c2" else "stack"] = stack_record(args, args.stack, args.stack_tie)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
