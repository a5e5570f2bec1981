"""Benchmark of the CertKV compression pass on one MI355X.

Workload: a Llama-3-8B-shaped cache, 32 layers x 8 KV heads (GQA 4), head
dim 128, 131072 tokens, 64-query observation window, bf16, ten-fold budget
(n_keep = 13108 live slots per head incl. the tail slot); synthetic seeded
inputs already resident in HBM.  One step = one full compression pass
(score, order + curves + allocation, selection, tail summary, compaction)
over all layers.

Prints one JSON line: KV tokens compressed per second per layer, the
roofline position of the dominant kernel (timed with HIP events on the
launch stream), and the CPU oracle timed on a bounded sample of the same
workload.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA


def algorithmic_model(cfg, n_keep):
    """Algorithmic bytes and flops per launch of each kernel (whole workload).

    Per (KV head, token) unit with d = head_dim, e = element bytes, keep
    fraction f = (n_keep - 1) / n:
      score pass 1          K read                                   d*e
      score pass 2          K read + score write                     d*e + 4
      sort                  score read + order write                 4 + 4
      curves                V gathered + order + key + curve write   d*e + 12
      curve block stats     curve read                               4
      allocate              curve read                               4
      select                score read + kept index write + bitmap   4 + 4f + 1/8
      tail+compact gather   kept index, score, K, V read; K, V and
                            position written                          f*(4*d*e + 12)
    MFMA flops of each scoring pass: 2 * M * d per (head, token), M = w*G.
    Small per-unit kernels (row combines, offsets, slot finalize) are
    modelled by their per-unit traffic only.
    """
    L, H, D = cfg.layers, cfg.kv_heads, cfg.head_dim
    e = 2 if cfg.dtype_name == "bf16" else 4
    ht = L * H * sum(cfg.seqlens)
    f = sum((nk - 1) for nk in n_keep) / sum(cfg.seqlens)
    M = cfg.window * cfg.group
    per = {
        "score_pass1_mfma": (D * e, 2 * M * D),
        "score_pass2_mfma": (D * e + 4, 2 * M * D),
        "sort_segments": (8, 0),
        "curves": (D * e + 12, 0),
        "curve_blockstats": (4, 0),
        "allocate": (4, 0),
        "select": (4 + 4 * f + 0.125, 0),
        "tail_compact_gather": (f * (4 * D * e + 12), 0),
    }
    return {k: (b * ht, fl * ht) for k, (b, fl) in per.items()}, ht


def cpu_baseline(cache, cfg, n_keep, log):
    """The fp64 oracle on one full layer of the workload (all KV heads)."""
    import oracle
    q = cache["q_win"][0, :cfg.window].double().cpu().numpy()
    k = cache["k"][0, :cfg.seqlens[0]].double().cpu().numpy()
    v = cache["v"][0, :cfg.seqlens[0]].double().cpu().numpy()
    log(f"cpu baseline: oracle on 1 layer x {cfg.kv_heads} heads x {cfg.seqlens[0]} tokens")
    t0 = time.perf_counter()
    oracle.compress_block(q, k, v, n_keep[0], 1.0 / math.sqrt(cfg.head_dim))
    dt = time.perf_counter() - t0
    return {"value": cfg.seqlens[0] / dt, "unit": "KV tokens/s per layer",
            "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"layer 0 of the workload: {cfg.kv_heads} KV heads x {cfg.seqlens[0]} tokens, "
                      f"full pass (score, order, curves, allocation, selection, tail), {dt:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="C3")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--quiet", action="store_true")
    args = ap.parse_args()

    def log(msg):
        if not args.quiet:
            print(msg, file=sys.stderr, flush=True)

    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on exactly one GPU; "
                                   "--gpus must be 1 (sharding is described in DESIGN.md)"}))
        sys.exit(2)

    import torch
    import paper_2608_21541_amd as ck
    import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    cfg = synth.config(args.config)
    cfg.dtype_name = "bf16" if cfg.dtype == torch.bfloat16 else "f32"
    log(f"generating {args.config}: {cfg.layers} layers, {cfg.seqlens} tokens")
    cache = synth.make_cache(cfg, dev)
    n_keep = cache["n_keep"]
    spec = ck.ProblemSpec(cfg.layers, cfg.kv_heads, cfg.group, cfg.head_dim, cfg.window,
                          cfg.seqlens, cfg.dtype)
    bufs = ck.CompressBuffers(spec, n_keep, dev)
    q, k, v = cache["q_win"], cache["k"], cache["v"]
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream(dev)
    for _ in range(args.warmup):
        ck.compress(spec, q, k, v, n_keep, bufs=bufs)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(args.steps):
        ck.compress(spec, q, k, v, n_keep, bufs=bufs)
    end.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / args.steps
    tokens = sum(cfg.seqlens)
    value = tokens * cfg.layers / (ms / 1e3) / cfg.layers  # tokens per second per layer
    log(f"pass: {ms:.3f} ms")

    # Per-kernel durations from HIP events around each launch (same stream).
    ck.profile_reset()
    ck.profile_enable(True)
    for _ in range(args.steps):
        ck.compress(spec, q, k, v, n_keep, bufs=bufs)
    torch.cuda.synchronize()
    prof = ck.profile_read()
    ck.profile_enable(False)
    ck.profile_reset()
    st = bufs.alloc_stats.cpu()
    alloc_diag = {"repairs_mean": float(st[:, 0].float().mean()), "repairs_max": int(st[:, 0].max()),
                  "bisect_us_mean": float(st[:, 1].float().mean()) / 100.0,
                  "repair_us_mean": float(st[:, 2].float().mean()) / 100.0}
    log(f"allocation: {alloc_diag}")
    model, ht = algorithmic_model(cfg, n_keep)
    kernels = {}
    for name, (cnt, tot) in prof.items():
        avg = tot / max(cnt, 1)
        kernels[name] = {"launches_per_step": cnt / args.steps, "avg_ms": avg}
    dom = max(kernels, key=lambda n_: kernels[n_]["avg_ms"] * kernels[n_]["launches_per_step"])
    dbytes, dflops = model.get(dom, (0, 0))
    davg = kernels[dom]["avg_ms"] / 1e3
    gbs = dbytes / davg / 1e9
    tfl = dflops / davg / 1e12
    if dflops and dflops / max(dbytes, 1) > BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9):
        roof = {"bound": "mfma", "achieved": tfl, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": tfl / BF16_PEAK_TFLOPS}
    else:
        roof = {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": gbs / HBM_PEAK_GBS}
    roof["kernel"] = dom
    roof["traffic"] = None
    pass_bytes = sum(b for b, _ in model.values())
    for name, kk in kernels.items():
        b_, f_ = model.get(name, (0, 0))
        if b_:
            kk["alg_GBps"] = b_ / (kk["avg_ms"] / 1e3) / 1e9
        if f_:
            kk["alg_TFLOPs"] = f_ / (kk["avg_ms"] / 1e3) / 1e12
    log(json.dumps(kernels, indent=1))

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cache, cfg, n_keep, log)

    rec = {
        "metric": "KV tokens compressed/sec per layer at 128K ctx; achieved HBM GB/s vs peak",
        "value": value,
        "unit": "KV tokens/s per layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype_name,
        "data": "synthetic",
        "config": {"workload": f"{args.config}: Llama-3-8B-shaped KV cache, {cfg.layers} layers x "
                               f"{cfg.kv_heads} KV heads (GQA {cfg.group}), d {cfg.head_dim}, "
                               f"{tokens} tokens, window {cfg.window}, n_keep {n_keep[0]}",
                   "layers": cfg.layers, "seq_len": tokens, "kv_heads": cfg.kv_heads,
                   "head_dim": cfg.head_dim, "window": cfg.window, "n_keep": n_keep[0]},
        "pass_alg_GBps": pass_bytes / (ms / 1e3) / 1e9,
        "pass_alg_frac_hbm": pass_bytes / (ms / 1e3) / 1e9 / HBM_PEAK_GBS,
        "roofline": roof,
        "kernels": kernels,
        "cpu_baseline": cpu,
        "allocation": alloc_diag,
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
