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
import statistics
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA, TFLOP/s
# Full-rate VALU lane operations per second: 256 CUs x 4 SIMDs x 16 lanes x
# 2.4 GHz.  (The published fp32 vector peak, 157.3 TFLOP/s, is this rate x 2
# for FMA x 2 for packed fp32; fp64 FMA issues at the same rate, 78.6 TFLOP/s.)
VALU_PEAK_TSLOTS = 256 * 4 * 16 * 2.4e9 / 1e12
COPY_BYTES = 1 << 30           # calibration copy: 1 GiB read, 1 GiB written

KERNEL_SOURCES = {
    "score_": "score.hip", "sort_segments": "sort.hip", "curves": "curves.hip",
    "curve_blockstats": "allocate.hip", "allocate": "allocate.hip", "select": "select.hip",
    "kept_offsets": "select.hip", "clamp_budgets": "select.hip", "packed_offsets": "select.hip",
    "coverage_budget": "select.hip", "tail_": "tail.hip", "compact_": "tail.hip",
    "kept_bitmap": "tail.hip", "decode": "decode.hip",
}


def algorithmic_model(cfg, n_keep, lse_in=False):
    """Algorithmic HBM bytes, MFMA flops and VALU slots per launch of each kernel.

    Per (KV head, token) unit with d = head_dim, e = element bytes, keep
    fraction f = (n_keep - 1) / n, M = w*G window rows:
      kernel                bytes                                   MFMA flops  VALU slots
      score pass 1          K read: d*e                              2*M*d       4*M
      score pass 2          K read + score write: d*e + 4            2*M*d       4*M
      sort                  score read + order write: 8
      curves                V gathered + order + key + curve: d*e+12             9*d
      curve block stats     curve read: 4
      allocate              curve read: 4
      select                score read + kept index + bitmap: 4+4f+1/8
      tail+compact gather   kept index, score, K, V read; K, V and
                            position written: f*(4*d*e + 12)
    A VALU slot is one full-rate lane operation: per softmax term the passes
    spend one multiply (or fma), one exp2 (half rate: 2 slots) and one add;
    the fp64 curves spend per (rank, dim) two conversions and two fma in the
    totals pass and two conversions and three fma in the walk.
    With the caller's row log-sum-exp (lse_in) score pass 1 does not run, so
    K is read once.
    """
    L, H, D = cfg.layers, cfg.kv_heads, cfg.head_dim
    e = 2 if cfg.dtype_name == "bf16" else 4
    ht = L * H * sum(cfg.seqlens)
    f = sum((nk - 1) for nk in n_keep) / sum(cfg.seqlens)
    M = cfg.window * cfg.group
    per = {
        "score_pass1_mfma": (D * e, 2 * M * D, 4 * M),
        "score_pass2_mfma": (D * e + 4, 2 * M * D, 4 * M),
        "sort_segments": (8, 0, 0),
        "curves": (D * e + 12, 0, 9 * D),
        "curve_blockstats": (4, 0, 0),
        "allocate": (4, 0, 0),
        "select": (4 + 4 * f + 0.125, 0, 0),
        "tail_compact_gather": (f * (4 * D * e + 12), 0, 0),
    }
    if lse_in:
        del per["score_pass1_mfma"]
    return {k: (b * ht, fl * ht, sl * ht) for k, (b, fl, sl) in per.items()}, ht


# One-factor ablations of the pass (appendix, one-factor ablations table).
VARIANTS = {
    "default": {},
    "tail_mass": {"statistic": "tail_mass"},
    "uncentered": {"statistic": "uncentered"},
    "uniform": {"allocator": "uniform"},
    "greedy": {"allocator": "greedy"},
    "no_slot": {"slot": False},
    "alpha0": {"alpha": 0.0},
    "alpha0.1": {"alpha": 0.1},
    "alpha0.4": {"alpha": 0.4},
    # the SnapKV-uniform baseline: n_keep real tokens per head, no slot
    "snapkv_uniform": {"allocator": "uniform", "slot": False},
}


def source_digest(kernel):
    """sha256 over the source file of a kernel and the shared headers."""
    import hashlib
    fname = next((f for pre, f in KERNEL_SOURCES.items() if kernel.startswith(pre)), None)
    if fname is None:
        return None
    h = hashlib.sha256()
    for part in ("common.h", "stages.h", fname):
        with open(os.path.join(ROOT, "paper_2608_21541_amd", "csrc", part), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def recorded_traffic(kernel, workload):
    """HBM bytes per launch from a committed counter summary, if its kernel
    source is unchanged since the counters were taken (else None)."""
    pdir = os.path.join(ROOT, "profiles")
    if not os.path.isdir(pdir):
        return None
    digest = source_digest(kernel)
    for name in sorted(os.listdir(pdir)):
        if not name.endswith(".md"):
            continue
        with open(os.path.join(pdir, name)) as fh:
            for line in fh:
                if line.startswith("traffic-record: "):
                    rec = json.loads(line[len("traffic-record: "):])
                    if rec.get("kernel") == kernel and rec.get("workload") == workload \
                            and rec.get("source_sha256") == digest:
                        return rec["bytes_per_launch"]
    return None


def roofline_of(name, model, avg_ms, workload):
    """Bound of one kernel: the resource with the largest lower-bound time."""
    b, fl, sl = model.get(name, (0, 0, 0))
    sec = avg_ms / 1e3
    cands = [("hbm", b / (HBM_PEAK_GBS * 1e9), b / sec / 1e9, HBM_PEAK_GBS, "GB/s"),
             ("mfma", fl / (BF16_PEAK_TFLOPS * 1e12), fl / sec / 1e12, BF16_PEAK_TFLOPS, "TFLOP/s"),
             ("alu", sl / (VALU_PEAK_TSLOTS * 1e12), sl / sec / 1e12, VALU_PEAK_TSLOTS,
              "T VALU lane-slots/s")]
    bound, _, ach, peak, unit = max(cands, key=lambda c: c[1])
    return {"bound": bound, "achieved": ach, "peak": peak, "unit": unit, "frac": ach / peak,
            "traffic": recorded_traffic(name, workload), "kernel": name,
            "lower_bounds_ms": {c[0]: c[1] * 1e3 for c in cands}}


def run_metadata(cfg, dev):
    """Digest of every source the run executes, of the workload's
    configuration, and the device's identity and peak clocks."""
    import ctypes
    import hashlib
    import torch
    h = hashlib.sha256()
    for sub in ("paper_2608_21541_amd/csrc", "include", "synth", "paper_2608_21541_amd"):
        d = os.path.join(ROOT, sub)
        for name in sorted(os.listdir(d)):
            if name.endswith((".hip", ".h", ".py")):
                with open(os.path.join(d, name), "rb") as fh:
                    h.update(name.encode() + b"\0" + fh.read())
    with open(os.path.abspath(__file__), "rb") as fh:
        h.update(fh.read())
    conf = json.dumps({k: (str(v) if k == "dtype" else v) for k, v in vars(cfg).items()},
                      sort_keys=True, default=str)
    props = torch.cuda.get_device_properties(dev)
    clocks = {}
    try:
        hip = ctypes.CDLL("libamdhip64.so")
        for name, attr in (("sclk_peak_mhz", 5), ("mclk_peak_mhz", 60)):
            val = ctypes.c_int(0)
            if hip.hipDeviceGetAttribute(ctypes.byref(val), attr, dev.index or 0) == 0:
                clocks[name] = val.value / 1000.0
    except OSError:
        pass
    return {"source_sha256": h.hexdigest(), "config_sha256": hashlib.sha256(conf.encode()).hexdigest(),
            "device": props.name, "arch": getattr(props, "gcnArchName", ""),
            "cus": props.multi_processor_count, **clocks}


def time_passes(run, steps, stream, profile, per_step=None):
    """Average milliseconds of `steps` calls of run(), timed with events on the
    launch stream; with profile the library brackets every launch with events
    and the per-kernel averages are returned too.  With a list `per_step`,
    an event at every step boundary (one per step, on the same stream) adds
    each step's time to it."""
    import torch
    import paper_2608_21541_amd as ck
    torch.cuda.synchronize()
    if profile:
        ck.profile_reset()
        ck.profile_enable(True)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1 if per_step is not None else 2)]
    ev[0].record(stream)
    for i in range(steps):
        run()
        if per_step is not None:
            ev[i + 1].record(stream)
    ev[-1].record(stream)
    torch.cuda.synchronize()
    if per_step is not None:
        per_step.extend(ev[i].elapsed_time(ev[i + 1]) for i in range(steps))
    kernels = None
    if profile:
        prof = ck.profile_read()
        ck.profile_enable(False)
        ck.profile_reset()
        kernels = {name: {"launches_per_step": cnt / steps, "avg_ms": tot / max(cnt, 1)}
                   for name, (cnt, tot) in prof.items()}
    return ev[0].elapsed_time(ev[-1]) / steps, kernels


def copy_bandwidth(dev, nbytes=1 << 30, reps=5):
    """GB/s of a plain device-to-device copy (bytes read + bytes written per
    second), the practical ceiling a streaming kernel is compared with."""
    import torch
    src = torch.empty(nbytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    gbps = 2.0 * nbytes * reps / (a.elapsed_time(b) / 1e3) / 1e9
    del src, dst
    return gbps


def cpu_baseline(cache, cfg, n_keep, log, layers=6):
    """The fp64 oracle on the first `layers` layers of the workload (all KV
    heads, full length): about ten seconds of host work."""
    import oracle
    layers = min(layers, cfg.layers)
    n = cfg.seqlens[0]
    log(f"cpu baseline: oracle on {layers} layers x {cfg.kv_heads} heads x {n} tokens")
    dt = 0.0
    for li in range(layers):
        q = cache["q_win"][li, :cfg.window].double().cpu().numpy()
        k = cache["k"][li, :n].double().cpu().numpy()
        v = cache["v"][li, :n].double().cpu().numpy()
        t0 = time.perf_counter()
        oracle.compress_block(q, k, v, n_keep[0], 1.0 / math.sqrt(cfg.head_dim))
        dt += time.perf_counter() - t0
    cpu_model = ""
    try:
        with open("/proc/cpuinfo") as fh:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")), "")
    except OSError:
        pass
    return {"value": n / (dt / layers), "unit": "KV tokens/s per layer",
            "cores": oracle.num_threads(), "cpu_model": cpu_model, "kind": "oracle",
            "sample": f"layers 0-{layers - 1} of the workload: {cfg.kv_heads} KV heads x {n} tokens "
                      f"each, full pass (score, order, curves, allocation, selection, tail), "
                      f"{dt:.1f} s of oracle time"}


def _read_csv(path):
    import csv
    with open(path, newline="") as fh:
        return list(csv.DictReader(fh))


def summarize_stats(csv_path, out, command):
    """Markdown summary of a rocprofv3 --kernel-trace --stats kernel table."""
    rows = _read_csv(csv_path)
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    lines = ["# Kernel time summary", "", "Command:", "", "```", command, "```", "",
             "| kernel | calls | avg us | total ms | % |", "|---|---:|---:|---:|---:|"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        lines.append("| %s | %s | %.1f | %.3f | %.1f |" % (
            r["Name"][:90].replace("|", "/"), r["Calls"], float(r["AverageNs"]) / 1e3,
            float(r["TotalDurationNs"]) / 1e6, 100.0 * float(r["TotalDurationNs"]) / total))
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")


def summarize_traffic(fetch_csv, write_csv, kernel_regex, kernel, workload, out, commands):
    """HBM traffic of one kernel from two rocprofv3 --pmc runs (FETCH_SIZE, then
    WRITE_SIZE, KiB per dispatch), scaled by the readings of a 1 GiB device
    copy in the same runs."""
    import re
    import statistics

    def per_kernel(path, counter):
        vals, copies = [], []
        for r in _read_csv(path):
            if r.get("Counter_Name") != counter:
                continue
            name, val = r["Kernel_Name"], float(r["Counter_Value"])
            if re.search(kernel_regex, name):
                vals.append(val)
            elif "copy" in name.lower():
                copies.append(val)
        return vals, copies

    fv, fc = per_kernel(fetch_csv, "FETCH_SIZE")
    wv, wc = per_kernel(write_csv, "WRITE_SIZE")
    f_copy, w_copy = max(fc), max(wc)
    f_scale = COPY_BYTES / 1024.0 / f_copy
    w_scale = COPY_BYTES / 1024.0 / w_copy
    fetch_b = statistics.mean(fv) * 1024.0 * f_scale
    write_b = statistics.mean(wv) * 1024.0 * w_scale
    rec = {"kernel": kernel, "workload": workload, "source_sha256": source_digest(kernel),
           "bytes_per_launch": fetch_b + write_b, "fetch_bytes": fetch_b, "write_bytes": write_b,
           "fetch_scale": f_scale, "write_scale": w_scale, "dispatches": [len(fv), len(wv)]}
    lines = ["# HBM traffic of %s (%s)" % (kernel, workload), "",
             "Counters FETCH_SIZE and WRITE_SIZE (KiB per dispatch) from two separate",
             "rocprofv3 --pmc runs, each scaled by the reading of a plain 1 GiB device",
             "copy in the same run (copy read %.0f KiB, written %.0f KiB: scale %.4f / %.4f)."
             % (f_copy, w_copy, f_scale, w_scale), "",
             "Commands:", "", "```"] + commands + ["```", "",
             "| | per launch |", "|---|---:|",
             "| fetched | %.3f GB |" % (fetch_b / 1e9), "| written | %.3f GB |" % (write_b / 1e9),
             "| total | %.3f GB |" % ((fetch_b + write_b) / 1e9), "",
             "traffic-record: " + json.dumps(rec)]
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")


def summarize_counters(csvs, kernel_regex, out, commands):
    """Markdown summary of SQ issue counters (rocprofv3 --pmc runs) of the
    kernels matching kernel_regex: per counter the mean over dispatches of the
    value summed over the device, and the derived busy fractions."""
    import re
    import statistics
    per = {}
    for path in csvs:
        for r in _read_csv(path):
            name = r["Kernel_Name"]
            if not re.search(kernel_regex, name):
                continue
            short = re.sub(r"^void ", "", name).split("(")[0]
            d = per.setdefault(short, {}).setdefault(r["Counter_Name"], {})
            d[r["Dispatch_Id"]] = d.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
    lines = ["# SQ issue counters (%s)" % kernel_regex, "",
             "Per counter: the mean over dispatches of the device-wide sum.  Busy",
             "fractions are per SIMD: MFMA-busy and VALU-active cycles over the",
             "wave-resident cycles of one SIMD (SQ_BUSY_CYCLES counts per shader",
             "engine, 32 of them; SQ_VALU_MFMA_BUSY_CYCLES per SIMD, 1024; SQ_ACTIVE_INST_*",
             "and SQ_WAVE_CYCLES per wave in units of 4 cycles).", "",
             "Commands:", "", "```"] + commands + ["```", ""]
    for k, cs in per.items():
        m = {c: statistics.mean(v.values()) for c, v in cs.items()}
        lines += ["## " + k, "", "| counter | value |", "|---|---:|"]
        lines += ["| %s | %.4g |" % (c, v) for c, v in sorted(m.items())]
        if "SQ_BUSY_CYCLES" in m and "SQ_VALU_MFMA_BUSY_CYCLES" in m:
            span = m["SQ_BUSY_CYCLES"] / 32.0           # cycles of one shader engine
            mfma = m["SQ_VALU_MFMA_BUSY_CYCLES"] / 1024.0
            lines += ["", "| derived (per SIMD) | value |", "|---|---:|",
                      "| busy span, cycles | %.4g |" % span,
                      "| MFMA busy, cycles | %.4g (%.0f %%) |" % (mfma, 100 * mfma / span)]
            if "SQ_ACTIVE_INST_VALU" in m:
                valu = 4.0 * m["SQ_ACTIVE_INST_VALU"] / 1024.0
                lines.append("| VALU active, cycles | %.4g (%.0f %%) |" % (valu, 100 * valu / span))
            if "SQ_VALU_MFMA_COEXEC_CYCLES" in m:
                co = m["SQ_VALU_MFMA_COEXEC_CYCLES"] / 1024.0
                lines.append("| MFMA and VALU together, cycles | %.4g |" % co)
            if "SQ_WAIT_ANY" in m and "SQ_WAVE_CYCLES" in m:
                lines.append("| waves waiting, share of wave cycles | %.0f %% |"
                             % (100 * m["SQ_WAIT_ANY"] / m["SQ_WAVE_CYCLES"]))
        lines.append("")
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")


def lift_diagnostic(cfg, cache, bufs, qn, out, tq, layers):
    """The future-query lift theorem's a-posteriori bound on a sample of the
    decode: for each sampled (layer, head) and new query row, the exact output
    O over the uncompressed cache (torch fp64 on the GPU, beside the HIP path),
    the decode output Ohat, and the bound V_max (2 |p - q| + min(p, q)
    |a - r|_1) + q |v*_stored - sum_E r v| (the last term: the bf16 rounding of
    the stored slot value), with p = sigmoid(Lambda_E - log Z_S), q =
    sigmoid(z* - log Z_S), a the query's attention over the evicted set E and r
    the slot's charge (the clipped window scores over E, normalized)."""
    import torch
    H, G, D = cfg.kv_heads, cfg.group, cfg.head_dim
    n = cfg.seqlens[0]
    scale = 1.0 / math.sqrt(D)
    ko = bufs.kept_offsets.cpu()
    po = bufs.packed_offsets.cpu()
    ratios, errs, bounds, ps, qs = [], [], [], [], []
    for li in layers:
        for h in range(H):
            u = li * H + h  # one sequence
            K = cache["k"][li, :n, h].double()
            V = cache["v"][li, :n, h].double()
            Q = qn[li, :tq, h * G:(h + 1) * G].double().reshape(-1, D)
            Z = torch.matmul(Q, K.t().contiguous()) * scale
            kept = torch.zeros(n, dtype=torch.bool, device=K.device)
            kept[bufs.kept_idx[int(ko[u]):int(ko[u + 1])].long()] = True
            ev = ~kept
            r = torch.clamp(bufs.scores[li, h, :n].double(), min=0.0)[ev]
            r = r / r.sum()
            o_full = torch.matmul(torch.softmax(Z, dim=1), V)
            o_hat = out[li, :tq, h * G:(h + 1) * G].double().reshape(-1, D)
            err = torch.linalg.vector_norm(o_full - o_hat, dim=1)
            lam_e = torch.logsumexp(Z[:, ev], dim=1)
            log_zs = torch.logsumexp(Z[:, kept], dim=1)
            slot = int(po[u + 1]) - 1
            zstar = torch.matmul(Q, bufs.k_packed[slot].double()) * scale
            p = torch.sigmoid(lam_e - log_zs)
            q = torch.sigmoid(zstar - log_zs)
            l1 = (torch.softmax(Z[:, ev], dim=1) - r).abs().sum(dim=1)
            vmax = torch.linalg.vector_norm(V, dim=1).max()
            slack = q * torch.linalg.vector_norm(bufs.v_packed[slot].double() - r @ V[ev])
            bound = vmax * (2 * (p - q).abs() + torch.minimum(p, q) * l1) + slack
            ratios.append(err / bound)
            errs.append(err)
            bounds.append(bound)
            ps.append(p)
            qs.append(q)
    cat = lambda xs: torch.cat(xs).cpu()
    ratio, err, bound, p, q = cat(ratios), cat(errs), cat(bounds), cat(ps), cat(qs)
    return {"sample": f"layers {list(layers)}, {H} KV heads, {tq * G} new query rows each; "
                      "exact attention over the uncompressed cache in torch fp64",
            "rows": int(ratio.numel()), "holds": float((ratio <= 1.0).double().mean()),
            "ratio_median": float(ratio.median()), "ratio_max": float(ratio.max()),
            "err_median": float(err.median()), "bound_median": float(bound.median()),
            "p_median": float(p.median()), "q_median": float(q.median())}


def run_decode_bench(args, cfg, cache, spec, bufs, n_keep, dev, log):
    """Decode over the packed cache: one compression pass (untimed) builds it,
    then `steps` decodes of `tq` new queries per sequence are timed.  The
    algorithmic bytes of one decode are the packed K and V rows, the new
    queries and the fp32 outputs; the split partials are overhead."""
    import torch
    import paper_2608_21541_amd as ck
    import synth

    ck.compress(spec, cache["q_win"], cache["k"], cache["v"], n_keep,
                alpha=VARIANTS[args.variant].get("alpha", 0.2), bufs=bufs)
    torch.cuda.synchronize()
    rows = int(bufs.packed_offsets[-1].item())
    # the budgets are known once compression has run: the longest segment
    # bounds the split partials (set before the timed region)
    max_rows = int((bufs.packed_offsets[1:] - bufs.packed_offsets[:-1]).max().item())
    e = 2 if cfg.dtype_name == "bf16" else 4
    hq = cfg.kv_heads * cfg.group
    stream = torch.cuda.current_stream(dev)

    def time_tq(tq, steps, warmup):
        qn = synth.make_queries(cfg, tq, dev)
        db = ck.DecodeBuffers(spec, tq, dev, max_rows=max_rows)
        for _ in range(warmup):
            ck.decode(spec, qn, bufs.k_packed, bufs.v_packed, bufs.packed_offsets, tq, bufs=db)
        torch.cuda.synchronize()
        ck.profile_reset()
        ck.profile_enable(True)
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for _ in range(steps):
            ck.decode(spec, qn, bufs.k_packed, bufs.v_packed, bufs.packed_offsets, tq, bufs=db)
        t1.record(stream)
        torch.cuda.synchronize()
        prof = ck.profile_read()
        ck.profile_enable(False)
        ck.profile_reset()
        ms = t0.elapsed_time(t1) / steps
        qrows = cfg.layers * cfg.batch * tq * hq
        alg = rows * cfg.head_dim * e * 2 + qrows * cfg.head_dim * (e + 4)
        kern = {n: {"launches_per_step": c / steps, "avg_ms": t / max(c, 1)}
                for n, (c, t) in prof.items()}
        kms = kern["decode"]["avg_ms"]
        roof = {"bound": "hbm", "achieved": alg / (kms / 1e3) / 1e9, "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": alg / (kms / 1e3) / 1e9 / HBM_PEAK_GBS,
                "traffic": recorded_traffic("decode", f"{args.config}-decode{tq}"), "kernel": "decode",
                "alg_bytes_per_launch": alg}
        return ms, kern, roof

    ms, kern, roof = time_tq(args.tq, args.steps, args.warmup)
    ms1, kern1, roof1 = time_tq(1, args.steps, args.warmup)
    log(f"decode tq={args.tq}: {ms:.3f} ms; tq=1: {ms1:.3f} ms")
    clusters = None
    if args.clusters > 0:
        assert not spec.slot, "clustered summaries replace the slot: use --variant no_slot"
        m = args.clusters
        cl = ck.cluster_tail(spec, cache["k"], cache["v"], bufs.perm, bufs.budgets, m)
        torch.cuda.synchronize()
        qn = synth.make_queries(cfg, args.tq, dev)
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for _ in range(args.steps):
            ck.cluster_tail(spec, cache["k"], cache["v"], bufs.perm, bufs.budgets, m)
        t1.record(stream)
        torch.cuda.synchronize()
        tail_ms = t0.elapsed_time(t1) / args.steps
        ck.decode_clustered(spec, qn, bufs.k_packed, bufs.v_packed, bufs.packed_offsets, args.tq,
                            cl, max_rows=max_rows)
        torch.cuda.synchronize()
        t0.record(stream)
        for _ in range(args.steps):
            _, _, bound = ck.decode_clustered(spec, qn, bufs.k_packed, bufs.v_packed,
                                              bufs.packed_offsets, args.tq, cl, max_rows=max_rows)
        t1.record(stream)
        torch.cuda.synchronize()
        dec_ms = t0.elapsed_time(t1) / args.steps
        evicted = int(cfg.layers * cfg.kv_heads * sum(cfg.seqlens)) - rows
        # algorithmic bytes: every evicted row's K and V slice and rank entry
        # once, the provisional centres' sample (every 16th member at most)
        # again, and every kept row's V slice and rank entry (the kept value
        # norm)
        cl_bytes = evicted * (2 * cfg.head_dim * e + 4) * (1 + 1 / 16) + rows * (cfg.head_dim * e + 4)
        clusters = {"m": m, "cluster_tail_ms": tail_ms, "cluster_tail_alg_bytes": cl_bytes,
                    "cluster_tail_GBps": cl_bytes / (tail_ms / 1e3) / 1e9,
                    "decode_clustered_ms": dec_ms,
                    "finite_certificates": float(torch.isfinite(bound).float().mean())}
        log(f"clusters: {clusters}")
    lift = None
    if cfg.batch == 1:
        qn = synth.make_queries(cfg, args.tq, dev)
        out = ck.decode(spec, qn, bufs.k_packed, bufs.v_packed, bufs.packed_offsets, args.tq,
                        max_rows=max_rows)
        torch.cuda.synchronize()
        lift = lift_diagnostic(cfg, cache, bufs, qn, out, args.tq,
                               sorted({0, cfg.layers - 1}))
        log(f"lift bound: holds on {lift['holds']:.4f} of {lift['rows']} rows, "
            f"median ratio {lift['ratio_median']:.3g}")
    tokens = cfg.batch * args.tq
    rec = {
        "metric": "decode over the packed cache: new tokens per second (all layers and heads)",
        "value": tokens / (ms / 1e3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": cfg.dtype_name, "data": "synthetic",
        "config": {"workload": f"{args.config} packed cache ({rows} rows of {cfg.layers} layers x "
                               f"{cfg.kv_heads} KV heads, n_keep {n_keep[0]}), {args.tq} new "
                               f"queries per sequence x {hq} query heads",
                   "tq": args.tq, "packed_rows": rows, "max_segment_rows": max_rows},
        "roofline": roof, "kernels": kern,
        "tq1": {"ms_per_step": ms1, "roofline": roof1, "kernels": kern1},
        "lift_bound": lift,
        "clusters": clusters,
    }
    print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="C3")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-lse-line", action="store_true",
                    help="skip the pass with the caller's row log-sum-exp")
    ap.add_argument("--quiet", action="store_true")
    ap.add_argument("--decode", action="store_true",
                    help="time decode over the packed cache instead of the pass")
    ap.add_argument("--tq", type=int, default=32, help="new queries per sequence (--decode)")
    ap.add_argument("--clusters", type=int, default=0,
                    help="with --decode --variant no_slot: time M clustered tail summaries "
                         "per head and the clustered decode")
    ap.add_argument("--variant", default="default", choices=sorted(VARIANTS),
                    help="a one-factor ablation of the pass (statistic, allocator, slot, alpha)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run a 1 GiB device copy first (counter calibration)")
    ap.add_argument("--summarize-stats", nargs=3, metavar=("CSV", "OUT", "COMMAND"),
                    help="write a markdown summary of a rocprofv3 kernel_stats.csv")
    ap.add_argument("--summarize-counters", nargs=6,
                    metavar=("CSV_A", "CSV_B", "REGEX", "OUT", "CMD1", "CMD2"),
                    help="write a markdown summary of SQ issue counters from two pmc runs")
    ap.add_argument("--summarize-traffic", nargs=7,
                    metavar=("FETCH_CSV", "WRITE_CSV", "REGEX", "KERNEL", "OUT", "CMD1", "CMD2"),
                    help="write the HBM traffic record of one kernel from two pmc runs")
    args = ap.parse_args()
    if args.summarize_stats:
        summarize_stats(*args.summarize_stats)
        return
    if args.summarize_counters:
        a, b, rx, out, c1, c2 = args.summarize_counters
        summarize_counters([a, b], rx, out, [c1, c2])
        return
    if args.summarize_traffic:
        fc, wc, rx, kn, out, c1, c2 = args.summarize_traffic
        workload = args.config + (f"-decode{args.tq}" if args.decode else "")
        summarize_traffic(fc, wc, rx, kn, workload, out, [c1, c2])
        return

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
    var = VARIANTS[args.variant]
    spec.statistic = var.get("statistic", "centered")
    spec.allocator = var.get("allocator", "lagrangian")
    spec.slot = var.get("slot", True)
    alpha = var.get("alpha", 0.2)
    bufs = ck.CompressBuffers(spec, n_keep, dev, with_perm=args.clusters > 0)
    q, k, v = cache["q_win"], cache["k"], cache["v"]
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream(dev)
    if args.calibrate_copy:
        # A plain device copy of known size: its FETCH_SIZE / WRITE_SIZE
        # readings scale the counters of the timed kernels to bytes.
        src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if args.decode:
        run_decode_bench(args, cfg, cache, spec, bufs, n_keep, dev, log)
        return
    run = lambda: ck.compress(spec, q, k, v, n_keep, alpha=alpha, bufs=bufs)
    for _ in range(args.warmup):
        run()
    # Timed region: the plain pass, no profiling events.  A second run of the
    # same steps with every launch bracketed by HIP events on its stream gives
    # the per-kernel durations (and the events' overhead on the pass).
    steps_ms = []
    ms, _ = time_passes(run, args.steps, stream, profile=False, per_step=steps_ms)
    ms_prof, kernels = time_passes(run, args.steps, stream, profile=True)
    copy_gbps = copy_bandwidth(dev)
    tokens = sum(cfg.seqlens)
    # KV tokens compressed per second per layer: n / (T_pass / L)
    value = tokens / (ms / 1e3 / cfg.layers)
    log(f"pass: {ms:.3f} ms ({ms_prof:.3f} ms with per-kernel events)")

    st = bufs.alloc_stats.cpu()
    alloc_diag = {"repairs_mean": float(st[:, 0].float().mean()), "repairs_max": int(st[:, 0].max()),
                  "bisect_us_mean": float(st[:, 1].float().mean()) / 100.0,
                  "repair_us_mean": float(st[:, 2].float().mean()) / 100.0}
    log(f"allocation: {alloc_diag}")
    model, ht = algorithmic_model(cfg, n_keep)

    def summarize(kernels, model):
        for name, kk in kernels.items():
            if name in model:
                r = roofline_of(name, model, kk["avg_ms"], args.config)
                kk.update({"bound": r["bound"], "frac": r["frac"]})
        dom = max(kernels, key=lambda n_: kernels[n_]["avg_ms"] * kernels[n_]["launches_per_step"])
        return roofline_of(dom, model, kernels[dom]["avg_ms"], args.config)

    roof = summarize(kernels, model)
    pass_bytes = sum(b for b, _, _ in model.values())
    log(json.dumps(kernels, indent=1))

    # The same pass with the caller's row log-sum-exp (as an attention prefill
    # already has it): pass 1 is skipped and K is read once.  The log-sum-exp
    # comes from an untimed pass that exports it.
    lse_line = None
    if args.variant == "default" and not args.no_lse_line:
        lbufs = ck.CompressBuffers(spec, n_keep, dev, with_lse=True)
        ck.compress(spec, q, k, v, n_keep, alpha=alpha, bufs=lbufs)
        lse = lbufs.lse.clone()
        del lbufs
        run_l = lambda: ck.compress(spec, q, k, v, n_keep, alpha=alpha, bufs=bufs, lse_in=lse)
        for _ in range(args.warmup):
            run_l()
        ms_l, _ = time_passes(run_l, args.steps, stream, profile=False)
        _, kern_l = time_passes(run_l, args.steps, stream, profile=True)
        model_l, _ = algorithmic_model(cfg, n_keep, lse_in=True)
        roof_l = summarize(kern_l, model_l)
        bytes_l = sum(b for b, _, _ in model_l.values())
        lse_line = {"value": tokens / (ms_l / 1e3 / cfg.layers), "unit": "KV tokens/s per layer",
                    "ms_per_step": ms_l, "pass_alg_bytes": bytes_l,
                    "pass_alg_GBps": bytes_l / (ms_l / 1e3) / 1e9,
                    "pass_alg_frac_hbm": bytes_l / (ms_l / 1e3) / 1e9 / HBM_PEAK_GBS,
                    "roofline": roof_l, "kernels": kern_l,
                    "note": "caller-supplied row log-sum-exp (from an untimed pass): score pass 1 "
                            "skipped, K read once"}
        log(f"pass with caller log-sum-exp: {ms_l:.3f} ms")

    cpu = None
    if not args.no_cpu_baseline and args.variant == "default":
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
                   "head_dim": cfg.head_dim, "window": cfg.window, "n_keep": n_keep[0],
                   "variant": args.variant},
        "pass_alg_bytes": pass_bytes,
        "pass_alg_GBps": pass_bytes / (ms / 1e3) / 1e9,
        "pass_alg_frac_hbm": pass_bytes / (ms / 1e3) / 1e9 / HBM_PEAK_GBS,
        "ms_median": statistics.median(steps_ms),
        "ms_min": min(steps_ms),
        "copy_GBps": copy_gbps,
        "pass_alg_frac_copy": pass_bytes / (ms / 1e3) / 1e9 / copy_gbps,
        "roofline": roof,
        "kernels": kernels,
        "ms_per_step_with_kernel_events": ms_prof,
        "cpu_baseline": cpu,
        "allocation": alloc_diag,
        "lse_in": lse_line,
        "meta": run_metadata(cfg, dev),
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
