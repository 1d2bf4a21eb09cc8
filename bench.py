"""Benchmark of the end-to-end functional-reconstruction step on one MI355X.

One step = teacher forward + student forward + Eq. 11 loss + backward to the five
converter-introduced projections, on one calibration minibatch of synthetic hidden states
resident in HBM.  Default workload: the Llama-3-8B-shaped layer (B=4, T=4096, D=4096,
H=32, G=8, d_k=128; student r_q=1536, r_kv=512, d_nope=128, d_rope=64).

Prints one JSON line: calibration tokens/s per layer (B*T / step time), the fraction of
the bf16 MFMA peak reached by the whole step, the roofline of the dominant kernel class
(a second pass over the same number of steps with every launch bracketed by HIP events
on the launch stream), and the float64 CPU oracle timed on a bounded sample of the same
workload on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--config", type=int, default=3)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-separate", action="store_true",
                   help="skip the reference timing of the four-call step (profiling runs)")
    p.add_argument("--no-graph", action="store_true",
                   help="skip the timing of the step replayed as a HIP graph (profiling runs)")
    p.add_argument("--no-rel", action="store_true",
                   help="skip the timing of the relative-error call (profiling runs)")
    p.add_argument("--no-cached", action="store_true",
                   help="skip the timing of the cached-teacher step (profiling runs)")
    p.add_argument("--no-train", action="store_true",
                   help="skip the timing of the step plus the AdamW update (profiling runs)")
    p.add_argument("--no-capture", action="store_true",
                   help="skip the timing of calibration capture (profiling runs)")
    p.add_argument("--no-decode", action="store_true",
                   help="skip the timing of absorbed-form decoding (profiling runs)")
    p.add_argument("--no-other-configs", action="store_true",
                   help="skip the timing of the other layer shapes (profiling runs)")
    p.add_argument("--decode-batch", type=int, default=64,
                   help="sequences per decoding step (each with a full-length cache)")
    p.add_argument("--cpu-seq", type=int, default=4096, help="oracle sample: tokens of one sequence")
    p.add_argument("--calib-copy-mb", type=int, default=0,
                   help="run one device-to-device copy of this many MiB first (HBM counter calibration)")
    p.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                   help="turn two rocprofv3 --pmc counter_collection.csv files (FETCH_SIZE, WRITE_SIZE) "
                        "of a --calib-copy-mb run into per-kernel HBM bytes per launch; print JSON")
    p.add_argument("--summarize-counters", nargs="+", metavar="CSV",
                   help="turn rocprofv3 --pmc counter_collection.csv files (and the kernel_trace.csv of "
                        "a --kernel-trace run given as --trace) into a per-kernel markdown table; print it")
    p.add_argument("--trace", help="kernel_trace.csv for --summarize-counters (durations)")
    return p.parse_args()


# Kernel names as the library's instrumentation reports them, derived from the names
# rocprofv3 reports (so that counter readings and live timings refer to the same kernel)
def rocprof_label(name):
    """The instrumentation's name for a kernel rocprofv3 reports as `name`."""
    import re
    base = name[5:] if name.startswith("void ") else name
    base = base.replace("(anonymous namespace)::", "").replace("mla::", "").replace("attn::", "")
    base = base.split("(")[0]
    m = re.match(r"(\w+)<(.*)>$", base.strip())
    if not m:
        return base.strip()
    fn, args = m.group(1), [x.strip() for x in m.group(2).split(",")]
    ty = lambda t: "fp32" if t == "float" else "bf16"
    if fn in ("gemm_mfma_persist_kernel", "gemm_mfma_kernel") and len(args) >= 7:
        lay = {("true", "true"): "NT", ("true", "false"): "NN", ("false", "false"): "TN",
               ("false", "true"): "TT"}[(args[4], args[5])]
        tag = fn if fn == "gemm_mfma_persist_kernel" else "gemm_mfma_kernel(masked loss)"
        return f"{tag}<{args[0]},{args[1]},{lay},{ty(args[6])}>"
    if fn == "gemm_nt4_persist_kernel" and len(args) == 2:
        return f"{fn}<256,{args[0]},NT,{ty(args[1])}>"
    if fn in ("attn_ds_gemm_persist_kernel", "attn_ds_gemm_kernel") and len(args) >= 7:
        return f"{fn}<{args[0]},{args[1]},{'dK' if args[4] == 'true' else 'dQ'},{ty(args[6])}>"
    if fn in ("attn_fwd_persist_kernel", "attn_fwd_mfma_kernel") and len(args) >= 3:
        return f"{fn}<{args[0]},{args[1]}{',lse' if args[2] == 'true' else ''}>"
    if fn.startswith("attn_dv_"):
        return f"{fn}<{args[0]},{args[1]}>"
    return fn


# sources whose change invalidates stored counter readings
TRAFFIC_SOURCES = ["paper_2607_27269_amd/csrc/gemm_mfma.hip", "paper_2607_27269_amd/csrc/attn_fwd.hip",
                   "paper_2607_27269_amd/csrc/attn_bwd.hip", "paper_2607_27269_amd/csrc/attn_common.h",
                   "paper_2607_27269_amd/csrc/common.h", "paper_2607_27269_amd/csrc/elementwise.hip",
                   "paper_2607_27269_amd/csrc/api.cpp"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")


def sources_digest():
    import hashlib
    h = hashlib.sha1()
    for f in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def summarize_traffic(fetch_csv, write_csv, copy_mb):
    """HBM bytes per launch of each kernel from FETCH_SIZE / WRITE_SIZE (KiB per dispatch),
    each scaled so that the calibration copy reads and writes copy_mb MiB."""
    import csv
    def read(path, counter):
        rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
        per = {}
        for r in rows:
            key = (r["Dispatch_Id"], r["Kernel_Name"])
            per[key] = per.get(key, 0.0) + float(r["Counter_Value"]) * 1024.0
        return per
    fetch, write = read(fetch_csv, "FETCH_SIZE"), read(write_csv, "WRITE_SIZE")
    known = copy_mb * 1024.0 * 1024.0
    def copy_value(d):
        # the calibration copy is the largest dispatch named like a copy
        cands = [v for (i, n), v in d.items() if "copy" in n.lower()]
        return max(cands) if cands else None
    fc, wc = copy_value(fetch), copy_value(write)
    out = {"copy_mb": copy_mb, "fetch_scale": known / fc if fc else None,
           "write_scale": known / wc if wc else None, "kernels": {}}
    if not fc or not wc:
        return out
    labels = sorted({rocprof_label(n) for (i, n) in fetch if "copy" not in n.lower()})
    for lab in labels:
        fv = [v for (i, n), v in fetch.items() if rocprof_label(n) == lab]
        wv = [v for (i, n), v in write.items() if rocprof_label(n) == lab]
        if not fv or not wv:
            continue
        out["kernels"][lab] = {"launches": len(fv),
                               "bytes_per_launch": sum(fv) * out["fetch_scale"] / len(fv) +
                                                   sum(wv) * out["write_scale"] / len(wv),
                               "read_bytes_per_launch": sum(fv) * out["fetch_scale"] / len(fv),
                               "write_bytes_per_launch": sum(wv) * out["write_scale"] / len(wv)}
    out["sources_sha1"] = sources_digest()
    return out


def summarize_counters(csvs, trace):
    """Per-kernel averages of rocprofv3 --pmc readings (one or more passes), with the MFMA
    and vector-ALU busy fractions and, from a kernel trace, the average duration."""
    import collections
    import csv
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    for path in csvs:
        per = collections.defaultdict(float)
        for r in csv.DictReader(open(path)):
            per[(r["Dispatch_Id"], r["Kernel_Name"], r["Counter_Name"])] += float(r["Counter_Value"])
        for (i, n, c), v in per.items():
            vals[rocprof_label(n)][c].append(v)
    dur = collections.defaultdict(list)
    if trace:
        for r in csv.DictReader(open(trace)):
            dur[rocprof_label(r["Kernel_Name"])].append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    mean = lambda xs: sum(xs) / len(xs) if xs else float("nan")
    rows = []
    for lab, cs in vals.items():
        m = {c: mean(v) for c, v in cs.items()}
        busy = m.get("SQ_BUSY_CYCLES")
        row = {"kernel": lab, "us": mean(dur.get(lab, [])) / 1e3}
        # SQ_BUSY_CYCLES counts per SE (32 per chip: 8 XCDs x 4), SQ_VALU_MFMA_BUSY_CYCLES per
        # SIMD (1024): the two ratios are the busy fraction of the matrix / vector units
        if busy:
            if "SQ_VALU_MFMA_BUSY_CYCLES" in m:
                row["mfma_busy"] = m["SQ_VALU_MFMA_BUSY_CYCLES"] / 1024 / (busy / 32)
            if "SQ_ACTIVE_INST_VALU" in m:
                row["valu_active_per_cu"] = m["SQ_ACTIVE_INST_VALU"] / 256 / (busy / 32)
        for c in ("SQ_INSTS_MFMA", "SQ_INSTS_VALU", "SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT",
                  "SQ_WAIT_INST_LDS", "SQ_INSTS_SALU"):
            if c in m:
                row[c] = m[c]
        rows.append(row)
    rows.sort(key=lambda r: -(r["us"] if r["us"] == r["us"] else 0))
    cols = ["kernel", "us", "mfma_busy", "valu_active_per_cu", "SQ_INSTS_MFMA", "SQ_INSTS_VALU",
            "SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_WAIT_INST_LDS", "SQ_INSTS_SALU"]
    cols = [c for c in cols if any(c in r for r in rows)]
    fmt = lambda v: f"{v:.3g}" if isinstance(v, float) else str(v)
    lines = ["| " + " | ".join(cols) + " |", "|" + "---|" * len(cols)]
    for r in rows:
        lines.append("| " + " | ".join(fmt(r.get(c, "")) for c in cols) + " |")
    return "\n".join(lines)


def stored_traffic(kernel):
    """Counter-derived HBM bytes per launch of `kernel`, if taken on the current sources."""
    try:
        with open(TRAFFIC_FILE) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("sources_sha1") != sources_digest():
        return None
    c = t.get("kernels", {}).get(kernel)
    return None if c is None else c["bytes_per_launch"]


def cpu_baseline(cfg, wl, seq):
    """The float64 oracle on one sequence of `seq` tokens of the same layer."""
    import numpy as np

    import oracle as O
    c = cfg
    h = wl.h[0:1, :seq]
    mask = np.ones((1, seq), dtype=np.uint8)
    t0 = time.perf_counter()
    A_t = O.teacher_forward(h, wl.Wq, wl.Wk, wl.Wv, wl.Wo, wl.inv_freq_t, c.n_heads,
                            c.n_kv_groups, c.softmax_scale)
    A_s, cache = O.student_forward(h, wl.Wdq, wl.Wuq, wl.Wdkv_kr, wl.Wuk, wl.Wuv, wl.Wo,
                                   wl.inv_freq_s, n_heads=c.n_heads, s_kv_groups=c.s_kv_groups,
                                   s_rope_groups=c.s_rope_groups, nope_dim=c.nope_dim,
                                   rope_dim=c.rope_dim, scale=c.softmax_scale)
    _, _, dA = O.recon_loss(A_s, A_t, mask)
    O.student_backward(cache, dA)
    dt = time.perf_counter() - t0
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count()
    threads = int(os.environ.get("OMP_NUM_THREADS", cores))
    return {"value": seq / dt, "unit": "tokens/s", "cores": min(cores, threads), "kind": "oracle",
            "sample": f"1 sequence x {seq} tokens of the {cfg.name} layer (full widths), "
                      f"teacher fwd + student fwd + Eq. 11 + backward, float64 numpy; {dt:.1f} s"}


def step_flops(cfg):
    """Algorithmic FLOPs of the single-call step as run: the paper's step with the two W_O
    products and dA W_O replaced by W_O^T W_O and one product with it."""
    HV = cfg.n_heads * cfg.head_dim
    return (cfg.total_flops() - 3 * cfg.flops()["T4_wo"] + 2.0 * HV * HV * cfg.hidden
            + 2.0 * cfg.tokens * HV * HV)


def time_config(idx, steps, warmup):
    """The timed step (mla_recon_step without dA) on another layer shape."""
    import torch
    from paper_2607_27269_amd import configs, synth
    from paper_2607_27269_amd.step import DeviceStep
    cfg = configs.get(idx)
    dev = DeviceStep(synth.make_workload(cfg))
    for _ in range(warmup):
        dev.fused_step(with_dA=False)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(steps):
        dev.fused_step(with_dA=False)
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / steps
    out = {"workload": f"{cfg.name}: B={cfg.batch} T={cfg.seq} D={cfg.hidden} H={cfg.n_heads} "
                       f"G={cfg.n_kv_groups} d_k={cfg.head_dim}; student r_q={cfg.q_rank} "
                       f"r_kv={cfg.kv_rank} d_nope={cfg.nope_dim} d_rope={cfg.rope_dim} "
                       f"G_kv={cfg.s_kv_groups} G_r={cfg.s_rope_groups}",
           "ms_per_step": round(ms, 4), "value": round(cfg.tokens / (ms / 1e3), 1),
           "unit": "tokens/s", "mfma_peak_frac": round(step_flops(cfg) / (ms / 1e3) / (PEAK_BF16_TFLOPS * 1e12), 4),
           "loss": float(dev.loss_buf[0])}
    del dev
    torch.cuda.empty_cache()
    return out


def decode_bench(cfg, wl, batch, steps):
    """One decoding step of `batch` sequences, each over a cache of cfg.seq latent rows
    (random bf16 stand-ins; the same shapes as the cache the student forward produces)."""
    import torch
    from paper_2607_27269_amd import _lib as L
    from paper_2607_27269_amd.step import _dev_tensor
    dcfg = cfg.replace(batch=batch)
    c = L.make_cfg(dcfg)
    T, H, dqk, ldc = cfg.seq, cfg.n_heads, cfg.qk_dim, cfg.kv_rank + cfg.rope_dim
    wsb = L.mla_recon_decode_workspace_size(c, T)
    if wsb == 0:
        return None
    g = torch.Generator(device="cuda").manual_seed(7)
    q = (torch.randn(batch, H, dqk, device="cuda", generator=g) * 0.5).to(torch.bfloat16)
    kv = torch.randn(batch, T, ldc, device="cuda", generator=g).to(torch.bfloat16)
    lens = torch.full((batch,), T, dtype=torch.int32, device="cuda")
    wuk, wuv = _dev_tensor(wl.Wuk, "bf16", "cuda"), _dev_tensor(wl.Wuv, "bf16", "cuda")
    o = torch.empty(batch, H, cfg.head_dim, dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream

    def run():
        L.mla_recon_decode(c, q.data_ptr(), kv.data_ptr(), T, lens.data_ptr(), wuk.data_ptr(),
                           wuv.data_ptr(), o.data_ptr(), ws.data_ptr(), wsb, stream)
    for _ in range(3):
        run()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(steps):
        run()
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / steps
    L.mla_recon_prof_enable(L.KC_ATTN_FWD, True)
    for _ in range(steps):
        run()
    attn = L.mla_recon_prof_read(L.KC_ATTN_FWD)
    L.mla_recon_prof_enable(L.KC_ATTN_FWD, False)
    attn_ms = attn["ms"] / steps
    cache_bytes = batch * T * ldc * 2
    return {"batch": batch, "cache_tokens": T, "ms_per_step": round(ms, 4),
            "value": round(batch / (ms / 1e3), 1), "unit": "tokens/s",
            "attention_kernel_ms": round(attn_ms, 4),
            "cache_GBps": round(cache_bytes / (attn_ms / 1e3) / 1e9, 1),
            "cache_frac_of_hbm_peak": round(cache_bytes / (attn_ms / 1e3) / 1e9 / PEAK_HBM_GBS, 4)}


def main():
    args = parse()
    if args.summarize_traffic:
        print(json.dumps(summarize_traffic(*args.summarize_traffic, args.calib_copy_mb or 1024), indent=1))
        return
    if args.summarize_counters:
        print(summarize_counters(args.summarize_counters, args.trace))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the reconstruction step is not sharded across "
              "GPUs (layers are independent); run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2607_27269_amd import _lib as L
    from paper_2607_27269_amd import configs, synth
    from paper_2607_27269_amd.step import DeviceStep

    if args.calib_copy_mb:
        n = args.calib_copy_mb * 1024 * 1024 // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    cfg = configs.get(args.config)
    wl = synth.make_workload(cfg)
    dev = DeviceStep(wl)
    # the step: teacher forward, student forward, Eq. 11 and the backward in one library call
    # (mla_recon_step: the shared frozen W_O applied to o_s - o_t; dL/dA_s not materialised,
    # the backward starts from (o_s - o_t) W_O^T W_O)
    for _ in range(args.warmup):
        dev.fused_step(with_dA=False)
    torch.cuda.synchronize()

    # headline: exactly `steps` steps, nothing else in the timed region
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        dev.fused_step(with_dA=False)
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    loss = float(dev.loss_buf[0].cpu())

    # also reported: the relative error on request (mla_recon_rel_error after the step; one
    # more [B T, H d_k] x [H d_k, D] product), timed alone over the same number of calls
    # also reported: the same step replayed as a HIP graph (captured once; the replays run
    # the same kernels on the same buffers without per-launch host work)
    ms_graph = None
    if not args.no_graph:
        graph = dev.capture_fused_step(with_dA=False)
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
        start.record()
        for _ in range(args.steps):
            graph.replay()
        stop.record()
        torch.cuda.synchronize()
        ms_graph = start.elapsed_time(stop) / args.steps
        del graph

    ms_rel = rel = None
    if not args.no_rel:
        dev.rel_error()
        torch.cuda.synchronize()
        start.record()
        for _ in range(args.steps):
            dev.rel_error()
        stop.record()
        torch.cuda.synchronize()
        ms_rel = start.elapsed_time(stop) / args.steps
        rel = float(dev.loss_buf[1].cpu())

    # also reported: the step with the teacher cached (its output depends only on h and the
    # frozen weights, so a training loop can compute it once per minibatch)
    ms_cached = None
    if not args.no_cached:
        dev.teacher_cache()
        dev.student_step(with_dA=False)
        torch.cuda.synchronize()
        start.record()
        for _ in range(args.steps):
            dev.student_step(with_dA=False)
        stop.record()
        torch.cuda.synchronize()
        ms_cached = start.elapsed_time(stop) / args.steps

    # also reported: a training iteration, the step followed by the AdamW update of the five
    # projections (its own copies of the weights, so the step timings above are unaffected)
    ms_train = None
    if not args.no_train:
        tr = DeviceStep(wl)
        tr.init_optimizer()
        for _ in range(2):
            tr.fused_step(with_dA=False)
            tr.optimizer_step(1e-4)
        torch.cuda.synchronize()
        start.record()
        for _ in range(args.steps):
            tr.fused_step(with_dA=False)
            tr.optimizer_step(1e-4)
        stop.record()
        torch.cuda.synchronize()
        ms_train = start.elapsed_time(stop) / args.steps
        del tr

    # also reported: calibration capture, one layer of the frozen stack (teacher forward with
    # W_O, then the residual update and RMS normalisation that give the next layer's input)
    ms_cap = None
    if not args.no_capture:
        x = dev.A_t.clone()
        h_next = torch.empty_like(dev.h)
        dt = L.MLA_FP32 if cfg.dtype == "fp32" else L.MLA_BF16

        def capture_layer():
            dev.teacher_fwd()
            L.mla_recon_residual_rmsnorm(x.data_ptr(), dev.A_t.data_ptr(), h_next.data_ptr(),
                                         cfg.tokens, cfg.hidden, dt, 1e-6, dev.stream)
        capture_layer()
        torch.cuda.synchronize()
        start.record()
        for _ in range(args.steps):
            capture_layer()
        stop.record()
        torch.cuda.synchronize()
        ms_cap = start.elapsed_time(stop) / args.steps
        del x, h_next

    decode = None if args.no_decode else decode_bench(cfg, wl, args.decode_batch, args.steps)

    # for reference: the four separate calls, which also form A_t and A_s (two W_O products)
    ms_sep = None
    if not args.no_separate:
        dev.step()
        torch.cuda.synchronize()
        start.record()
        for _ in range(args.steps):
            dev.step()
        stop.record()
        torch.cuda.synchronize()
        ms_sep = round(start.elapsed_time(stop) / args.steps, 4)

    # per-kernel-class times: the same steps again, each launch of a class bracketed by
    # HIP events on the launch stream (inside the library)
    classes = list(L.KCLASS_NAMES)
    for k in classes:
        L.mla_recon_prof_enable(k, True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        dev.fused_step(with_dA=False)
    stop.record()
    torch.cuda.synchronize()
    ms_instr = start.elapsed_time(stop) / args.steps
    kern = [dict(k, cls=L.KCLASS_NAMES[c]) for c in classes for k in L.mla_recon_prof_kernels(c)]
    prof = {L.KCLASS_NAMES[k]: L.mla_recon_prof_read(k) for k in classes}
    for k in classes:
        L.mla_recon_prof_enable(k, False)

    tokens = cfg.tokens
    flops = step_flops(cfg)
    tok_s = tokens / (ms / 1e3)

    def rate(p):
        """(bound, achieved, peak, unit) of a kernel's algorithmic work over its time"""
        if p["flops"] > 0:
            return "mfma", p["flops"] / (p["ms"] / 1e3) / 1e12, PEAK_BF16_TFLOPS, "TFLOP/s"
        return "hbm", p["bytes"] / (p["ms"] / 1e3) / 1e9, PEAK_HBM_GBS, "GB/s"
    # the dominant single kernel (one kernel function and template instance)
    top = max(kern, key=lambda k: k["ms"])
    bound, achieved, peak, unit = rate(top)
    kernels = []
    for k in sorted(kern, key=lambda k: -k["ms"]):
        kb, ka, kp, ku = rate(k)
        kernels.append({"kernel": k["kernel"], "ms_per_step": round(k["ms"] / args.steps, 4),
                        "launches_per_step": k["launches"] / args.steps, "bound": kb,
                        "achieved": round(ka, 1), "unit": ku, "frac": round(ka / kp, 4)})
    dom = max(prof, key=lambda k: prof[k]["ms"])
    cb, ca, cp, cu = rate(prof[dom])
    kernel_share = {k: round(v["ms"] / args.steps, 4) for k, v in prof.items()}
    # the other layer shapes (the tiny fp32 one is a parity case only)
    others = None
    if not args.no_other_configs:
        others = {str(i): time_config(i, args.steps, args.warmup) for i in (1, 2, 4) if i != args.config}
    out = {
        "metric": "calibration tokens/sec per layer (fwd+bwd recon)",
        "value": round(tok_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: B={cfg.batch} T={cfg.seq} D={cfg.hidden} "
                               f"H={cfg.n_heads} G={cfg.n_kv_groups} d_k={cfg.head_dim}; student "
                               f"r_q={cfg.q_rank} r_kv={cfg.kv_rank} d_nope={cfg.nope_dim} "
                               f"d_rope={cfg.rope_dim} G_kv={cfg.s_kv_groups} G_r={cfg.s_rope_groups}",
                   "global_batch": cfg.batch, "seq_len": cfg.seq, "parallelism": "none (1 GPU)"},
        "mfma_peak_frac": round(flops / (ms / 1e3) / (PEAK_BF16_TFLOPS * 1e12), 4),
        "alg_gflop_per_step": round(flops / 1e9, 1),
        "ms_per_step_instrumented": round(ms_instr, 4),
        "ms_per_step_separate_outputs": ms_sep,
        "train_step": None if ms_train is None else
                      {"ms_per_step": round(ms_train, 4), "optimizer": "AdamW",
                       "value": round(tokens / (ms_train / 1e3), 1), "unit": "tokens/s"},
        "capture": None if ms_cap is None else
                   {"ms_per_layer": round(ms_cap, 4),
                    "value": round(tokens / (ms_cap / 1e3), 1), "unit": "tokens/s per layer"},
        "decode_absorbed": decode,
        "graph_step": None if ms_graph is None else
                      {"ms_per_step": round(ms_graph, 4),
                       "value": round(tokens / (ms_graph / 1e3), 1), "unit": "tokens/s"},
        "cached_teacher": None if ms_cached is None else
                          {"ms_per_step": round(ms_cached, 4),
                           "value": round(tokens / (ms_cached / 1e3), 1), "unit": "tokens/s"},
        "kernel_ms_per_step": kernel_share,
        "roofline": {"kernel": top["kernel"], "bound": bound, "achieved": round(achieved, 2),
                     "peak": peak, "unit": unit, "frac": round(achieved / peak, 4),
                     "traffic": stored_traffic(top["kernel"]),
                     "launches_per_step": top["launches"] / args.steps,
                     "ms_per_launch": round(top["ms"] / top["launches"], 4),
                     "alg_per_launch": top["flops"] / top["launches"] if bound == "mfma"
                     else top["bytes"] / top["launches"]},
        "kernels": kernels,
        "class_roofline": {"class": f"{dom}: {L.KCLASS_KERNELS[dom]}", "bound": cb,
                           "achieved": round(ca, 2), "peak": cp, "unit": cu,
                           "frac": round(ca / cp, 4)},
        "other_configs": others,
        "loss": loss,
        "rel_error": None if ms_rel is None else
                     {"value": rel, "ms_per_call": round(ms_rel, 4),
                      "call": "mla_recon_rel_error after the step"},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, wl, min(args.cpu_seq, cfg.seq))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
