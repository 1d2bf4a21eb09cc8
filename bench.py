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
    p.add_argument("--no-cached", action="store_true",
                   help="skip the timing of the cached-teacher step (profiling runs)")
    p.add_argument("--no-train", action="store_true",
                   help="skip the timing of the step plus the AdamW update (profiling runs)")
    p.add_argument("--no-capture", action="store_true",
                   help="skip the timing of calibration capture (profiling runs)")
    p.add_argument("--no-decode", action="store_true",
                   help="skip the timing of absorbed-form decoding (profiling runs)")
    p.add_argument("--decode-batch", type=int, default=64,
                   help="sequences per decoding step (each with a full-length cache)")
    p.add_argument("--cpu-seq", type=int, default=4096, help="oracle sample: tokens of one sequence")
    p.add_argument("--calib-copy-mb", type=int, default=0,
                   help="run one device-to-device copy of this many MiB first (HBM counter calibration)")
    p.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                   help="turn two rocprofv3 --pmc counter_collection.csv files (FETCH_SIZE, WRITE_SIZE) "
                        "of a --calib-copy-mb run into per-class HBM bytes per launch; print JSON")
    return p.parse_args()


# kernel-name fragments of each timing class, as rocprofv3 reports them
# kernel-name patterns of each timing class: a kernel belongs to the class when every
# substring of one of the alternatives occurs in its name
CLASS_PATTERNS = {
    "gemm_nt": [("gemm_mfma_kernel<", ", true, true,"), ("gemm_mfma_persist_kernel<", ", true, true,")],
    "gemm_nn": [("gemm_mfma_kernel<", ", true, false,"), ("gemm_mfma_persist_kernel<", ", true, false,")],
    "gemm_tn": [("gemm_mfma_kernel<", ", false, false,"), ("gemm_mfma_persist_kernel<", ", false, false,")],
    "attn_fwd": [("attn_fwd_mfma_kernel<",), ("attn_fwd_persist_kernel<",)],
    "attn_bwd_dkdv": [("attn_dv_mfma_kernel<",), ("attn_dkdv_mfma_kernel<",)],
    "attn_bwd_dq": [("attn_ds_gemm_kernel<", ", false, false,"), ("attn_ds_gemm_persist_kernel<", ", false, false,"),
                    ("attn_dq_mfma_kernel<",)],
    "attn_bwd_dk": [("attn_ds_gemm_kernel<", ", true, false,"), ("attn_ds_gemm_persist_kernel<", ", true, false,")],
    "loss": [("loss_main_kernel<",)],
}


def _in_class(name, alts):
    return any(all(p in name for p in pats) for pats in alts)


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
    """HBM bytes per launch of each timing class from FETCH_SIZE / WRITE_SIZE (KiB per
    dispatch), each scaled so that the calibration copy reads and writes copy_mb MiB."""
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
        # the calibration copy is the largest non-library dispatch named like a copy
        cands = [v for (i, n), v in d.items() if "copy" in n.lower() or "Copy" in n]
        return max(cands) if cands else None
    fc, wc = copy_value(fetch), copy_value(write)
    out = {"copy_mb": copy_mb, "fetch_scale": known / fc if fc else None,
           "write_scale": known / wc if wc else None, "classes": {}}
    for cls, alts in CLASS_PATTERNS.items():
        fv = [v for (i, n), v in fetch.items() if _in_class(n, alts)]
        wv = [v for (i, n), v in write.items() if _in_class(n, alts)]
        if not fv or not wv or not fc or not wc:
            continue
        out["classes"][cls] = {"launches": len(fv),
                               "bytes_per_launch": (sum(fv) * out["fetch_scale"] + sum(wv) * out["write_scale"]) / len(fv),
                               "read_bytes_per_launch": sum(fv) * out["fetch_scale"] / len(fv),
                               "write_bytes_per_launch": sum(wv) * out["write_scale"] / len(wv)}
    out["sources_sha1"] = sources_digest()
    return out


def stored_traffic(cls):
    """Counter-derived HBM bytes per launch for `cls`, if taken on the current sources."""
    try:
        with open(TRAFFIC_FILE) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("sources_sha1") != sources_digest():
        return None
    c = t.get("classes", {}).get(cls)
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
    prof = {L.KCLASS_NAMES[k]: L.mla_recon_prof_read(k) for k in classes}
    for k in classes:
        L.mla_recon_prof_enable(k, False)

    loss = float(dev.loss_buf[0])
    tokens = cfg.tokens
    # algorithmic work of the step as run: the two W_O products and dA W_O replaced by
    # W_O^T W_O and one product with it
    HV = cfg.n_heads * cfg.head_dim
    flops = (cfg.total_flops() - 3 * cfg.flops()["T4_wo"] + 2.0 * HV * HV * cfg.hidden
             + 2.0 * cfg.tokens * HV * HV)
    tok_s = tokens / (ms / 1e3)
    dom = max(prof, key=lambda k: prof[k]["ms"])
    p = prof[dom]
    bound = "mfma" if p["flops"] > 0 else "hbm"
    if bound == "mfma":
        achieved = p["flops"] / (p["ms"] / 1e3) / 1e12
        peak, unit = PEAK_BF16_TFLOPS, "TFLOP/s"
    else:
        achieved = p["bytes"] / (p["ms"] / 1e3) / 1e9
        peak, unit = PEAK_HBM_GBS, "GB/s"
    kernel_share = {k: round(v["ms"] / args.steps, 4) for k, v in prof.items()}
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
        "cached_teacher": None if ms_cached is None else
                          {"ms_per_step": round(ms_cached, 4),
                           "value": round(tokens / (ms_cached / 1e3), 1), "unit": "tokens/s"},
        "kernel_ms_per_step": kernel_share,
        "roofline": {"kernel": f"{dom}: {L.KCLASS_KERNELS[dom]}", "bound": bound, "achieved": round(achieved, 2),
                     "peak": peak, "unit": unit, "frac": round(achieved / peak, 4),
                     "traffic": stored_traffic(dom),
                     "launches_per_step": p["launches"] / args.steps},
        "loss": loss,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, wl, min(args.cpu_seq, cfg.seq))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
