"""Throughput of one Early-Bird denoising step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--legs A,B]
                    [--no-cpu-baseline]
    python bench.py --ingest-counters DIR    (rocprofv3 FETCH_SIZE / WRITE_SIZE runs -> traffic)

A step is eb_decode_step over one batch of synthetic, seeded input already resident in HBM:
block attention over the cached prefix + block keys, the fused LM head with its
softmax / entropy / confidence / argmax reduction, and threshold unmasking in every block.
Prints ONE JSON line for the headline workload (default: the Dream-7B-shaped batch-64 step,
the largest configuration that fits one GPU): positions/s = block positions / step time, the
roofline of the fused LM-head kernel (timed with hipEvents recorded by the library around that
kernel), further workloads as nested legs with the same fields (default: the LLaDA-8B-shaped
batch-1 step, the HBM-bound case), and the fp64 CPU oracle timed on a bounded sample of the
headline workload.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import math
import os
import platform
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "block positions scored+unmasked/sec per denoising step; % HBM or MFMA peak"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA, TFLOP/s
MFMA_F32_PEAK_TFLOPS = 157.3    # fp32 vector peak (the fp32 path uses plain FMA)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "lmhead_traffic.json")
LMHEAD_SOURCES = [os.path.join(ROOT, "paper_2609_16450_amd", "csrc", f)
                  for f in ("lmhead.hip", "eb_common.hpp", "attn_small.hpp", "attn_common.hpp")]


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def lmhead_source_hash() -> str:
    """Hash of the code (comments and whitespace removed) of the LM-head launch's sources."""
    h = hashlib.sha256()
    for p in LMHEAD_SOURCES:
        with open(p, encoding="utf-8") as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def lmhead_work(cfg, T: int):
    """Algorithmic bytes and flops of one fused LM-head launch: W and h read once, 12 B of
    results per row (kappa, entropy, argmax); the logits are never written."""
    e = 4 if cfg.dtype == "f32" else 2
    nbytes = cfg.vocab * cfg.hidden * e + T * cfg.hidden * e + 12 * T
    flops = 2.0 * T * cfg.hidden * cfg.vocab
    return nbytes, flops


def attention_bytes(cfg, T: int, S: int) -> int:
    """Algorithmic bytes of the block attention: prefix K/V once, block Q/K/V in, O out."""
    e = 4 if cfg.dtype == "f32" else 2
    return 2 * S * cfg.hkv * cfg.head_dim * e + T * (2 * cfg.hq + 2 * cfg.hkv) * cfg.head_dim * e


def lmhead_kernel_name(dtype: str, T: int) -> str:
    """The LM-head kernel the library launches for T rows (the streaming kernel for at most 64
    bf16 rows, the tile kernel above)."""
    if dtype == "f32":
        return "lmhead_f32_kernel"
    return "lmhead_stream16_kernel" if T <= 64 else "lmhead_tile_kernel"


def measured_traffic(workload: str):
    """HBM bytes per launch from rocprofv3 counters, if taken on the current kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f).get(workload)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_hash") != lmhead_source_hash():
        return None
    return rec.get("bytes_per_launch")


def cpu_model() -> str:
    """The host CPU's model name from /proc/cpuinfo (platform.processor() gives only the ISA)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def cpu_baseline(case, budget_s: float = 15.0):
    """Time the fp64 oracle (as it stands) on a bounded sample of the workload.

    The oracle's step is block_attention, then lmhead_confidence, then unmask_select (what
    oracle.decode_step runs); the three are timed one after another so that each stage's time
    is reported, and their sum is the step time."""
    from threadpoolctl import threadpool_info, threadpool_limits

    import oracle
    from workloads import bf16_bits_to_f32

    threads = max(1, min(16, os.cpu_count() or 1))
    f = (lambda x: bf16_bits_to_f32(x)) if case.dtype == "bf16" else (lambda x: np.asarray(x))
    # sample: whole blocks from the front of the batch, at most 64 block positions
    nb, rows = 0, 0
    while nb < case.batch and (rows == 0 or rows + int(case.block_lens[nb]) <= 64):
        rows += int(case.block_lens[nb])
        nb += 1
    cu_b = case.cu_block[:nb + 1]
    cu_p = case.cu_prefix[:nb + 1]
    T, S = int(cu_b[-1]), int(cu_p[-1])
    w = f(case.w)
    q, kb, vb = f(case.q[:T]), f(case.k_blk[:T]), f(case.v_blk[:T])
    kp, vp, h = f(case.k_pre[:S]), f(case.v_pre[:S]), f(case.h[:T])
    stage = {"attention": 0.0, "lmhead_and_statistics": 0.0, "unmask": 0.0}
    reps, t_total = 0, 0.0
    with threadpool_limits(limits=threads):
        blas = [{k: d.get(k) for k in ("internal_api", "version", "num_threads", "threading_layer")}
                for d in threadpool_info() if d.get("user_api") == "blas"]
        while t_total < budget_s and reps < 50:
            t0 = time.perf_counter()
            oracle.block_attention(q, kb, vb, kp, vp, cu_b, cu_p, case.cfg.hq, case.cfg.hkv)
            t1 = time.perf_counter()
            st = oracle.lmhead_confidence(h, w)
            t2 = time.perf_counter()
            oracle.unmask_select(st["conf"], st["argmax"], case.masked[:T], case.tokens[:T],
                                 case.tau[:nb], cu_b)
            t3 = time.perf_counter()
            stage["attention"] += t1 - t0
            stage["lmhead_and_statistics"] += t2 - t1
            stage["unmask"] += t3 - t2
            t_total += t3 - t0
            reps += 1
    return {"value": reps * T / t_total, "unit": "positions/s", "cores": threads, "kind": "oracle",
            "sample": f"{reps} x the oracle's step (block_attention, lmhead_confidence, "
                      f"unmask_select) over the first {nb} block(s) of the workload ({T} block "
                      f"positions, full vocabulary {case.cfg.vocab}, prefix {S}), fp64 numpy, "
                      f"{t_total:.1f} s",
            "threads": threads, "host_cpu_count": os.cpu_count(), "cpu_model": cpu_model(),
            "blas": blas,
            "stage_seconds_per_step": {k: v / reps for k, v in stage.items()}}


SUFFIX_LEN = 256         # cached suffix rows per sequence on the dual-cache leg
LBS_WINDOW = 512         # generation window of the LBS leg (generation length 512, App. F)
TAU_PSI = 0.9            # LPS acceptance threshold on the lps leg
TOP_M = 2                # per-block budget on the topm leg


def timed(torch, stream, steps, run):
    """Milliseconds per call of run(i) over `steps` calls, host clock between synchronisations."""
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        run(i)
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / steps


def measured_peaks(torch, eb) -> dict:
    """Same-box reference rates beside the spec peaks: a 1 GiB device-to-device copy (read +
    write bytes per second), a bf16 8192^3 GEMM through torch's library path and the library's
    register-only bf16 MFMA loop (the matrix-core rate at the clock the chip holds under load)."""
    def ev_ms(fn, reps):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    copy_ms = ev_ms(lambda: dst.copy_(src), 10)
    del src, dst
    k = 8192
    x = torch.randn(k, k, device="cuda:0").to(torch.bfloat16)
    y = torch.randn(k, k, device="cuda:0").to(torch.bfloat16)
    gemm_ms = ev_ms(lambda: torch.mm(x, y), 10)
    del x, y
    groups, iters = 4096, 4096
    out = torch.empty(groups * 256, dtype=torch.float32, device="cuda:0")
    flops = eb.eb_probe_mfma_bf16(out, groups, iters)
    mfma_ms = ev_ms(lambda: eb.eb_probe_mfma_bf16(out, groups, iters), 5)
    del out
    return {"copy_GBps": 2 * n / (copy_ms * 1e-3) / 1e9,
            "gemm_bf16_TFLOPs": 2.0 * k ** 3 / (gemm_ms * 1e-3) / 1e12,
            "mfma_loop_bf16_TFLOPs": flops / (mfma_ms * 1e-3) / 1e12,
            "note": ("1 GiB device copy (read + write), bf16 8192^3 torch.mm, register-only bf16 "
                     "32x32x16 MFMA loop (eb_probe_mfma_bf16, 4096 groups x 4096 iterations); "
                     "same box, same run")}


def variant_leg(args, torch, eb, case, copies, stream) -> int:
    """The next-row paths: one JSON line with the same fields as the headline."""
    from workloads import lbs_window, router_scores, suffix_segment

    cfg, T, B = case.cfg, case.T, case.batch
    dev = "cuda:0"
    u8 = lambda n: torch.empty(max(n, 1), dtype=torch.uint8, device=dev)
    bf = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    dt_code = eb.EB_BF16 if cfg.dtype == "bf16" else eb.EB_F32
    extra = []
    for ds in copies:
        x = {"attn_ws": u8(eb.eb_block_attn_workspace(dt_code, ds.ragged, cfg.hq, cfg.hkv,
                                                       cfg.head_dim)),
             "lm_ws": u8(eb.eb_lmhead_features_workspace(dt_code, T, cfg.hidden, cfg.vocab)),
             "gap": torch.empty(T, device=dev), "feat": torch.empty((T, 4), device=dev),
             "pos": torch.empty(T, device=dev), "rho": torch.empty(B, device=dev),
             "p_psi": torch.from_numpy(router_scores(cfg.seed, "p_psi", T)).to(dev)}
        if args.path == "dual":
            cu_s, k_s, v_s = suffix_segment(cfg.seed, [SUFFIX_LEN] * B, cfg.hkv, cfg.head_dim,
                                            cfg.dtype)
            conv = (lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)) \
                if cfg.dtype == "bf16" else torch.from_numpy
            x.update(cu_s=torch.from_numpy(cu_s).to(dev), k_s=conv(k_s).to(dev),
                     v_s=conv(v_s).to(dev))
            from paper_2609_16450_amd.binding import eb_suffix
            x["attn_ws"] = u8(eb.load().eb_block_attn_dual_workspace(
                dt_code, ctypes.byref(ds.ragged.c()),
                ctypes.byref(eb_suffix(SUFFIX_LEN * B, SUFFIX_LEN, 0)), cfg.hq, cfg.hkv,
                cfg.head_dim))
        extra.append(x)
    if args.path == "lbs":
        m, p, xh = lbs_window(cfg.seed, B, LBS_WINDOW, cfg.vocab, cfg.vocab - 1)
        lb = [dict(m=torch.from_numpy(m).to(dev), p=torch.from_numpy(p).to(dev),
                   x=torch.from_numpy(xh).to(dev),
                   block=torch.empty((B, LBS_WINDOW), dtype=torch.uint8, device=dev),
                   size=torch.empty(B, dtype=torch.int32, device=dev),
                   first=torch.empty(B, dtype=torch.int32, device=dev)) for _ in copies]

    def run(i, lm_events=None):
        ds, x = copies[i % len(copies)], extra[i % len(copies)]
        if args.path == "lbs":
            L = lb[i % len(copies)]
            eb.eb_lbs_select(L["m"], L["p"], L["x"], cfg.vocab - 1, 4, 32, 5, L["block"],
                             L["size"], L["first"], stream=stream)
            return
        if args.path == "dual":
            eb.eb_block_attn_dual(ds.ragged, x["cu_s"], SUFFIX_LEN, ds.q, ds.k_blk, ds.v_blk,
                                  ds.k_pre, ds.v_pre, x["k_s"], x["v_s"], ds.attn_out,
                                  ws=x["attn_ws"], stream=stream)
        else:
            eb.eb_block_attn(ds.ragged, ds.q, ds.k_blk, ds.v_blk, ds.k_pre, ds.v_pre, ds.attn_out,
                             ws=x["attn_ws"], stream=stream)
        if lm_events:
            lm_events[0].record(stream)
        if args.path == "lps":
            eb.eb_lmhead_features(ds.h, ds.w, ds.conf, ds.entropy, ds.argmax, x["gap"],
                                  ds.max_logit, ws=x["lm_ws"], stream=stream)
        else:
            eb.eb_lmhead_confidence(ds.h, ds.w, ds.conf, ds.entropy, ds.argmax, ds.max_logit,
                                    ws=x["lm_ws"], stream=stream)
        if lm_events:
            lm_events[1].record(stream)
        if args.path == "lps":
            eb.eb_lps_features(ds.ragged, cfg.vocab, ds.conf, ds.entropy, x["gap"], ds.masked,
                               x["feat"], x["pos"], x["rho"], stream=stream)
            eb.eb_unmask_select_lps(ds.ragged, ds.conf, ds.argmax, ds.tau, x["p_psi"], TAU_PSI,
                                    ds.masked, ds.tokens, ds.unmask, ds.n_commit, ds.resolved,
                                    stream=stream)
        elif args.path == "topm":
            eb.eb_unmask_select_topm(ds.ragged, ds.conf, ds.argmax, ds.tau, TOP_M, ds.masked,
                                     ds.tokens, ds.unmask, ds.n_commit, ds.resolved,
                                     stream=stream)
        else:
            eb.eb_unmask_select(ds.ragged, ds.conf, ds.argmax, ds.tau, ds.masked, ds.tokens,
                                ds.unmask, ds.n_commit, ds.resolved, stream=stream)

    for i in range(args.warmup):
        run(i)
    ms = timed(torch, stream, args.steps, run)
    units = B * LBS_WINDOW if args.path == "lbs" else T
    config = {"workload": cfg.name, "path": args.path, "batch": B, "block_positions": T,
              "prefix_positions": case.S, "heads": f"{cfg.hq}/{cfg.hkv}x{cfg.head_dim}",
              "hidden": cfg.hidden, "vocab": cfg.vocab, "input_copies": len(copies)}
    if args.path == "lbs":
        nbytes = units * (1 + 4 + 4 + 1) + 8 * B   # masked, p_phi, x_hat in; block, size, first out
        roof = {"bound": "hbm", "achieved": nbytes / (ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                "traffic": None, "kernel": "lbs_select_kernel", "kernel_us": ms * 1e3,
                "algorithmic_bytes": nbytes, "algorithmic_flops": 0.0}
        config.update(window=LBS_WINDOW, l_min=4, l_b=32, g_max=5)
        metric, unit = "generation-window positions selected/sec (LBS post-pass)", "positions/s"
    else:
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
        for i, pair in enumerate(evs):
            run(i, pair)
        torch.cuda.synchronize()
        lm_ms = sum(a.elapsed_time(b) for a, b in evs) / len(evs)
        nbytes, flops = lmhead_work(cfg, T)
        if cfg.dtype == "f32":
            bound, peak, unit_r, achieved = "alu", MFMA_F32_PEAK_TFLOPS, "TFLOP/s", flops / (lm_ms * 1e-3) / 1e12
        elif flops / nbytes < (MFMA_BF16_PEAK_TFLOPS * 1e12) / (HBM_PEAK_GBS * 1e9):
            bound, peak, unit_r, achieved = "hbm", HBM_PEAK_GBS, "GB/s", nbytes / (lm_ms * 1e-3) / 1e9
        else:
            bound, peak, unit_r, achieved = "mfma", MFMA_BF16_PEAK_TFLOPS, "TFLOP/s", flops / (lm_ms * 1e-3) / 1e12
        roof = {"bound": bound, "achieved": achieved, "peak": peak, "unit": unit_r,
                "frac": achieved / peak, "traffic": None,
                "kernel": lmhead_kernel_name(cfg.dtype, T) + " + lmhead_combine_kernel",
                "kernel_us": lm_ms * 1e3, "algorithmic_bytes": nbytes, "algorithmic_flops": flops}
        if args.path == "dual":
            config["suffix_positions"] = SUFFIX_LEN * B
        if args.path == "lps":
            config["tau_psi"] = TAU_PSI
        if args.path == "topm":
            config["m"] = TOP_M
        metric, unit = METRIC, "positions/s"
    print(json.dumps({"metric": metric, "value": units / (ms * 1e-3), "unit": unit, "n_gpus": 1,
                      "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
                      "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
                      "dtype": cfg.dtype, "data": "synthetic", "config": config,
                      "roofline": roof}), flush=True)
    return 0


def roofline_of(cfg, T: int, S: int, kernel_ms: float, with_attn: bool) -> dict:
    """Roofline object of the fused LM-head launch: algorithmic bytes (W, h, results; plus the
    attention's Q, K, V and O when that launch also runs it) or flops over its duration, bound
    chosen by arithmetic intensity against the ridge of the spec peaks."""
    nbytes, flops = lmhead_work(cfg, T)
    if with_attn:
        nbytes += attention_bytes(cfg, T, S)
    ai = flops / nbytes
    if cfg.dtype == "f32":
        bound, peak, unit, achieved = "alu", MFMA_F32_PEAK_TFLOPS, "TFLOP/s", flops / (kernel_ms * 1e-3) / 1e12
    elif ai < (MFMA_BF16_PEAK_TFLOPS * 1e12) / (HBM_PEAK_GBS * 1e9):
        bound, peak, unit, achieved = "hbm", HBM_PEAK_GBS, "GB/s", nbytes / (kernel_ms * 1e-3) / 1e9
    else:
        bound, peak, unit, achieved = "mfma", MFMA_BF16_PEAK_TFLOPS, "TFLOP/s", flops / (kernel_ms * 1e-3) / 1e12
    return {"bound": bound, "achieved": achieved, "peak": peak, "unit": unit,
            "frac": achieved / peak, "traffic": measured_traffic(cfg.name),
            "kernel": lmhead_kernel_name(cfg.dtype, T), "kernel_us": kernel_ms * 1e3,
            "algorithmic_bytes": nbytes, "includes_attention": bool(with_attn),
            "algorithmic_flops": flops}


def step_leg(torch, eb, name: str, steps: int, warmup: int, n_copies: int, stream) -> tuple:
    """Time `steps` whole eb_decode_step calls of workload `name` (after `warmup`), then the same
    steps again with hipEvents recorded by the library around the fused LM-head kernel.
    Returns (fields of the JSON line, the generated case)."""
    from paper_2609_16450_amd.binding import eb_step_trace
    from paper_2609_16450_amd.device_case import DeviceStep
    from workloads import CONFIGS, make_step

    cfg = CONFIGS[name]
    log(f"bench: generating {cfg.name}")
    case = make_step(cfg)
    T = case.T
    copies = [DeviceStep(case, device="cuda:0") for _ in range(max(1, n_copies))]
    log(f"bench: {cfg.name} T={T} S={case.S} warmup={warmup} steps={steps}")

    def run(i, trace=None):
        ds = copies[i % len(copies)]
        eb.eb_decode_step(ds.buffers, stream=stream, trace=trace)

    for i in range(warmup):
        run(i)
    torch.cuda.synchronize()

    # K whole steps, host clock between two synchronisations (events beside it)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for i in range(steps):
        run(i)
    ev1.record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / steps
    ms_events = ev0.elapsed_time(ev1) / steps
    log(f"bench: {cfg.name} {ms_per_step:.4f} ms/step (events {ms_events:.4f})")

    # the same steps again with hipEvents recorded around the fused LM-head kernel, on the
    # step's stream
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    for a, b in evs:            # create the events
        a.record(stream)
        b.record(stream)
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(evs):
        run(i, eb_step_trace(0, 0, a.cuda_event, b.cuda_event, 0, 0))
    torch.cuda.synchronize()
    lm_ms = sum(a.elapsed_time(b) for a, b in evs) / len(evs)
    # in small steps the launch also runs the attention: count its algorithmic bytes as well
    with_attn = eb.eb_decode_step_attn_in_lmhead(copies[0].buffers)
    roof = roofline_of(cfg, T, case.S, lm_ms, with_attn)
    log(f"bench: {cfg.name} fused LM-head kernel {lm_ms * 1e3:.1f} us, "
        f"{roof['achieved']:.1f} {roof['unit']} ({100 * roof['frac']:.1f}%)")
    fields = {
        "value": T / (ms_per_step * 1e-3),
        "unit": "positions/s",
        "ms_per_step": ms_per_step,
        "dtype": cfg.dtype,
        "config": {"workload": cfg.name, "batch": cfg.batch, "block_positions": T,
                   "prefix_positions": case.S, "heads": f"{cfg.hq}/{cfg.hkv}x{cfg.head_dim}",
                   "hidden": cfg.hidden, "vocab": cfg.vocab, "input_copies": len(copies),
                   "ms_per_step_events": ms_events},
        "roofline": roof,
    }
    del copies
    torch.cuda.empty_cache()
    return fields, case


def ingest_counters(directory: str) -> int:
    """Turn rocprofv3 counter runs into profiles/lmhead_traffic.json.

    `directory` holds one rocprofv3 output folder per run, named <run>_FETCH_SIZE and
    <run>_WRITE_SIZE, each with a *counter_collection.csv: the run "copy" is
    `bench.py --calibrate-copy 1073741824` (three 1 GiB device-to-device copies); every other
    run is a bench.py step run whose workloads are listed in the file <run>.workloads (one name
    per line; a missing file means the run's name is the workload).  Each counter is averaged
    over the dispatches of the workload's fused LM-head kernel (matched by name), scaled by the
    factor that makes the copy's reading equal its true bytes (read for FETCH_SIZE, written for
    WRITE_SIZE), and stored with the hash of the kernel source it was taken on."""
    import csv
    import glob

    from workloads import CONFIGS, make_step

    def rows(run, counter):
        paths = glob.glob(os.path.join(directory, f"{run}_{counter}", "**",
                                       "*counter_collection.csv"), recursive=True)
        if not paths:
            raise SystemExit(f"no counter_collection.csv for {run}_{counter} under {directory}")
        out = []
        for p in paths:
            with open(p, newline="") as f:
                out += [r for r in csv.DictReader(f) if r["Counter_Name"] == counter]
        return out

    copy_bytes = 1 << 30
    factor = {}
    for counter in ("FETCH_SIZE", "WRITE_SIZE"):
        vals = [float(r["Counter_Value"]) for r in rows("copy", counter)
                if "copyBuffer" in r["Kernel_Name"]]
        vals = [v for v in vals if v > 0.25 * copy_bytes / 1024 / 2]   # the 1 GiB copies only
        if not vals:
            raise SystemExit(f"no 1 GiB copy dispatch in copy_{counter}")
        factor[counter] = (copy_bytes / 1024) / (sum(vals) / len(vals))
    runs = sorted({os.path.basename(d).rsplit("_", 2)[0]
                   for d in glob.glob(os.path.join(directory, "*_FETCH_SIZE"))} - {"copy"})
    try:
        with open(TRAFFIC_FILE) as f:
            table = json.load(f)
    except (OSError, ValueError):
        table = {}
    src_hash = lmhead_source_hash()
    for run in runs:
        wl_file = os.path.join(directory, f"{run}.workloads")
        names = ([ln.strip() for ln in open(wl_file) if ln.strip()] if os.path.exists(wl_file)
                 else [run])
        for name in names:
            cfg = CONFIGS[name]
            kernel = lmhead_kernel_name(cfg.dtype, make_step(cfg).T)
            rec = {"kernel": kernel}
            total = 0.0
            for counter, key in (("FETCH_SIZE", "fetch_kib"), ("WRITE_SIZE", "write_kib")):
                vals = [float(r["Counter_Value"]) for r in rows(run, counter)
                        if kernel in r["Kernel_Name"]]
                if not vals:
                    raise SystemExit(f"{run}_{counter}: no dispatch of {kernel}")
                rec[key] = sum(vals) / len(vals)
                rec.setdefault("dispatches", []).append(len(vals))
                total += rec[key] * 1024 * factor[counter]
            rec["bytes_per_launch"] = total
            rec["source_hash"] = src_hash
            table[name] = rec
            log(f"ingest: {name} {kernel} {total / 1e9:.4f} GB per launch")
    table["_note"] = (
        "HBM-side bytes per launch of the fused LM-head kernel from rocprofv3 FETCH_SIZE and "
        "WRITE_SIZE (KiB per dispatch, mean over the dispatches of the run), each scaled by what "
        f"the counter reads for a 1 GiB device-to-device copy: fetch factor "
        f"{factor['FETCH_SIZE']:.4f}, write factor {factor['WRITE_SIZE']:.4f}. source_hash = "
        "sha256 of the code of lmhead.hip, eb_common.hpp, attn_small.hpp and attn_common.hpp "
        "with comments and whitespace removed (first 16 hex digits) when the counters were "
        "taken. Written by `python bench.py --ingest-counters DIR`; commands in "
        "profiles/lmhead_counters.md. For a batch-1 step the launch also runs the step's block "
        "attention (queued behind the vocabulary slices), whose bytes are included.")
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(dict(sorted(table.items())), f, indent=1)
        f.write("\n")
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="dream7b_b64",
                    help="headline workload (default: the batch-64 Dream-7B-shaped step)")
    ap.add_argument("--legs", default="llada8b_b1",
                    help="comma-separated further workloads timed as nested legs of the same "
                         "line (default: the batch-1 LLaDA-8B-shaped step; '' for none)")
    ap.add_argument("--copies", type=int, default=2, help="input copies rotated between steps")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="only run 3 device-to-device copies of BYTES (calibrates HBM counters)")
    ap.add_argument("--ingest-counters", metavar="DIR",
                    help="write profiles/lmhead_traffic.json from rocprofv3 counter runs in DIR")
    ap.add_argument("--no-peaks", action="store_true",
                    help="skip the same-box copy and GEMM reference rates (e.g. under a profiler)")
    ap.add_argument("--path", default="step", choices=["step", "lps", "topm", "dual", "lbs"],
                    help="step: eb_decode_step (the headline); lps: attention + LM head with the "
                         "top-2 gap + LPS features + union accept rule; topm: attention + LM head "
                         "+ top-m commit; dual: dual-cache attention + LM head + unmask; lbs: the "
                         "LBS post-pass over a 512-position generation window per sequence")
    args = ap.parse_args()

    if args.ingest_counters:
        return ingest_counters(args.ingest_counters)
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the step is built and timed on a single MI355X "
              "(how the step would shard across GPUs is a design note only).", file=sys.stderr)
        return 2

    import torch

    import paper_2609_16450_amd as eb
    from paper_2609_16450_amd.device_case import DeviceStep
    from workloads import CONFIGS, make_step

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    if args.calibrate_copy:
        src = torch.ones(args.calibrate_copy, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": args.calibrate_copy, "copies": 3}), flush=True)
        return 0
    eb.load()
    stream = torch.cuda.current_stream()

    if args.path != "step":
        cfg = CONFIGS[args.workload]
        log(f"bench: generating {cfg.name}")
        case = make_step(cfg)
        copies = [DeviceStep(case, device="cuda:0") for _ in range(max(1, args.copies))]
        log(f"bench: T={case.T} S={case.S} warmup={args.warmup} steps={args.steps}")
        return variant_leg(args, torch, eb, case, copies, stream)

    # the legs run first, each with its inputs freshly allocated and freed afterwards, then the
    # headline workload
    legs = {}
    for name in [x.strip() for x in args.legs.split(",") if x.strip() and x.strip() != args.workload]:
        leg, _ = step_leg(torch, eb, name, args.steps, args.warmup, args.copies, stream)
        legs[name] = leg
    head, case = step_leg(torch, eb, args.workload, args.steps, args.warmup, args.copies, stream)
    result = {
        "metric": METRIC,
        "value": head["value"],
        "unit": head["unit"],
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": head["dtype"],
        "data": "synthetic",
        "config": head["config"],
        "roofline": head["roofline"],
    }
    if legs:
        result["legs"] = legs
    if not args.no_peaks:
        result["roofline"]["measured_peak"] = measured_peaks(torch, eb)
        log(f"bench: measured peaks {result['roofline']['measured_peak']}")
    if not args.no_cpu_baseline:
        log("bench: timing the fp64 oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(case)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
