"""Throughput of the compressed ternary GEMV stack on one MI355X.

One step = one token through a synthetic linear stack: every layer's fused
QKV, O, fused gate_up and down GEMV, each matrix with its own seeded weights
and its own seeded activations.  Weights are packed once (untimed) and stay
resident in HBM, as do the activations, before the timed region.

Two executions of the same step are timed:
  grouped  one qtea_grouped_gemv launch computes all of the token's GEMVs
           (their inputs are independent, as generated); the weight stream
           runs back to back across matrices.  This is `value`.
  chained  one qtea_gemm_lowbatch launch per GEMV, in order on one stream,
           captured as one HIP graph (the paper times per-token latency with
           CUDA Graph); each launch starts after the previous one ends, as in
           a decoder where each product feeds the next.  Reported beside it.

Default workload: the 32-layer Llama-3-8B-shaped stack at batch 1
(1.48 GB of packed weights per token, far beyond the 256 MB last-level
cache, so every token streams its weights from HBM).

Printed: one JSON line with the weight-stream GB/s (algorithmic bytes per
token / time per token), us per token, the roofline of the dominant kernel
(timed live with HIP events around graph replays on its stream), the
chained figures and the CPU oracle baseline.
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

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def build_stack(wl, B, dev, seed, layers=None):
    import numpy as np
    import torch

    import paper_2609_00224_amd as q
    import synth

    mats = []
    t0 = time.time()
    for layer, mat, role, N, K in wl.matrices():
        if layers is not None and layer >= layers:
            break
        L = synth.layer_inputs(seed, layer, mat, N, K, p0=wl.p0, frac=wl.frac, resid=wl.resid,
                               groups=wl.groups)
        x = synth.activations(seed, layer, mat, B, K)
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        nS = int(L["S"].size)
        if wl.groups:
            pm = q.pack_matrix_g128(t(L["trits"]), t(L["alpha_g"]), t(L["beta_g"]), t(L["v"]), t(L["bitmap"]), nS,
                                    t(L["R8"]), t(L["idx"]))
        elif wl.resid == "e4m3":
            pm = q.pack_matrix_e4m3(t(L["trits"]), t(L["alpha"]), t(L["v"]), t(L["bitmap"]), nS, t(L["R8"]),
                                    t(L["idx"]))
        else:
            pm = q.pack_matrix(t(L["trits"]), t(L["alpha"]), t(L["v"]), t(L["S"]), t(L["R"]), t(L["idx"]))
        mats.append({
            "layer": layer, "mat": mat, "role": role, "N": N, "K": K, "nS": nS, "pm": pm, "x": t(x),
            "y": torch.empty((B, N), dtype=torch.float32, device=dev),
            "bytes": (q.algorithmic_bytes_g128(N, K, nS) if wl.groups else
                      q.algorithmic_bytes(N, K, nS, value_bytes=1 if wl.resid == "e4m3" else 2)),
        })
        if layer == 0 or (layer + 1) % 8 == 0 and mat == len(wl.shapes) - 1:
            log(f"packed layer {layer} {role} {N}x{K} ({time.time() - t0:.1f}s)")
    torch.cuda.synchronize()
    return mats


def capture(mats, B, ws, stream):
    import torch

    import paper_2609_00224_amd as q

    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(stream):
        # one eager pass first (module load, workspace counters settle)
        for m in mats:
            q.qtea_gemm_lowbatch(m["pm"].desc, m["pm"].packed, m["x"], B, m["y"], ws, stream=stream)
        stream.synchronize()
        with torch.cuda.graph(g, stream=stream):
            for m in mats:
                q.qtea_gemm_lowbatch(m["pm"].desc, m["pm"].packed, m["x"], B, m["y"], ws, stream=stream)
    stream.synchronize()
    return g


def capture_grouped(gp, stream):
    import torch

    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(stream):
        gp.run(stream=stream)
        stream.synchronize()
        with torch.cuda.graph(g, stream=stream):
            gp.run(stream=stream)
    stream.synchronize()
    return g


def time_graph(g, stream, reps, warmup):
    import torch

    with torch.cuda.stream(stream):
        for _ in range(warmup):
            g.replay()
        stream.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            g.replay()
        e1.record(stream)
    e1.synchronize()
    return e0.elapsed_time(e1) / reps  # ms per replay


def time_calls(fn, stream, reps, warmup):
    """ms per call of fn() (which enqueues one step on `stream`), called back
    to back: `warmup` calls, a synchronize, then `reps` calls between two
    events on the stream."""
    import torch

    with torch.cuda.stream(stream):
        for _ in range(warmup):
            fn()
        stream.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
    e1.synchronize()
    return e0.elapsed_time(e1) / reps


def replay_spread(g, stream, reps):
    """Median, p10 and p90 of single replays, each between its own pair of
    events (a separate pass after the timed one)."""
    import numpy as np
    import torch

    ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    with torch.cuda.stream(stream):
        ev[0].record(stream)
        for i in range(reps):
            g.replay()
            ev[i + 1].record(stream)
    ev[-1].synchronize()
    us = np.array([ev[i].elapsed_time(ev[i + 1]) * 1e3 for i in range(reps)])
    p10, p50, p90 = np.percentile(us, [10, 50, 90])
    return {"median": round(float(p50), 2), "p10": round(float(p10), 2), "p90": round(float(p90), 2),
            "replays": reps}


def kernel_name(B, grouped=False, rows_per_panel=1024, e4m3=False, g128=False):
    f8 = "true" if e4m3 else "false"
    # the grouped format runs every batch row through the batch-1 table kernel
    if grouped and g128:
        return f"grouped_gemv_kernel<{rows_per_panel // 128}, true, true>"
    if g128:
        return "grouped_gemv_kernel<4, true, true, true>"
    if grouped and B > 1:
        # hi/lo activation halves in one or two MFMAs
        return f"grouped_mma_kernel<{1 if B <= 8 else 2}, {f8}>"
    if grouped:
        return f"grouped_gemv_kernel<{rows_per_panel // 128}, {f8}, false>"  # 8 waves x 16 rows per row block
    # one matrix per launch (qtea_gemm_lowbatch): the same kernels in their single-problem form
    if B > 1:
        return f"grouped_mma_kernel<{1 if B <= 8 else 2}, {f8}, true>"
    return f"grouped_gemv_kernel<4, {f8}, {'true' if g128 else 'false'}, true>"


def traffic_per_launch(kernel, algorithmic_bytes, workload="llama3_8b_stack batch 1"):
    """HBM bytes per launch from the committed counter summary, if it was
    taken on this kernel and workload and on the current kernel source
    (sha256 recorded in the summary)."""
    import hashlib

    path = os.path.join(ROOT, "profiles", "traffic_grouped_gemv_b1_llama3_8b_stack.txt")
    srcs = ["grouped.hip", "grouped_plan.h", "plan_host.h", "qtea_internal.h"]
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if "=" in line and not line.lstrip().startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    h = hashlib.sha256()
    for f in srcs:  # the kernel's source file, then the shared headers
        h.update(open(os.path.join(ROOT, "paper_2609_00224_amd", "csrc", f), "rb").read())
    digest = h.hexdigest()
    if kv.get("kernel") != kernel or kv.get("source_sha256") != digest or kv.get("workload") != workload:
        return None
    try:
        return int(float(kv["hbm_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def read_ceiling(dev, stream, nbytes=2 << 30, warm=200, reps=20, passes=5):
    """GB/s of the library's plain streaming-read kernel over a buffer far
    beyond the last-level cache (16-byte non-temporal loads, nothing else),
    after `warm` launches of sustained load; the best of `passes` timed
    passes of `reps` launches, and their mean."""
    import torch

    import paper_2609_00224_amd as q

    buf = torch.ones(nbytes, dtype=torch.uint8, device=dev)
    sink = torch.zeros(q.read_ceiling_sink_words(nbytes), dtype=torch.int32, device=dev)
    rates = []
    with torch.cuda.stream(stream):
        for _ in range(warm):
            q.qtea_read_ceiling(buf, sink, stream=stream)
        for _ in range(passes):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                q.qtea_read_ceiling(buf, sink, stream=stream)
            e1.record(stream)
            e1.synchronize()
            rates.append(nbytes * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9)
    del buf
    return max(rates), sum(rates) / len(rates)


def gpu_clock():
    """Current shader clock level as the driver reports it, if readable."""
    import glob

    for path in sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk")):
        try:
            for line in open(path):
                if "*" in line:
                    return line.split(":", 1)[1].replace("*", "").strip()
        except OSError:
            continue
    return None


def copy_calibration(nbytes, dev):
    """A plain device copy of known size, for scaling the HBM counters."""
    import torch

    n = nbytes // 4
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        torch.neg(src, out=dst)  # one elementwise kernel: reads and writes 4n bytes
    torch.cuda.synchronize()
    log(f"copy calibration: {4 * n} bytes read and written per launch, 3 launches")


def cpu_baseline(mats, wl, seed, B, min_s=10.0):
    """The oracle (plain fp64 C, OpenMP over rows) over whole tokens of the
    same stack: every matrix once per pass, passes repeated until at least
    `min_s` seconds of oracle time.  The first pass also reports how far the
    GPU outputs of every matrix are from it."""
    import numpy as np

    import oracle
    import synth

    nthreads = oracle.threads()
    token_bytes = sum(m["bytes"] for m in mats)
    inputs = []
    worst = 0.0
    t_oracle = 0.0
    for m in mats:
        L = synth.layer_inputs(seed, m["layer"], m["mat"], m["N"], m["K"], p0=wl.p0, frac=wl.frac,
                               resid=wl.resid, groups=wl.groups)
        if wl.resid == "e4m3":
            L["R"] = oracle.e4m3_as_half(L["R8"])
        x = synth.activations(seed, m["layer"], m["mat"], B, m["K"])
        if wl.groups:
            gemv = oracle.gemv128
            args = (m["N"], m["K"], oracle.pack128(L.pop("trits")), L["alpha_g"], L["beta_g"], L["v"], L["S"],
                    L["R"], L["idx"], x)
        else:
            gemv = oracle.gemv
            args = (m["N"], m["K"], oracle.pack(L.pop("trits")), L["alpha"], L["v"], L["S"], L["R"], L["idx"], x)
        t0 = time.perf_counter()
        y = gemv(*args, nthreads=nthreads)
        t_oracle += time.perf_counter() - t0
        yg = m["y"].cpu().numpy().astype(np.float64)
        rel = np.linalg.norm(yg - y, axis=1) / np.linalg.norm(y, axis=1)
        worst = max(worst, float(rel.max()))
        inputs.append(args)
    passes = 1
    while t_oracle < min_s:
        for args in inputs:
            t0 = time.perf_counter()
            gemv(*args, nthreads=nthreads)
            t_oracle += time.perf_counter() - t0
        passes += 1
    us_token = t_oracle / passes * 1e6
    single = None
    if len(inputs) <= 4:  # the single GEMV and the one-layer workloads: one thread as well
        t1, p1 = 0.0, 0
        while t1 < min_s / 2:
            for args in inputs:
                t0 = time.perf_counter()
                gemv(*args, nthreads=1)
                t1 += time.perf_counter() - t0
            p1 += 1
        single = {"value": round(token_bytes * p1 / t1 / 1e9, 4), "unit": "GB/s", "cores": 1,
                  "us_per_step": round(t1 / p1 * 1e6, 1)}
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {
        "value": round(token_bytes * passes / t_oracle / 1e9, 4),
        "unit": "GB/s",
        "cores": nthreads,
        "kind": "oracle",
        "sample": f"{passes} whole tokens of {wl.name} at batch {B} ({len(mats)} GEMVs, "
                  f"{token_bytes / 1e9:.3f} GB of packed weights each), {t_oracle:.1f} s of oracle time",
        "us_per_token": round(us_token, 1),
        "single_thread": single,
        "gpu_vs_oracle_max_rel_l2": worst,
        "host": {"cpu_model": model, "usable_cores": len(os.sched_getaffinity(0)), "nproc": os.cpu_count()},
    }


FP64_PEAK_TFLOPS = 78.6  # MI355X dense fp64 (vector and matrix)
QUANT_LAYER = (("qkv", 6144, 4096), ("o", 4096, 4096), ("gate_up", 28672, 4096), ("down", 4096, 14336))
QUANT_SALIENT = 0.05  # the paper's salient-column fraction
QUANT_LAMBDA = 1.0
QUANT_ITERS = 2


def cold_main(args):
    """Warm and cold timing of a small workload (one GEMV, one layer), each
    as C steps back to back in one graph: warm repeats one copy, whose packed
    bytes stay in the caches; cold walks C copies, each its own seeded
    weights, so every step streams its weights from HBM."""
    import dataclasses

    import torch

    import paper_2609_00224_amd as q
    import synth
    from synth.workloads import WORKLOADS

    q.load()
    assert torch.cuda.is_available(), "no GPU"
    dev = torch.device("cuda:0")
    base = WORKLOADS[args.workload]
    assert base.layers == 1, "--cold-copies takes a one-layer workload"
    C, B = args.cold_copies, args.batch
    seed = synth.DEFAULT_SEED if args.seed is None else args.seed
    mats = build_stack(dataclasses.replace(base, layers=C), B, dev, seed)
    per = len(base.shapes)
    copies = [mats[i * per:(i + 1) * per] for i in range(C)]
    step_bytes = sum(m["bytes"] for m in copies[0])
    stream = torch.cuda.Stream(device=dev)
    plans = [q.plan_grouped([m["pm"] for m in c], [m["x"] for m in c], [m["y"] for m in c], batch=B) for c in copies]
    ws = torch.zeros(max(max(q.qtea_workspace_bytes(m["pm"].desc, B) for m in mats), 4), dtype=torch.uint8,
                     device=dev)

    def graph(fn):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.stream(stream):
            fn()
            stream.synchronize()
            with torch.cuda.graph(g, stream=stream):
                fn()
        stream.synchronize()
        return g

    def grouped(cs):
        return lambda: [plans[i].run(stream=stream) for i in cs]

    def chained(cs):
        return lambda: [q.qtea_gemm_lowbatch(m["pm"].desc, m["pm"].packed, m["x"], B, m["y"], ws, stream=stream)
                        for i in cs for m in copies[i]]

    res = {}
    for name, mk in (("grouped", grouped), ("chained", chained)):
        # both graphs run C steps back to back; warm repeats copy 0, cold walks the copies
        reps, warm_reps = max(1, args.steps // C), max(1, args.warmup // C)
        warm = time_graph(graph(mk([0] * C)), stream, reps, warm_reps) / C
        cold = time_graph(graph(mk(range(C))), stream, reps, warm_reps) / C
        res[name] = {"warm_us": round(warm * 1e3, 2), "cold_us": round(cold * 1e3, 2),
                     "warm_gbs": round(step_bytes / (warm * 1e-3) / 1e9, 1),
                     "cold_gbs": round(step_bytes / (cold * 1e-3) / 1e9, 1)}
        log(f"{base.name} B={B} {name}: warm {res[name]['warm_us']} us ({res[name]['warm_gbs']} GB/s), cold "
            f"{res[name]['cold_us']} us ({res[name]['cold_gbs']} GB/s) over {C} copies "
            f"({C * step_bytes / 1e6:.0f} MB)")
    out = {"metric": "weight-stream GB/s and us per step, warm and cold", "unit": "GB/s",
           "value": res["grouped"]["cold_gbs"], "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
           "config": {"workload": base.name, "batch": B, "copies": C, "bytes_per_step": step_bytes,
                      "cold_bytes": C * step_bytes, "seed": seed},
           "grouped": res["grouped"], "chained": res["chained"]}
    print(json.dumps(out), flush=True)


def quantizer_main(args):
    """Offline quantizer: Hessian and quantization of the four matrices of
    one Llama-3-8B-shaped layer (synthetic full-precision weights and
    calibration rows); one step = all four matrices."""
    import torch

    import paper_2609_00224_amd as q
    import synth

    q.load()
    assert torch.cuda.is_available(), "no GPU"
    dev = torch.device("cuda:0")
    seed = synth.DEFAULT_SEED if args.seed is None else args.seed
    mats = []
    for i, (role, N, K) in enumerate(QUANT_LAYER):
        W, X = synth.quant_inputs(seed + i, N, K, args.calib_rows)
        mats.append({"role": role, "N": N, "K": K, "W": torch.from_numpy(W).to(dev), "X": torch.from_numpy(X).to(dev),
                     "H": torch.empty((K, K), dtype=torch.float64, device=dev),
                     "nS": synth.n_salient(K, QUANT_SALIENT)})
        log(f"quantizer input {role} {N}x{K} ready")
    weights = sum(m["N"] * m["K"] for m in mats)

    # The matrices are independent and the library is reentrant: each gets
    # its own stream and host thread (the column phase of one matrix keeps
    # only a few dozen CUs busy, so the four overlap).
    from concurrent.futures import ThreadPoolExecutor

    streams = [torch.cuda.Stream(device=dev) for _ in mats]
    pool = ThreadPoolExecutor(max_workers=len(mats)) if args.quant_concurrent else None

    def one(m, st, times):
        with torch.cuda.stream(st):
            t0 = time.perf_counter()
            q.qtea_quant_hessian(m["X"], m["H"], stream=st)
            st.synchronize()
            t1 = time.perf_counter()
            m["out"] = q.quantize_matrix(m["W"], m["H"], m["nS"], lambda_decay=QUANT_LAMBDA, iters=QUANT_ITERS,
                                         stream=st)
            t2 = time.perf_counter()
        if times is not None:
            times.setdefault(m["role"], []).append((t1 - t0, t2 - t1))

    def step(times=None):
        if pool is None:
            for m, st in zip(mats, streams):
                one(m, st, times)
        else:
            for f in [pool.submit(one, m, st, times) for m, st in zip(mats, streams)]:
                f.result()

    for _ in range(args.warmup):
        step()
    times = {}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(times)
    torch.cuda.synchronize()
    sec = (time.perf_counter() - t0) / args.steps
    per = {m["role"]: {"N": m["N"], "K": m["K"],
                       "hessian_ms": round(1e3 * sum(a for a, _ in times[m["role"]]) / args.steps, 2),
                       "quantize_ms": round(1e3 * sum(b for _, b in times[m["role"]]) / args.steps, 2)}
           for m in mats}
    for r, v in per.items():
        log(f"  {r:8s} {v['N']}x{v['K']}: hessian {v['hessian_ms']} ms, quantize {v['quantize_ms']} ms")
    log(f"quantizer: {weights / sec / 1e6:.1f} M weights/s ({sec * 1e3:.1f} ms per layer)")
    # algorithmic fp64 work per step: Hessian 2 n K^2, reverse Cholesky K^3/3,
    # triangular inverse K^3/3, GPTQ error updates 2 N K (K - 1) / 2
    flops = sum(2.0 * args.calib_rows * m["K"] ** 2 + 2.0 * m["K"] ** 3 / 3 + float(m["N"]) * m["K"] * (m["K"] - 1)
                for m in mats)
    roof = {"bound": "alu", "achieved": round(flops / sec / 1e12, 3), "peak": FP64_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(flops / sec / 1e12 / FP64_PEAK_TFLOPS, 4), "traffic": None,
            "kernel": "whole quantizer (all kernels of the step)", "flops_per_step": flops}
    cpu = None
    if not args.no_cpu_baseline:
        cpu = quantizer_cpu_baseline(mats[1], seed + 1, args.calib_rows)
        log(f"oracle: {cpu['value'] / 1e6:.2f} M weights/s on the {cpu['sample']}; GPU outputs equal: "
            f"{cpu['gpu_vs_oracle']}")
    out = {
        "metric": "offline QTEA quantization rate, one Llama-3-8B-shaped layer (Hessian + quantize)",
        "value": round(weights / sec, 1), "unit": "weights/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(sec * 1e3, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": "llama3_8b_layer_quantize", "matrices": [list(x) for x in QUANT_LAYER],
                   "calib_rows": args.calib_rows, "salient_frac": QUANT_SALIENT, "lambda_decay": QUANT_LAMBDA,
                   "iters": QUANT_ITERS, "seed": seed,
                   "execution": "four streams, one host thread each" if args.quant_concurrent else "sequential"},
        "per_matrix": per,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def quantizer_cpu_baseline(m, seed, calib_rows):
    """The quantizer oracle (fp64 numpy) on one whole matrix of the layer,
    timed, and the GPU's outputs for that matrix compared with it."""
    import numpy as np

    import synth
    from oracle import quantizer as qz

    W, X = synth.quant_inputs(seed, m["N"], m["K"], calib_rows)
    t0 = time.perf_counter()
    ref = qz.quantize(W, qz.hessian(X), m["nS"], lam=QUANT_LAMBDA, iters=QUANT_ITERS)
    t = time.perf_counter() - t0
    o = m["out"]
    f16 = lambda a: np.asarray(a, np.float16).view(np.uint16)
    eq = {
        "codes": bool(np.array_equal(o["T"].cpu().numpy(), ref["T"])),
        "alpha_beta_v": bool(np.array_equal(o["alpha"].cpu().numpy().view(np.uint16), f16(ref["alpha"]))
                             and np.array_equal(o["beta"].cpu().numpy().view(np.uint16), f16(ref["beta"]))
                             and np.array_equal(o["v"].cpu().numpy().view(np.uint16), f16(ref["v"]))),
        "salient_and_residual": bool(np.array_equal(o["S"].cpu().numpy(), ref["S"])
                                     and np.array_equal(o["R8"].cpu().numpy(), ref["rval"])
                                     and np.array_equal(o["idx"].cpu().numpy(), ref["ridx"])),
    }
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": round(m["N"] * m["K"] / t, 1), "unit": "weights/s", "cores": len(os.sched_getaffinity(0)),
            "kind": "oracle", "sample": f"{m['role']} matrix {m['N']}x{m['K']} (Hessian from {calib_rows} rows "
            f"+ quantization), {t:.1f} s of oracle time", "gpu_vs_oracle": eq,
            "host": {"cpu_model": model, "nproc": os.cpu_count()}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # The grouped kernel draws enough power that the shader clock settles only
    # after about 60 back-to-back tokens; the default warmup covers that, so
    # the timed steps measure sustained decode throughput.
    ap.add_argument("--steps", type=int, default=300)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--batch", type=int, default=1)
    ap.add_argument("--workload", default="llama3_8b_stack")
    ap.add_argument("--layers", type=int, default=None, help="use only the first L layers")
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-timing", action="store_true")
    ap.add_argument("--chained-only", action="store_true", help="time only the per-GEMV launches")
    ap.add_argument("--grouped-only", action="store_true",
                    help="skip the per-GEMV launches (profiling the grouped kernel)")
    ap.add_argument("--quantizer", action="store_true",
                    help="time the offline quantizer on one Llama-3-8B-shaped layer instead of the GEMV")
    ap.add_argument("--calib-rows", type=int, default=2048, help="calibration rows per Hessian (--quantizer)")
    ap.add_argument("--quant-sequential", dest="quant_concurrent", action="store_false",
                    help="quantize the layer's matrices one after another instead of on four streams")
    ap.add_argument("--cold-copies", type=int, default=0,
                    help="time the workload warm (one copy replayed) and cold (rotating through this many "
                         "copies, each with its own weights, far beyond the 256 MB last-level cache)")
    ap.add_argument("--chained-batches", type=lambda v: [int(b) for b in v.split(",") if b], default=[4, 16],
                    help="further batch sizes timed through the chained per-GEMV launches (comma list)")
    ap.add_argument("--residual-off", action="store_true",
                    help="the ternary-only stack: same shapes and seeds, no salient columns (residual cost)")
    ap.add_argument("--copy-calibration", type=int, default=0,
                    help="after the bench, copy this many bytes device-to-device 3 times "
                         "(known-size reference for HBM counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the multi-GPU "
              "sharding of this path is described, not built", file=sys.stderr)
        sys.exit(2)

    if args.quantizer:
        quantizer_main(args)
        return
    if args.cold_copies:
        cold_main(args)
        return

    import dataclasses
    from fractions import Fraction

    import torch

    import paper_2609_00224_amd as q
    import synth
    from synth.workloads import WORKLOADS

    q.load()
    assert torch.cuda.is_available(), "no GPU"
    dev = torch.device("cuda:0")
    wl = WORKLOADS[args.workload]
    if args.residual_off:  # the ternary-only stack: same shapes and seeds, no salient columns
        wl = dataclasses.replace(wl, name=wl.name + "_ternary_only", frac=Fraction(0))
    B = args.batch
    seed = synth.DEFAULT_SEED if args.seed is None else args.seed
    # chained timing at further batch sizes from the same stack (activation rows sliced)
    extra_b = [b for b in args.chained_batches if b != B] if not args.grouped_only else []
    Bmax = max([B] + extra_b)
    mats = build_stack(wl, Bmax, dev, seed, args.layers)
    full_x = [m["x"] for m in mats]
    full_y = [m["y"] for m in mats]
    for m in mats:
        m["x"], m["y"] = m["x"][:B], m["y"][:B]
    n_layers = len({m["layer"] for m in mats})
    ws_bytes = max(q.qtea_workspace_bytes(m["pm"].desc, b) for m in mats for b in [B] + extra_b)
    ws = torch.zeros(max(ws_bytes, 4), dtype=torch.uint8, device=dev)
    stream = torch.cuda.Stream(device=dev)
    token_bytes = sum(m["bytes"] for m in mats)

    # The grouped plan and its graph are made before anything is timed, so
    # that the timed replays follow the read-ceiling passes with no idle gap:
    # from idle, this chip lowers its shader clock hard a few replays into a
    # sustained load and takes about a hundred replays to recover, while a
    # load already running keeps that dip small.
    grouped = not args.chained_only
    if grouped:
        gp = q.plan_grouped([m["pm"] for m in mats], [m["x"] for m in mats], [m["y"] for m in mats], batch=B)
        gg = capture_grouped(gp, stream)

    # 1. The measured streaming-read ceiling, the reference the path's rate is
    # compared with (a plain read of 2 GiB, held under load).
    clock_before = gpu_clock()
    ceiling, ceiling_mean = read_ceiling(dev, stream)

    # 2. Grouped: every GEMV of the token in one launch (`value`: a throughput
    # bound for independent GEMVs, whose activations are all ready at launch).
    # A step is one qtea_grouped_gemv call (its two kernels, no host work),
    # called once per token as a caller would; the host stays far ahead of
    # the device.  The same step replayed as a captured graph is reported
    # beside it: each graph launch adds about 4 us between steps here.  The
    # graph replays and their spread are measured first, so that the calls
    # of `value` (its own warmup, then the timed steps) run a few dozen steps
    # into the token's load: the shader clock dips when this load follows
    # another one and recovers over about a hundred steps.
    if grouped:
        ms_graph = time_graph(gg, stream, args.steps, args.warmup)
        spread = replay_spread(gg, stream, min(args.steps, 200))
        ms = time_calls(lambda: gp.run(stream=stream), stream, args.steps, args.warmup)
        log(f"streaming-read ceiling {ceiling:.1f} GB/s (mean of passes {ceiling_mean:.1f}), shader clock "
            f"{clock_before}")
        log(f"{wl.name} B={B} grouped: {ms * 1e3:.1f} us/token ({gp.info.n_units} units, "
            f"{gp.info.rows_per_panel}-row panels, {gp.info.grid} workgroups); as graph replays "
            f"{ms_graph * 1e3:.1f} us; single replays median {spread['median']} p10 {spread['p10']} "
            f"p90 {spread['p90']} us")
        if q.qtea_grouped_status(gp.workspace, stream=stream):
            raise RuntimeError("grouped GEMV reported a queue error")

    # 3. Chained: one qtea_gemm_lowbatch launch per GEMV in decode order (each
    # launch starts after the previous one ends, as when each product feeds
    # the next): the per-token latency of the named per-product call.
    ms_chain = float("nan")
    chained_more = {}
    if not args.grouped_only:
        g = capture(mats, B, ws, stream)
        ms_chain = time_graph(g, stream, args.steps, args.warmup)
        del g
        for b in extra_b:
            sub = [dict(m, x=fx[:b], y=fy[:b]) for m, fx, fy in zip(mats, full_x, full_y)]
            gb_ = capture(sub, b, ws, stream)
            ms_b = time_graph(gb_, stream, max(10, args.steps // 2), max(3, args.warmup // 2))
            del gb_
            chained_more[str(b)] = {"us_per_token": round(ms_b * 1e3, 2),
                                    "gbs": round(token_bytes / (ms_b * 1e-3) / 1e9, 1),
                                    "kernel": kernel_name(b, e4m3=wl.resid == "e4m3", g128=bool(wl.groups))}
            log(f"{wl.name} B={b} chained: {ms_b * 1e3:.1f} us/token, {chained_more[str(b)]['gbs']} GB/s")
    gbs_chain = token_bytes / (ms_chain * 1e-3) / 1e9
    log(f"{wl.name} B={B} chained: {ms_chain * 1e3:.1f} us/token, {gbs_chain:.1f} GB/s "
        f"({gbs_chain / HBM_PEAK_GBS:.1%} of peak)")
    if not grouped:
        log(f"streaming-read ceiling {ceiling:.1f} GB/s (mean of passes {ceiling_mean:.1f}), shader clock "
            f"{clock_before}")
        ms = ms_chain
        spread = None
    gbs = token_bytes / (ms * 1e-3) / 1e9
    log(f"{wl.name} B={B}: {ms * 1e3:.1f} us/token, {gbs:.1f} GB/s ({gbs / HBM_PEAK_GBS:.1%} of peak)")

    # Per role: the role's launches over all layers in one graph, per launch,
    # through qtea_gemm_lowbatch, and the same matrices each through a
    # one-problem grouped plan (the grouped kernel on that matrix alone).
    roles = {}
    if not args.no_kernel_timing and not args.grouped_only:
        for mat, (role, N, K) in enumerate(wl.shapes):
            sub = [m for m in mats if m["mat"] == mat]
            gr = capture(sub, B, ws, stream)
            ms_r = time_graph(gr, stream, max(10, args.steps // 4), 5)
            del gr
            per = ms_r / len(sub)
            roles[role] = {"N": N, "K": K, "us_per_launch": round(per * 1e3, 3),
                           "gbs": round(sub[0]["bytes"] / (per * 1e-3) / 1e9, 1)}
            plans = [q.plan_grouped([m["pm"]], [m["x"]], [m["y"]], batch=B) for m in sub[:8]]
            g1 = torch.cuda.CUDAGraph()
            with torch.cuda.stream(stream):
                for p_ in plans:
                    p_.run(stream=stream)
                stream.synchronize()
                with torch.cuda.graph(g1, stream=stream):
                    for p_ in plans:
                        p_.run(stream=stream)
            stream.synchronize()
            ms_g1 = time_graph(g1, stream, max(10, args.steps // 4), 5) / len(plans)
            del g1, plans
            roles[role]["grouped_one_us"] = round(ms_g1 * 1e3, 3)
            log(f"  {role:8s} {N}x{K}: {per * 1e3:.2f} us/launch, {roles[role]['gbs']} GB/s "
                f"(grouped kernel on the same matrix alone: {ms_g1 * 1e3:.2f} us)")
    # Roofline of the dominant kernel.  Grouped: one launch per step moves
    # the token's bytes.  Chained: every GEMV is a launch of the same kernel,
    # so the average launch moves token_bytes / launches.  Durations come
    # from HIP events on the stream around the timed steps above.
    n_launch = 1 if grouped else len(mats)
    kname = kernel_name(B, grouped, gp.info.rows_per_panel if grouped else 1024, wl.resid == "e4m3",
                        bool(wl.groups))
    per_launch_bytes = token_bytes / n_launch
    us_launch = ms * 1e3 / n_launch
    ach = per_launch_bytes / (us_launch * 1e-6) / 1e9
    roof = {"bound": "hbm", "achieved": round(ach, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(ach / HBM_PEAK_GBS, 4),
            "traffic": traffic_per_launch(kname, per_launch_bytes, f"{wl.name} batch {B}"),
            "kernel": kname, "launches_per_step": n_launch,
            "algorithmic_bytes_per_launch": int(per_launch_bytes), "us_per_launch": round(us_launch, 3)}
    chained = {"us_per_token": round(ms_chain * 1e3, 2), "value": round(gbs_chain, 2), "unit": "GB/s",
               "frac_hbm_peak": round(gbs_chain / HBM_PEAK_GBS, 4), "kernel": kernel_name(B, e4m3=wl.resid == "e4m3",
                                                                                        g128=bool(wl.groups)),
               "launches_per_step": len(mats), "us_per_launch": round(ms_chain * 1e3 / len(mats), 3),
               "per_role": roles, "other_batches": chained_more} if not args.grouped_only else None

    clock_after = gpu_clock()
    trit_bytes = sum(m["N"] * m["pm"].desc.n_packs for m in mats)
    device_bytes = sum(int(m["pm"].desc.bytes_total) for m in mats)
    device_gbs = device_bytes / (ms * 1e-3) / 1e9
    log(f"this path: {gbs / ceiling:.1%} of the streaming-read ceiling in algorithmic bytes, "
        f"{device_gbs / ceiling:.1%} in device bytes")
    if grouped:  # leave the grouped outputs in y for the oracle comparison
        with torch.cuda.stream(stream):
            gg.replay()
        stream.synchronize()
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(mats, wl, seed, B)
        log(f"oracle: {cpu['value']} GB/s on {cpu['cores']} threads; "
            f"GPU vs oracle max relL2 {cpu['gpu_vs_oracle_max_rel_l2']:.2e}")

    out = {
        "metric": "weight-stream GB/s (% HBM peak) & us/token, batch-1 8B-shaped ternary stack",
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "layers": n_layers, "matrices_per_token": len(mats),
                   "batch": B, "weight_bytes_per_token": token_bytes, "seed": seed,
                   "residual": "off" if args.residual_off else "on"},
        "us_per_token": round(ms * 1e3, 2),
        "us_per_token_graph_replays": round(ms_graph * 1e3, 2) if grouped else None,
        "us_per_token_single_replays": spread,
        "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
        "read_ceiling": {"gbs": round(ceiling, 1), "mean_gbs": round(ceiling_mean, 1),
                         "frac": round(gbs / ceiling, 4), "device_frac": round(device_gbs / ceiling, 4),
                         "kernel": "read_ceiling_kernel", "bytes": 2 << 30,
                         "passes": "best of 5 x 20 launches after 200 launches of load, measured first"},
        "trit_bytes_per_token": trit_bytes, "trit_gbs": round(trit_bytes / (ms * 1e-3) / 1e9, 2),
        "device_bytes_per_token": device_bytes, "device_gbs": round(device_gbs, 2),
        "shader_clock_before_timing": clock_before,
        "shader_clock_after_timing": clock_after,
        "execution": "grouped" if grouped else "chained",
        "execution_note": ("grouped: every GEMV of the token in one launch, a throughput bound for independent "
                           "GEMVs; chained: one qtea_gemm_lowbatch launch per GEMV in decode order, the "
                           "per-token latency when each product feeds the next"),
        "chained": chained,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration, dev)


if __name__ == "__main__":
    main()
