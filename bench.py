"""Benchmark of the batched serving step on one MI355X.

A step is one full serving run (every row of the hot path: admission and
continuous batching under the batch-weight budget, packed prefill, KV-cached
greedy decode, latency accounting) over the seeded 8B-shape GQA workload:
256 requests, 64 concurrent users in a closed loop (the batch is held at 64 by
continuous admission), input lengths lognormal(6.0, 0.8) clipped to [16, 4096],
output lengths lognormal(5.0, 0.7) clipped to [8, 1024].  Weights are
generated on the device (bf16 values ~N(0, 0.02)) and prompts are uploaded
before the timed region.

Prints one JSON line: whole-job output tokens/s over the timed steps, the
decode throughput and HBM fraction of full-batch decode steps, p50 TTFT/ITL,
the roofline of the dominant kernel (decode gate/up GEMM, timed per launch
with HIP events inside the timed region) and the CPU oracle's rate on a
bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2410_02425_amd import lp, synth  # noqa: E402

HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0  # dense fp16 / bf16

# HBM bytes per decode gate/up launch, measured with rocprofv3 --pmc FETCH_SIZE and
# WRITE_SIZE (one pass each, 8B workload with 72 requests, averaged over the
# 16928 gate/up dispatches of all row counts) and scaled by what the same
# counters read for a plain 1 GiB device copy: FETCH_SIZE x2.0 (it reads
# 524302 KiB for 1048576 KiB fetched), WRITE_SIZE x1.0.  The figure holds for
# the kernel source and launch plan it was measured on and is dropped when
# they change.
GATE_UP_TRAFFIC = {"bytes_per_launch": 237385249, "kernel_source": "153f83bdfcdcd181",
                   "profile": "profiles/decode_gate_up_gemm_8b.md"}


def skinny_kernel_fingerprint() -> str:
    """sha256 prefix of the source text the decode GEMM launch executes: the
    kernel's section of gemm.hip, its launch plan and launcher, the tiled
    weight layout helpers of kernels.hpp, and the device helpers."""
    csrc = os.path.join(ROOT, "paper_2410_02425_amd", "csrc")
    s = open(os.path.join(csrc, "gemm.hip")).read()
    h = open(os.path.join(csrc, "kernels.hpp")).read()

    def cut(text, start, end):
        a = text.index(start)
        return text[a:text.index(end, a)]
    parts = [cut(s, "// ------------------------------------------------------------------ skinny (decode)",
                 "// ------------------------------------------------------------------ split-K finish"),
             cut(s, "struct SkinnyPlan {", "int skinny_effective_splits("),
             cut(s, "template <typename T, int MT>\nstatic void launch_skinny_mt(", "template <typename T>\nstatic"),
             cut(h, "// Tiled layout of 16-bit weight matrices", "// Where the rows of a step read"),
             open(os.path.join(csrc, "device.hpp")).read()]
    return hashlib.sha256("".join(parts).encode()).hexdigest()[:16]


def decode_step_bytes(shape: synth.ModelShape, rows: int, sum_ctx: int, esz: int = 2) -> int:
    """Algorithmic HBM bytes of one decode step: every weight once (LM head
    included), the KV cache of every row's context once, the new K/V entries,
    and the embedding rows."""
    d, hd, F, V, L = shape.d_model, shape.head_dim, shape.ffn_dim, shape.vocab, shape.n_layers
    Hq, Hkv = shape.n_heads, shape.n_kv_heads
    weights = esz * (L * (d * (Hq + 2 * Hkv) * hd + Hq * hd * d + 3 * d * F) + V * d)
    gains = 4 * (L * 2 * d + d)
    kv_read = sum_ctx * 2 * L * Hkv * hd * esz
    kv_write = rows * 2 * L * Hkv * hd * esz
    embed = rows * d * esz
    return weights + gains + kv_read + kv_write + embed


def gate_up_bytes(shape: synth.ModelShape, launches: int, rows_sum: int, esz: int = 2) -> int:
    """Algorithmic bytes of the decode gate/up GEMM launches: the fused [2F x d]
    weight once per launch, plus each launch's activation rows in and out."""
    d, F = shape.d_model, shape.ffn_dim
    return launches * 2 * F * d * esz + rows_sum * (d + F) * esz


def prefill_flops(shape: synth.ModelShape, prompt_lens) -> int:
    """Algorithmic flops of one prefill step: the linear layers over every
    prompt token, causal attention (QK^T and PV over n(n+1)/2 pairs per head)
    and the LM head at each request's last position."""
    d, hd, F, V, L = shape.d_model, shape.head_dim, shape.ffn_dim, shape.vocab, shape.n_layers
    Hq, Hkv = shape.n_heads, shape.n_kv_heads
    lin = 2 * L * (d * (Hq + 2 * Hkv) * hd + Hq * hd * d + 3 * d * F)
    return sum(n * lin + 2 * n * (n + 1) * Hq * hd * L + 2 * d * V for n in prompt_lens)


def copy_bandwidth_gbs(torch, reps: int = 10) -> float:
    """Device-to-device copy rate of 1 GiB buffers (read + write bytes over
    time): the HBM bandwidth a plain streaming kernel reaches here."""
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1)
    b.copy_(a)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del a, b
    return 2 * n / (ms * 1e-3) / 1e9


def host_info() -> dict:
    """The host the oracle runs on: CPU model, cores it may use, and the BLAS
    library numpy calls with its thread count."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = {"vendor": "unknown", "threads": None}
    try:
        import threadpoolctl
        for lib in threadpoolctl.threadpool_info():
            if lib.get("user_api") == "blas":
                blas = {"vendor": f"{lib.get('internal_api')} {lib.get('version')}", "threads": lib.get("num_threads")}
                break
    except ImportError:
        pass
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    return {"cpu_model": model, "cores": cores, "cpu_count": os.cpu_count(), "blas": blas["vendor"],
            "blas_threads": blas["threads"]}


def step_contexts(eng, reqs, log, idx):
    """Context length of every row of decode step idx of the last run: the
    row's prompt plus the tokens it produced before that step."""
    end = log[idx]["end_ns"]
    in_len = {r.id: r.in_len for r in reqs}
    return [in_len[i] + int(np.sum(eng.token_times(i) < end)) for i in log[idx]["ids"]]


def cpu_baseline(shape: synth.ModelShape, ctxs, seed: int, budget_s: float = 20.0, prompt_lens=None):
    """The oracle, unchanged (float64, one request at a time, as it is
    written), on a bounded sample of a full-batch decode step of the
    benchmark run: ``ctxs`` are the context lengths of that step's rows.  A
    sample of the rows, spread over their contexts, runs one decode step
    (oracle.transformer.decode_step_batch) at depth 1 and 2 with full-width
    weights; the KV caches hold seeded random values of each row's context
    length (the step's cost does not depend on them).  The per-layer time is
    the difference, extrapolated linearly to the full depth, and the rows'
    time scales with their count because the oracle processes them one by
    one.  The sample size comes from a one-row probe so that the timed runs
    take about budget_s.  Returns decode tokens/s of the whole step.
    ``prompt_lens`` (a prefill step of the same run): the oracle prefills
    each of its prompts (oracle.transformer.forward on a fresh cache, one
    request at a time) at depth 1 and 2, extrapolated the same way; reported
    as prefill tokens/s beside the decode figure."""
    from oracle import transformer as T

    models = {}
    for depth in (1, 2):
        sh = shape.with_layers(depth)
        w = {}
        for name, tid, (rows, cols) in synth.tensor_shapes(sh):
            if name == "embed":
                w[name] = np.zeros((1, cols), dtype=np.float32)  # token 0's row, the one fed; set below
                emb_tid, emb_cols = tid, cols
            elif name == "lm_head":
                w[name] = models[1].w["lm_head"] if depth == 2 else synth.tensor_values(
                    seed, 2 + 9 * shape.n_layers, np.arange(rows), cols, 0.02, sh.dtype)
            else:
                v = synth.tensor_values(seed, tid, np.arange(rows), cols, 0.02, sh.dtype, gain=synth.is_gain(name))
                w[name] = v.reshape(cols) if rows == 1 else v
        cfg = dict(n_layers=depth, d_model=sh.d_model, n_heads=sh.n_heads, n_kv_heads=sh.n_kv_heads,
                   ffn_dim=sh.ffn_dim, vocab=sh.vocab, rope_theta=sh.rope_theta, norm_eps=sh.norm_eps)
        models[depth] = T.Model(cfg, w)
        models[depth].w["embed"] = synth.tensor_values(seed, emb_tid, [0], emb_cols, 0.02,
                                                       sh.dtype).astype(np.float64)
    rng = np.random.default_rng(seed)
    order = np.argsort(ctxs)

    def caches(m, sample):
        # a row of context c attends to c positions: c - 1 cached, one appended by the step
        out = []
        for c in sample:
            kv = T.KVCache(m)
            kv.k = [rng.standard_normal((c - 1, m.Hkv, m.hd)) * 0.5 for _ in range(m.L)]
            kv.v = [rng.standard_normal((c - 1, m.Hkv, m.hd)) * 0.5 for _ in range(m.L)]
            out.append(kv)
        return out

    def timed(depth, sample):
        cs = caches(models[depth], sample)
        t0 = time.perf_counter()
        T.decode_step_batch(models[depth], cs, [0] * len(sample))
        return time.perf_counter() - t0

    probe = timed(2, [int(np.median(ctxs))])
    n = int(min(len(ctxs), max(2, budget_s / (3.6 * probe))))
    sample = [int(ctxs[order[int(i)]]) for i in np.linspace(0, len(ctxs) - 1, n).round()]
    # each depth timed twice, alternating, the faster kept: the per-layer
    # time is a difference of two timings and one slow run would swing it
    t1 = t2 = float("inf")
    for _ in range(2):
        t1, t2 = min(t1, timed(1, sample)), min(t2, timed(2, sample))
    per_layer = max(t2 - t1, 1e-9)
    fixed = max(t1 - per_layer, 0.0)
    step_s = (fixed + per_layer * shape.n_layers) * len(ctxs) / n
    prefill = {}
    if prompt_lens:
        def timed_prefill(depth):
            t0 = time.perf_counter()
            for n_tok in prompt_lens:
                T.forward(models[depth], [0] * int(n_tok), T.KVCache(models[depth]))
            return time.perf_counter() - t0
        p1 = p2 = float("inf")
        for _ in range(2):
            p1, p2 = min(p1, timed_prefill(1)), min(p2, timed_prefill(2))
        p_layer = max(p2 - p1, 1e-9)
        p_s = max(p1 - p_layer, 0.0) + p_layer * shape.n_layers
        prefill = {
            "prefill_value": round(sum(prompt_lens) / p_s, 3),
            "prefill_unit": "prompt tokens/s",
            "prefill_s_extrapolated": round(p_s, 3),
            "prefill_sample": (f"one prefill step of the benchmark run ({len(prompt_lens)} prompt(s), "
                               f"{sum(prompt_lens)} tokens), the median-sized one: float64 oracle at depth 1 "
                               f"({p1:.1f} s) and 2 ({p2:.1f} s), extrapolated linearly to {shape.n_layers} layers"),
        }
    info = host_info()
    return {
        "value": round(len(ctxs) / step_s, 3),
        "unit": "decode tokens/s",
        "cores": info["blas_threads"] or info["cores"],
        "kind": "oracle",
        "precision": "fp64",
        "cpu_model": info["cpu_model"],
        "cpu_cores_available": info["cores"],
        "blas": info["blas"],
        "blas_threads": info["blas_threads"],
        "step_s_extrapolated": round(step_s, 3),
        "sample": (f"one full-batch decode step of the benchmark run ({len(ctxs)} rows, contexts "
                   f"{min(ctxs)}..{max(ctxs)}, sum {sum(ctxs)}): {n} of its rows spread over the contexts, "
                   f"float64 oracle with full-width weights at depth 1 ({t1:.1f} s) and 2 ({t2:.1f} s, each the faster of two runs), "
                   f"extrapolated linearly to {shape.n_layers} layers and to all {len(ctxs)} rows"),
        **prefill,
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="8b")
    ap.add_argument("--requests", type=int, default=0, help="override the workload's request count")
    ap.add_argument("--act", choices=["f16", "bf16"], default="f16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-timing", action="store_true")
    ap.add_argument("--step-log", default="",
                    help="write the last timed run's steps (kind, rows, context sum, duration, decode "
                         "algorithmic bytes) to this JSON file")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only copy 1 GiB device-to-device 5 times (a plain copy kernel of known size, "
                         "the reference for the HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)

    import torch
    torch.cuda.set_device(0)
    if args.copy_calibration:
        a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        a.fill_(1)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_per_launch": 1 << 30, "launches": 5}))
        return
    copy_gbs = copy_bandwidth_gbs(torch)
    shape = synth.SHAPES[args.config]
    wl = synth.WORKLOADS[args.config]
    key = synth.workload_seeds(wl.base_seed)[0]
    reqs = synth.make_requests(wl, shape.vocab, args.requests or None)
    max_seq = wl.in_range[1] + wl.out_range[1]
    flags = 0 if args.no_kernel_timing else lp.LP_FLAG_TIME_KERNEL
    if args.act == "bf16":
        flags |= lp.LP_FLAG_BF16_ACTIVATIONS
    opt = lp.EngineOptions(wl.max_batch, max_seq, 0, 65536, 0, flags)
    eng = lp.Engine(lp.make_config(shape), opt)
    eng.init_weights_random(key, 0.02)
    eng.submit(reqs)
    mode = lp.LP_CLOSED_LOOP if wl.mode == "closed" else lp.LP_OPEN_LOOP
    for _ in range(args.warmup):
        eng.run(mode, wl.max_batch)
        print(f"warmup run done: {eng.stats()['output_tokens']} tokens", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    agg = None
    for k in range(args.steps):
        eng.run(mode, wl.max_batch)
        s = eng.stats()
        agg = s if agg is None else {kk: agg[kk] + s[kk] for kk in s}
        print(f"timed run {k + 1}/{args.steps}: {s['output_tokens']} tokens in {s['wall_ns'] / 1e9:.2f} s",
              file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    # per-request latency medians (TTFT over requests, ITL pooled), last timed run
    log = eng.step_log()
    res = {r.id: eng.result(r.id) for r in reqs}
    ttft = [res[r.id]["ttft_ns"] for r in reqs]
    itl = np.concatenate([res[r.id]["itl_ns"] for r in reqs if r.out_len > 1])
    nttft = [res[r.id]["ttft_ns"] / r.in_len for r in reqs]
    # full-batch decode steps: throughput and HBM fraction
    full = [st for st in log if st["kind"] == "decode" and st["n_rows"] == wl.max_batch]
    prev_end = {i: (log[i - 1]["end_ns"] if i else 0) for i in range(len(log))}
    full_idx = [i for i, st in enumerate(log) if st["kind"] == "decode" and st["n_rows"] == wl.max_batch]
    full_ns = sum(log[i]["end_ns"] - prev_end[i] for i in full_idx)
    if args.step_log:
        with open(args.step_log, "w") as f:
            in_len_of = {r.id: r.in_len for r in reqs}
            json.dump([{"kind": st["kind"], "n_rows": st["n_rows"], "sum_ctx": st["sum_ctx"],
                        "ns": st["end_ns"] - prev_end[i],
                        "bytes": decode_step_bytes(shape, st["n_rows"], st["sum_ctx"])
                        if st["kind"] == "decode" else None,
                        "prompt_lens": [in_len_of[j] for j in st["ids"]] if st["kind"] == "prefill" else None}
                       for i, st in enumerate(log)], f)
    full_bytes = sum(decode_step_bytes(shape, log[i]["n_rows"], log[i]["sum_ctx"]) for i in full_idx)
    full_tokens = sum(log[i]["n_rows"] for i in full_idx)
    decode_gbs = full_bytes / full_ns if full_ns else 0.0
    out_tokens = agg["output_tokens"]
    in_len = {r.id: r.in_len for r in reqs}
    pre_idx = [i for i, st in enumerate(log) if st["kind"] == "prefill"]
    pre_ns = sum(log[i]["end_ns"] - prev_end[i] for i in pre_idx)
    pre_flops = sum(prefill_flops(shape, [in_len[j] for j in log[i]["ids"]]) for i in pre_idx)
    pre_tflops = pre_flops / pre_ns / 1e3 if pre_ns else 0.0

    roofline = None
    # the fp32 configuration is cache-resident and launch-bound: latency only
    if agg["timed_kernel_launches"] and shape.dtype != synth.DTYPE_F32:
        launches = agg["timed_kernel_launches"]
        avg_ms = agg["timed_kernel_ms"] / launches
        bytes_total = gate_up_bytes(shape, launches, agg["timed_kernel_rows"])
        achieved = bytes_total / launches / (avg_ms * 1e-3) / 1e9
        # the counter figure belongs to the 8B-shape gate/up launch it was measured on
        traffic = (GATE_UP_TRAFFIC["bytes_per_launch"]
                   if args.config == "8b" and skinny_kernel_fingerprint() == GATE_UP_TRAFFIC["kernel_source"]
                   else None)
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                    "traffic_unit": "bytes per launch",
                    "kernel": "gemm_skinny_kernel (decode gate/up, fused SiLU gate)",
                    "avg_launch_us": round(avg_ms * 1e3, 2), "launches": launches,
                    "bytes_per_launch": int(bytes_total / launches)}

    result = {
        "metric": "decode tokens/sec at fixed batch + p50 ITL/TTFT; % of HBM peak (1 MI355X)",
        "value": round(out_tokens / elapsed, 1),
        "unit": "output tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 1),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if shape.dtype == synth.DTYPE_F32 else ("f16" if args.act == "f16" else "bf16"),
        "data": "synthetic",
        "config": {"workload": f"{args.config}-shape decoder, closed loop, {wl.max_batch} users, "
                               f"{len(reqs)} requests, lognormal lengths",
                   "weights": ("fp32 ~N(0,0.02)" if shape.dtype == synth.DTYPE_F32 else
                               "bf16 values ~N(0,0.02), held exactly in fp16" if args.act == "f16"
                               else "bf16 ~N(0,0.02)"),
                   "global_batch": wl.max_batch, "parallelism": "none (1 GPU)"},
        "decode_tok_s_full_batch": round(full_tokens / (full_ns * 1e-9), 1) if full_ns else None,
        "decode_hbm_gbs_full_batch": round(decode_gbs, 1),
        "decode_hbm_frac_full_batch": round(decode_gbs / HBM_PEAK_GBS, 4),
        "decode_ms_per_step_full_batch": round(full_ns / max(len(full_idx), 1) / 1e6, 3),
        "ttft_p50_ms": round(float(np.median(ttft)) / 1e6, 2),
        "nttft_p50_ms": round(float(np.median(nttft)) / 1e6, 4),
        "itl_p50_ms": round(float(np.median(itl)) / 1e6, 3),
        "prefill_tflops": round(pre_tflops, 1),
        "prefill_mfma_frac": round(pre_tflops / MFMA_F16_PEAK_TFLOPS, 4),
        "copy_gbs_measured": round(copy_gbs, 1),
        "decode_frac_of_copy_full_batch": round(decode_gbs / copy_gbs, 4),
        "prefill_steps": agg["n_prefill_steps"],
        "decode_steps": agg["n_decode_steps"],
        "roofline": roofline,
        # the same measure for the whole full-batch decode step (every kernel
        # of the step), the fraction the target is stated for
        "step_roofline": None if shape.dtype == synth.DTYPE_F32 else {
                          "bound": "hbm", "achieved": round(decode_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                          "frac": round(decode_gbs / HBM_PEAK_GBS, 4),
                          "what": f"full-batch decode step ({wl.max_batch} rows)",
                          "bytes_per_step": int(full_bytes / max(len(full_idx), 1)),
                          "ms_per_step": round(full_ns / max(len(full_idx), 1) / 1e6, 3),
                          "steps": len(full_idx)},
    }
    if not args.no_cpu_baseline and full_idx:
        # the full-batch decode step whose context sum is the median one
        med = sorted(full_idx, key=lambda i: log[i]["sum_ctx"])[len(full_idx) // 2]
        # the prefill step whose prompt-token count is the median one
        pf = sorted(pre_idx, key=lambda i: sum(in_len[j] for j in log[i]["ids"]))
        pf_lens = [in_len[j] for j in log[pf[len(pf) // 2]]["ids"]] if pf else None
        result["cpu_baseline"] = cpu_baseline(shape, step_contexts(eng, reqs, log, med), key, prompt_lens=pf_lens)
    eng.close()
    print(json.dumps(result))


if __name__ == "__main__":
    main()
