#!/usr/bin/env python3
"""Benchmark of the PARD decode step on one MI355X.

A step is one pass of the whole hot path: one draft forward over the pending
tokens plus K-1 mask tokens, one target verify forward over K+1 rows, argmax,
greedy acceptance and KV rollback, all on the device (fused loop,
``pard_generate``).  The workload is the LLaMA3.1-8B-shaped target with the
LLaMA3.2-1B-shaped draft, bf16, batch 1, K = 8, 512-token prompt, seeded
random weights (synthetic data).  Prints one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

``--workload llama8b_1b_batch32`` measures the batched workload instead (32
sequences with ragged prompts stepped together; MFMA-bound GEMMs);
``--workload cod`` the COD training-data processing of a synthetic dataset.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import pard_inputs as pi  # noqa: E402
from paper_2504_18583_amd import bytes_model as bm  # noqa: E402

METRIC = "tokens/sec batch-1 PARD decode, 1B draft/8B target K=8; step HBM GB/s vs peak"
PEAK_HBM_GBPS = 8000.0
SAMPLING_T, SAMPLING_SEED = 1.0, 2504   # speculative-sampling measurement beside the greedy headline
# measured HBM traffic of the dominant kernel (rocprofv3 FETCH_SIZE / WRITE_SIZE,
# scaled by a copy of known size); valid only while the kernel source is unchanged:
# the 8B gate/up GEMM launched on its own, and the 8B decode layer's one launch
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_gemm_swiglu_8b_gateup_traffic.txt")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2504_18583_amd", "csrc", f) for f in ("gemm.hip", "pard_internal.h")]
LAYER_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_qkv_attn_8b_layer_traffic.txt")
LAYER_SOURCES = [os.path.join(ROOT, "paper_2504_18583_amd", "csrc", f)
                 for f in ("gemm.hip", "attn_tile.h", "pard_internal.h")]
# measured HBM traffic of whole decode steps of the 8B/1B K = 8 workload (every
# kernel of the step), valid while the decode path's sources are unchanged
STEP_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "step_8b_1b_k8_counters.txt")
STEP_SOURCES = [os.path.join(ROOT, "paper_2504_18583_amd", "csrc", f)
                for f in ("attention.hip", "attn_tile.h", "device_init.h", "device_init.hip", "engine.hip",
                          "gemm.hip", "pard_internal.h")]


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def kernel_source_sha256(sources=KERNEL_SOURCES) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in sources:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(path=TRAFFIC_FILE, sources=KERNEL_SOURCES, key="traffic_bytes_per_launch"):
    """HBM bytes per launch of the dominant kernel (or, with key, another
    figure) from the committed counter summary, or None when it is missing or
    the kernel source changed since."""
    try:
        kv = {}
        with open(path) as fh:
            for line in fh:
                if ":" in line and not line.startswith("#"):
                    k, v = line.split(":", 1)
                    kv[k.strip()] = v.strip()
        if kv.get("kernel_source_sha256") != kernel_source_sha256(sources):
            return None
        return int(float(kv[key]))
    except (OSError, KeyError, ValueError):
        return None


def copy_calibration() -> int:
    """A device-to-device copy of known size, for scaling rocprofv3 byte counters."""
    import torch
    n = 1 << 30
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "copies": 3}), flush=True)
    return 0


DTYPE = "bf16 weights (fp16 encoding), fp16 activations/KV, fp16 MFMA, fp32 accumulate"


def host_description() -> str:
    """CPU model and numpy's BLAS, for the CPU-baseline record."""
    model = "unknown CPU"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = "unknown BLAS"
    try:
        b = np.show_config(mode="dicts")["Build Dependencies"]["blas"]
        blas = f"{b.get('name', '?')} {b.get('version', '')}".strip()
    except Exception:
        pass
    return f"{model}; numpy {np.__version__} with {blas}"


def cpu_baseline_full(wl, tokens_per_step: float, context: int, steps: int = 2) -> dict:
    """The oracle, as it is, timed on the host for whole steps at full depth.

    The oracle's float32 weights of both models are generated first (not
    timed), the KV caches hold `context` positions of random keys and values
    (the step's arithmetic does not depend on their values), and `steps`
    steps -- one draft pass over 1 pending token and K-1 masks, one verify pass
    over K+1 rows -- are timed; the median step is reported."""
    import oracle
    threads = len(os.sched_getaffinity(0))
    k = wl.k
    rng = np.random.default_rng(0)
    t0 = time.perf_counter()
    target, draft = oracle.build_model(wl.target), oracle.build_model(wl.draft)
    gen_s = time.perf_counter() - t0
    log(f"cpu_baseline: oracle weights generated in {gen_s:.1f} s")
    caches = []
    for model in (target, draft):
        s_ = model.spec
        cache = oracle.KVCache(model)
        for l in range(s_.n_layers):
            cache.k[l] = rng.standard_normal((context, s_.n_kv_heads, s_.head_dim))
            cache.v[l] = rng.standard_normal((context, s_.n_kv_heads, s_.head_dim))
        caches.append(cache)
    times = []
    for i in range(steps):
        t0 = time.perf_counter()
        oracle.draft_step(draft, caches[1], [1], k, wl.mask_id)
        oracle.verify_step(target, caches[0], 1, list(range(2, 2 + k)))
        times.append(time.perf_counter() - t0)
        log(f"cpu_baseline: full-depth step {i + 1}: {times[-1]:.2f} s")
        caches[0].truncate(context)
        caches[1].truncate(context)
    step = statistics.median(times)
    return {"value": round(tokens_per_step / step, 4), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": (f"{steps} whole steps at full depth ({wl.target.n_layers}/{wl.draft.n_layers} layers): one "
                       f"draft pass over 1 pending + {k - 1} mask rows and one verify pass over {k + 1} rows, "
                       f"context {context}, float64 numpy on {threads} threads; median step {step:.2f} s "
                       f"(steps {', '.join(f'{t:.2f}' for t in times)} s; weights generated beforehand in "
                       f"{gen_s:.0f} s, not timed); {tokens_per_step:.3f} tokens/step as measured on the GPU; "
                       f"host: {host_description()}")}


def copy_ceiling(nbytes: int = 2 << 30, reps: int = 10):
    """Plain device bandwidths this box reaches, in GB/s: a device-to-device
    copy (bytes read + written) and a read-dominated reduction (torch.sum over
    fp16 values, bytes read); practical references beside the 8 TB/s peak."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    dst.copy_(src)
    halves = src.view(torch.float16)
    torch.sum(halves, dtype=torch.float32)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(reps):
        dst.copy_(src)
    ev1.record()
    torch.cuda.synchronize()
    copy_ms = ev0.elapsed_time(ev1) / reps
    ev0.record()
    for _ in range(reps):
        torch.sum(halves, dtype=torch.float32)
    ev1.record()
    torch.cuda.synchronize()
    read_ms = ev0.elapsed_time(ev1) / reps
    del src, dst, halves
    torch.cuda.empty_cache()
    return 2 * nbytes / (copy_ms * 1e-3) / 1e9, nbytes / (read_ms * 1e-3) / 1e9


def cpu_baseline(wl, tokens_per_step: float, context: int) -> dict:
    """The oracle, as it is, timed on the host for one step at this workload's shapes.

    Bounded sample: the target and draft run with 1 and with 2 of their layers
    (embedding and lm_head in full) against a synthetic KV cache of `context`
    positions; the per-layer cost is extrapolated linearly to all layers."""
    import oracle
    from dataclasses import replace
    threads = len(os.sched_getaffinity(0))
    k = wl.k
    rng = np.random.default_rng(0)
    t_full = 0.0
    for spec, is_target in ((wl.target, True), (wl.draft, False)):
        full = oracle.build_model(replace(spec, n_layers=2))
        times = {}
        for n_layers in (1, 2):
            layers = {l: full.weights["layers"][l] for l in range(n_layers)}
            model = oracle.Model(replace(spec, n_layers=n_layers), dict(full.weights, layers=layers))
            samples = []
            for _ in range(2):
                cache = oracle.KVCache(model)
                for l in range(n_layers):
                    cache.k[l] = rng.standard_normal((context, spec.n_kv_heads, spec.head_dim))
                    cache.v[l] = rng.standard_normal((context, spec.n_kv_heads, spec.head_dim))
                t0 = time.perf_counter()
                if is_target:
                    oracle.verify_step(model, cache, 1, list(range(2, 2 + k)))
                else:
                    oracle.draft_step(model, cache, [1], k, wl.mask_id)
                samples.append(time.perf_counter() - t0)
            times[n_layers] = min(samples)
        per_layer = max(times[2] - times[1], 0.0)
        fixed = max(times[1] - per_layer, 0.0)
        t_full += fixed + per_layer * spec.n_layers
        log(f"cpu_baseline: {'target' if is_target else 'draft'} 1 layer {times[1]:.2f}s, "
            f"2 layers {times[2]:.2f}s")
    return {"value": round(tokens_per_step / t_full, 4), "unit": "tokens/s", "cores": threads,
            "kind": "oracle",
            "sample": (f"one step (draft pass over 1 pending + {k - 1} mask rows, verify pass over "
                       f"{k + 1} rows) at these shapes, context {context}, float64 numpy; target and "
                       f"draft timed with 1 and 2 layers (full embedding/lm_head), per-layer time "
                       f"extrapolated to {wl.target.n_layers}/{wl.draft.n_layers} layers; "
                       f"{tokens_per_step:.3f} tokens/step as measured on the GPU; "
                       f"step {t_full:.2f} s")}


PEAK_F16_TFLOPS = 2500.0   # MI355X dense fp16 / bf16 MFMA


def measure_baselines(eng, B, prompt, k, pard_step_s, pard_tok_s, steps=64, warmup=4):
    """The decoding schemes PARD is compared with, on the same kernels and the
    same prompt: plain greedy target steps (K = 0, one target pass per token)
    and vanilla speculative decoding (K sequential one-row draft passes, then
    the verify pass; eq. 3).  Each is timed over `steps` fused steps after a
    fresh prefill; per step, T_AR = T_T, T_vanilla = K*T_D + T_T and
    T_PARD = T_D' + T_T (T_D' one draft pass over K + a rows)."""
    import torch
    out = {"steps": steps}
    for name, kk, mode in (("ar", 0, B.PARD_MODE_PARALLEL), ("vanilla_sd", k, B.PARD_MODE_VANILLA)):
        eng.prefill(prompt)
        eng.generate(kk, eng.max_ctx - len(prompt) - 2 * k - 2, max_steps=warmup, mode=mode)
        budget = eng.max_ctx - eng.kv_len(B.PARD_TARGET) - 2 * k - 2
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        _, st = eng.generate(kk, budget, max_steps=steps, mode=mode)
        torch.cuda.synchronize()
        w = time.perf_counter() - t0
        hist = list(st.accept_hist)
        em = sum((a + 1) * c for a, c in enumerate(hist))
        out[name] = {"ms_per_step": round(w / st.steps * 1e3, 4), "tokens_per_step": round(em / st.steps, 4),
                     "tokens_per_s": round(em / w, 3)}
    t_ar = out["ar"]["ms_per_step"]
    out["pard"] = {"ms_per_step": round(pard_step_s * 1e3, 4), "tokens_per_s": round(pard_tok_s, 3)}
    out["draft_ms_per_step"] = {"pard": round(pard_step_s * 1e3 - t_ar, 4),
                                "vanilla_sd": round(out["vanilla_sd"]["ms_per_step"] - t_ar, 4)}
    out["note"] = ("acceptance with random weights is ~0, so every scheme emits ~1 token per step; "
                   "draft_ms_per_step = step time minus the plain target step")
    # speculative sampling (temperature 1): PARD and plain target sampling
    samp = {"temperature": SAMPLING_T, "seed": SAMPLING_SEED}
    eng.set_sampling(SAMPLING_T, SAMPLING_SEED)
    try:
        for name, kk in (("pard", k), ("ar", 0)):
            eng.prefill(prompt)
            eng.generate(kk, eng.max_ctx - len(prompt) - 2 * k - 2, max_steps=warmup)
            budget = eng.max_ctx - eng.kv_len(B.PARD_TARGET) - 2 * k - 2
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            _, st = eng.generate(kk, budget, max_steps=steps)
            torch.cuda.synchronize()
            w = time.perf_counter() - t0
            hist = list(st.accept_hist)
            em = sum((a + 1) * c for a, c in enumerate(hist))
            samp[name] = {"ms_per_step": round(w / st.steps * 1e3, 4), "tokens_per_step": round(em / st.steps, 4),
                          "tokens_per_s": round(em / w, 3), "accept_hist": hist[:kk + 1]}
    finally:
        eng.set_sampling(0.0)
    samp["note"] = ("random weights: both models' distributions at T=1 are broad, so candidates are kept "
                    "often; the figure shows the sampled step's cost, not a trained pair's speedup")
    out["sampling"] = samp
    return out


def bench_batched(args, wl) -> int:
    """The batched workload: wl.batch independent sequences with ragged prompt
    lengths, stepped together (one batched draft pass and one batched verify
    pass per step, every sequence with its own acceptance and KV rollback).
    Prints one JSON line; its metric is aggregate tokens/s, its roofline the
    MFMA rate of the target's gate/up GEMM over the verify pass's rows."""
    import torch
    from paper_2504_18583_amd import binding as B

    k = args.k if args.k is not None else wl.k
    n = wl.batch
    t_spec, d_spec = pi.with_dtype(wl.target, "bf16"), pi.with_dtype(wl.draft, "bf16")
    prompts = [[int(x) for x in p] for p in pi.workload_prompts(wl)]
    max_len = max(len(p) for p in prompts)
    max_ctx = max_len + (args.warmup + 2 * args.steps + 4) * (k + 1) + 2 * k + 8
    slots = list(range(n))

    t0 = time.perf_counter()
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=max_ctx, max_k=max(k, 1), max_batch=n)
    torch.cuda.synchronize()
    log(f"load + weight generation: {time.perf_counter() - t0:.2f}s")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s, p in zip(slots, prompts):
        eng.prefill(p, seq=s)
    torch.cuda.synchronize()
    prefill_ms = (time.perf_counter() - t0) * 1e3
    n_prompt = sum(len(p) for p in prompts)
    log(f"prefill ({n} prompts, {n_prompt} tokens, both models): {prefill_ms:.1f} ms")

    def budget():
        return max_ctx - max(eng.kv_len(B.PARD_TARGET, seq=s) for s in slots) - 2 * k - 2

    if args.warmup:
        eng.generate_batch(slots, k, budget(), max_steps=args.warmup)
    l_t0 = [eng.kv_len(B.PARD_TARGET, seq=s) for s in slots]
    l_d0 = [eng.kv_len(B.PARD_DRAFT, seq=s) for s in slots]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    _, stats = eng.generate_batch(slots, k, budget(), max_steps=args.steps)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    steps = int(stats.steps)
    hist = list(stats.accept_hist)
    emitted = sum((a + 1) * c for a, c in enumerate(hist))
    assert steps == args.steps, (steps, args.steps)
    tokens_per_seq_step = emitted / (steps * n)
    step_s = wall / steps
    l_t1 = [eng.kv_len(B.PARD_TARGET, seq=s) for s in slots]

    # algorithmic bytes and GEMM flops of the timed steps (contexts grow by a+1 per step)
    tot_bytes = 0.0
    acc = round(tokens_per_seq_step - 1.0)
    for i in range(steps):
        grow = i * tokens_per_seq_step
        tot_bytes += bm.batch_step_bytes(t_spec, d_spec, k, [int(l + grow) for l in l_t0],
                                         [int(l + grow) for l in l_d0], [acc + 1] * n)
    step_gbps = tot_bytes / wall / 1e9
    step_flops = bm.gemm_flops(t_spec, n * (k + 1)) + bm.gemm_flops(d_spec, n * (acc + k))
    step_tflops = step_flops / step_s / 1e12

    # dominant kernel: the target's gate/up GEMM over the verify pass's n*(K+1)
    # rows, timed with HIP events attached to each launch over a second run
    kclass = B.PARD_TARGET * 8 + B.OP_GATEUP
    eng.timer_enable(kclass, min(steps * t_spec.n_layers, 1 << 16))
    eng.generate_batch(slots, k, budget(), max_steps=steps)
    launches, total_ms = eng.timer_read()
    eng.timer_enable(-1, 1)
    avg_s = total_ms / 1e3 / max(launches, 1)
    f_pad = (t_spec.ffn_dim + 31) // 32 * 32
    rows = n * (k + 1)
    gu_flops = 2 * rows * (2 * f_pad) * t_spec.d_model
    achieved = gu_flops / avg_s / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_F16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_F16_TFLOPS, 4), "traffic": None,
                "kernel": f"k_gemm_rows<EPI_SWIGLU> (target gate/up, 8B shape, {rows} rows)",
                "launches": launches, "avg_us": round(avg_s * 1e6, 2), "flops_per_launch": gu_flops}
    result = {
        "metric": f"tokens/sec batch-{n} PARD decode (ragged prompts), 1B draft/8B target K={k}; MFMA TFLOP/s vs peak",
        "value": round(emitted / wall, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_s * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DTYPE,
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: {wl.target.n_layers}-layer d{wl.target.d_model} target / "
                               f"{wl.draft.n_layers}-layer d{wl.draft.d_model} draft, batch {n}, prompts "
                               f"{min(len(p) for p in prompts)}-{max_len}, K={k}, seed {wl.seed}",
                   "batch": n, "prompt_lens": [len(p) for p in prompts], "k": k, "seed": wl.seed},
        "tokens_per_step": round(emitted / steps, 4),
        "accept_hist": hist[:k + 1],
        "step_hbm_gbps": round(step_gbps, 1),
        "step_hbm_frac": round(step_gbps / PEAK_HBM_GBPS, 4),
        "step_gemm_tflops": round(step_tflops, 1),
        "step_mfma_frac": round(step_tflops / PEAK_F16_TFLOPS, 4),
        "bytes_per_step": round(tot_bytes / steps),
        "context": [min(l_t0), max(l_t1)],
        "prefill_ms": round(prefill_ms, 1),
        "device_ms_per_step": round(stats.elapsed_ms / steps, 4),
        "roofline": roofline,
    }
    eng.close()
    del eng
    if not args.no_cpu_baseline:
        cb = cpu_baseline(wl, tokens_per_seq_step, int(statistics.mean(l_t0)))
        cb["sample"] += f"; the oracle runs the {n} sequences one after another, so its aggregate rate equals this per-sequence rate"
        result["cpu_baseline"] = cb
    print(json.dumps(result), flush=True)
    return 0


COD_SAMPLES, COD_LEN, COD_K, COD_R, COD_RMIN, COD_SEED = 4096, (256, 1024), 8, 0.7, 0.2, 6


def bench_cod(args) -> int:
    """COD training-data processing (Sec. 3.2, Alg. 1) of a synthetic dataset:
    COD_SAMPLES token sequences with lengths uniform in COD_LEN (the paper's
    training sequence lengths reach 1024), K = 8, r = 0.7, r_min = 0.2 (the
    setting App. A counts).  A step is one pass over the whole dataset (one
    pard_cod_build call); the line's value is samples per second."""
    import torch
    from paper_2504_18583_amd import binding as B

    lo, hi = COD_LEN
    lens = pi.gen_prompt_lengths(COD_SEED, COD_SAMPLES, lo, hi)
    vocab = pi.WORKLOADS["llama8b_1b"].target.vocab
    samples = [pi.gen_prompt(COD_SEED, vocab, int(n), b) for b, n in enumerate(lens)]
    offs = np.zeros(COD_SAMPLES + 1, np.int64)
    offs[1:] = np.cumsum(lens)
    flat = torch.from_numpy(np.concatenate(samples).astype(np.int32)).cuda()
    mask_id = vocab - 1
    run = lambda: B.cod_build(flat, offs, COD_K, COD_R, COD_RMIN, mask_id, COD_SEED, timing=True)
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    kernel_ms = []
    for _ in range(args.steps):
        _, _, out_len, ms = run()
        kernel_ms.append(ms)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    packed = int(out_len.sum().item())
    dev_ms = sum(kernel_ms) / len(kernel_ms)
    n_tok = int(offs[-1])
    algo_bytes = 4 * n_tok + 5 * 4 * packed + 4 * COD_SAMPLES
    achieved = algo_bytes / (dev_ms * 1e-3) / 1e9
    line = {
        "metric": "COD training-data processing samples/s (K=8, r=0.7, r_min=0.2)",
        "value": round(COD_SAMPLES * args.steps / wall, 1),
        "unit": "samples/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int32", "data": "synthetic",
        "config": {"workload": f"cod: {COD_SAMPLES} samples, lengths U[{lo},{hi}], K={COD_K}, r={COD_R}, "
                               f"r_min={COD_RMIN}, seed {COD_SEED}",
                   "samples": COD_SAMPLES, "tokens": n_tok, "packed_tokens": packed,
                   "packed_per_column": round(packed / (n_tok - COD_SAMPLES), 4)},
        "device_ms_per_step": round(dev_ms, 4),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBPS, 4), "traffic": None,
                     "kernel": "k_cod (one 256-thread workgroup per sample)",
                     "bytes_per_launch": algo_bytes,
                     "note": "HIP events around each k_cod launch on its stream (pard_cod_build's kernel_ms); "
                             "bound by per-subtask LDS sorts and barriers, not by HBM"},
    }
    if not args.no_cpu_baseline:
        from oracle import cod
        t0 = time.perf_counter()
        n_s = 0
        while time.perf_counter() - t0 < 15.0 and n_s < COD_SAMPLES:
            cod.cod_process(samples[n_s], COD_K, COD_R, COD_RMIN, mask_id, COD_SEED, n_s)
            n_s += 1
        w = time.perf_counter() - t0
        line["cpu_baseline"] = {"value": round(n_s / w, 2), "unit": "samples/s", "cores": 1, "kind": "oracle",
                                "sample": f"the first {n_s} samples of the same dataset, pure-Python oracle "
                                          f"(one thread), {w:.1f} s"}
    print(json.dumps(line), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", default="llama8b_1b")
    ap.add_argument("--k", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-baselines", action="store_true",
                    help="skip the plain-target and vanilla-SD comparison runs (profiling runs)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy (byte-counter calibration under rocprofv3)")
    args = ap.parse_args()
    if args.copy_calibration:
        return copy_calibration()
    if args.gpus != 1:
        log("bench.py measures one GPU: the decode step of one batch-1 sequence does not shard "
            "(see the design notes); run with --gpus 1")
        return 2

    import torch
    from paper_2504_18583_amd import binding as B

    if args.workload == "cod":
        return bench_cod(args)
    wl = pi.WORKLOADS[args.workload]
    if wl.batch != 1:
        return bench_batched(args, wl)
    k = args.k if args.k is not None else wl.k
    t_spec, d_spec = pi.with_dtype(wl.target, "bf16"), pi.with_dtype(wl.draft, "bf16")
    prompt = [int(x) for x in pi.workload_prompts(wl)[0]]
    max_ctx = len(prompt) + (args.warmup + args.steps + 2) * (k + 1) + 2 * k + 8

    t0 = time.perf_counter()
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=max_ctx, max_k=max(k, 1))
    torch.cuda.synchronize()
    log(f"load + weight generation: {time.perf_counter() - t0:.2f}s")

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    eng.prefill(prompt)
    torch.cuda.synchronize()
    ttft_ms = (time.perf_counter() - t0) * 1e3
    log(f"prefill ({len(prompt)} tokens, both models): {ttft_ms:.1f} ms")

    big = max_ctx  # n_tokens bound; max_steps decides
    # capture every step graph the timed steps will replay (one per attention
    # length class the context passes through), then start again from the prompt
    eng.generate(k, big - eng.kv_len(B.PARD_TARGET) - 2 * k - 2, max_steps=args.warmup + args.steps)
    eng.prefill(prompt)
    if args.warmup:
        eng.generate(k, big - eng.kv_len(B.PARD_TARGET) - 2 * k - 2, max_steps=args.warmup)
    l_t0 = eng.kv_len(B.PARD_TARGET)

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    _, stats = eng.generate(k, big - l_t0 - 2 * k - 2, max_steps=args.steps)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    steps = int(stats.steps)
    hist = list(stats.accept_hist)
    emitted = sum((a + 1) * n for a, n in enumerate(hist))
    assert steps == args.steps, (steps, args.steps)
    tokens_per_step = emitted / steps
    step_s = wall / steps
    l_t1 = eng.kv_len(B.PARD_TARGET)

    # algorithmic bytes of the timed steps (context grows by a+1 per step)
    mean_acc = tokens_per_step - 1.0
    tot_bytes = 0.0
    for i in range(steps):
        lt = l_t0 + i * tokens_per_step
        tot_bytes += bm.step_bytes(t_spec, d_spec, k, round(mean_acc), int(lt), int(lt) + 1)
    step_gbps = tot_bytes / wall / 1e9

    phases = {"draft_ms_per_step": round(stats.draft_ms / steps, 4),
              "verify_ms_per_step": round(stats.verify_ms / steps, 4),
              "accept_ms_per_step": round(stats.accept_ms / steps, 4),
              "note": ("device clock at pass boundaries inside the timed steps: draft pass incl. its tail; "
                       "target pass through its lm_head; verify tail (argmax, acceptance, rollback, staging)")}
    latency = {"p50_ms": round(stats.step_ms_p50, 4), "p90_ms": round(stats.step_ms_p90, 4),
               "mean_ms": round(step_s * 1e3, 4)}

    # dominant kernel, timed with HIP events around each launch on the engine's
    # stream over a second run of the same steps: the target's gate/up GEMM,
    # or, where the engine runs gate/up inside the decode layer's launch (QKV,
    # attention, O-projection and gate/up), that launch
    def time_class(op, n_steps=steps):
        eng.timer_enable(B.PARD_TARGET * 8 + op, min(n_steps * t_spec.n_layers, 1 << 16))
        eng.generate(k, big - eng.kv_len(B.PARD_TARGET) - 2 * k - 2,
                     max_steps=max(1, min(n_steps, (max_ctx - eng.kv_len(B.PARD_TARGET) - 2 * k - 2) // (k + 1))))
        n, ms = eng.timer_read()
        eng.timer_enable(-1, 1)
        return n, ms

    f_pad = (t_spec.ffn_dim + 31) // 32 * 32
    launches, total_ms = time_class(B.OP_GATEUP)
    if launches > 0:
        # bf16 weights [2*F, d] once, fp16 activations in, fp16 h = silu(gate)*up out
        kbytes = 2 * (2 * f_pad * t_spec.d_model) + (k + 1) * t_spec.d_model * 2 + (k + 1) * f_pad * 2
        kname = f"k_gemm<MT=1,EPI_SWIGLU> (target gate/up, [{2 * f_pad}, {t_spec.d_model}] weight, {k + 1} rows)"
        # the counter summary covers the 8B-shaped gate/up launch with 9 rows only
        traffic = measured_traffic() if (t_spec.d_model, t_spec.ffn_dim, k) == (4096, 14336, 8) else None
    else:
        with_down = time_class(B.OP_DOWN, 1)[0] == 0   # the down projection runs inside the launch too
        l_mean = eng.kv_len(B.PARD_TARGET) + steps * tokens_per_step / 2
        launches, total_ms = time_class(B.OP_QKV)
        # the timer run's mean committed target length (it continues after the timed steps)
        kbytes = bm.layer_launch_bytes(t_spec, k + 1, int(round(l_mean)), with_down)
        kname = (f"k_qkv_attn (target decode layer: QKV GEMM, attention, O-projection, gate/up"
                 f"{' and down' if with_down else ''} GEMMs, {k + 1} rows)")
        # the counter summary covers the 8B-shaped launch with the down projection, 9 rows
        traffic = (measured_traffic(LAYER_TRAFFIC_FILE, LAYER_SOURCES)
                   if (t_spec.d_model, t_spec.ffn_dim, k) == (4096, 14336, 8) and with_down else None)
    avg_s = total_ms / 1e3 / max(launches, 1)
    achieved = kbytes / avg_s / 1e9 if launches > 0 else 0.0
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBPS, 4), "traffic": traffic,
                "kernel": kname, "launches": launches, "avg_us": round(avg_s * 1e6, 2),
                "bytes_per_launch": kbytes}

    baselines = None if args.no_baselines else measure_baselines(eng, B, prompt, k, wall / steps, emitted / wall)
    eng.close()
    del eng
    copy_gbps, read_gbps = copy_ceiling()
    log(f"device copy: {copy_gbps:.0f} GB/s (read + write); torch.sum read: {read_gbps:.0f} GB/s")
    # HBM bytes per step counted by rocprofv3 over whole steps of this workload
    # (FETCH_SIZE / WRITE_SIZE of every kernel, scaled by a copy of known size)
    step_traffic = None
    if wl.name == "llama8b_1b" and k == 8:
        counted = measured_traffic(STEP_TRAFFIC_FILE, STEP_SOURCES, "traffic_bytes_per_step")
        algo = measured_traffic(STEP_TRAFFIC_FILE, STEP_SOURCES, "algorithmic_bytes_per_step")
        if counted and algo:
            step_traffic = {"bytes_per_step": counted, "over_algorithmic": round(counted / algo, 4),
                            "gbps": round(counted / step_s / 1e9, 1),
                            "frac": round(counted / step_s / 1e9 / PEAK_HBM_GBPS, 4),
                            "source": os.path.relpath(STEP_TRAFFIC_FILE, ROOT)}

    result = {
        "metric": METRIC,
        "value": round(emitted / wall, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_s * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DTYPE,
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: {wl.target.n_layers}-layer d{wl.target.d_model} target / "
                               f"{wl.draft.n_layers}-layer d{wl.draft.d_model} draft, batch 1, "
                               f"prompt {len(prompt)}, K={k}, seed {wl.seed}",
                   "batch": 1, "prompt_len": len(prompt), "k": k, "seed": wl.seed},
        "tokens_per_step": round(tokens_per_step, 4),
        "accept_hist": hist[:k + 1],
        "step_hbm_gbps": round(step_gbps, 1),
        "step_hbm_frac": round(step_gbps / PEAK_HBM_GBPS, 4),
        "copy_gbps": round(copy_gbps, 1),
        "read_gbps": round(read_gbps, 1),
        "step_frac_of_copy": round(step_gbps / copy_gbps, 4),
        "bytes_per_step": round(tot_bytes / steps),
        "step_traffic": step_traffic,
        "context": [l_t0, l_t1],
        "ttft_ms": round(ttft_ms, 2),
        "device_ms_per_step": round(stats.elapsed_ms / steps, 4),
        "step_latency": latency,
        "phases": phases,
        "roofline": roofline,
        "baselines": baselines,
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline_full(wl, tokens_per_step, len(prompt))
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
