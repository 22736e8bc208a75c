"""Throughput of one DC-Leap denoising iteration on one MI355X.

A step = dcl_denoise_step (bidirectional transformer forward, fused LM head + vocabulary softmax /
top-2 reduction over the masked rows) + dcl_select_contiguous (DCV, commit, drafts, remask), on
one HIP stream, preceded by a device-to-device restore of the frozen decode state (tokens + p,
1.5 KB) so every timed step sees the same input. Weights and inputs are seeded synthetic data
resident in HBM before timing starts.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
import argparse
import dataclasses
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "denoising steps/sec and scored tokens/sec at LLaDA-8B shape; MFMA util %"
BF16_PEAK_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
HBM_PEAK_GBS = 8000.0


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def step_work(w, R):
    """Algorithmic FLOPs per launch of each kernel class for workload w with R scored rows."""
    g = w.geom
    T = w.batch * w.seq
    Sk = w.kv_prefix + w.seq
    d, H, Hkv, dh, F, V = g.d_model, g.n_heads, g.n_kv_heads, g.head_dim, g.d_ffn, g.vocab
    return {
        "gemm_qkv_rope": 2.0 * T * (H + 2 * Hkv) * dh * d,
        "attention": 4.0 * w.batch * H * w.seq * Sk * dh,
        "gemm_o_residual": 2.0 * T * d * H * dh,
        "gemm_gate_up_swiglu": 2.0 * T * 2 * F * d,
        "gemm_down_residual": 2.0 * T * d * F,
        "gemm_lm_head_top2": 2.0 * R * V * d,
    }


def step_bytes(w, R):
    """Algorithmic HBM bytes per launch of each kernel class: every operand read once, every result
    written once (bf16 weights and activations, fp32 residual stream and split-K slices)."""
    g = w.geom
    T = w.batch * w.seq
    P = w.kv_prefix
    d, H, Hkv, dh, F, V = g.d_model, g.n_heads, g.n_kv_heads, g.head_dim, g.d_ffn, g.vocab
    nq = (H + 2 * Hkv) * dh
    return {
        "gemm_qkv_rope": 2 * (nq * d + T * d + T * nq),
        "attention": 2 * (T * H * dh + 2 * w.batch * Hkv * (w.seq + P) * dh + T * H * dh),
        "gemm_o_residual": 2 * (d * H * dh + T * H * dh) + 4 * T * d,
        "gemm_gate_up_swiglu": 2 * (2 * F * d + T * d + T * F),
        "gemm_down_residual": 2 * (d * F + T * F) + 4 * T * d,
        "gemm_lm_head_top2": 2 * (V * d + R * d),
    }


# Kernel sources whose change invalidates stored hardware-counter traffic figures.
# the sources that define the dominant kernel (the GEMM family, its plans and device helpers)
TRAFFIC_SOURCES = ["paper_2607_20467_amd/csrc/k_gemm.hip", "paper_2607_20467_amd/csrc/gemm_tuned.inc",
                   "paper_2607_20467_amd/csrc/dcl_internal.h"]


def kernel_source_digest():
    import hashlib
    h = hashlib.sha256()
    for rel in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def stored_traffic(kernel_class, workload_key):
    """HBM bytes per launch from a committed rocprofv3 FETCH_SIZE / WRITE_SIZE summary, or None when
    there is none or the kernel sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{kernel_class}_{workload_key}_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    start = text.find("```json")
    if start < 0:
        return None
    rec = json.loads(text[start + 7:text.index("```", start + 7)])
    if rec.get("source_digest") != kernel_source_digest():
        log(f"traffic figures in {os.path.basename(path)} predate the current kernel sources: not used")
        return None
    return rec


# rocprofv3 kernel names -> bench kernel classes (split-K slice GEMMs alternate o-proj, down-proj per layer)
def kernel_class(name):
    for key, cls in (("EpiSwiglu", "gemm_gate_up_swiglu"), ("EpiQkv", "gemm_qkv_rope"), ("EpiLm", "gemm_lm_head_top2"),
                     ("attn_kernel", "attention"), ("rmsnorm_kernel", "rmsnorm"), ("embed_kernel", "embed"),
                     ("compact_kernel", "compact"), ("merge_kernel", "merge"), ("select_kernel", "select"),
                     ("copyBuffer", "copy"), ("pack_", "weight_packing")):
        if key in name:
            return cls
    if "EpiPartial" in name or "EpiResid" in name:
        return "gemm_o_or_down_residual"
    return "other"


def pmc_summary(csv_path, copy_mib):
    """Per-kernel-class average of each counter in a rocprofv3 --pmc counter_collection.csv, with the
    calibration factor from the largest plain copy (copy_mib MiB read and written once)."""
    import collections
    import csv
    rows = list(csv.DictReader(open(csv_path)))
    per = collections.defaultdict(lambda: collections.defaultdict(list))
    order = sorted({(int(r["Dispatch_Id"]), r["Kernel_Name"]) for r in rows})
    split_seq = [d for d, n in order if kernel_class(n) == "gemm_o_or_down_residual"]
    split_cls = {d: ("gemm_o_residual" if i % 2 == 0 else "gemm_down_residual") for i, d in enumerate(split_seq)}
    for r in rows:
        d = int(r["Dispatch_Id"])
        cls = split_cls.get(d) or kernel_class(r["Kernel_Name"])
        per[(cls, r["Counter_Name"])][d].append(float(r["Counter_Value"]))
    out = {}
    for (cls, ctr), disp in sorted(per.items()):
        vals = [sum(v) for v in disp.values()]
        out.setdefault(cls, {})[ctr] = {"dispatches": len(vals), "avg": sum(vals) / len(vals), "max": max(vals)}
    if "copy" in out and copy_mib:
        for ctr, ent in out["copy"].items():
            kib = ent["max"]  # the calibration copy is the largest copyBuffer dispatch
            ent["factor_bytes_per_unit"] = copy_mib * 1024 * 1024 / (kib * 1024.0) if kib else None
    return out


def gpu_clock_mhz():
    """Current shader clock (MHz) read from the amdgpu driver's sysfs table right after the timed steps: the
    level marked '*' in pp_dpm_sclk of the first card that has one (None if unreadable). A file read, so
    nothing is started from the process that holds the GPU."""
    import glob
    import re
    for path in sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk")):
        try:
            with open(path) as f:
                for line in f:
                    if "*" in line:
                        m = re.search(r"(\d+)\s*Mhz", line, re.IGNORECASE)
                        if m:
                            return int(m.group(1))
        except OSError:
            continue
    return None


def step_flops(w, R):
    per = step_work(w, R)
    L = w.geom.n_layers
    return L * sum(v for k, v in per.items() if k != "gemm_lm_head_top2") + per["gemm_lm_head_top2"]


def host_description():
    """Host CPU model, logical CPUs, and the BLAS library numpy uses with its thread count."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas, threads = None, None
    try:
        from threadpoolctl import threadpool_info
        for info in threadpool_info():
            if info.get("user_api") == "blas":
                blas = f"{info.get('internal_api')} {info.get('version')}"
                threads = info.get("num_threads")
                break
    except Exception:
        pass
    return {"cpu_model": model, "logical_cpus": os.cpu_count(), "blas": blas, "blas_threads": threads}


def cpu_baseline(w, stored, tok, p, R, kv_host=None, full=True, layers_sample=8, rows_sample=64):
    """The float64 oracle on the same step, timed on the host. With ``full`` one whole oracle step (forward
    of every sequence over every layer, statistics of every scored row); otherwise a sample (the forward over
    ``layers_sample`` layers and the statistics of ``rows_sample`` rows) scaled to one step."""
    import numpy as np
    import oracle
    from oracle.numerics import WeightView
    host = host_description()
    cores = host["blas_threads"] or os.cpu_count() or 1
    W = WeightView(stored)
    g = w.geom
    kv = None
    if kv_host is not None:
        def kv(b, l):
            import synth
            k, v = kv_host[l]
            return synth.bf16_bits_to_f32(k[b]), synth.bf16_bits_to_f32(v[b])
        kv.prefix = w.kv_prefix
    if full:
        t0 = time.perf_counter()
        oracle.step(g, W, tok, p, w.gen_end, kv=kv)
        est = time.perf_counter() - t0
        sample = (f"one full float64 oracle step of the same workload (forward of {tok.shape[0]} x {tok.shape[1]} "
                  f"tokens over {g.n_layers} layers, statistics of {R} scored rows), measured: {est:.1f} s")
    else:
        gs = dataclasses.replace(g, n_layers=layers_sample)
        pos = w.kv_prefix + np.arange(w.seq)
        t0 = time.perf_counter()
        hf = oracle.forward(gs, W, tok[0], pos)
        t1 = time.perf_counter()
        rows = np.nonzero(oracle.scored_mask(tok, p, w.gen_end, g.mask_id)[0])[0][:rows_sample]
        oracle.row_stats(oracle.lm_logits(W, hf[rows]))
        t2 = time.perf_counter()
        est = ((t1 - t0) * g.n_layers / layers_sample * tok.shape[0] + (t2 - t1) * R / max(len(rows), 1))
        sample = (f"float64 oracle forward of one sequence over {layers_sample} of {g.n_layers} layers ({t1 - t0:.1f} s)"
                  f" and statistics of {len(rows)} of {R} scored rows ({t2 - t1:.1f} s), scaled to one step: "
                  f"{est:.1f} s")
    return {"value": 1.0 / est, "unit": "steps/s", "cores": int(cores), "kind": "oracle", "sample": sample,
            "seconds_per_step": est, "host": host}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="c2", help="synth workload key (c2 = LLaDA-8B shape, B1, S384)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="skip the event-timed kernel-class pass")
    ap.add_argument("--no-generate", action="store_true", help="skip the end-to-end decode (dcl_generate) run")
    ap.add_argument("--select", choices=("dcv", "noncontiguous", "chain-drafts"), default="dcv",
                    help="selection rule: Dynamic Contiguous Verification with drafts (default), the independent "
                         "threshold rule, or drafts restricted to the leading chain")
    ap.add_argument("--score-all", action="store_true", help="score every uncommitted position, not only masks")
    ap.add_argument("--suppress-mask", action="store_true", help="leave the [MASK] id out of the vocabulary")
    ap.add_argument("--graph", choices=("auto", "on", "off"), default="auto",
                    help="also time the step replayed from a captured HIP graph and report that rate (auto: for the "
                         "launch-bound tiny workload c1)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after timing, copy a buffer of this many MiB (hardware-counter calibration)")
    ap.add_argument("--pmc-summary", metavar="CSV", help="summarise a rocprofv3 --pmc counter_collection.csv "
                    "per kernel class and exit (with --copy-calibration-mib of the profiled run)")
    args = ap.parse_args()
    if args.pmc_summary:
        summ = pmc_summary(args.pmc_summary, args.copy_calibration_mib)
        print(json.dumps({"source_digest": kernel_source_digest(), "classes": summ}, indent=1))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the library has no multi-GPU path (asked for --gpus {args.gpus}); "
              "one process drives one GPU", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2607_20467_amd as dcl
    import synth

    w = synth.WORKLOADS[args.workload]
    g = w.geom
    log(f"workload {w.key}: {w.description}")
    t = time.perf_counter()
    stored = synth.make_weights(g)
    log(f"generated {g.name} weights in {time.perf_counter() - t:.1f} s")
    names = [n for n, _, _ in synth.tensor_specs(g)]
    t = time.perf_counter()
    run = dcl.Runner(g, [stored[n] for n in names], max_positions=max(4096, w.kv_prefix + w.seq))
    log(f"loaded weights into HBM in {time.perf_counter() - t:.1f} s")
    tok_h, p_h = synth.initial_state(w)
    B, S = tok_h.shape
    inside = (np.arange(S)[None] >= p_h[:, None]) & (np.arange(S)[None] < w.gen_end)
    R = int((inside if args.score_all else inside & (tok_h == g.mask_id)).sum())
    score_flags = (dcl.DCL_SCORE_ALL_UNCOMMITTED if args.score_all else 0) | \
        (dcl.DCL_SCORE_SUPPRESS_MASK if args.suppress_mask else 0)
    sel_flags = (dcl.DCL_SEL_SCORE_ALL if args.score_all else 0) | \
        {"dcv": 0, "noncontiguous": dcl.DCL_SEL_NONCONTIGUOUS, "chain-drafts": dcl.DCL_SEL_CONTIGUOUS_DRAFTS}[args.select]
    tok0 = torch.from_numpy(tok_h).cuda()
    p0 = torch.from_numpy(p_h).cuda()
    tok = tok0.clone()
    p = p0.clone()
    kv = None
    if w.kv_prefix:
        caches = [synth.kv_cache_layer(w, l) for l in range(g.n_layers)]
        kv = ([torch.from_numpy(c[0].view(np.int16)).cuda() for c in caches],
              [torch.from_numpy(c[1].view(np.int16)).cuda() for c in caches], w.kv_prefix)
        del caches
    stats = run.new_stats(B, S)
    ws, ws_bytes = run.workspace(B, S, w.kv_prefix)
    k_raw = torch.zeros(B, dtype=torch.int32, device="cuda")
    k_eff = torch.zeros(B, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()

    def one_step(st=None):
        st = stream if st is None else st
        tok.copy_(tok0, non_blocking=True)
        p.copy_(p0, non_blocking=True)
        dcl.dcl_denoise_step(run.model, tok, B, S, p, w.gen_end, kv, score_flags, stats, ws, ws_bytes, st)
        dcl.dcl_select_contiguous(tok, B, S, p, w.gen_end, w.window, w.tau_commit, w.tau_draft, g.mask_id, stats,
                                  k_raw, k_eff, sel_flags, st)

    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    log(f"timing {args.steps} steps")
    # per-step HIP events on the launch stream (the whole-run clock below gives `value`)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t0 = time.perf_counter()
    evs[0].record(stream)
    for i in range(args.steps):
        one_step()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    step_ms = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
    clock = gpu_clock_mhz()
    ms = 1000.0 * elapsed / args.steps
    launch = {"mode": "eager", "eager_ms_per_step": round(ms, 4)}
    if args.graph == "on" or (args.graph == "auto" and w.key == "c1"):
        # the same step captured once into a HIP graph (torch's CUDAGraph on a side stream) and replayed:
        # for a launch-latency-bound step this removes the per-kernel host launch cost
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            with torch.cuda.graph(graph, stream=side):
                one_step(side)
        torch.cuda.synchronize()
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        evs[0].record(stream)
        for i in range(args.steps):
            graph.replay()
            evs[i + 1].record(stream)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        step_ms = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
        ms = 1000.0 * elapsed / args.steps
        launch.update(mode="hip graph replay", graph_ms_per_step=round(ms, 4))
        log(f"eager {launch['eager_ms_per_step']:.4f} ms/step, graph replay {ms:.4f} ms/step")
    steps_per_s = 1000.0 / ms
    flops = step_flops(w, R)
    mfma_util = 100.0 * flops / (ms * 1e-3) / (BF16_PEAK_TFLOPS * 1e12)
    log(f"{ms:.3f} ms/step, {steps_per_s:.1f} steps/s, {R * steps_per_s:.0f} scored tok/s, "
        f"{flops / 1e12:.3f} TFLOP/step -> {mfma_util:.1f}% of bf16 peak; K_eff {k_eff.cpu().tolist()}")

    roofline = None
    classes = None
    if not args.no_profile:
        dcl.dcl_profile_enable(True)
        for _ in range(args.steps):
            one_step()
        torch.cuda.synchronize()
        prof = dcl.dcl_profile_read()
        dcl.dcl_profile_enable(False)
        per = step_work(w, R)
        classes = {}
        for name, (n, tms) in prof.items():
            if n == 0:
                continue
            avg_us = 1000.0 * tms / n
            ent = {"launches_per_step": n / args.steps, "avg_us": round(avg_us, 2),
                   "ms_per_step": round(tms / args.steps, 4)}
            if name in per:
                ent["tflops"] = round(per[name] / (avg_us * 1e-6) / 1e12, 1)
            classes[name] = ent
            log(f"  {name:22s} {n / args.steps:6.1f} launches/step  avg {avg_us:9.2f} us  "
                f"{tms / args.steps:8.3f} ms/step" + (f"  {ent['tflops']:7.1f} TFLOP/s" if "tflops" in ent else ""))
        launch["kernels_per_step"] = round(sum(e["launches_per_step"] for e in classes.values()), 2)
        launch["event_timed_kernel_ms_per_step"] = round(sum(e["ms_per_step"] for e in classes.values()), 4)
        alg_bytes = step_bytes(w, R)
        for name, ent in classes.items():
            if name in alg_bytes:
                ent["gbs"] = round(alg_bytes[name] / (ent["avg_us"] * 1e-6) / 1e9, 1)
        dom = max((k for k in classes if k in per), key=lambda k: classes[k]["ms_per_step"])
        ach = per[dom] / (classes[dom]["avg_us"] * 1e-6) / 1e12
        tr = stored_traffic(dom, w.key)
        roofline = {"bound": "mfma", "kernel": dom, "achieved": round(ach, 1), "peak": BF16_PEAK_TFLOPS,
                    "unit": "TFLOP/s", "frac": round(ach / BF16_PEAK_TFLOPS, 4),
                    "traffic": tr["hbm_bytes_per_launch"] if tr else None,
                    "flop_per_launch": per[dom], "algorithmic_bytes_per_launch": alg_bytes[dom],
                    "avg_launch_us": classes[dom]["avg_us"]}

    gen = None
    if not args.no_generate:
        # Algorithm 1 end to end from the workload's initial state (dcl_generate: graph-replayed
        # iterations, completion checked on the host after each one): block-free with the workload's
        # window, then semi-autoregressive blocks of 32 with windows of 32 and 128 (the paper's setup)
        def generate(L, block_len):
            torch.cuda.synchronize()
            tok.copy_(tok0)
            p.copy_(p0)
            hist = torch.zeros(L + 1, dtype=torch.int32, device="cuda")
            max_steps = int(w.gen_end - p_h.min())
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            n_it = dcl.dcl_generate(run.model, tok, B, S, p, w.gen_end, kv, score_flags, L, w.tau_commit,
                                    w.tau_draft, sel_flags, max_steps, 1, stats, k_raw, k_eff, hist, ws, ws_bytes,
                                    stream, block_origin=w.prompt_len if not w.kv_prefix else 0,
                                    block_len=block_len)
            torch.cuda.synchronize()
            t_gen = time.perf_counter() - t1
            new_tok = int((w.gen_end - p_h).clip(min=0).sum())
            done = bool((p.cpu().numpy() >= w.gen_end).all())
            rec = {"window": L, "block_len": block_len, "iterations": n_it, "finished": done, "tokens": new_tok,
                   "seconds": round(t_gen, 4), "tokens_per_s": round(new_tok / t_gen, 1),
                   "tokens_per_iteration": round(new_tok / max(n_it, 1), 3),
                   "ms_per_iteration": round(1000 * t_gen / max(n_it, 1), 4), "k_eff_hist": hist.cpu().tolist()}
            log(f"generation (window {L}, blocks {block_len or 'none'}): {n_it} iterations for {new_tok} tokens "
                f"in {t_gen:.3f} s ({new_tok / t_gen:.0f} tok/s, {1000 * t_gen / max(n_it, 1):.2f} ms/iteration)")
            return rec

        gen = generate(w.window, 0)
        gen["blocked"] = [generate(L, 32) for L in (32, 128)]

    if args.copy_calibration_mib:
        n = args.copy_calibration_mib * 1024 * 1024 // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copied {args.copy_calibration_mib} MiB three times (counter calibration)")
        del src, dst

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the float64 oracle on a bounded sample (CPU baseline)")
        kv_host = [synth.kv_cache_layer(w, l) for l in range(g.n_layers)] if w.kv_prefix else None
        cpu = cpu_baseline(w, stored, tok_h, p_h, R, kv_host, full=w.key in ("c1", "c2", "c5"))
        cpu = {k: (round(v, 6) if isinstance(v, float) else v) for k, v in cpu.items()}
        del kv_host
        log(f"  {cpu['sample']}")

    out = {
        "metric": METRIC, "value": round(steps_per_s, 3), "unit": "steps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{w.key}: {w.description}", "geometry": g.name, "batch": B, "seq_len": S,
                   "kv_prefix": w.kv_prefix, "scored_rows": R, "window": w.window, "tau_commit": w.tau_commit,
                   "tau_draft": w.tau_draft, "parallelism": "single GPU", "select": args.select,
                   "score_all": bool(args.score_all), "suppress_mask": bool(args.suppress_mask)},
        "step_ms": {"median": round(float(np.median(step_ms)), 4), "p10": round(float(np.percentile(step_ms, 10)), 4),
                    "p90": round(float(np.percentile(step_ms, 90)), 4)},
        "gpu_sclk_mhz": clock,
        "launch": launch,
        "scored_tokens_per_s": round(R * steps_per_s, 1),
        "mfma_util_pct": round(mfma_util, 2),
        "tflop_per_step": round(flops / 1e12, 4),
        "roofline": roofline,
        "kernel_classes": classes,
        "generation": gen,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
