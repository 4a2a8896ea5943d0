"""Benchmark: stream-batched rectified-flow steps on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config s512] [--no-cpu]

A step is one sf_stream_step over a full queue: one heterogeneous-timestep velocity
network call over every in-flight latent, each latent's Euler update, and the shift
that admits the next fresh latent (one finished latent leaves per step). Inputs
(weights, latents, a pool of fresh latents) are resident in HBM before timing.

The headline (value, ms_per_step, images/s) is the step replayed from captured HIP
graphs (sf_graph_enable: the same kernels, captured once per distinct call); the
eagerly launched step is reported beside it under "eager" (--no-graph makes it the
headline). The replayed step with the modulation cache on (sf_modulation_cache: the
per-sample conditioning computed once while every slot keeps its t) is reported
separately under "graph_replay_modulation_cached" and is never the headline.

Prints one JSON line: latent-steps/s (value), images/s, the median step, the roofline
of the dominant kernel class (timed with HIP events attached to its dispatches during
the timed steps), the per-class time breakdown and the achieved GB/s of the
memory-bound classes, the Alg. 2 rate over 100 images including the fill phase, the
one-latent-at-a-time rate (no stream batching), and the oracle timed on the host
cores as a CPU baseline.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402

METRIC = "stream-batched RF latent-steps/s and images/s at 512² (K=4); MFMA util %"
MI355X_PEAK_BF16_TFLOPS = 2500.0
MI355X_PEAK_FP32_TFLOPS = 157.3
MI355X_HBM_GBS = 8000.0

# HBM bytes per launch of a kernel class, from two rocprofv3 --pmc passes (FETCH_SIZE,
# then WRITE_SIZE, KiB per dispatch) over `bench.py --steps 5 --warmup 2 --no-cpu --no-graph
# --no-sequential --copy-calibration`, each scaled by what the same counter reads for a
# plain 256 MiB elementwise copy (FETCH_SIZE x 2.000, WRITE_SIZE x 1.000). An entry holds
# only for the kernel sources it was measured on (hash below); otherwise traffic is null.
KERNEL_SOURCES = ("k_gemm.hip", "k_attn.hip", "sf_device.h", "sf_launch.h")
TRAFFIC = {
    ("s512", "bf16", "FC2"): {"bytes": 94525086, "sources": "cac1cfd0c9deab6b",
                              "profile": "profiles/stream_step_s512_bf16_hbm_traffic.md"},
    ("s512", "bf16", "FC1"): {"bytes": 59987705, "sources": "cac1cfd0c9deab6b",
                              "profile": "profiles/stream_step_s512_bf16_hbm_traffic.md"},
    ("s512_large", "bf16", "FC2"): {"bytes": 187609226, "sources": "cac1cfd0c9deab6b",
                                    "profile": "profiles/stream_step_s512_large_bf16.md"},
    ("s512_large", "bf16", "FC1"): {"bytes": 134056520, "sources": "cac1cfd0c9deab6b",
                                    "profile": "profiles/stream_step_s512_large_bf16.md"},
    ("s512_cfg", "bf16", "FC2"): {"bytes": 392050527, "sources": "cac1cfd0c9deab6b",
                                  "profile": "profiles/stream_step_s512_cfg_bf16.md"},
    ("s1024", "bf16", "ATTN"): {"bytes": 161797938, "sources": "cac1cfd0c9deab6b",
                                "profile": "profiles/stream_step_s1024_bf16.md"},
}


def kernel_sources_hash():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2511_22009_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def class_work(cfg, kc, rows):
    """Algorithmic FLOPs of ONE launch of kernel class kc (GEMM classes and attention)."""
    from paper_2511_22009_amd import KernelClass as KC
    M, D, N, F = rows * cfg.N, cfg.D, cfg.N, cfg.mlp
    return {
        KC.QKV: 2.0 * M * D * 3 * D,
        KC.PROJ: 2.0 * M * D * D,
        KC.FC1: 2.0 * M * D * F,
        KC.FC2: 2.0 * M * F * D,
        KC.ATTN: 4.0 * rows * N * N * D,
    }.get(kc)


def class_bytes(cfg, kc, es):
    """Algorithmic HBM bytes of ONE launch of a memory-bound kernel class (read once +
    write once at the kernel's dtypes); es = bytes per element of bf16/fp32 operands."""
    from paper_2511_22009_amd import KernelClass as KC
    R, N, D, E, P = cfg.rows, cfg.N, cfg.D, cfg.C * cfg.H * cfg.W, cfg.patch_dim
    M, B = R * N, cfg.K
    modw = cfg.L * 6 * D + 2 * D
    return {
        KC.TEMB: cfg.tdim * D * 4 + D * D * 4 + modw * D * es + B * modw * 4,
        KC.EMBED: B * E * 4 + P * D * 4 + N * D * 4 + M * D * 4,
        KC.LN: M * D * 4 + M * D * es,
        KC.HEAD: M * D * 4 + P * D * 4 + R * E * 4,
        KC.EULER: (B + R + 1) * E * 4 + (B + 1) * E * 4,
    }.get(kc)


def cpu_baseline(cfg, budget_s=12.0):
    """Oracle stream steps on the host cores until about budget_s seconds of work."""
    import oracle
    from threadpoolctl import threadpool_info
    blob = W.make_blob(cfg)
    m = oracle.load_blob(blob)
    t, dt = W.slot_times(cfg)
    x = W.latents(cfg, cfg.K)
    kw = {}
    if cfg.cfg:
        kw = dict(ctx=W.context(cfg, cfg.K), null_ctx=W.null_context(cfg), guidance=cfg.guidance)
    # one sample's forward first, to size the run
    t0 = time.perf_counter()
    oracle.stream_step(m, x[:1], t[:1], dt[:1], x[0], **({k: (v[:1] if k == "ctx" else v) for k, v in kw.items()}))
    one = time.perf_counter() - t0
    steps = max(1, int(budget_s / max(one * cfg.K, 1e-9)))
    t0 = time.perf_counter()
    for _ in range(steps):
        x, _, _ = oracle.stream_step(m, x, t, dt, x[0], **kw)
    el = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
    return {"value": cfg.K * steps / el, "unit": "latent-steps/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{steps} full stream step(s) of the {cfg.name} workload ({cfg.K} latents each), "
                      f"NumPy fp32, {el:.1f} s",
            "single_thread": single_thread_baseline(cfg, m, x, t, dt, kw)}


def single_thread_baseline(cfg, m, x, t, dt, kw):
    """The oracle on ONE host thread: the bench workload on a bounded sample (one
    latent's network call and Euler update, i.e. one latent-step) and Tiny over 100
    full stream steps."""
    import oracle
    from threadpoolctl import threadpool_limits
    out = {}
    with threadpool_limits(limits=1):
        one_kw = {k: (v[:1] if k == "ctx" else v) for k, v in kw.items()}
        t0 = time.perf_counter()
        oracle.stream_step(m, x[:1], t[:1], dt[:1], x[0], **one_kw)
        el = time.perf_counter() - t0
        out[cfg.name] = {"value": 1.0 / el, "unit": "latent-steps/s", "cores": 1,
                         "sample": f"one latent-step of the {cfg.name} workload, {el:.1f} s"}
        tiny = W.get_config("tiny")
        tm = oracle.load_blob(W.make_blob(tiny))
        tt, tdt = W.slot_times(tiny)
        tx = W.latents(tiny, tiny.K)
        t0 = time.perf_counter()
        for _ in range(100):
            tx, _, _ = oracle.stream_step(tm, tx, tt, tdt, tx[0])
        el = time.perf_counter() - t0
        out["tiny"] = {"value": tiny.K * 100 / el, "unit": "latent-steps/s", "cores": 1,
                       "sample": f"100 full stream steps of the tiny workload ({tiny.K} latents each), {el:.2f} s"}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="s512")
    ap.add_argument("--precision", default="bf16", choices=["bf16", "fp32"])
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--no-graph", action="store_true", help="skip the graph-replay measurement")
    ap.add_argument("--no-sequential", action="store_true",
                    help="skip the one-latent-at-a-time comparison run (keeps profiles to the batched step)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed steps, run a plain 256 MiB elementwise copy kernel (three times) "
                         "whose FETCH_SIZE / WRITE_SIZE counters scale the kernels' HBM traffic")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (--gpus {args.gpus} requested): the stream step has no "
              "multi-GPU path; independent queues per GPU would each report this single-GPU rate.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2511_22009_amd import Cond, KernelClass, Model, Precision

    cfg = W.get_config(args.config)
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    blob = W.make_blob(cfg)
    m = Model(blob, Precision[args.precision.upper()], max_rows=cfg.rows)
    t, dt = W.slot_times(cfg)
    K = cfg.K
    x = torch.from_numpy(W.latents(cfg, K)).to(dev)
    pool = torch.from_numpy(W.latents(cfg, 16, seed=W.gen.SEED_IMAGE_BASE)).to(dev)
    done = torch.empty(cfg.latent_shape, device=dev)
    cond = None
    if cfg.has_cross:
        cond = Cond(torch.from_numpy(W.context(cfg, K)).to(dev), torch.from_numpy(W.null_context(cfg)).to(dev),
                    cfg.guidance)
    stream = torch.cuda.current_stream()

    def step(i):
        m.stream_step(x, t, dt, K, pool[i % pool.shape[0]], done, cond, stream)

    # warmup (untimed), then a separate pass with every kernel class event-timed to
    # get the per-class breakdown and pick the dominant class
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    n_break = max(3, min(10, args.steps))
    for kc in KernelClass:
        m.timing_enable(kc, True)
    for i in range(n_break):
        step(i)
    torch.cuda.synchronize()
    breakdown = {}
    for kc in KernelClass:
        ms, n = m.timing_read(kc)
        m.timing_enable(kc, False)
        if n:
            breakdown[kc.name] = {"ms_per_step": ms / n_break, "launches_per_step": n / n_break}
    dom = max((kc for kc in KernelClass if kc.name in breakdown and class_work(cfg, kc, cfg.rows)),
              key=lambda kc: breakdown[kc.name]["ms_per_step"])

    # timed region: exactly `steps` steps, events on the dominant class only
    m.timing_enable(dom, True)
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        marks[i].record(stream)
        step(args.warmup + i)
    marks[-1].record(stream)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    per_step_ms = sorted(marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps))
    dom_ms, dom_n = m.timing_read(dom)
    m.timing_enable(dom, False)
    if not bool(torch.isfinite(x).all()):
        raise RuntimeError("non-finite latents after the timed steps")

    ms_step = 1e3 * el / args.steps
    value = K / (el / args.steps)
    work = class_work(cfg, dom, cfg.rows)
    avg_launch_s = dom_ms / 1e3 / max(dom_n, 1)
    achieved = work / avg_launch_s / 1e12
    peak = MI355X_PEAK_BF16_TFLOPS if args.precision == "bf16" else MI355X_PEAK_FP32_TFLOPS
    es = 2 if args.precision == "bf16" else 4
    mem = {}
    for kc in KernelClass:
        b = class_bytes(cfg, kc, es)
        if b and kc.name in breakdown:
            us = 1e3 * breakdown[kc.name]["ms_per_step"] / breakdown[kc.name]["launches_per_step"]
            mem[kc.name] = {"us_per_launch": round(us, 2), "bytes_per_launch": b,
                            "GBps": round(b / us / 1e3, 1), "frac_of_hbm": round(b / us / 1e3 / MI355X_HBM_GBS, 3)}
    tr = TRAFFIC.get((cfg.name, args.precision, dom.name))
    traffic = tr["bytes"] if tr and tr["sources"] == kernel_sources_hash() else None
    gemm_ms = sum(breakdown[k]["ms_per_step"] for k in ("QKV", "PROJ", "FC1", "FC2") if k in breakdown)
    gemm_tflops = cfg.gemm_flops_per_step() / (gemm_ms / 1e3) / 1e12 if gemm_ms else None

    # the same kernels one latent at a time (no stream batching): K network calls per image
    # the same steps replayed from captured HIP graphs on a side stream (one graph per
    # distinct call: the fresh-latent pool has 16 entries, so 16 graphs after warm-up)
    graph = None
    cached_mod = None
    ctx_reuse = None
    if not args.no_graph:
        gs = torch.cuda.Stream()

        def gstep(i):
            m.stream_step(x, t, dt, K, pool[i % pool.shape[0]], done, cond, gs)

        def replay_run(fn=gstep):
            torch.cuda.synchronize()
            for i in range(pool.shape[0] + max(2, args.warmup)):
                fn(i)
            # the timed steps carry no per-step events (an event between two graph
            # launches adds a few microseconds to every step); the median step comes
            # from a separate pass with an event before every step
            torch.cuda.synchronize()
            g0 = time.perf_counter()
            for i in range(args.steps):
                fn(i)
            torch.cuda.synchronize()
            gel = time.perf_counter() - g0
            if not bool(torch.isfinite(x).all()):
                raise RuntimeError("non-finite latents after the graph-replay steps")
            n_med = min(args.steps, 20)
            gmarks = [torch.cuda.Event(enable_timing=True) for _ in range(n_med + 1)]
            for i in range(n_med):
                gmarks[i].record(gs)
                fn(i)
            gmarks[-1].record(gs)
            torch.cuda.synchronize()
            g_steps = sorted(gmarks[i].elapsed_time(gmarks[i + 1]) for i in range(n_med))
            return {"ms_per_step": 1e3 * gel / args.steps, "latent_steps_per_s": K / (gel / args.steps),
                    "median_ms_per_step": g_steps[len(g_steps) // 2]}

        m.graph_enable(True)
        graph = replay_run()
        graph["graphs_cached"], graph["replays"] = m.graph_stats()
        # reported separately, never the headline: the same replayed steps with the
        # modulation cache on (in the steady state every slot keeps its t, so the
        # conditioning launches run once and later steps reuse the adaLN table)
        m.modulation_cache(True)
        cached_mod = replay_run()
        cached_mod["skipped_conditioning_calls"] = m.modulation_cache_stats()
        m.modulation_cache(False)
        # reported separately too: with cross-attention, the replayed steps with the
        # context entries kept across calls while the contexts move through the queue as
        # in Alg. 2 (a window sliding down a pool of contexts: each step's slot k holds
        # the context slot k - 1 held the step before, and slot 0 a new one)
        if cond is not None:
            P = pool.shape[0]
            ctx_pool = torch.from_numpy(W.context(cfg, P + K, seed=W.gen.SEED_IMAGE_BASE + 7)).to(dev)

            def cstep(i):
                w = (P - 1) - (i % P)
                m.stream_step(x, t, dt, K, pool[i % P], done, Cond(ctx_pool[w:w + K], cond.null_ctx, cond.guidance), gs)

            m.context_cache(True)
            ctx_reuse = replay_run(cstep)
            calls, projected = m.context_cache_stats()
            ctx_reuse["contexts_projected_per_step"] = projected / max(calls, 1)
            m.context_cache(False)
        m.graph_enable(False)

    # Alg. 2 end to end: M = 100 images through the fill phase and the full queue
    # (M + K - 1 stream steps, host driver included)
    fill_img_s = None
    if not args.no_sequential:
        from paper_2511_22009_amd.pipeline import run_images
        grid = W.schedule(cfg)
        ctx_of = None
        if cond is not None:
            ctx_of = lambda j: cond.ctx[j % K]  # noqa: E731
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        imgs = run_images(m, grid, 100, lambda j: pool[j % pool.shape[0]], ctx_of,
                          cond.null_ctx if cond is not None else None, cfg.guidance if cond is not None else None)
        torch.cuda.synchronize()
        fill_img_s = len(imgs) / (time.perf_counter() - t2)
        del imgs

    seq_img_s = None
    if not args.no_sequential:
        seq_steps = max(4, args.steps // 10)
        x1 = x[:1].clone()
        done1 = torch.empty_like(done)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        cond1 = None if cond is None else Cond(cond.ctx[:1], cond.null_ctx, cond.guidance)
        for i in range(seq_steps):
            for s in range(K):
                # a one-slot queue: the updated latent leaves through `done1` and, until the
                # image is finished, re-enters slot 0 as the "fresh" latent
                z = done1 if s < K - 1 else pool[i % pool.shape[0]]
                m.stream_step(x1, t[s:s + 1], dt[s:s + 1], 1, z, done1, cond1, stream)
        torch.cuda.synchronize()
        seq_img_s = seq_steps / (time.perf_counter() - t1)

    # The headline is the graph-replayed step (the library's static-execution mode: one
    # capture per distinct call, replayed with the same kernels and bit-identical
    # results); the eagerly launched step is reported beside it.
    eager = {"ms_per_step": ms_step, "latent_steps_per_s": value, "images_per_s": 1e3 / ms_step,
             "median_ms_per_step": per_step_ms[len(per_step_ms) // 2]}
    if graph is not None:
        head_ms, head_value, head_median = graph["ms_per_step"], graph["latent_steps_per_s"], graph["median_ms_per_step"]
    else:
        head_ms, head_value, head_median = ms_step, value, eager["median_ms_per_step"]
    out = {
        "metric": METRIC,
        "value": head_value,
        "unit": "latent-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.precision,
        "data": "synthetic (seeded random-init weights N(0,0.02), N(0,1) latents)",
        "config": {
            "workload": f"{cfg.name}: latent {cfg.C}x{cfg.H}x{cfg.W}, {cfg.N} tokens, width {cfg.D}, depth {cfg.L}, "
                        f"{cfg.heads} heads, MLP {cfg.mlp}, {K} stream slots ({cfg.rows} network rows), "
                        f"schedule {cfg.schedule}",
            "slots": K, "rows": cfg.rows, "tokens": cfg.N, "width": cfg.D, "depth": cfg.L,
        },
        "execution": "hip-graph replay" if graph is not None else "eager launches",
        "images_per_s": 1e3 / head_ms,
        "median_ms_per_step": head_median,
        "fill_inclusive_images_per_s_M100": fill_img_s,
        "graph_replay": graph,
        "eager": eager,
        "graph_replay_modulation_cached": cached_mod,
        "graph_replay_context_reuse": ctx_reuse,
        "step_tflops": cfg.flops_per_step() / (head_ms / 1e3) / 1e12,
        "step_frac_of_peak": cfg.flops_per_step() / (head_ms / 1e3) / 1e12 / peak,
        "gemm_tflops": gemm_tflops,
        "gemm_frac_of_peak": (gemm_tflops / peak) if gemm_tflops else None,
        "sequential_images_per_s": seq_img_s,
        "roofline": {
            "kernel": dom.name,
            "bound": "mfma",
            "achieved": achieved,
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": achieved / peak,
            "traffic": traffic,
            "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
            "traffic_profile": tr["profile"] if traffic else None,
            "flops_per_launch": work,
            "avg_launch_us": avg_launch_s * 1e6,
            "launches_timed": dom_n,
        },
        "breakdown_ms_per_step": {k: round(v["ms_per_step"], 4) for k, v in breakdown.items()},
        "memory_kernels": mem,
    }
    m.close()
    if args.copy_calibration:
        src = torch.ones(64 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)  # an elementwise kernel: reads and writes 256 MiB
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = src.numel() * 4
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(cfg)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
