#!/usr/bin/env python3
"""Benchmark of the R-iKFAD optimiser step on one MI355X.

Workload: the GPT2-S-shaped parameter set (124,439,808 parameters: 50
matrices + 98 bias / LayerNorm vectors), seeded synthetic data resident in
HBM: x ~ N(0, 0.02^2), gradients g_ij = s_i t_j z_ij with log-normal row and
column scales, p = r = c = 0 at the start.  A step is one rikfad_step over
all 148 tensors (streaming kernel + finalisation kernel, deferred form).

Prints ONE JSON line.  value = parameters updated per second (whole job);
roofline = the streaming kernel's compulsory HBM bytes per launch divided
by its average duration (HIP events recorded by the library around each
launch on the step's stream) against the 8 TB/s HBM peak; cpu_baseline =
the fp64 oracle timed on the host cores on a bounded sample.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "optimiser-step params/sec and achieved HBM GB/s (% of peak), GPT2-S-shaped"
PEAK_GBPS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "stream_kernel_gpt2s_traffic.json")


def kernel_source_hash():
    h = hashlib.sha256()
    for nm in ("kernels.hip", "device.hpp", "layout.hpp", "plan.cpp"):
        with open(os.path.join(ROOT, "paper_2609_30342_amd", "csrc", nm), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(dtype):
    """HBM bytes per streaming launch from the committed rocprofv3 counter
    runs, or None if they were taken on a different kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_hash") != kernel_source_hash():
        return None
    entry = rec.get(dtype)
    return None if entry is None else entry.get("bytes_per_launch")


# The chip's clocks ramp over the first ~20 ms of sustained load (shader
# clock 2.1 -> 2.38 GHz on MI355X; a GPT2-S step goes from ~516 us in its
# first ten steps to a steady ~415 us after about fifty) and drop again
# when it idles.  Every measurement, the headline included, therefore first
# keeps the GPU busy with the operation it is about to time for WARM_MS
# (the pre-warm), then makes its `warmup` untimed calls, then times.  In
# training the optimiser step follows the forward and backward passes,
# which keep the clocks up; a step timed on a cold chip measures the
# clock ramp, not the step.
WARM_MS = 60.0


def warm_up(step, count, warm_ms=WARM_MS):
    """Pre-warm: calls of step() until the GPU has been busy for at least
    warm_ms (synchronising every 8 calls); then `count` untimed calls.
    Returns the pre-warm's milliseconds and number of calls."""
    import torch
    calls, ms = 0, 0.0
    if warm_ms > 0:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        while (time.perf_counter() - t0) * 1e3 < warm_ms:
            for _ in range(8):
                step()
            calls += 8
            torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3
    for _ in range(count):
        step()
    return ms, calls


def build_workload(specs, dtype, seed, device, scales="lognormal"):
    """dtype None: each tensor in its own spec's storage type.  scales:
    "lognormal" row and column scales LogNormal(0, 0.5); "student_t" row
    scales |T| with T ~ Student-t(3) (drawn as z0 / sqrt((z1^2 + z2^2 +
    z3^2) / 3)), column scales 1."""
    import torch
    gen = torch.Generator(device=device).manual_seed(seed)
    xs, gs = [], []
    for sp in specs:
        dt = torch.bfloat16 if (dtype or sp.dtype) == "bf16" else torch.float32
        x = (torch.randn((sp.m, sp.n), generator=gen, device=device) * 0.02).to(dt)
        if scales == "student_t":
            z = torch.randn((4, sp.m), generator=gen, device=device)
            s = (z[0] / torch.sqrt((z[1:] ** 2).sum(0) / 3.0)).abs()
            t = torch.ones(sp.n, device=device)
        else:
            s = torch.exp(0.5 * torch.randn(sp.m, generator=gen, device=device))
            t = torch.exp(0.5 * torch.randn(sp.n, generator=gen, device=device))
        g = (torch.randn((sp.m, sp.n), generator=gen, device=device) * s[:, None]
             * t[None, :]).to(dt)
        xs.append(x.contiguous())
        gs.append(g.contiguous())
    return xs, gs


def time_rikfad(specs, dtype, hp, steps, warmup, two_pass=False, seed=0, scales="lognormal",
                warm_ms=WARM_MS):
    import torch
    from paper_2609_30342_amd import rikfad as R
    dev = torch.device("cuda:0")
    xs, gs = build_workload(specs, dtype, seed, dev, scales)
    opt = R.RIKFAD(xs, gs, two_pass=two_pass, **hp)
    info = opt.query()
    prewarm_ms, prewarm_steps = warm_up(opt.step, warmup, warm_ms)
    # Timed region: exactly `steps` steps, free of timing events.
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(steps):
        opt.step()
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end)
    # Kernel times: the same number of steps right after, with the library's
    # kernel timing (HIP start / stop events attached to the dispatches of
    # each phase, on the step's stream).  Timing events change the step --
    # a timed step takes 12-20 us longer and its streaming kernel runs up to
    # ~1% slower -- so they stay out of the timed region.
    R.rikfad_timing_enable(opt.ctx, True)
    for _ in range(steps):
        opt.step()
    R.rikfad_timing_enable(opt.ctx, False)
    k1, k2, k3, n = R.rikfad_timing_read(opt.ctx)
    nonfinite = opt.nonfinite()
    opt.close()
    del xs, gs
    torch.cuda.empty_cache()
    return dict(ms_per_step=ms / steps, stream_ms=k1 / n, finalize_ms=k2 / n,
                apply_ms=k3 / n, timed_steps=n, info=info, nonfinite=nonfinite,
                prewarm_ms=prewarm_ms, prewarm_steps=prewarm_steps)


def time_ikfad(specs, hp, steps, warmup, seed=0, dtype="fp32"):
    import torch
    from paper_2609_30342_amd import rikfad as R
    xs, gs = build_workload(specs, dtype, seed, torch.device("cuda:0"))
    ik = R.IKFAD(xs, gs, h=hp["h"], gamma=hp["gamma"], alpha=hp["alpha"], mu=hp["mu"])
    warm_up(ik.step, warmup)
    torch.cuda.synchronize()
    R.ikfad_timing_enable(ik.ctx, True)
    for _ in range(steps):
        ik.step()
    ms, n = R.ikfad_timing_read(ik.ctx)
    ik.close()
    del xs, gs
    torch.cuda.empty_cache()
    return ms / n


def time_adafm(specs, dtype, steps, warmup, seed=0, **hp):
    """Adafactor-m (the paper's baseline) on the same parameter set: whole
    step time and the library's per-pass event timing."""
    import torch
    from paper_2609_30342_amd import rikfad as R
    xs, gs = build_workload(specs, dtype, seed, torch.device("cuda:0"))
    opt = R.ADAFM(xs, gs, **hp)
    total, upd_bytes, state = R.adafm_min_bytes(opt.ctx)
    warm_up(opt.step, warmup)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(steps):
        opt.step()
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / steps
    R.adafm_timing_enable(opt.ctx, True)
    for _ in range(steps):
        opt.step()
    (stats, fin, rms, scale, upd), n = R.adafm_timing_read(opt.ctx)
    opt.close()
    del xs, gs
    torch.cuda.empty_cache()
    stats_b, rms_b = adafm_read_pass_bytes(specs, dtype)
    return {"ms_per_step": ms, "params_per_s": sum(s.numel for s in specs) / (ms * 1e-3),
            "hbm_gbps_step": total / (ms * 1e-3) / 1e9, "min_bytes_per_step": total,
            "state_bytes": state,
            "pass_ms": {"stats": stats / n, "finalize": fin / n, "rms": rms / n,
                        "scale": scale / n, "update": upd / n},
            "stats_gbps": stats_b / (stats / n * 1e-3) / 1e9,
            "rms_gbps": rms_b / (rms / n * 1e-3) / 1e9,
            "update_gbps": upd_bytes / (upd / n * 1e-3) / 1e9}


def adafm_read_pass_bytes(specs, dtype):
    """Compulsory bytes of Adafactor-m's two read passes (no parameter
    scaling): the statistics pass reads each matrix's gradient once and a
    vector's gradient plus its second moment, which it also writes; the RMS
    pass reads each matrix's gradient once (vectors finish in pass 1)."""
    es = 2 if dtype == "bf16" else 4
    mat = sum(s.numel for s in specs if s.m > 1 and s.n > 1)
    vec = sum(s.numel for s in specs if s.m == 1 or s.n == 1)
    return es * mat + (es + 8) * vec, es * mat


def time_small(specs, hp, steps, warmup, seed=0):
    """Launch-bound parameter sets: microseconds per step issued eagerly and
    replayed from a HIP graph that holds one captured step."""
    import torch
    from paper_2609_30342_amd import rikfad as R
    xs, gs = build_workload(specs, None, seed, torch.device("cuda:0"))
    opt = R.RIKFAD(xs, gs, **hp)
    warm_up(opt.step, warmup)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    for _ in range(steps):
        opt.step()
    b.record()
    torch.cuda.synchronize()
    eager = a.elapsed_time(b) / steps
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        opt.step()
    warm_up(g.replay, 1)
    a.record()
    for _ in range(steps):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    graph = a.elapsed_time(b) / steps
    # Ten steps in one graph: a graph launch has a fixed cost, which a
    # graph holding a whole training iteration pays once.
    g10 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g10):
        for _ in range(10):
            opt.step()
    warm_up(g10.replay, 1)
    a.record()
    for _ in range(max(1, steps // 10)):
        g10.replay()
    b.record()
    torch.cuda.synchronize()
    graph10 = a.elapsed_time(b) / (max(1, steps // 10) * 10)
    n = sum(sp.numel for sp in specs)
    info = opt.query()
    opt.close()
    del g, g10, xs, gs
    torch.cuda.empty_cache()
    best = min(eager, graph, graph10)
    # The ceiling at this size: the step's access mix without arithmetic,
    # in the streaming kernel's tiles, over the same number of elements of
    # the set's storage type (one launch, no finalisation).
    dt = "bf16" if all(sp.dtype == "bf16" for sp in specs) else "fp32"
    nel = (n // 256) * 256
    probe_gbps = time_probe_mix(nel, dt, 1, reps=200)
    return {"params": n, "eager_us": eager * 1e3, "graph_us": graph * 1e3,
            "graph_10_steps_us": graph10 * 1e3,
            "graph_params_per_s": n / (graph * 1e-3),
            "min_bytes_per_step": info["min_bytes_per_step"],
            "hbm_frac_step": info["min_bytes_per_step"] / (best * 1e-3) / 1e9 / PEAK_GBPS,
            "probe_mix_tiles_us": info["min_bytes_per_step"] / (probe_gbps * 1e9) * 1e6,
            "probe_mix_tiles_frac": probe_gbps / PEAK_GBPS}


def time_friction_report(m, n, iters=30, reps=3):
    """Rank-1 friction diagnostic on an m x n friction tensor: ms per call and
    GB/s on the passes over xi it makes, 4 m n bytes each: iters + 2 when
    n <= 1024 (factors; errors with the first power iteration; one pass per
    iteration; sigma_1), 2 iters + 4 otherwise."""
    import torch
    from paper_2609_30342_amd import rikfad as R
    gen = torch.Generator(device="cuda:0").manual_seed(7)
    xi = torch.rand((m, n), generator=gen, device="cuda:0")
    s = torch.cuda.current_stream().cuda_stream
    warm_up(lambda: R.rikfad_friction_report(xi.data_ptr(), m, n, 1e-16, iters, s), 1)
    t0 = time.perf_counter()
    for _ in range(reps):
        R.rikfad_friction_report(xi.data_ptr(), m, n, 1e-16, iters, s)
    ms = (time.perf_counter() - t0) / reps * 1e3
    passes = iters + 2 if n <= 1024 else 2 * iters + 4
    del xi
    torch.cuda.empty_cache()
    return {"shape": [m, n], "power_iters": iters, "ms": ms,
            "gbps": passes * 4.0 * m * n / (ms * 1e-3) / 1e9}


def _time_calls(fn, reps):
    import torch
    warm_up(fn, 1)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        fn()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps


def time_probe(nfloat, reps=50):
    """3-read / 2-write fp32 stream of the same byte count as the step, over
    five separate buffers (d = a + b, e = a * c)."""
    import torch
    from paper_2609_30342_amd import rikfad as R
    bufs = [torch.empty(nfloat, device="cuda:0") for _ in range(5)]
    for b in bufs[:3]:
        b.normal_()
    s = torch.cuda.current_stream().cuda_stream
    ptrs = [b.data_ptr() for b in bufs]
    ms = _time_calls(lambda: R.rikfad_probe_stream(*ptrs, nfloat, s), reps)
    del bufs
    torch.cuda.empty_cache()
    return 20.0 * nfloat / (ms * 1e-3) / 1e9


def time_probe_mix(nelem, dtype, shape, reps=50):
    """The step's access mix without its arithmetic, in place: read x, g, p
    and write x, p (20 B per element fp32, 14 B bf16); shape 0 contiguous,
    shape 1 the streaming kernel's tiles.  GB/s."""
    import torch
    from paper_2609_30342_amd import rikfad as R
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    x = torch.randn(nelem, device="cuda:0").to(dt)
    g = torch.randn(nelem, device="cuda:0").to(dt)
    p = torch.randn(nelem, device="cuda:0")
    code = R.RIKFAD_BF16 if dtype == "bf16" else R.RIKFAD_FP32
    s = torch.cuda.current_stream().cuda_stream
    ms = _time_calls(lambda: R.rikfad_probe_mix(x.data_ptr(), g.data_ptr(), p.data_ptr(), nelem,
                                                code, shape, s), reps)
    per = 14.0 if dtype == "bf16" else 20.0
    del x, g, p
    torch.cuda.empty_cache()
    return per * nelem / (ms * 1e-3) / 1e9


def time_probe_write(nbytes, reps=50):
    """Write-only stream of nbytes.  GB/s."""
    import torch
    from paper_2609_30342_amd import rikfad as R
    a = torch.empty(nbytes // 4, device="cuda:0")
    s = torch.cuda.current_stream().cuda_stream
    ms = _time_calls(lambda: R.rikfad_probe_write(a.data_ptr(), nbytes, 0x3f800000, s), reps)
    del a
    torch.cuda.empty_cache()
    return nbytes / (ms * 1e-3) / 1e9


def measure_probes(n):
    """The chip's ceilings for the step's access mixes over n elements:
    the 3-read/2-write stream of five fp32 buffers, the step's own mix
    without arithmetic (fp32 and bf16, contiguous and in the streaming
    kernel's tiles), and read-only and write-only streams of 4 n bytes.
    GB/s on each probe's own bytes."""
    probes = {"stream_3r2w": time_probe(n)}
    probes.update({f"mix_{dt}_{nm}": time_probe_mix(n, dt, sh)
                   for dt in ("fp32", "bf16") for sh, nm in ((0, "contig"), (1, "tiles"))})
    probes["read_only"] = time_probe_read(4 * n)
    probes["write_only"] = time_probe_write(4 * n)
    return probes


def time_probe_read(nbytes, reps=50):
    """Read-only stream of nbytes.  GB/s."""
    import torch
    from paper_2609_30342_amd import rikfad as R
    a = torch.randn(nbytes // 4, device="cuda:0")
    out = torch.zeros(1, device="cuda:0")
    s = torch.cuda.current_stream().cuda_stream
    ms = _time_calls(lambda: R.rikfad_probe_read(a.data_ptr(), nbytes, out.data_ptr(), s), reps)
    del a, out
    torch.cuda.empty_cache()
    return nbytes / (ms * 1e-3) / 1e9


def cpu_baseline(specs, hp, budget_s):
    """The fp64 oracle (as it stands) on a bounded sample of the workload:
    the position embedding, block 0's four matrices and its eight vectors
    (7.9M of the 124.4M parameters), stepped until budget_s seconds pass."""
    import numpy as np

    import oracle as O
    from paper_2609_30342_amd import synth
    names = {"wpe"} | {s.name for s in specs if s.name.startswith("h0.")}
    sample = [s for s in specs if s.name in names]
    wl = synth.Workload(sample, seed=0)
    ts = [O.make_tensor(wl.x0(i)) for i in range(len(sample))]
    grads = [wl.grad(i, 0).astype(np.float64) for i in range(len(sample))]
    threads = len(os.sched_getaffinity(0))
    ohp = O.HParams(**hp)

    def rate(nthreads, seconds):
        n, t0 = 0, time.perf_counter()
        while True:
            O.step_list(ts, grads, ohp, threads=nthreads)
            n += 1
            el = time.perf_counter() - t0
            if el >= seconds:
                return n, el

    elems = sum(s.numel for s in sample)
    n, el = rate(threads, budget_s)
    n1, el1 = rate(1, max(1.0, budget_s / 6))
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")),
                         "")
    except OSError:
        pass
    return {"value": elems * n / el, "unit": "params/s", "cores": threads, "kind": "oracle",
            "single_thread_value": elems * n1 / el1, "cpu_model": model,
            "sample": f"fp64 oracle, {n} steps over wpe + block 0 of the GPT2-S set "
                      f"({elems} params, {len(sample)} tensors), OpenMP over tensors, "
                      f"{el:.1f} s; single thread: {n1} steps in {el1:.1f} s"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10,
                    help="untimed steps after the pre-warm and before the timed ones")
    ap.add_argument("--dtype", choices=["fp32", "bf16"], default="fp32")
    ap.add_argument("--cpu-budget", type=float, default=12.0,
                    help="seconds of oracle time for cpu_baseline (0 = skip)")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the bf16 / two-pass / full-iKFAD / probe side measurements")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="also run the copy probe 3 times over this many MiB (a kernel of "
                         "known traffic for scaling hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: the step runs on one GPU (no multi-GPU path); --gpus {args.gpus} is not "
              "supported", file=sys.stderr)
        return 2

    import torch
    from paper_2609_30342_amd import synth
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 1

    hp = dict(synth.HP_BASE)
    specs = synth.gpt2_small(args.dtype)
    N = sum(s.numel for s in specs)
    main_run = time_rikfad(specs, args.dtype, hp, args.steps, args.warmup)
    info = main_run["info"]
    stream_bytes = info["stream_min_bytes"]
    achieved = stream_bytes / (main_run["stream_ms"] * 1e-3) / 1e9
    step_gbps = info["min_bytes_per_step"] / (main_run["ms_per_step"] * 1e-3) / 1e9
    kernel_sum = main_run["stream_ms"] + main_run["finalize_ms"]
    traffic = measured_traffic(args.dtype)
    out = {
        "metric": METRIC,
        "value": N / (main_run["ms_per_step"] * 1e-3),
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_run["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if args.dtype == "fp32" else "bf16 x/g, f32 p/r/c (f32 math)",
        "data": "synthetic (seeded; GPT2-S shapes, random gradients)",
        "config": {
            "workload": f"GPT2-S-shaped parameter set, {args.dtype} x/g: {N} params "
                        f"({info['matrices']} matrices + {info['vectors']} vectors), "
                        "deferred single-pass step",
            "params": N,
            "hparams": hp,
            "stream_tiles": info["stream_tiles"],
            "finalize_items": info["finalize_items"],
        },
        "prewarm": {"ms": main_run["prewarm_ms"], "steps": main_run["prewarm_steps"]},
        "hbm_gbps_step": step_gbps,
        "hbm_frac_step": step_gbps / PEAK_GBPS,
        "kernel_ms": {"stream": main_run["stream_ms"], "finalize": main_run["finalize_ms"],
                      "sum": kernel_sum},
        "step_vs_kernel_sum": main_run["ms_per_step"] / kernel_sum,
        "roofline": {
            "bound": "hbm",
            "achieved": achieved,
            "peak": PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / PEAK_GBPS,
            "traffic": traffic,
            "kernel": "rikfad_stream_kernel",
            "bytes_per_launch": stream_bytes,
            "launches_timed": main_run["timed_steps"],
            "step_frac": step_gbps / PEAK_GBPS,
            "step_bytes": info["min_bytes_per_step"],
        },
        "state_bytes": {"rikfad": info["state_bytes"], "ikfad": info["ikfad_state_bytes"]},
        "nonfinite": main_run["nonfinite"],
    }
    if not args.no_variants:
        var = {}
        other = "bf16" if args.dtype == "fp32" else "fp32"
        r2 = time_rikfad(synth.gpt2_small(other), other, hp, args.steps, args.warmup)
        var[f"rikfad_{other}"] = {
            "ms_per_step": r2["ms_per_step"], "params_per_s": N / (r2["ms_per_step"] * 1e-3),
            "hbm_frac_step": r2["info"]["min_bytes_per_step"] / (r2["ms_per_step"] * 1e-3)
            / 1e9 / PEAK_GBPS,
            "stream_ms": r2["stream_ms"], "finalize_ms": r2["finalize_ms"],
            "stream_gbps": r2["info"]["stream_min_bytes"] / (r2["stream_ms"] * 1e-3) / 1e9}
        tp = time_rikfad(specs, args.dtype, hp, args.steps, args.warmup, two_pass=True)
        var["rikfad_two_pass"] = {"ms_per_step": tp["ms_per_step"],
                                  "params_per_s": N / (tp["ms_per_step"] * 1e-3)}
        for idt, per in (("fp32", 28.0), ("bf16", 22.0)):
            ik_ms = time_ikfad(synth.gpt2_small(idt), hp, args.steps, args.warmup, dtype=idt)
            var[f"ikfad_full_{idt}"] = {"ms_per_step": ik_ms, "params_per_s": N / (ik_ms * 1e-3),
                                        "hbm_gbps": per * N / (ik_ms * 1e-3) / 1e9,
                                        "state_bytes": info["ikfad_state_bytes"]}
        var["adafm_fp32"] = time_adafm(synth.gpt2_small("fp32"), "fp32", args.steps,
                                       args.warmup, h=1e-3, beta1=0.9)
        var["adafm_bf16"] = time_adafm(synth.gpt2_small("bf16"), "bf16", args.steps,
                                       args.warmup, h=1e-3, beta1=0.9)
        big = synth.distilbert_stress()
        rb = time_rikfad(big, None, hp, 10, 3, scales="student_t")
        nb = sum(sp.numel for sp in big)
        var["distilbert_plus_32_large_bf16"] = {
            "params": nb, "ms_per_step": rb["ms_per_step"],
            "params_per_s": nb / (rb["ms_per_step"] * 1e-3),
            "min_bytes_per_step": rb["info"]["min_bytes_per_step"],
            "hbm_gbps_step": rb["info"]["min_bytes_per_step"] / (rb["ms_per_step"] * 1e-3) / 1e9,
            "stream_ms": rb["stream_ms"],
            "stream_gbps": rb["info"]["stream_min_bytes"] / (rb["stream_ms"] * 1e-3) / 1e9}
        # The chip's ceiling for each access mix, measured in the same run:
        # the plain 3-read/2-write stream, the step's own mix without
        # arithmetic (contiguous and in the streaming kernel's tiles), and
        # read-only (what Adafactor-m's read passes move) and write-only
        # streams of the gradient's fp32 bytes.
        probes = measure_probes(N)
        var["probe_3r2w_gbps"] = probes.pop("stream_3r2w")
        var["stream_kernel_vs_probe"] = achieved / var["probe_3r2w_gbps"]
        var["probes_gbps"] = probes
        ceil = {dt: max(probes[f"mix_{dt}_contig"], probes[f"mix_{dt}_tiles"],
                        *( [var["probe_3r2w_gbps"]] if dt == "fp32" else []))
                for dt in ("fp32", "bf16")}
        runs = {args.dtype: (main_run, info), other: (r2, r2["info"])}
        var["vs_ceiling"] = {
            dt: {"ceiling_gbps": ceil[dt],
                 "ceiling_frac_of_peak": ceil[dt] / PEAK_GBPS,
                 "step_over_ceiling_time": (run["ms_per_step"] * 1e-3)
                 / (inf["min_bytes_per_step"] / (ceil[dt] * 1e9)),
                 "stream_over_ceiling_time": (run["stream_ms"] * 1e-3)
                 / (inf["stream_min_bytes"] / (ceil[dt] * 1e9)),
                 "gate_us": inf["min_bytes_per_step"] / (0.75 * PEAK_GBPS * 1e9) * 1e6,
                 "step_us": run["ms_per_step"] * 1e3,
                 "ceiling_us": inf["min_bytes_per_step"] / (ceil[dt] * 1e9) * 1e6}
            for dt, (run, inf) in runs.items()}
        for nm in ("adafm_fp32", "adafm_bf16"):
            var[nm]["read_passes_vs_read_probe"] = {
                "stats": var[nm]["stats_gbps"] / probes["read_only"],
                "rms": var[nm]["rms_gbps"] / probes["read_only"]}
        var["friction_report_wte"] = time_friction_report(50257, 768)
        var["launch_bound_sets"] = {
            "single_256x512_fp32": time_small(synth.single_matrix(), hp, 200, 5),
            "gpt2_nano_fp32": time_small(synth.gpt2_nano(), hp, 100, 5),
            "tinyvit_bf16": time_small(synth.tinyvit_like(), hp, 100, 5),
        }
        out["variants"] = var
    if args.calibrate_copy_mib > 0:
        nbytes = args.calibrate_copy_mib << 20
        src = torch.ones(nbytes // 4, device="cuda:0")
        dst = torch.empty_like(src)
        from paper_2609_30342_amd import rikfad as R
        for _ in range(3):
            R.rikfad_probe_copy(src.data_ptr(), dst.data_ptr(), nbytes,
                                torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        out["calibration_copy_bytes"] = nbytes
        del src, dst
    if args.cpu_budget > 0:
        out["cpu_baseline"] = cpu_baseline(specs, hp, args.cpu_budget)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
