"""Benchmark of the cached Picard sampler on one MI355X.

    python bench.py [--steps K] [--warmup W] [--gpus 1]

Workload: the SD-latent patch-MLP case (latent 4x64x64, T = 100 DDIM steps, window 32,
hidden 1024 over 1024 tokens, tau = 1e-3), synthetic seeded inputs already resident in HBM.
One step = one complete sample (every sweep until the window reaches T) through the C ABI.
value = sweeps/s at delta = 0.05; eps evals/s and NFE saved against delta = 0 are reported
beside it, as are the other cache tolerances of the sweep {0, 0.02, 0.05, 0.1}.

Beside the headline line (same JSON object, extra keys):
  revisit_statistic  the delta = 0 run's fraction of requested drift evaluations that
                     revisit a timestep whose input moved by less than 0.05 (Sec. 1);
  batched            8 samples per handle at the same workload (one network launch per
                     sweep serves every sample's misses): samples/s, eps evals/s;
  ddpm_window64      ancestral DDPM (eta = 1, pre-drawn step noise) over T = 1000 with a
                     window of 64 on the same latent and network, delta in {0, 0.05}.
  long_window128     the deterministic sampler over T = 1000 (the full schedule) with a window
                     of 128 on the same latent and network, delta in {0, 0.05}: long-window
                     prefix sums and 128-wide miss compaction; with the Picard kernel's rate.
  parareal           the Parareal-style cached sampler: 4x96x96 latent, T = 100 in 10 blocks,
                     patch-MLP H = 2048 over 2304 tokens, delta in {0, 0.05}.
  picard_beyond_cache  the solver kernels at 64 samples per handle of the same workload: one
                     Picard launch then touches ~0.5 GB, more than the 256 MB Infinity Cache,
                     so its rate is that of HBM (the one- and eight-sample figures are not).
  shard_share        one GPU's share of a sweep's misses if they were split over G GPUs: the
                     network launch with 32 / G misses at the same shape (window 32 / G at
                     delta = 0, so every launch evaluates that many latents), G in {1, 2, 4, 8}.

Prints one JSON line (rank 0). Throughput figures (value, ms_per_step, ε evals/s, and those of
the extra measurements) come from samples launched exactly as a user launches them, with no
timing events. Kernel durations come from a second pass over the same samples on a handle
whose network launches carry start/stop HIP events attached to their dispatches on the
sampler's stream (the events add stream time, so that pass is not the throughput). An event
pair can include idle time before its kernel on the stream: without a profiler attached the
event-timed network duration is within about 1% of rocprofv3's kernel duration, while a
profiler spaces the kernels further apart and the event figure of a profiled run grows with
it. The roofline object describes the
dominant kernel (the fused patch-MLP network kernel): achieved = algorithmic FLOPs of its
launches / their summed event-timed duration.
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

METRIC = "cached Picard sweeps/s + ε evals/s at 4×64×64, T=100; NFE saved vs δ=0"
PEAK_BF16_TFLOPS = 2500.0          # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0              # MI355X HBM3E
PRIMARY_DELTA = 0.05


TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "k_eps_mlp_traffic_sd_4x64x64_T100_P32_H1024.md")
PICARD64_RECORD = os.path.join(ROOT, "profiles", "k_picard_batched64_sd_4x64x64_T100_P32_H1024.md")
MFMA_RECORD = os.path.join(ROOT, "profiles", "k_eps_mlp_mfma_sd_4x64x64_T100_P32_H1024.md")


def counter_record(record):
    """The machine-readable record of a committed counter summary, or None when the kernel
    sources changed since the counters were taken."""
    import hashlib
    import re
    try:
        text = open(record).read()
        rec = json.loads(re.search(r"```json\n(.*?)```", text, re.S).group(1))
        h = hashlib.sha256()
        for src in rec["sources"]:
            h.update(open(os.path.join(ROOT, src), "rb").read())
        return rec if h.hexdigest() == rec["source_sha256"] else None
    except (OSError, AttributeError, KeyError, ValueError):
        return None


def measured_traffic(record=TRAFFIC_RECORD):
    """HBM bytes per launch of a kernel from a committed counter summary, or None."""
    rec = counter_record(record)
    return rec["traffic_bytes_per_launch"] if rec else None


def mfma_counters():
    """MFMA utilisation counters of the network kernel from the committed summary, or None."""
    rec = counter_record(MFMA_RECORD)
    if rec is None:
        return None
    return {k: rec[k] for k in ("mfma_busy_frac", "mfma_flop_executed_per_launch",
                                "algorithmic_flop_per_launch", "valu_active_frac",
                                "mfma_cycles_with_valu_coissue_frac", "clock_GHz")}


def flops_per_eval(wl) -> float:
    """Algorithmic FLOPs of one patch-MLP evaluation: 2 * tokens * (16 H + H^2 + 16 H)."""
    H = wl.hidden
    return 2.0 * wl.tokens * (16 * H + H * H + 16 * H)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=600)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--deltas", type=str, default="0,0.02,0.05,0.1")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--headline-only", action="store_true",
                    help="skip the revisit, batched, DDPM and Parareal measurements")
    ap.add_argument("--extras", type=str, default="revisit,batched,ddpm,long,parareal,hbm,shard",
                    help="which extra measurements to run (comma list)")
    ap.add_argument("--cpu-seconds", type=float, default=6.0,
                    help="budget of each of the oracle's two bounded samples (all threads, one)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run a plain device copy of this size (counter calibration)")
    return ap.parse_args()


def timed_samples(sampler, x, steps, warmup, torch, profiled):
    out = torch.empty_like(x)
    for _ in range(warmup):                         # untimed warm-up generations
        sampler.sample(x, out)
    torch.cuda.synchronize()
    if profiled:
        sampler.kernel_times()                      # restart the kernel timers
    sweeps = nfe = hits = revisits = below = 0
    per_sample = []
    t0 = time.perf_counter()
    for _ in range(steps):
        ts = time.perf_counter()
        sampler.sample(x, out)                      # returns once every sample is done
        per_sample.append(time.perf_counter() - ts)
        st = sampler.stats()                        # final counters, taken from the done words
        sweeps += st["sweeps"]
        nfe += st["nfe"]
        hits += st["hits"]
        revisits += st["revisits"]
        below += st["revisits_below"]
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    per_sample.sort()
    r = {"seconds": dt, "sweeps": sweeps, "nfe": nfe, "hits": hits, "revisits": revisits,
         "revisits_below": below, "out": out,
         "median_sample_s": per_sample[len(per_sample) // 2] if len(per_sample) % 2 else
         0.5 * (per_sample[len(per_sample) // 2 - 1] + per_sample[len(per_sample) // 2])}
    if profiled:
        kt = sampler.kernel_times()                 # every launch of the timed samples
        r.update({"eps_ms": kt["eps_ms_total"], "launches": kt["launches"],
                  "picard_ms": kt["picard_ms_total"], "slide_ms": kt["slide_ms_total"],
                  "solver_launches": kt["solver_launches"], "profiled_seconds": dt,
                  "profiled_nfe": nfe, "profiled_sweeps": sweeps, "profiled_hits": hits})
    return r


def parareal_case(wl, delta, steps, warmup, torch, weights):
    """Timed Parareal samples: plain launches for the throughput, then the same samples on a
    handle with events on the network launches for the kernel durations."""
    from paper_2609_36522_amd import binding, inputs
    x = torch.from_numpy(inputs.x_init(wl.latent).reshape(-1)).cuda()
    out = torch.empty_like(x)
    res = {}
    for profiled in (False, True):
        with binding.parareal_from_workload(wl, delta, seed_weights=weights, profile=profiled) as s:
            for _ in range(warmup):
                s.sample(x, out)
            torch.cuda.synchronize()
            if profiled:
                s.kernel_times()                    # restart the kernel timers
            nfe = hits = iters = 0
            t0 = time.perf_counter()
            for _ in range(steps):
                s.sample(x, out)
                st = s.stats()
                nfe += st["nfe"]
                hits += st["hits"]
                iters += st["iterations"]
            torch.cuda.synchronize()
            dt = time.perf_counter() - t0
            if profiled:
                kt = s.kernel_times()
                res.update({"eps_ms": kt["eps_ms_total"], "launches": kt["launches"],
                            "profiled_nfe": nfe})
            else:
                res.update({"seconds": dt, "nfe": nfe, "hits": hits, "iters": iters})
    return res


def solver_kernels(r, D):
    """HBM view of the two solver kernels from their event times (a separate run whose
    handle times them: their events add stream time, so it is not the headline run).

    k_picard's algorithmic bytes per sweep are the Picard update's (3W + 1) * 4D (read the
    W + 1 window states and the W assembled outputs, write W states) plus 4D per miss (the
    Eq. (7) cache write of its input). Not counted: the Eq. (7) write of the fresh output (the
    network kernel's whole outputs land in the cache directly; only launches with split
    outputs leave it to k_picard), and the cache inputs of hit slots it reads for the next
    sweep's Eq. (4) test. Summed over a run: 4D * (3 * (nfe + hits) + sweeps + nfe). k_slide
    moves only the fp64 partial sums and the control block: it is bound by latency."""
    byts = 4.0 * D * (3 * (r["profiled_nfe"] + r["profiled_hits"]) + r["profiled_sweeps"]
                      + r["profiled_nfe"])
    n = max(r["solver_launches"], 1)
    gbs = byts / (r["picard_ms"] * 1e-3) / 1e9 if r["picard_ms"] > 0 else None
    return {"k_picard": {"bound": "hbm", "achieved": gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": (gbs / PEAK_HBM_GBS) if gbs else None,
                         "bytes_per_launch": byts / n, "avg_launch_us": 1e3 * r["picard_ms"] / n},
            "k_slide": ({"bound": "latency", "avg_launch_us": 1e3 * r["slide_ms"] / n}
                        if r["slide_ms"] > 0 else
                        {"fused": "computed at the start of the next network kernel (one "
                                  "patch-MLP sample): no launch of its own"})}


def sweep_breakdown(p, rs, steps):
    """Where a sweep's stream time goes at the headline workload, in microseconds per sweep:
    total = wall time of a sample (plain launches) / its sweeps; network = event-timed
    duration of the network launches of a sample / sweeps; picard = event-timed duration of
    the Picard launches (a run whose handle also times them) / sweeps; rest = total - network
    - picard: launch gaps, the window slide's own launch when it has one, and the host's
    enqueue and final copy."""
    sweeps = p["sweeps"] / steps
    total = 1e6 * p["seconds"] / steps / sweeps
    net = 1e3 * p["eps_ms"] / steps / sweeps
    pic = 1e3 * rs["picard_ms"] / rs["profiled_sweeps"] if rs["profiled_sweeps"] else 0.0
    sld = 1e3 * rs["slide_ms"] / rs["profiled_sweeps"] if rs["profiled_sweeps"] else 0.0
    return {"total": total, "network": net, "picard": pic, "slide": sld,
            "rest": total - net - pic - sld, "sweeps_per_sample": sweeps}


def run_case(wl, delta, steps, warmup, torch, weights, *, batch=1, eta=0.0, solver=False):
    """Timed samples of one configuration. The throughput comes from a handle with plain
    launches; the kernel durations from a second pass over the same samples on a handle whose
    network launches (with ``solver`` also the Picard and slide launches) carry start/stop
    events (the events add stream time, ~4 us per sweep, so they stay out of the throughput)."""
    from paper_2609_36522_amd import binding, inputs
    if batch == 1:
        xs = inputs.x_init(wl.latent).reshape(-1)
    else:
        xs = inputs.x_init_batch(wl.latent, batch).reshape(-1)
    x = torch.from_numpy(xs).cuda()
    noise = (torch.from_numpy(inputs.step_noise(batch, wl.T, wl.D).reshape(-1)).cuda()
             if eta > 0 else None)
    res = None
    for profiled in (False, True):
        with binding.from_workload(wl, delta, seed_weights=weights, profile=profiled, batch=batch,
                                   eta=eta, profile_solver=profiled and solver) as s:
            if noise is not None:
                s.set_noise(noise)
            r = timed_samples(s, x, steps, warmup, torch, profiled)
        if res is None:
            res = r
        else:
            res.update({k: v for k, v in r.items() if k.startswith("profiled_") or k in (
                "eps_ms", "launches", "picard_ms", "slide_ms", "solver_launches")})
    return res


def measured_ceilings(torch, gemm_m):
    """Ceilings measured on this GPU beside the vendor peaks: HBM streams of 1 GiB arrays
    through torch (a copy, a fill that only writes, and z = x + y, two reads per write), and
    hipBLASLt bf16 GEMMs run as a library through torch.matmul, at the network's GEMM2 shape
    for one sweep's misses ([gemm_m x 1024] x [1024 x 1024]) and at 8192^3."""
    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        b.synchronize()
        return a.elapsed_time(b) / reps * 1e-3
    n = (1 << 30) // 4
    src = torch.ones(n, device="cuda")
    dst = torch.empty_like(src)
    t = timed(lambda: dst.copy_(src), 10)
    copy_gbs = 2 * n * 4 / t / 1e9
    t = timed(lambda: dst.fill_(2.0), 10)
    fill_gbs = n * 4 / t / 1e9
    third = torch.empty_like(src)
    t = timed(lambda: torch.add(src, dst, out=third), 10)
    add_gbs = 3 * n * 4 / t / 1e9
    del src, dst, third
    out = {"copy_1GiB_GBps": copy_gbs, "fill_1GiB_GBps": fill_gbs, "add_1GiB_GBps": add_gbs}
    for name, (m, k, nn) in {"gemm2_shape": (gemm_m, 1024, 1024), "square_8192": (8192, 8192, 8192)}.items():
        A = torch.randn(m, k, device="cuda", dtype=torch.bfloat16)
        Bm = torch.randn(k, nn, device="cuda", dtype=torch.bfloat16)
        t = timed(lambda: torch.matmul(A, Bm), 20)
        out[f"bf16_{name}_TFLOPs"] = 2.0 * m * k * nn / t / 1e12
        out[f"bf16_{name}"] = [m, k, nn]
        del A, Bm
    torch.cuda.empty_cache()
    return out


def cpu_baseline(wl, delta, budget_s):
    """The oracle (as it stands) on a bounded prefix of the same sample."""
    import numpy as np
    from oracle import eps_models as em
    from oracle import sampler as sp
    from oracle import schedule as sch
    from paper_2609_36522_amd import inputs
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    ab, t = sch.sampler_alpha_bar(wl.T)
    alpha, b = sch.ddim_coefficients(ab)
    net = em.PatchMLP(inputs.mlp_weights(wl.hidden, temb_dim=wl.temb_dim), t, wl.latent)
    st = sp.init_state(inputs.x_init(wl.latent), wl.T)
    t0 = time.perf_counter()
    while not st.done and time.perf_counter() - t0 < budget_s:
        sp.sweep(st, wl.window, delta, wl.tol, alpha, b, net)
    dt = time.perf_counter() - t0
    return {"value": st.sweeps / dt, "unit": "sweeps/s", "cores": int(threads), "kind": "oracle",
            "sample": f"first {st.sweeps} sweeps (NFE {st.nfe}, {dt:.1f} s) of the delta={delta} "
                      f"sample, float64 NumPy oracle",
            "eps_evals_per_s": st.nfe / dt, "cpu_model": cpu_model(),
            "os_cpu_count": os.cpu_count()}


def cpu_model() -> str:
    """The host CPU's model name (/proc/cpuinfo), or "unknown"."""
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus}); the sampler has no "
              f"multi-GPU path.", file=sys.stderr, flush=True)
        sys.exit(2)
    import torch
    from paper_2609_36522_amd import binding, inputs, workloads

    binding.load_library()
    torch.cuda.set_device(0)
    wl = workloads.SD_MLP
    deltas = [float(v) for v in args.deltas.split(",")]
    if PRIMARY_DELTA not in deltas:
        deltas.append(PRIMARY_DELTA)
    weights = inputs.mlp_weights(wl.hidden, temb_dim=wl.temb_dim)
    fpe = flops_per_eval(wl)

    per_delta = {}
    for d in deltas:
        r = run_case(wl, d, args.steps, args.warmup, torch, weights)
        per_delta[d] = r
        print(f"[bench] delta={d}: {r['sweeps'] / args.steps:.1f} sweeps/sample, "
              f"NFE {r['nfe'] / args.steps:.1f}, {1e3 * r['seconds'] / args.steps:.3f} ms/sample",
              file=sys.stderr, flush=True)

    extras = {}
    if not args.headline_only:
        want = set(args.extras.split(","))
        # revisit statistic of the delta = 0 run (the cache's motivation figure, Sec. 1)
        if "revisit" in want and 0.0 in per_delta:
            r0 = per_delta[0.0]
            req = r0["nfe"] + r0["hits"]
            extras["revisit_statistic"] = {
                "threshold": 0.05, "delta": 0.0,
                "fraction_of_requests": r0["revisits_below"] / req,
                "revisit_fraction": r0["revisits"] / req,
                "requests_per_sample": req / args.steps}
    if not args.headline_only and "batched" in want:
        # several samples per handle
        nb = 8
        bsteps = max(args.steps // 3, 3)
        rb = run_case(wl, PRIMARY_DELTA, bsteps, 1, torch, weights, batch=nb)
        extras["batched"] = {
            "samples": nb, "delta": PRIMARY_DELTA, "steps": bsteps,
            "ms_per_batch": 1e3 * rb["seconds"] / bsteps,
            "samples_per_s": nb * bsteps / rb["seconds"],
            "eps_evals_per_s": rb["nfe"] / rb["seconds"],
            "batched_sweeps_per_batch": rb["sweeps"] / bsteps,
            "nfe_per_sample": rb["nfe"] / (nb * bsteps),
            "eps_kernel_tflops": (rb["profiled_nfe"] * fpe) / (rb["eps_ms"] * 1e-3) / 1e12 if rb["eps_ms"] > 0 else None,
            "solver_kernels": solver_kernels(
                run_case(wl, PRIMARY_DELTA, 3, 1, torch, weights, batch=nb, solver=True), wl.D)}
        print(f"[bench] batch {nb}: {extras['batched']['ms_per_batch']:.3f} ms/batch, "
              f"{extras['batched']['samples_per_s']:.0f} samples/s", file=sys.stderr, flush=True)
    if not args.headline_only and "hbm" in want:
        # Picard launches whose touched set exceeds the Infinity Cache
        nh = 64
        rh = run_case(wl, PRIMARY_DELTA, 2, 1, torch, weights, batch=nh, solver=True)
        sk = solver_kernels(rh, wl.D)
        traffic = measured_traffic(PICARD64_RECORD)
        sk["k_picard"]["traffic"] = traffic
        sk["k_picard"]["traffic_unit"] = "bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)"
        if traffic is not None:
            sk["k_picard"]["traffic_GBps"] = traffic / (sk["k_picard"]["avg_launch_us"] * 1e-6) / 1e9
        extras["picard_beyond_cache"] = {
            "samples": nh, "delta": PRIMARY_DELTA, "steps": 2, "solver_kernels": sk}
        print(f"[bench] picard at batch {nh}: {sk['k_picard']['bytes_per_launch'] / 1e6:.0f} MB/launch, "
              f"{sk['k_picard']['achieved']:.0f} GB/s", file=sys.stderr, flush=True)
    if not args.headline_only and "shard" in want:
        # the network kernel on one GPU's share of the misses (m / G latents per launch)
        fpe = flops_per_eval(wl)
        share = {}
        for G in (1, 2, 4, 8):
            ws = wl.with_(window=wl.window // G)
            r = run_case(ws, 0.0, max(args.steps // 40, 3), 1, torch, weights)
            per = r["eps_ms"] * 1e3 / max(r["launches"], 1)
            m = r["profiled_nfe"] / max(r["launches"], 1)
            share[str(G)] = {"misses_per_launch": m, "avg_launch_us": per,
                             "tflops": m * fpe / (per * 1e-6) / 1e12 if per > 0 else None}
            print(f"[bench] shard share G={G}: {m:.1f} misses/launch, {per:.1f} us/launch",
                  file=sys.stderr, flush=True)
        extras["shard_share"] = {"workload": wl.name, "delta": 0.0, "per_G": share}
    if not args.headline_only and "ddpm" in want:
        # the window study's stochastic setting
        wd = wl.with_(T=1000, window=64)
        dsteps = max(args.steps // 6, 3)
        dd = {}
        for d in (0.0, PRIMARY_DELTA):
            r = run_case(wd, d, dsteps, 1, torch, weights, eta=1.0)
            dd[d] = r
            print(f"[bench] ddpm T=1000 P=64 delta={d}: {1e3 * r['seconds'] / dsteps:.3f} ms/sample, "
                  f"NFE {r['nfe'] / dsteps:.0f}", file=sys.stderr, flush=True)
        extras["ddpm_window64"] = {
            "T": 1000, "window": 64, "eta": 1.0, "steps": dsteps,
            "per_delta": {str(d): {"ms_per_sample": 1e3 * r["seconds"] / dsteps,
                                   "sweeps_per_s": r["sweeps"] / r["seconds"],
                                   "eps_evals_per_s": r["nfe"] / r["seconds"],
                                   "nfe_per_sample": r["nfe"] / dsteps,
                                   "sweeps_per_sample": r["sweeps"] / dsteps}
                          for d, r in dd.items()},
            "nfe_saved_vs_delta0": 1.0 - dd[PRIMARY_DELTA]["nfe"] / dd[0.0]["nfe"]}
    if not args.headline_only and "long" in want:
        # the long-window deterministic setting: T = 1000, window 128
        wlg = workloads.LONG_MLP
        lsteps = max(args.steps // 6, 3)
        ll = {}
        for d in (0.0, PRIMARY_DELTA):
            r = run_case(wlg, d, lsteps, 1, torch, weights, solver=(d == PRIMARY_DELTA))
            ll[d] = r
            print(f"[bench] long T=1000 P=128 delta={d}: {1e3 * r['seconds'] / lsteps:.3f} ms/sample, "
                  f"NFE {r['nfe'] / lsteps:.0f}, {r['sweeps'] / lsteps:.0f} sweeps", file=sys.stderr, flush=True)
        extras["long_window128"] = {
            "workload": wlg.name, "T": wlg.T, "window": wlg.window, "steps": lsteps,
            "per_delta": {str(d): {"ms_per_sample": 1e3 * r["seconds"] / lsteps,
                                   "sweeps_per_s": r["sweeps"] / r["seconds"],
                                   "eps_evals_per_s": r["nfe"] / r["seconds"],
                                   "nfe_per_sample": r["nfe"] / lsteps,
                                   "hits_per_sample": r["hits"] / lsteps,
                                   "sweeps_per_sample": r["sweeps"] / lsteps,
                                   "eps_kernel_tflops": (r["profiled_nfe"] * fpe) / (r["eps_ms"] * 1e-3) / 1e12
                                   if r["eps_ms"] > 0 else None}
                          for d, r in ll.items()},
            "nfe_saved_vs_delta0": 1.0 - ll[PRIMARY_DELTA]["nfe"] / ll[0.0]["nfe"],
            "solver_kernels": solver_kernels(ll[PRIMARY_DELTA], wlg.D)}
    if not args.headline_only and "parareal" in want:
        # the Parareal-style cached sampler
        wp = workloads.PARAREAL_MLP
        wts = inputs.mlp_weights(wp.hidden, temb_dim=wp.temb_dim)
        fpp = flops_per_eval(wp)
        psteps = max(args.steps // 10, 3)
        pp = {}
        for d in (0.0, PRIMARY_DELTA):
            r = parareal_case(wp, d, psteps, 1, torch, wts)
            pp[d] = r
            print(f"[bench] parareal delta={d}: {1e3 * r['seconds'] / psteps:.3f} ms/sample, "
                  f"NFE {r['nfe'] / psteps:.0f}, {r['iters'] / psteps:.1f} iterations",
                  file=sys.stderr, flush=True)
        extras["parareal"] = {
            "workload": wp.name, "latent": list(wp.latent), "T": wp.T, "blocks": wp.blocks,
            "hidden": wp.hidden, "tokens": wp.tokens, "gflop_per_eval": fpp / 1e9, "steps": psteps,
            "per_delta": {str(d): {"ms_per_sample": 1e3 * r["seconds"] / psteps,
                                   "eps_evals_per_s": r["nfe"] / r["seconds"],
                                   "nfe_per_sample": r["nfe"] / psteps,
                                   "hits_per_sample": r["hits"] / psteps,
                                   "iterations_per_sample": r["iters"] / psteps,
                                   "eps_kernel_tflops": (r["profiled_nfe"] * fpp) / (r["eps_ms"] * 1e-3) / 1e12
                                   if r["eps_ms"] > 0 else None}
                          for d, r in pp.items()},
            "nfe_saved_vs_delta0": 1.0 - pp[PRIMARY_DELTA]["nfe"] / pp[0.0]["nfe"]}

    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib * (1 << 20) // 4
        a = torch.ones(n, device="cuda")
        bb = torch.empty_like(a)
        for _ in range(3):
            bb.copy_(a)
        torch.cuda.synchronize()

    p = per_delta[PRIMARY_DELTA]
    d0 = per_delta.get(0.0)
    rs = run_case(wl, PRIMARY_DELTA, 10, 1, torch, weights, solver=True)
    sweeps_per_s = p["sweeps"] / p["seconds"]
    eps_per_s = p["nfe"] / p["seconds"]
    achieved = (p["profiled_nfe"] * fpe) / (p["eps_ms"] * 1e-3) / 1e12 if p["eps_ms"] > 0 else 0.0
    line = {
        "metric": METRIC,
        "value": sweeps_per_s,
        "unit": "sweeps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * p["seconds"] / args.steps,
        "ms_per_sample_mean": 1e3 * p["seconds"] / args.steps,
        "ms_per_sample_median": 1e3 * p["median_sample_s"],
        "sweeps_per_s_median": (p["sweeps"] / args.steps) / p["median_sample_s"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "latent": list(wl.latent), "T": wl.T,
                   "window": wl.window, "delta": PRIMARY_DELTA, "tau": wl.tol,
                   "eps_net": f"patch-MLP 16-{wl.hidden}-{wl.hidden}-16 bf16 MFMA, fp32 state",
                   "tokens": wl.tokens, "step": "one full sample (all sweeps until done)",
                   "parallelism": "single GPU"},
        "eps_evals_per_s": eps_per_s,
        "nfe_per_sample": p["nfe"] / args.steps,
        "hits_per_sample": p["hits"] / args.steps,
        "sweeps_per_sample": p["sweeps"] / args.steps,
        "nfe_saved_vs_delta0": (1.0 - p["nfe"] / d0["nfe"]) if d0 else None,
        "per_delta": {str(d): {"sweeps_per_s": r["sweeps"] / r["seconds"],
                               "eps_evals_per_s": r["nfe"] / r["seconds"],
                               "ms_per_sample": 1e3 * r["seconds"] / args.steps,
                               "ms_per_sample_median": 1e3 * r["median_sample_s"],
                               "nfe_per_sample": r["nfe"] / args.steps,
                               "hits_per_sample": r["hits"] / args.steps,
                               "sweeps_per_sample": r["sweeps"] / args.steps,
                               "nfe_saved_vs_delta0": (1.0 - r["nfe"] / d0["nfe"]) if d0 else None,
                               "eps_kernel_tflops": ((r["profiled_nfe"] * fpe) / (r["eps_ms"] * 1e-3) / 1e12
                                                     if r["eps_ms"] > 0 else None)}
                      for d, r in per_delta.items()},
        "solver_kernels": solver_kernels(rs, wl.D),
        "sweep_breakdown_us": sweep_breakdown(p, rs, args.steps),
        "roofline": {"bound": "mfma", "kernel": "k_eps_mlp<1024, 128>",
                     "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS, "traffic": measured_traffic(),
                     "traffic_unit": "bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                     "counters": mfma_counters(),
                     "avg_launch_us": 1e3 * p["eps_ms"] / max(p["launches"], 1),
                     "flops_per_launch": p["profiled_nfe"] * fpe / max(p["launches"], 1),
                     "timing": "kernel durations from a second pass of the timed samples with "
                               "start/stop events attached to every network launch"},
    }
    line.update(extras)
    # The second kernel of every sweep beside the dominant one: the Picard kernel's fraction of
    # the HBM peak at the headline workload (its launches run from the Infinity Cache and are
    # latency-bound) and, when measured, with 64 samples per handle (streaming from HBM).
    pk1 = line["solver_kernels"]["k_picard"]
    pk64 = line.get("picard_beyond_cache", {}).get("solver_kernels", {}).get("k_picard", {})
    line["roofline"]["second_kernel"] = {
        "kernel": "k_picard", "bound": "hbm", "peak": PEAK_HBM_GBS, "unit": "GB/s",
        "achieved": pk1.get("achieved"), "frac": pk1.get("frac"),
        "achieved_beyond_cache": pk64.get("achieved"), "frac_beyond_cache": pk64.get("frac")}
    if not args.headline_only:
        ceil = measured_ceilings(torch, int(round(p["nfe"] / p["sweeps"])) * wl.tokens)
        line["measured_ceilings"] = ceil
        line["roofline"]["frac_vs_measured_square_gemm"] = achieved / ceil["bf16_square_8192_TFLOPs"]
        line["roofline"]["frac_vs_measured_gemm2_shape"] = achieved / ceil["bf16_gemm2_shape_TFLOPs"]
        pks = [line["solver_kernels"]["k_picard"]]
        if "picard_beyond_cache" in line:
            pks.append(line["picard_beyond_cache"]["solver_kernels"]["k_picard"])
        for pk in pks:
            if pk["achieved"]:
                pk["frac_vs_measured_copy"] = pk["achieved"] / ceil["copy_1GiB_GBps"]
                pk["frac_vs_measured_add"] = pk["achieved"] / ceil["add_1GiB_GBps"]
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, PRIMARY_DELTA, args.cpu_seconds)
        if not args.headline_only:
            try:
                from threadpoolctl import threadpool_limits
                with threadpool_limits(limits=1):
                    one = cpu_baseline(wl, PRIMARY_DELTA, args.cpu_seconds)
                line["cpu_baseline_1thread"] = dict(one, cores=1)
            except ImportError:
                pass
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
