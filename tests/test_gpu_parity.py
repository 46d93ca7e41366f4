"""Device parity against the oracle through the C ABI (MI355X only).

Every case runs the device sampler sweep by sweep; the oracle repeats each sweep on the
device's own pre-sweep state (step-locked) and then follows its own trajectory from the
same initial latent. Decisions must agree except inside the 1e-6 relative band around
delta/tau; final latents agree within 1e-4 x RMS. Fresh patch-MLP outputs are compared one
by one with the oracle network (every output of a run, or every output of its first sweep
and a fixed stride after that for the largest runs), within 1e-2 x the larger of the
output's RMS and the token's own output scale (parity_harness.eps_error).
"""
import math
import sys

import numpy as np
import pytest

from paper_2609_36522_amd import workloads as W
from paper_2609_36522_amd.workloads import Workload

import parity_harness as H

pytestmark = pytest.mark.gpu

INF = math.inf

LIN = W.TINY_LINEAR
CASES = [
    # tiny closed-form workload and its degenerate settings
    ("tiny", LIN, 0.05),
    ("tiny_delta0", LIN, 0.0),
    ("tiny_delta_inf", LIN, INF),
    ("tiny_window1", LIN.with_(window=1), 0.05),
    ("tiny_windowT", LIN.with_(window=10), 0.05),
    ("T1", LIN.with_(T=1, window=1), 0.05),
    ("tau0", LIN.with_(tol=0.0), 0.05),
    # ragged sizes: partial cache-test chunks and Picard column blocks
    ("ragged_4x10x10", Workload("lin_4x10x10", (4, 10, 10), 30, 7, 0.05, 1e-3, "linear"), 0.05),
    ("ragged_3x5x4", Workload("lin_3x5x4", (3, 5, 4), 12, 5, 0.1, 1e-3, "linear"), 0.1),
    ("D4", Workload("lin_1x2x2", (1, 2, 2), 8, 3, 0.05, 1e-3, "linear"), 0.05),
    ("big_D_linear", Workload("lin_4x64x64", (4, 64, 64), 100, 32, 0.05, 1e-3, "linear"), 0.05),
    # maximum window
    ("max_window", Workload("lin_4x8x8_P256", (4, 8, 8), 256, 256, 0.05, 1e-3, "linear"), 0.05),
    ("long_window_128", Workload("lin_4x16x16_P128", (4, 16, 16), 300, 128, 0.05, 1e-3, "linear"), 0.05),
    # patch-MLP; every fresh network output is checked against the oracle network unless the
    # case names a stride (then every output of the first sweep and every stride-th after)
    ("mlp_16x32_H512", Workload("mlp_4x16x32_H512", (4, 16, 32), 20, 8, 0.05, 1e-3, "patch_mlp",
                                hidden=512), 0.05),
    # W/2 = 48 patch columns: 128-token blocks start and end inside patch rows
    ("mlp_32x96_H1024", Workload("mlp_4x32x96_T10_P5_H1024", (4, 32, 96), 10, 5, 0.05, 1e-3,
                                 "patch_mlp", hidden=1024), 0.05),
    ("mlp_96x96_H512", Workload("mlp_4x96x96_T8_P4_H512", (4, 96, 96), 8, 4, 0.05, 1e-3,
                                "patch_mlp", hidden=512), 0.05),
    ("mlp_small", W.SMALL_MLP, 0.05, dict(independent=True)),
    ("mlp_small_delta0", W.SMALL_MLP, 0.0, dict(independent=True)),
    ("mlp_sd", W.SD_MLP, 0.05, dict(independent=True)),
    ("mlp_sd_delta0", W.SD_MLP, 0.0, dict(independent=True)),
    # the rest of the headline delta sweep
    ("mlp_sd_delta002", W.SD_MLP, 0.02, dict(eps_stride=4)),
    ("mlp_sd_delta01", W.SD_MLP, 0.1, dict(eps_stride=4)),
    # several samples per handle: every sample step-locked and followed on its own
    ("batch5_tiny", LIN, 0.05, dict(batch=5)),
    ("batch3_ragged", Workload("lin_3x5x4", (3, 5, 4), 12, 5, 0.1, 1e-3, "linear"), 0.1, dict(batch=3)),
    ("batch3_mlp_small", W.SMALL_MLP, 0.05, dict(batch=3)),
    ("batch4_mlp_sd", W.SD_MLP, 0.05, dict(batch=4, eps_stride=4)),
    # stochastic step (ancestral DDPM) with pre-drawn step noise
    ("ddpm_tiny", LIN, 0.05, dict(eta=1.0)),
    ("ddpm_tiny_delta0", LIN, 0.0, dict(eta=1.0)),
    ("ddpm_window1", LIN.with_(window=1), 0.05, dict(eta=1.0)),
    ("ddpm_batch3_tiny", LIN, 0.05, dict(eta=1.0, batch=3)),
    ("ddpm_mlp_small", W.SMALL_MLP, 0.05, dict(eta=1.0)),
    ("ddpm_eta_half", W.SMALL_MLP, 0.05, dict(eta=0.5)),
    # widest network (four partial outputs per fresh output) in the Picard sampler
    ("mlp_H2048", Workload("mlp_4x32x32_T20_P8_H2048", (4, 32, 32), 20, 8, 0.05, 1e-3, "patch_mlp",
                           hidden=2048), 0.05, dict(eps_stride=2)),
    # largest batch: the network kernel's prefix over 64 samples
    ("batch64_mlp", Workload("mlp_4x16x32_T12_P6_H512", (4, 16, 32), 12, 6, 0.05, 1e-3, "patch_mlp",
                             hidden=512), 0.05, dict(batch=64)),
]
CASES = [c if len(c) == 4 else (*c, {}) for c in CASES]


@pytest.mark.parametrize("name,wl,delta,kw", CASES, ids=[c[0] for c in CASES])
def test_parity(name, wl, delta, kw, gpu_lib):
    print(f"[parity] {name}: {wl.name} delta={delta} {kw}", flush=True)
    kw = dict(kw)
    independent = kw.pop("independent", False)
    run = H.Run(wl, delta, **kw).run()
    try:
        for n in range(run.N):
            st = run.stats_n[n]
            recs = run.records[n]
            assert st["done"] and st["sweeps"] == len(recs) <= wl.T
            assert st["nfe"] >= wl.T and st["nfe"] == sum(r["m"] for r in recs)
            assert st["hits"] == sum(r["e"] - r["s"] - r["m"] for r in recs)
            if delta == 0.0:
                assert st["hits"] == 0
            if delta == INF:
                assert st["nfe"] == wl.T
            if wl.window == 1:
                assert st["sweeps"] == wl.T and st["nfe"] == wl.T
            assert recs[0]["m"] == min(wl.window, wl.T)
            err = run.follow(n)
            assert err <= H.FINAL_RTOL, f"sample {n}: final latent off by {err:.3g} x RMS"
            print(f"[parity] {name}[{n}]: sweeps={st['sweeps']} nfe={st['nfe']} hits={st['hits']} "
                  f"revisits={st['revisits']} below={st['revisits_below']} "
                  f"final_err={err:.2e} {run.eps_summary()} "
                  f"state_ulp_diffs={run.state_diffs} "
                  f"flips={len(run.log.flips) + len(run.follow_log.flips)}", flush=True)
            if independent:
                # reported, not gated: the oracle's own network drives its own run
                print(f"[parity] {name}[{n}] independent follow: {run.follow_independent(n)}", flush=True)
        agg = run.stats
        assert agg["nfe"] == sum(x["nfe"] for x in run.stats_n)
        assert agg["sweeps"] == max(x["sweeps"] for x in run.stats_n)
    finally:
        run.close()


def test_long_window_sd(gpu_lib):
    """Full-size long-window workload (T=1000, window 128): every sweep step-locked, sampled
    network outputs checked one by one, eps-locked follow to the final latent."""
    _long_window(0.05)


def test_long_window_sd_delta0(gpu_lib):
    """The long-window workload uncached (delta = 0): every window slot a miss, up to 128
    misses per network launch."""
    _long_window(0.0)


def _long_window(delta):
    wl = W.LONG_MLP
    print(f"[parity] long: {wl.name} delta={delta}", flush=True)
    run = H.Run(wl, delta, eps_stride=16).run()
    try:
        err = run.follow()
        assert err <= H.FINAL_RTOL
        assert run.stats["nfe"] >= wl.T
        if delta == 0.0:
            assert run.stats["hits"] == 0
        print(f"[parity] long: sweeps={run.stats['sweeps']} nfe={run.stats['nfe']} "
              f"hits={run.stats['hits']} final_err={err:.2e} {run.eps_summary()}", flush=True)
    finally:
        run.close()


def test_long_ddpm_window64(gpu_lib):
    """The window study's stochastic setting at full size: ancestral DDPM over T=1000 with a
    window of 64 on the SD latent shape, step-locked and followed to the final latent."""
    wl = W.LONG_MLP.with_(window=64)
    print(f"[parity] long ddpm: {wl.name} P=64 eta=1", flush=True)
    run = H.Run(wl, 0.05, eps_stride=32, eta=1.0).run()
    try:
        err = run.follow()
        assert err <= H.FINAL_RTOL
        print(f"[parity] long ddpm: sweeps={run.stats['sweeps']} nfe={run.stats['nfe']} "
              f"hits={run.stats['hits']} final_err={err:.2e} {run.eps_summary()}", flush=True)
    finally:
        run.close()
