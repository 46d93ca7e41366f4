"""Seeded random configurations through the step-locked parity harness (MI355X only).

Beyond the hand-picked cases of test_gpu_parity.py: 24 configurations drawn from a fixed
seed over the valid domain of the sampler -- linear network (latents C x H x W with C*H*W a
multiple of 4, 1..5 x 1..20 x 1..20, T up to 300) or patch-MLP (hidden 512, 1024 or 2048,
4 x H x W latents whose token count is a multiple of 128, T up to 100), any window 1..min(T,
256), delta in {0, 0.01, 0.05, 0.1, 0.3, inf}, tau in {0, 1e-4, 1e-3, 1e-2, 1e-1}, 1 to 8
samples per handle, eta in {0, 0.5, 1}. Each run is checked as in test_gpu_parity.py: every
sweep step-locked against the oracle (decisions exactly, states within one fp32 ulp),
counters consistent with the traces, network outputs against the oracle network, and the
followed final latent within 1e-4 x RMS. Then 12 seeded random configurations of the
Parareal sampler, checked as in test_gpu_parareal.py.
"""
import math
import random

import pytest

import parity_harness as H
from paper_2609_36522_amd.workloads import Workload

INF = math.inf
SEED = 20260201
COUNT = 24


def _configs():
    rng = random.Random(SEED)
    out = []
    for i in range(COUNT):
        mlp = rng.random() < 0.35
        if mlp:
            hidden = rng.choice([512, 1024, 1024, 2048])
            hw = rng.choice([(16, 32), (32, 32), (32, 16), (16, 64), (32, 64), (64, 32), (48, 64), (32, 96)])
            latent = (4, hw[0], hw[1])
            T = rng.randint(2, 24) if rng.random() < 0.8 else rng.randint(24, 100)
        else:
            hidden = 0
            while True:
                latent = (rng.randint(1, 5), rng.randint(1, 20), rng.randint(1, 20))
                if (latent[0] * latent[1] * latent[2]) % 4 == 0:
                    break
            T = rng.choice([1, 2, 3, rng.randint(4, 40), rng.randint(40, 300)])
        P = rng.randint(1, min(T, 256)) if rng.random() < 0.8 else min(T, 256, rng.choice([1, 2, T]))
        delta = rng.choice([0.0, 0.01, 0.05, 0.1, 0.3, INF])
        tol = rng.choice([0.0, 1e-4, 1e-3, 1e-2, 1e-1])
        batch = rng.choice([1, 1, 1, 2, 3, 5, 8]) if not (mlp and hidden == 2048) else rng.choice([1, 2])
        eta = rng.choice([0.0, 0.0, 0.0, 1.0, 0.5])
        wl = Workload(f"rand{i}", latent, T, P, delta, tol, "patch_mlp" if mlp else "linear", hidden=hidden)
        out.append((wl, batch, eta))
    return out


CONFIGS = _configs()


@pytest.mark.gpu
@pytest.mark.parametrize("wl,batch,eta", CONFIGS, ids=[c[0].name for c in CONFIGS])
def test_random_configuration(wl, batch, eta, gpu_lib):
    T, P, delta = wl.T, wl.window, wl.delta
    print(f"[random] {wl.name}: {wl.model} H={wl.hidden} latent={wl.latent} T={T} P={P} "
          f"delta={delta} tol={wl.tol} batch={batch} eta={eta}", flush=True)
    run = H.Run(wl, delta, batch=batch, eta=eta, eps_stride=3).run()
    try:
        for n in range(run.N):
            st, recs = run.stats_n[n], run.records[n]
            assert st["done"] and st["sweeps"] == len(recs) <= T
            assert st["nfe"] >= T and st["nfe"] == sum(r["m"] for r in recs)
            assert st["hits"] == sum(r["e"] - r["s"] - r["m"] for r in recs)
            if delta == 0.0:
                assert st["hits"] == 0
            if delta == INF:
                assert st["nfe"] == T
            assert recs[0]["m"] == min(P, T)
            err = run.follow(n)
            assert err <= H.FINAL_RTOL, f"sample {n}: final latent off by {err:.3g} x RMS"
        print(f"[random] {wl.name}: sweeps={run.stats['sweeps']} nfe={run.stats['nfe']} {run.eps_summary()}",
              flush=True)
    finally:
        run.close()


def _parareal_configs():
    import test_gpu_parareal as TP
    rng = random.Random(SEED + 1)
    out = []
    for i in range(12):
        mlp = rng.random() < 0.4
        B = rng.randint(1, 12)
        T = B * rng.randint(1, 10)
        if mlp:
            hw = rng.choice([(16, 32), (32, 32), (32, 64), (48, 64), (32, 96)])
            wl = TP._wl(f"pr_rand{i}", (4, hw[0], hw[1]), T, B, "patch_mlp", rng.choice([512, 1024, 2048]))
        else:
            while True:
                lat = (rng.randint(1, 5), rng.randint(1, 16), rng.randint(1, 16))
                if (lat[0] * lat[1] * lat[2]) % 4 == 0:
                    break
            wl = TP._wl(f"pr_rand{i}", lat, T, B)
        out.append((wl, rng.choice([0.0, 0.01, 0.05, 0.2, INF])))
    return out


PR_CONFIGS = _parareal_configs()


@pytest.mark.gpu
@pytest.mark.parametrize("wl,delta", PR_CONFIGS, ids=[c[0].name for c in PR_CONFIGS])
def test_random_parareal_configuration(wl, delta, gpu_lib):
    """The Parareal sampler on 12 seeded random configurations (1 to 12 blocks of 1 to 10 fine
    steps; linear or patch-MLP), checked as in test_gpu_parareal.py."""
    import test_gpu_parareal as TP
    TP.test_parareal_parity(wl.name, wl, delta, gpu_lib)
