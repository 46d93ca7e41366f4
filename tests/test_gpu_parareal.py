"""Cached Parareal on the device against the oracle (MI355X only), through the C ABI.

Every request of the device run (coarse initialization, batched fine steps, coarse
corrections) is compared with the oracle's request sequence: the same timestep, the same
Eq. (4) deviation up to fp64 summation order, the same hit decision (a flip allowed only
inside the 1e-6 relative band around delta). The linear network runs the oracle fully
independently; the patch-MLP runs it eps-locked (the oracle consumes the device's fresh
outputs, in request order) and fresh outputs are checked against the oracle network: all of
the initialization and of the first fine step, the first of every phase of every iteration,
and every 16th of the rest. Boundary residuals, counters, boundary states and the output are
compared.
"""
import math

import numpy as np
import pytest
import torch

from oracle import eps_models as em
from oracle import parareal as pr
from oracle import schedule as sch
from paper_2609_36522_amd import binding as B
from paper_2609_36522_amd import inputs
from paper_2609_36522_amd import workloads as W
from paper_2609_36522_amd.workloads import Workload

import parity_harness as H

pytestmark = pytest.mark.gpu

INF = math.inf


def _wl(name, latent, T, blocks, model="linear", hidden=0):
    return Workload(name, latent, T, 1, 0.05, 1e-3, model, hidden=hidden, blocks=blocks)


CASES = [
    ("lin_tiny", _wl("pr_lin_4x8x8_T20_B4", (4, 8, 8), 20, 4), 0.05),
    ("lin_tiny_delta0", _wl("pr_lin_4x8x8_T20_B4", (4, 8, 8), 20, 4), 0.0),
    ("lin_tiny_delta_inf", _wl("pr_lin_4x8x8_T20_B4", (4, 8, 8), 20, 4), INF),
    ("lin_ragged", _wl("pr_lin_3x5x4_T12_B3", (3, 5, 4), 12, 3), 0.1),
    ("lin_one_block", _wl("pr_lin_4x8x8_T10_B1", (4, 8, 8), 10, 1), 0.05),
    ("lin_unit_blocks", _wl("pr_lin_4x8x8_T8_B8", (4, 8, 8), 8, 8), 0.05),
    ("lin_c5_shape", _wl("pr_lin_4x96x96_T100_B10", (4, 96, 96), 100, 10), 0.05),
    ("lin_max_blocks", _wl("pr_lin_4x8x8_T64_B64", (4, 8, 8), 64, 64), 0.05),
    ("mlp_small", _wl("pr_mlp_4x32x32_T20_B4_H512", (4, 32, 32), 20, 4, "patch_mlp", 512), 0.05),
    # the most blocks, two fine steps each: fine-step launches of up to 64 latents through the
    # network kernel, over several iterations (all misses at delta = 0)
    ("mlp_max_blocks", _wl("pr_mlp_4x16x32_T128_B64_H512", (4, 16, 32), 128, 64, "patch_mlp", 512), 0.05),
    ("mlp_max_blocks_delta0", _wl("pr_mlp_4x16x32_T128_B64_H512", (4, 16, 32), 128, 64, "patch_mlp", 512), 0.0),
    ("mlp_c5", W.PARAREAL_MLP, 0.05),
    ("mlp_c5_delta0", W.PARAREAL_MLP, 0.0),
]


EPS_STRIDE = 16   # every 16th fresh output, besides those always checked (see eps_fn)


def _oracle_requests(trace):
    out = []
    for rec in trace:
        groups = [(0, -1, r) for r in rec["coarse"]] if rec["kind"] == "init" else \
            [(1, rec["k"], r) for r in rec["fine"]] + [(2, rec["k"], r) for r in rec["coarse"]]
        for phase, k, r in groups:
            for t, d, h in zip(r["t"], r["dev"], r["hit"]):
                out.append({"phase": phase, "iteration": k, "t": t, "dev": float(d), "hit": bool(h)})
    return out


@pytest.mark.parametrize("name,wl,delta", CASES, ids=[c[0] for c in CASES])
def test_parareal_parity(name, wl, delta, gpu_lib):
    print(f"[parareal] {name}: {wl.name} delta={delta}", flush=True)
    T, Bk = wl.T, wl.blocks
    ab, t_values = sch.sampler_alpha_bar(T)
    alpha, b = sch.ddim_coefficients(ab)
    x = inputs.x_init(wl.latent).reshape(-1)
    mlp = wl.model != "linear"
    with B.parareal_from_workload(wl, delta, trace=True) as s:
        out = s.sample(torch.from_numpy(x).cuda()).cpu().numpy()
        st = s.stats()
        recs = [s.trace(i, with_eps=mlp) for i in range(st["requests"])]
        res = [s.residuals(k) for k in range(st["iterations"])]
        U = s.boundaries()
    assert st["done"] and not st["nonfinite"] and 1 <= st["iterations"] <= Bk
    assert st["nfe"] == sum(1 for r, _ in recs if not r["hit"])
    if mlp:
        net = em.PatchMLP(inputs.mlp_weights(wl.hidden, temb_dim=wl.temb_dim), t_values, wl.latent)
        queue = [(r["t"], (r["phase"], r["iteration"]), e) for r, e in recs if not r["hit"]]
        checked = []
        seen = {}
        fresh = [0]

        # Fresh outputs checked against the oracle network: every output of the
        # initialization (single-latent coarse launches, 64-token items) and of the first fine
        # step (one batched launch over all blocks, 128-token items, which cross patch rows
        # when W/2 does not divide 128, as at 4x96x96), the first output of every phase of
        # every iteration (the corrections are single-latent launches too), and every
        # EPS_STRIDE-th fresh output of the run.
        def eps_fn(Xb, ts, _q=queue):
            rows = []
            for r, t in enumerate(ts):
                t_dev, grp, e = _q.pop(0)
                assert t_dev == t, f"miss order differs: device {t_dev}, oracle {t}"
                k = seen.get(grp, 0)
                seen[grp] = k + 1
                check = (grp[0] == 0 or (grp == (1, 0) and k < Bk) or k == 0 or fresh[0] % EPS_STRIDE == 0)
                fresh[0] += 1
                if check:
                    ref = net.eval_one(Xb[r], t)
                    e_rel = H.eps_error(e, ref, wl.latent)
                    checked.append(e_rel)
                    assert e_rel <= H.EPS_RTOL, f"network output at t={t} off by {e_rel:.3g} x its scale"
                rows.append(e)
            return np.stack(rows)
    else:
        eps_fn = em.linear_eps(inputs.linear_coefficients(T))
    xo, trace, sto = pr.sample(x, T, Bk, delta, wl.tol, ab, alpha, b, eps_fn)
    oreq = _oracle_requests(trace)
    assert len(oreq) == len(recs), (len(oreq), len(recs))
    flips = 0
    for i, ((g, _), o) in enumerate(zip(recs, oreq)):
        assert (g["phase"], g["iteration"], g["t"]) == (o["phase"], o["iteration"], o["t"]), (i, g, o)
        assert np.isnan(g["dev"]) == np.isnan(o["dev"]), (i, g, o)
        if not np.isnan(o["dev"]):
            assert abs(g["dev"] - o["dev"]) <= H.SUM_RTOL * o["dev"] + 1e-300, (i, g["dev"], o["dev"])
        if g["hit"] != o["hit"]:
            assert abs(o["dev"] - delta) <= H.BAND * delta, f"request {i}: hit differs outside the band"
            flips += 1
    assert st["nfe"] == sto["nfe"] and st["hits"] == sto["hits"] and st["iterations"] == sto["iters"]
    for k, rec in enumerate(r for r in trace if r["kind"] == "iter"):
        ro = rec["r"]
        rg = res[k][k + 1:]
        assert np.all(np.abs(rg - ro) <= 1e-9 * np.abs(ro) + 1e-30), (k, rg, ro)
    sc = max(H.rms(xo), 1e-30)
    err = float(np.max(np.abs(out.astype(np.float64) - xo)) / sc)
    uerr = float(np.max(np.abs(U.astype(np.float64) - sto["U"])) / sc)
    assert err <= H.FINAL_RTOL and uerr <= H.FINAL_RTOL
    if delta == 0.0:
        assert st["hits"] == 0
    if delta == INF:
        assert st["nfe"] == T
    print(f"[parareal] {name}: iterations={st['iterations']} nfe={st['nfe']} hits={st['hits']} "
          f"requests={st['requests']} final_err={err:.2e} boundary_err={uerr:.2e} flips={flips}"
          + (f" eps_checked={len(checked)} eps_err_max={max(checked):.2e}" if mlp else ""), flush=True)


def test_parareal_repeatable_and_state_errors(gpu_lib):
    wl = _wl("pr_lin_4x8x8_T20_B4", (4, 8, 8), 20, 4)
    x = torch.from_numpy(inputs.x_init(wl.latent).reshape(-1)).cuda()
    with B.parareal_from_workload(wl, 0.05) as s:
        with pytest.raises(B.PAError) as ei:
            s.stats()
        assert ei.value.code == B.PA_ERR_STATE
        a = s.sample(x).cpu().numpy()
        st1 = s.stats()
        b_ = s.sample(x).cpu().numpy()
        st2 = s.stats()
        with pytest.raises(B.PAError) as ei:
            s.trace(0)
        assert ei.value.code == B.PA_ERR_STATE          # no trace flag
    assert np.array_equal(a, b_) and st1 == st2


@pytest.mark.parametrize("T,Bk", [(20, 4), (12, 3), (10, 10)])
def test_parareal_identity_steps_stop_after_one_iteration(T, Bk, gpu_lib):
    """alpha_bar = 1 at every state: coarse and fine steps are the identity, the first
    iteration moves no boundary (every Eq. (2) residual exactly 0), and at tau = 0 (r <= tau)
    the sampler stops there: one iteration, NFE = T + 2B - 1 at delta = 0 (the B coarse
    requests of the initialization, T fine steps, B - 1 coarse corrections), the initial
    latent returned bit for bit."""
    wl = Workload(f"pr_identity_T{T}_B{Bk}", (4, 8, 8), T, 1, 0.0, 0.0, "linear", blocks=Bk)
    sched = {"alpha_bar": np.ones(T + 1), "t_values": sch.trailing_timesteps(T)}
    x = torch.from_numpy(inputs.x_init(wl.latent).reshape(-1)).cuda()
    with B.parareal_from_workload(wl, 0.0, schedule=sched) as s:
        out = s.sample(x).cpu().numpy()
        st = s.stats()
    assert np.array_equal(out, x.cpu().numpy())
    assert st["iterations"] == 1 and st["done"] == 1 and st["nfe"] == T + 2 * Bk - 1 and st["hits"] == 0


def test_parareal_repeated_samples_are_bitwise_identical(gpu_lib):
    """Soak for races: 20 Parareal samples back to back at the full 4x96x96, H = 2048 shape
    give the same output bits and counters every time."""
    wl = W.PARAREAL_MLP
    x = torch.from_numpy(inputs.x_init(wl.latent).reshape(-1)).cuda()
    with B.parareal_from_workload(wl, 0.05) as s:
        outs, stats = [], []
        for _ in range(20):
            outs.append(s.sample(x).cpu().numpy())
            stats.append(s.stats())
    assert all(np.array_equal(o, outs[0]) for o in outs)
    assert all(st == stats[0] for st in stats)
