"""C-ABI behaviour on the device: sample() against sweep-by-sweep, determinism, the state
machine, non-finite input, explicit schedules, and the uploaded coefficient tables."""
import math

import numpy as np
import pytest
import torch

from oracle import eps_models as em
from oracle import schedule as sch
from paper_2609_36522_amd import binding as B
from paper_2609_36522_amd import inputs
from paper_2609_36522_amd import workloads as W

pytestmark = pytest.mark.gpu


def _x(wl, seed=0):
    return torch.from_numpy(inputs.x_init(wl.latent, seed).reshape(-1)).cuda()


# mlp_window1: a fused patch-MLP handle whose sample needs exactly T sweeps (window 1), so its
# last slide runs in a network kernel launched after the T-th sweep.
@pytest.mark.parametrize("wl", [W.TINY_LINEAR, W.SMALL_MLP,
                                W.Workload("mlp_4x16x32_T6_P1", (4, 16, 32), 6, 1, 0.05, 1e-3,
                                           "patch_mlp", hidden=512)],
                         ids=["linear", "mlp", "mlp_window1"])
def test_sample_equals_sweep_by_sweep_and_is_deterministic(wl, gpu_lib):
    x = _x(wl)
    with B.from_workload(wl, trace=True) as s:
        out1 = s.sample(x).cpu().numpy()
        st1 = s.stats()
        tr1 = s.traces()
        out2 = s.sample(x).cpu().numpy()
        st2 = s.stats()
        tr2 = s.traces()
        s.reset(x)
        while not s.sweep(sync=True):
            pass
        st3 = s.stats()
        X, _, _, _ = s.read_state(wl.T, wl.T + 1)
    assert np.array_equal(out1, out2) and np.array_equal(out1, X[0])
    assert st1 == st2 == st3
    if wl.window == 1:
        assert st1["sweeps"] == wl.T
    for a, b in zip(tr1, tr2):
        assert a["miss"] == b["miss"] and a["c"] == b["c"]
        assert np.array_equal(a["dev"], b["dev"], equal_nan=True) and np.array_equal(a["r"], b["r"])


def test_state_machine(gpu_lib):
    wl = W.TINY_LINEAR
    with B.from_workload(wl) as s:
        with pytest.raises(B.PAError) as ei:
            s.sweep()
        assert ei.value.code == B.PA_ERR_STATE
        with pytest.raises(B.PAError) as ei:
            s.stats()
        assert ei.value.code == B.PA_ERR_STATE
        with pytest.raises(B.PAError) as ei:
            s.trace(0)
        assert ei.value.code == B.PA_ERR_STATE      # no trace flag
        s.sample(_x(wl))
        with pytest.raises(B.PAError) as ei:
            s.sweep()
        assert ei.value.code == B.PA_ERR_STATE      # already done
        with pytest.raises(B.PAError) as ei:
            s.kernel_times()
        assert ei.value.code == B.PA_ERR_STATE
    with B.from_workload(wl, trace=True) as s:
        s.sample(_x(wl))
        n = s.stats()["sweeps"]
        with pytest.raises(B.PAError) as ei:
            s.trace(n)
        assert ei.value.code == B.PA_ERR_INVALID_ARG


def test_nonfinite_input_is_reported(gpu_lib):
    wl = W.TINY_LINEAR
    x = _x(wl)
    x[5] = float("nan")
    with B.from_workload(wl) as s:
        with pytest.raises(B.PAError) as ei:
            s.sample(x)
        assert ei.value.code == B.PA_ERR_NONFINITE
        st = s.stats()
        assert st["done"] and st["nonfinite"] and st["sweeps"] == wl.T   # stride 1 on NaN
        out = s.sample(_x(wl))                  # the handle recovers after reset
        assert np.isfinite(out.cpu().numpy()).all()


def test_explicit_schedule_matches_scaled_linear(gpu_lib):
    wl = W.TINY_LINEAR
    ab, t = sch.sampler_alpha_bar(wl.T)
    x = _x(wl)
    with B.from_workload(wl) as s1, B.from_workload(wl, schedule={"alpha_bar": ab, "t_values": t}) as s2:
        a1, b1, _, _ = s1.coefficients()
        a2, b2, _, _ = s2.coefficients()
        assert np.array_equal(a1, a2) and np.array_equal(b1, b2)
        assert np.array_equal(s1.sample(x).cpu().numpy(), s2.sample(x).cpu().numpy())


@pytest.mark.parametrize("eta", [0.0, 1.0])
@pytest.mark.parametrize("delta", [0.0, 0.05])
def test_identity_steps_converge_in_one_sweep_per_window(delta, eta, gpu_lib):
    """alpha_bar = 1 at every state: every step is the identity (alpha = b = sigma = 0 in the
    uploaded tables, no NaN), every Eq. (2) residual is exactly 0, and at tau = 0 (r <= tau)
    each sweep slides the window to its end: ceil(T / P) sweeps, every step evaluated once,
    the initial latent returned bit for bit."""
    T, P = 12, 5
    wl = W.TINY_LINEAR.with_(T=T, window=P, tol=0.0)
    sched = {"alpha_bar": np.ones(T + 1), "t_values": sch.trailing_timesteps(T)}
    x = _x(wl)
    with B.from_workload(wl, delta, schedule=sched, eta=eta) as s:
        a, b, sig, _ = s.coefficients()
        assert np.all(a == 0.0) and np.all(b == 0.0) and np.all(sig == 0.0)
        if eta > 0.0:
            s.set_noise(torch.from_numpy(inputs.step_noise(1, T, wl.D).reshape(-1)).cuda())
        out = s.sample(x).cpu().numpy()
        st = s.stats()
    assert np.array_equal(out, x.cpu().numpy())
    assert st["sweeps"] == -(-T // P) and st["nfe"] == T and st["hits"] == 0


@pytest.mark.parametrize("T", [10, 50, 100, 1000])
def test_uploaded_coefficients_are_rounded_oracle_values(T, gpu_lib):
    wl = W.TINY_LINEAR.with_(T=T, window=min(4, T))
    ab, t = sch.sampler_alpha_bar(T)
    alpha, b = sch.ddim_coefficients(ab)
    with B.from_workload(wl) as s:
        a32, b32, _, _ = s.coefficients()
    # Same fp64 definition on both sides: bit-identical coefficient tables.
    assert np.array_equal(a32, alpha) and np.array_equal(b32, b)


def test_time_embedding_table(gpu_lib):
    wl = W.SMALL_MLP
    ab, t = sch.sampler_alpha_bar(wl.T)
    net = em.PatchMLP(inputs.mlp_weights(wl.hidden), t, wl.latent)
    with B.from_workload(wl) as s:
        _, _, _, temb = s.coefficients()
    diff = np.abs(temb.astype(np.float64) - net.temb.astype(np.float64))
    assert np.all(diff <= np.abs(net.temb) * 2.0 ** -23 + 1e-30)


def test_profile_counts_launches(gpu_lib):
    wl = W.SMALL_MLP
    with B.from_workload(wl, profile=True) as s:
        s.sample(_x(wl))
        kt = s.kernel_times()
        st = s.stats()
        # several samples between reads: each sample folds its launches into the totals
        for _ in range(3):
            s.sample(_x(wl))
        kt3 = s.kernel_times()
    # sample() may enqueue a sweep or two past done; those network launches exit at once.
    assert kt["launches"] >= st["sweeps"] and kt["eps_latents"] == st["nfe"]
    assert kt["eps_ms_total"] > 0
    assert kt3["launches"] >= 3 * st["sweeps"] and kt3["eps_latents"] == 3 * st["nfe"]
    assert kt["solver_launches"] == 0 and kt["picard_ms_total"] == 0.0
    with B.from_workload(wl, profile_solver=True) as s:
        s.sample(_x(wl))
        kt = s.kernel_times()
    assert kt["solver_launches"] == kt["launches"] >= st["sweeps"]
    # One patch-MLP sample: the window slide runs inside the next network kernel (no k_slide).
    assert kt["picard_ms_total"] > 0 and kt["slide_ms_total"] == 0.0
    with B.from_workload(wl, profile_solver=True, batch=2) as s:
        xs = torch.from_numpy(inputs.x_init_batch(wl.latent, 2).reshape(-1)).cuda()
        s.sample(xs)
        kt = s.kernel_times()
    assert kt["solver_launches"] == kt["launches"] > 0
    assert kt["picard_ms_total"] > 0 and kt["slide_ms_total"] > 0


@pytest.mark.parametrize("T,eta", [(10, 1.0), (100, 1.0), (1000, 1.0), (50, 0.5)])
def test_stochastic_coefficients_are_oracle_values(T, eta, gpu_lib):
    wl = W.TINY_LINEAR.with_(T=T, window=min(4, T))
    ab, t = sch.sampler_alpha_bar(T)
    alpha, b, sigma = sch.step_coefficients(ab, eta)
    with B.from_workload(wl, eta=eta) as s:
        a, bb, sg, _ = s.coefficients()
    assert np.array_equal(a, alpha) and np.array_equal(bb, b) and np.array_equal(sg, sigma)


def test_stochastic_handle_needs_noise(gpu_lib):
    wl = W.TINY_LINEAR
    x = _x(wl)
    with B.from_workload(wl, eta=1.0) as s:
        with pytest.raises(B.PAError) as ei:
            s.sample(x)
        assert ei.value.code == B.PA_ERR_STATE
        z = torch.from_numpy(inputs.step_noise(1, wl.T, wl.D).reshape(-1)).cuda()
        s.set_noise(z)
        out1 = s.sample(x).cpu().numpy()
        z2 = torch.zeros_like(z)
        s.set_noise(z2)
        out0 = s.sample(x).cpu().numpy()
    assert not np.array_equal(out1, out0)          # the noise term is live
    with B.from_workload(wl) as s:
        with pytest.raises(B.PAError) as ei:
            s.set_noise(torch.zeros(wl.T * wl.D, device="cuda"))
        assert ei.value.code == B.PA_ERR_INVALID_ARG


@pytest.mark.parametrize("wl,eta,N", [(W.TINY_LINEAR, 0.0, 4), (W.SMALL_MLP, 0.0, 4), (W.SD_MLP, 0.0, 4),
                                      (W.TINY_LINEAR, 1.0, 4), (W.SMALL_MLP, 1.0, 4),
                                      (W.SD_MLP, 0.0, 8), (W.SMALL_MLP, 1.0, 8), (W.TINY_LINEAR, 0.0, 8)],
                         ids=["linear", "mlp_small", "mlp_sd", "linear_ddpm", "mlp_small_ddpm",
                              "mlp_sd_batch8", "mlp_small_ddpm_batch8", "linear_batch8"])
def test_batch_equals_independent_samples(wl, eta, N, gpu_lib):
    """A handle with N samples gives each sample exactly what a single-sample handle gives
    it: the same final latent bit for bit, counters and sweep traces. Handles of eight or more
    samples run the Picard kernel builds capped for occupancy (deterministic, stochastic and
    linear-network builds)."""
    xb = inputs.x_init_batch(wl.latent, N).reshape(N, -1)
    Z = inputs.step_noise(N, wl.T, wl.D) if eta > 0 else None
    with B.from_workload(wl, batch=N, eta=eta, trace=True) as s:
        if Z is not None:
            s.set_noise(torch.from_numpy(Z.reshape(-1)).cuda())
        outb = s.sample(torch.from_numpy(xb.reshape(-1)).cuda()).cpu().numpy().reshape(N, -1)
        stb = [s.stats(n) for n in range(N)]
        trb = [s.traces(n) for n in range(N)]
        agg = s.stats()
    for n in range(N):
        with B.from_workload(wl, eta=eta, trace=True) as s1:
            if Z is not None:
                s1.set_noise(torch.from_numpy(Z[n].reshape(-1)).cuda())
            out1 = s1.sample(torch.from_numpy(xb[n]).cuda()).cpu().numpy()
            st1 = s1.stats()
            tr1 = s1.traces()
        assert np.array_equal(outb[n], out1), f"sample {n}"
        assert stb[n] == st1, (n, stb[n], st1)
        assert len(trb[n]) == len(tr1)
        for a, b in zip(trb[n], tr1):
            assert a["miss"] == b["miss"] and a["c"] == b["c"]
            assert np.array_equal(a["dev"], b["dev"], equal_nan=True) and np.array_equal(a["r"], b["r"])
    assert agg["nfe"] == sum(x["nfe"] for x in stb) and agg["done"]
    assert agg["sweeps"] == max(x["sweeps"] for x in stb)
    assert agg["window_start"] == min(x["window_start"] for x in stb)


def test_revisit_threshold(gpu_lib):
    wl = W.SMALL_MLP
    x = _x(wl)
    with B.from_workload(wl, 0.0) as s:
        s.sample(x)
        st = s.stats()
        assert st["revisits"] == st["nfe"] + st["hits"] - wl.T
        s.set_revisit_threshold(math.inf)
        s.sample(x)
        assert s.stats()["revisits_below"] == s.stats()["revisits"]
        s.set_revisit_threshold(0.0)
        s.sample(x)
        assert s.stats()["revisits_below"] == 0
        with pytest.raises(B.PAError) as ei:
            s.set_revisit_threshold(-1.0)
        assert ei.value.code == B.PA_ERR_INVALID_ARG
        with pytest.raises(B.PAError) as ei:
            s.set_revisit_threshold(float("nan"))
        assert ei.value.code == B.PA_ERR_INVALID_ARG


def test_batch_argument_checks(gpu_lib):
    wl = W.TINY_LINEAR
    with B.from_workload(wl, batch=3, trace=True) as s:
        xb = torch.from_numpy(inputs.x_init_batch(wl.latent, 3).reshape(-1)).cuda()
        s.sample(xb)
        for bad in (-1, 3):
            with pytest.raises(B.PAError) as ei:
                s.stats(bad)
            assert ei.value.code == B.PA_ERR_INVALID_ARG
            with pytest.raises(B.PAError) as ei:
                s.trace(0, bad)
            assert ei.value.code == B.PA_ERR_INVALID_ARG
            with pytest.raises(B.PAError) as ei:
                s.read_state(0, 1, bad)
            assert ei.value.code == B.PA_ERR_INVALID_ARG


@pytest.mark.parametrize("wl,batch", [(W.SMALL_MLP, 1), (W.SD_MLP, 1), (W.SD_MLP, 4),
                                      (W.Workload("mlp_4x32x32_T20_P8_H2048", (4, 32, 32), 20, 8, 0.05,
                                                  1e-3, "patch_mlp", hidden=2048), 1)],
                         ids=["mlp_small", "mlp_sd", "mlp_sd_batch4", "mlp_h2048"])
def test_whole_outputs_equal_split_outputs(wl, batch, gpu_lib):
    """A network launch writes whole outputs into the cache when that costs no extra time and
    split partials otherwise; both give the same bits. A handle forced to split outputs on
    every launch must end in the same trajectory, cache, counters and traces."""
    xb = inputs.x_init_batch(wl.latent, batch).reshape(-1) if batch > 1 else inputs.x_init(wl.latent).reshape(-1)
    x = torch.from_numpy(xb).cuda()
    res = []
    for split in (False, True):
        with B.from_workload(wl, batch=batch, trace=True, split_outputs=split) as s:
            out = s.sample(x).cpu().numpy()
            per = [(s.stats(n), s.traces(n), s.read_state(0, None, n)) for n in range(batch)]
        res.append((out, per))
    (o0, p0), (o1, p1) = res
    assert np.array_equal(o0, o1)
    for n in range(batch):
        (st0, tr0, S0), (st1, tr1, S1) = p0[n], p1[n]
        assert st0 == st1, (n, st0, st1)
        assert len(tr0) == len(tr1)
        for a, b in zip(tr0, tr1):
            assert a["miss"] == b["miss"] and a["c"] == b["c"]
            assert np.array_equal(a["dev"], b["dev"], equal_nan=True) and np.array_equal(a["r"], b["r"])
        for A, Bv in zip(S0, S1):
            assert np.array_equal(A, Bv), n


@pytest.mark.parametrize("wl,batch", [(W.TINY_LINEAR, 3), (W.SMALL_MLP, 1)], ids=["linear_batch3", "mlp"])
def test_sample_output_alignment(wl, batch, gpu_lib):
    """Buffers at any 4-byte offset and an aliased x_init == x_out give the same final
    latents, bit for bit, and the same counters."""
    xs = inputs.x_init_batch(wl.latent, batch).reshape(-1) if batch > 1 else inputs.x_init(wl.latent).reshape(-1)
    n = xs.size
    big = torch.zeros(n + 4, device="cuda")
    with B.from_workload(wl, batch=batch) as s:
        x = torch.from_numpy(xs).cuda()
        ref = s.sample(x).cpu().numpy()
        st = s.stats()
        big[1:n + 1] = x                      # 4-byte offset: not 16-byte aligned
        out_big = torch.zeros(n + 4, device="cuda")
        s.sample(big[1:n + 1], out_big[3:n + 3])
        assert np.array_equal(out_big[3:n + 3].cpu().numpy(), ref)
        assert s.stats() == st
        y = x.clone()
        s.sample(y, y)                        # in place
        assert np.array_equal(y.cpu().numpy(), ref)


def _create_raw(latent, T, window, c):
    """paraanya_create through ctypes, *out preset to a non-NULL value; returns (rc, handle)."""
    import ctypes as C
    lib = B.load_library()
    keep = []
    sc, em_ = B._schedule_and_model(keep, None, 0.0, "linear", c, None, 0)
    shape = (C.c_int32 * 4)(1, *latent)
    h = C.c_void_p(0x1234)
    rc = lib.paraanya_create(shape, int(T), C.byref(sc), int(window), 0.05, 1e-3, C.byref(em_),
                             C.c_void_p(torch.cuda.current_stream().cuda_stream), 0, C.byref(h))
    return rc, h


def test_create_out_of_memory_fails_cleanly(gpu_lib):
    """Device buffers beyond the device's memory: create fails with PA_ERR_OOM before any
    sweep, sets *out to NULL and frees whatever it had allocated; the next valid create and
    sample work. Two sizes: the first buffer (the trajectory) alone is too large, and the
    trajectory and cached inputs fit but the cached outputs do not."""
    torch.cuda.synchronize()
    free0, total = torch.cuda.mem_get_info()
    lat = (4, 8192, 8192)                       # 1 GiB per state
    row = 4 * 8192 * 8192 * 4
    for T in (1000, int(0.4 * free0 // row)):
        assert 1 <= T <= 1000 and (T == 1000 or 2 * (T + 1) * row < free0)
        c = np.full(T, 0.9, np.float32)
        print(f"[oom] T={T}: {T * row / 2**30:.1f} GiB per [T][D] buffer, {free0 / 2**30:.1f} GiB free", flush=True)
        rc, h = _create_raw(lat, T, 1, c)
        assert rc == B.PA_ERR_OOM, (rc, B.status_str(rc))
        assert h.value is None
        torch.cuda.synchronize()
        free1, _ = torch.cuda.mem_get_info()
        assert free1 >= free0 - (64 << 20), f"{(free0 - free1) / 2**20:.0f} MiB not returned"
    wl = W.TINY_LINEAR
    with B.from_workload(wl) as s:
        out = s.sample(_x(wl)).cpu().numpy()
        assert s.stats()["done"] and np.isfinite(out).all()


def test_largest_handle_offsets(gpu_lib):
    """Maximum sizes: 64 samples (PA_MAX_BATCH), window 256 (PA_MAX_WINDOW), T = 1000 and 4x96x96
    latents, so the trajectory alone holds 64 x 1001 x 36864 = 2.36e9 floats (beyond 2^31): a
    32-bit element offset anywhere in a kernel or a host copy would read or write another
    sample's rows. tau = inf makes every window converge in one sweep (slides of 256), delta =
    0.05. Linear network: the last and the first sample end on the oracle's final latent (same
    NFE and hits). Patch-MLP (H = 1024): the last sample's cached outputs at the last timesteps
    equal the oracle network's outputs for the device's cached inputs, and its final latent
    differs from the first sample's."""
    from oracle import sampler as sp
    import parity_harness as H
    N, T, P = B.PA_MAX_BATCH, 1000, B.PA_MAX_WINDOW
    shape = (4, 96, 96)
    D = int(np.prod(shape))
    assert N * (T + 1) * D > 2 ** 31
    ab, tv = sch.sampler_alpha_bar(T)
    alpha, b = sch.ddim_coefficients(ab)
    xs = inputs.x_init_batch(shape, N).reshape(N, -1)
    x = torch.from_numpy(xs.reshape(-1)).cuda()
    lin = W.Workload("lin_64x4x96x96_T1000_P256", shape, T, P, 0.05, math.inf, "linear")
    print(f"[max-size] linear N={N} T={T} P={P} latent={shape}", flush=True)
    with B.from_workload(lin, batch=N) as s:
        out = s.sample(x).cpu().numpy().reshape(N, -1)
        st = [s.stats(n) for n in (0, N - 1)]
    c = inputs.linear_coefficients(T)
    for k, n in enumerate((0, N - 1)):
        xo, _, ost = sp.sample(xs[n], T, P, 0.05, math.inf, alpha, b, em.linear_eps(c))
        assert (st[k]["nfe"], st[k]["hits"]) == (ost.nfe, ost.hits), (n, st[k], ost)
        rms = float(np.sqrt(np.mean(xo.astype(np.float64) ** 2)))
        assert np.max(np.abs(out[n].astype(np.float64) - xo)) <= 1e-4 * rms, n
    del out
    mlp = W.Workload("mlp_64x4x96x96_T1000_P256_H1024", shape, T, P, 0.05, math.inf, "patch_mlp", hidden=1024)
    print(f"[max-size] patch-MLP H=1024 N={N} T={T} P={P} latent={shape}", flush=True)
    net = em.PatchMLP(inputs.mlp_weights(1024), tv, shape)
    with B.from_workload(mlp, batch=N) as s:
        out = s.sample(x).cpu().numpy().reshape(N, -1)
        _, Xh, Eh, valid = s.read_state(T - 2, T, N - 1)
    assert valid.all()
    for i, t in enumerate((T - 2, T - 1)):
        ref = net.eval_one(Xh[i], t)
        assert H.eps_error(Eh[i], ref, shape) <= H.EPS_RTOL, t
    assert np.isfinite(out).all() and not np.array_equal(out[0], out[N - 1])


@pytest.mark.parametrize("wl,batch", [(W.TINY_LINEAR, 3), (W.SMALL_MLP, 1), (W.SD_MLP, 1), (W.SMALL_MLP, 2)],
                         ids=["linear_batch3", "mlp_small", "mlp_sd", "mlp_small_batch2"])
def test_sample_counters_from_done_words(wl, batch, gpu_lib):
    """paraanya_sample returns once every sample's done word is seen, without draining the
    stream, and takes the counters from the final counter words the last slide wrote (tagged
    with the sample's epoch). They must equal what the control blocks hold after a full
    synchronization (a profiling handle always takes that path), sample by sample, over
    several samples in a row on one handle; the outputs, read after the stream, must agree
    bit for bit, and a reset right after a sample must not see the previous sample's words."""
    xb = inputs.x_init_batch(wl.latent, batch).reshape(-1) if batch > 1 else inputs.x_init(wl.latent).reshape(-1)
    x = torch.from_numpy(xb).cuda()
    runs = []
    for profile in (False, True):
        with B.from_workload(wl, batch=batch, profile=profile) as s:
            got = []
            for _ in range(3):
                out = s.sample(x)
                st = [s.stats()] + [s.stats(n) for n in range(batch)]
                got.append((out.cpu().numpy(), st))
            s.reset(x)                       # the next sample starts from a clean slate
            s.sweep(sync=True)
            assert s.stats()["sweeps"] == 1
        runs.append(got)
    for (o0, s0), (o1, s1) in zip(*runs):
        assert np.array_equal(o0, o1)
        assert s0 == s1, (s0, s1)
    assert runs[0][0][1] == runs[0][2][1]    # the same input gives the same counters each time


@pytest.mark.parametrize("wl", [W.TINY_LINEAR, W.SMALL_MLP], ids=["linear", "mlp"])
def test_chained_samples_are_stream_ordered(wl, gpu_lib):
    """paraanya_sample returns before its output copy has run; feeding each output straight
    back as the next sample's input (no synchronization in between, in place and into a second
    tensor) must give what a synchronizing handle gives."""
    x = _x(wl)
    results = []
    for profile in (False, True):
        with B.from_workload(wl, profile=profile) as s:
            a = x.clone()
            b = torch.empty_like(a)
            s.sample(a, b)          # b <- sample(x)
            s.sample(b, b)          # in place
            s.sample(b, a)          # a <- sample(b)
            results.append(a.cpu().numpy())
    assert np.array_equal(results[0], results[1])
    assert np.isfinite(results[0]).all()


def test_concurrent_handles_on_separate_streams_and_threads(gpu_lib):
    """Handles share no state: two host threads, each with its own handle on its own stream
    (default priority), and a third calling the allocation-free entry point (which shares one
    locked workspace per device) run at the same time; every output and counter equals the
    same calls made one after another on the current stream."""
    import threading
    jobs = [(W.SD_MLP, 1), (W.SMALL_MLP, 2), (W.TINY_LINEAR, 3)]
    reps = 4

    def xs(wl, n):
        a = inputs.x_init(wl.latent).reshape(-1) if n == 1 else inputs.x_init_batch(wl.latent, n).reshape(-1)
        return torch.from_numpy(a)

    def chain(wl, n, stream=None):
        out, sts = [], []
        with B.from_workload(wl, batch=n, stream=stream) as s:
            x = xs(wl, n).cuda()
            for _ in range(reps):
                x = s.sample(x)
                out.append(x.cpu().numpy())
                sts.append(s.stats())
        return out, sts

    def noalloc_chain(stream=None):
        out = []
        x = xs(W.SMALL_MLP, 1).cuda()
        for _ in range(reps):
            x, st = B.sample_noalloc_workload(W.SMALL_MLP, x, stream=stream)
            out.append((x.cpu().numpy(), st))
        return out

    ref = [chain(wl, n) for wl, n in jobs]
    ref_na = noalloc_chain()
    torch.cuda.synchronize()

    results, errors = {}, []

    def run(key, fn):
        try:
            st = torch.cuda.Stream()
            with torch.cuda.stream(st):
                results[key] = fn(st)
                st.synchronize()
        except Exception as e:      # reported below, in the test's thread
            errors.append((key, repr(e)))

    threads = [threading.Thread(target=run, args=(i, lambda st, wl=wl, n=n: chain(wl, n, st)))
               for i, (wl, n) in enumerate(jobs)]
    threads.append(threading.Thread(target=run, args=("na", lambda st: noalloc_chain(st))))
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a thread did not finish"
    assert not errors, errors
    for i in range(len(jobs)):
        out, sts = results[i]
        for a, b in zip(out, ref[i][0]):
            assert np.array_equal(a, b), jobs[i][0].name
        assert sts == ref[i][1]
    for (a, sa), (b, sb) in zip(results["na"], ref_na):
        assert np.array_equal(a, b) and sa == sb


@pytest.mark.parametrize("wl,batch,reps", [(W.SD_MLP, 1, 200), (W.SD_MLP, 8, 40), (W.TINY_LINEAR, 5, 300)])
def test_repeated_samples_are_bitwise_identical(wl, batch, reps, gpu_lib):
    """Soak for races: many samples back to back on one handle (each returning before its
    output copy has run, the counters taken from the final progress and counter words) give
    the same output bits and counters every time."""
    xs = inputs.x_init(wl.latent).reshape(-1) if batch == 1 else inputs.x_init_batch(wl.latent, batch).reshape(-1)
    x = torch.from_numpy(xs).cuda()
    with B.from_workload(wl, batch=batch) as s:
        outs = [torch.empty_like(x) for _ in range(reps)]
        stats = []
        for o in outs:
            s.sample(x, o)
            stats.append(s.stats())
        first = outs[0].cpu().numpy()
        for i, o in enumerate(outs):
            assert np.array_equal(o.cpu().numpy(), first), f"sample {i} differs"
    assert all(st == stats[0] for st in stats)
