"""The allocation-free entry point (paraanya_sample_noalloc) through the C ABI: the same final
latents and counters, bit for bit, as a handle created and sampled through paraanya_create /
paraanya_sample, on two calls in a row (the second with a smaller input, which reuses the
workspace the first one filled), a batched linear request, and a clear error for a request
beyond the workspace."""
import numpy as np
import pytest
import torch

from paper_2609_36522_amd import binding as B
from paper_2609_36522_amd import inputs
from paper_2609_36522_amd import workloads as W

pytestmark = pytest.mark.gpu


def _x(wl, batch=1):
    xs = inputs.x_init(wl.latent).reshape(-1) if batch == 1 else inputs.x_init_batch(wl.latent, batch).reshape(-1)
    return torch.from_numpy(xs).cuda()


def _reference(wl, x, batch=1):
    with B.from_workload(wl, batch=batch) as s:
        out = s.sample(x).cpu().numpy()
        return out, s.stats()


def test_noalloc_equals_handle_path(gpu_lib):
    cases = [(W.SD_MLP, 1), (W.SMALL_MLP, 1), (W.TINY_LINEAR, 3)]
    refs = [(_x(wl, n), *_reference(wl, _x(wl, n), n)) for wl, n in cases]
    torch.cuda.synchronize()
    for rep in range(2):
        for (wl, n), (x, ref, st_ref) in zip(cases, refs):
            free0, _ = torch.cuda.mem_get_info()
            out, st = B.sample_noalloc_workload(wl, x, batch=n)
            torch.cuda.synchronize()
            free1, _ = torch.cuda.mem_get_info()
            print(f"[noalloc] {wl.name} batch={n} rep={rep}: nfe={st['nfe']} sweeps={st['sweeps']}", flush=True)
            assert np.array_equal(out.cpu().numpy(), ref), (wl.name, n, rep)
            assert st == st_ref, (wl.name, st, st_ref)
            if rep == 1:   # everything the library needs was set up by the first round
                assert free1 >= free0 - (4 << 20), f"{(free0 - free1) / 2**20:.1f} MiB taken"


def test_noalloc_in_place_and_limits(gpu_lib):
    wl = W.SMALL_MLP
    x = _x(wl)
    ref, st_ref = _reference(wl, x)
    y = x.clone()
    out, st = B.sample_noalloc_workload(wl, y, y)             # x_init and x_out alias
    assert out.data_ptr() == y.data_ptr() and np.array_equal(y.cpu().numpy(), ref) and st == st_ref
    big = W.LONG_MLP                                          # ~200 MB of buffers
    with pytest.raises(B.PAError) as ei:
        B.sample_noalloc_workload(big, _x(big))
    assert ei.value.code == B.PA_ERR_INVALID_ARG and "workspace" in str(ei.value)
    out, st = B.sample_noalloc_workload(wl, x)                # still works after the refusal
    assert np.array_equal(out.cpu().numpy(), ref) and st == st_ref


def test_noalloc_random_configurations(gpu_lib):
    """Ten seeded random deterministic-step configurations (linear or patch-MLP, ragged linear
    latents, any window, delta and tau, 1 to 5 samples): the allocation-free call equals the
    handle path bit for bit, or, if its buffers do not fit the workspace, refuses with
    PA_ERR_INVALID_ARG and leaves the next call working."""
    import math
    import random
    from paper_2609_36522_amd.workloads import Workload
    rng = random.Random(20260202)
    ran = 0
    for i in range(10):
        if rng.random() < 0.4:
            hw = rng.choice([(16, 32), (32, 32), (32, 64), (48, 64)])
            wl = Workload(f"na_rand{i}", (4, hw[0], hw[1]), rng.randint(2, 60), 1, 0.05, 1e-3, "patch_mlp",
                          hidden=rng.choice([512, 1024]))
        else:
            while True:
                lat = (rng.randint(1, 5), rng.randint(1, 20), rng.randint(1, 20))
                if (lat[0] * lat[1] * lat[2]) % 4 == 0:
                    break
            wl = Workload(f"na_rand{i}", lat, rng.randint(1, 300), 1, 0.05, 1e-3, "linear")
        wl = wl.with_(window=rng.randint(1, min(wl.T, 256)), delta=rng.choice([0.0, 0.05, 0.3, math.inf]),
                      tol=rng.choice([0.0, 1e-3, 1e-1]))
        n = rng.choice([1, 1, 2, 5])
        x = _x(wl, n)
        print(f"[noalloc] {wl.name}: {wl.model} latent={wl.latent} T={wl.T} P={wl.window} "
              f"delta={wl.delta} tol={wl.tol} batch={n}", flush=True)
        ref, st_ref = _reference(wl, x, n)
        try:
            out, st = B.sample_noalloc_workload(wl, x, batch=n)
        except B.PAError as e:
            assert e.code == B.PA_ERR_INVALID_ARG and "workspace" in str(e), str(e)
            continue
        ran += 1
        assert np.array_equal(out.cpu().numpy(), ref) and st == st_ref, wl.name
    assert ran >= 5
