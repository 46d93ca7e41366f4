"""The C-ABI library on the CPU: it loads, exports every entry point the header declares,
and rejects invalid arguments before making any HIP call (no GPU needed)."""
import ctypes as C
import math
import os
import re

import numpy as np
import pytest

from paper_2609_36522_amd import binding as B
from paper_2609_36522_amd import inputs

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "paraanya.h")


def _declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"PA_API\s+[\w\s\*]*?\b(paraanya_\w+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = B.load_library()
    names = _declared()
    assert len(names) == 26
    assert sorted(B.EXPORTED) == names
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    assert B.status_str(0) == "PA_OK"
    assert B.status_str(-1) == "PA_ERR_INVALID_ARG"
    assert B.status_str(-6) == "PA_ERR_UNSUPPORTED"
    assert B.status_str(-99) == "PA_ERR_UNKNOWN"


def _create(shape=(1, 4, 8, 8), T=10, window=4, delta=0.05, tol=1e-3, kind=B.PA_EPS_LINEAR,
            hidden=1024, patch=2, temb_dim=128, sched=None, flags=0, null_c=False, eta=0.0):
    lib = B.load_library()
    sh = (C.c_int32 * 4)(*shape)
    sc = sched or B.Schedule(B.PA_SCHED_SCALED_LINEAR, 0.00085, 0.012, 1000, 0, 1, None, None, eta)
    c = np.ones(max(T, 1), np.float32)
    w = {k: np.zeros(1, np.uint16) for k in ("w1", "wt", "w2", "w3")}
    em = B.EpsModel(kind, None if null_c else c.ctypes.data_as(C.POINTER(C.c_float)), patch,
                    hidden, temb_dim, *(w[k].ctypes.data_as(C.POINTER(C.c_uint16))
                                        for k in ("w1", "wt", "w2", "w3")))
    h = C.c_void_p(1234)
    rc = lib.paraanya_create(sh, T, C.byref(sc), window, delta, tol, C.byref(em), None, flags,
                             C.byref(h))
    return rc, h.value, lib.paraanya_last_error().decode()


@pytest.mark.parametrize("kw,frag", [
    (dict(shape=(0, 4, 8, 8)), "batch"),
    (dict(shape=(B.PA_MAX_BATCH + 1, 4, 8, 8)), "batch"),
    (dict(eta=-0.5), "eta"),
    (dict(eta=1.5), "eta"),
    (dict(eta=float("nan")), "eta"),
    (dict(shape=(1, 3, 3, 3)), "multiple of 4"),
    (dict(T=0, window=1), "T must"),
    (dict(T=B.PA_MAX_STEPS + 1, window=4), "T must"),
    (dict(window=0), "window"),
    (dict(window=11), "window"),
    (dict(T=300, window=257), "window"),
    (dict(delta=-0.1), "delta"),
    (dict(delta=float("nan")), "delta"),
    (dict(tol=-1.0), "tol"),
    (dict(tol=float("nan")), "tol"),
    (dict(flags=32), "flags"),
    (dict(flags=16), "flags"),
    (dict(null_c=True), "c is NULL"),
    (dict(kind=7), "kind"),
    (dict(kind=B.PA_EPS_PATCH_MLP, shape=(1, 4, 7, 8)), "even"),
    (dict(T=2000, window=4), "train_steps"),
])
def test_create_rejects_invalid_arguments(kw, frag):
    rc, h, msg = _create(**kw)
    assert rc == B.PA_ERR_INVALID_ARG, msg
    assert h is None
    assert frag in msg


@pytest.mark.parametrize("kw", [
    dict(kind=B.PA_EPS_PATCH_MLP, hidden=768),
    dict(kind=B.PA_EPS_PATCH_MLP, patch=4),
    dict(kind=B.PA_EPS_PATCH_MLP, temb_dim=64),
    dict(kind=B.PA_EPS_PATCH_MLP, shape=(1, 4, 10, 10)),   # 25 tokens: not a multiple of 128
    dict(kind=B.PA_EPS_PATCH_MLP, shape=(1, 4, 16, 16)),   # 64 tokens
    dict(kind=B.PA_EPS_PATCH_MLP, shape=(1, 3, 16, 16)),
])
def test_create_reports_unbuilt_shapes(kw):
    rc, h, msg = _create(**kw)
    assert rc == B.PA_ERR_UNSUPPORTED, msg
    assert h is None


def test_explicit_schedule_validation():
    ab = np.array([0.5, 0.7, 1.5], np.float64)       # > 1: invalid
    tv = np.array([10, 5], np.int32)
    sc = B.Schedule(B.PA_SCHED_EXPLICIT, 0, 0, 0, 0, 0, ab.ctypes.data_as(C.POINTER(C.c_double)),
                    tv.ctypes.data_as(C.POINTER(C.c_int32)), 0.0)
    rc, h, msg = _create(T=2, window=2, sched=sc)
    assert rc == B.PA_ERR_INVALID_ARG and "alpha_bar[2]" in msg


def test_explicit_schedule_must_not_decrease_with_noise():
    """With eta > 0 the noise scale needs ab_i <= ab_{i+1}: a decreasing explicit schedule is
    refused at create (with eta = 0 the DDIM step is defined for it)."""
    ab = np.array([0.5, 0.4, 1.0], np.float64)
    tv = np.array([10, 5], np.int32)
    sc = B.Schedule(B.PA_SCHED_EXPLICIT, 0, 0, 0, 0, 0, ab.ctypes.data_as(C.POINTER(C.c_double)),
                    tv.ctypes.data_as(C.POINTER(C.c_int32)), 1.0)
    rc, h, msg = _create(T=2, window=2, sched=sc)
    assert rc == B.PA_ERR_INVALID_ARG and h is None and "must not decrease" in msg


def test_null_handle_calls_fail_cleanly():
    lib = B.load_library()
    assert lib.paraanya_reset(None, None) == B.PA_ERR_INVALID_ARG
    assert lib.paraanya_sweep(None, None) == B.PA_ERR_INVALID_ARG
    assert lib.paraanya_sample(None, None, None) == B.PA_ERR_INVALID_ARG
    st = B.Stats()
    assert lib.paraanya_stats(None, C.byref(st)) == B.PA_ERR_INVALID_ARG
    assert lib.paraanya_stats_sample(None, 0, C.byref(st)) == B.PA_ERR_INVALID_ARG
    assert lib.paraanya_set_noise(None, None) == B.PA_ERR_INVALID_ARG
    assert lib.paraanya_set_revisit_threshold(None, 0.05) == B.PA_ERR_INVALID_ARG
    tr = B.SweepTrace()
    assert lib.paraanya_trace_sample(None, 0, 0, C.byref(tr)) == B.PA_ERR_INVALID_ARG
    assert lib.paraanya_read_state_sample(None, 0, 0, 1, None, None, None, None) == B.PA_ERR_INVALID_ARG
    lib.paraanya_destroy(None)   # NULL-safe


def test_struct_layouts_match_the_header(tmp_path):
    """The binding's ctypes structures have the sizes and field offsets of the header's C
    structs (compiled here with the host C compiler)."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no host C compiler")
    fields = {"pa_schedule_t": (B.Schedule, ["kind", "beta_start", "train_steps", "alpha_bar", "t_values", "eta"]),
              "pa_stats_t": (B.Stats, ["nfe", "sweeps", "window_start", "nonfinite", "revisits", "revisits_below"]),
              "pa_sweep_trace_t": (B.SweepTrace, ["s", "sweep", "dev", "resid", "miss_idx", "hit"]),
              "pa_eps_model_t": (B.EpsModel, ["kind", "c", "hidden", "w1", "w3"]),
              "pa_ktimes_t": (B.KTimes, ["launches", "eps_ms_total", "eps_latents", "solver_launches",
                                         "picard_ms_total", "slide_ms_total"]),
              "pa_parareal_stats_t": (B.PrStats, ["nfe", "hits", "requests", "iterations", "done", "nonfinite"]),
              "pa_request_trace_t": (B.RequestTrace, ["iteration", "phase", "t", "block", "hit", "dev"])}
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "paraanya.h"', "int main(void) {"]
    for st, (_, fs) in fields.items():
        lines.append(f'printf("%zu\\n", sizeof({st}));')
        lines += [f'printf("%zu\\n", offsetof({st}, {f}));' for f in fs]
    lines.append("return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run([cc, "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)], check=True)
    vals = [int(v) for v in subprocess.run([str(exe)], check=True, capture_output=True,
                                           text=True).stdout.split()]
    it = iter(vals)
    for st, (cls, fs) in fields.items():
        assert next(it) == C.sizeof(cls), st
        for f in fs:
            assert next(it) == getattr(cls, f).offset, f"{st}.{f}"


def _pr_create(shape=(1, 4, 8, 8), T=20, blocks=4, delta=0.05, tol=1e-3, eta=0.0, flags=0,
               kind=B.PA_EPS_LINEAR):
    lib = B.load_library()
    sh = (C.c_int32 * 4)(*shape)
    sc = B.Schedule(B.PA_SCHED_SCALED_LINEAR, 0.00085, 0.012, 1000, 0, 1, None, None, eta)
    c = np.ones(max(T, 1), np.float32)
    w = {k: np.zeros(1, np.uint16) for k in ("w1", "wt", "w2", "w3")}
    em = B.EpsModel(kind, c.ctypes.data_as(C.POINTER(C.c_float)), 2, 1024, 128,
                    *(w[k].ctypes.data_as(C.POINTER(C.c_uint16)) for k in ("w1", "wt", "w2", "w3")))
    h = C.c_void_p(1234)
    rc = lib.paraanya_parareal_create(sh, T, C.byref(sc), blocks, delta, tol, C.byref(em), None,
                                      flags, C.byref(h))
    return rc, h.value, lib.paraanya_last_error().decode()


@pytest.mark.parametrize("kw,code,frag", [
    (dict(shape=(2, 4, 8, 8)), B.PA_ERR_INVALID_ARG, "batch"),
    (dict(blocks=3), B.PA_ERR_INVALID_ARG, "blocks"),
    (dict(blocks=0), B.PA_ERR_INVALID_ARG, "blocks"),
    (dict(T=B.PA_MAX_STEPS + 1, blocks=1), B.PA_ERR_INVALID_ARG, "T must"),
    (dict(T=130, blocks=65), B.PA_ERR_INVALID_ARG, "blocks"),
    (dict(delta=-1.0), B.PA_ERR_INVALID_ARG, "delta"),
    (dict(tol=float("nan")), B.PA_ERR_INVALID_ARG, "tol"),
    (dict(flags=4), B.PA_ERR_INVALID_ARG, "flags"),
    (dict(eta=1.0), B.PA_ERR_UNSUPPORTED, "eta"),
    (dict(kind=B.PA_EPS_PATCH_MLP, shape=(1, 4, 16, 16)), B.PA_ERR_UNSUPPORTED, "token"),
])
def test_parareal_create_rejects(kw, code, frag):
    rc, h, msg = _pr_create(**kw)
    assert rc == code, msg
    assert h is None and frag in msg


def test_parareal_null_handle_calls_fail_cleanly():
    lib = B.load_library()
    assert lib.paraanya_parareal_sample(None, None, None) == B.PA_ERR_INVALID_ARG
    st = B.PrStats()
    assert lib.paraanya_parareal_stats(None, C.byref(st)) == B.PA_ERR_INVALID_ARG
    r = B.RequestTrace()
    assert lib.paraanya_parareal_trace(None, 0, C.byref(r), None) == B.PA_ERR_INVALID_ARG
    assert lib.paraanya_parareal_residuals(None, 0, None) == B.PA_ERR_INVALID_ARG
    assert lib.paraanya_parareal_read_boundaries(None, None) == B.PA_ERR_INVALID_ARG
    lib.paraanya_parareal_destroy(None)


@pytest.mark.parametrize("kw,code,frag", [
    (dict(T=1025), B.PA_ERR_INVALID_ARG, "at most 1024"),
    (dict(eta=0.5), B.PA_ERR_UNSUPPORTED, "eta"),
    (dict(window=0), B.PA_ERR_INVALID_ARG, "window"),
    (dict(null_x=True), B.PA_ERR_INVALID_ARG, "NULL"),
])
def test_noalloc_rejects_before_any_hip_call(kw, code, frag):
    """The allocation-free entry point checks its arguments and limits before any HIP call."""
    lib = B.load_library()
    T = kw.get("T", 10)
    sh = (C.c_int32 * 4)(1, 4, 8, 8)
    sc = B.Schedule(B.PA_SCHED_SCALED_LINEAR, 0.00085, 0.012, 1000 if T <= 1000 else 2000, 0, 1, None, None,
                    kw.get("eta", 0.0))
    c = np.ones(T, np.float32)
    em = B.EpsModel(B.PA_EPS_LINEAR, c.ctypes.data_as(C.POINTER(C.c_float)), 0, 0, 0, None, None, None, None)
    x = None if kw.get("null_x") else C.c_void_p(16)
    st = B.Stats()
    rc = lib.paraanya_sample_noalloc(sh, T, C.byref(sc), kw.get("window", 4), 0.05, 1e-3, C.byref(em), None,
                                     x, C.c_void_p(16), C.byref(st))
    assert rc == code, (rc, lib.paraanya_last_error())
    assert frag in lib.paraanya_last_error().decode()
