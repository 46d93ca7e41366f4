"""ctypes binding of libparaanya.so (the C ABI in include/paraanya.h).

Argument marshalling only: every step of a sweep runs in the library's HIP kernels.
PyTorch provides device memory (fp32 CUDA tensors) and the stream handle. There is no
fallback: if the library is missing or cannot be loaded, :func:`load_library` raises.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libparaanya.so")

PA_OK = 0
PA_ERR_INVALID_ARG = -1
PA_ERR_HIP = -2
PA_ERR_OOM = -3
PA_ERR_STATE = -4
PA_ERR_NONFINITE = -5
PA_ERR_UNSUPPORTED = -6
PA_MAX_WINDOW = 256
PA_MAX_BATCH = 64
PA_MAX_STEPS = 1 << 20
PA_PR_MAX_BLOCKS = 64

PA_SCHED_SCALED_LINEAR = 0
PA_SCHED_EXPLICIT = 1
PA_SPACING_TRAILING = 0
PA_EPS_LINEAR = 0
PA_EPS_PATCH_MLP = 1
PA_FLAG_TRACE = 1
PA_FLAG_PROFILE = 2
PA_FLAG_PROFILE_SOLVER = 4
PA_FLAG_SPLIT_OUTPUTS = 8

EXPORTED = ("paraanya_create", "paraanya_reset", "paraanya_sweep", "paraanya_sample",
            "paraanya_stats", "paraanya_trace", "paraanya_read_state", "paraanya_coefficients",
            "paraanya_kernel_times", "paraanya_destroy", "paraanya_last_error",
            "paraanya_status_str", "paraanya_set_noise", "paraanya_set_revisit_threshold",
            "paraanya_stats_sample", "paraanya_trace_sample", "paraanya_read_state_sample",
            "paraanya_parareal_create", "paraanya_parareal_sample", "paraanya_parareal_stats",
            "paraanya_parareal_trace", "paraanya_parareal_residuals",
            "paraanya_parareal_read_boundaries", "paraanya_parareal_kernel_times",
            "paraanya_parareal_destroy", "paraanya_sample_noalloc")
PA_NOALLOC_WORKSPACE_BYTES = 64 << 20
PA_NOALLOC_MAX_STEPS = 1024


class Schedule(C.Structure):
    _fields_ = [("kind", C.c_int32), ("beta_start", C.c_double), ("beta_end", C.c_double),
                ("train_steps", C.c_int32), ("spacing", C.c_int32),
                ("final_alpha_one", C.c_int32), ("alpha_bar", C.POINTER(C.c_double)),
                ("t_values", C.POINTER(C.c_int32)), ("eta", C.c_double)]


class EpsModel(C.Structure):
    _fields_ = [("kind", C.c_int32), ("c", C.POINTER(C.c_float)), ("patch", C.c_int32),
                ("hidden", C.c_int32), ("temb_dim", C.c_int32),
                ("w1", C.POINTER(C.c_uint16)), ("wt", C.POINTER(C.c_uint16)),
                ("w2", C.POINTER(C.c_uint16)), ("w3", C.POINTER(C.c_uint16))]


class Stats(C.Structure):
    _fields_ = [("nfe", C.c_int64), ("hits", C.c_int64), ("misses", C.c_int64),
                ("sweeps", C.c_int64), ("window_start", C.c_int32), ("window_end", C.c_int32),
                ("done", C.c_int32), ("nonfinite", C.c_int32),
                ("revisits", C.c_int64), ("revisits_below", C.c_int64)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class SweepTrace(C.Structure):
    _fields_ = [("s", C.c_int32), ("e", C.c_int32), ("m", C.c_int32), ("c", C.c_int32),
                ("s_next", C.c_int32), ("sweep", C.c_int32),
                ("dev", C.c_double * PA_MAX_WINDOW), ("resid", C.c_double * PA_MAX_WINDOW),
                ("miss_idx", C.c_int32 * PA_MAX_WINDOW), ("hit", C.c_uint8 * PA_MAX_WINDOW)]

    def as_dict(self):
        W = self.e - self.s
        return {"s": self.s, "e": self.e, "m": self.m, "c": self.c, "s_next": self.s_next,
                "sweep": self.sweep,
                "dev": np.frombuffer(self.dev, dtype=np.float64, count=W).copy(),
                "hit": np.frombuffer(self.hit, dtype=np.uint8, count=W).astype(bool),
                "miss": list(np.frombuffer(self.miss_idx, dtype=np.int32, count=self.m)),
                "r": np.frombuffer(self.resid, dtype=np.float64, count=W).copy()}


class KTimes(C.Structure):
    _fields_ = [("launches", C.c_int64), ("eps_ms_total", C.c_double),
                ("eps_latents", C.c_int64), ("solver_launches", C.c_int64),
                ("picard_ms_total", C.c_double), ("slide_ms_total", C.c_double)]


class PrStats(C.Structure):
    _fields_ = [("nfe", C.c_int64), ("hits", C.c_int64), ("requests", C.c_int64),
                ("iterations", C.c_int32), ("done", C.c_int32), ("nonfinite", C.c_int32),
                ("pad", C.c_int32)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_ if k != "pad"}


class RequestTrace(C.Structure):
    _fields_ = [("iteration", C.c_int32), ("phase", C.c_int32), ("t", C.c_int32),
                ("block", C.c_int32), ("hit", C.c_int32), ("pad", C.c_int32),
                ("dev", C.c_double)]


_LIB = None


def load_library(path: str = LIB_PATH):
    """Load the built library (raises if it is missing: there is no fallback path)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2609_36522_amd.build`")
    lib = C.CDLL(path)
    P, I32, F64, V = C.c_void_p, C.c_int32, C.c_double, C.c_void_p
    lib.paraanya_create.argtypes = [C.POINTER(C.c_int32), I32, C.POINTER(Schedule), I32, F64, F64,
                                    C.POINTER(EpsModel), V, C.c_uint32, C.POINTER(P)]
    lib.paraanya_reset.argtypes = [P, P]
    lib.paraanya_sweep.argtypes = [P, C.POINTER(I32)]
    lib.paraanya_sample.argtypes = [P, P, P]
    lib.paraanya_stats.argtypes = [P, C.POINTER(Stats)]
    lib.paraanya_stats_sample.argtypes = [P, I32, C.POINTER(Stats)]
    lib.paraanya_trace.argtypes = [P, I32, C.POINTER(SweepTrace)]
    lib.paraanya_trace_sample.argtypes = [P, I32, I32, C.POINTER(SweepTrace)]
    lib.paraanya_read_state.argtypes = [P, I32, I32, P, P, P, P]
    lib.paraanya_read_state_sample.argtypes = [P, I32, I32, I32, P, P, P, P]
    lib.paraanya_coefficients.argtypes = [P, P, P, P, P]
    lib.paraanya_set_noise.argtypes = [P, P]
    lib.paraanya_set_revisit_threshold.argtypes = [P, F64]
    lib.paraanya_kernel_times.argtypes = [P, C.POINTER(KTimes)]
    lib.paraanya_destroy.argtypes = [P]
    lib.paraanya_destroy.restype = None
    lib.paraanya_parareal_create.argtypes = [C.POINTER(C.c_int32), I32, C.POINTER(Schedule), I32, F64,
                                             F64, C.POINTER(EpsModel), V, C.c_uint32, C.POINTER(P)]
    lib.paraanya_parareal_sample.argtypes = [P, P, P]
    lib.paraanya_parareal_stats.argtypes = [P, C.POINTER(PrStats)]
    lib.paraanya_parareal_trace.argtypes = [P, I32, C.POINTER(RequestTrace), P]
    lib.paraanya_parareal_residuals.argtypes = [P, I32, P]
    lib.paraanya_parareal_read_boundaries.argtypes = [P, P]
    lib.paraanya_parareal_kernel_times.argtypes = [P, C.POINTER(KTimes)]
    lib.paraanya_parareal_destroy.argtypes = [P]
    lib.paraanya_parareal_destroy.restype = None
    lib.paraanya_sample_noalloc.argtypes = [C.POINTER(C.c_int32), I32, C.POINTER(Schedule), I32, F64, F64,
                                            C.POINTER(EpsModel), V, P, P, C.POINTER(Stats)]
    lib.paraanya_last_error.restype = C.c_char_p
    lib.paraanya_status_str.argtypes = [C.c_int]
    lib.paraanya_status_str.restype = C.c_char_p
    for name in EXPORTED:
        if name not in ("paraanya_destroy", "paraanya_last_error", "paraanya_status_str",
                        "paraanya_parareal_destroy"):
            getattr(lib, name).restype = C.c_int
    _LIB = lib
    return lib


class PAError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{status_str(code)}: {msg}")
        self.code = code


def status_str(code: int) -> str:
    return load_library().paraanya_status_str(code).decode()


def _check(rc: int):
    if rc != PA_OK:
        raise PAError(rc, load_library().paraanya_last_error().decode())


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(C.POINTER(ctype))


def _schedule_and_model(keep, schedule, eta, model, c, weights, hidden):
    """ctypes Schedule and EpsModel; arrays they point to are appended to ``keep``."""
    if schedule is None:
        sc = Schedule(PA_SCHED_SCALED_LINEAR, 0.00085, 0.012, 1000, PA_SPACING_TRAILING, 1,
                      None, None, float(eta))
    else:
        ab = np.ascontiguousarray(schedule["alpha_bar"], dtype=np.float64)
        tv = np.ascontiguousarray(schedule["t_values"], dtype=np.int32)
        keep += [ab, tv]
        sc = Schedule(PA_SCHED_EXPLICIT, 0.0, 0.0, 0, 0, 0, _ptr(ab, C.c_double),
                      _ptr(tv, C.c_int32), float(eta))
    if model == "linear":
        cc = np.ascontiguousarray(c, dtype=np.float32)
        keep.append(cc)
        em = EpsModel(PA_EPS_LINEAR, _ptr(cc, C.c_float), 0, 0, 0, None, None, None, None)
    elif model == "patch_mlp":
        ws = {k: np.ascontiguousarray(weights[k], dtype=np.uint16) for k in ("w1", "wt", "w2", "w3")}
        keep.append(ws)
        em = EpsModel(PA_EPS_PATCH_MLP, None, 2, int(hidden), int(ws["wt"].shape[0]),
                      _ptr(ws["w1"], C.c_uint16), _ptr(ws["wt"], C.c_uint16),
                      _ptr(ws["w2"], C.c_uint16), _ptr(ws["w3"], C.c_uint16))
    else:
        raise ValueError(f"unknown model {model!r}")
    return sc, em


class Sampler:
    """One handle of the cached Picard sampler.

    ``model`` is "linear" (needs ``c``) or "patch_mlp" (needs ``weights`` as a dict of bf16
    bit-pattern arrays w1, wt, w2, w3). ``batch`` independent samples share the handle
    (tensors passed to reset/sample hold batch x D values). ``eta`` > 0 selects the
    stochastic step (1 = ancestral DDPM); its step noise is given with :meth:`set_noise`.
    ``stream`` is a torch.cuda.Stream or None (the current stream). ``split_outputs`` (test
    hook) keeps the network's outputs split over its partial buffers on every launch."""

    def __init__(self, latent, T, window, delta, tol, model, *, c=None, weights=None,
                 hidden=0, schedule=None, stream=None, trace=False, profile=False, batch=1,
                 eta=0.0, profile_solver=False, split_outputs=False):
        import torch
        self.lib = load_library()
        self.latent = tuple(int(v) for v in latent)
        self.T, self.P = int(T), int(window)
        self.D = int(np.prod(self.latent))
        self.N = int(batch)
        self.torch = torch
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        shape = (C.c_int32 * 4)(self.N, *self.latent)
        self._keep = []
        sc, em = _schedule_and_model(self._keep, schedule, eta, model, c, weights, hidden)
        flags = (PA_FLAG_TRACE if trace else 0) | (PA_FLAG_PROFILE if profile else 0) | \
            (PA_FLAG_PROFILE | PA_FLAG_PROFILE_SOLVER if profile_solver else 0) | \
            (PA_FLAG_SPLIT_OUTPUTS if split_outputs else 0)
        h = C.c_void_p()
        _check(self.lib.paraanya_create(shape, self.T, C.byref(sc), self.P, float(delta),
                                        float(tol), C.byref(em), C.c_void_p(self.stream.cuda_stream),
                                        flags, C.byref(h)))
        self.h = h
        self.model = model
        self.hidden = int(hidden)

    # ------------------------------------------------------------------ lifetime
    def close(self):
        if getattr(self, "h", None):
            self.lib.paraanya_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    # ------------------------------------------------------------------ sampling
    def _dev(self, x, count=None):
        t = self.torch
        count = self.N * self.D if count is None else count
        if not (isinstance(x, t.Tensor) and x.is_cuda and x.dtype == t.float32 and x.is_contiguous()
                and x.numel() == count):
            raise ValueError(f"expected a contiguous fp32 CUDA tensor of {count} elements")
        return C.c_void_p(x.data_ptr())

    def reset(self, x_init):
        _check(self.lib.paraanya_reset(self.h, self._dev(x_init)))

    def set_noise(self, z):
        """Step noise z[n][i][D] (fp32 CUDA tensor) of the stochastic step (eta > 0)."""
        _check(self.lib.paraanya_set_noise(self.h, self._dev(z, self.N * self.T * self.D)))

    def set_revisit_threshold(self, threshold: float):
        _check(self.lib.paraanya_set_revisit_threshold(self.h, float(threshold)))

    def sweep(self, sync: bool = False):
        if not sync:
            _check(self.lib.paraanya_sweep(self.h, None))
            return None
        done = C.c_int32(0)
        _check(self.lib.paraanya_sweep(self.h, C.byref(done)))
        return bool(done.value)

    def sample(self, x_init, x_out=None):
        """paraanya_sample: returns once every sample is done; x_out is written by work queued
        on the handle's stream (torch operations on that stream see it)."""
        if x_out is None:
            x_out = self.torch.empty_like(x_init)
        _check(self.lib.paraanya_sample(self.h, self._dev(x_init), self._dev(x_out)))
        return x_out

    # ------------------------------------------------------------------ inspection
    def stats(self, n=None) -> dict:
        """Counters aggregated over the samples, or of sample ``n``."""
        st = Stats()
        if n is None:
            _check(self.lib.paraanya_stats(self.h, C.byref(st)))
        else:
            _check(self.lib.paraanya_stats_sample(self.h, int(n), C.byref(st)))
        return st.as_dict()

    def trace(self, k: int, n: int = 0) -> dict:
        tr = SweepTrace()
        _check(self.lib.paraanya_trace_sample(self.h, int(n), int(k), C.byref(tr)))
        return tr.as_dict()

    def traces(self, n: int = 0) -> list:
        return [self.trace(k, n) for k in range(self.stats(n)["sweeps"])]

    def read_state(self, t0: int = 0, t1=None, n: int = 0):
        """Host copies of sample n's X[t0:t1], Xh/Eh/valid[t0:min(t1, T)]."""
        t1 = self.T + 1 if t1 is None else int(t1)
        c1 = min(t1, self.T)
        X = np.empty((t1 - t0, self.D), np.float32)
        Xh = np.empty((max(c1 - t0, 0), self.D), np.float32)
        Eh = np.empty_like(Xh)
        valid = np.empty(max(c1 - t0, 0), np.uint8)
        _check(self.lib.paraanya_read_state_sample(self.h, int(n), int(t0), int(t1), X.ctypes.data_as(C.c_void_p),
                                            Xh.ctypes.data_as(C.c_void_p), Eh.ctypes.data_as(C.c_void_p),
                                            valid.ctypes.data_as(C.c_void_p)))
        return X, Xh, Eh, valid.astype(bool)

    def coefficients(self):
        """(alpha, b, sigma, temb) as the device uses them (temb None for the linear model)."""
        a = np.empty(self.T, np.float64)
        b = np.empty(self.T, np.float64)
        sg = np.empty(self.T, np.float64)
        temb = np.empty((self.T, self.hidden), np.float32) if self.model == "patch_mlp" else None
        _check(self.lib.paraanya_coefficients(self.h, a.ctypes.data_as(C.c_void_p),
                                              b.ctypes.data_as(C.c_void_p),
                                              sg.ctypes.data_as(C.c_void_p),
                                              None if temb is None else temb.ctypes.data_as(C.c_void_p)))
        return a, b, sg, temb

    def kernel_times(self) -> dict:
        kt = KTimes()
        _check(self.lib.paraanya_kernel_times(self.h, C.byref(kt)))
        return {"launches": kt.launches, "eps_ms_total": kt.eps_ms_total,
                "eps_latents": kt.eps_latents, "solver_launches": kt.solver_launches,
                "picard_ms_total": kt.picard_ms_total, "slide_ms_total": kt.slide_ms_total}


def from_workload(wl, delta=None, *, seed_weights=None, **kw) -> "Sampler":
    """Sampler for a :class:`~paper_2609_36522_amd.workloads.Workload` with its seeded inputs."""
    from . import inputs
    d = wl.delta if delta is None else delta
    if wl.model == "linear":
        return Sampler(wl.latent, wl.T, wl.window, d, wl.tol, "linear",
                       c=inputs.linear_coefficients(wl.T), **kw)
    w = inputs.mlp_weights(wl.hidden, temb_dim=wl.temb_dim) if seed_weights is None else seed_weights
    return Sampler(wl.latent, wl.T, wl.window, d, wl.tol, "patch_mlp", weights=w,
                   hidden=wl.hidden, **kw)



def sample_noalloc(latent, T, window, delta, tol, model, x_init, x_out=None, *, c=None, weights=None,
                   hidden=0, schedule=None, stream=None, batch=1):
    """paraanya_sample_noalloc: one sample with every device buffer in the library's static
    workspace (no allocation by the library). ``x_init`` (and ``x_out``, allocated here by torch
    when None) are contiguous fp32 CUDA tensors of batch x D values. Returns (x_out, stats)."""
    import torch
    lib = load_library()
    latent = tuple(int(v) for v in latent)
    D = int(np.prod(latent))
    st = stream if stream is not None else torch.cuda.current_stream()
    for t in (x_init,) + (() if x_out is None else (x_out,)):
        if not (isinstance(t, torch.Tensor) and t.is_cuda and t.dtype == torch.float32 and t.is_contiguous()
                and t.numel() == batch * D):
            raise ValueError(f"expected a contiguous fp32 CUDA tensor of {batch * D} elements")
    if x_out is None:
        x_out = torch.empty_like(x_init)
    keep = []
    sc, em = _schedule_and_model(keep, schedule, 0.0, model, c, weights, hidden)
    shape = (C.c_int32 * 4)(int(batch), *latent)
    out = Stats()
    _check(lib.paraanya_sample_noalloc(shape, int(T), C.byref(sc), int(window), float(delta), float(tol),
                                       C.byref(em), C.c_void_p(st.cuda_stream), C.c_void_p(x_init.data_ptr()),
                                       C.c_void_p(x_out.data_ptr()), C.byref(out)))
    return x_out, out.as_dict()


def sample_noalloc_workload(wl, x_init, x_out=None, delta=None, *, seed_weights=None, **kw):
    """sample_noalloc for a :class:`~paper_2609_36522_amd.workloads.Workload` with its seeded inputs."""
    from . import inputs
    d = wl.delta if delta is None else delta
    if wl.model == "linear":
        return sample_noalloc(wl.latent, wl.T, wl.window, d, wl.tol, "linear", x_init, x_out,
                              c=inputs.linear_coefficients(wl.T), **kw)
    w = inputs.mlp_weights(wl.hidden, temb_dim=wl.temb_dim) if seed_weights is None else seed_weights
    return sample_noalloc(wl.latent, wl.T, wl.window, d, wl.tol, "patch_mlp", x_init, x_out, weights=w,
                          hidden=wl.hidden, **kw)


class Parareal:
    """One handle of the cached Parareal sampler (T steps in ``blocks`` blocks)."""

    def __init__(self, latent, T, blocks, delta, tol, model, *, c=None, weights=None, hidden=0,
                 schedule=None, stream=None, trace=False, profile=False):
        import torch
        self.lib = load_library()
        self.latent = tuple(int(v) for v in latent)
        self.T, self.B = int(T), int(blocks)
        self.D = int(np.prod(self.latent))
        self.torch = torch
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        self._keep = []
        sc, em = _schedule_and_model(self._keep, schedule, 0.0, model, c, weights, hidden)
        shape = (C.c_int32 * 4)(1, *self.latent)
        flags = (PA_FLAG_TRACE if trace else 0) | (PA_FLAG_PROFILE if profile else 0)
        h = C.c_void_p()
        _check(self.lib.paraanya_parareal_create(shape, self.T, C.byref(sc), self.B, float(delta),
                                                 float(tol), C.byref(em),
                                                 C.c_void_p(self.stream.cuda_stream), flags, C.byref(h)))
        self.h = h

    def close(self):
        if getattr(self, "h", None):
            self.lib.paraanya_parareal_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def _dev(self, x):
        t = self.torch
        if not (isinstance(x, t.Tensor) and x.is_cuda and x.dtype == t.float32 and x.is_contiguous()
                and x.numel() == self.D):
            raise ValueError(f"expected a contiguous fp32 CUDA tensor of {self.D} elements")
        return C.c_void_p(x.data_ptr())

    def sample(self, x_init, x_out=None):
        if x_out is None:
            x_out = self.torch.empty_like(x_init)
        _check(self.lib.paraanya_parareal_sample(self.h, self._dev(x_init), self._dev(x_out)))
        return x_out

    def stats(self) -> dict:
        st = PrStats()
        _check(self.lib.paraanya_parareal_stats(self.h, C.byref(st)))
        return st.as_dict()

    def trace(self, i: int, with_eps: bool = False):
        """(record dict, fresh output or None) of request i of the last sample."""
        r = RequestTrace()
        eps = np.empty(self.D, np.float32) if with_eps else None
        _check(self.lib.paraanya_parareal_trace(self.h, int(i), C.byref(r),
                                                None if eps is None else eps.ctypes.data_as(C.c_void_p)))
        rec = {"iteration": r.iteration, "phase": r.phase, "t": r.t, "block": r.block,
               "hit": bool(r.hit), "dev": r.dev}
        return rec, (eps if (with_eps and not r.hit) else None)

    def residuals(self, k: int) -> np.ndarray:
        r = np.empty(self.B + 1, np.float64)
        _check(self.lib.paraanya_parareal_residuals(self.h, int(k), r.ctypes.data_as(C.c_void_p)))
        return r

    def boundaries(self) -> np.ndarray:
        U = np.empty((self.B + 1, self.D), np.float32)
        _check(self.lib.paraanya_parareal_read_boundaries(self.h, U.ctypes.data_as(C.c_void_p)))
        return U

    def kernel_times(self) -> dict:
        kt = KTimes()
        _check(self.lib.paraanya_parareal_kernel_times(self.h, C.byref(kt)))
        return {"launches": kt.launches, "eps_ms_total": kt.eps_ms_total,
                "eps_latents": kt.eps_latents}


def parareal_from_workload(wl, delta=None, *, seed_weights=None, **kw) -> "Parareal":
    """Parareal handle for a workload with ``wl.blocks`` blocks and its seeded inputs."""
    from . import inputs
    d = wl.delta if delta is None else delta
    if wl.model == "linear":
        return Parareal(wl.latent, wl.T, wl.blocks, d, wl.tol, "linear",
                        c=inputs.linear_coefficients(wl.T), **kw)
    w = inputs.mlp_weights(wl.hidden, temb_dim=wl.temb_dim) if seed_weights is None else seed_weights
    return Parareal(wl.latent, wl.T, wl.blocks, d, wl.tol, "patch_mlp", weights=w,
                    hidden=wl.hidden, **kw)
