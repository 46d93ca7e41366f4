"""GPU-vs-oracle parity harness (used by the -m gpu tests; needs the built library).

Two checks per workload, both through the C ABI (binding.Sampler):

* step-locked: before every device sweep the harness reads the device state (window rows of
  X, Xh, Eh, valid); the oracle then runs the same sweep on that state and the harness
  compares the decisions (deviation, hit mask, miss list, residuals, slide) and the updated
  rows. For the patch-MLP the oracle consumes the device's fresh outputs for the misses
  ("eps-locked"), and those outputs are checked separately against the oracle network.
* follow: the oracle runs its own trajectory from the same initial latent (fully independent
  for the linear network; eps-locked for the patch-MLP), advanced sweep by sweep beside the
  device run, and must reproduce every decision and the final latent within 1e-4 x RMS.

Decision rule: the device decides in fp32, the oracle in fp64. A decision may differ only if
the oracle's deviation lies within BAND (relative) of delta, or the deciding residual within
BAND of tau; such flips are logged and the oracle adopts the device's decision.
"""
from __future__ import annotations

import numpy as np

from oracle import eps_models as em
from oracle import sampler as sp
from oracle import schedule as sch
from paper_2609_36522_amd import binding, inputs

# Tolerances, derived from the arithmetic:
# both sides form the drift, the Picard sum, the deviations and the residuals in fp64 from
# the same fp32 inputs; they differ only in the association of fp64 sums (~1e-16 relative),
# so an updated fp32 state can differ by at most one fp32 ulp (a rounding tie), and a
# deviation or residual by a few fp64 ulps of the sum.
BAND = 1e-6                 # relative decision band around delta and tau (logged, not failed)
STATE_ULPS = 1              # per-sweep updated states, in fp32 ulps of the oracle value
# At most max(1, STATE_FRAC x n) of the n state elements a sweep updates may differ at all. A
# tie needs the fp64 sum within a few fp64 ulps of an fp32 rounding midpoint: 10 of the 1.24e9
# updated elements checked over 1000 random configurations differed (8e-9); one tie in a
# sweep of a tiny latent (80 elements, 51 states) is that event, while a systematic change of
# the arithmetic (an fp32 partial sum, a dropped term) moves many elements at once.
STATE_FRAC = 1e-4
FINAL_RTOL = 1e-4           # final latent, max-abs x RMS
SUM_RTOL = 1e-11            # deviations/residuals: fp64 sums in different orders
# Fresh network outputs: max-abs error <= EPS_RTOL x the larger of the output's RMS over the
# latent and the largest magnitude among the 16 outputs of the same token (eps_error). Both
# sides round every activation to bf16; the device accumulates in fp32, the oracle in fp64, so
# an activation near a bf16 rounding boundary can round differently, and its step (half a bf16
# ulp, proportional to the activation) moves that token's outputs by an amount proportional to
# the token's own scale. Seen on the device: one token of a late state (latent RMS 12) with
# activations up to 79 (bf16 step 0.5) deviated by 1.01e-2 x the latent RMS, 2.3e-3 x its own
# output scale; a CPU evaluation of the same latent with fp32 accumulation and the exact erf
# GELU deviates from the oracle by the same 1.01e-2 there, so the deviation is the arithmetic's.
EPS_RTOL = 1e-2
REVISIT_THR = 0.05          # default threshold of the device's revisit counters
# An oracle trajectory of its own (follow) stores its own fp32 states, which may differ from
# the device's by a rounding in a few elements, then by what the dynamics make of it. For
# every cached slot the harness measures, before the sweep, a = mean |x_o - x_d| +
# mean |x^_o - x^_d| over the D entries; by the triangle inequality the two Eq. (4)
# deviations, means of |x - x^|, differ by at most a, plus the fp64 sum order (SUM_RTOL).


def coefficients(T, eta=0.0):
    ab, t = sch.sampler_alpha_bar(T)
    alpha, b, sigma = sch.step_coefficients(ab, eta)
    return ab, t, alpha, b, sigma


def oracle_network(wl, t_values):
    if wl.model == "linear":
        return em.linear_eps(inputs.linear_coefficients(wl.T))
    return em.PatchMLP(inputs.mlp_weights(wl.hidden, temb_dim=wl.temb_dim), t_values, wl.latent)


def rms(a) -> float:
    a = np.asarray(a, dtype=np.float64)
    return float(np.sqrt(np.mean(a * a))) if a.size else 0.0


def eps_error(got, ref, shape) -> float:
    """Largest |got - ref| of a network output (flat [D]) relative to max(RMS of ref, the
    largest |ref| among the outputs of the same token): the quantity EPS_RTOL bounds."""
    ref = np.asarray(ref, np.float64).reshape(shape)
    d = np.abs(np.asarray(got, np.float64).reshape(shape) - ref)
    scale = np.maximum(np.abs(em.patchify(ref, 2)).max(axis=1), max(rms(ref), 1e-30))
    return float((em.patchify(d, 2).max(axis=1) / scale).max())


class Log:
    def __init__(self):
        self.flips = []

    def flip(self, kind, sweep, slot, value, threshold):
        self.flips.append((kind, sweep, slot, float(value), float(threshold)))


def _in_band(v, thr, extra=0.0) -> bool:
    """v within BAND (relative) of the threshold, widened by ``extra`` (follow: how far the
    two sides' states can move v)."""
    return abs(v - thr) <= BAND * max(abs(thr), 1e-30) + extra


def _check_hits(k, dev_o, gpu, delta, log, allow=None):
    """Compare the oracle's deviations/hits (fp64) with the device's; returns the mask to use.
    ``allow`` (follow only): per window slot, how far the two sides' states can move the
    deviation (mean |x_o - x_d| + mean |x^_o - x^_d|); step-locked, both hold the same states."""
    W = len(dev_o)
    assert gpu["e"] - gpu["s"] == W
    dev_g = gpu["dev"]
    assert np.array_equal(np.isnan(dev_o), np.isnan(dev_g)), f"sweep {k}: first-entry slots differ"
    ok = ~np.isnan(dev_o)
    if ok.any():
        err = np.abs(dev_g[ok] - dev_o[ok])
        bound = SUM_RTOL * np.maximum(dev_o[ok], dev_g[ok])
        if allow is not None:
            bound = bound + (1.0 + SUM_RTOL) * allow[ok]
        j = int(np.argmax(err - bound))
        assert np.all(err <= bound + 1e-300), \
            f"sweep {k}: deviation mismatch {err[j]!r} (oracle {dev_o[ok][j]!r}, bound {bound[j]!r})"
    hit_o = ok & (np.nan_to_num(dev_o, nan=np.inf) < delta)
    hit_g = gpu["hit"]
    for j in np.nonzero(hit_o != hit_g)[0]:
        extra = 0.0 if allow is None else (1.0 + SUM_RTOL) * allow[j]
        assert _in_band(dev_o[j], delta, extra), f"sweep {k} slot {j}: hit decision differs outside the band " \
                                          f"(dev {dev_o[j]!r}, delta {delta!r})"
        log.flip("hit", k, int(j), dev_o[j], delta)
    return hit_g.copy()


def _check_slide(k, r_o, gpu, tau, log, state_err=0.0):
    """Residuals: fp64 sums of the same squares, plus the effect of state differences e
    (|r' - r| <= 2 sqrt(r) max|e| + max|e|^2)."""
    W = len(r_o)
    r_g = gpu["r"].astype(np.float64)
    tol = SUM_RTOL * np.abs(r_o) + 2.0 * np.sqrt(np.abs(r_o)) * state_err + state_err ** 2 + 1e-300
    assert np.all(np.abs(r_g - r_o) <= tol), f"sweep {k}: residual mismatch {np.max(np.abs(r_g - r_o) - tol)}"
    c_o = sp.leading_converged(r_o, tau)
    if c_o != gpu["c"]:
        j = min(c_o, gpu["c"])
        assert j < W - 1 and _in_band(r_o[j], tau), f"sweep {k}: slide differs outside the band"
        log.flip("tau", k, j, r_o[j], tau)
    assert gpu["s_next"] == gpu["s"] + 1 + gpu["c"]


class Run:
    """A device run driven sweep by sweep with the step-locked check after each sweep.

    ``batch`` > 1 drives one handle with that many samples (initial latents from
    inputs.x_init_batch) and checks every sample that is still running after each batched
    sweep. ``eta`` > 0 runs the stochastic step with the seeded step noise."""

    def __init__(self, wl, delta, *, eps_stride=1, seed_x=inputs.SEED_X_INIT,
                 x_init=None, batch=1, eta=0.0):
        import torch
        self.wl, self.delta = wl, float(delta)
        self.T, self.P, self.D = wl.T, wl.window, wl.D
        self.N, self.eta = int(batch), float(eta)
        self.ab, self.t_values, self.alpha, self.b, self.sigma = coefficients(wl.T, self.eta)
        self.net = oracle_network(wl, self.t_values)
        if x_init is not None:
            xs = np.asarray(x_init, np.float32).reshape(self.N, self.D)
        elif self.N == 1:
            xs = inputs.x_init(wl.latent, seed_x).reshape(1, -1)
        else:
            xs = inputs.x_init_batch(wl.latent, self.N).reshape(self.N, -1)
        self.xs = xs
        self.x_init = xs[0]
        self.noise = None
        if self.eta > 0.0:
            self.Z = inputs.step_noise(self.N, self.T, self.D)
            self.noise = [sp.step_noise_terms(self.sigma, self.Z[n]) for n in range(self.N)]
        self.log = Log()
        self.records = [[] for _ in range(self.N)]    # device trace records per sample
        # follow: the oracle's own trajectory per sample, its decision log and trace
        self.fol = [sp.init_state(self.xs[n], self.T) for n in range(self.N)]
        self.follow_logs = [Log() for _ in range(self.N)]
        self.follow_traces = [[] for _ in range(self.N)]
        # Fresh network outputs checked one by one against the oracle network: every output
        # of the first sweep, then every eps_stride-th fresh output of the run (counted over
        # all samples in sweep order); eps_stride = 1 checks every output, 0 none.
        self.eps_stride = int(eps_stride)
        self.eps_err = []          # max-abs/RMS of every checked fresh output
        self._eps_seen = 0
        self.state_diffs = 0       # updated state elements that differ (by one ulp) at all
        self.sampler = binding.from_workload(wl, delta, trace=True, batch=self.N, eta=self.eta)
        self.torch = torch
        self.xd = torch.from_numpy(np.ascontiguousarray(xs, np.float32).reshape(-1)).cuda()
        if self.eta > 0.0:
            self.sampler.set_noise(torch.from_numpy(self.Z.reshape(-1)).cuda())

    def close(self):
        self.sampler.close()

    def run(self):
        s = self.sampler
        s.reset(self.xd)
        T, D, N = self.T, self.D, self.N
        ost = [sp.init_state(np.zeros(D, np.float32), T) for _ in range(N)]
        newest = [0] * N
        k = 0
        while True:
            active = [n for n in range(N) if not s.stats(n)["done"]]
            if not active:
                break
            pre = {}
            for n in active:
                st = s.stats(n)
                sw, e = st["window_start"], st["window_end"]
                Xg, Xhg, Ehg, vg = s.read_state(sw, max(newest[n], sw) + 1, n)
                o = ost[n]
                o.X[sw:sw + len(Xg)] = Xg
                c1 = min(max(newest[n], sw) + 1, T)
                o.Xh[sw:c1] = Xhg
                o.Eh[sw:c1] = Ehg
                o.valid[:] = False
                o.valid[sw:c1] = vg
                o.s, o.newest = sw, newest[n]
                pre[n] = (sw, e, self._follow_allowance(n, k, sw, e, Xg, Xhg, c1))
            s.sweep(sync=True)
            for n in active:
                sw, e, allow = pre[n]
                g, gpu_eps = self._check_sweep(n, k, sw, e, ost[n], newest[n])
                self._follow_sweep(n, k, g, gpu_eps, allow)
                newest[n] = max(newest[n], e)
            k += 1
            assert k <= T, "more sweeps than steps"
        self.stats = s.stats()
        self.stats_n = [s.stats(n) for n in range(N)]
        self.x_T_all = [s.read_state(T, T + 1, n)[0][0].copy() for n in range(N)]
        self.x_T = self.x_T_all[0]
        return self

    def _check_sweep(self, n, k, sw, e, ost, newest):
        s = self.sampler
        g = s.trace(k, n)
        assert (g["s"], g["e"]) == (sw, e), f"sample {n} sweep {k}: window mismatch"
        # device post-state of the window
        Xp, Xhp, Ehp, vp = s.read_state(sw, e + 1, n)
        gpu_eps = {t: Ehp[t - sw].copy() for t in g["miss"]}
        if self.wl.model == "linear":
            eps_fn = self.net
        else:
            def eps_fn(Xb, steps, _g=gpu_eps):
                assert list(steps) == list(_g.keys()), "miss lists differ"
                return np.stack([_g[t] for t in steps]).astype(Xb.dtype)
        noise = None if self.noise is None else self.noise[n]
        # oracle: same sweep on the device's pre-state
        sp.fill_new_states(ost.X, newest, e)
        dev_o, hit_o = sp.cache_test(ost.X, ost.Xh, ost.valid, sw, e, self.delta)
        hit = _check_hits(k, dev_o, g, self.delta, self.log)
        X_before = ost.X[sw:e + 1].copy()
        rec = sp.sweep(ost, self.P, self.delta, self.wl.tol, self.alpha, self.b, eps_fn,
                       force_hit=hit, noise=noise)
        assert rec["miss"] == g["miss"] and rec["m"] == g["m"], f"sample {n} sweep {k}: miss list"
        # updated states s+1..e: at most one fp32 ulp apart, rarely
        ref = ost.X[sw + 1:e + 1]
        diff = np.abs(Xp[1:].astype(np.float64) - ref.astype(np.float64))
        ulp = np.spacing(np.abs(ref)).astype(np.float64)
        assert np.all(diff <= STATE_ULPS * ulp), f"sample {n} sweep {k}: states differ by {np.max(diff / ulp):.3g} ulp"
        nd = int(np.count_nonzero(diff))
        assert nd <= max(1, STATE_FRAC * diff.size), f"sample {n} sweep {k}: {nd} of {diff.size} state elements differ"
        self.state_diffs += nd
        _check_slide(k, rec["r"], g, self.wl.tol, self.log, float(diff.max(initial=0.0)))
        # cache: inputs of the misses are the pre-update states, hits untouched
        for j in range(e - sw):
            t = sw + j
            if t in gpu_eps:
                assert np.array_equal(Xhp[j], X_before[j]), f"sample {n} sweep {k}: cached input of miss {t}"
                assert vp[j]
            else:
                assert np.array_equal(Xhp[j], ost.Xh[t]) and np.array_equal(Ehp[j], ost.Eh[t])
        if self.wl.model == "linear":
            for t, row in gpu_eps.items():     # exact fp32 product on both sides
                assert np.array_equal(row, ost.Eh[t]), f"sample {n} sweep {k}: linear output of {t}"
        elif self.eps_stride > 0:
            for t in g["miss"]:
                pick = k == 0 or self._eps_seen % self.eps_stride == 0
                self._eps_seen += 1
                if not pick:
                    continue
                ref = self.net.eval_one(X_before[t - sw], t)
                e_rel = eps_error(gpu_eps[t], ref, self.wl.latent)
                self.eps_err.append(e_rel)
                assert e_rel <= EPS_RTOL, f"sample {n} sweep {k}: network output of {t} off by {e_rel:.3g} x its scale"
        self.records[n].append(g)
        return g, gpu_eps

    def _follow_allowance(self, n, k, sw, e, Xg, Xhg, c1):
        """Before device sweep k: bring the followed trajectory of sample n to the same window
        and measure, per cached slot, mean |x_o - x_d| + mean |x^_o - x^_d| against the
        device's pre-state rows (Xg from state sw, Xhg for sw..c1-1)."""
        f = self.fol[n]
        assert f.s == sw, f"follow sweep {k}: window start {f.s} vs {sw}"
        sp.fill_new_states(f.X, f.newest, e)
        allow = np.zeros(e - sw)
        for j in range(e - sw):
            t = sw + j
            if t < c1 and f.valid[t]:
                allow[j] = (np.abs(f.X[t].astype(np.float64) - Xg[j]).mean()
                            + np.abs(f.Xh[t].astype(np.float64) - Xhg[j]).mean())
        return allow

    def _follow_sweep(self, n, k, g, gpu_eps, allow):
        """Sweep k of the followed trajectory of sample n, after the device's: its own states,
        the device's decisions within the band, and for the patch-MLP the device's fresh outputs."""
        f, log = self.fol[n], self.follow_logs[n]
        e = sp.window_end(f.s, self.T, self.P)
        dev_o, _ = sp.cache_test(f.X, f.Xh, f.valid, f.s, e, self.delta)
        hit = _check_hits(k, dev_o, g, self.delta, log, allow=allow)
        if self.wl.model == "linear":
            eps_fn = self.net
        else:
            def eps_fn(Xb, steps, _r=gpu_eps):
                assert list(steps) == list(_r.keys())
                return np.stack([_r[t] for t in steps]).astype(Xb.dtype)
        noise = None if self.noise is None else self.noise[n]
        rec = sp.sweep(f, self.P, self.delta, self.wl.tol, self.alpha, self.b, eps_fn,
                       force_hit=hit, noise=noise)
        rec["allow"] = allow
        self.follow_traces[n].append(rec)
        assert rec["miss"] == g["miss"]
        if rec["c"] != g["c"]:
            j = min(rec["c"], g["c"])
            assert _in_band(rec["r"][j], self.wl.tol), f"follow sweep {k}: slide differs"
            log.flip("tau", k, j, rec["r"][j], self.wl.tol)
            f.s = g["s_next"]

    def follow(self, n=0):
        """The followed trajectory of sample n (advanced during run()): its counters, revisit
        counters and final latent against the device's; returns the x_T error / RMS."""
        T = self.T
        st, trace, log = self.fol[n], self.follow_traces[n], self.follow_logs[n]
        assert len(trace) == len(self.records[n])
        stn = self.stats_n[n]
        assert st.done and st.nfe == stn["nfe"] and st.hits == stn["hits"]
        # revisit counters (default threshold 0.05): the oracle's count from its own trace;
        # a deviation within the band of the threshold may fall either way.
        req, rev, below = sp.revisit_counts(trace, REVISIT_THR)
        assert req == stn["nfe"] + stn["hits"] and rev == stn["revisits"]
        near = sum(int(np.count_nonzero(np.abs(np.nan_to_num(np.asarray(r["dev"]), nan=-1.0) - REVISIT_THR)
                                        <= BAND * REVISIT_THR + (1.0 + SUM_RTOL) * r["allow"])) for r in trace)
        assert abs(below - stn["revisits_below"]) <= near, (below, stn["revisits_below"])
        ref = st.X[T].astype(np.float64)
        x_T = self.x_T_all[n]
        err = float(np.max(np.abs(x_T.astype(np.float64) - ref)) / max(rms(ref), 1e-30))
        self.follow_log = log
        return err

    def eps_summary(self) -> str:
        """Count, maximum and 99th percentile of the checked network-output errors (eps_error)."""
        if not self.eps_err:
            return "eps_checked=0"
        e = np.asarray(self.eps_err)
        return (f"eps_checked={len(e)}/{sum(r['m'] for recs in self.records for r in recs)} "
                f"eps_err_max={e.max():.2e} eps_err_p99={np.percentile(e, 99):.2e}")

    def follow_independent(self, n=0) -> dict:
        """The oracle's own run of sample n with its own network (not eps-locked): reported,
        not gated. The device's and the oracle's network outputs differ by bf16 rounding
        flips (about 1e-3 x RMS), so once a deviation or residual lands near its threshold
        the two runs may part. Returns how many sweeps agree in every decision before the
        first difference, whether that difference lies within the decision band, the
        counters of both runs and the final-latent error."""
        T, P = self.T, self.P
        noise = None if self.noise is None else self.noise[n]
        xo, trace, st = sp.sample(self.xs[n], T, P, self.delta, self.wl.tol, self.alpha, self.b,
                                  self.net, noise=noise)
        dev = self.records[n]
        agree, first = 0, None
        for ro, rg in zip(trace, dev):
            same = (ro["s"], ro["e"], list(ro["miss"]), ro["c"]) == (rg["s"], rg["e"], list(rg["miss"]), rg["c"])
            if not same:
                W = ro["e"] - ro["s"]
                flips = [j for j in range(W) if bool(ro["hit"][j]) != bool(rg["hit"][j])] \
                    if (ro["s"], ro["e"]) == (rg["s"], rg["e"]) else []
                in_band = all(_in_band(ro["dev"][j], self.delta) for j in flips)
                if not flips and ro["c"] != rg["c"] and (ro["s"], ro["e"]) == (rg["s"], rg["e"]):
                    j = min(ro["c"], rg["c"])
                    in_band = _in_band(ro["r"][j], self.wl.tol)
                    kind = "tau"
                else:
                    kind = "hit" if flips else "window"
                first = {"sweep": agree, "kind": kind, "hit_flips": len(flips), "in_band": bool(in_band)}
                break
            agree += 1
        stn = self.stats_n[n]
        ref = xo.astype(np.float64)
        err = float(np.max(np.abs(self.x_T_all[n].astype(np.float64) - ref)) / max(rms(ref), 1e-30))
        return {"agree_sweeps": agree, "oracle_sweeps": len(trace), "device_sweeps": len(dev),
                "first_difference": first, "nfe": (st.nfe, stn["nfe"]), "hits": (st.hits, stn["hits"]),
                "final_err": err}
