"""The oracle's pins catch plausible mistakes (CPU only).

Each case plants one mistake in a copy of ``oracle/`` -- a dropped term, a wrong sign or index,
a transposed operand, a non-strict comparison, a missing update -- and runs the oracle pin
tests (closed forms, textbook and library special cases, brute force, the scalar simulator,
the uncached references) against the copy in a fresh interpreter. Every mistake must make at
least one pin fail; the unmutated copy must pass, so a failure is the mistake's and not the
harness's. The mistakes live only in the temporary copy; the oracle itself is not touched.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PIN_TESTS = ["test_oracle_pieces.py", "test_oracle_sampler.py", "test_oracle_extensions.py",
             "test_oracle_parareal.py"]

# (name, oracle file, exact text, replacement). Every text occurs exactly once in its file.
MUTATIONS = [
    # schedule and step coefficients
    ("betas_not_squared", "schedule.py", "betas = root * root", "betas = root"),
    ("timesteps_off_by_one", "schedule.py", "(np.round(train_steps - j * train_steps / T) - 1)",
     "(np.round(train_steps - j * train_steps / T))"),
    ("final_alpha_bar", "schedule.py", "ab[T] = 1.0", "ab[T] = abar[0]"),
    ("ddim_alpha_not_increment", "schedule.py",
     "alpha = a - 1.0\n    b = np.sqrt(1.0 - ab[1:])", "alpha = a\n    b = np.sqrt(1.0 - ab[1:])"),
    ("ddim_b_sign", "schedule.py", "b = np.sqrt(1.0 - ab[1:]) - a * np.sqrt(1.0 - ab[:-1])",
     "b = np.sqrt(1.0 - ab[1:]) + a * np.sqrt(1.0 - ab[:-1])"),
    ("sigma_second_factor", "schedule.py",
     "full = eta * np.sqrt((1.0 - ab1) / (1.0 - ab0)) * np.sqrt(1.0 - ab0 / ab1)",
     "full = eta * np.sqrt((1.0 - ab1) / (1.0 - ab0))"),
    ("sigma_noiseless_rule_dropped", "schedule.py", "noiseless = (ab1 == ab0) | (eta == 0.0)",
     "noiseless = eta == 0.0"),
    ("b_without_sigma", "schedule.py", "x0_coef_eps = np.sqrt(1.0 - ab1 - sigma * sigma)",
     "x0_coef_eps = np.sqrt(1.0 - ab1)"),
    # networks
    ("bf16_ties_up", "eps_models.py", "(u + (((u >> 16) & np.uint32(1)) + np.uint32(0x7FFF)))",
     "(u + np.uint32(0x8000))"),
    ("patchify_dh_dw_swapped", "eps_models.py", "t = x.reshape(C, H // p, p, W // p, p).transpose(1, 3, 0, 2, 4)",
     "t = x.reshape(C, H // p, p, W // p, p).transpose(1, 3, 0, 4, 2)"),
    ("temb_sin_cos_swapped", "eps_models.py", "np.concatenate([np.sin(arg), np.cos(arg)], axis=1)",
     "np.concatenate([np.cos(arg), np.sin(arg)], axis=1)"),
    ("gelu_scale", "eps_models.py", "_erf(x / math.sqrt(2.0))", "_erf(x / 2.0)"),
    ("mlp_no_time_embedding", "eps_models.py", "pre1 = (xb @ self.W1 + self.temb[j].astype(F64)).astype(F32)",
     "pre1 = (xb @ self.W1).astype(F32)"),
    ("mlp_h1_not_rounded", "eps_models.py", "h1 = bf16_round(gelu(pre1).astype(F32)).astype(F64)",
     "h1 = gelu(pre1).astype(F32).astype(F64)"),
    ("mlp_second_gelu_dropped", "eps_models.py", "h2 = bf16_round(gelu(pre2).astype(F32)).astype(F64)",
     "h2 = bf16_round(pre2.astype(F32)).astype(F64)"),
    ("linear_step_index", "eps_models.py", "c64[np.asarray(steps)]", "c64[np.asarray(steps) - 1]"),
    ("unpatchify_dh_dw_swapped", "eps_models.py", "t = tok.reshape(H // p, W // p, C, p, p).transpose(2, 0, 3, 1, 4)",
     "t = tok.reshape(H // p, W // p, C, p, p).transpose(2, 0, 4, 1, 3)"),
    # the references the pins compare against
    ("scalar_recurrence_cached_state", "scalar_sim.py", "run += alpha[t] * g[t] + b[t] * c[t] * gh[t]",
     "run += alpha[t] * gh[t] + b[t] * c[t] * gh[t]"),
    ("uncached_slide_takes_last_state", "sampler.py", "while c < e - s - 1 and r[c] <= tau:",
     "while c < e - s and r[c] <= tau:"),
    ("textbook_ddpm_variance", "sampler.py", "var = beta * (1.0 - ab[i + 1]) / (1.0 - ab[i])", "var = beta"),
    # the cached Picard sampler
    ("picard_anchor", "sampler.py", "    acc = X[s].astype(F64)\n    Y = np.empty((e - s, X.shape[1]), dtype=X.dtype)",
     "    acc = X[s + 1].astype(F64)\n    Y = np.empty((e - s, X.shape[1]), dtype=X.dtype)"),
    ("drift_output_term_dropped", "sampler.py",
     "d = float(alpha[t]) * X[t].astype(F64) + float(b[t]) * Eh[t].astype(F64)",
     "d = float(alpha[t]) * X[t].astype(F64)"),
    ("residual_index", "sampler.py", "diff = Y[j].astype(F64) - X[s + 1 + j].astype(F64)",
     "diff = Y[j].astype(F64) - X[s + j].astype(F64)"),
    ("hit_not_strict", "sampler.py", "hit[j] = dev[j] < delta", "hit[j] = dev[j] <= delta"),
    ("deviation_sum_not_mean", "sampler.py", "return float(np.abs(x - np.asarray(xh, dtype=F64)).sum() / x.size)",
     "return float(np.abs(x - np.asarray(xh, dtype=F64)).sum())"),
    ("first_entry_rule_dropped", "sampler.py", "        if valid[t]:\n            dev[j] = mean_abs_deviation",
     "        if True:\n            dev[j] = mean_abs_deviation"),
    ("tau_strict", "sampler.py", "        if r[j] <= tau:", "        if r[j] < tau:"),
    ("last_state_decides_slide", "sampler.py", "    for j in range(len(r) - 1):\n        if r[j] <= tau:",
     "    for j in range(len(r)):\n        if r[j] <= tau:"),
    ("cache_input_not_updated", "sampler.py", "        st.Xh[t] = st.X[t]\n", "        pass\n"),
    ("new_states_from_initial", "sampler.py",
     "copies of the newest state.\"\"\"\n    for t in range(newest + 1, e + 1):\n        X[t] = X[newest]",
     "copies of the newest state.\"\"\"\n    for t in range(newest + 1, e + 1):\n        X[t] = X[0]"),
    ("noise_of_previous_step", "sampler.py", "            d = d + noise[t]\n        acc = acc + d",
     "            d = d + noise[t - 1]\n        acc = acc + d"),
    ("misses_descending", "sampler.py", "return [s + j for j in range(len(hit)) if not hit[j]]",
     "return [s + j for j in reversed(range(len(hit))) if not hit[j]]"),
    ("revisit_threshold_not_strict", "sampler.py", "below += int(np.count_nonzero(dev[seen] < threshold))",
     "below += int(np.count_nonzero(dev[seen] <= threshold))"),
    ("nan_counted_as_revisit", "sampler.py", "revisits += int(np.count_nonzero(seen))", "revisits += dev.size"),
    # Parareal
    ("parareal_correction_sign", "parareal.py",
     "            coarse.append(rec)\n            g = _step(U[n], e, ac[n], bc[n], store_dtype)\n"
     "            U[n + 1] = (g.astype(F64) + (Xf[n].astype(F64) - G[n].astype(F64))).astype(store_dtype)",
     "            coarse.append(rec)\n            g = _step(U[n], e, ac[n], bc[n], store_dtype)\n"
     "            U[n + 1] = (g.astype(F64) - (Xf[n].astype(F64) - G[n].astype(F64))).astype(store_dtype)"),
    ("parareal_coarse_b", "parareal.py", "bc = np.sqrt(1.0 - a1) - (1.0 + ac) * np.sqrt(1.0 - a0)",
     "bc = np.sqrt(1.0 - a1) - ac * np.sqrt(1.0 - a0)"),
    ("parareal_exact_copy_dropped", "parareal.py",
     "        U[k + 1] = Xf[k]                       # exact: the fine solve of a final state\n", ""),
    ("parareal_coarse_timestep", "parareal.py",
     "            (e,), rec = cache.request([n * L], [U[n]], eps_fn)\n            coarse.append(rec)",
     "            (e,), rec = cache.request([n * L + L - 1], [U[n]], eps_fn)\n            coarse.append(rec)"),
    ("parareal_hit_not_strict", "parareal.py", "hit[i] = dev[i] < self.delta", "hit[i] = dev[i] <= self.delta"),
    ("parareal_cache_input_not_updated", "parareal.py", "                self.Xh[t] = xs[i]\n", ""),
    ("parareal_no_stop_after_B", "parareal.py", "done = bool(np.all(r <= tau)) or k + 1 == B",
     "done = bool(np.all(r <= tau))"),
    ("parareal_tau_strict", "parareal.py", "done = bool(np.all(r <= tau)) or k + 1 == B",
     "done = bool(np.all(r < tau)) or k + 1 == B"),
    ("parareal_final_blocks_recomputed", "parareal.py", "        active = list(range(k, B))",
     "        active = list(range(0, B))"),
]


def _tree(tmp, name=None):
    """A directory holding a copy of oracle/ (with the named mutation), the pin tests, the
    seeded input generators and the binding's Python side (imported, never loaded by the pins);
    returns its path."""
    d = os.path.join(tmp, name or "control")
    shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(d, "oracle"),
                    ignore=shutil.ignore_patterns("__pycache__"))
    os.makedirs(os.path.join(d, "tests"))
    for f in ["conftest.py", "parity_harness.py", *PIN_TESTS]:
        shutil.copy(os.path.join(ROOT, "tests", f), os.path.join(d, "tests", f))
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), os.path.join(d, "tests", "golden"))
    pkg = os.path.join(d, "paper_2609_36522_amd")
    os.makedirs(pkg)
    for f in ["__init__.py", "inputs.py", "workloads.py", "binding.py"]:   # no library is loaded
        shutil.copy(os.path.join(ROOT, "paper_2609_36522_amd", f), os.path.join(pkg, f))
    if name is not None:
        mut = {m[0]: m for m in MUTATIONS}[name]
        _, fname, old, new = mut
        path = os.path.join(d, "oracle", fname)
        src = open(path).read()
        assert src.count(old) == 1, f"{name}: the text to replace occurs {src.count(old)} times"
        open(path, "w").write(src.replace(old, new))
    return d


def _run(d):
    env = dict(os.environ)
    env["PYTHONDONTWRITEBYTECODE"] = "1"
    env["OMP_NUM_THREADS"] = "1"
    env.pop("PYTHONPATH", None)
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
           *[os.path.join("tests", f) for f in PIN_TESTS]]
    r = subprocess.run(cmd, cwd=d, env=env, capture_output=True, text=True, timeout=600)
    return r.returncode, r.stdout[-3000:] + r.stderr[-2000:]


def test_every_planted_mistake_fails_a_pin(tmp_path):
    names = [m[0] for m in MUTATIONS]
    assert len(set(names)) == len(names)
    trees = {None: _tree(str(tmp_path))}
    for n in names:
        trees[n] = _tree(str(tmp_path), n)
    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        results = dict(zip(trees, ex.map(_run, trees.values())))
    rc, out = results.pop(None)
    assert rc == 0, f"the unmutated oracle copy fails its pins:\n{out}"
    missed = [n for n, (rc, _) in results.items() if rc != 1]
    detail = "\n".join(f"--- {n} (exit {results[n][0]}):\n{results[n][1][-1500:]}" for n in missed)
    # exit 1 = tests ran and at least one failed; 2-5 would be an interrupted or broken run
    assert not missed, f"planted mistakes no pin caught (or broken runs):\n{detail}"
