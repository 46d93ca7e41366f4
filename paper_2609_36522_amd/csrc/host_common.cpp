// Host-side helpers shared by the sampler handles (see pa_host.h).
#include "pa_host.h"

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <chrono>

#include <hip/hip_ext.h>

namespace pa {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int hip_fail(hipError_t e, const char* what) {
    if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation)
        return fail(PA_ERR_OOM, "%s: out of memory (%s)", what, hipGetErrorString(e));
    return fail(PA_ERR_HIP, "%s failed: %s", what, hipGetErrorString(e));
}

int build_schedule(const pa_schedule_t* sc, int T, double* ab, double* tv) {
    for (int i = 0; i <= T; ++i) ab[i] = 0.0;
    for (int j = 0; j < T; ++j) tv[j] = 0.0;
    if (sc->kind == PA_SCHED_SCALED_LINEAR) {
        const int N = sc->train_steps;
        if (!(N >= 2) || !(T <= N)) return fail(PA_ERR_INVALID_ARG, "schedule: need 2 <= train_steps and T <= train_steps");
        if (!(sc->beta_start > 0.0) || !(sc->beta_end > 0.0) || !(sc->beta_end < 1.0) || !(sc->beta_start < 1.0))
            return fail(PA_ERR_INVALID_ARG, "schedule: betas must lie in (0, 1)");
        if (sc->spacing != PA_SPACING_TRAILING) return fail(PA_ERR_UNSUPPORTED, "schedule: only trailing spacing is built");
        if (sc->final_alpha_one != 1) return fail(PA_ERR_UNSUPPORTED, "schedule: only final_alpha_one = 1 is built");
        for (int j = 0; j < T; ++j) {
            const long t = lrint(nearbyint((double)N - j * (double)N / T)) - 1;  // ties to even
            if (t < 0 || t >= N) return fail(PA_ERR_INVALID_ARG, "schedule: timestep out of range");
            tv[j] = (double)t;
        }
        // alpha_bar(t) = prod_{k <= t} (1 - beta_k), taken at the timesteps t_j as the running
        // product passes them (t_j strictly decreases with j: consecutive steps are at least
        // one train step apart).
        double prod = 1.0;
        const double r0 = sqrt(sc->beta_start), r1 = sqrt(sc->beta_end);
        int j = T - 1;
        for (int k = 0; k < N && j >= 0; ++k) {
            const double r = r0 + k * (r1 - r0) / (N - 1);
            prod *= 1.0 - r * r;
            while (j >= 0 && tv[j] == (double)k) ab[j--] = prod;
        }
        ab[T] = 1.0;
    } else if (sc->kind == PA_SCHED_EXPLICIT) {
        if (!sc->alpha_bar || !sc->t_values) return fail(PA_ERR_INVALID_ARG, "schedule: explicit arrays are NULL");
        for (int i = 0; i <= T; ++i) {
            const double a = sc->alpha_bar[i];
            if (!(a > 0.0 && a <= 1.0)) return fail(PA_ERR_INVALID_ARG, "schedule: alpha_bar[%d] outside (0, 1]", i);
            ab[i] = a;
        }
        for (int j = 0; j < T; ++j) tv[j] = (double)sc->t_values[j];
    } else {
        return fail(PA_ERR_INVALID_ARG, "schedule: unknown kind %d", sc->kind);
    }
    if (!(sc->eta >= 0.0 && sc->eta <= 1.0)) return fail(PA_ERR_INVALID_ARG, "schedule: eta must lie in [0, 1] (got %g)", sc->eta);
    if (sc->eta > 0.0) {
        // The noise scale sigma_i needs ab_i <= ab_{i+1} (no real square root otherwise).
        for (int i = 0; i < T; ++i)
            if (!(ab[i + 1] >= ab[i]))
                return fail(PA_ERR_INVALID_ARG, "schedule: alpha_bar must not decrease when eta > 0 (state %d)", i + 1);
    }
    return PA_OK;
}

int build_schedule(const pa_schedule_t* sc, int T, std::vector<double>& ab, std::vector<double>& tv) {
    ab.assign(T + 1, 0.0);
    tv.assign(T, 0.0);
    return build_schedule(sc, T, ab.data(), tv.data());
}

void step_coefficients(const double* ab, int T, double eta, double* coef) {
    // One-step increment d_i = alpha_i x_i + b_i eps_i + sigma_i z_i of the generalized DDIM
    // step with eta (eta = 0: DDIM; eta = 1: ancestral DDPM). sigma_i is 0 at eta = 0, and
    // where ab_{i+1} = ab_i (its second factor is 0 and its first at most 1; for
    // ab_i = ab_{i+1} = 1 the first is 0/0), so a degenerate step has no NaN coefficients.
    for (int i = 0; i < T; ++i) {
        const double a = sqrt(ab[i + 1] / ab[i]);
        const double sig = (eta == 0.0 || ab[i + 1] == ab[i])
                               ? 0.0
                               : eta * sqrt((1.0 - ab[i + 1]) / (1.0 - ab[i])) * sqrt(1.0 - ab[i] / ab[i + 1]);
        coef[3 * i] = a - 1.0;
        coef[3 * i + 1] = sqrt(1.0 - ab[i + 1] - sig * sig) - a * sqrt(1.0 - ab[i]);
        coef[3 * i + 2] = sig;
    }
}

std::vector<double> step_coefficients(const std::vector<double>& ab, int T, double eta) {
    std::vector<double> coef(3 * (size_t)T);
    step_coefficients(ab.data(), T, eta, coef.data());
    return coef;
}

int check_eps_model(const pa_eps_model_t* em, int C, int Hi, int Wi, int T) {
    if (em->kind == PA_EPS_LINEAR) {
        if (!em->c) return fail(PA_ERR_INVALID_ARG, "linear model: c is NULL");
        for (int j = 0; j < T; ++j)
            if (!isfinite(em->c[j])) return fail(PA_ERR_INVALID_ARG, "linear model: c[%d] is not finite", j);
    } else if (em->kind == PA_EPS_PATCH_MLP) {
        if (!em->w1 || !em->wt || !em->w2 || !em->w3) return fail(PA_ERR_INVALID_ARG, "patch-MLP: weight pointer is NULL");
        if (em->patch != 2) return fail(PA_ERR_UNSUPPORTED, "patch-MLP: only patch = 2 is built");
        if (C != 4) return fail(PA_ERR_UNSUPPORTED, "patch-MLP: only C = 4 is built");
        if (Hi % 2 || Wi % 2) return fail(PA_ERR_INVALID_ARG, "patch-MLP: H and W must be even");
        if (em->temb_dim != 128) return fail(PA_ERR_UNSUPPORTED, "patch-MLP: only temb_dim = 128 is built");
        if (!mlp_supported(em->hidden)) return fail(PA_ERR_UNSUPPORTED, "patch-MLP: hidden %d not built (512, 1024, 2048)", em->hidden);
        if (((Hi / 2) * (Wi / 2)) % mlp_tokens_per_item())
            return fail(PA_ERR_UNSUPPORTED, "patch-MLP: token count must be a multiple of %d", mlp_tokens_per_item());
    } else {
        return fail(PA_ERR_INVALID_ARG, "unknown eps model kind %d", em->kind);
    }
    return PA_OK;
}

bool QueryPacer::due() {
    const int64_t now = std::chrono::duration_cast<std::chrono::nanoseconds>(
                            std::chrono::steady_clock::now().time_since_epoch()).count();
    if (next_ns == 0) next_ns = now + kIntervalNs;   // the first query one interval from now
    if (now < next_ns) return false;
    next_ns = now + kIntervalNs;
    return true;
}

int KernelTimer::pair(int k, hipEvent_t* e0, hipEvent_t* e1) {
    for (hipEvent_t* out : {e0, e1}) {
        if (used == pool.size()) {
            hipEvent_t e;
            // Timing only: no system-scope fence, so the events do not disturb the stream.
            PA_HIP(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
            pool.push_back(e);
        }
        *out = pool[used++];
    }
    kind.push_back(k);
    return PA_OK;
}

int KernelTimer::drain() {
    for (size_t i = 0; i + 1 < used; i += 2) {
        float t = 0.f;
        PA_HIP(hipEventElapsedTime(&t, pool[i], pool[i + 1]));
        const int k = kind[i / 2];
        ms[k] += t;
        launches[k] += 1;
    }
    used = 0;
    kind.clear();
    return PA_OK;
}

void KernelTimer::clear() {
    used = 0;
    kind.clear();
    for (int k = 0; k < kKinds; ++k) {
        launches[k] = 0;
        ms[k] = 0.0;
    }
}

int setup_network(Dev& d, DevMem& mem, const pa_eps_model_t* em, const double* tv,
                  int cus, size_t ep_rows, hipStream_t st) {
    const int T = d.T;
    const size_t Dz = (size_t)d.D;
    int rc;
    if (em->kind == PA_EPS_LINEAR) {
        if ((rc = mem.alloc(&d.lin_c, (size_t)T, "lin_c"))) return rc;
        PA_HIP(hipMemcpyAsync(d.lin_c, em->c, (size_t)T * sizeof(float), hipMemcpyHostToDevice, st));
        PA_HIP(hipStreamSynchronize(st));
        return PA_OK;
    }
    const int Hd = em->hidden;
    d.hidden = Hd;
    d.ntok = (d.Himg / 2) * (d.Wimg / 2);
    d.mlp_grid = mlp_grid_size(cus);
    // The caller's weights ([in][out] bf16) are copied as they are and rearranged on the device
    // into the network kernel's layouts (launch_pack_weights).
    uint16_t *w1r, *w2r, *w3r;
    __bf16 *w1d, *w2d, *w3d, *wtd;
    double* tvd;
    if ((rc = mem.alloc(&w1r, (size_t)Hd * 16, "w1 (as given)"))) return rc;
    if ((rc = mem.alloc(&w2r, (size_t)Hd * Hd, "w2 (as given)"))) return rc;
    if ((rc = mem.alloc(&w3r, (size_t)Hd * 16, "w3 (as given)"))) return rc;
    if ((rc = mem.alloc(&w1d, (size_t)Hd * 16, "w1t"))) return rc;
    if ((rc = mem.alloc(&w2d, (size_t)Hd * Hd, "w2f"))) return rc;
    if ((rc = mem.alloc(&w3d, (size_t)Hd * 32, "w3p"))) return rc;
    if ((rc = mem.alloc(&wtd, (size_t)em->temb_dim * Hd, "wt"))) return rc;
    if ((rc = mem.alloc(&tvd, (size_t)T, "t_values"))) return rc;
    if ((rc = mem.alloc(&d.temb, (size_t)T * Hd, "temb"))) return rc;
    d.nsplit = mlp_splits(Hd);
    if ((rc = mem.alloc(&d.Ep, (size_t)d.nsplit * ep_rows * Dz, "Ep"))) return rc;
    PA_HIP(hipMemcpyAsync(w1r, em->w1, (size_t)Hd * 16 * 2, hipMemcpyHostToDevice, st));
    PA_HIP(hipMemcpyAsync(w2r, em->w2, (size_t)Hd * Hd * 2, hipMemcpyHostToDevice, st));
    PA_HIP(hipMemcpyAsync(w3r, em->w3, (size_t)Hd * 16 * 2, hipMemcpyHostToDevice, st));
    PA_HIP(hipMemcpyAsync(wtd, em->wt, (size_t)em->temb_dim * Hd * 2, hipMemcpyHostToDevice, st));
    PA_HIP(hipMemcpyAsync(tvd, tv, (size_t)T * sizeof(double), hipMemcpyHostToDevice, st));
    PA_HIP(launch_pack_weights(w1r, w2r, w3r, Hd, w1d, w2d, w3d, st));
    d.w1t = w1d;
    d.w2f = w2d;
    d.w3p = w3d;
    PA_HIP(launch_temb_table(d, tvd, wtd, em->temb_dim, st));
    return PA_OK;
}

}  // namespace pa
