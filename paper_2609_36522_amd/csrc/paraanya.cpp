// Host side of the C ABI declared in include/paraanya.h: argument validation (before any
// HIP call), schedule and DDIM coefficients in fp64, device buffers and weight layouts,
// the sweep enqueue loop. Every compute step of a sweep runs in the gfx950 kernels.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <new>
#include <string>
#include <vector>

#include "pa_internal.h"

using pa::Ctrl;
using pa::Dev;

namespace {

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

#define PA_HIP(call)                                           \
    do {                                                       \
        hipError_t e_ = (call);                                \
        if (e_ != hipSuccess) return hip_fail(e_, #call);      \
    } while (0)

}  // namespace

struct paraanya {
    Dev d{};
    hipStream_t stream = nullptr;
    uint32_t flags = 0;
    int model = PA_EPS_LINEAR;
    int temb_dim = 0;
    std::vector<double> coef_host;    // [T][3] as uploaded
    Ctrl* ctrl_host = nullptr;        // pinned mirror, one block per sample
    uint64_t* progress_host = nullptr; // pinned, device-mapped progress words (see k_slide)
    float* noise_buf = nullptr;       // [N][T][D] step noise (eta > 0)
    bool noise_set = false;
    bool ctrl_fresh = false;           // ctrl_host matches the device and nothing is queued
    bool have_reset = false;
    bool host_done = false;           // done flag of the last synchronized read
    std::vector<void*> allocs;        // device allocations
    // profiling
    std::vector<hipEvent_t> ev_pool;
    size_t ev_used = 0;
    std::vector<int> ev_kind;         // kernel kind of each event pair
    int64_t prof_kernel_launches[3] = {0, 0, 0};
    double prof_kernel_ms[3] = {0.0, 0.0, 0.0};

    ~paraanya() {
        (void)hipStreamSynchronize(stream);
        for (hipEvent_t e : ev_pool) (void)hipEventDestroy(e);
        for (void* p : allocs) (void)hipFree(p);
        if (ctrl_host) (void)hipHostFree(ctrl_host);
        if (progress_host) (void)hipHostFree(progress_host);
    }

    template <class T>
    int alloc(T** p, size_t count, const char* what) {
        void* q = nullptr;
        hipError_t e = hipMalloc(&q, count * sizeof(T) + 256);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return fail(PA_ERR_OOM, "hipMalloc(%s, %zu bytes): %s", what, count * sizeof(T),
                        hipGetErrorString(e));
        }
        allocs.push_back(q);
        *p = static_cast<T*>(q);
        return PA_OK;
    }

    int read_ctrl() {
        // The mirror stays valid until the next enqueue, so repeated queries cost nothing.
        if (ctrl_fresh) return PA_OK;
        PA_HIP(hipMemcpyAsync(ctrl_host, d.ctrl, (size_t)d.N * sizeof(Ctrl), hipMemcpyDeviceToHost, stream));
        PA_HIP(hipStreamSynchronize(stream));
        host_done = true;
        for (int n = 0; n < d.N; ++n) host_done = host_done && ctrl_host[n].done != 0;
        ctrl_fresh = true;
        return PA_OK;
    }

    bool any_nonfinite() const {
        for (int n = 0; n < d.N; ++n)
            if (ctrl_host[n].nonfinite) return true;
        return false;
    }

    int drain_profile() {
        // Event pairs recorded since the last drain; the stream is synchronized by the caller.
        for (size_t i = 0; i + 1 < ev_used; i += 2) {
            float ms = 0.f;
            PA_HIP(hipEventElapsedTime(&ms, ev_pool[i], ev_pool[i + 1]));
            const int k = ev_kind[i / 2];
            prof_kernel_ms[k] += ms;
            prof_kernel_launches[k] += 1;
        }
        ev_used = 0;
        ev_kind.clear();
        return PA_OK;
    }

    // Start/stop events of one timed launch of kernel kind k (0 network, 1 Picard, 2 slide),
    // or nulls when the handle is not profiling.
    int timed(int k, hipEvent_t* e0, hipEvent_t* e1) {
        *e0 = *e1 = nullptr;
        if (!(flags & PA_FLAG_PROFILE)) return PA_OK;
        if (k > 0 && !(flags & PA_FLAG_PROFILE_SOLVER)) return PA_OK;
        int rc = next_event(e0);
        if (rc) return rc;
        if ((rc = next_event(e1))) return rc;
        ev_kind.push_back(k);
        return PA_OK;
    }

    int next_event(hipEvent_t* out) {
        if (ev_used == ev_pool.size()) {
            hipEvent_t e;
            // Timing only: no system-scope fence, so the events do not disturb the stream.
            PA_HIP(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
            ev_pool.push_back(e);
        }
        *out = ev_pool[ev_used++];
        return PA_OK;
    }

    int enqueue_sweep() {
        // The miss list of this sweep was published by the previous k_slide (or k_reset).
        // Under PROFILE every launch carries its own start/stop events (no marker packets
        // between kernels).
        ctrl_fresh = false;
        hipEvent_t e0, e1;
        int rc;
        if (model == PA_EPS_PATCH_MLP) {
            if ((rc = timed(0, &e0, &e1))) return rc;
            PA_HIP(pa::launch_eps_mlp(d, stream, e0, e1));
        }
        if ((rc = timed(1, &e0, &e1))) return rc;
        PA_HIP(pa::launch_picard(d, stream, model == PA_EPS_LINEAR, e0, e1));
        if ((rc = timed(2, &e0, &e1))) return rc;
        PA_HIP(pa::launch_slide(d, stream, e0, e1));
        return PA_OK;
    }
};

namespace {

int build_schedule(const pa_schedule_t* sc, int T, std::vector<double>& ab, std::vector<double>& tv) {
    ab.assign(T + 1, 0.0);
    tv.assign(T, 0.0);
    if (sc->kind == PA_SCHED_SCALED_LINEAR) {
        const int N = sc->train_steps;
        if (!(N >= 2) || !(T <= N)) return fail(PA_ERR_INVALID_ARG, "schedule: need 2 <= train_steps and T <= train_steps");
        if (!(sc->beta_start > 0.0) || !(sc->beta_end > 0.0) || !(sc->beta_end < 1.0) || !(sc->beta_start < 1.0))
            return fail(PA_ERR_INVALID_ARG, "schedule: betas must lie in (0, 1)");
        if (sc->spacing != PA_SPACING_TRAILING) return fail(PA_ERR_UNSUPPORTED, "schedule: only trailing spacing is built");
        if (sc->final_alpha_one != 1) return fail(PA_ERR_UNSUPPORTED, "schedule: only final_alpha_one = 1 is built");
        std::vector<double> abar(N);
        double prod = 1.0;
        const double r0 = sqrt(sc->beta_start), r1 = sqrt(sc->beta_end);
        for (int j = 0; j < N; ++j) {
            const double r = r0 + j * (r1 - r0) / (N - 1);
            prod *= 1.0 - r * r;
            abar[j] = prod;
        }
        for (int j = 0; j < T; ++j) {
            const long t = lrint(nearbyint((double)N - j * (double)N / T)) - 1;  // ties to even
            if (t < 0 || t >= N) return fail(PA_ERR_INVALID_ARG, "schedule: timestep out of range");
            tv[j] = (double)t;
            ab[j] = abar[t];
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
    return PA_OK;
}

}  // namespace

extern "C" {

const char* paraanya_last_error(void) { return g_err.c_str(); }

const char* paraanya_status_str(int s) {
    switch (s) {
        case PA_OK: return "PA_OK";
        case PA_ERR_INVALID_ARG: return "PA_ERR_INVALID_ARG";
        case PA_ERR_HIP: return "PA_ERR_HIP";
        case PA_ERR_OOM: return "PA_ERR_OOM";
        case PA_ERR_STATE: return "PA_ERR_STATE";
        case PA_ERR_NONFINITE: return "PA_ERR_NONFINITE";
        case PA_ERR_UNSUPPORTED: return "PA_ERR_UNSUPPORTED";
        default: return "PA_ERR_UNKNOWN";
    }
}

int paraanya_create(const int32_t latent_shape[4], int32_t T, const pa_schedule_t* schedule,
                    int32_t window, double delta, double tol, const pa_eps_model_t* eps_model,
                    void* stream, uint32_t flags, paraanya_t** out) {
    g_err.clear();
    if (!out) return fail(PA_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    // ---- validation: no HIP call before this block completes
    if (!latent_shape || !schedule || !eps_model) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    const int N = latent_shape[0], C = latent_shape[1], Hi = latent_shape[2], Wi = latent_shape[3];
    if (N < 1 || N > PA_MAX_BATCH) return fail(PA_ERR_INVALID_ARG, "batch N must be in [1, %d] (got %d)", PA_MAX_BATCH, N);
    if (C < 1 || Hi < 1 || Wi < 1) return fail(PA_ERR_INVALID_ARG, "latent dims must be positive");
    const long long Dl = (long long)C * Hi * Wi;
    if (Dl % 4 != 0) return fail(PA_ERR_INVALID_ARG, "C*H*W must be a multiple of 4");
    if (Dl > (1ll << 30)) return fail(PA_ERR_INVALID_ARG, "latent too large");
    if (T < 1) return fail(PA_ERR_INVALID_ARG, "T must be >= 1");
    if (window < 1 || window > T || window > PA_MAX_WINDOW)
        return fail(PA_ERR_INVALID_ARG, "window must be in [1, min(T, %d)]", PA_MAX_WINDOW);
    if (!(delta >= 0.0)) return fail(PA_ERR_INVALID_ARG, "delta must be >= 0 (got %g)", delta);
    if (!(tol >= 0.0)) return fail(PA_ERR_INVALID_ARG, "tol must be >= 0 (got %g)", tol);
    if (flags & ~(PA_FLAG_TRACE | PA_FLAG_PROFILE | PA_FLAG_PROFILE_SOLVER)) return fail(PA_ERR_INVALID_ARG, "unknown flags");
    const int D = (int)Dl;
    const pa_eps_model_t* em = eps_model;
    if (em->kind == PA_EPS_LINEAR) {
        if (!em->c) return fail(PA_ERR_INVALID_ARG, "linear model: c is NULL");
    } else if (em->kind == PA_EPS_PATCH_MLP) {
        if (!em->w1 || !em->wt || !em->w2 || !em->w3) return fail(PA_ERR_INVALID_ARG, "patch-MLP: weight pointer is NULL");
        if (em->patch != 2) return fail(PA_ERR_UNSUPPORTED, "patch-MLP: only patch = 2 is built");
        if (C != 4) return fail(PA_ERR_UNSUPPORTED, "patch-MLP: only C = 4 is built");
        if (Hi % 2 || Wi % 2) return fail(PA_ERR_INVALID_ARG, "patch-MLP: H and W must be even");
        if (em->temb_dim != 128) return fail(PA_ERR_UNSUPPORTED, "patch-MLP: only temb_dim = 128 is built");
        if (!pa::mlp_supported(em->hidden)) return fail(PA_ERR_UNSUPPORTED, "patch-MLP: hidden %d not built (512, 1024)", em->hidden);
        if (((Hi / 2) * (Wi / 2)) % pa::mlp_tokens_per_item())
            return fail(PA_ERR_UNSUPPORTED, "patch-MLP: token count must be a multiple of %d", pa::mlp_tokens_per_item());
    } else {
        return fail(PA_ERR_INVALID_ARG, "unknown eps model kind %d", em->kind);
    }
    std::vector<double> ab, tv;
    int rc = build_schedule(schedule, T, ab, tv);
    if (rc) return rc;
    // One-step increment d_i = alpha_i x_i + b_i eps_i + sigma_i z_i of the generalized DDIM
    // step with eta (eta = 0: DDIM; eta = 1: ancestral DDPM), fp64.
    const double eta = schedule->eta;
    std::vector<double> coef(3 * (size_t)T);
    for (int i = 0; i < T; ++i) {
        const double a = sqrt(ab[i + 1] / ab[i]);
        const double sig = eta * sqrt((1.0 - ab[i + 1]) / (1.0 - ab[i])) * sqrt(1.0 - ab[i] / ab[i + 1]);
        coef[3 * i] = a - 1.0;
        coef[3 * i + 1] = sqrt(1.0 - ab[i + 1] - sig * sig) - a * sqrt(1.0 - ab[i]);
        coef[3 * i + 2] = sig;
    }
    if (em->kind == PA_EPS_LINEAR)
        for (int j = 0; j < T; ++j)
            if (!isfinite(em->c[j])) return fail(PA_ERR_INVALID_ARG, "linear model: c[%d] is not finite", j);

    // ---- resources
    paraanya* h = new (std::nothrow) paraanya();
    if (!h) return fail(PA_ERR_OOM, "host allocation failed");
    h->stream = (hipStream_t)stream;
    h->flags = flags;
    h->model = em->kind;
    h->coef_host = coef;
    Dev& d = h->d;
    d.N = N; d.T = T; d.P = window; d.D = D; d.C = C; d.Himg = Hi; d.Wimg = Wi;
    d.delta = delta; d.tol = tol;
    d.revisit_thr = 0.05;
    d.picard_blocks = pa::picard_blocks(D);
    auto bail = [&](int code) { delete h; return code; };

    int dev_id = 0;
    hipError_t he = hipGetDevice(&dev_id);
    if (he != hipSuccess) return bail(hip_fail(he, "hipGetDevice"));
    int cus = 0;
    he = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev_id);
    if (he != hipSuccess) return bail(hip_fail(he, "hipDeviceGetAttribute"));

    const size_t Dz = (size_t)D;
    const size_t Nz = (size_t)N;
    if ((rc = h->alloc(&d.X, Nz * (T + 1) * Dz, "X"))) return bail(rc);
    if ((rc = h->alloc(&d.Xh, Nz * T * Dz, "Xh"))) return bail(rc);
    if ((rc = h->alloc(&d.Eh, Nz * T * Dz, "Eh"))) return bail(rc);
    if ((rc = h->alloc(&d.valid, Nz * T, "valid"))) return bail(rc);
    if ((rc = h->alloc(&d.coef, 3 * (size_t)T, "coef"))) return bail(rc);
    if ((rc = h->alloc(&d.part_res, Nz * window * d.picard_blocks, "part_res"))) return bail(rc);
    if ((rc = h->alloc(&d.part_dev, Nz * window * d.picard_blocks, "part_dev"))) return bail(rc);
    if ((rc = h->alloc(&d.ctrl, Nz, "ctrl"))) return bail(rc);
    if (flags & PA_FLAG_TRACE)
        if ((rc = h->alloc(&d.trace, Nz * T, "trace"))) return bail(rc);
    if (eta > 0.0) {
        if ((rc = h->alloc(&h->noise_buf, Nz * T * Dz, "noise"))) return bail(rc);
        d.noise = h->noise_buf;
    }
    he = hipHostMalloc((void**)&h->ctrl_host, Nz * sizeof(Ctrl), hipHostMallocDefault);
    if (he != hipSuccess) return bail(hip_fail(he, "hipHostMalloc"));
    memset(h->ctrl_host, 0, Nz * sizeof(Ctrl));
    he = hipHostMalloc((void**)&h->progress_host, Nz * sizeof(uint64_t) < 256 ? 256 : Nz * sizeof(uint64_t),
                       hipHostMallocMapped | hipHostMallocCoherent);
    if (he != hipSuccess) return bail(hip_fail(he, "hipHostMalloc(progress)"));
    for (int n = 0; n < N; ++n) h->progress_host[n] = 0;
    he = hipHostGetDevicePointer((void**)&d.progress, h->progress_host, 0);
    if (he != hipSuccess) return bail(hip_fail(he, "hipHostGetDevicePointer"));

#define PA_HIP_BAIL(call)                                        \
    do {                                                         \
        hipError_t e_ = (call);                                  \
        if (e_ != hipSuccess) return bail(hip_fail(e_, #call));  \
    } while (0)

    PA_HIP_BAIL(hipMemcpyAsync(d.coef, coef.data(), coef.size() * sizeof(double), hipMemcpyHostToDevice, h->stream));
    if (em->kind == PA_EPS_LINEAR) {
        if ((rc = h->alloc(&d.lin_c, (size_t)T, "lin_c"))) return bail(rc);
        PA_HIP_BAIL(hipMemcpyAsync(d.lin_c, em->c, (size_t)T * sizeof(float), hipMemcpyHostToDevice, h->stream));
        PA_HIP_BAIL(hipStreamSynchronize(h->stream));
    } else {
        const int Hd = em->hidden;
        d.hidden = Hd;
        d.ntok = (Hi / 2) * (Wi / 2);
        d.mlp_grid = pa::mlp_grid_size(cus);
        h->temb_dim = em->temb_dim;
        // Device layouts: W1^T [H][16]; W2^T as MFMA A fragments, fragment (b, ks) = lanes
        // l = 0..63 x 8 values W2[16 ks + 8 (l/32) + i][32 b + l%32]; W3 fragments permuted
        // to the GEMM2 accumulator layout (see k_epsnet.hip).
        std::vector<uint16_t> w1t((size_t)Hd * 16), w2f((size_t)Hd * Hd), w3p((size_t)Hd * 32);
        for (int f = 0; f < 16; ++f)
            for (int n = 0; n < Hd; ++n) w1t[(size_t)n * 16 + f] = em->w1[(size_t)f * Hd + n];
        const int KS = Hd / 16;
        for (int b = 0; b < Hd / 32; ++b)
            for (int ks = 0; ks < KS; ++ks)
                for (int lane = 0; lane < 64; ++lane)
                    for (int i = 0; i < 8; ++i) {
                        const int n = b * 32 + (lane & 31), k = ks * 16 + (lane >> 5) * 8 + i;
                        w2f[(((size_t)b * KS + ks) * 64 + lane) * 8 + i] = em->w2[(size_t)k * Hd + n];
                    }
        for (int hbg = 0; hbg < Hd / 32; ++hbg)
            for (int jj = 0; jj < 2; ++jj)
                for (int lane = 0; lane < 64; ++lane)
                    for (int i = 0; i < 8; ++i) {
                        const int g = lane >> 5, f = lane & 31;
                        const int n = hbg * 32 + (jj * 2 + i / 4) * 8 + g * 4 + (i % 4);
                        w3p[(((size_t)hbg * 2 + jj) * 64 + lane) * 8 + i] =
                            f < 16 ? em->w3[(size_t)n * 16 + f] : (uint16_t)0;
                    }
        __bf16 *w1d, *w2d, *w3d, *wtd;
        double* tvd;
        if ((rc = h->alloc(&w1d, w1t.size(), "w1t"))) return bail(rc);
        if ((rc = h->alloc(&w2d, w2f.size(), "w2f"))) return bail(rc);
        if ((rc = h->alloc(&w3d, w3p.size(), "w3p"))) return bail(rc);
        if ((rc = h->alloc(&wtd, (size_t)em->temb_dim * Hd, "wt"))) return bail(rc);
        if ((rc = h->alloc(&tvd, (size_t)T, "t_values"))) return bail(rc);
        if ((rc = h->alloc(&d.temb, (size_t)T * Hd, "temb"))) return bail(rc);
        d.nsplit = pa::mlp_splits(Hd);
        if ((rc = h->alloc(&d.Ep, (size_t)d.nsplit * Nz * window * Dz, "Ep"))) return bail(rc);
        PA_HIP_BAIL(hipMemcpyAsync(w1d, w1t.data(), w1t.size() * 2, hipMemcpyHostToDevice, h->stream));
        PA_HIP_BAIL(hipMemcpyAsync(w2d, w2f.data(), w2f.size() * 2, hipMemcpyHostToDevice, h->stream));
        PA_HIP_BAIL(hipMemcpyAsync(w3d, w3p.data(), w3p.size() * 2, hipMemcpyHostToDevice, h->stream));
        PA_HIP_BAIL(hipMemcpyAsync(wtd, em->wt, (size_t)em->temb_dim * Hd * 2, hipMemcpyHostToDevice, h->stream));
        PA_HIP_BAIL(hipMemcpyAsync(tvd, tv.data(), (size_t)T * sizeof(double), hipMemcpyHostToDevice, h->stream));
        d.w1t = w1d;
        d.w2f = w2d;
        d.w3p = w3d;
        PA_HIP_BAIL(pa::launch_temb_table(d, tvd, wtd, em->temb_dim, h->stream));
        PA_HIP_BAIL(hipStreamSynchronize(h->stream));   // host staging vectors die here
    }
#undef PA_HIP_BAIL
    *out = h;
    return PA_OK;
}

int paraanya_reset(paraanya_t* h, const float* x_init) {
    g_err.clear();
    if (!h || !x_init) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    if (h->noise_buf && !h->noise_set) return fail(PA_ERR_STATE, "eta > 0: set the step noise first (paraanya_set_noise)");
    // No kernel of this handle may still publish progress from an earlier sample.
    PA_HIP(hipStreamSynchronize(h->stream));
    for (int n = 0; n < h->d.N; ++n) h->progress_host[n] = 0;
    h->ctrl_fresh = false;
    const size_t row = (size_t)h->d.D * sizeof(float);
    PA_HIP(hipMemcpy2DAsync(h->d.X, (size_t)(h->d.T + 1) * row, x_init, row, row, (size_t)h->d.N,
                            hipMemcpyDeviceToDevice, h->stream));
    PA_HIP(pa::launch_reset(h->d, h->stream));
    h->have_reset = true;
    h->host_done = false;
    h->ev_used = 0;
    h->ev_kind.clear();
    for (int k = 0; k < 3; ++k) {
        h->prof_kernel_ms[k] = 0.0;
        h->prof_kernel_launches[k] = 0;
    }
    return PA_OK;
}

int paraanya_set_noise(paraanya_t* h, const float* z) {
    g_err.clear();
    if (!h || !z) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    if (!h->noise_buf) return fail(PA_ERR_INVALID_ARG, "handle has eta = 0: no step noise");
    PA_HIP(hipMemcpyAsync(h->noise_buf, z, (size_t)h->d.N * h->d.T * h->d.D * sizeof(float),
                          hipMemcpyDeviceToDevice, h->stream));
    h->noise_set = true;
    return PA_OK;
}

int paraanya_set_revisit_threshold(paraanya_t* h, double threshold) {
    g_err.clear();
    if (!h) return fail(PA_ERR_INVALID_ARG, "NULL handle");
    if (!(threshold >= 0.0)) return fail(PA_ERR_INVALID_ARG, "threshold must be >= 0 (got %g)", threshold);
    h->d.revisit_thr = threshold;
    return PA_OK;
}

int paraanya_sweep(paraanya_t* h, int32_t* done) {
    g_err.clear();
    if (!h) return fail(PA_ERR_INVALID_ARG, "NULL handle");
    if (!h->have_reset) return fail(PA_ERR_STATE, "sweep before reset");
    if (h->host_done) return fail(PA_ERR_STATE, "sweep after the sampler finished");
    int rc = h->enqueue_sweep();
    if (rc) return rc;
    if (done) {
        if ((rc = h->read_ctrl())) return rc;
        *done = h->host_done ? 1 : 0;
        if (h->any_nonfinite()) return fail(PA_ERR_NONFINITE, "non-finite residual");
    }
    return PA_OK;
}

int paraanya_sample(paraanya_t* h, const float* x_init, float* x_out) {
    g_err.clear();
    if (!h || !x_init || !x_out) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    int rc = paraanya_reset(h, x_init);
    if (rc) return rc;
    const int T = h->d.T, P = h->d.P, N = h->d.N;
    // Launch loop without per-sweep synchronisation: k_slide publishes (completed sweeps,
    // done, s) of every sample to a pinned host word after each sweep; the host keeps enough
    // sweeps in flight -- at least the kLookahead next ones and at least the ceil((T - s)/P)
    // that the slowest sample certainly still needs (s advances by at most P per sweep) --
    // and stops enqueuing once every sample is done. Sweeps enqueued after that exit at
    // their first instruction. Every sweep advances each unfinished sample's s by at least 1,
    // so at most T sweeps are ever enqueued. The stream is polled while waiting, so a failed
    // or idle stream ends the loop.
    constexpr int kLookahead = 2;
    volatile uint64_t* prog = h->progress_host;
    auto scan = [&](int* completed, int* need) {      // returns true once all are done
        bool all = true;
        *completed = 0;
        *need = 0;
        for (int n = 0; n < N; ++n) {
            const uint64_t w = prog[n];
            const int c = (int)(w >> 32), s_now = (int)(w & 0x7fffffffu);
            if (c > *completed) *completed = c;
            if ((w >> 31) & 1u) continue;
            all = false;
            const int q = (T - s_now + P - 1) / P;
            if (q > *need) *need = q;
        }
        return all;
    };
    int enqueued = 0;
    for (unsigned spin = 0;; ++spin) {
        int completed, need;
        if (scan(&completed, &need)) break;
        const int want = completed + (need > kLookahead ? need : kLookahead);
        if (enqueued < want && enqueued < T) {
            const int k = (want < T ? want : T) - enqueued;
            for (int i = 0; i < k; ++i)
                if ((rc = h->enqueue_sweep())) return rc;
            enqueued += k;
            continue;
        }
        if (spin % 256 != 255) continue;        // poll the stream now and then, not per spin
        const hipError_t q = hipStreamQuery(h->stream);
        if (q == hipSuccess) {
            // Stream idle: the words are final for the enqueued work.
            if (scan(&completed, &need)) break;
            if (enqueued >= T) return fail(PA_ERR_HIP, "sampler did not finish within T sweeps");
        } else if (q != hipErrorNotReady) {
            return hip_fail(q, "hipStreamQuery");
        }
    }
    // One synchronization for the output copy and the counters.
    const size_t row = (size_t)h->d.D * sizeof(float);
    PA_HIP(hipMemcpy2DAsync(x_out, row, h->d.X + (size_t)T * h->d.D, (size_t)(T + 1) * row, row,
                            (size_t)N, hipMemcpyDeviceToDevice, h->stream));
    h->ctrl_fresh = false;
    if ((rc = h->read_ctrl())) return rc;
    if (h->any_nonfinite()) return fail(PA_ERR_NONFINITE, "non-finite residual during sampling");
    return PA_OK;
}

namespace {

void fill_stats(const Ctrl& c, pa_stats_t* out) {
    out->nfe = c.nfe;
    out->hits = c.hits;
    out->misses = c.nfe;
    out->sweeps = c.sweep;
    out->window_start = c.s;
    out->window_end = c.e;
    out->done = c.done;
    out->nonfinite = c.nonfinite;
    out->revisits = c.revisits;
    out->revisits_below = c.revisits_below;
}

}  // namespace

int paraanya_stats(paraanya_t* h, pa_stats_t* out) {
    g_err.clear();
    if (!h || !out) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    if (!h->have_reset) return fail(PA_ERR_STATE, "stats before reset");
    int rc = h->read_ctrl();
    if (rc) return rc;
    fill_stats(h->ctrl_host[0], out);
    for (int n = 1; n < h->d.N; ++n) {
        pa_stats_t o;
        fill_stats(h->ctrl_host[n], &o);
        out->nfe += o.nfe;
        out->hits += o.hits;
        out->misses += o.misses;
        out->revisits += o.revisits;
        out->revisits_below += o.revisits_below;
        if (o.sweeps > out->sweeps) out->sweeps = o.sweeps;
        if (o.window_start < out->window_start) out->window_start = o.window_start;
        if (o.window_end < out->window_end) out->window_end = o.window_end;
        out->done = out->done && o.done;
        out->nonfinite = out->nonfinite || o.nonfinite;
    }
    return PA_OK;
}

int paraanya_stats_sample(paraanya_t* h, int32_t n, pa_stats_t* out) {
    g_err.clear();
    if (!h || !out) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    if (n < 0 || n >= h->d.N) return fail(PA_ERR_INVALID_ARG, "sample %d outside [0, %d)", n, h->d.N);
    if (!h->have_reset) return fail(PA_ERR_STATE, "stats before reset");
    int rc = h->read_ctrl();
    if (rc) return rc;
    fill_stats(h->ctrl_host[n], out);
    return PA_OK;
}

int paraanya_trace_sample(paraanya_t* h, int32_t n, int32_t k, pa_sweep_trace_t* out) {
    g_err.clear();
    if (!h || !out) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    if (!(h->flags & PA_FLAG_TRACE)) return fail(PA_ERR_STATE, "handle created without PA_FLAG_TRACE");
    if (n < 0 || n >= h->d.N) return fail(PA_ERR_INVALID_ARG, "sample %d outside [0, %d)", n, h->d.N);
    if (!h->have_reset) return fail(PA_ERR_STATE, "trace before reset");
    int rc = h->read_ctrl();
    if (rc) return rc;
    if (k < 0 || k >= h->ctrl_host[n].sweep) return fail(PA_ERR_INVALID_ARG, "sweep %d not completed", k);
    PA_HIP(hipMemcpy(out, h->d.trace + (size_t)n * h->d.T + k, sizeof(pa_sweep_trace_t), hipMemcpyDeviceToHost));
    return PA_OK;
}

int paraanya_trace(paraanya_t* h, int32_t k, pa_sweep_trace_t* out) {
    return paraanya_trace_sample(h, 0, k, out);
}

int paraanya_read_state_sample(paraanya_t* h, int32_t n, int32_t t0, int32_t t1, float* X, float* Xh,
                               float* Eh, uint8_t* valid) {
    g_err.clear();
    if (!h) return fail(PA_ERR_INVALID_ARG, "NULL handle");
    const int T = h->d.T;
    if (n < 0 || n >= h->d.N) return fail(PA_ERR_INVALID_ARG, "sample %d outside [0, %d)", n, h->d.N);
    if (t0 < 0 || t1 < t0 || t1 > T + 1) return fail(PA_ERR_INVALID_ARG, "row range [%d, %d) invalid", t0, t1);
    PA_HIP(hipStreamSynchronize(h->stream));
    const size_t D = (size_t)h->d.D;
    const float* Xs = h->d.X + (size_t)n * (T + 1) * D;
    const float* Xhs = h->d.Xh + (size_t)n * T * D;
    const float* Ehs = h->d.Eh + (size_t)n * T * D;
    const uint8_t* vs = h->d.valid + (size_t)n * T;
    const int c1 = t1 < T ? t1 : T;
    if (X && t1 > t0) PA_HIP(hipMemcpy(X, Xs + t0 * D, (size_t)(t1 - t0) * D * 4, hipMemcpyDeviceToHost));
    if (c1 > t0) {
        if (Xh) PA_HIP(hipMemcpy(Xh, Xhs + t0 * D, (size_t)(c1 - t0) * D * 4, hipMemcpyDeviceToHost));
        if (Eh) PA_HIP(hipMemcpy(Eh, Ehs + t0 * D, (size_t)(c1 - t0) * D * 4, hipMemcpyDeviceToHost));
        if (valid) PA_HIP(hipMemcpy(valid, vs + t0, (size_t)(c1 - t0), hipMemcpyDeviceToHost));
    }
    return PA_OK;
}

int paraanya_read_state(paraanya_t* h, int32_t t0, int32_t t1, float* X, float* Xh, float* Eh,
                        uint8_t* valid) {
    return paraanya_read_state_sample(h, 0, t0, t1, X, Xh, Eh, valid);
}

int paraanya_coefficients(paraanya_t* h, double* alpha, double* b, double* sigma, float* temb) {
    g_err.clear();
    if (!h) return fail(PA_ERR_INVALID_ARG, "NULL handle");
    const int T = h->d.T;
    for (int i = 0; i < T; ++i) {
        if (alpha) alpha[i] = h->coef_host[3 * i];
        if (b) b[i] = h->coef_host[3 * i + 1];
        if (sigma) sigma[i] = h->coef_host[3 * i + 2];
    }
    if (temb) {
        if (h->model != PA_EPS_PATCH_MLP) return fail(PA_ERR_INVALID_ARG, "temb requested for a linear model");
        PA_HIP(hipStreamSynchronize(h->stream));
        PA_HIP(hipMemcpy(temb, h->d.temb, (size_t)T * h->d.hidden * 4, hipMemcpyDeviceToHost));
    }
    return PA_OK;
}

int paraanya_kernel_times(paraanya_t* h, pa_ktimes_t* out) {
    g_err.clear();
    if (!h || !out) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    if (!(h->flags & PA_FLAG_PROFILE)) return fail(PA_ERR_STATE, "handle created without PA_FLAG_PROFILE");
    PA_HIP(hipStreamSynchronize(h->stream));
    int rc = h->drain_profile();
    if (rc) return rc;
    rc = h->read_ctrl();
    if (rc) return rc;
    out->launches = h->prof_kernel_launches[0];
    out->eps_ms_total = h->prof_kernel_ms[0];
    out->solver_launches = h->prof_kernel_launches[1];
    out->picard_ms_total = h->prof_kernel_ms[1];
    out->slide_ms_total = h->prof_kernel_ms[2];
    out->eps_latents = 0;
    for (int n = 0; n < h->d.N; ++n) out->eps_latents += h->ctrl_host[n].nfe;
    return PA_OK;
}

void paraanya_destroy(paraanya_t* h) { delete h; }

}  // extern "C"
