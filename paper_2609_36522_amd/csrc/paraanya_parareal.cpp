// Host side of the cached Parareal sampler (include/paraanya.h, "Parareal sampler"):
// validation, coarse and fine step coefficients in fp64, device buffers, and the launch
// sequence of one sample. Every compute step runs in the gfx950 kernels (k_parareal.hip
// and the batched network kernel); the host only orders the launches and waits for each
// iteration's convergence word.
#include <hip/hip_runtime.h>
#include <math.h>
#include <string.h>

#include <new>
#include <vector>

#include "pa_host.h"
#include "pa_parareal.h"

using pa::Ctrl;
using pa::Dev;
using pa::fail;
using pa::hip_fail;
using pa::PrArgs;
using pa::PrCtrl;

struct paraanya_parareal {
    Dev d{};
    hipStream_t stream = nullptr;
    uint32_t flags = 0;
    int model = PA_EPS_LINEAR;
    int B = 0, L = 0;
    int nchunk = 0;
    int max_records = 0;
    int records = 0;                  // requests of the last sample
    bool have_sample = false;
    PrCtrl* pc = nullptr;             // device control block
    uint64_t* progress_host = nullptr;
    pa::DevMem mem;
    pa::KernelTimer timer;
    int64_t timed_latents = 0;        // network latents of the samples the timer covers
    pa_parareal_stats_t last{};       // counters of the last sample, read at its end

    ~paraanya_parareal() {
        (void)hipStreamSynchronize(stream);
        if (progress_host) (void)hipHostFree(progress_host);
    }

    PrArgs args(int mode, int k, int j, int n, int rec) const {
        PrArgs a;
        a.mode = mode;
        a.L = L;
        a.k = k;
        a.j = j;
        a.n = n;
        a.rec = rec;
        a.nchunk = nchunk;
        a.pc = pc;
        return a;
    }

    // One batch of requests: hit test, network on the misses, then the step kernel.
    int request(const PrArgs& a, int step_kernel) {
        PA_HIP(pa::launch_pr(d, a, pa::PRK_TEST, stream));
        if (model == PA_EPS_PATCH_MLP) {
            hipEvent_t e0 = nullptr, e1 = nullptr;
            if (flags & PA_FLAG_PROFILE) {
                const int rc = timer.pair(0, &e0, &e1);
                if (rc) return rc;
            }
            // A coarse request evaluates one latent: 64-token work items spread it over twice
            // as many CUs.
            PA_HIP(pa::launch_eps_mlp(d, stream, e0, e1, step_kernel == pa::PRK_COARSE ? 1 : 0));
        }
        PA_HIP(pa::launch_pr(d, a, step_kernel, stream));
        return PA_OK;
    }

    // Waits for the convergence word of iteration k; returns 1 if done, 0 if not, < 0 on error.
    int wait_iteration(int k) {
        volatile uint64_t* w = progress_host;
        pa::QueryPacer pacer;
        for (unsigned spin = 0;; ++spin) {
            const uint64_t v = *w;
            if ((int)(v >> 32) >= k + 1) return (v >> 31) & 1u ? 1 : 0;
            if (spin % 64 != 63 || !pacer.due()) continue;
            const hipError_t q = hipStreamQuery(stream);
            if (q == hipSuccess) {
                const uint64_t v2 = *w;
                if ((int)(v2 >> 32) >= k + 1) return (v2 >> 31) & 1u ? 1 : 0;
                return fail(PA_ERR_HIP, "Parareal iteration %d did not report", k);
            }
            if (q != hipErrorNotReady) return hip_fail(q, "hipStreamQuery");
        }
    }
};

extern "C" {

int paraanya_parareal_create(const int32_t latent_shape[4], int32_t T, const pa_schedule_t* schedule,
                             int32_t blocks, double delta, double tol, const pa_eps_model_t* eps_model,
                             void* stream, uint32_t flags, paraanya_parareal_t** out) {
    pa::g_err.clear();
    if (!out) return fail(PA_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    // ---- validation: no HIP call before this block completes
    if (!latent_shape || !schedule || !eps_model) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    const int N = latent_shape[0], C = latent_shape[1], Hi = latent_shape[2], Wi = latent_shape[3];
    if (N != 1) return fail(PA_ERR_INVALID_ARG, "Parareal: batch N must be 1 (got %d)", N);
    if (C < 1 || Hi < 1 || Wi < 1) return fail(PA_ERR_INVALID_ARG, "latent dims must be positive");
    const long long Dl = (long long)C * Hi * Wi;
    if (Dl % 4 != 0) return fail(PA_ERR_INVALID_ARG, "C*H*W must be a multiple of 4");
    if (Dl > (1ll << 30)) return fail(PA_ERR_INVALID_ARG, "latent too large");
    if (T < 1 || T > PA_MAX_STEPS) return fail(PA_ERR_INVALID_ARG, "T must be in [1, %d] (got %d)", PA_MAX_STEPS, T);
    if (blocks < 1 || blocks > PA_PR_MAX_BLOCKS || blocks > T || T % blocks)
        return fail(PA_ERR_INVALID_ARG, "blocks must divide T and lie in [1, %d]", PA_PR_MAX_BLOCKS);
    if (!(delta >= 0.0)) return fail(PA_ERR_INVALID_ARG, "delta must be >= 0 (got %g)", delta);
    if (!(tol >= 0.0)) return fail(PA_ERR_INVALID_ARG, "tol must be >= 0 (got %g)", tol);
    if (flags & ~(PA_FLAG_TRACE | PA_FLAG_PROFILE)) return fail(PA_ERR_INVALID_ARG, "unknown flags");
    const int D = (int)Dl;
    int rc = pa::check_eps_model(eps_model, C, Hi, Wi, T);
    if (rc) return rc;
    std::vector<double> ab, tv;
    if ((rc = pa::build_schedule(schedule, T, ab, tv))) return rc;
    if (schedule->eta != 0.0) return fail(PA_ERR_UNSUPPORTED, "Parareal: only the deterministic step (eta = 0) is built");
    const std::vector<double> coef = pa::step_coefficients(ab, T, 0.0);
    const int L = T / blocks;
    // Coarse step of block n: one DDIM step from state nL to state (n+1)L, fp64.
    std::vector<double> pcoef(2 * (size_t)blocks);
    for (int n = 0; n < blocks; ++n) {
        const double a0 = ab[(size_t)n * L], a1 = ab[(size_t)(n + 1) * L];
        const double ac = sqrt(a1 / a0) - 1.0;
        pcoef[2 * n] = ac;
        pcoef[2 * n + 1] = sqrt(1.0 - a1) - (1.0 + ac) * sqrt(1.0 - a0);
    }

    // ---- resources
    paraanya_parareal* h = new (std::nothrow) paraanya_parareal();
    if (!h) return fail(PA_ERR_OOM, "host allocation failed");
    h->stream = (hipStream_t)stream;
    h->flags = flags;
    h->model = eps_model->kind;
    h->B = blocks;
    h->L = L;
    h->nchunk = pa::pr_chunks(D);
    h->max_records = blocks + L * blocks * (blocks + 1) / 2 + blocks * (blocks - 1) / 2;
    Dev& d = h->d;
    d.N = blocks; d.T = T; d.P = 1; d.D = D; d.C = C; d.Himg = Hi; d.Wimg = Wi;
    d.delta = delta; d.tol = tol;
    auto bail = [&](int code) { delete h; return code; };

    int dev_id = 0;
    hipError_t he = hipGetDevice(&dev_id);
    if (he != hipSuccess) return bail(hip_fail(he, "hipGetDevice"));
    int cus = 0;
    he = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev_id);
    if (he != hipSuccess) return bail(hip_fail(he, "hipDeviceGetAttribute"));

    const size_t Dz = (size_t)D, Bz = (size_t)blocks;
    pa::DevMem& m = h->mem;
    if ((rc = m.alloc(&d.X, (Bz + 1) * (T + 1) * Dz, "X"))) return bail(rc);
    if ((rc = m.alloc(&d.Xh, (size_t)T * Dz, "Xh"))) return bail(rc);
    if ((rc = m.alloc(&d.Eh, (size_t)T * Dz, "Eh"))) return bail(rc);
    if ((rc = m.alloc(&d.valid, (size_t)T, "valid"))) return bail(rc);
    if ((rc = m.alloc(&d.coef, 3 * (size_t)T, "coef"))) return bail(rc);
    if ((rc = m.alloc(&d.pr_coef, 2 * Bz, "pr_coef"))) return bail(rc);
    if ((rc = m.alloc(&d.Gc, Bz * Dz, "Gc"))) return bail(rc);
    if ((rc = m.alloc(&d.part_res, (Bz + 1) * h->nchunk, "part_res"))) return bail(rc);
    if ((rc = m.alloc(&d.ctrl, Bz, "ctrl"))) return bail(rc);
    if ((rc = m.alloc(&h->pc, 1, "pr_ctrl"))) return bail(rc);
    if (flags & PA_FLAG_TRACE) {
        if ((rc = m.alloc(&d.trace_pr, (size_t)h->max_records, "trace_pr"))) return bail(rc);
        if ((rc = m.alloc(&d.trace_eps, (size_t)h->max_records * Dz, "trace_eps"))) return bail(rc);
        if ((rc = m.alloc(&d.trace_res, Bz * (Bz + 1), "trace_res"))) return bail(rc);
    }
    he = hipHostMalloc((void**)&h->progress_host, 256, hipHostMallocMapped | hipHostMallocCoherent);
    if (he != hipSuccess) return bail(hip_fail(he, "hipHostMalloc(progress)"));
    *h->progress_host = 0;
    he = hipHostGetDevicePointer((void**)&d.progress, h->progress_host, 0);
    if (he != hipSuccess) return bail(hip_fail(he, "hipHostGetDevicePointer"));
    he = hipMemcpyAsync(d.coef, coef.data(), coef.size() * sizeof(double), hipMemcpyHostToDevice, h->stream);
    if (he != hipSuccess) return bail(hip_fail(he, "hipMemcpyAsync(coef)"));
    he = hipMemcpyAsync(d.pr_coef, pcoef.data(), pcoef.size() * sizeof(double), hipMemcpyHostToDevice, h->stream);
    if (he != hipSuccess) return bail(hip_fail(he, "hipMemcpyAsync(pr_coef)"));
    he = hipMemsetAsync(d.ctrl, 0, Bz * sizeof(Ctrl), h->stream);
    if (he != hipSuccess) return bail(hip_fail(he, "hipMemsetAsync(ctrl)"));
    if ((rc = pa::setup_network(d, m, eps_model, tv.data(), cus, Bz, h->stream))) return bail(rc);
    // The host vectors above die at return: wait for the copies that read them.
    he = hipStreamSynchronize(h->stream);
    if (he != hipSuccess) return bail(hip_fail(he, "hipStreamSynchronize"));
    *out = h;
    return PA_OK;
}

int paraanya_parareal_sample(paraanya_parareal_t* h, const float* x_init, float* x_out) {
    pa::g_err.clear();
    if (!h || !x_init || !x_out) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    Dev& d = h->d;
    const int B = h->B, L = h->L, T = d.T;
    const size_t D = (size_t)d.D, rows = (size_t)T + 1;
    PA_HIP(hipStreamSynchronize(h->stream));      // nothing of an earlier sample still runs
    *h->progress_host = 0;
    PA_HIP(hipMemcpyAsync(d.X, x_init, D * sizeof(float), hipMemcpyDeviceToDevice, h->stream));
    PA_HIP(pa::launch_pr(d, h->args(pa::PR_INIT, 0, 0, 0, 0), pa::PRK_RESET, h->stream));
    int rc, rec = 0;
    // initialization: U_{n+1} = G_n(U_n), serially
    for (int n = 0; n < B; ++n, ++rec)
        if ((rc = h->request(h->args(pa::PR_INIT, 0, 0, n, rec), pa::PRK_COARSE))) return rc;
    for (int k = 0; k < B; ++k) {
        for (int j = 0; j < L; ++j) {
            if ((rc = h->request(h->args(pa::PR_FINE, k, j, 0, rec), pa::PRK_FINE))) return rc;
            rec += B - k;
        }
        PA_HIP(pa::launch_pr(d, h->args(pa::PR_COPY, k, 0, k, rec), pa::PRK_COARSE, h->stream));
        for (int n = k + 1; n < B; ++n, ++rec)
            if ((rc = h->request(h->args(pa::PR_COARSE, k, 0, n, rec), pa::PRK_COARSE))) return rc;
        PA_HIP(pa::launch_pr(d, h->args(pa::PR_COARSE, k, 0, 0, rec), pa::PRK_CHECK, h->stream));
        const int done = h->wait_iteration(k);
        if (done < 0) return done;
        if (done) break;
    }
    h->records = rec;
    h->have_sample = true;
    PA_HIP(hipMemcpyAsync(x_out, d.X + ((size_t)B * rows + T) * D, D * sizeof(float),
                          hipMemcpyDeviceToDevice, h->stream));
    PrCtrl pc;
    std::vector<Ctrl> c((size_t)B);
    PA_HIP(hipMemcpyAsync(&pc, h->pc, sizeof(PrCtrl), hipMemcpyDeviceToHost, h->stream));
    PA_HIP(hipMemcpyAsync(c.data(), d.ctrl, c.size() * sizeof(Ctrl), hipMemcpyDeviceToHost, h->stream));
    PA_HIP(hipStreamSynchronize(h->stream));
    pa_parareal_stats_t& st = h->last;
    memset(&st, 0, sizeof st);
    for (const Ctrl& x : c) {
        st.nfe += x.nfe;
        st.hits += x.hits;
    }
    st.requests = st.nfe + st.hits;
    st.iterations = pc.iters;
    st.done = pc.done;
    st.nonfinite = pc.nonfinite;
    h->timed_latents += st.nfe;
    // The stream is idle: fold this sample's event pairs into the running totals, so the
    // pool stays at one sample's launches however many samples run between reads.
    if (h->flags & PA_FLAG_PROFILE)
        if ((rc = h->timer.drain())) return rc;
    if (pc.nonfinite) return fail(PA_ERR_NONFINITE, "non-finite boundary residual");
    return PA_OK;
}

int paraanya_parareal_stats(paraanya_parareal_t* h, pa_parareal_stats_t* out) {
    pa::g_err.clear();
    if (!h || !out) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    if (!h->have_sample) return fail(PA_ERR_STATE, "stats before the first sample");
    *out = h->last;   // read back at the end of the sample; nothing has run since
    return PA_OK;
}

int paraanya_parareal_trace(paraanya_parareal_t* h, int32_t i, pa_request_trace_t* out, float* eps) {
    pa::g_err.clear();
    if (!h || !out) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    if (!(h->flags & PA_FLAG_TRACE)) return fail(PA_ERR_STATE, "handle created without PA_FLAG_TRACE");
    if (!h->have_sample) return fail(PA_ERR_STATE, "trace before the first sample");
    if (i < 0 || i >= h->records) return fail(PA_ERR_INVALID_ARG, "request %d outside [0, %d)", i, h->records);
    PA_HIP(hipStreamSynchronize(h->stream));
    PA_HIP(hipMemcpy(out, h->d.trace_pr + i, sizeof *out, hipMemcpyDeviceToHost));
    if (eps && !out->hit)
        PA_HIP(hipMemcpy(eps, h->d.trace_eps + (size_t)i * h->d.D, (size_t)h->d.D * sizeof(float),
                         hipMemcpyDeviceToHost));
    return PA_OK;
}

int paraanya_parareal_residuals(paraanya_parareal_t* h, int32_t k, double* r) {
    pa::g_err.clear();
    if (!h || !r) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    if (!(h->flags & PA_FLAG_TRACE)) return fail(PA_ERR_STATE, "handle created without PA_FLAG_TRACE");
    if (!h->have_sample) return fail(PA_ERR_STATE, "residuals before the first sample");
    PrCtrl pc;
    PA_HIP(hipStreamSynchronize(h->stream));
    PA_HIP(hipMemcpy(&pc, h->pc, sizeof(PrCtrl), hipMemcpyDeviceToHost));
    if (k < 0 || k >= pc.iters) return fail(PA_ERR_INVALID_ARG, "iteration %d not completed", k);
    PA_HIP(hipMemcpy(r, h->d.trace_res + (size_t)k * (h->B + 1), (size_t)(h->B + 1) * sizeof(double),
                     hipMemcpyDeviceToHost));
    for (int n = 0; n <= k; ++n) r[n] = 0.0;
    return PA_OK;
}

int paraanya_parareal_read_boundaries(paraanya_parareal_t* h, float* U) {
    pa::g_err.clear();
    if (!h || !U) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    const size_t D = (size_t)h->d.D, rows = (size_t)h->d.T + 1;
    PA_HIP(hipStreamSynchronize(h->stream));
    for (int n = 0; n <= h->B; ++n)
        PA_HIP(hipMemcpy(U + (size_t)n * D, h->d.X + ((size_t)n * rows + (size_t)n * h->L) * D,
                         D * sizeof(float), hipMemcpyDeviceToHost));
    return PA_OK;
}

int paraanya_parareal_kernel_times(paraanya_parareal_t* h, pa_ktimes_t* out) {
    pa::g_err.clear();
    if (!h || !out) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    if (!(h->flags & PA_FLAG_PROFILE)) return fail(PA_ERR_STATE, "handle created without PA_FLAG_PROFILE");
    PA_HIP(hipStreamSynchronize(h->stream));
    int rc = h->timer.drain();
    if (rc) return rc;
    memset(out, 0, sizeof *out);
    out->launches = h->timer.launches[0];
    out->eps_ms_total = h->timer.ms[0];
    out->eps_latents = h->timed_latents;
    h->timer.clear();
    h->timed_latents = 0;
    return PA_OK;
}

void paraanya_parareal_destroy(paraanya_parareal_t* h) { delete h; }

}  // extern "C"
