// Host side of the C ABI declared in include/paraanya.h: argument validation (before any
// HIP call), schedule and DDIM coefficients in fp64, device buffers and weight layouts,
// the sweep enqueue loop. Every compute step of a sweep runs in the gfx950 kernels.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stddef.h>
#include <string.h>

#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "pa_host.h"

using pa::Ctrl;
using pa::Dev;
using pa::fail;
using pa::hip_fail;

struct paraanya {
    Dev d{};
    hipStream_t stream = nullptr;
    uint32_t flags = 0;
    int model = PA_EPS_LINEAR;
    std::vector<double> coef_host;    // [T][3] as uploaded
    Ctrl* ctrl_host = nullptr;        // pinned mirror, one block per sample
    uint64_t* progress_host = nullptr; // pinned, device-mapped: [N] progress words, then [N][4]
                                       // final counter words (see publish_progress, slide_core)
    float* noise_buf = nullptr;       // [N][T][D] step noise (eta > 0)
    bool noise_set = false;
    bool ctrl_fresh = false;           // ctrl_host matches the device and nothing is queued
    bool have_reset = false;
    bool host_done = false;           // done flag of the last synchronized read
    pa::DevMem mem;                   // device allocations
    pa::KernelTimer timer;            // kinds: 0 network, 1 Picard, 2 slide
    int64_t timed_latents = 0;        // network latents of the samples the timer covers
    bool slide_pending = false;       // fused sweep: the last sweep's slide is not computed yet
    bool head_valid = false;          // ctrl_host's counters are final (taken from the counter
                                      // words by paraanya_sample; work may still be queued)
    bool progress_quiet = false;      // nothing queued can still write a progress word

    ~paraanya() {
        (void)hipStreamSynchronize(stream);
        if (ctrl_host) (void)hipHostFree(ctrl_host);
        if (progress_host) (void)hipHostFree(progress_host);
    }

    template <class T>
    int alloc(T** p, size_t count, const char* what) { return mem.alloc(p, count, what); }

    int read_ctrl() {
        // The mirror stays valid until the next enqueue, so repeated queries cost nothing.
        if (ctrl_fresh) return PA_OK;
        if (slide_pending) {
            // Fused sweep: bring the control block up to date (the next network kernel computes
            // the same slide again and writes the same values).
            PA_HIP(pa::launch_slide_pending(d, stream));
            slide_pending = false;
        }
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

    // Every sample is done (its progress word says so): fills the counters of ctrl_host from
    // the done words and the final counter words the last slide wrote before them, if all of
    // those carry this sample's epoch (else the caller reads the control blocks the
    // synchronizing way). The words are written by the device with system-scope stores that
    // may reach host memory in any order, hence the epoch tag on each.
    bool take_final_counters() {
        const volatile uint64_t* w = progress_host;
        const volatile uint64_t* cw = progress_host + d.N;
        const uint64_t tag = (uint64_t)(d.epoch & 0xffffffu);
        uint64_t v[PA_MAX_BATCH][4];
        for (int n = 0; n < d.N; ++n)
            for (int k = 0; k < 4; ++k) {
                v[n][k] = cw[4 * n + k];
                if ((v[n][k] >> 40) != tag) return false;
            }
        for (int n = 0; n < d.N; ++n) {
            const uint64_t p = w[n];
            Ctrl& c = ctrl_host[n];
            c.sweep = (int32_t)(p >> 32);
            c.done = (int32_t)((p >> 31) & 1u);
            c.nonfinite = (int32_t)((p >> 30) & 1u);
            c.s = (int32_t)(p & 0x3fffffffu);
            c.e = c.s + d.P < d.T ? c.s + d.P : d.T;
            const uint64_t mask = (1ull << 40) - 1;
            c.nfe = (int64_t)(v[n][0] & mask);
            c.hits = (int64_t)(v[n][1] & mask);
            c.revisits = (int64_t)(v[n][2] & mask);
            c.revisits_below = (int64_t)(v[n][3] & mask);
        }
        head_valid = true;
        return true;
    }

    // Start/stop events of one timed launch of kernel kind k, or nulls when untimed. Samples
    // drain the pool when they end; a handle driven sweep by sweep drains it (after waiting
    // for the stream) once kMaxPendingPairs launches are pending.
    static constexpr size_t kMaxPendingPairs = 4096;
    int timed(int k, hipEvent_t* e0, hipEvent_t* e1) {
        *e0 = *e1 = nullptr;
        if (!(flags & PA_FLAG_PROFILE)) return PA_OK;
        if (k > 0 && !(flags & PA_FLAG_PROFILE_SOLVER)) return PA_OK;
        if (timer.pending() >= kMaxPendingPairs) {
            PA_HIP(hipStreamSynchronize(stream));
            const int rc = timer.drain();
            if (rc) return rc;
        }
        return timer.pair(k, e0, e1);
    }

    int enqueue_sweep() {
        // The miss list of this sweep was published by the previous k_slide (or k_reset).
        // Under PROFILE every timed launch carries its own start/stop events (no marker
        // packets between kernels).
        ctrl_fresh = false;
        head_valid = false;
        hipEvent_t e0, e1;
        int rc;
        if (model == PA_EPS_PATCH_MLP) {
            if ((rc = timed(0, &e0, &e1))) return rc;
            PA_HIP(pa::launch_eps_mlp(d, stream, e0, e1));
        }
        if ((rc = timed(1, &e0, &e1))) return rc;
        PA_HIP(pa::launch_picard(d, stream, model == PA_EPS_LINEAR, e0, e1));
        if (d.fused_slide) {
            // The slide runs at the start of the next network kernel (or of a finishing
            // k_slide when the host needs the control block first).
            slide_pending = true;
            return PA_OK;
        }
        if ((rc = timed(2, &e0, &e1))) return rc;
        PA_HIP(pa::launch_slide(d, stream, e0, e1));
        return PA_OK;
    }
};

extern "C" {

const char* paraanya_last_error(void) { return pa::g_err.c_str(); }

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

}  // extern "C"

namespace {

// Validated arguments of a sampler request.
struct Request {
    int N, C, Hi, Wi, D, T, P;
    double delta, tol, eta;
    const pa_eps_model_t* em;
};

// Argument checks shared by paraanya_create and paraanya_sample_noalloc; no HIP call.
int validate(const int32_t latent_shape[4], int32_t T, const pa_schedule_t* schedule, int32_t window,
             double delta, double tol, const pa_eps_model_t* eps_model, Request* r) {
    if (!latent_shape || !schedule || !eps_model) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    const int N = latent_shape[0], C = latent_shape[1], Hi = latent_shape[2], Wi = latent_shape[3];
    if (N < 1 || N > PA_MAX_BATCH) return fail(PA_ERR_INVALID_ARG, "batch N must be in [1, %d] (got %d)", PA_MAX_BATCH, N);
    if (C < 1 || Hi < 1 || Wi < 1) return fail(PA_ERR_INVALID_ARG, "latent dims must be positive");
    const long long Dl = (long long)C * Hi * Wi;
    if (Dl % 4 != 0) return fail(PA_ERR_INVALID_ARG, "C*H*W must be a multiple of 4");
    if (Dl > (1ll << 30)) return fail(PA_ERR_INVALID_ARG, "latent too large");
    if (T < 1 || T > PA_MAX_STEPS) return fail(PA_ERR_INVALID_ARG, "T must be in [1, %d] (got %d)", PA_MAX_STEPS, T);
    if (window < 1 || window > T || window > PA_MAX_WINDOW)
        return fail(PA_ERR_INVALID_ARG, "window must be in [1, min(T, %d)]", PA_MAX_WINDOW);
    if (!(delta >= 0.0)) return fail(PA_ERR_INVALID_ARG, "delta must be >= 0 (got %g)", delta);
    if (!(tol >= 0.0)) return fail(PA_ERR_INVALID_ARG, "tol must be >= 0 (got %g)", tol);
    int rc = pa::check_eps_model(eps_model, C, Hi, Wi, T);
    if (rc) return rc;
    *r = Request{N, C, Hi, Wi, (int)Dl, T, window, delta, tol, schedule->eta, eps_model};
    return PA_OK;
}

// Geometry and device buffers of a handle (allocated, or carved from a workspace, by h->mem);
// coef: the [T][3] step coefficients (host), tv: the T time values (host). The pinned host
// mirror and progress words are the caller's business. Enqueues the uploads on h->stream.
int setup_handle(paraanya* h, const Request& q, const double* coef, const double* tv) {
    Dev& d = h->d;
    d.N = q.N; d.T = q.T; d.P = q.P; d.D = q.D; d.C = q.C; d.Himg = q.Hi; d.Wimg = q.Wi;
    d.delta = q.delta; d.tol = q.tol;
    d.revisit_thr = 0.05;
    d.picard_blocks = pa::picard_blocks(q.D, q.P);
    h->model = q.em->kind;
    int dev_id = 0;
    PA_HIP(hipGetDevice(&dev_id));
    int cus = 0;
    PA_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev_id));
    const size_t Dz = (size_t)q.D, Nz = (size_t)q.N, T = (size_t)q.T, P = (size_t)q.P;
    int rc;
    if ((rc = h->alloc(&d.X, Nz * (T + 1) * Dz, "X"))) return rc;
    if ((rc = h->alloc(&d.Xh, Nz * T * Dz, "Xh"))) return rc;
    if ((rc = h->alloc(&d.Eh, Nz * T * Dz, "Eh"))) return rc;
    if ((rc = h->alloc(&d.valid, Nz * T, "valid"))) return rc;
    if ((rc = h->alloc(&d.coef, 3 * T, "coef"))) return rc;
    if ((rc = h->alloc(&d.part_res, Nz * P * d.picard_blocks, "part_res"))) return rc;
    if ((rc = h->alloc(&d.part_dev, Nz * P * d.picard_blocks, "part_dev"))) return rc;
    if ((rc = h->alloc(&d.ctrl, Nz, "ctrl"))) return rc;
    // Fused sweep (network -> Picard, the slide computed by every block of the next network
    // kernel): one sample, patch-MLP, and a partial-sum volume that a block reduces quickly.
    d.fused_slide = (q.em->kind == PA_EPS_PATCH_MLP && q.N == 1 &&
                     2 * P * d.picard_blocks * sizeof(double) <= pa::kFusedSlideMaxBytes) ? 1 : 0;
    if ((rc = h->alloc(&d.pre, Nz, "pre"))) return rc;
    if (h->flags & PA_FLAG_TRACE)
        if ((rc = h->alloc(&d.trace, Nz * T, "trace"))) return rc;
    if (q.eta > 0.0) {
        if ((rc = h->alloc(&h->noise_buf, Nz * T * Dz, "noise"))) return rc;
        d.noise = h->noise_buf;
    }
    // Whole network outputs written straight into the cache (unless split ones are forced).
    if (q.em->kind == PA_EPS_PATCH_MLP && !(h->flags & PA_FLAG_SPLIT_OUTPUTS))
        if ((rc = h->alloc(&d.eps_whole, 1, "eps_whole"))) return rc;
    // setup_network takes all its buffers before it enqueues anything, so a request that does
    // not fit fails before the first upload.
    if ((rc = pa::setup_network(d, h->mem, q.em, tv, cus, Nz * P, h->stream))) return rc;
    PA_HIP(hipMemcpyAsync(d.coef, coef, 3 * T * sizeof(double), hipMemcpyHostToDevice, h->stream));
    return PA_OK;
}

}  // namespace

extern "C" {

int paraanya_create(const int32_t latent_shape[4], int32_t T, const pa_schedule_t* schedule,
                    int32_t window, double delta, double tol, const pa_eps_model_t* eps_model,
                    void* stream, uint32_t flags, paraanya_t** out) {
    pa::g_err.clear();
    if (!out) return fail(PA_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    // ---- validation: no HIP call before this block completes
    Request q;
    int rc = validate(latent_shape, T, schedule, window, delta, tol, eps_model, &q);
    if (rc) return rc;
    if (flags & ~(PA_FLAG_TRACE | PA_FLAG_PROFILE | PA_FLAG_PROFILE_SOLVER | PA_FLAG_SPLIT_OUTPUTS))
        return fail(PA_ERR_INVALID_ARG, "unknown flags");
    std::vector<double> ab, tv;
    if ((rc = pa::build_schedule(schedule, T, ab, tv))) return rc;
    std::vector<double> coef = pa::step_coefficients(ab, T, q.eta);

    // ---- resources
    paraanya* h = new (std::nothrow) paraanya();
    if (!h) return fail(PA_ERR_OOM, "host allocation failed");
    h->stream = (hipStream_t)stream;
    h->flags = flags;
    h->coef_host = coef;
    auto bail = [&](int code) { delete h; return code; };
    if ((rc = setup_handle(h, q, coef.data(), tv.data()))) return bail(rc);
    Dev& d = h->d;
    const size_t Nz = (size_t)q.N;
    hipError_t he = hipHostMalloc((void**)&h->ctrl_host, Nz * sizeof(Ctrl), hipHostMallocDefault);
    if (he != hipSuccess) return bail(hip_fail(he, "hipHostMalloc"));
    memset(h->ctrl_host, 0, Nz * sizeof(Ctrl));
    // Progress words [N], then the final counter words [N][4].
    const size_t words = 5 * Nz;
    he = hipHostMalloc((void**)&h->progress_host, words * sizeof(uint64_t) < 256 ? 256 : words * sizeof(uint64_t),
                       hipHostMallocMapped | hipHostMallocCoherent);
    if (he != hipSuccess) return bail(hip_fail(he, "hipHostMalloc(progress)"));
    for (size_t i = 0; i < words; ++i) h->progress_host[i] = 0;
    he = hipHostGetDevicePointer((void**)&d.progress, h->progress_host, 0);
    if (he != hipSuccess) return bail(hip_fail(he, "hipHostGetDevicePointer"));
    d.counters = d.progress + Nz;
    // The host vectors above die at return: wait for the uploads that read them.
    he = hipStreamSynchronize(h->stream);
    if (he != hipSuccess) return bail(hip_fail(he, "hipStreamSynchronize"));
    *out = h;
    return PA_OK;
}

int paraanya_reset(paraanya_t* h, const float* x_init) {
    pa::g_err.clear();
    if (!h || !x_init) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    if (h->noise_buf && !h->noise_set) return fail(PA_ERR_STATE, "eta > 0: set the step noise first (paraanya_set_noise)");
    // No kernel of this handle may still publish progress from an earlier sample. After a
    // paraanya_sample that saw every sample done, none can (the slide that published done was
    // the last writer; later queued sweeps leave at once), so the stream need not be drained.
    if (!h->progress_quiet) PA_HIP(hipStreamSynchronize(h->stream));
    h->progress_quiet = false;
    for (int n = 0; n < h->d.N; ++n) h->progress_host[n] = 0;
    h->d.epoch = (h->d.epoch + 1) & 0xffffffu;    // counter words of this sample carry it
    h->ctrl_fresh = false;
    h->head_valid = false;
    const size_t row = (size_t)h->d.D * sizeof(float);
    PA_HIP(hipMemcpy2DAsync(h->d.X, (size_t)(h->d.T + 1) * row, x_init, row, row, (size_t)h->d.N,
                            hipMemcpyDeviceToDevice, h->stream));
    PA_HIP(pa::launch_reset(h->d, h->stream));
    h->slide_pending = false;
    h->have_reset = true;
    h->host_done = false;
    return PA_OK;
}

int paraanya_set_noise(paraanya_t* h, const float* z) {
    pa::g_err.clear();
    if (!h || !z) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    if (!h->noise_buf) return fail(PA_ERR_INVALID_ARG, "handle has eta = 0: no step noise");
    PA_HIP(hipMemcpyAsync(h->noise_buf, z, (size_t)h->d.N * h->d.T * h->d.D * sizeof(float),
                          hipMemcpyDeviceToDevice, h->stream));
    h->noise_set = true;
    return PA_OK;
}

int paraanya_set_revisit_threshold(paraanya_t* h, double threshold) {
    pa::g_err.clear();
    if (!h) return fail(PA_ERR_INVALID_ARG, "NULL handle");
    if (!(threshold >= 0.0)) return fail(PA_ERR_INVALID_ARG, "threshold must be >= 0 (got %g)", threshold);
    h->d.revisit_thr = threshold;
    return PA_OK;
}

int paraanya_sweep(paraanya_t* h, int32_t* done) {
    pa::g_err.clear();
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
    pa::g_err.clear();
    if (!h || !x_init || !x_out) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    int rc = paraanya_reset(h, x_init);
    if (rc) return rc;
    const int T = h->d.T, P = h->d.P, N = h->d.N;
    // Launch loop without per-sweep synchronisation: the window slide (k_slide, or the next
    // network kernel in a fused sweep) publishes (completed sweeps, done, s) of every sample to
    // a pinned host word after each sweep; the host keeps enough sweeps in flight -- at least
    // the kLookahead next ones and at least the ceil((T - s)/P) that the slowest sample
    // certainly still needs (s advances by at most P per sweep) -- and stops enqueuing once
    // every sample is done. Sweeps enqueued after that exit at their first instruction. Every
    // sweep advances each unfinished sample's s by at least 1, so at most T sweeps are ever
    // enqueued (T + 1 for a fused sweep, see below). The stream is polled (at most once per
    // millisecond, see QueryPacer) while waiting, so a failed or idle stream ends the loop.
    constexpr int kLookahead = 2;
    volatile uint64_t* prog = h->progress_host;
    auto scan = [&](int* completed, int* need) {      // returns true once all are done
        bool all = true;
        *completed = 0;
        *need = 0;
        for (int n = 0; n < N; ++n) {
            const uint64_t w = prog[n];
            const int c = (int)(w >> 32), s_now = (int)(w & 0x3fffffffu);
            if (c > *completed) *completed = c;
            if ((w >> 31) & 1u) continue;
            all = false;
            const int q = (T - s_now + P - 1) / P;
            if (q > *need) *need = q;
        }
        return all;
    };
    // A fused sweep's slide runs in the next sweep's network kernel, so the sweep that finishes
    // the sample is followed by one more (its network kernel only computes that slide).
    const int cap = T + (h->d.fused_slide ? 1 : 0);
    int enqueued = 0;
    pa::QueryPacer pacer;
    for (unsigned spin = 0;; ++spin) {
        int completed, need;
        if (scan(&completed, &need)) break;
        const int want = completed + (need > kLookahead ? need : kLookahead);
        if (enqueued < want && enqueued < cap) {
            const int k = (want < cap ? want : cap) - enqueued;
            for (int i = 0; i < k; ++i)
                if ((rc = h->enqueue_sweep())) return rc;
            enqueued += k;
            continue;
        }
        if (spin % 64 != 63 || !pacer.due()) continue;   // poll the stream rarely, not per spin
        const hipError_t q = hipStreamQuery(h->stream);
        if (q == hipSuccess) {
            // Stream idle: the words are final for the enqueued work.
            if (scan(&completed, &need)) break;
            if (enqueued >= cap) return fail(PA_ERR_HIP, "sampler did not finish within T sweeps");
        } else if (q != hipErrorNotReady) {
            return hip_fail(q, "hipStreamQuery");
        }
    }
    // Every sample is done: the slide that published that also wrote the control block, so no
    // finishing slide is needed. The output copy is queued behind the sample's last kernels.
    h->slide_pending = false;
    const size_t row = (size_t)h->d.D * sizeof(float);
    PA_HIP(hipMemcpy2DAsync(x_out, row, h->d.X + (size_t)T * h->d.D, (size_t)(T + 1) * row, row,
                            (size_t)N, hipMemcpyDeviceToDevice, h->stream));
    h->ctrl_fresh = false;
    h->host_done = true;
    if (!(h->flags & PA_FLAG_PROFILE) && h->take_final_counters()) {
        // No synchronization: the counters came with the done words, and what is still queued
        // (the tail of the last kernels, the copy) is ordered before the caller's next work on
        // the stream.
        h->progress_quiet = true;
    } else {
        if ((rc = h->read_ctrl())) return rc;
        for (int n = 0; n < N; ++n) h->timed_latents += h->ctrl_host[n].nfe;
        // The stream is idle (read_ctrl synchronized it): fold this sample's event pairs into
        // the running totals, so the pool stays at one sample's launches.
        if (h->flags & PA_FLAG_PROFILE)
            if ((rc = h->timer.drain())) return rc;
    }
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
    pa::g_err.clear();
    if (!h || !out) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    if (!h->have_reset) return fail(PA_ERR_STATE, "stats before reset");
    int rc = h->head_valid ? PA_OK : h->read_ctrl();
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
    pa::g_err.clear();
    if (!h || !out) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    if (n < 0 || n >= h->d.N) return fail(PA_ERR_INVALID_ARG, "sample %d outside [0, %d)", n, h->d.N);
    if (!h->have_reset) return fail(PA_ERR_STATE, "stats before reset");
    int rc = h->head_valid ? PA_OK : h->read_ctrl();
    if (rc) return rc;
    fill_stats(h->ctrl_host[n], out);
    return PA_OK;
}

int paraanya_trace_sample(paraanya_t* h, int32_t n, int32_t k, pa_sweep_trace_t* out) {
    pa::g_err.clear();
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
    pa::g_err.clear();
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
    pa::g_err.clear();
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
    pa::g_err.clear();
    if (!h || !out) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    if (!(h->flags & PA_FLAG_PROFILE)) return fail(PA_ERR_STATE, "handle created without PA_FLAG_PROFILE");
    PA_HIP(hipStreamSynchronize(h->stream));
    int rc = h->timer.drain();
    if (rc) return rc;
    rc = h->read_ctrl();
    if (rc) return rc;
    out->launches = h->timer.launches[0];
    out->eps_ms_total = h->timer.ms[0];
    out->solver_launches = h->timer.launches[1];
    out->picard_ms_total = h->timer.ms[1];
    out->slide_ms_total = h->timer.ms[2];
    out->eps_latents = h->timed_latents;
    h->timer.clear();
    h->timed_latents = 0;
    return PA_OK;
}

void paraanya_destroy(paraanya_t* h) { delete h; }

}  // extern "C"

// ---------------------------------------------------------------------------- no allocation
namespace {

constexpr int kMaxDevices = 64;

// Workspace of paraanya_sample_noalloc. Every device the library runs on holds its own copy
// until the process ends. In host code the name stands for a host-side shadow, not a device
// address: host code uses only the device address hipGetSymbolAddress returns for the
// current device (g_scratch_addr), for the kernels' arguments and every copy.
static __device__ __align__(256) unsigned char scratch[PA_NOALLOC_WORKSPACE_BYTES];

std::mutex g_scratch_lock[kMaxDevices];   // one call at a time per device shares the workspace
void* g_scratch_addr[kMaxDevices];        // device address of scratch, per device (under the lock)

// Leading fields of a control block (the counters and the window), read back at the end.
constexpr size_t kCtrlHead = offsetof(Ctrl, miss_idx);

}  // namespace

extern "C" {

int paraanya_sample_noalloc(const int32_t latent_shape[4], int32_t T, const pa_schedule_t* schedule,
                            int32_t window, double delta, double tol, const pa_eps_model_t* eps_model,
                            void* stream, const float* x_init, float* x_out, pa_stats_t* stats) {
    pa::g_err.clear();
    if (!x_init || !x_out) return fail(PA_ERR_INVALID_ARG, "NULL argument");
    Request q;
    int rc = validate(latent_shape, T, schedule, window, delta, tol, eps_model, &q);
    if (rc) return rc;
    if (T > PA_NOALLOC_MAX_STEPS)
        return fail(PA_ERR_INVALID_ARG, "allocation-free sampling: T must be at most %d (got %d)", PA_NOALLOC_MAX_STEPS, T);
    if (schedule->eta != 0.0)
        return fail(PA_ERR_UNSUPPORTED, "allocation-free sampling: only the deterministic step (eta = 0) is built");
    // Schedule tables on the stack (no host allocation either).
    double ab[PA_NOALLOC_MAX_STEPS + 1], tv[PA_NOALLOC_MAX_STEPS], coef[3 * PA_NOALLOC_MAX_STEPS];
    if ((rc = pa::build_schedule(schedule, T, ab, tv))) return rc;
    pa::step_coefficients(ab, T, 0.0, coef);

    int dev = 0;
    PA_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices)
        return fail(PA_ERR_UNSUPPORTED, "allocation-free sampling: device %d beyond the first %d", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_lock[dev]);
    if (!g_scratch_addr[dev]) {
        void* p = nullptr;
        PA_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));   // this device's copy
        if (!p) return fail(PA_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
        g_scratch_addr[dev] = p;
    }

    // A handle on the stack: its containers stay empty; every buffer is carved from the
    // workspace in order (the carve fails before anything is enqueued if it does not fit).
    paraanya h;
    h.stream = (hipStream_t)stream;
    h.flags = 0;
    h.mem.workspace(g_scratch_addr[dev], PA_NOALLOC_WORKSPACE_BYTES);
    Dev& d = h.d;
    const size_t Nz = (size_t)q.N;
    if ((rc = h.alloc(&d.progress, Nz, "progress"))) return rc;
    if ((rc = setup_handle(&h, q, coef, tv))) return rc;

    // Reset. The workspace keeps the previous call's contents: the progress words are
    // cleared here; the reset kernel clears the cache flags and the control blocks.
    const size_t row = (size_t)q.D * sizeof(float);
    PA_HIP(hipMemsetAsync(d.progress, 0, Nz * sizeof(uint64_t), h.stream));
    PA_HIP(hipMemcpy2DAsync(d.X, (size_t)(T + 1) * row, x_init, row, row, Nz, hipMemcpyDeviceToDevice, h.stream));
    PA_HIP(pa::launch_reset(d, h.stream));
    h.have_reset = true;

    // Sweeps in batches: the progress words are device memory here, so the host reads them
    // back after each batch and enqueues the ceil((T - s)/P) sweeps that the slowest sample
    // certainly still needs (at least one). A fused sweep publishes its slide from the next
    // network kernel, so one sweep beyond T may be needed; later sweeps exit at once.
    const int cap = T + (d.fused_slide ? 1 : 0);
    int enqueued = 0, need = (T + q.P - 1) / q.P;
    uint64_t words[PA_MAX_BATCH];
    for (;;) {
        const int k = need < cap - enqueued ? need : cap - enqueued;
        if (k <= 0) return fail(PA_ERR_HIP, "sampler did not finish within T sweeps");
        for (int i = 0; i < k; ++i)
            if ((rc = h.enqueue_sweep())) return rc;
        enqueued += k;
        PA_HIP(hipMemcpyAsync(words, d.progress, Nz * sizeof(uint64_t), hipMemcpyDeviceToHost, h.stream));
        PA_HIP(hipStreamSynchronize(h.stream));
        bool all = true;
        need = 1;
        for (size_t n = 0; n < Nz; ++n) {
            if ((words[n] >> 31) & 1u) continue;
            all = false;
            const int s_now = (int)(words[n] & 0x3fffffffu);
            const int qn = (T - s_now + q.P - 1) / q.P;
            if (qn > need) need = qn;
        }
        if (all) break;
    }
    // Every sample is done; the slide that published that also wrote its control block.
    h.slide_pending = false;
    PA_HIP(hipMemcpy2DAsync(x_out, row, d.X + (size_t)T * q.D, (size_t)(T + 1) * row, row, Nz,
                            hipMemcpyDeviceToDevice, h.stream));
    unsigned char heads[PA_MAX_BATCH][kCtrlHead];
    PA_HIP(hipMemcpy2DAsync(heads, kCtrlHead, d.ctrl, sizeof(Ctrl), kCtrlHead, Nz, hipMemcpyDeviceToHost, h.stream));
    PA_HIP(hipStreamSynchronize(h.stream));
    bool nonfinite = false;
    pa_stats_t agg{};
    for (size_t n = 0; n < Nz; ++n) {
        Ctrl c;
        memcpy(&c, heads[n], kCtrlHead);
        pa_stats_t o;
        fill_stats(c, &o);
        nonfinite = nonfinite || o.nonfinite;
        if (n == 0) {
            agg = o;
            continue;
        }
        agg.nfe += o.nfe;
        agg.hits += o.hits;
        agg.misses += o.misses;
        agg.revisits += o.revisits;
        agg.revisits_below += o.revisits_below;
        if (o.sweeps > agg.sweeps) agg.sweeps = o.sweeps;
        if (o.window_start < agg.window_start) agg.window_start = o.window_start;
        if (o.window_end < agg.window_end) agg.window_end = o.window_end;
        agg.done = agg.done && o.done;
        agg.nonfinite = agg.nonfinite || o.nonfinite;
    }
    if (stats) *stats = agg;
    if (nonfinite) return fail(PA_ERR_NONFINITE, "non-finite residual during sampling");
    return PA_OK;
}

}  // extern "C"
