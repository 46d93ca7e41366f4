/*
 * paraanya.h — C ABI of the MI355X (gfx950) cached Picard sliding-window sampler.
 *
 * The sampler is the output-cached parallel-in-time diffusion sampler of
 * "ParaAnya: Accelerating Parallel Diffusion Sampling with Plug-and-Play Output
 * Caching": Picard iteration over a sliding window of P timesteps (Sec. 2.1, Eq. (1),
 * convergence test Eq. (2)) with an output cache in front of the noise network
 * (Sec. 2.2, Eq. (3)-(7)). One sweep on the device is:
 *   (1) per-timestep cache test, mean |x_t - x^_t| < delta        (Eq. (4), (5));
 *   (2) compaction of the misses into a dense batch                 (Eq. (5));
 *   (3) one batched network evaluation of the misses only           (Sec. 2.2);
 *   (4) scatter of the fresh outputs into the cache                 (Eq. (6), (7));
 *   (5) DDIM drift at the current latents and the Picard prefix sum
 *       anchored at the window start                                (Eq. (1));
 *   (6) residuals, convergence test against tau, window slide       (Eq. (2)).
 *
 * Conventions
 *   - All entry points return PA_OK (0) or a negative PA_ERR_* code; no C++ exception
 *     crosses this boundary. paraanya_last_error() gives a thread-local message.
 *   - One handle = one HIP stream (given at create). Every device operation of the
 *     handle is enqueued on that stream. A handle is not thread-safe.
 *   - Device pointers are HIP device addresses on the handle's current device; host
 *     pointers are ordinary CPU memory. The library never takes ownership of caller
 *     memory: it copies what it needs and owns every buffer it allocates.
 *   - Latents are fp32, layout [N][C][H][W] row-major, D = C*H*W elements per sample.
 *     N independent samples share one handle (same T, window, thresholds, network): each
 *     has its own trajectory, cache and window, and one batched sweep advances every sample
 *     that is not done, with all their misses evaluated by one network launch.
 *   - Sampler state index i = 0..T: state 0 is the initial noise, state T the output.
 */
#ifndef PARAANYA_H
#define PARAANYA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define PA_API __attribute__((visibility("default")))
#else
#define PA_API
#endif

/* ------------------------------------------------------------------ status codes */
#define PA_OK               0
#define PA_ERR_INVALID_ARG (-1)  /* argument outside the documented domain; nothing enqueued */
#define PA_ERR_HIP         (-2)  /* a HIP runtime call failed (message names the call) */
#define PA_ERR_OOM         (-3)  /* device or pinned-host allocation failed */
#define PA_ERR_STATE       (-4)  /* call not valid in the handle's current state */
#define PA_ERR_NONFINITE   (-5)  /* a residual of Eq. (2) was NaN/Inf; the sweep completed */
#define PA_ERR_UNSUPPORTED (-6)  /* valid request the library does not implement */

#define PA_MAX_WINDOW 256        /* largest window P */
#define PA_MAX_BATCH  64         /* largest number of samples N per handle */
#define PA_MAX_STEPS  (1 << 20)  /* largest number of sampling steps T (keeps T + 1 and every
                                    row count of the trajectory within int) */

/* ------------------------------------------------------------------ schedule */
#define PA_SCHED_SCALED_LINEAR 0
#define PA_SCHED_EXPLICIT      1
#define PA_SPACING_TRAILING    0

/* Noise schedule of the DDIM sampler (the paper uses the SD-v1.5 DDIM scheduler,
 * Sec. 3.3). SCALED_LINEAR: betas (sqrt(beta_start) + j*(sqrt(beta_end)-sqrt(beta_start))
 * /(train_steps-1))^2, alpha_bar = cumprod(1-beta), trailing timesteps
 * t_j = round(train_steps - j*train_steps/T) - 1, alpha_bar of the final state = 1
 * (final_alpha_one must be 1). EXPLICIT: the caller gives alpha_bar[0..T] (host, state
 * order, alpha_bar[T] is the clean end) and t_values[0..T-1] (host; used only for the
 * time embedding of the patch-MLP). Copied at create.
 * eta in [0, 1] selects the step (the generalized DDIM step of the DDIM paper):
 * x_{i+1} = sqrt(ab_{i+1}) x0^ + sqrt(1 - ab_{i+1} - sigma_i^2) eps + sigma_i z_i with
 * sigma_i = eta sqrt((1 - ab_{i+1}) / (1 - ab_i)) sqrt(1 - ab_i / ab_{i+1}), taken as 0 at
 * eta = 0 and where ab_{i+1} = ab_i (a step with no noise; with eta > 0 alpha_bar must not
 * decrease, else PA_ERR_INVALID_ARG). eta = 0 is
 * deterministic DDIM; eta = 1 is ancestral DDPM sampling (the stochastic sampler of the
 * paper's window study, Sec. 3.4), whose per-step noise z_i is drawn before sampling and
 * given with paraanya_set_noise, so that Picard iteration solves a fixed recurrence. */
typedef struct {
    int32_t kind;
    double beta_start, beta_end;
    int32_t train_steps;
    int32_t spacing;
    int32_t final_alpha_one;
    const double* alpha_bar;
    const int32_t* t_values;
    double eta;
} pa_schedule_t;

/* ------------------------------------------------------------------ noise network */
#define PA_EPS_LINEAR    0
#define PA_EPS_PATCH_MLP 1

/* Synthetic noise-prediction network standing in for the paper's SD-v1.5 UNet (Sec. 3.2).
 * LINEAR: eps_j(x) = c[j] * x with c[0..T-1] (host fp32), j the sampling step.
 * PATCH_MLP: 2x2 patchify (token = (h/2)*(W/2) + w/2, feature = c*4 + (h%2)*2 + (w%2),
 * C = 4 channels, 16 features), h1 = GELU(bf16(x) W1 + e_j), h2 = GELU(bf16(h1) W2),
 * eps = bf16(h2) W3, unpatchify; e_j = temb(t_j) Wt with the 128-d sinusoidal embedding
 * (sin for k < 64, cos above, frequency exp(-ln(1e4) k/64)); erf GELU; bf16 x bf16
 * products accumulated in fp32. Weights are bf16 bit patterns, row-major [in][out]:
 * w1[16][hidden], wt[temb_dim][hidden], w2[hidden][hidden], w3[hidden][16]; host memory,
 * copied at create. Supported: patch = 2, C = 4, temb_dim = 128, hidden in {512, 1024, 2048},
 * (H/2)*(W/2) a multiple of 128. */
typedef struct {
    int32_t kind;
    const float* c;
    int32_t patch;
    int32_t hidden;
    int32_t temb_dim;
    const uint16_t* w1;
    const uint16_t* wt;
    const uint16_t* w2;
    const uint16_t* w3;
} pa_eps_model_t;

/* ------------------------------------------------------------------ create flags */
#define PA_FLAG_TRACE   1u   /* keep a per-sweep trace record (paraanya_trace) */
#define PA_FLAG_PROFILE 2u   /* time every network launch with HIP events (paraanya_kernel_times) */
#define PA_FLAG_PROFILE_SOLVER 4u  /* with PA_FLAG_PROFILE: time the Picard and slide launches
                                      too (their events add ~7 us per sweep of stream time) */
#define PA_FLAG_SPLIT_OUTPUTS 8u   /* test hook (patch-MLP): every network launch writes split
                                      partial outputs that the Picard kernel sums, instead of
                                      choosing whole outputs written straight into the cache
                                      when they cost no extra time; the results are the same
                                      bit for bit either way */

typedef struct paraanya paraanya_t;

/* Counters of Sec. 3.1 / Tab. cache_tol: nfe = single-latent network evaluations (the
 * misses), hits = window slots served from the cache, sweeps = Picard iterations.
 * revisits / revisits_below feed the revisit statistic of Sec. 1: of all requested drift
 * evaluations (nfe + hits, one per window slot and sweep), revisits are those at a
 * timestep evaluated before, and revisits_below those whose input moved by less than the
 * revisit threshold (Eq. (4) deviation from the cached input; paraanya_set_revisit_threshold,
 * default 0.05). Run at delta = 0, revisits_below / (nfe + hits) is the fraction of
 * requested evaluations that a cache with tolerance equal to the threshold would first
 * target. For a batched handle paraanya_stats sums the counters over the samples and
 * reports sweeps = the largest per-sample count, window_start/window_end = the smallest
 * per-sample values, done = all samples done, nonfinite = any. */
typedef struct {
    int64_t nfe;
    int64_t hits;
    int64_t misses;       /* == nfe */
    int64_t sweeps;
    int32_t window_start; /* s: states 0..s are final */
    int32_t window_end;   /* e = min(s + P, T) */
    int32_t done;         /* s >= T */
    int32_t nonfinite;    /* a non-finite residual was seen (sticky until reset) */
    int64_t revisits;
    int64_t revisits_below;
} pa_stats_t;

/* One sweep's decisions (test hook). Slot j <-> timestep s + j, j < e - s. */
typedef struct {
    int32_t s, e, m, c, s_next, sweep;
    double  dev[PA_MAX_WINDOW];       /* Eq. (4) per slot (fp64 sum); NaN for a first entry */
    double  resid[PA_MAX_WINDOW];     /* Eq. (2) residual of state s + 1 + j (fp64 sum) */
    int32_t miss_idx[PA_MAX_WINDOW];  /* ascending timesteps of the misses, m of them */
    uint8_t hit[PA_MAX_WINDOW];       /* Eq. (5) hit mask per slot */
} pa_sweep_trace_t;

/* Device time of the kernels since reset (PA_FLAG_PROFILE): each launch carries start/stop
 * events attached to its dispatch on the handle's stream. A pair can also cover idle time
 * between the kernel and the work before it on the stream (little without a profiler
 * attached, more under one, which spaces the kernels further apart). */
typedef struct {
    int64_t launches;         /* network launches */
    double  eps_ms_total;     /* summed kernel durations of the network launches */
    int64_t eps_latents;      /* latents evaluated by those launches (= nfe) */
    int64_t solver_launches;  /* Picard launches (= window-slide launches) */
    double  picard_ms_total;  /* summed durations of the drift / Picard / cache-update kernel */
    double  slide_ms_total;   /* summed durations of the residual / slide / hit-test kernel
                                 (0 for a fused handle, see paraanya_sweep: its slide runs in
                                 the network kernel) */
} pa_ktimes_t;

/* ------------------------------------------------------------------ entry points */

/* Create a sampler. latent_shape = {N, C, H, W} with 1 <= N <= PA_MAX_BATCH samples; T in [1, PA_MAX_STEPS] sampling steps;
 * window P in [1, min(T, PA_MAX_WINDOW)]; delta >= 0 the cache tolerance of Eq. (5)
 * (strict '<'; 0 disables hits; +inf allowed); tol >= 0 the tau of Eq. (2) (mean
 * square, '<='). Both thresholds are compared against fp64 sums: states and network
 * outputs are stored in fp32, and the drift, the Picard sum, the deviations and the
 * residuals are computed in fp64 from them, then rounded once on store. stream is a hipStream_t (NULL = the null stream). On success *out
 * holds the handle; on failure *out = NULL and nothing is left allocated.
 * Errors: INVALID_ARG (N outside [1, PA_MAX_BATCH], C*H*W % 4 != 0, T outside [1, PA_MAX_STEPS], window outside
 * range, delta or tol negative/NaN, eta outside [0, 1], bad schedule or model fields),
 * UNSUPPORTED (model shape not built), OOM, HIP. */
PA_API int paraanya_create(const int32_t latent_shape[4], int32_t T, const pa_schedule_t* schedule,
                           int32_t window, double delta, double tol, const pa_eps_model_t* eps_model,
                           void* stream, uint32_t flags, paraanya_t** out);

/* Start new samples: state 0 of sample n <- x_init[n] (device, N x D fp32, read on the
 * stream), every cache entry invalid, windows [0, min(P, T)), counters zero. Waits for the
 * handle's earlier work on the stream, then enqueues the reset and returns without waiting
 * for it. STATE if eta > 0 and no noise was given (paraanya_set_noise). */
PA_API int paraanya_reset(paraanya_t* h, const float* x_init);

/* Pre-sampled per-step noise of the stochastic sampler (eta > 0): z (device, N x T x D
 * fp32, layout [n][i][D], i the sampling step) is copied on the stream into the handle and
 * used by every following sample until replaced; sigma_i z_i is added to the drift of
 * step i. INVALID_ARG for eta = 0 handles or z == NULL. */
PA_API int paraanya_set_noise(paraanya_t* h, const float* z);

/* Threshold of the revisit statistic (see pa_stats_t); >= 0, +inf allowed; applies to the
 * sweeps enqueued after the call. */
PA_API int paraanya_set_revisit_threshold(paraanya_t* h, double threshold);

/* Enqueue one sweep (steps (1)-(6) above) of every sample not yet done. If done != NULL
 * the stream is synchronized and *done receives 1 once every sample is done. Errors: STATE
 * (before reset, or the last synchronized state was already done), NONFINITE (only when
 * done != NULL and a residual was NaN/Inf).
 * A handle of one patch-MLP sample whose window's fp64 partial sums are small (2 P times the
 * Picard kernel's D/64 column blocks, at most 256 KiB) runs its sweeps fused: the window
 * slide of step (6) runs at the start of the next sweep's network kernel (every block
 * computes it; one publishes it), and whenever the host reads the state (done != NULL,
 * stats, trace, read_state) a finishing slide runs first, so every call observes the same
 * state as with a separate slide kernel. */
PA_API int paraanya_sweep(paraanya_t* h, int32_t* done);

/* reset, sweeps until every sample is done, then x_out (device, N x D fp32) <- state T of
 * each sample. x_init and x_out may alias. The host does not synchronize per sweep: it
 * follows a progress word that each sweep writes to pinned host memory and keeps a few sweeps
 * queued ahead; sweeps queued past the end exit at once. The call returns once every sample
 * is done, without draining the stream: the copy into x_out (and the tail of the last
 * kernels) is queued on the stream, so work the caller enqueues on that stream afterwards
 * sees x_out; synchronize the stream before reading x_out any other way. The final counters
 * come with the done words, so paraanya_stats / paraanya_stats_sample right after return
 * them without synchronizing; every other query synchronizes first. With PA_FLAG_PROFILE
 * (or if the counter words are not yet visible) the call synchronizes before returning.
 * NONFINITE as paraanya_sweep. */
PA_API int paraanya_sample(paraanya_t* h, const float* x_init, float* x_out);

/* Counters and window position; synchronizes the stream (not right after paraanya_sample,
 * whose counters are already final). STATE before the first reset.
 * paraanya_stats aggregates over the samples (see pa_stats_t); paraanya_stats_sample
 * reports sample n alone (INVALID_ARG for n outside [0, N)). */
PA_API int paraanya_stats(paraanya_t* h, pa_stats_t* out);
PA_API int paraanya_stats_sample(paraanya_t* h, int32_t n, pa_stats_t* out);

/* Trace record of sweep k (0-based) since reset; needs PA_FLAG_TRACE. Synchronizes.
 * INVALID_ARG if k is not a completed sweep of that sample or n is out of range; STATE
 * without the flag. paraanya_trace is sample 0. */
PA_API int paraanya_trace(paraanya_t* h, int32_t k, pa_sweep_trace_t* out);
PA_API int paraanya_trace_sample(paraanya_t* h, int32_t n, int32_t k, pa_sweep_trace_t* out);

/* Test hook: copy state rows to host memory; synchronizes. Any pointer may be NULL.
 * X receives states [t0, t1) (t1 <= T+1); Xh, Eh, valid receive cache rows [t0, min(t1, T)).
 * A state above the newest computed one is not materialized: its current estimate is the
 * newest computed state (the window start's row shows which rows were computed). */
PA_API int paraanya_read_state(paraanya_t* h, int32_t t0, int32_t t1, float* X, float* Xh,
                        float* Eh, uint8_t* valid);
/* The same for sample n (paraanya_read_state is sample 0). */
PA_API int paraanya_read_state_sample(paraanya_t* h, int32_t n, int32_t t0, int32_t t1, float* X,
                                      float* Xh, float* Eh, uint8_t* valid);

/* Test hook: the fp64 step coefficients the device uses (host arrays of T, any may be
 * NULL): alpha[i] = a_i - 1, b[i], sigma[i], with the drift d_i = alpha_i x_i + b_i eps_i
 * + sigma_i z_i, a_i = sqrt(ab_{i+1}/ab_i), b_i = sqrt(1 - ab_{i+1} - sigma_i^2)
 * - a_i sqrt(1 - ab_i) and sigma_i as under pa_schedule_t; and, for the patch-MLP, the
 * fp32 time-embedding table e[T][hidden]. */
PA_API int paraanya_coefficients(paraanya_t* h, double* alpha, double* b, double* sigma, float* temb);

/* Kernel timings (PA_FLAG_PROFILE) of every launch since the previous call (or since
 * create): the totals restart after each call, so a caller can time many samples and read
 * once. eps_latents counts the network latents of the completed samples among them.
 * Synchronizes. STATE without the flag. */
PA_API int paraanya_kernel_times(paraanya_t* h, pa_ktimes_t* out);

/* Free every resource of the handle (synchronizes its stream first). NULL-safe. */
PA_API void paraanya_destroy(paraanya_t* h);

/* ------------------------------------------------------------------ allocation-free sampling
 * For callers that cannot allocate: code that must not call hipMalloc, hipHostMalloc or
 * hipFree (tight serving loops, harnesses that forbid allocation). One complete sample, the
 * same bit for bit as paraanya_create (flags 0) + paraanya_sample + paraanya_stats +
 * paraanya_destroy with the same arguments, but every device buffer of the sampler
 * (trajectory, cache, partial sums, control blocks, progress words, network tables) is carved
 * from a static device workspace of PA_NOALLOC_WORKSPACE_BYTES that the library holds on each
 * device it runs on until the process ends, and the host side uses the stack only. No device,
 * pinned or host heap memory is allocated (an error message may allocate its text).
 * Arguments as for paraanya_create, plus: x_init, x_out device N x D fp32 (may alias);
 * stats (host, may be NULL) receives the counters as paraanya_stats reports them. Limits:
 * T <= PA_NOALLOC_MAX_STEPS, deterministic step (schedule eta = 0), and the request's
 * buffers must fit the workspace (e.g. one 4x64x64 latent, T = 100, window 32, patch-MLP
 * hidden 1024 takes about 28 MiB); otherwise INVALID_ARG (UNSUPPORTED for eta != 0) before
 * anything is enqueued. Returns after x_out is written (the stream is synchronized). Calls on
 * one device share its workspace and are serialized by a lock inside the library; every call
 * rebuilds the workspace's contents (the previous call's are overwritten), and calls that
 * overlapped on one device without that lock would race. Other errors as paraanya_sample. */
#define PA_NOALLOC_WORKSPACE_BYTES (64u << 20)
#define PA_NOALLOC_MAX_STEPS 1024
PA_API int paraanya_sample_noalloc(const int32_t latent_shape[4], int32_t T,
                                   const pa_schedule_t* schedule, int32_t window, double delta,
                                   double tol, const pa_eps_model_t* eps_model, void* stream,
                                   const float* x_init, float* x_out, pa_stats_t* stats);

/* ------------------------------------------------------------------ Parareal sampler
 * The Parareal-based sampler family of Sec. 2.1 (coarse solver initializing, fine solvers
 * refining; SRDS) with the Sec. 2.2 cache on every network evaluation, coarse or fine. The
 * T sampling steps form B blocks of L = T / B fine DDIM steps. Coarse step of block n: one
 * DDIM step from state nL to state (n+1)L with the network at timestep nL. Initialization:
 * U_0 = x_init, U_{n+1} = G_n(U_n). Iteration k: fine solves of the blocks n >= k (all
 * blocks advance one fine step per batched network launch), then U_{k+1} <- F_k and, for
 * n = k+1..B-1 in order, U_{n+1} <- G_n(U_n) + (F_n - G_n^previous) (textbook Parareal
 * predictor-corrector); stop when every boundary's Eq. (2) residual is <= tol, or after B
 * iterations (then U_B equals serial fine DDIM). The cache holds one entry per fine-grid
 * timestep; a coarse request at nL shares the entry of the first fine step of block n.
 * Storage fp32, arithmetic fp64 with one rounding per stored value, as in the Picard
 * sampler. Deterministic DDIM only (schedule eta must be 0). */
#define PA_PR_MAX_BLOCKS 64

typedef struct paraanya_parareal paraanya_parareal_t;

typedef struct {
    int64_t nfe;          /* network evaluations (cache misses) */
    int64_t hits;         /* requests served from the cache */
    int64_t requests;     /* nfe + hits */
    int32_t iterations;   /* Parareal iterations after the initialization */
    int32_t done;
    int32_t nonfinite;    /* a boundary residual was NaN/Inf */
    int32_t pad;
} pa_parareal_stats_t;

/* One network request (test hook). Requests are numbered in issue order: the B coarse
 * requests of the initialization, then per iteration the fine steps (blocks k..B-1 each)
 * and the coarse requests of blocks k+1..B-1. */
typedef struct {
    int32_t iteration;    /* -1 for the initialization */
    int32_t phase;        /* 0 initialization, 1 fine step, 2 coarse correction */
    int32_t t;            /* fine-grid timestep */
    int32_t block;
    int32_t hit;          /* Eq. (5) */
    int32_t pad;
    double  dev;          /* Eq. (4) (fp64 sum); NaN without a cache entry */
} pa_request_trace_t;

/* Create a Parareal sampler. latent_shape = {1, C, H, W}; T in [1, PA_MAX_STEPS]; blocks in
 * [1, PA_PR_MAX_BLOCKS] dividing T; delta, tol as for paraanya_create; flags: PA_FLAG_TRACE (request records,
 * fresh outputs and boundary residuals), PA_FLAG_PROFILE (network launch timings).
 * Errors: INVALID_ARG, UNSUPPORTED (eta != 0, model shape not built), OOM, HIP. */
PA_API int paraanya_parareal_create(const int32_t latent_shape[4], int32_t T,
                                    const pa_schedule_t* schedule, int32_t blocks, double delta,
                                    double tol, const pa_eps_model_t* eps_model, void* stream,
                                    uint32_t flags, paraanya_parareal_t** out);

/* One full sample: initialization and iterations until done; x_init, x_out device D fp32
 * (may alias); returns after x_out is written. NONFINITE if a residual was NaN/Inf. */
PA_API int paraanya_parareal_sample(paraanya_parareal_t* h, const float* x_init, float* x_out);

/* Counters of the last sample; STATE before the first. */
PA_API int paraanya_parareal_stats(paraanya_parareal_t* h, pa_parareal_stats_t* out);

/* Test hook (PA_FLAG_TRACE): request i of the last sample; eps (host, D fp32, may be NULL)
 * receives its fresh network output when it was a miss. INVALID_ARG for i out of range. */
PA_API int paraanya_parareal_trace(paraanya_parareal_t* h, int32_t i, pa_request_trace_t* out,
                                   float* eps);

/* Test hook (PA_FLAG_TRACE): boundary residuals r[0..B] of iteration k (entries 0..k are 0). */
PA_API int paraanya_parareal_residuals(paraanya_parareal_t* h, int32_t k, double* r);

/* Test hook: the boundary states U_0..U_B of the last sample, host (B+1) x D fp32. */
PA_API int paraanya_parareal_read_boundaries(paraanya_parareal_t* h, float* U);

/* Network-launch timings since the previous call (or create), as paraanya_kernel_times;
 * STATE without PA_FLAG_PROFILE. */
PA_API int paraanya_parareal_kernel_times(paraanya_parareal_t* h, pa_ktimes_t* out);

/* Free the handle (synchronizes its stream first). NULL-safe. */
PA_API void paraanya_parareal_destroy(paraanya_parareal_t* h);

/* Thread-local message of the last failing call on this thread ("" if none). */
PA_API const char* paraanya_last_error(void);

/* Static name of a status code. */
PA_API const char* paraanya_status_str(int status);

#ifdef __cplusplus
}
#endif
#endif /* PARAANYA_H */
