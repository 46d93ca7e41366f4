// Host-code exercise of the C ABI, built against a copy of the library whose host code carries
// AddressSanitizer and UndefinedBehaviorSanitizer (device code built as usual). Any
// sanitizer report ends the run with a non-zero status; so does any unexpected return code.
//
//   abi_driver cpu   argument checks, NULL handles, status strings, the allocation-free entry
//                    point's limits (no HIP call needed), and one valid create, which ends in
//                    PA_OK (then destroyed) or, on a machine without a GPU, PA_ERR_HIP with no
//                    handle and nothing leaked;
//   abi_driver gpu   the above, then every entry point on small workloads: the linear and
//                    patch-MLP samplers (one and two samples, split outputs, step noise),
//                    step-by-step sweeps and every query, the allocation-free sample twice,
//                    the Parareal sampler, and a create that runs out of device memory.
//
// Prints one line per section; the last line is "abi_driver ok".
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "paraanya.h"

namespace {

int g_checks = 0;

#define EXPECT(cond)                                                                        \
    do {                                                                                    \
        ++g_checks;                                                                         \
        if (!(cond)) {                                                                      \
            fprintf(stderr, "%s:%d: expectation failed: %s (last error: %s)\n", __FILE__, \
                    __LINE__, #cond, paraanya_last_error());                                \
            exit(1);                                                                        \
        }                                                                                   \
    } while (0)

#define EXPECT_RC(call, want)                                                                  \
    do {                                                                                       \
        const int rc_ = (call);                                                                \
        ++g_checks;                                                                            \
        if (rc_ != (want)) {                                                                   \
            fprintf(stderr, "%s:%d: %s returned %s, expected %s (last error: %s)\n", __FILE__, \
                    __LINE__, #call, paraanya_status_str(rc_), paraanya_status_str(want),      \
                    paraanya_last_error());                                                    \
            exit(1);                                                                           \
        }                                                                                      \
    } while (0)

#define HIP_OK(call)                                                                     \
    do {                                                                                 \
        const hipError_t e_ = (call);                                                    \
        if (e_ != hipSuccess) {                                                          \
            fprintf(stderr, "%s:%d: %s: %s\n", __FILE__, __LINE__, #call, hipGetErrorString(e_)); \
            exit(1);                                                                     \
        }                                                                                \
    } while (0)

// Deterministic uniform numbers in [-1, 1) (64-bit LCG, top 24 bits).
struct Lcg {
    uint64_t s;
    explicit Lcg(uint64_t seed) : s(seed) {}
    float next() {
        s = s * 6364136223846793005ull + 1442695040888963407ull;
        return (float)((double)(s >> 40) / (double)(1u << 23) - 1.0);
    }
};

uint16_t bf16_bits(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

pa_schedule_t sd_schedule(double eta) {
    pa_schedule_t s;
    memset(&s, 0, sizeof s);
    s.kind = PA_SCHED_SCALED_LINEAR;
    s.beta_start = 0.00085;
    s.beta_end = 0.012;
    s.train_steps = 1000;
    s.spacing = PA_SPACING_TRAILING;
    s.final_alpha_one = 1;
    s.eta = eta;
    return s;
}

// Network description and the host arrays it points to.
struct Model {
    std::vector<float> c;
    std::vector<uint16_t> w1, wt, w2, w3;
    pa_eps_model_t em;
};

void linear_model(Model& m, int T) {
    m.c.resize(T > 0 ? T : 1);
    for (int j = 0; j < (int)m.c.size(); ++j) m.c[j] = 0.1f + 0.001f * j;
    memset(&m.em, 0, sizeof m.em);
    m.em.kind = PA_EPS_LINEAR;
    m.em.c = m.c.data();
}

void mlp_model(Model& m, int hidden) {
    Lcg g(1234 + hidden);
    auto fill = [&](std::vector<uint16_t>& w, int fan_in, int fan_out) {
        w.resize((size_t)fan_in * fan_out);
        const float a = sqrtf(3.0f / fan_in);
        for (auto& v : w) v = bf16_bits(a * g.next());
    };
    fill(m.w1, 16, hidden);
    fill(m.wt, 128, hidden);
    fill(m.w2, hidden, hidden);
    fill(m.w3, hidden, 16);
    memset(&m.em, 0, sizeof m.em);
    m.em.kind = PA_EPS_PATCH_MLP;
    m.em.patch = 2;
    m.em.hidden = hidden;
    m.em.temb_dim = 128;
    m.em.w1 = m.w1.data();
    m.em.wt = m.wt.data();
    m.em.w2 = m.w2.data();
    m.em.w3 = m.w3.data();
}

// ---------------------------------------------------------------- checks without a GPU
void cpu_checks(bool have_gpu) {
    for (int s = -8; s <= 1; ++s) EXPECT(paraanya_status_str(s) != nullptr && paraanya_status_str(s)[0]);
    EXPECT(strcmp(paraanya_status_str(PA_OK), "PA_OK") == 0);

    const pa_schedule_t sc = sd_schedule(0.0);
    Model lin;
    linear_model(lin, 2048);                  // c covers every T tried below
    const int32_t shape[4] = {1, 4, 8, 8};
    paraanya_t* h = (paraanya_t*)0x1;
    EXPECT_RC(paraanya_create(shape, 10, &sc, 4, 0.05, 1e-3, &lin.em, nullptr, 0, nullptr), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_create(nullptr, 10, &sc, 4, 0.05, 1e-3, &lin.em, nullptr, 0, &h), PA_ERR_INVALID_ARG);
    EXPECT(h == nullptr);
    EXPECT(strlen(paraanya_last_error()) > 0);
    struct Bad {
        int32_t shape[4];
        int T, window;
        double delta, tol;
        uint32_t flags;
    } bad[] = {
        {{0, 4, 8, 8}, 10, 4, 0.05, 1e-3, 0},   {{PA_MAX_BATCH + 1, 4, 8, 8}, 10, 4, 0.05, 1e-3, 0},
        {{1, 3, 3, 3}, 10, 4, 0.05, 1e-3, 0},   {{1, 4, 8, 8}, 0, 1, 0.05, 1e-3, 0},
        {{1, 4, 8, 8}, 10, 0, 0.05, 1e-3, 0},   {{1, 4, 8, 8}, 10, 11, 0.05, 1e-3, 0},
        {{1, 4, 8, 8}, 10, 4, -1.0, 1e-3, 0},   {{1, 4, 8, 8}, 10, 4, NAN, 1e-3, 0},
        {{1, 4, 8, 8}, 10, 4, 0.05, -1.0, 0},   {{1, 4, 8, 8}, 10, 4, 0.05, 1e-3, 64u},
        {{1, 4, 8, 8}, 2000, 4, 0.05, 1e-3, 0},
    };
    for (const Bad& b : bad) {
        h = (paraanya_t*)0x1;
        EXPECT_RC(paraanya_create(b.shape, b.T, &sc, b.window, b.delta, b.tol, &lin.em, nullptr, b.flags, &h),
                  PA_ERR_INVALID_ARG);
        EXPECT(h == nullptr);
    }
    EXPECT_RC(paraanya_create(shape, 10, nullptr, 4, 0.05, 1e-3, &lin.em, nullptr, 0, &h), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_create(shape, 10, &sc, 4, 0.05, 1e-3, nullptr, nullptr, 0, &h), PA_ERR_INVALID_ARG);
    pa_schedule_t ex = sc;
    ex.kind = PA_SCHED_EXPLICIT;
    EXPECT_RC(paraanya_create(shape, 10, &ex, 4, 0.05, 1e-3, &lin.em, nullptr, 0, &h), PA_ERR_INVALID_ARG);
    std::vector<double> ab(11, 0.5);
    std::vector<int32_t> tv(10, 0);
    ab[3] = 1.5;
    ex.alpha_bar = ab.data();
    ex.t_values = tv.data();
    EXPECT_RC(paraanya_create(shape, 10, &ex, 4, 0.05, 1e-3, &lin.em, nullptr, 0, &h), PA_ERR_INVALID_ARG);
    Model mlp;
    mlp_model(mlp, 512);
    const int32_t odd[4] = {1, 4, 7, 8};
    EXPECT_RC(paraanya_create(odd, 10, &sc, 4, 0.05, 1e-3, &mlp.em, nullptr, 0, &h), PA_ERR_INVALID_ARG);
    mlp.em.hidden = 768;
    const int32_t mshape[4] = {1, 4, 32, 32};
    EXPECT_RC(paraanya_create(mshape, 10, &sc, 4, 0.05, 1e-3, &mlp.em, nullptr, 0, &h), PA_ERR_UNSUPPORTED);
    mlp.em.hidden = 512;

    // NULL handles
    float dummy[4] = {0, 0, 0, 0};
    int32_t done = 0;
    pa_stats_t st;
    pa_sweep_trace_t* tr = (pa_sweep_trace_t*)calloc(1, sizeof(pa_sweep_trace_t));
    pa_ktimes_t kt;
    EXPECT_RC(paraanya_reset(nullptr, dummy), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_set_noise(nullptr, dummy), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_set_revisit_threshold(nullptr, 0.1), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_sweep(nullptr, &done), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_sample(nullptr, dummy, dummy), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_stats(nullptr, &st), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_stats_sample(nullptr, 0, &st), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_trace(nullptr, 0, tr), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_trace_sample(nullptr, 0, 0, tr), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_read_state(nullptr, 0, 1, dummy, nullptr, nullptr, nullptr), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_read_state_sample(nullptr, 0, 0, 1, dummy, nullptr, nullptr, nullptr), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_coefficients(nullptr, nullptr, nullptr, nullptr, nullptr), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_kernel_times(nullptr, &kt), PA_ERR_INVALID_ARG);
    paraanya_destroy(nullptr);

    // Parareal: argument checks and NULL handles
    paraanya_parareal_t* ph = (paraanya_parareal_t*)0x1;
    EXPECT_RC(paraanya_parareal_create(mshape, 12, &sc, 5, 0.05, 1e-3, &mlp.em, nullptr, 0, &ph), PA_ERR_INVALID_ARG);
    EXPECT(ph == nullptr);
    EXPECT_RC(paraanya_parareal_create(mshape, 12, &sc, 0, 0.05, 1e-3, &mlp.em, nullptr, 0, &ph), PA_ERR_INVALID_ARG);
    const pa_schedule_t sc1 = sd_schedule(1.0);
    EXPECT_RC(paraanya_parareal_create(mshape, 12, &sc1, 4, 0.05, 1e-3, &mlp.em, nullptr, 0, &ph), PA_ERR_UNSUPPORTED);
    pa_parareal_stats_t pst;
    pa_request_trace_t prt;
    double r[PA_PR_MAX_BLOCKS + 1];
    EXPECT_RC(paraanya_parareal_sample(nullptr, dummy, dummy), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_parareal_stats(nullptr, &pst), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_parareal_trace(nullptr, 0, &prt, nullptr), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_parareal_residuals(nullptr, 0, r), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_parareal_read_boundaries(nullptr, dummy), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_parareal_kernel_times(nullptr, &kt), PA_ERR_INVALID_ARG);
    paraanya_parareal_destroy(nullptr);

    // Allocation-free entry point: limits checked before any HIP call
    EXPECT_RC(paraanya_sample_noalloc(shape, PA_NOALLOC_MAX_STEPS + 1, &sc, 4, 0.05, 1e-3, &lin.em, nullptr,
                                      dummy, dummy, &st), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_sample_noalloc(shape, 10, &sc1, 4, 0.05, 1e-3, &lin.em, nullptr, dummy, dummy, &st),
              PA_ERR_UNSUPPORTED);
    EXPECT_RC(paraanya_sample_noalloc(shape, 10, &sc, 4, 0.05, 1e-3, &lin.em, nullptr, nullptr, dummy, &st),
              PA_ERR_INVALID_ARG);
    // Beyond the workspace: found once the device is known (no GPU: the HIP call fails first).
    const int32_t big[4] = {1, 4, 64, 64};
    EXPECT_RC(paraanya_sample_noalloc(big, 1000, &sc, 128, 0.05, 1e-3, &mlp.em, nullptr, dummy, dummy, &st),
              have_gpu ? PA_ERR_INVALID_ARG : PA_ERR_HIP);

    // One valid create
    h = (paraanya_t*)0x1;
    const int rc = paraanya_create(shape, 10, &sc, 4, 0.05, 1e-3, &lin.em, nullptr, 0, &h);
    if (have_gpu) {
        EXPECT(rc == PA_OK && h != nullptr);
        paraanya_destroy(h);
    } else {
        EXPECT(rc == PA_ERR_HIP && h == nullptr);
    }
    free(tr);
    printf("cpu checks ok (%d expectations)\n", g_checks);
}

// ---------------------------------------------------------------- full runs on a GPU
float* device_latents(int n, size_t D, uint64_t seed) {
    std::vector<float> x((size_t)n * D);
    Lcg g(seed);
    for (auto& v : x) v = 1.7f * g.next();
    float* p = nullptr;
    HIP_OK(hipMalloc((void**)&p, x.size() * sizeof(float)));
    HIP_OK(hipMemcpy(p, x.data(), x.size() * sizeof(float), hipMemcpyHostToDevice));
    return p;
}

void expect_finite_device(const float* p, size_t count) {
    std::vector<float> h(count);
    HIP_OK(hipMemcpy(h.data(), p, count * sizeof(float), hipMemcpyDeviceToHost));
    for (float v : h) EXPECT(isfinite(v));
}

// Step-by-step sweeps and every query on one handle.
void run_handle(const int32_t shape[4], int T, int window, const pa_schedule_t& sc, const Model& m,
                uint32_t flags, const char* name) {
    const int N = shape[0];
    const size_t D = (size_t)shape[1] * shape[2] * shape[3];
    paraanya_t* h = nullptr;
    EXPECT_RC(paraanya_create(shape, T, &sc, window, 0.05, 1e-3, &m.em, nullptr, flags, &h), PA_OK);
    float* x = device_latents(N, D, 7);
    float* z = nullptr;
    if (sc.eta > 0.0) {
        EXPECT_RC(paraanya_reset(h, x), PA_ERR_STATE);          // no noise given yet
        z = device_latents(N, (size_t)T * D, 11);
        EXPECT_RC(paraanya_set_noise(h, z), PA_OK);
    }
    pa_stats_t st;
    EXPECT_RC(paraanya_stats(h, &st), PA_ERR_STATE);             // before the first reset
    EXPECT_RC(paraanya_set_revisit_threshold(h, 0.1), PA_OK);
    EXPECT_RC(paraanya_reset(h, x), PA_OK);
    int32_t done = 0;
    int sweeps = 0;
    while (!done) {
        EXPECT_RC(paraanya_sweep(h, &done), PA_OK);
        EXPECT(++sweeps <= T + 1);
    }
    EXPECT_RC(paraanya_sweep(h, &done), PA_ERR_STATE);           // already done
    EXPECT_RC(paraanya_stats(h, &st), PA_OK);
    EXPECT(st.done == 1 && st.nfe + st.hits >= T && st.sweeps > 0 && st.sweeps <= sweeps);
    for (int n = 0; n < N; ++n) EXPECT_RC(paraanya_stats_sample(h, n, &st), PA_OK);
    EXPECT_RC(paraanya_stats_sample(h, N, &st), PA_ERR_INVALID_ARG);
    pa_sweep_trace_t* tr = (pa_sweep_trace_t*)calloc(1, sizeof(pa_sweep_trace_t));
    if (flags & PA_FLAG_TRACE) {
        EXPECT_RC(paraanya_trace(h, 0, tr), PA_OK);
        EXPECT(tr->m > 0);
        EXPECT_RC(paraanya_trace_sample(h, N - 1, 0, tr), PA_OK);
        EXPECT_RC(paraanya_trace(h, sweeps + 5, tr), PA_ERR_INVALID_ARG);
        EXPECT_RC(paraanya_trace(h, -1, tr), PA_ERR_INVALID_ARG);
        EXPECT_RC(paraanya_trace_sample(h, N, 0, tr), PA_ERR_INVALID_ARG);
        EXPECT_RC(paraanya_trace(h, 0, nullptr), PA_ERR_INVALID_ARG);
    } else {
        EXPECT_RC(paraanya_trace(h, 0, tr), PA_ERR_STATE);
    }
    std::vector<float> X((size_t)(T + 1) * D), Xh((size_t)T * D), Eh((size_t)T * D);
    std::vector<uint8_t> valid(T);
    EXPECT_RC(paraanya_read_state(h, 0, T + 1, X.data(), Xh.data(), Eh.data(), valid.data()), PA_OK);
    for (size_t i = (size_t)T * D; i < X.size(); ++i) EXPECT(isfinite(X[i]));
    EXPECT_RC(paraanya_read_state_sample(h, N - 1, T - 1, T + 1, X.data(), nullptr, nullptr, nullptr), PA_OK);
    EXPECT_RC(paraanya_read_state(h, 0, T + 2, X.data(), nullptr, nullptr, nullptr), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_read_state(h, -1, 1, X.data(), nullptr, nullptr, nullptr), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_read_state(h, 2, 1, X.data(), nullptr, nullptr, nullptr), PA_ERR_INVALID_ARG);
    EXPECT_RC(paraanya_read_state(h, 1, 1, X.data(), Xh.data(), Eh.data(), valid.data()), PA_OK);   // empty
    EXPECT_RC(paraanya_read_state_sample(h, -1, 0, 1, X.data(), nullptr, nullptr, nullptr), PA_ERR_INVALID_ARG);
    std::vector<double> a(T), b(T), s(T);
    std::vector<float> temb(m.em.kind == PA_EPS_PATCH_MLP ? (size_t)T * m.em.hidden : 1);
    EXPECT_RC(paraanya_coefficients(h, a.data(), b.data(), s.data(),
                                    m.em.kind == PA_EPS_PATCH_MLP ? temb.data() : nullptr), PA_OK);
    pa_ktimes_t kt;
    if (flags & PA_FLAG_PROFILE) {
        EXPECT_RC(paraanya_kernel_times(h, &kt), PA_OK);
    } else {
        EXPECT_RC(paraanya_kernel_times(h, &kt), PA_ERR_STATE);
    }
    // Two whole samples, the output aliasing the input.
    for (int k = 0; k < 2; ++k) EXPECT_RC(paraanya_sample(h, x, x), PA_OK);
    expect_finite_device(x, (size_t)N * D);
    free(tr);
    paraanya_destroy(h);
    HIP_OK(hipFree(x));
    if (z) HIP_OK(hipFree(z));
    printf("%s ok (%d sweeps)\n", name, sweeps);
}

void gpu_checks() {
    const pa_schedule_t sc = sd_schedule(0.0), sc1 = sd_schedule(1.0);
    Model lin, mlp, mlp1k;
    linear_model(lin, 12);
    mlp_model(mlp, 512);
    mlp_model(mlp1k, 1024);
    const uint32_t all = PA_FLAG_TRACE | PA_FLAG_PROFILE | PA_FLAG_PROFILE_SOLVER;
    const int32_t s_lin[4] = {2, 4, 8, 8}, s_mlp1[4] = {1, 4, 32, 32}, s_mlp2[4] = {2, 4, 32, 32};
    run_handle(s_lin, 12, 4, sc, lin, all, "linear, two samples");
    run_handle(s_lin, 12, 4, sc1, lin, 0, "linear with step noise");
    run_handle(s_mlp1, 12, 6, sc, mlp, all, "patch-MLP, one sample");
    run_handle(s_mlp2, 12, 6, sc, mlp, PA_FLAG_TRACE | PA_FLAG_PROFILE, "patch-MLP, two samples");
    run_handle(s_mlp1, 12, 6, sc, mlp1k, PA_FLAG_SPLIT_OUTPUTS | PA_FLAG_TRACE, "patch-MLP, split outputs");

    // Allocation-free sample, twice (the second smaller), in place.
    {
        const size_t D = 4 * 32 * 32;
        float* x = device_latents(1, D, 5);
        pa_stats_t st;
        EXPECT_RC(paraanya_sample_noalloc(s_mlp1, 12, &sc, 6, 0.05, 1e-3, &mlp.em, nullptr, x, x, &st), PA_OK);
        EXPECT(st.done == 1);
        const int32_t small[4] = {1, 4, 16, 32};
        EXPECT_RC(paraanya_sample_noalloc(small, 8, &sc, 4, 0.05, 1e-3, &mlp.em, nullptr, x, x, nullptr), PA_OK);
        expect_finite_device(x, 4 * 16 * 32);
        HIP_OK(hipFree(x));
        printf("allocation-free sample ok\n");
    }

    // Parareal sampler.
    {
        const size_t D = 4 * 32 * 32;
        const int T = 12, B = 4;
        paraanya_parareal_t* ph = nullptr;
        EXPECT_RC(paraanya_parareal_create(s_mlp1, T, &sc, B, 0.05, 1e-3, &mlp.em, nullptr,
                                           PA_FLAG_TRACE | PA_FLAG_PROFILE, &ph), PA_OK);
        pa_parareal_stats_t pst;
        EXPECT_RC(paraanya_parareal_stats(ph, &pst), PA_ERR_STATE);
        float* x = device_latents(1, D, 9);
        EXPECT_RC(paraanya_parareal_sample(ph, x, x), PA_OK);
        EXPECT_RC(paraanya_parareal_stats(ph, &pst), PA_OK);
        EXPECT(pst.done == 1 && pst.requests == pst.nfe + pst.hits && pst.requests > 0);
        pa_request_trace_t prt;
        std::vector<float> eps(D);
        EXPECT_RC(paraanya_parareal_trace(ph, 0, &prt, eps.data()), PA_OK);
        EXPECT_RC(paraanya_parareal_trace(ph, (int32_t)pst.requests, &prt, nullptr), PA_ERR_INVALID_ARG);
        double r[PA_PR_MAX_BLOCKS + 1];
        EXPECT_RC(paraanya_parareal_residuals(ph, 0, r), PA_OK);
        std::vector<float> U((size_t)(B + 1) * D);
        EXPECT_RC(paraanya_parareal_read_boundaries(ph, U.data()), PA_OK);
        for (float v : U) EXPECT(isfinite(v));
        pa_ktimes_t kt;
        EXPECT_RC(paraanya_parareal_kernel_times(ph, &kt), PA_OK);
        EXPECT(kt.launches > 0);
        paraanya_parareal_destroy(ph);
        HIP_OK(hipFree(x));
        printf("parareal ok (%d iterations)\n", pst.iterations);
    }

    // A request larger than device memory: OOM, no handle, nothing kept.
    {
        const int32_t huge[4] = {1, 4, 8192, 8192};     // 1 GiB per state, 1001 states
        Model lin1k;
        linear_model(lin1k, 1000);
        paraanya_t* h = (paraanya_t*)0x1;
        EXPECT_RC(paraanya_create(huge, 1000, &sc, 32, 0.05, 1e-3, &lin1k.em, nullptr, 0, &h), PA_ERR_OOM);
        EXPECT(h == nullptr);
        printf("out-of-memory create ok\n");
    }
}

}  // namespace

int main(int argc, char** argv) {
    if (argc != 2 || (strcmp(argv[1], "cpu") && strcmp(argv[1], "gpu"))) {
        fprintf(stderr, "usage: %s cpu|gpu\n", argv[0]);
        return 2;
    }
    const bool gpu = strcmp(argv[1], "gpu") == 0;
    int ndev = 0;
    const bool have_gpu = hipGetDeviceCount(&ndev) == hipSuccess && ndev > 0;
    if (gpu && !have_gpu) {
        fprintf(stderr, "gpu mode needs a GPU\n");
        return 2;
    }
    cpu_checks(have_gpu);
    if (gpu) gpu_checks();
    printf("abi_driver ok (%d expectations)\n", g_checks);
    return 0;
}
