// Kernels of the cached Parareal sampler (Sec. 2.1 Parareal-based samplers with the Sec. 2.2
// output cache), for gfx950 (wave64). The noise network is the batched network kernel of
// the Picard sampler: Parareal block n plays the role of sample n with at most one miss per
// batch (Ctrl[n].m in {0, 1}, miss_idx[0] = its timestep), so one network launch serves the
// requests of all blocks at one fine step, or the single request of one coarse step.
//
// Buffers (Dev): X[n][t] (slab n, fine-grid row t) holds block n's trajectory: row nL is the
// boundary state U_n, rows nL+1..(n+1)L its fine solve (row (n+1)L = F_n); slab B row T holds
// the output U_B. Xh/Eh/valid are the timestep cache [T][D]. Per request:
//   k_pr_test          Eq. (4)-(5) hit test of the request's input against the cache entry
//                      of its timestep (one block per Parareal block, fp64 fixed-order sum);
//   k_eps_mlp          the network on the misses;
//   k_pr_fine_step     Eq. (6)-(7) assembly and cache update, then one fine DDIM step;
//   k_pr_coarse        Eq. (6)-(7), then the coarse step and the Parareal correction
//                      U_{n+1} <- G_n(U_n) + (F_n - G_n^old), or the copy U_{k+1} <- F_k,
//                      with per-chunk fp64 partials of the Eq. (2) boundary residual;
//   k_pr_check         residuals, convergence, iteration count, progress word.
#include <math.h>

#include "pa_parareal.h"

namespace pa {

namespace {

constexpr int kTestThreads = 1024;
constexpr int kStepThreads = 256;

__device__ __forceinline__ double block_sum_1024(double v, double* sh) {
    // Fixed-order sum over the 1024 threads of a block: wave butterflies, then wave 0.
    v = wave_sum(v);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    if (lane == 0) sh[w] = v;
    __syncthreads();
    double r = 0.0;
    if (threadIdx.x < 64) {
        r = threadIdx.x < (int)(blockDim.x >> 6) ? sh[threadIdx.x] : 0.0;
        r = wave_sum(r);
    }
    return r;   // valid in thread 0
}

__device__ __forceinline__ float4 f4_fresh(const Dev& d, int n, int c4, int t, float4 x) {
    // Fresh network output of block n's miss at timestep t with input x: the linear network
    // in place, or the fixed-order sum of the network kernel's partial outputs.
    if (d.lin_c) {
        const float c = d.lin_c[t];
        return make_float4(c * x.x, c * x.y, c * x.z, c * x.w);
    }
    const size_t D = (size_t)d.D;
    const float* ep = d.Ep + (size_t)n * d.P * D;
    float4 e = reinterpret_cast<const float4*>(ep)[c4];
    for (int h = 1; h < d.nsplit; ++h) {
        const float4 p = reinterpret_cast<const float4*>(ep + (size_t)h * d.N * d.P * D)[c4];
        e = make_float4(e.x + p.x, e.y + p.y, e.z + p.z, e.w + p.w);
    }
    return e;
}

// x + (a x + b e) in fp64 from fp32 operands, rounded once.
__device__ __forceinline__ float4 ddim_step(float4 x, float4 e, double a, double b) {
    return make_float4((float)((double)x.x + fma(b, (double)e.x, a * (double)x.x)),
                       (float)((double)x.y + fma(b, (double)e.y, a * (double)x.y)),
                       (float)((double)x.z + fma(b, (double)e.z, a * (double)x.z)),
                       (float)((double)x.w + fma(b, (double)e.w, a * (double)x.w)));
}

}  // namespace

// Which request, if any, Parareal block n makes in this launch (uniform per block).
__device__ __forceinline__ bool pr_request(const PrArgs& a, int n, int* t) {
    if (a.mode == PR_FINE) {
        *t = n * a.L + a.j;
        return n >= a.k;
    }
    *t = n * a.L;
    return n == a.n;
}

__global__ __launch_bounds__(kTestThreads) void k_pr_test(Dev d, PrArgs a) {
    const int n = blockIdx.x;
    Ctrl* c = d.ctrl + n;
    int t = 0;
    const bool act = pr_request(a, n, &t) && !a.pc->done;
    if (!act) {                                     // uniform over the block
        if (threadIdx.x == 0) c->m = 0;
        return;
    }
    const size_t D = (size_t)d.D;
    const float* x = d.X + ((size_t)n * (d.T + 1) + t) * D;
    const bool entry = d.valid[t] != 0;
    __shared__ double sh[kTestThreads / 64];
    double dev = __builtin_nan("");
    if (entry) {
        const float4* x4 = reinterpret_cast<const float4*>(x);
        const float4* h4 = reinterpret_cast<const float4*>(d.Xh + (size_t)t * D);
        double acc = 0.0;
        for (int i = threadIdx.x; i < d.D / 4; i += kTestThreads) {
            const float4 u = x4[i], v = h4[i];
            acc += (fabs((double)u.x - (double)v.x) + fabs((double)u.y - (double)v.y)) +
                   (fabs((double)u.z - (double)v.z) + fabs((double)u.w - (double)v.w));
        }
        dev = block_sum_1024(acc, sh) / (double)d.D;
    }
    if (threadIdx.x == 0) {
        const bool hit = entry && dev < d.delta;    // strict: delta == 0 never hits
        c->m = hit ? 0 : 1;
        c->miss_idx[0] = t;
        c->newest = t;
        c->done = 0;
        c->slot_miss[0] = hit ? 0 : 1;
        if (hit) c->hits += 1;
        else c->nfe += 1;
        if (d.trace_pr) {
            pa_request_trace_t* r = d.trace_pr + a.rec + (a.mode == PR_FINE ? n - a.k : 0);
            r->iteration = a.mode == PR_INIT ? -1 : a.k;
            r->phase = a.mode;
            r->t = t;
            r->block = n;
            r->hit = hit ? 1 : 0;
            r->dev = dev;
        }
    }
}

// One fine step of every active block: Eq. (6)-(7) for its request, then the DDIM step.
__global__ __launch_bounds__(kStepThreads) void k_pr_fine_step(Dev d, PrArgs a) {
    const int n = blockIdx.y;
    int t = 0;
    if (!pr_request(a, n, &t) || a.pc->done) return;
    const Ctrl* c = d.ctrl + n;
    const int c4 = blockIdx.x * kStepThreads + threadIdx.x;
    const bool miss = c->slot_miss[0] != 0;
    if (c4 < d.D / 4) {
        const size_t D = (size_t)d.D;
        float* xr = d.X + ((size_t)n * (d.T + 1) + t) * D;
        const float4 x = reinterpret_cast<const float4*>(xr)[c4];
        float4 e;
        if (miss) {
            e = f4_fresh(d, n, c4, t, x);
            reinterpret_cast<float4*>(d.Eh + (size_t)t * D)[c4] = e;
            reinterpret_cast<float4*>(d.Xh + (size_t)t * D)[c4] = x;
            if (d.trace_eps) reinterpret_cast<float4*>(d.trace_eps + (size_t)(a.rec + n - a.k) * D)[c4] = e;
        } else {
            e = reinterpret_cast<const float4*>(d.Eh + (size_t)t * D)[c4];
        }
        reinterpret_cast<float4*>(xr + D)[c4] = ddim_step(x, e, d.coef[3 * t], d.coef[3 * t + 1]);
    }
    if (miss && blockIdx.x == 0 && threadIdx.x == 0) d.valid[t] = 1;
}

// Coarse request of block a.n (PR_INIT / PR_COARSE), or the copy U_{k+1} <- F_k (PR_COPY).
__global__ __launch_bounds__(kStepThreads) void k_pr_coarse(Dev d, PrArgs a) {
    if (a.pc->done) return;
    const int n = a.n, L = a.L;
    const size_t D = (size_t)d.D, rows = (size_t)d.T + 1;
    const int c4 = blockIdx.x * kStepThreads + threadIdx.x;
    const bool ok = c4 < d.D / 4;
    float* unext = d.X + ((size_t)(n + 1) * rows + (size_t)(n + 1) * L) * D;   // U_{n+1}
    const float* fn = d.X + ((size_t)n * rows + (size_t)(n + 1) * L) * D;      // F_n
    double part = 0.0;
    if (a.mode == PR_COPY) {
        if (ok) {
            const float4 f = reinterpret_cast<const float4*>(fn)[c4];
            const float4 o = reinterpret_cast<const float4*>(unext)[c4];
            reinterpret_cast<float4*>(unext)[c4] = f;
            const double dx = (double)f.x - o.x, dy = (double)f.y - o.y, dz = (double)f.z - o.z, dw = (double)f.w - o.w;
            part = (dx * dx + dy * dy) + (dz * dz + dw * dw);
        }
    } else {
        const int t = n * L;
        const Ctrl* c = d.ctrl + n;
        const bool miss = c->slot_miss[0] != 0;
        if (ok) {
            const float* u = d.X + ((size_t)n * rows + (size_t)t) * D;
            const float4 x = reinterpret_cast<const float4*>(u)[c4];
            float4 e;
            if (miss) {
                e = f4_fresh(d, n, c4, t, x);
                reinterpret_cast<float4*>(d.Eh + (size_t)t * D)[c4] = e;
                reinterpret_cast<float4*>(d.Xh + (size_t)t * D)[c4] = x;
                if (d.trace_eps) reinterpret_cast<float4*>(d.trace_eps + (size_t)a.rec * D)[c4] = e;
            } else {
                e = reinterpret_cast<const float4*>(d.Eh + (size_t)t * D)[c4];
            }
            const float4 g = ddim_step(x, e, d.pr_coef[2 * n], d.pr_coef[2 * n + 1]);
            float4* gst = reinterpret_cast<float4*>(d.Gc + (size_t)n * D) + c4;
            float4 un = g;
            if (a.mode == PR_COARSE) {
                const float4 f = reinterpret_cast<const float4*>(fn)[c4];
                const float4 go = *gst;
                un = make_float4((float)((double)g.x + ((double)f.x - (double)go.x)),
                                 (float)((double)g.y + ((double)f.y - (double)go.y)),
                                 (float)((double)g.z + ((double)f.z - (double)go.z)),
                                 (float)((double)g.w + ((double)f.w - (double)go.w)));
                const float4 o = reinterpret_cast<const float4*>(unext)[c4];
                const double dx = (double)un.x - o.x, dy = (double)un.y - o.y;
                const double dz = (double)un.z - o.z, dw = (double)un.w - o.w;
                part = (dx * dx + dy * dy) + (dz * dz + dw * dw);
            }
            *gst = g;
            reinterpret_cast<float4*>(unext)[c4] = un;
        }
        if (miss && blockIdx.x == 0 && threadIdx.x == 0) d.valid[t] = 1;
    }
    if (a.mode != PR_INIT) {
        __shared__ double sh[kStepThreads / 64];
        part = wave_sum(part);
        if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = part;
        __syncthreads();
        if (threadIdx.x == 0) {
            double s = 0.0;
            for (int w = 0; w < kStepThreads / 64; ++w) s += sh[w];
            d.part_res[(size_t)(n + 1) * gridDim.x + blockIdx.x] = s;
        }
    }
}

// Boundary residuals r_n, n = k+1..B, convergence and the iteration count.
__global__ __launch_bounds__(kTestThreads) void k_pr_check(Dev d, PrArgs a) {
    PrCtrl* pc = a.pc;
    if (pc->done) return;
    const int B = d.N, k = a.k, nchunk = a.nchunk;
    __shared__ double r_s[PA_PR_MAX_BLOCKS + 1];
    static_assert(PA_PR_MAX_BLOCKS <= PA_MAX_BATCH, "a Parareal block is a sample of the network kernel");
    // wave w sums boundary w (fixed order within the wave, then the butterfly)
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    for (int nb = k + 1 + w; nb <= B; nb += kTestThreads / 64) {
        double acc = 0.0;
        for (int q = lane; q < nchunk; q += 64) acc += d.part_res[(size_t)nb * nchunk + q];
        acc = wave_sum(acc);
        if (lane == 0) r_s[nb] = acc / (double)d.D;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        bool conv = true, bad = false;
        for (int nb = k + 1; nb <= B; ++nb) {
            const double r = r_s[nb];
            conv = conv && (r <= d.tol);
            bad = bad || !isfinite(r);
            if (d.trace_res) d.trace_res[(size_t)k * (B + 1) + nb] = r;
        }
        if (bad) pc->nonfinite = 1;
        pc->iters = k + 1;
        pc->done = (conv || k + 1 >= B) ? 1 : 0;
        const uint64_t word = ((uint64_t)(uint32_t)pc->iters << 32) | ((uint64_t)pc->done << 31);
        __hip_atomic_store(d.progress, word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
}

__global__ void k_pr_reset(Dev d, PrArgs a) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    for (int t = i; t < d.T; t += gridDim.x * blockDim.x) d.valid[t] = 0;
    for (int n = i; n < d.N; n += gridDim.x * blockDim.x) {
        Ctrl* c = d.ctrl + n;
        c->m = 0;
        c->done = 0;
        c->nfe = 0;
        c->hits = 0;
        c->slot_miss[0] = 0;
    }
    if (i == 0) {
        a.pc->done = 0;
        a.pc->iters = 0;
        a.pc->nonfinite = 0;
    }
}

hipError_t launch_pr(const Dev& d, const PrArgs& a, int kernel, hipStream_t st) {
    const int chunks = (d.D / 4 + kStepThreads - 1) / kStepThreads;
    switch (kernel) {
        case PRK_RESET:
            hipLaunchKernelGGL(k_pr_reset, dim3(4), dim3(256), 0, st, d, a);
            break;
        case PRK_TEST:
            hipLaunchKernelGGL(k_pr_test, dim3(d.N), dim3(kTestThreads), 0, st, d, a);
            break;
        case PRK_FINE:
            hipLaunchKernelGGL(k_pr_fine_step, dim3(chunks, d.N), dim3(kStepThreads), 0, st, d, a);
            break;
        case PRK_COARSE:
            hipLaunchKernelGGL(k_pr_coarse, dim3(chunks), dim3(kStepThreads), 0, st, d, a);
            break;
        case PRK_CHECK:
            hipLaunchKernelGGL(k_pr_check, dim3(1), dim3(kTestThreads), 0, st, d, a);
            break;
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

int pr_chunks(int D) { return (D / 4 + kStepThreads - 1) / kStepThreads; }

}  // namespace pa
