// Solver-side kernels of one sweep, for gfx950 (wave64):
//   k_cache_test : Eq. (4) mean absolute deviation per window slot, Eq. (5) hit test,
//                  first-entry rule, ballot + LDS-offset compaction of the misses, and the
//                  initial estimate of states entering the window.
//   k_picard     : Eq. (6) assembly (cached output for hits, fresh for misses), Eq. (7)
//                  cache-input update, DDIM drift at the current latents, the Eq. (1)
//                  prefix sum over the window anchored at its start (blocked scan: register
//                  scan per thread, chunk carries through LDS), Eq. (2) residual partial
//                  sums; the last block turns them into residuals, counts the leading
//                  converged states and slides the window.
// Both finalize in their last-arriving block (integer arrival counter; partial sums are
// reduced in a fixed order, so every decision is bitwise reproducible run to run).
// Arithmetic: states and network outputs are stored in fp32; the drift, the Picard sum,
// the deviations and the residuals are computed in fp64 from them (coefficients are fp64),
// and every state is rounded once on store. The decisions of Eq. (2) and Eq. (5) are
// therefore taken on fp64 sums, the precision the method is defined in, at no bandwidth
// cost (these kernels are bound by HBM, not by VALU).
#include <math.h>

#include "pa_internal.h"

namespace pa {

namespace {

constexpr int kThreads = 256;           // 4 waves
constexpr int kTestF4PerThread = 4;
constexpr int kTestChunkF4 = kThreads * kTestF4PerThread;   // 4096 floats per block
constexpr int kPicardCols = 16;         // float4 columns per Picard block (a 16-lane DPP row)
constexpr int kPicardRows = kThreads / kPicardCols;         // 16 time rows

__device__ __forceinline__ double wave_sum(double v) {
    // Butterfly over the 64 lanes; the fixed pattern makes the result order-deterministic.
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__device__ __forceinline__ double row16_sum(double v) {
    // Sum inside each aligned group of 16 lanes (one DPP row).
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) v += __shfl_xor(v, off, 16);
    return v;
}

__device__ __forceinline__ double4 d4_add(double4 a, double4 b) {
    return make_double4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

__device__ __forceinline__ double4 d4_of(float4 v) {
    return make_double4((double)v.x, (double)v.y, (double)v.z, (double)v.w);
}

// alpha * x + b * e, elementwise in fp64 (x, e are fp32 values, exact in fp64).
__device__ __forceinline__ double4 drift(double alpha, float4 x, double b, float4 e) {
    return make_double4(fma(b, (double)e.x, alpha * (double)x.x), fma(b, (double)e.y, alpha * (double)x.y),
                        fma(b, (double)e.z, alpha * (double)x.z), fma(b, (double)e.w, alpha * (double)x.w));
}

// Last-block pattern across the grid: one thread per block publishes its partial sums
// (agent-scope release: L2 writeback, no invalidate), bumps the arrival counter, and only
// the last arriving block acquires (invalidate) before it reads every partial.
__device__ __forceinline__ bool arrive_last(uint32_t* counter) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    const uint32_t prev = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return prev == gridDim.x - 1;
}

__device__ __forceinline__ void acquire_partials() { __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent"); }

__device__ __forceinline__ unsigned long long lanemask_lt() {
    const int lane = threadIdx.x & 63;
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

}  // namespace

// ---------------------------------------------------------------------------- reset
__global__ void k_reset(Dev d) {
    const int tid = blockIdx.x * blockDim.x + threadIdx.x;
    for (int t = tid; t < d.T; t += gridDim.x * blockDim.x) d.valid[t] = 0;
    if (tid == 0) {
        Ctrl* c = d.ctrl;
        c->s = 0;
        c->e = min(d.P, d.T);
        c->newest = 0;
        c->m = 0;
        c->done = 0;
        c->nonfinite = 0;
        c->c = 0;
        c->sweep = 0;
        c->nfe = 0;
        c->hits = 0;
        c->cnt_test = 0;
        c->cnt_picard = 0;
    }
}

hipError_t launch_reset(const Dev& d, hipStream_t st) {
    int blocks = (d.T + kThreads - 1) / kThreads;
    if (blocks < 1) blocks = 1;
    if (blocks > 64) blocks = 64;
    hipLaunchKernelGGL(k_reset, dim3(blocks), dim3(kThreads), 0, st, d);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------- cache test
int cache_test_chunks(int D) { return (D / 4 + kTestChunkF4 - 1) / kTestChunkF4; }

__global__ __launch_bounds__(kThreads) void k_cache_test(Dev d) {
    Ctrl* ctrl = d.ctrl;
    if (ctrl->done) return;                 // uniform over the grid
    const int s = ctrl->s, e = ctrl->e, newest = ctrl->newest;
    const int chunks = d.test_chunks;
    const int slot = blockIdx.x / chunks, chunk = blockIdx.x - slot * chunks;
    const int t = s + slot;
    const int n4 = d.D >> 2;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int base = chunk * kTestChunkF4 + tid;

    double acc = 0.0;
    if (t <= e && t > newest) {
        // A state entering the window starts as a copy of the newest estimate.
        const float4* src = reinterpret_cast<const float4*>(d.X + (size_t)newest * d.D);
        float4* dst = reinterpret_cast<float4*>(d.X + (size_t)t * d.D);
#pragma unroll
        for (int k = 0; k < kTestF4PerThread; ++k) {
            const int i = base + k * kThreads;
            if (i < n4) dst[i] = src[i];
        }
    } else if (t < e && d.valid[t]) {
        const float4* x = reinterpret_cast<const float4*>(d.X + (size_t)t * d.D);
        const float4* xh = reinterpret_cast<const float4*>(d.Xh + (size_t)t * d.D);
        float4 a[kTestF4PerThread], b[kTestF4PerThread];
#pragma unroll
        for (int k = 0; k < kTestF4PerThread; ++k) {
            const int i = base + k * kThreads;
            a[k] = i < n4 ? x[i] : make_float4(0.f, 0.f, 0.f, 0.f);
            b[k] = i < n4 ? xh[i] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int k = 0; k < kTestF4PerThread; ++k)
            acc += (fabs((double)a[k].x - (double)b[k].x) + fabs((double)a[k].y - (double)b[k].y)) +
                   (fabs((double)a[k].z - (double)b[k].z) + fabs((double)a[k].w - (double)b[k].w));
    }

    __shared__ double wsum[kThreads / 64];
    __shared__ int is_last;
    acc = wave_sum(acc);
    if (lane == 0) wsum[wave] = acc;
    __syncthreads();
    if (tid == 0) {
        d.part_test[slot * chunks + chunk] = (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]);
        is_last = arrive_last(&ctrl->cnt_test);
    }
    __syncthreads();
    if (!is_last) return;
    acquire_partials();

    // ---- last block: per-slot deviation, hit test, compaction (slot j <-> t = s + j)
    const int W = e - s;
    const int j = tid;                      // kThreads >= PA_MAX_WINDOW
    double dev = __builtin_nan("");
    bool hit = false, miss = false;
    if (j < W) {
        if (d.valid[s + j]) {
            double sum = 0.0;
            for (int c = 0; c < chunks; ++c) sum += d.part_test[j * chunks + c];
            dev = sum / (double)d.D;
            hit = dev < d.delta;            // strict: delta == 0 never hits
        }
        miss = !hit;                        // first entry (no cache entry) is a miss
    }
    const unsigned long long mask = __ballot(miss);
    const int rank = __popcll(mask & lanemask_lt());
    __shared__ int wcount[kThreads / 64];
    if (lane == 0) wcount[wave] = __popcll(mask);
    __syncthreads();
    int off = 0;
    for (int w = 0; w < wave; ++w) off += wcount[w];
    const int m = wcount[0] + wcount[1] + wcount[2] + wcount[3];
    if (miss) {
        ctrl->miss_idx[off + rank] = s + j;
        d.valid[s + j] = 1;                 // Eq. (7): the miss gets its cache entry now
    }
    if (j < W) ctrl->slot_miss[j] = miss ? 1 : 0;
    if (d.trace) {
        pa_sweep_trace_t* rec = d.trace + ctrl->sweep;
        if (j < W) {
            rec->dev[j] = dev;
            rec->hit[j] = hit ? 1 : 0;
        }
        if (miss) rec->miss_idx[off + rank] = s + j;
        if (tid == 0) {
            rec->s = s;
            rec->e = e;
            rec->m = m;
        }
    }
    if (tid == 0) {
        ctrl->m = m;
        ctrl->nfe += m;
        ctrl->hits += W - m;
        ctrl->newest = max(newest, e);
        ctrl->cnt_test = 0;
    }
}

hipError_t launch_cache_test(const Dev& d, hipStream_t st) {
    const int blocks = (d.P + 1) * d.test_chunks;
    hipLaunchKernelGGL(k_cache_test, dim3(blocks), dim3(kThreads), 0, st, d);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------- Picard
int picard_blocks(int D) { return (D / 4 + kPicardCols - 1) / kPicardCols; }

int picard_tpt(int P) {
    int tpt = 1;
    while (tpt * kPicardRows < P) tpt <<= 1;
    return tpt;
}

// Block = 16 float4 columns x 16 time rows; thread (col, row) owns TPT consecutive window
// slots of one float4 column. LINEAR computes eps = c_t * x for the misses in place.
template <int TPT, bool LINEAR>
__global__ __launch_bounds__(kThreads) void k_picard(Dev d) {
    Ctrl* ctrl = d.ctrl;
    if (ctrl->done) return;
    const int s = ctrl->s, e = ctrl->e, W = e - s;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col = tid % kPicardCols, row = tid / kPicardCols;
    const int n4 = d.D >> 2;
    const int c4 = blockIdx.x * kPicardCols + col;
    const bool colok = c4 < n4;
    const int j0 = row * TPT;
    const size_t D = (size_t)d.D;
    const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
    const double4 dzero = make_double4(0.0, 0.0, 0.0, 0.0);

    // xs[k] = state s + j0 + k for j0 + k <= W: xs[k] (k < TPT) is the drift input of slot
    // j0 + k, xs[k + 1] the previous iterate of the state that slot updates.
    float4 xs[TPT + 1], anchor = zero;
    double4 dr[TPT];
#pragma unroll
    for (int k = 0; k <= TPT; ++k) {
        const int j = j0 + k;
        xs[k] = (j <= W && colok) ? reinterpret_cast<const float4*>(d.X + (s + j) * D)[c4] : zero;
    }
#pragma unroll
    for (int k = 0; k < TPT; ++k) {
        const int j = j0 + k;
        dr[k] = dzero;
        if (j < W && colok) {
            const int t = s + j;
            const float4 x = xs[k];
            float4 eps;
            if (ctrl->slot_miss[j]) {
                if (LINEAR) {
                    const float ct = d.lin_c[t];
                    eps = make_float4(ct * x.x, ct * x.y, ct * x.z, ct * x.w);
                    reinterpret_cast<float4*>(d.Eh + t * D)[c4] = eps;
                } else {
                    eps = reinterpret_cast<const float4*>(d.Eh + t * D)[c4];
                }
                reinterpret_cast<float4*>(d.Xh + t * D)[c4] = x;   // Eq. (7) input
            } else {
                eps = reinterpret_cast<const float4*>(d.Eh + t * D)[c4];  // Eq. (6) hit
            }
            dr[k] = drift(d.coef[2 * t], x, d.coef[2 * t + 1], eps);
        }
    }
    if (colok) anchor = reinterpret_cast<const float4*>(d.X + s * D)[c4];

#pragma unroll
    for (int k = 1; k < TPT; ++k) dr[k] = d4_add(dr[k], dr[k - 1]);

    __shared__ double4 tot[kPicardRows][kPicardCols];
    tot[row][col] = dr[TPT - 1];
    __builtin_amdgcn_s_waitcnt(0);          // all loads of X consumed before any store below
    __syncthreads();
    double4 pre = d4_of(anchor);
    for (int r = 0; r < row; ++r) pre = d4_add(pre, tot[r][col]);

    const int nblk = gridDim.x;
    __shared__ double rpart[PA_MAX_WINDOW];
#pragma unroll
    for (int k = 0; k < TPT; ++k) {
        const int j = j0 + k;
        if (j >= W) break;                  // uniform over the 16-lane row
        const double4 yd = d4_add(pre, dr[k]);
        const float4 y = make_float4((float)yd.x, (float)yd.y, (float)yd.z, (float)yd.w);
        const float4 xo = xs[k + 1];
        double rs = 0.0;
        if (colok) {
            reinterpret_cast<float4*>(d.X + (s + 1 + j) * D)[c4] = y;
            const double dx = (double)y.x - (double)xo.x, dy = (double)y.y - (double)xo.y;
            const double dz = (double)y.z - (double)xo.z, dw = (double)y.w - (double)xo.w;
            rs = (dx * dx + dy * dy) + (dz * dz + dw * dw);
        }
        rs = row16_sum(rs);
        if (col == 0) rpart[j] = rs;
    }

    __shared__ int is_last;
    __syncthreads();
    if (tid == 0) {
        for (int j = 0; j < W; ++j) d.part_res[j * nblk + blockIdx.x] = rpart[j];
        is_last = arrive_last(&ctrl->cnt_picard);
    }
    __syncthreads();
    if (!is_last) return;
    acquire_partials();

    // ---- last block: residuals of states s+1..e, convergence count, slide.
    __shared__ double r_s[PA_MAX_WINDOW];
    for (int jj = wave; jj < W; jj += kThreads / 64) {
        double acc = 0.0;
        for (int b = lane; b < nblk; b += 64) acc += d.part_res[jj * nblk + b];
        acc = wave_sum(acc);
        if (lane == 0) r_s[jj] = acc / (double)d.D;
    }
    __syncthreads();
    const int j = tid;
    const double r = j < W ? r_s[j] : 0.0;
    // Slot j stops the leading run if it is not converged or is the last slot (state e).
    const bool stop = (j >= W - 1) || !(r <= d.tol);
    const bool bad = (j < W) && !isfinite(r);
    const unsigned long long sm = __ballot(stop);
    const unsigned long long bm = __ballot(bad);
    __shared__ int wfirst[kThreads / 64];
    __shared__ int wbad[kThreads / 64];
    if (lane == 0) {
        wfirst[wave] = sm ? wave * 64 + __ffsll((long long)sm) - 1 : 1 << 30;
        wbad[wave] = bm != 0ull;
    }
    if (d.trace && j < W) d.trace[ctrl->sweep].resid[j] = r;
    __syncthreads();
    if (tid == 0) {
        int c = 1 << 30, anybad = 0;
        for (int w = 0; w < kThreads / 64; ++w) {
            c = min(c, wfirst[w]);
            anybad |= wbad[w];
        }
        const int s2 = s + 1 + c;
        if (anybad) ctrl->nonfinite = 1;
        if (d.trace) {
            pa_sweep_trace_t* rec = d.trace + ctrl->sweep;
            rec->c = c;
            rec->s_next = s2;
            rec->sweep = ctrl->sweep;
        }
        ctrl->c = c;
        ctrl->s = s2;
        ctrl->e = min(s2 + d.P, d.T);
        ctrl->done = s2 >= d.T;
        ctrl->sweep += 1;
        ctrl->cnt_picard = 0;
    }
}

template <bool LINEAR>
static hipError_t launch_picard_t(const Dev& d, hipStream_t st) {
    const dim3 grid(d.picard_blocks), block(kThreads);
    switch (picard_tpt(d.P)) {
        case 1: hipLaunchKernelGGL((k_picard<1, LINEAR>), grid, block, 0, st, d); break;
        case 2: hipLaunchKernelGGL((k_picard<2, LINEAR>), grid, block, 0, st, d); break;
        case 4: hipLaunchKernelGGL((k_picard<4, LINEAR>), grid, block, 0, st, d); break;
        case 8: hipLaunchKernelGGL((k_picard<8, LINEAR>), grid, block, 0, st, d); break;
        case 16: hipLaunchKernelGGL((k_picard<16, LINEAR>), grid, block, 0, st, d); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_picard(const Dev& d, hipStream_t st, int linear) {
    return linear ? launch_picard_t<true>(d, st) : launch_picard_t<false>(d, st);
}

// ---------------------------------------------------------------------------- t-emb table
// e[j][n] = sum_k temb_k(t_j) Wt[k][n], accumulated in fp64 and rounded once to fp32.
__global__ void k_temb(float* out, const double* tv, const __bf16* wt, int H, int dim) {
    const int n = blockIdx.x * blockDim.x + threadIdx.x;
    const int j = blockIdx.y;
    if (n >= H) return;
    const int half = dim / 2;
    const double t = tv[j];
    double acc = 0.0;
    for (int k = 0; k < half; ++k) {
        const double w = exp(-log(10000.0) * k / half);
        acc += sin(t * w) * (double)(float)wt[(size_t)k * H + n];
        acc += cos(t * w) * (double)(float)wt[(size_t)(k + half) * H + n];
    }
    out[(size_t)j * H + n] = (float)acc;
}

hipError_t launch_temb_table(const Dev& d, const double* t_values_dev, const __bf16* wt_dev,
                             int temb_dim, hipStream_t st) {
    const dim3 grid((d.hidden + 255) / 256, d.T), block(256);
    hipLaunchKernelGGL(k_temb, grid, block, 0, st, d.temb, t_values_dev, wt_dev, d.hidden,
                       temb_dim);
    return hipGetLastError();
}

}  // namespace pa
