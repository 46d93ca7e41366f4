// Solver-side kernels of the sampler, for gfx950 (wave64). One sweep is
//   [k_eps_mlp: network on the misses (patch-MLP only)] -> k_picard -> k_slide
// and k_reset prepares the first window. Every kernel handles the N samples of a handle
// at once (grid dimension y of k_reset and k_picard, the blocks of k_slide); a sample that
// is done makes its blocks exit at once.
//   k_picard : Eq. (6) assembly (cached output for hits, fresh for misses: in the cache
//              already when the network launch wrote whole outputs, else the fixed-order sum
//              of its split partials), Eq. (7) cache update, DDIM drift at the current latents, the Eq. (1) prefix sum over the
//              window anchored at its start (blocked scan: register scan per thread, chunk
//              carries through LDS). Per block it writes partial sums of the Eq. (2)
//              residuals and, for the states it just updated, of the Eq. (4) deviation from
//              the cache entry they will be tested against in the next sweep (every drift
//              point of the window holds a cache entry after the sweep), so the next sweep
//              needs no separate pass over the window.
//   k_slide  : residuals from the partials, leading converged count, window slide, done;
//              then, for the next window, Eq. (5) hit test (first entries are misses) and
//              ballot + LDS-offset compaction of the misses into an ascending list.
// A state that enters the window is never copied: its estimate is the newest computed state
// (Sec. 2.1 gives no initial trajectory; reading X[min(t, newest)] is that copy, virtually).
// Kernel boundaries order all partial sums and their consumers: no cross-block fence or float
// atomic anywhere, and every partial is reduced in a fixed order, so each decision is bitwise
// reproducible run to run.
// Arithmetic: states and network outputs are stored in fp32; the drift, the Picard sum, the
// deviations and the residuals are computed in fp64 from them (coefficients are fp64), and
// every state is rounded once on store. The decisions of Eq. (2) and Eq. (5) are therefore
// taken on fp64 sums at no bandwidth cost (these kernels are bound by memory, not by VALU).
#include <math.h>

#include <hip/hip_ext.h>

#include "pa_device.h"
#include "pa_slide.h"

namespace pa {

namespace {

constexpr int kThreads = 256;           // 4 waves
constexpr int kSlideThreads = 1024;     // k_slide: 16 waves for the partial reductions

template <int WIDTH>
__device__ __forceinline__ double group_sum(double v) {
    // Sum inside each aligned group of WIDTH lanes (butterfly, fixed order).
#pragma unroll
    for (int off = WIDTH / 2; off >= 1; off >>= 1) v += __shfl_xor(v, off, WIDTH);
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

// d += sigma * z (the pre-sampled noise term of a stochastic step).
__device__ __forceinline__ double4 add_noise(double4 d, double sigma, float4 z) {
    return make_double4(fma(sigma, (double)z.x, d.x), fma(sigma, (double)z.y, d.y),
                        fma(sigma, (double)z.z, d.z), fma(sigma, (double)z.w, d.w));
}

__device__ __forceinline__ double abs_dev(float4 a, float4 b) {
    return (fabs((double)a.x - (double)b.x) + fabs((double)a.y - (double)b.y)) +
           (fabs((double)a.z - (double)b.z) + fabs((double)a.w - (double)b.w));
}

__device__ __forceinline__ double sq_dev(float4 a, float4 b) {
    const double dx = (double)a.x - (double)b.x, dy = (double)a.y - (double)b.y;
    const double dz = (double)a.z - (double)b.z, dw = (double)a.w - (double)b.w;
    return (dx * dx + dy * dy) + (dz * dz + dw * dw);
}

}  // namespace

// ---------------------------------------------------------------------------- reset
// Window [0, min(P, T)); no timestep has a cache entry, so every slot is a first-entry miss.
__global__ void k_reset(Dev d) {
    const int n = blockIdx.y;
    const int tid = blockIdx.x * blockDim.x + threadIdx.x;
    Ctrl* c = d.ctrl + n;
    uint8_t* valid = d.valid + (size_t)n * d.T;
    pa_sweep_trace_t* tr = d.trace ? d.trace + (size_t)n * d.T : nullptr;
    const int W = min(d.P, d.T);
    for (int t = tid; t < d.T; t += gridDim.x * blockDim.x) valid[t] = 0;
    for (int j = tid; j < W; j += gridDim.x * blockDim.x) {
        c->miss_idx[j] = j;
        c->slot_miss[j] = 1;
        c->slot_rank[j] = (uint8_t)j;
        if (tr) {
            tr[0].dev[j] = __builtin_nan("");
            tr[0].hit[j] = 0;
            tr[0].miss_idx[j] = j;
        }
    }
    if (tid == 0) {
        if (d.pre) d.pre[n].pending = 0;
        c->s = 0;
        c->e = W;
        c->newest = 0;
        c->m = W;
        c->done = 0;
        c->nonfinite = 0;
        c->c = 0;
        c->sweep = 0;
        c->nfe = W;
        c->hits = 0;
        c->revisits = 0;
        c->revisits_below = 0;
        if (tr) {
            tr[0].s = 0;
            tr[0].e = W;
            tr[0].m = W;
        }
    }
}

hipError_t launch_reset(const Dev& d, hipStream_t st) {
    int blocks = (d.T + kThreads - 1) / kThreads;
    if (blocks < 1) blocks = 1;
    if (blocks > 64) blocks = 64;
    hipLaunchKernelGGL(k_reset, dim3(blocks, d.N), dim3(kThreads), 0, st, d);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------- Picard
// Block = COLS float4 columns (one DPP row of lanes) x ROWS time rows, TPT slots per thread:
//   P <= 16: 16 x 16 x 1;  P <= 32: 16 x 16 x 2;  P <= 64: 16 x 32 x 2;  P <= 128: 16 x 64 x 2;
//   P <= 256: 8 x 128 x 2.
// Narrow blocks give the most blocks, which this latency-bound kernel needs more than fewer
// partial sums (measured: 64-column blocks at P = 32 take twice as long). Longer windows take
// more rows rather than more slots per thread: each slot holds ~30 registers, and at 8 slots
// per thread the kernel ran at one wave per SIMD (16 slots spilled).
struct PicardShape {
    int cols, rows, tpt;
};

static PicardShape picard_shape(int P) {
    if (P <= 16) return {16, 16, 1};
    if (P <= 32) return {16, 16, 2};
    if (P <= 64) return {16, 32, 2};
    if (P <= 128) return {16, 64, 2};
    return {8, 128, 2};
}

int picard_blocks(int D, int P) {
    const int cols = picard_shape(P).cols;
    return (D / 4 + cols - 1) / cols;
}

// LINEAR computes eps = c_t * x for the misses in place; otherwise the fresh outputs are the
// fixed-order sum of the network kernel's partial outputs.
// NS: partial outputs per fresh network output (the network kernel's splits of the output
// units; 1 for the linear network).
// Zero vectors as values: a named local zero vector was kept in scratch memory by the compiler.
__device__ __forceinline__ float4 f4_zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
__device__ __forceinline__ double4 d4_zero() { return make_double4(0.0, 0.0, 0.0, 0.0); }

// MINB: minimum blocks per CU the compiler must fit (1, or 6 (5 with step noise or one
// partial output) for the 256-thread shape of batched handles: at most 76 (96) registers). NOISE: the step adds the
// pre-drawn noise term (stochastic sampler).
template <int COLS, int ROWS, int TPT, bool LINEAR, int NS, int MINB, bool NOISE>
__global__ __launch_bounds__(COLS * ROWS, MINB) void k_picard(Dev d) {
    constexpr int kThr = COLS * ROWS;
    const int n = blockIdx.y;
    const Ctrl* ctrl = d.ctrl + n;
    // The network launch wrote the fresh outputs of the misses into Eh (whole outputs) rather
    // than split partials into Ep.
    const bool whole = !LINEAR && d.eps_whole != nullptr && *d.eps_whole != 0;
    if (ctrl->done) return;
    const int s = ctrl->s, e = ctrl->e, W = e - s, newest = ctrl->newest;
    const int tid = threadIdx.x;
    const int col = tid % COLS, row = tid / COLS;
    const int n4 = d.D >> 2;
    const int c4 = blockIdx.x * COLS + col;
    const bool colok = c4 < n4;
    const int j0 = row * TPT;
    const size_t D = (size_t)d.D;
    float* X = d.X + (size_t)n * (d.T + 1) * D;
    float* Xh = d.Xh + (size_t)n * d.T * D;
    float* Eh = d.Eh + (size_t)n * d.T * D;
    const float* noise = NOISE ? d.noise + (size_t)n * d.T * D : nullptr;

    // ---- the states (independent of the miss list) first; meanwhile the block stages the
    // per-slot miss flags and ranks in LDS, so that the address of every other load is known
    // after one barrier instead of a chain of dependent global byte loads.
    // xs[k] = current estimate of state s + j0 + k (k <= TPT, j0 + k <= W): the drift input of
    // slot j0 + k and the previous iterate of the state slot j0 + k - 1 updates.
    float4 xs[TPT + 1], e0[TPT], ex[TPT][NS > 1 ? NS - 1 : 1], zt[TPT], xhn[TPT];
    double cf[TPT][3];
    float4 anchor = f4_zero();
    if (colok) anchor = reinterpret_cast<const float4*>(X + min(s, newest) * D)[c4];
#pragma unroll
    for (int k = 0; k <= TPT; ++k) {
        const int j = j0 + k;
        xs[k] = (j <= W && colok) ? reinterpret_cast<const float4*>(X + min(s + j, newest) * D)[c4] : f4_zero();
    }
    // Loads that do not depend on the miss flags, issued before the flags are staged: the
    // coefficients, the step noise and, when the network launch wrote whole outputs, each
    // slot's row of Eh.
#pragma unroll
    for (int k = 0; k < TPT; ++k) {
        const int j = j0 + k, t = s + j;
        const bool act = j < W && colok;
        e0[k] = f4_zero();
        zt[k] = f4_zero();
        xhn[k] = f4_zero();
#pragma unroll
        for (int h = 0; h < (NS > 1 ? NS - 1 : 1); ++h) ex[k][h] = f4_zero();
        cf[k][0] = cf[k][1] = cf[k][2] = 0.0;
        if (act) {
            // Eq. (6) with whole outputs: the cache row holds the output of a hit and the
            // fresh output of a miss alike.
            if (whole) e0[k] = reinterpret_cast<const float4*>(Eh + t * D)[c4];
            cf[k][0] = d.coef[3 * t];
            cf[k][1] = d.coef[3 * t + 1];
            if (NOISE) {
                cf[k][2] = d.coef[3 * t + 2];
                zt[k] = reinterpret_cast<const float4*>(noise + t * D)[c4];
            }
        }
    }
    __shared__ uint8_t sm[PA_MAX_WINDOW + TPT + 1];
    __shared__ uint8_t sr[PA_MAX_WINDOW + TPT];
    static_assert(kThr >= PA_MAX_WINDOW, "one thread per window slot");
    if (tid < W) {
        sm[tid] = ctrl->slot_miss[tid];
        sr[tid] = ctrl->slot_rank[tid];
    }
    __syncthreads();
    // f[k]: slot j0 + k is a miss (k <= TPT; slot j0 + TPT decides where the last updated
    // state's next cache entry comes from); rk[k]: its place in the miss list.
    int f[TPT + 1], rk[TPT];
#pragma unroll
    for (int k = 0; k <= TPT; ++k) f[k] = (j0 + k < W) ? sm[j0 + k] : 0;
#pragma unroll
    for (int k = 0; k < TPT; ++k) rk[k] = (j0 + k < W) ? sr[j0 + k] : 0;

    // ---- the loads that depend on the flags, issued before any store.
#pragma unroll
    for (int k = 0; k < TPT; ++k) {
        const int j = j0 + k, t = s + j;
        const bool act = j < W && colok;
        const bool miss = f[k] != 0;
        if (act && !whole) {
            // Eq. (6): the cached output of a hit, or the network kernel's split partial
            // outputs of a miss (LINEAR: computed below from the state).
            const float* ep = d.Ep + ((size_t)n * d.P + rk[k]) * D;
            if (!(LINEAR && miss)) e0[k] = reinterpret_cast<const float4*>(miss ? ep : Eh + t * D)[c4];
            if (!LINEAR && miss) {
#pragma unroll
                for (int h = 1; h < NS; ++h)
                    ex[k][h - 1] = reinterpret_cast<const float4*>(ep + (size_t)h * d.N * d.P * D)[c4];
            }
        }
        // Cache entry the updated state s + 1 + j is tested against in the next sweep: the
        // state itself if slot j + 1 is a miss now (its entry is refreshed below), else Xh.
        if (j + 1 < W && colok && !f[k + 1]) xhn[k] = reinterpret_cast<const float4*>(Xh + (s + 1 + j) * D)[c4];
    }

    // ---- Eq. (6)-(7) and the drift at the current latents (fp64), cache writes of misses.
    double4 dr[TPT];
#pragma unroll
    for (int k = 0; k < TPT; ++k) {
        const int j = j0 + k, t = s + j;
        dr[k] = d4_zero();
        if (j + 1 < W && f[k + 1]) xhn[k] = xs[k + 1];
        if (j < W && colok) {
            const float4 x = xs[k];
            float4 eps = e0[k];
            if (f[k]) {
                if (LINEAR) {
                    const float ct = d.lin_c[t];
                    eps = make_float4(ct * x.x, ct * x.y, ct * x.z, ct * x.w);
                } else if (!whole) {
                    // Fresh output = fixed-order sum of the network kernel's partials.
#pragma unroll
                    for (int h = 1; h < NS; ++h) {
                        const float4 p = ex[k][h - 1];
                        eps = make_float4(eps.x + p.x, eps.y + p.y, eps.z + p.z, eps.w + p.w);
                    }
                }
            }
            dr[k] = drift(cf[k][0], x, cf[k][1], eps);
            if (NOISE) dr[k] = add_noise(dr[k], cf[k][2], zt[k]);
            e0[k] = eps;
        }
    }
#pragma unroll
    for (int k = 1; k < TPT; ++k) dr[k] = d4_add(dr[k], dr[k - 1]);

    __shared__ double4 tot[ROWS][COLS];
    __shared__ double rres[PA_MAX_WINDOW];
    __shared__ double rdev[PA_MAX_WINDOW];
    tot[row][col] = dr[TPT - 1];
    __builtin_amdgcn_s_waitcnt(0);          // all loads of X consumed before any store below
    __syncthreads();
#pragma unroll
    for (int k = 0; k < TPT; ++k) {
        const int j = j0 + k, t = s + j;
        if (j < W && colok && f[k]) {
            if (!whole) reinterpret_cast<float4*>(Eh + t * D)[c4] = e0[k];   // Eq. (7) output
            reinterpret_cast<float4*>(Xh + t * D)[c4] = xs[k];               // Eq. (7) input
        }
    }
    // pre = anchor + the totals of the rows above, added in row order.
    double4 pre;
    if constexpr (ROWS <= 16) {
        pre = d4_of(anchor);
        for (int r = 0; r < row; ++r) pre = d4_add(pre, tot[r][col]);
    } else {
        // Tall blocks: one thread per column turns the row totals into that same prefix in
        // place (the same additions in the same order), instead of every thread re-reading
        // up to ROWS - 1 totals.
        if (tid < COLS) {
            double4 acc = d4_of(anchor);
            for (int r = 0; r < ROWS; ++r) {
                const double4 tr = tot[r][tid];
                tot[r][tid] = acc;
                acc = d4_add(acc, tr);
            }
        }
        __syncthreads();
        pre = tot[row][col];
    }

#pragma unroll
    for (int k = 0; k < TPT; ++k) {
        const int j = j0 + k;
        double rs = 0.0, ds = 0.0;
        if (j < W && colok) {
            const double4 yd = d4_add(pre, dr[k]);
            const float4 y = make_float4((float)yd.x, (float)yd.y, (float)yd.z, (float)yd.w);
            reinterpret_cast<float4*>(X + (s + 1 + j) * D)[c4] = y;
            rs = sq_dev(y, xs[k + 1]);                   // Eq. (2) vs the previous iterate
            if (j + 1 < W) ds = abs_dev(y, xhn[k]);      // Eq. (4) for the next sweep
        }
        rs = group_sum<COLS>(rs);                        // j is uniform over the row's lanes
        ds = group_sum<COLS>(ds);
        if (col == 0 && j < W) {
            rres[j] = rs;
            rdev[j] = ds;
        }
    }
    __syncthreads();
    const int nblk = gridDim.x;
    if (tid < W) {
        const size_t pbase = (size_t)n * d.P * nblk;
        d.part_res[pbase + tid * nblk + blockIdx.x] = rres[tid];
        d.part_dev[pbase + tid * nblk + blockIdx.x] = rdev[tid];
        if (blockIdx.x == 0 && ctrl->slot_miss[tid]) d.valid[(size_t)n * d.T + s + tid] = 1;   // Eq. (7) entry
    }
    // Fused sweep: the state this sweep started from, for the slide of the next network kernel.
    if (d.fused_slide && blockIdx.x == 0 && tid == 0) d.pre[n] = slide_pre_of(*ctrl);
}

template <bool LINEAR, int NS, bool NOISE>
static hipError_t launch_picard_t(const Dev& d, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    const PicardShape sh = picard_shape(d.P);
    const dim3 grid(d.picard_blocks, d.N), block(sh.cols * sh.rows);
    if (d.picard_blocks != picard_blocks(d.D, d.P)) return hipErrorInvalidValue;
    // Batched handles stream from HBM with many blocks per CU: a build capped at 76 registers
    // (six waves per SIMD; 96 and five with step noise or one partial output, whose registers
    // would otherwise spill) instead of four waves (one sample: within 2% either way, and the four-wave build is kept
    // there). With four partial outputs the register cap would spill.
    const bool occ = d.N >= 8;
    switch (sh.rows * 4 + sh.tpt) {
        case 16 * 4 + 1: hipExtLaunchKernelGGL((k_picard<16, 16, 1, LINEAR, NS, 1, NOISE>), grid, block, 0, st, e0, e1, 0, d); break;
        case 16 * 4 + 2:
            if constexpr (NS <= 2) {
                if (occ) {
                    constexpr int kMinb = (NOISE || NS == 1) ? 5 : 6;
                    hipExtLaunchKernelGGL((k_picard<16, 16, 2, LINEAR, NS, kMinb, NOISE>), grid, block, 0, st, e0, e1, 0, d);
                    break;
                }
            }
            hipExtLaunchKernelGGL((k_picard<16, 16, 2, LINEAR, NS, 1, NOISE>), grid, block, 0, st, e0, e1, 0, d);
            break;
        case 32 * 4 + 2: hipExtLaunchKernelGGL((k_picard<16, 32, 2, LINEAR, NS, 1, NOISE>), grid, block, 0, st, e0, e1, 0, d); break;
        case 64 * 4 + 2: hipExtLaunchKernelGGL((k_picard<16, 64, 2, LINEAR, NS, 1, NOISE>), grid, block, 0, st, e0, e1, 0, d); break;
        case 128 * 4 + 2: hipExtLaunchKernelGGL((k_picard<8, 128, 2, LINEAR, NS, 1, NOISE>), grid, block, 0, st, e0, e1, 0, d); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <bool NOISE>
static hipError_t launch_picard_n(const Dev& d, hipStream_t st, int linear, hipEvent_t e0, hipEvent_t e1) {
    if (linear) return launch_picard_t<true, 1, NOISE>(d, st, e0, e1);
    switch (d.nsplit) {
        case 1: return launch_picard_t<false, 1, NOISE>(d, st, e0, e1);
        case 2: return launch_picard_t<false, 2, NOISE>(d, st, e0, e1);
        case 4: return launch_picard_t<false, 4, NOISE>(d, st, e0, e1);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_picard(const Dev& d, hipStream_t st, int linear, hipEvent_t e0, hipEvent_t e1) {
    return d.noise ? launch_picard_n<true>(d, st, linear, e0, e1) : launch_picard_n<false>(d, st, linear, e0, e1);
}

// ---------------------------------------------------------------------------- slide
// One block per sample: the slide of its current state (FROM_PRE: of the Picard kernel's
// snapshot, outstanding after a fused sweep; nothing to do if there is none).
template <bool FROM_PRE>
__global__ __launch_bounds__(kSlideThreads) void k_slide(Dev d) {
    const int n = blockIdx.x;
    const Ctrl* ctrl = d.ctrl + n;
    __shared__ SlideScratch sc;
    __shared__ double sub[kSlideSubDoubles];
    slide_partials<kSlideThreads>(d, n, sub);    // issued while the control block is read
    if (ctrl->done) return;
    SlidePre pre;
    if (FROM_PRE) {
        pre = d.pre[n];
        if (!pre.pending) return;
    } else {
        pre = slide_pre_of(*ctrl);
    }
    __syncthreads();
    slide_core<kSlideThreads>(d, n, pre, true, sc, sub);
}

hipError_t launch_slide(const Dev& d, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    hipExtLaunchKernelGGL(k_slide<false>, dim3(d.N), dim3(kSlideThreads), 0, st, e0, e1, 0, d);
    return hipGetLastError();
}

hipError_t launch_slide_pending(const Dev& d, hipStream_t st) {
    hipLaunchKernelGGL(k_slide<true>, dim3(d.N), dim3(kSlideThreads), 0, st, d);
    return hipGetLastError();
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
