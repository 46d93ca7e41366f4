// Internal declarations shared by the host library and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "paraanya.h"

namespace pa {

// Device-resident control block of one sample. Every per-sweep decision lives here, so
// the host can enqueue sweeps without reading anything back.
struct alignas(256) Ctrl {
    int32_t s;          // window start: states 0..s are final
    int32_t e;          // window end: drift points s..e-1, updated states s+1..e
    int32_t newest;     // highest computed state; a state above it reads as X[newest]
    int32_t m;          // misses of the current sweep
    int32_t done;       // s >= T
    int32_t nonfinite;  // sticky: a residual was NaN/Inf
    int32_t c;          // leading converged count of the last sweep
    int32_t sweep;      // completed sweeps since reset
    int64_t nfe;
    int64_t hits;
    int64_t revisits;       // window slots whose timestep holds a cache entry
    int64_t revisits_below; // ... with Eq. (4) deviation below Dev::revisit_thr
    int32_t miss_idx[PA_MAX_WINDOW];  // ascending miss timesteps
    uint8_t slot_miss[PA_MAX_WINDOW]; // per window slot j: 1 if t = s + j is a miss
    uint8_t slot_rank[PA_MAX_WINDOW]; // per miss slot j: its position in miss_idx
};

// The control-block fields the window slide reads, as they were before it (the fused sweep's
// Picard kernel leaves this snapshot for the slide that the next network kernel computes).
struct SlidePre {
    int32_t s, e, newest, sweep, nonfinite;
    int32_t pending;    // a slide of this state is outstanding (0 right after reset)
    int64_t nfe, hits, revisits, revisits_below;
};

// Geometry and device buffers handed to every kernel launcher. Per-sample buffers are
// stacked along a leading sample index n < N.
struct Dev {
    int32_t N;                 // samples
    int32_t T, P, D;
    int32_t C, Himg, Wimg;
    int32_t ntok, hidden;      // patch-MLP only
    double delta, tol;
    double revisit_thr;        // threshold of the revisit counters
    float* X;                  // [N][T+1][D] trajectories
    float* Xh;                 // [N][T][D]   cached inputs
    float* Eh;                 // [N][T][D]   cached outputs
    uint8_t* valid;            // [N][T]
    const float* noise;        // [N][T][D]   pre-sampled step noise z (eta > 0), else null
    double* coef;              // [T][3]      (alpha_i, b_i, sigma_i) in fp64
    float* lin_c;              // [T]         linear network coefficients (or null)
    double* part_res;          // [N][P][picard_blocks] fp64 partial sums of Eq. (2) residuals
    double* part_dev;          // [N][P][picard_blocks] fp64 partial sums of Eq. (4) deviations
    Ctrl* ctrl;                // [N]
    SlidePre* pre;             // [N] pre-slide snapshots (fused sweep), or null
    int32_t fused_slide;       // 1: the network kernel computes the slide (N = 1), no k_slide
    uint64_t* progress;        // [N] host-mapped words: sweeps << 32 | done << 31 | nonfinite << 30 | s
    uint64_t* counters;        // [N][4] host-mapped final counters (epoch << 40 | value) or null
    uint32_t epoch;            // sample epoch of the counter words (24 bits, set at reset)
    pa_sweep_trace_t* trace;   // [N][T] or null
    // patch-MLP weights in device layouts
    const __bf16* w1t;         // [hidden][16]     (transposed W1)
    const __bf16* w2f;         // W2^T fragment-major: [hidden/32][hidden/16][64 lanes][8]
    const __bf16* w3p;         // [hidden/32][2][64][8] lane-permuted W3 fragments
    float* temb;               // [T][hidden]      e_j = temb(t_j) Wt
    float* Ep;                 // [nsplit][N][P][D] per-half network outputs of the misses
    int32_t nsplit;            // halves of the output units (partials summed by k_picard)
    int32_t* eps_whole;        // [1] set by each network launch: 1 = it wrote whole outputs
                               // into Eh, 0 = split partials into Ep; null = always split
    int32_t picard_blocks;
    int32_t mlp_grid;
    // Parareal sampler only (k_parareal.hip)
    float* Gc;                         // [B][D] stored coarse values G_n
    double* pr_coef;                   // [B][2] coarse step (ac_n, bc_n)
    pa_request_trace_t* trace_pr;      // request records or null
    float* trace_eps;                  // [records][D] fresh outputs of the misses, or null
    double* trace_res;                 // [B][B+1] boundary residuals per iteration, or null
};

// Kernel launchers (all asynchronous on `st`).
hipError_t launch_reset(const Dev& d, hipStream_t st);
// start/stop: optional events attached to the kernel's dispatch (null = untimed).
hipError_t launch_slide(const Dev& d, hipStream_t st, hipEvent_t start, hipEvent_t stop);
// The slide outstanding after a fused sweep, from the Picard kernel's snapshot (no-op if none).
hipError_t launch_slide_pending(const Dev& d, hipStream_t st);
// Largest fp64 partial-sum volume per sample the network kernel reduces redundantly per block.
constexpr size_t kFusedSlideMaxBytes = 256 * 1024;
hipError_t launch_picard(const Dev& d, hipStream_t st, int linear, hipEvent_t start, hipEvent_t stop);
// single: the launch evaluates at most one latent (64-token work items).
hipError_t launch_eps_mlp(const Dev& d, hipStream_t st, hipEvent_t start, hipEvent_t stop, int single = 0);
// Rearranges the patch-MLP weights ([in][out] bf16 bit patterns, device) into the network
// kernel's layouts: w1t [H][16], w2f (W2^T fragments, halved), w3p (lane-permuted W3
// fragments, halved).
hipError_t launch_pack_weights(const uint16_t* w1, const uint16_t* w2, const uint16_t* w3, int H,
                               __bf16* w1t, __bf16* w2f, __bf16* w3p, hipStream_t st);
hipError_t launch_temb_table(const Dev& d, const double* t_values_dev, const __bf16* wt_dev,
                             int temb_dim, hipStream_t st);
int picard_blocks(int D, int P);
int mlp_supported(int hidden);
int mlp_tokens_per_item();
int mlp_splits(int hidden);
int mlp_grid_size(int device_cus);

}  // namespace pa
