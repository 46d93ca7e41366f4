// Internal declarations shared by the host library and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "paraanya.h"

namespace pa {

// Device-resident control block of one handle. Every per-sweep decision lives here, so
// the host can enqueue sweeps without reading anything back.
struct alignas(256) Ctrl {
    int32_t s;          // window start: states 0..s are final
    int32_t e;          // window end: drift points s..e-1, updated states s+1..e
    int32_t newest;     // highest state index holding an estimate (above: stale)
    int32_t m;          // misses of the current sweep
    int32_t done;       // s >= T
    int32_t nonfinite;  // sticky: a residual was NaN/Inf
    int32_t c;          // leading converged count of the last sweep
    int32_t sweep;      // completed sweeps since reset
    int64_t nfe;
    int64_t hits;
    uint32_t cnt_test;    // arrival counter of the cache-test kernel (last block finalizes)
    uint32_t cnt_picard;  // arrival counter of the Picard kernel
    int32_t pad[2];
    int32_t miss_idx[PA_MAX_WINDOW];  // ascending miss timesteps
    uint8_t slot_miss[PA_MAX_WINDOW]; // per window slot j: 1 if t = s + j is a miss
};

// Geometry and device buffers handed to every kernel launcher.
struct Dev {
    int32_t T, P, D;
    int32_t C, Himg, Wimg;
    int32_t ntok, hidden;      // patch-MLP only
    double delta, tol;
    float* X;                  // [T+1][D] trajectory
    float* Xh;                 // [T][D]   cached inputs
    float* Eh;                 // [T][D]   cached outputs
    uint8_t* valid;            // [T]
    double* coef;              // [T][2]   (alpha_i, b_i) in fp64
    float* lin_c;              // [T]      linear network coefficients (or null)
    double* part_test;         // [(P+1) * test_chunks] fp64 partial sums
    double* part_res;          // [P * picard_blocks]   fp64 partial sums
    Ctrl* ctrl;
    pa_sweep_trace_t* trace;   // [T] or null
    // patch-MLP weights in device layouts
    const __bf16* w1t;         // [hidden][16]     (transposed W1)
    const __bf16* w2t;         // [hidden][hidden] (transposed W2: row = output unit)
    const __bf16* w3p;         // [hidden/32][2][64][8] lane-permuted W3 fragments
    float* temb;               // [T][hidden]      e_j = temb(t_j) Wt
    int32_t test_chunks;
    int32_t picard_blocks;
    int32_t mlp_grid;
};

// Kernel launchers (all asynchronous on `st`).
hipError_t launch_reset(const Dev& d, hipStream_t st);
hipError_t launch_cache_test(const Dev& d, hipStream_t st);
hipError_t launch_picard(const Dev& d, hipStream_t st, int linear);
hipError_t launch_eps_mlp(const Dev& d, hipStream_t st);
hipError_t launch_temb_table(const Dev& d, const double* t_values_dev, const __bf16* wt_dev,
                             int temb_dim, hipStream_t st);
int cache_test_chunks(int D);
int picard_blocks(int D);
int picard_tpt(int P);
int mlp_supported(int hidden);
int mlp_grid_size(int device_cus);

}  // namespace pa
