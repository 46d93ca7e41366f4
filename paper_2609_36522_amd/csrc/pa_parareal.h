// Internal declarations of the cached Parareal sampler (kernels in k_parareal.hip).
#pragma once

#include "pa_device.h"

namespace pa {

// Device control block of one Parareal handle.
struct alignas(64) PrCtrl {
    int32_t done;       // converged (Eq. (2) on every boundary) or B iterations done
    int32_t iters;      // completed iterations
    int32_t nonfinite;  // sticky: a boundary residual was NaN/Inf
    int32_t pad;
};

enum PrMode : int32_t { PR_INIT = 0, PR_FINE = 1, PR_COARSE = 2, PR_COPY = 3 };
enum PrKernel : int32_t { PRK_RESET, PRK_TEST, PRK_FINE, PRK_COARSE, PRK_CHECK };

// Per-launch arguments: which requests this launch serves.
struct PrArgs {
    int32_t mode;       // PrMode
    int32_t L;          // fine steps per block
    int32_t k;          // iteration (fine: blocks n >= k are active)
    int32_t j;          // fine step within the block
    int32_t n;          // block of a coarse request or copy
    int32_t rec;        // trace record index of the launch's first request
    int32_t nchunk;     // residual partials per boundary
    PrCtrl* pc;
};

hipError_t launch_pr(const Dev& d, const PrArgs& a, int kernel, hipStream_t st);
int pr_chunks(int D);

}  // namespace pa
