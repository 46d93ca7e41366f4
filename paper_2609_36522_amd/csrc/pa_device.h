// Device helpers shared by the solver and network kernels (wave64, gfx950).
#pragma once

#include "pa_internal.h"

namespace pa {

__device__ __forceinline__ double wave_sum(double v) {
    // Butterfly over the 64 lanes; the fixed pattern makes the result order-deterministic.
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__device__ __forceinline__ unsigned long long lanemask_lt() {
    const int lane = threadIdx.x & 63;
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

}  // namespace pa
