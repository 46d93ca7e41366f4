// Host-side helpers shared by the sampler handles of the C ABI: error reporting, the noise
// schedule, device allocations, kernel-attached timing events and the network upload.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "pa_internal.h"

namespace pa {

extern thread_local std::string g_err;

int fail(int code, const char* fmt, ...);
int hip_fail(hipError_t e, const char* what);

#define PA_HIP(call)                                           \
    do {                                                       \
        hipError_t e_ = (call);                                \
        if (e_ != hipSuccess) return ::pa::hip_fail(e_, #call); \
    } while (0)

// alpha_bar of the sampler states 0..T and the time values of steps 0..T-1 (see
// pa_schedule_t); validates the schedule, eta included.
int build_schedule(const pa_schedule_t* sc, int T, std::vector<double>& ab, std::vector<double>& tv);
// The same into caller arrays ab[T + 1], tv[T] (no allocation).
int build_schedule(const pa_schedule_t* sc, int T, double* ab, double* tv);

// Generalized DDIM step coefficients [T][3] = (alpha_i, b_i, sigma_i), fp64.
std::vector<double> step_coefficients(const std::vector<double>& ab, int T, double eta);
void step_coefficients(const double* ab, int T, double eta, double* coef);

// Validates the network description for a C x Hi x Wi latent and T steps.
int check_eps_model(const pa_eps_model_t* em, int C, int Hi, int Wi, int T);

// Device buffers of a handle: each allocated with hipMalloc and freed in the destructor, or,
// in workspace mode (workspace()), carved in order from a caller-given device range that
// the handle does not own (no allocation at all). Every buffer gets 256 bytes of slack past
// its end and starts 256-byte aligned.
struct DevMem {
    std::vector<void*> ptrs;
    char* ws = nullptr;       // workspace mode: base, capacity and bytes handed out
    size_t ws_cap = 0, ws_used = 0;
    DevMem() = default;
    DevMem(const DevMem&) = delete;
    DevMem& operator=(const DevMem&) = delete;
    ~DevMem() {
        for (void* p : ptrs) (void)hipFree(p);
    }
    void workspace(void* base, size_t cap) {
        ws = static_cast<char*>(base);
        ws_cap = cap;
        ws_used = 0;
    }
    template <class T>
    int alloc(T** p, size_t count, const char* what) {
        const size_t bytes = count * sizeof(T) + 256;
        if (ws) {
            const size_t need = ws_used + (bytes + 255) / 256 * 256;
            if (need > ws_cap)
                return fail(PA_ERR_INVALID_ARG, "workspace of %zu bytes too small: %s needs %zu more bytes after %zu",
                            ws_cap, what, bytes, ws_used);
            *p = reinterpret_cast<T*>(ws + ws_used);
            ws_used = need;
            return PA_OK;
        }
        void* q = nullptr;
        hipError_t e = hipMalloc(&q, bytes);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return fail(PA_ERR_OOM, "hipMalloc(%s, %zu bytes): %s", what, count * sizeof(T),
                        hipGetErrorString(e));
        }
        ptrs.push_back(q);
        *p = static_cast<T*>(q);
        return PA_OK;
    }
};

// Rate limit for polling a stream while the host spins on a progress word: hipStreamQuery on a
// stream with queued kernels delays the next dispatch on it (measured: ~5.5 us gaps between
// kernels that otherwise run back to back), so a waiting loop asks at most once per interval
// (and only to notice a failed or idle stream; progress itself comes from the word).
struct QueryPacer {
    static constexpr int64_t kIntervalNs = 1000000;   // 1 ms
    int64_t next_ns = 0;
    bool due();                        // true at most once per interval
};

// Start/stop event pairs attached to kernel dispatches (hipExtLaunchKernelGGL), summed per
// kernel kind when drained. A pair's interval can include idle time between the kernel and
// the work before it on the stream.
struct KernelTimer {
    static constexpr int kKinds = 3;
    std::vector<hipEvent_t> pool;
    std::vector<int> kind;             // kernel kind of each used pair
    size_t used = 0;                   // events handed out since the last drain
    int64_t launches[kKinds] = {0, 0, 0};
    double ms[kKinds] = {0.0, 0.0, 0.0};
    KernelTimer() = default;
    KernelTimer(const KernelTimer&) = delete;
    KernelTimer& operator=(const KernelTimer&) = delete;
    ~KernelTimer() {
        for (hipEvent_t e : pool) (void)hipEventDestroy(e);
    }
    int pair(int k, hipEvent_t* e0, hipEvent_t* e1);
    size_t pending() const { return kind.size(); }   // pairs handed out since the last drain
    int drain();                       // the stream must be synchronized
    void clear();
};

// Network tables on the device: the linear coefficients, or the patch-MLP weights in their
// device layouts and the time-embedding table (tv: time values of the T steps, host), plus
// the partial-output buffer Ep of nsplit x ep_rows latents. Enqueued on the stream; the
// caller's host arrays must stay valid until the stream has run the copies.
int setup_network(Dev& d, DevMem& mem, const pa_eps_model_t* em, const double* tv,
                  int cus, size_t ep_rows, hipStream_t st);

}  // namespace pa
