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

// Generalized DDIM step coefficients [T][3] = (alpha_i, b_i, sigma_i), fp64.
std::vector<double> step_coefficients(const std::vector<double>& ab, int T, double eta);

// Validates the network description for a C x Hi x Wi latent and T steps.
int check_eps_model(const pa_eps_model_t* em, int C, int Hi, int Wi, int T);

// Device allocations owned by a handle (freed in the destructor).
struct DevMem {
    std::vector<void*> ptrs;
    DevMem() = default;
    DevMem(const DevMem&) = delete;
    DevMem& operator=(const DevMem&) = delete;
    ~DevMem() {
        for (void* p : ptrs) (void)hipFree(p);
    }
    template <class T>
    int alloc(T** p, size_t count, const char* what) {
        void* q = nullptr;
        hipError_t e = hipMalloc(&q, count * sizeof(T) + 256);
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
// device layouts and the time-embedding table, plus the partial-output buffer Ep of
// nsplit x ep_rows latents. Synchronizes the stream before returning.
int setup_network(Dev& d, DevMem& mem, const pa_eps_model_t* em, const std::vector<double>& tv,
                  int cus, size_t ep_rows, hipStream_t st);

}  // namespace pa
