// The window slide of one sample (Eq. (2) convergence, Sec. 2.1 slide; then the next window's
// Eq. (4)-(5) hit test and the ascending compaction of its misses), as a block-wide device
// function. It runs in k_slide (one block per sample) and, in the fused sweep, redundantly in
// every block of the network kernel, which needs the next window's miss list before its first
// work item.
//
// Everything it writes is a function of the pre-slide state `pre` and the Picard kernel's
// partial sums, never of the control block it writes: computing the same slide twice (a
// finishing k_slide and then the next network kernel, or two network kernels without a Picard
// kernel between them once the sample is done) writes the same values.
#pragma once

#include "pa_device.h"

namespace pa {

// Sub-sums per reduced value, and the LDS they need (doubles): fixed, so the order of every
// fp64 sum is the same in every kernel that computes the slide.
constexpr int kSlideSubs = 8;
constexpr int kSlideSubDoubles = 2 * PA_MAX_WINDOW * kSlideSubs;

// LDS of one slide. The caller's block must have at least 256 threads (waves 0-3 vote on the
// slots of the window).
struct SlideScratch {
    double r[PA_MAX_WINDOW];        // residuals of states s+1..e
    double dv[PA_MAX_WINDOW];       // deviations of states s+1..e-1 from their cache entries
    int wfirst[4], wbad[4], wcount[4], wrev[4], wbelow[4];
    int s2;                         // new window start
    int nonfinite;                  // sticky non-finite flag after this slide (writer only)
    // results for the caller (valid after the call on every thread)
    int done, m, newest;
    int miss_idx[PA_MAX_WINDOW];    // ascending misses of the next window
};

__device__ __forceinline__ SlidePre slide_pre_of(const Ctrl& c) {
    SlidePre p;
    p.s = c.s;
    p.e = c.e;
    p.newest = c.newest;
    p.sweep = c.sweep;
    p.nonfinite = c.nonfinite;
    p.pending = 1;
    p.nfe = c.nfe;
    p.hits = c.hits;
    p.revisits = c.revisits;
    p.revisits_below = c.revisits_below;
    return p;
}

// Sub-sums of the Picard kernel's partials of sample n into sub (kSlideSubDoubles doubles of
// LDS), for all P window slots whatever the window: it reads nothing else, so a caller can
// issue it before the pre-slide snapshot arrives. Reduction q (q < P: residual q; q >= P:
// deviation q - P) is later the fixed-order sum of its kSlideSubs sub-sums, sub-sum u adding
// the partials u, u + kSlideSubs, ... in order. The order does not depend on the block size,
// so every caller (k_slide, the fused network kernel) obtains the same fp64 values bit for
// bit; the loads of a sub-sum are independent. Slots beyond the window hold stale partials,
// summed and never used. The caller synchronizes the block before slide_core. A thread issues
// the loads of kSlideBatch partials of a sub-sum at once (one base address, constant offsets),
// then adds them in order: one round trip to L2 per 32 partials instead of one per few loads;
// the partials after the last whole batch follow one by one, in the same order.
constexpr int kSlideBatch = 32;

template <int NT>
__device__ void slide_partials(const Dev& d, int n, double* sub) {
    const int tid = threadIdx.x;
    const int nblk = d.picard_blocks, P = d.P;
    const size_t pbase = (size_t)n * P * nblk;
    for (int idx = tid; idx < 2 * P * kSlideSubs; idx += NT) {
        const int q = idx / kSlideSubs, u = idx - q * kSlideSubs;
        const double* pr = (q < P) ? d.part_res + pbase + (size_t)q * nblk
                                   : d.part_dev + pbase + (size_t)(q - P) * nblk;
        double acc = 0.0;
        int b = u;
        for (; b + (kSlideBatch - 1) * kSlideSubs < nblk; b += kSlideBatch * kSlideSubs) {
            double v[kSlideBatch];
#pragma unroll
            for (int i = 0; i < kSlideBatch; ++i) v[i] = pr[b + i * kSlideSubs];
#pragma unroll
            for (int i = 0; i < kSlideBatch; ++i) acc += v[i];
        }
        for (; b < nblk; b += kSlideSubs) acc += pr[b];
        sub[idx] = acc;
    }
}

// Progress word of sample n for the host's launch loop (pinned host memory, system scope):
// completed sweeps << 32 | done << 31 | nonfinite << 30 | window start (at most T < 2^30).
// The host reads the words, and the counter words of a done sample; anything else only after
// synchronizing the stream.
__device__ __forceinline__ void publish_progress(const Dev& d, int n, int sweeps, int done, int nonfinite,
                                                 int s) {
    const uint64_t word = ((uint64_t)(uint32_t)sweeps << 32) | ((uint64_t)(done ? 1 : 0) << 31) |
                          ((uint64_t)(nonfinite ? 1 : 0) << 30) | (uint64_t)(uint32_t)s;
    __hip_atomic_store(d.progress + n, word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Every thread of the block calls it (it synchronizes the block), after slide_partials into
// sub and a block barrier. With `writer` the block publishes the result to the control block,
// the trace and the progress word.
template <int NT>
__device__ void slide_core(const Dev& d, int n, const SlidePre& pre, bool writer, SlideScratch& sc,
                           const double* sub) {
    static_assert(NT >= 256, "block too small for the slide");
    Ctrl* ctrl = d.ctrl + n;
    pa_sweep_trace_t* const trace = (writer && d.trace) ? d.trace + (size_t)n * d.T : nullptr;
    const int s = pre.s, e = pre.e, W = e - s;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int P = d.P;

    // Residuals r of states s+1..e and deviations of states s+1..e-1.
    for (int i = tid; i < 2 * W; i += NT) {
        const int q = i < W ? i : P + (i - W);
        double v = 0.0;
#pragma unroll
        for (int u = 0; u < kSlideSubs; ++u) v += sub[q * kSlideSubs + u];
        if (i < W) sc.r[i] = v / (double)d.D;
        else sc.dv[i - W] = v / (double)d.D;
    }
    __syncthreads();

    // Eq. (2): slot j stops the leading run if not converged or if it is the last slot.
    {
        const int j = tid;
        const double r = j < W ? sc.r[j] : 0.0;
        const bool stop = (j < 256) && ((j >= W - 1) || !(r <= d.tol));
        const bool bad = (j < W) && !isfinite(r);
        const unsigned long long sm = __ballot(stop);
        const unsigned long long bm = __ballot(bad);
        if (wave < 4 && lane == 0) {
            sc.wfirst[wave] = sm ? wave * 64 + __ffsll((long long)sm) - 1 : 1 << 30;
            sc.wbad[wave] = bm != 0ull;
        }
        if (trace && j < W) trace[pre.sweep].resid[j] = r;
    }
    __syncthreads();
    if (tid == 0) {
        int c = 1 << 30, anybad = 0;
        for (int w = 0; w < 4; ++w) {
            c = min(c, sc.wfirst[w]);
            anybad |= sc.wbad[w];
        }
        const int s2 = s + 1 + c;
        sc.s2 = s2;
        sc.done = s2 >= d.T;
        sc.newest = max(pre.newest, e);
        sc.m = 0;
        if (writer) {
            if (trace) {
                pa_sweep_trace_t* rec = trace + pre.sweep;
                rec->c = c;
                rec->s_next = s2;
                rec->sweep = pre.sweep;
            }
            ctrl->nonfinite = (pre.nonfinite || anybad) ? 1 : 0;
            ctrl->c = c;
            ctrl->newest = sc.newest;
            ctrl->s = s2;
            ctrl->e = min(s2 + d.P, d.T);
            ctrl->done = s2 >= d.T;
            ctrl->sweep = pre.sweep + 1;
            sc.nonfinite = (pre.nonfinite || anybad) ? 1 : 0;
        }
    }
    __syncthreads();
    const int s2 = sc.s2;
    if (s2 >= d.T) {                        // uniform; no next window, counters unchanged
        if (writer && tid == 0) {
            // The sample is done: its final counters for the host (tagged with the sample's
            // epoch, so that the host can tell them from an earlier sample's), then the word.
            if (d.counters) {
                const uint64_t tag = (uint64_t)(d.epoch & 0xffffffu) << 40;
                const int64_t v[4] = {pre.nfe, pre.hits, pre.revisits, pre.revisits_below};
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    __hip_atomic_store(d.counters + 4 * n + k, tag | ((uint64_t)v[k] & ((1ull << 40) - 1)),
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
            }
            publish_progress(d, n, pre.sweep + 1, 1, sc.nonfinite, d.T);
        }
        return;
    }

    // Next window [s2, e2): Eq. (4)-(5) for slots that hold a cache entry (t < e); first
    // entries (t >= e) are misses; compaction by wave ballots and LDS offsets.
    const int e2 = min(s2 + d.P, d.T), W2 = e2 - s2;
    const int next = pre.sweep + 1;         // index of the next sweep
    const int j = tid, t = s2 + j;
    double dev = __builtin_nan("");
    bool hit = false, miss = false, rev = false, below = false;
    if (j < W2) {
        if (t < e) {
            dev = sc.dv[t - s - 1];
            hit = dev < d.delta;            // strict: delta == 0 never hits
            rev = true;                     // t holds a cache entry: a revisit
            below = dev < d.revisit_thr;
        }
        miss = !hit;
    }
    const unsigned long long mask = __ballot(miss);
    const unsigned long long rmask = __ballot(rev);
    const unsigned long long bmask = __ballot(below);
    const int rank = __popcll(mask & lanemask_lt());
    if (wave < 4 && lane == 0) {
        sc.wcount[wave] = __popcll(mask);
        sc.wrev[wave] = __popcll(rmask);
        sc.wbelow[wave] = __popcll(bmask);
    }
    __syncthreads();
    if (j < 256) {
        int off = 0;
        for (int w = 0; w < wave; ++w) off += sc.wcount[w];
        const int m = sc.wcount[0] + sc.wcount[1] + sc.wcount[2] + sc.wcount[3];
        if (miss) sc.miss_idx[off + rank] = t;
        if (tid == 0) sc.m = m;
        if (writer) {
            if (miss) ctrl->miss_idx[off + rank] = t;
            if (j < W2) {
                ctrl->slot_miss[j] = miss ? 1 : 0;
                ctrl->slot_rank[j] = miss ? (uint8_t)(off + rank) : 0;
            }
            if (trace) {
                pa_sweep_trace_t* rec = trace + next;
                if (j < W2) {
                    rec->dev[j] = dev;
                    rec->hit[j] = hit ? 1 : 0;
                }
                if (miss) rec->miss_idx[off + rank] = t;
                if (tid == 0) {
                    rec->s = s2;
                    rec->e = e2;
                    rec->m = m;
                }
            }
            if (tid == 0) {
                ctrl->m = m;
                ctrl->nfe = pre.nfe + m;
                ctrl->hits = pre.hits + (W2 - m);
                ctrl->revisits = pre.revisits + sc.wrev[0] + sc.wrev[1] + sc.wrev[2] + sc.wrev[3];
                ctrl->revisits_below = pre.revisits_below + sc.wbelow[0] + sc.wbelow[1] + sc.wbelow[2] + sc.wbelow[3];
                publish_progress(d, n, pre.sweep + 1, 0, sc.nonfinite, s2);
            }
        }
    }
    __syncthreads();                        // results in sc visible to every thread
}

}  // namespace pa
