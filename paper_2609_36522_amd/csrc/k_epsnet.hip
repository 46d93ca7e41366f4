// Batched evaluation of the cache misses by the patch-MLP noise network, one fused
// persistent kernel for gfx950 (the single batched forward pass over the misses, Sec. 2.2).
//
// Work item = (miss j, block of 128 tokens, half of the hidden-out units of GEMM2). The
// misses of all samples of a handle form one list (sample-major, each sample's misses in
// its ascending order); a prefix over the samples' miss counts maps a list entry back to
// (sample, miss). For one item the block
//   0. gathers the 128 tokens (2x2 patches, 16 features) of latent x_t, rounds to bf16;
//   1. h1^T = GELU(W1^T x^T + e_t) in K-chunks of 256 units: MFMA 32x32x16 bf16, K = 16, e_t as
//      the accumulator's initial value; bf16 result (as 2 h1, with W2 stored halved) in LDS
//      ([token][unit], padded rows), two chunk buffers of 66 KB;
//   2. h2^T += W2^T h1^T chunk by chunk: each of the 8 waves owns 64 output units x 128
//      tokens (128 accumulator registers); W2^T fragments stream from L2 in MFMA-fragment
//      order (1 KB contiguous per wave load), two register stages in flight; the GEMM1 and
//      GELU of the next chunk are computed between the MFMA groups of the current one;
//   3. eps^T = W3^T GELU(h2^T), MFMA fed straight from the GEMM2 accumulators (reduction
//      index permuted to the accumulator layout; W3 stored pre-permuted);
//   4. per-wave partials summed in a fixed order through LDS and unpatchified.
// Two ways to finish (chosen per launch from the miss count, identically in every block,
// by the time each takes):
//   split outputs: each item is a work item of its own and writes its half's partial output;
//      the Picard kernel adds the halves in a fixed order and writes the cache;
//   whole outputs (at most two halves): one block runs both halves of a token block in turn,
//      adds their outputs in the same fixed order and writes the fresh output straight into
//      the cache (Eq. (6)-(7), output side). The second half takes its K-chunks in the order
//      2, 3, 1, 0 (generally H/256 - 2, H/256 - 1, H/256 - 3, ..., 0), so the first of them is
//      the h1 chunk the first half left in LDS: no gather, no h1 prologue, one chunk of GELU
//      work less. Odd halves take that order in both ways, so both give the same bits.
// 128 tokens per item make every W2 byte feed 128 FLOP, which keeps the W2 stream under the
// per-CU vector-memory bandwidth; the price is computing h1 (largely) once per half.
// All products are bf16 x bf16 with fp32 accumulation.
//
// Accumulator layout of v_mfma_f32_32x32x16_bf16 (C/D, 16 floats per lane):
//   reg r of lane l holds row (r/4)*8 + (l/32)*4 + r%4, column l%32.
// Operands: lane l supplies row l%32 of A (column l%32 of B) and 8 reduction slots; A and B
// use the same lane->slot convention, so any consistent slot->k assignment is valid.
#include <math.h>

#include <type_traits>

#include <hip/hip_ext.h>

#include "pa_device.h"
#include "pa_slide.h"

namespace pa {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kTokMax = 128;            // tokens per work item (64 for single-latent launches)
constexpr int kNH = 512;                // GEMM2 output units per work item
constexpr int kKC = 256;                // h1 units per LDS buffer (K-chunk); two buffers
constexpr int kWaves = 8;               // wave w owns output units [64w, 64w + 64) of the item
constexpr int kFeat = 16;               // 2x2 patch x 4 channels
constexpr int kXRow = kFeat + 8;        // padded LDS row of the token tile (bf16)

// Twice the erf-GELU: 2 x Phi(x) = (x + a) - a 2Q(a) with a = |x| and Q the normal upper tail,
// branch-free (x + a = 2 max(x, 0) exactly). 2Q(a) = 2^(-(P(a) - 1)) with P a degree-7
// polynomial fitted to -log2 Q on [0, 7] toward the minimax absolute error of the result
// (derivation: gelu_fit.py: what a deviation costs once the output is rounded to bf16 is its
// absolute size), its constant term lowered by 1. P increases monotonically for all a >= 0 and
// keeps tracking -log2 Q beyond 7 (a Q(a) < 1e-11 there); for very large a it overflows to
// +inf and Q to 0, so no clamp is needed. One v_add_f32, eight FMAs and one v_exp_f32 per
// element; in fp32 the result is within 4e-7 max(1, |x|) of twice the exact erf GELU. The
// factor 2 is exact and is undone exactly in the next product: W2 and W3 are stored halved
// (bf16 halving is exact for normal values), and bf16(2g) = 2 bf16(g), so every bf16 x bf16
// product equals the one with GELU(x) and the unhalved weight. Every GELU output is rounded to
// bf16 next; the residual error is kept within a few fp32 rounding errors of the result so
// that it adds few rounding flips to those of the fp32 accumulation of the products.
__device__ __forceinline__ float gelu2_erf(float x) {
    const float a = fabsf(x);
    float p = fmaf(a, 1.1180667343069217e-06f, -4.9184127419721335e-05f);
    p = fmaf(p, a, 0.0008520559640601277f);
    p = fmaf(p, a, -0.008282574824988842f);
    p = fmaf(p, a, 0.05366271361708641f);
    p = fmaf(p, a, 0.45861566066741943f);
    p = fmaf(p, a, 1.1512444019317627f);
    p = fmaf(p, a, -1.0669231414794922e-05f);   // P(a) - 1
    const float q2 = __builtin_amdgcn_exp2f(-p);  // 2 Q(a)
    return fmaf(-a, q2, x + a);
}

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Element index of the token tile <-> latent position. Consecutive e walk along w so that
// global accesses of a block are row-contiguous.
struct TokPos {
    int tl, f, idx;
};
template <int kTok>
__device__ __forceinline__ TokPos tok_pos(int e, int tb, int Himg, int Wimg) {
    constexpr int kLog = kTok == 128 ? 7 : 6;
    static_assert(kTok == (1 << kLog), "64 or 128 tokens per item");
    const int dw = e & 1, tl = (e >> 1) & (kTok - 1), dh = (e >> (kLog + 1)) & 1, c = e >> (kLog + 2);
    const int half_w = Wimg >> 1;
    const int tok = tb * kTok + tl;
    const int hp = tok / half_w, wp = tok - hp * half_w;
    TokPos p;
    p.tl = tl;
    p.f = c * 4 + dh * 2 + dw;
    p.idx = (c * Himg + 2 * hp + dh) * Wimg + 2 * wp + dw;
    return p;
}

}  // namespace

// TOK: tokens per work item, 128, or 64 for launches of a single latent (twice the work items,
// each half as long, where 128-token items would leave most CUs idle).
template <int H, int TOK>
__global__ __launch_bounds__(kWaves * 64) void k_eps_mlp(Dev d) {
    constexpr int NT = kWaves * 64;
    constexpr int kTok = TOK;
    constexpr int TB4 = kTok / 32;       // 32-token slices per item
    constexpr int NS = H / kNH;          // halves of the output units (work items per tokens)
    constexpr int KCH = H / kKC;         // K-chunks of h1
    constexpr int HRow = kKC + 8;        // padded LDS row of h1 (bf16)
    constexpr int KS = H / 16;           // GEMM2 k-steps (fragment columns of W2^T)
    constexpr int KBC = kKC / 32;        // k-blocks (two k-steps) per chunk
    constexpr int ITER = KBC / 2;        // pipelined iterations per chunk
    static_assert(H % kNH == 0 && H % kKC == 0 && ITER == 4, "unsupported hidden width");
    static_assert(kKC == kWaves * 32, "each wave computes 32 h1 units of a chunk");
    // h1 chunks, double-buffered: chunk c + 1 is computed while GEMM2 consumes chunk c.
    __shared__ __attribute__((aligned(16))) __bf16 h1s[2][kTok * HRow];
    __shared__ __attribute__((aligned(16))) __bf16 xs[kTok * kXRow];
    // e_t of the item's timestep. Read from LDS in the GELU slices: a global load there
    // would share the in-order vector-memory counter with the W2 prefetch, and waiting for
    // it would wait for the prefetched fragments too.
    __shared__ __attribute__((aligned(16))) float es[H];
    // [kWaves][kTok][16] after GEMM2, in the h1 buffer of the last chunk (the other buffer keeps
    // the chunk a whole-output block reuses for the item's second half).
    float* red = reinterpret_cast<float*>(&h1s[1][0]);
    static_assert(kWaves * kTok * kFeat * 4 <= kTok * HRow * 2, "reduction buffer must fit");
    static_assert(KCH % 2 == 0, "the last chunk of either order is consumed from buffer 1");

    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave index, in a scalar register
    // Misses per sample (0 once a sample is done), inclusive prefix over the samples.
    __shared__ int mpre[PA_MAX_BATCH + 1];
    static_assert(PA_MAX_BATCH <= 64, "one wave scans the samples");
    // Fused sweep (one sample): every block computes the outstanding window slide itself from
    // the Picard kernel's snapshot and partial sums (block 0 publishes it), and keeps the miss
    // list and the newest computed state in LDS; nothing this kernel writes is read back by it.
    __shared__ int fmiss[PA_MAX_WINDOW];
    __shared__ int fnewest;
    if (d.fused_slide) {
        // A launch queued after the one that finished the sample (that launch computed the last
        // slide and published done) has nothing to do: every block leaves at once.
        if (d.ctrl->done) return;
        static_assert(sizeof(SlideScratch) + 16 + kSlideSubDoubles * sizeof(double) <= sizeof(h1s),
                      "slide scratch must fit");
        SlideScratch& sc = *reinterpret_cast<SlideScratch*>(&h1s[0][0]);
        double* sub = reinterpret_cast<double*>(&h1s[0][0] + (sizeof(SlideScratch) + 15) / 16 * 8);
        const SlidePre pre = d.pre[0];
        slide_partials<NT>(d, 0, sub);       // its loads do not wait for the snapshot
        __syncthreads();
        if (pre.pending) {
            slide_core<NT>(d, 0, pre, blockIdx.x == 0, sc, sub);
            const int m = sc.done ? 0 : sc.m;
            for (int j = tid; j < m; j += NT) fmiss[j] = sc.miss_idx[j];
            if (tid == 0) {
                mpre[0] = 0;
                mpre[1] = m;
                fnewest = sc.newest;
            }
        } else {                             // first sweep after reset: the reset's window
            const Ctrl* c = d.ctrl;
            const int m = c->done ? 0 : c->m;
            for (int j = tid; j < m; j += NT) fmiss[j] = c->miss_idx[j];
            if (tid == 0) {
                mpre[0] = 0;
                mpre[1] = m;
                fnewest = c->newest;
            }
        }
    } else if (w == 0) {
        int v = 0;
        if (lane < d.N) v = d.ctrl[lane].done ? 0 : d.ctrl[lane].m;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int u = __shfl_up(v, off, 64);
            if (lane >= off) v += u;
        }
        if (lane < d.N) mpre[lane + 1] = v;
        if (lane == 0) mpre[0] = 0;
    }
    __syncthreads();
    const int nblk = d.ntok / kTok;
    const int tblocks = mpre[d.N] * nblk;            // (miss, token block) pairs
    const int G = gridDim.x;
    // Whole outputs (if the handle takes fresh outputs in the cache directly) unless they
    // lengthen the launch: a block's whole item costs about 15/16 of NS half items (one
    // gather and one h1 chunk fewer per extra half, measured ~4-6%), so they are taken when
    // 15/16 x NS x the rounds of whole items do not exceed the rounds of half items spread
    // over all blocks: with one item per block when more than half of the blocks get one,
    // and always from about 7 rounds on.
    const bool whole = d.eps_whole != nullptr && NS <= 2 &&
                       15 * NS * ((tblocks + G - 1) / G) <= 16 * ((tblocks * NS + G - 1) / G);
    if (d.eps_whole != nullptr && blockIdx.x == 0 && tid == 0) *d.eps_whole = whole ? 1 : 0;
    const int g = lane >> 5, l32 = lane & 31;
    // W2^T as a buffer resource (out-of-range loads would return zero)
    const __amdgpu_buffer_rsrc_t w2r = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<__bf16*>(d.w2f), (short)0, H * H * 2, 0x00020000);
    const f32x16 zero16 = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f,
                           0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    // K-chunk taken at position i: natural order for even halves; odd halves start with the
    // chunk a whole-output block still holds in buffer 0 (KCH - 2), then KCH - 1, KCH - 3, ..., 0.
    auto korder = [&](int odd, int i) {
        return !odd ? i : (i == 0 ? KCH - 2 : (i == 1 ? KCH - 1 : KCH - 1 - i));
    };
    float4 run = make_float4(0.f, 0.f, 0.f, 0.f);   // whole outputs: sum of the halves so far
    // One half (output units [512 ns, 512 ns + 512)) of the item (list entry gm, token block tb).
    // WHOLE: part of a whole-output block's item (ns > 0: the gather and the first h1 chunk of
    // the previous half are still in LDS).
    auto half = [&](int gm, int tb, int ns, bool whole_item) {
        int n = 0;
        while (mpre[n + 1] <= gm) ++n;               // sample of list entry gm (uniform)
        const int jm = gm - mpre[n];
        const Ctrl* ctrl = d.ctrl + n;
        const int t = d.fused_slide ? fmiss[jm] : ctrl->miss_idx[jm];
        const int newest = d.fused_slide ? fnewest : ctrl->newest;
        const int hb0 = ns * (kNH / 32) + w * 2;   // this wave's first 32-unit block of W2^T

        const int odd = ns & 1;
        const bool reuse = whole_item && ns > 0;      // tokens, e_t and chunk KCH - 2 in LDS
        // ---- 0. gather + patchify + bf16; e_t into LDS
        if (reuse) {
            __syncthreads();                 // the previous half's reduction reads are done
        } else {
            const float* xt = d.X + ((size_t)n * (d.T + 1) + min(t, newest)) * d.D;   // beyond newest: its copy
            const float* et = d.temb + (size_t)t * H;
            // Every load of the thread is issued before the first LDS store, so the block waits
            // for one round trip to memory instead of one per element.
            constexpr int kPer = kTok * kFeat / NT;
            static_assert(kPer * NT == kTok * kFeat, "one element per thread and round");
            constexpr int kEs = (H / 4 + NT - 1) / NT;
            float xv[kPer];
            float4 ev[kEs];
#pragma unroll
            for (int k = 0; k < kPer; ++k) xv[k] = xt[tok_pos<kTok>(tid + k * NT, tb, d.Himg, d.Wimg).idx];
#pragma unroll
            for (int k = 0; k < kEs; ++k)
                if (tid + k * NT < H / 4) ev[k] = reinterpret_cast<const float4*>(et)[tid + k * NT];
#pragma unroll
            for (int k = 0; k < kPer; ++k) {
                const TokPos p = tok_pos<kTok>(tid + k * NT, tb, d.Himg, d.Wimg);
                xs[p.tl * kXRow + p.f] = (__bf16)xv[k];
            }
#pragma unroll
            for (int k = 0; k < kEs; ++k)
                if (tid + k * NT < H / 4) reinterpret_cast<float4*>(es)[tid + k * NT] = ev[k];
            __syncthreads();
        }

        // ---- 1. h1 = GELU(x W1 + e_t): wave w computes units [32w, 32w + 32) of a chunk,
        // one 32-token slice per call, into LDS rows [token][unit].
        bf16x8 w1a;
        const float* ek = es;                // e_t of the chunk's units (LDS)
        auto h1_setup = [&](int kc) {
            const int n0 = kc * kKC + w * 32;
            w1a = *reinterpret_cast<const bf16x8*>(d.w1t + (size_t)(n0 + l32) * kFeat + g * 8);
            ek = es + n0 + g * 4;
        };
        f32x16 h1acc;
        // The accumulator starts at e_t (row = unit), so the MFMA returns x W1 + e_t; the
        // GELU slices store 2 h1 (W2 is stored halved, see gelu2_erf).
        auto h1_mfma = [&](int tb4) {
            const bf16x8 b = *reinterpret_cast<const bf16x8*>(xs + (tb4 * 32 + l32) * kXRow + g * 8);
            f32x16 c0;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float4 ev = *reinterpret_cast<const float4*>(ek + q * 8);
                c0[q * 4 + 0] = ev.x;
                c0[q * 4 + 1] = ev.y;
                c0[q * 4 + 2] = ev.z;
                c0[q * 4 + 3] = ev.w;
            }
            h1acc = mfma32(w1a, b, c0);
        };
        auto h1_gelu = [&](__bf16* buf, int kc, int tb4, int q0) {   // units q0*8.. of the slice
            const int tok = tb4 * 32 + l32;
#pragma unroll
            for (int q = q0; q < q0 + 2; ++q) {
                bf16x4 v;
#pragma unroll
                for (int i = 0; i < 4; ++i) v[i] = (__bf16)gelu2_erf(h1acc[q * 4 + i]);
                *reinterpret_cast<bf16x4*>(buf + tok * HRow + w * 32 + q * 8 + g * 4) = v;
            }
        };
        auto h1_slice = [&](__bf16* buf, int kc, int tb4) {
            h1_mfma(tb4);
            h1_gelu(buf, kc, tb4, 0);
            h1_gelu(buf, kc, tb4, 2);
        };
        if (!reuse) {
            const int k0 = korder(odd, 0);
            h1_setup(k0);
#pragma unroll
            for (int tb4 = 0; tb4 < TB4; ++tb4) h1_slice(h1s[0], k0, tb4);
            __syncthreads();
        }

        f32x16 acc2[2][TB4];
#pragma unroll
        for (int hb = 0; hb < 2; ++hb)
#pragma unroll
            for (int tb4 = 0; tb4 < TB4; ++tb4) acc2[hb][tb4] = zero16;

        // W2^T fragments of k-block kb of chunk kc, for this wave's two 32-unit blocks.
        // Buffer loads: the fragment's byte offset is wave-uniform (a scalar register), the
        // lane's 16-byte slot is the only per-lane address part.
        auto load_a = [&](bf16x8 (&A)[2][2], int kc, int kb) {
            const int sb = (hb0 * KS + kc * (kKC / 16) + 2 * kb) * 64 * 16;
#pragma unroll
            for (int hb = 0; hb < 2; ++hb)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    A[hb][j] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(
                        w2r, lane * 16, sb + (hb * KS + j) * 64 * 16, 0));
        };
        bf16x8 A0[2][2], A1[2][2];
        // GEMM2 MFMA group of k-block kb: 16 MFMAs over the four 32-token slices; the B
        // operands (h1^T from LDS) of slice tb4 + 1 are read while slice tb4 multiplies.
        auto mma = [&](const bf16x8 (&A)[2][2], const __bf16* h1b, int kb) {
            bf16x8 B[2][2];
#pragma unroll
            for (int j = 0; j < 2; ++j) B[0][j] = *reinterpret_cast<const bf16x8*>(h1b + kb * 32 + j * 16);
#pragma unroll
            for (int tb4 = 0; tb4 < TB4; ++tb4) {
                if (tb4 + 1 < TB4) {
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        B[(tb4 + 1) & 1][j] = *reinterpret_cast<const bf16x8*>(
                            h1b + (tb4 + 1) * 32 * HRow + kb * 32 + j * 16);
                }
#pragma unroll
                for (int j = 0; j < 2; ++j)
#pragma unroll
                    for (int hb = 0; hb < 2; ++hb)
                        acc2[hb][tb4] = mfma32(A[hb][j], B[tb4 & 1][j], acc2[hb][tb4]);
            }
        };
        // One chunk of GEMM2 at position i of the half's chunk order (two register stages of
        // W2^T fragments, the stream running on across chunk boundaries); position i is in
        // buffer i & 1. MORE: a chunk follows; its h1 slices are computed between the MFMA
        // groups (same basic block, so the VALU work of the GELU can be interleaved with the
        // MFMAs). A wave raises its issue priority while it feeds MFMA groups, so that the two
        // waves of a SIMD drift out of step (one in its MFMA group while the other is in its
        // GELU slice).
        auto chunk = [&](int i, auto more_c) {
            constexpr bool more = decltype(more_c)::value;
            const int kc = korder(odd, i);
            const int kn = more ? korder(odd, i + 1) : 0;
            if constexpr (more) h1_setup(kn);
            __bf16* nbuf = h1s[(i + 1) & 1];
            const __bf16* h1b = h1s[i & 1] + l32 * HRow + g * 8;
#pragma unroll
            for (int it = 0; it < ITER; ++it) {
                const int kb = 2 * it;
                load_a(A1, kc, kb + 1);
                __builtin_amdgcn_sched_barrier(0);
                __builtin_amdgcn_s_setprio(1);
                mma(A0, h1b, kb);
                if constexpr (more) {
                    if (it < TB4) h1_slice(nbuf, kn, it);   // one 32-token slice per iteration
                }
                __builtin_amdgcn_sched_barrier(0);
                __builtin_amdgcn_s_setprio(0);
                // Next fragments: this chunk's, or the first of the next chunk (after the
                // last chunk an unused reload of chunk 0, kept unconditional so the wait for
                // A1 below counts exactly these four loads as younger).
                if (kb + 2 < KBC) load_a(A0, kc, kb + 2);
                else load_a(A0, kn, 0);
                __builtin_amdgcn_sched_barrier(0);
                __builtin_amdgcn_s_setprio(1);
                mma(A1, h1b, kb + 1);
                __builtin_amdgcn_s_setprio(0);
                __builtin_amdgcn_sched_barrier(0);
            }
            __syncthreads();                 // chunk kc + 1 complete; chunk kc's buffer free
        };
        load_a(A0, korder(odd, 0), 0);
        for (int i = 0; i + 1 < KCH; ++i) chunk(i, std::true_type{});
        chunk(KCH - 1, std::false_type{});

        // ---- 3. eps^T partial = W3p GELU(h2^T) straight from the accumulators (2 GELU with W3
        // stored halved)
        f32x16 acc3[TB4];
#pragma unroll
        for (int tb4 = 0; tb4 < TB4; ++tb4) acc3[tb4] = zero16;
#pragma unroll
        for (int hb = 0; hb < 2; ++hb) {
#pragma unroll
            for (int jj = 0; jj < 2; ++jj) {
                const bf16x8 a3 = *reinterpret_cast<const bf16x8*>(
                    d.w3p + (((size_t)(hb0 + hb) * 2 + jj) * 64 + lane) * 8);
#pragma unroll
                for (int tb4 = 0; tb4 < TB4; ++tb4) {
                    bf16x8 b3;
#pragma unroll
                    for (int i = 0; i < 8; ++i) b3[i] = (__bf16)gelu2_erf(acc2[hb][tb4][jj * 8 + i]);
                    acc3[tb4] = mfma32(a3, b3, acc3[tb4]);
                }
            }
        }
        // valid rows of acc3: regs 0..7 -> feature (r/4)*8 + g*4 + r%4, token tb4*32 + l32
#pragma unroll
        for (int tb4 = 0; tb4 < TB4; ++tb4) {
            float* dst = red + ((size_t)w * kTok + tb4 * 32 + l32) * kFeat;
            *reinterpret_cast<float4*>(dst + g * 4) =
                make_float4(acc3[tb4][0], acc3[tb4][1], acc3[tb4][2], acc3[tb4][3]);
            *reinterpret_cast<float4*>(dst + 8 + g * 4) =
                make_float4(acc3[tb4][4], acc3[tb4][5], acc3[tb4][6], acc3[tb4][7]);
        }
        __syncthreads();

        // ---- 4. fixed-order sum over waves, unpatchify, store this half's partial output.
        // Thread = (channel c, token tl): its four features c*4 + dh*2 + dw are contiguous in
        // the reduction buffer and form two float2 pairs (dw = 0, 1) in rows 2hp and 2hp + 1.
        // Split outputs: this half's partial output; whole outputs: the running sum of the
        // halves (half 0 + half 1, the order the Picard kernel adds split partials in), stored
        // by the last half into the cache output of the miss.
        float* out = whole_item ? d.Eh + ((size_t)n * d.T + t) * d.D
                                : d.Ep + (((size_t)ns * d.N + n) * d.P + jm) * d.D;
        static_assert(kTok * (kFeat / 4) <= NT, "one token and channel per thread");
        if (tid < kTok * (kFeat / 4)) {
            const int tl = tid & (kTok - 1), c = tid / kTok;
            float4 sum = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int ww = 0; ww < kWaves; ++ww) {
                const float4 v = *reinterpret_cast<const float4*>(red + ((size_t)ww * kTok + tl) * kFeat + c * 4);
                sum.x += v.x;
                sum.y += v.y;
                sum.z += v.z;
                sum.w += v.w;
            }
            if (whole_item) {
                run = ns == 0 ? sum : make_float4(run.x + sum.x, run.y + sum.y, run.z + sum.z, run.w + sum.w);
                sum = run;
            }
            if (!whole_item || ns == NS - 1) {
                const int half_w = d.Wimg >> 1;
                const int tok = tb * kTok + tl;
                const int hp = tok / half_w, wp = tok - hp * half_w;
                float* o = out + ((size_t)c * d.Himg + 2 * hp) * d.Wimg + 2 * wp;
                *reinterpret_cast<float2*>(o) = make_float2(sum.x, sum.y);
                *reinterpret_cast<float2*>(o + d.Wimg) = make_float2(sum.z, sum.w);
            }
        }
        // No barrier: the next item's gather writes xs and es only, and its barrier comes
        // before anything overwrites the reduction buffer (h1 buffer 1); a whole-output
        // block's next half starts with one.
    };

    // One block item: both halves of a token block (whole) or one half (split).
    const int per = whole ? NS : 1;
    for (int item = blockIdx.x; item < tblocks * (NS / per); item += G) {
        const int tbk = whole ? item : item / NS;
        for (int q = 0; q < per; ++q) half(tbk / nblk, tbk % nblk, whole ? q : item % NS, whole);
    }
}

namespace {

// Half of a bf16 value on its bit pattern, rounded to nearest even. An exponent field of 2 or
// more drops by one (exact). Below that (subnormals and the smallest binade) the magnitude
// bits read as an integer are the value in units of 2^-133, which is halved with ties to even;
// the result is again such a magnitude. NaN is returned quiet, infinity unchanged.
__device__ __forceinline__ uint16_t bf16_half_bits(uint16_t b) {
    const uint16_t sgn = b & 0x8000u, mag = b & 0x7fffu;
    if (mag > 0x7f80u) return b | 0x0040u;
    if (mag == 0x7f80u) return b;
    if (mag >= 0x0100u) return sgn | (uint16_t)(mag - 0x0080u);
    const uint16_t q = mag >> 1;
    return sgn | (uint16_t)(q + ((mag & 1u) & (q & 1u)));
}

// Device layouts of the weights (grid-stride over the three outputs):
//   w1t[n][f] = W1[f][n];
//   w2f: W2^T as MFMA A fragments, fragment (b, ks) = lanes l = 0..63 x 8 values
//        W2[16 ks + 8 (l/32) + i][32 b + l%32] / 2;
//   w3p: fragment (hb, jj) = lanes l x 8 values W3[32 hb + (2 jj + i/4) 8 + 4 (l/32) + i%4][l%32] / 2
//        for l%32 < 16, else 0 (the reduction index permuted to the GEMM2 accumulator layout).
// W2 and W3 are stored halved because the kernel feeds them twice the GELU outputs.
__global__ void k_pack_weights(const uint16_t* __restrict__ w1, const uint16_t* __restrict__ w2,
                               const uint16_t* __restrict__ w3, int H, uint16_t* __restrict__ w1t,
                               uint16_t* __restrict__ w2f, uint16_t* __restrict__ w3p) {
    const size_t n1 = (size_t)H * 16, n2 = (size_t)H * H, n3 = (size_t)H * 32;
    const int KS = H / 16;
    for (size_t e = blockIdx.x * (size_t)blockDim.x + threadIdx.x; e < n1 + n2 + n3;
         e += (size_t)gridDim.x * blockDim.x) {
        if (e < n1) {
            const int n = (int)(e / 16), f = (int)(e % 16);
            w1t[e] = w1[(size_t)f * H + n];
        } else if (e < n1 + n2) {
            const size_t q = e - n1;
            const int i = (int)(q & 7), lane = (int)((q >> 3) & 63);
            const size_t frag = q >> 9;
            const int ks = (int)(frag % KS), b = (int)(frag / KS);
            const int n = b * 32 + (lane & 31), k = ks * 16 + (lane >> 5) * 8 + i;
            w2f[q] = bf16_half_bits(w2[(size_t)k * H + n]);
        } else {
            const size_t q = e - n1 - n2;
            const int i = (int)(q & 7), lane = (int)((q >> 3) & 63);
            const size_t rest = q >> 9;
            const int jj = (int)(rest & 1), hb = (int)(rest >> 1);
            const int g = lane >> 5, f = lane & 31;
            const int n = hb * 32 + (jj * 2 + i / 4) * 8 + g * 4 + (i % 4);
            w3p[q] = f < 16 ? bf16_half_bits(w3[(size_t)n * 16 + f]) : (uint16_t)0;
        }
    }
}

}  // namespace

hipError_t launch_pack_weights(const uint16_t* w1, const uint16_t* w2, const uint16_t* w3, int H,
                               __bf16* w1t, __bf16* w2f, __bf16* w3p, hipStream_t st) {
    hipLaunchKernelGGL(k_pack_weights, dim3(1024), dim3(256), 0, st, w1, w2, w3, H,
                       reinterpret_cast<uint16_t*>(w1t), reinterpret_cast<uint16_t*>(w2f),
                       reinterpret_cast<uint16_t*>(w3p));
    return hipGetLastError();
}

int mlp_supported(int hidden) { return hidden == 512 || hidden == 1024 || hidden == 2048; }

int mlp_tokens_per_item() { return kTokMax; }

int mlp_splits(int hidden) { return hidden / kNH; }

int mlp_grid_size(int device_cus) { return device_cus > 0 ? device_cus : 256; }

hipError_t launch_eps_mlp(const Dev& d, hipStream_t st, hipEvent_t start, hipEvent_t stop, int single) {
    const dim3 grid(d.mlp_grid), block(kWaves * 64);
    switch (d.hidden * 2 + (single ? 1 : 0)) {
        case 512 * 2: hipExtLaunchKernelGGL((k_eps_mlp<512, 128>), grid, block, 0, st, start, stop, 0, d); break;
        case 512 * 2 + 1: hipExtLaunchKernelGGL((k_eps_mlp<512, 64>), grid, block, 0, st, start, stop, 0, d); break;
        case 1024 * 2: hipExtLaunchKernelGGL((k_eps_mlp<1024, 128>), grid, block, 0, st, start, stop, 0, d); break;
        case 1024 * 2 + 1: hipExtLaunchKernelGGL((k_eps_mlp<1024, 64>), grid, block, 0, st, start, stop, 0, d); break;
        case 2048 * 2: hipExtLaunchKernelGGL((k_eps_mlp<2048, 128>), grid, block, 0, st, start, stop, 0, d); break;
        case 2048 * 2 + 1: hipExtLaunchKernelGGL((k_eps_mlp<2048, 64>), grid, block, 0, st, start, stop, 0, d); break;
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace pa
