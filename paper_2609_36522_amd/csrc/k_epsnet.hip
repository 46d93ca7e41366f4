// Batched evaluation of the cache misses by the patch-MLP noise network, one fused
// persistent kernel for gfx950 (the "single batched forward pass" over the misses, Sec. 2.2).
//
// Work item = (miss j, block of 64 tokens). For one item the block
//   0. gathers the 64 tokens (2x2 patches, 16 features) of latent x_t, rounds to bf16;
//   1. h1^T = GELU(W1^T x^T + e_t)     : MFMA 32x32x16 bf16, K = 16; bf16 result kept in LDS;
//   2. h2^T = GELU(W2^T h1^T)          : MFMA 32x32x16 bf16, K = hidden; each wave owns 128
//                                        output units and streams its W2^T rows from L2;
//   3. eps^T = W3^T h2^T               : MFMA again, fed straight from the GEMM2 accumulators
//                                        (the reduction index is permuted to match the
//                                        accumulator layout; W3 is stored pre-permuted);
//   4. sums the per-wave partials in a fixed order, unpatchifies and writes Eh[t].
// All products are bf16 x bf16 with fp32 accumulation.
//
// Accumulator layout of v_mfma_f32_32x32x16_bf16 (C/D, 16 floats per lane):
//   reg r of lane l holds row (r/4)*8 + (l/32)*4 + r%4, column l%32.
// Operands: lane l supplies row l%32 of A (column l%32 of B) and 8 reduction slots; A and B
// use the same lane->slot convention, so any consistent slot->k assignment is valid.
#include <math.h>

#include "pa_internal.h"

namespace pa {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kTok = 64;                // tokens per work item
constexpr int kFeat = 16;               // 2x2 patch x 4 channels
constexpr int kXRow = kFeat + 8;        // padded LDS row of the token tile (bf16)

// erf-GELU, x * Phi(x), branch-free. The normal upper tail Q(a) = 1 - Phi(a), a = |x|, is
// Hastings' approximation (Abramowitz & Stegun 26.2.17): Q(a) = phi(a) t (b1 + t (b2 + ...)),
// t = 1 / (1 + p a), |error| < 7.5e-8; phi(a) = exp(-a^2/2) / sqrt(2 pi) is folded into the
// coefficients. Error of the result <= ~2.2e-7 |x| in fp32, far below the bf16 rounding that
// follows. One v_rcp_f32 and one v_exp_f32 per element.
__device__ __forceinline__ float gelu_erf(float x) {
    constexpr float kP = 0.2316419f;
    constexpr float kB1 = 0.319381530f * 0.39894228040143268f;
    constexpr float kB2 = -0.356563782f * 0.39894228040143268f;
    constexpr float kB3 = 1.781477937f * 0.39894228040143268f;
    constexpr float kB4 = -1.821255978f * 0.39894228040143268f;
    constexpr float kB5 = 1.330274429f * 0.39894228040143268f;
    constexpr float kHalfLog2e = -0.72134752044448170f;   // -log2(e) / 2
    const float a = fabsf(x);
    const float t = __builtin_amdgcn_rcpf(fmaf(kP, a, 1.0f));
    float poly = fmaf(t, kB5, kB4);
    poly = fmaf(t, poly, kB3);
    poly = fmaf(t, poly, kB2);
    poly = fmaf(t, poly, kB1);
    const float q = __builtin_amdgcn_exp2f(a * (a * kHalfLog2e)) * (poly * t);
    return x * (x >= 0.0f ? 1.0f - q : q);
}

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Element index of the token tile <-> latent position. Consecutive e walk along w so that
// global accesses of a block are row-contiguous.
struct TokPos {
    int tl, f, idx;
};
__device__ __forceinline__ TokPos tok_pos(int e, int tb, int Himg, int Wimg) {
    const int dw = e & 1, tl = (e >> 1) & 63, dh = (e >> 7) & 1, c = e >> 8;
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

template <int H>
__global__ __launch_bounds__(H / 2) void k_eps_mlp(Dev d) {
    constexpr int NW = H / 128;          // waves; wave w owns hidden units [128w, 128w+128)
    constexpr int NT = NW * 64;
    constexpr int HRow = H + 8;          // padded LDS row of h1 (bf16)
    constexpr int KB = H / 32;           // GEMM2 k-blocks of 32
    __shared__ __attribute__((aligned(16))) __bf16 h1s[kTok * HRow];
    __shared__ __attribute__((aligned(16))) __bf16 xs[kTok * kXRow];
    float* red = reinterpret_cast<float*>(h1s);   // [NW][kTok][16] after GEMM2

    const Ctrl* ctrl = d.ctrl;
    if (ctrl->done) return;
    const int nblk = d.ntok / kTok;
    const int items = ctrl->m * nblk;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int g = lane >> 5, l32 = lane & 31;
    const f32x16 zero16 = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f,
                           0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};

    for (int item = blockIdx.x; item < items; item += gridDim.x) {
        const int jm = item / nblk, tb = item - jm * nblk;
        const int t = ctrl->miss_idx[jm];
        const float* xt = d.X + (size_t)t * d.D;

        // ---- 0. gather + patchify + bf16
        for (int e = tid; e < kTok * kFeat; e += NT) {
            const TokPos p = tok_pos(e, tb, d.Himg, d.Wimg);
            xs[p.tl * kXRow + p.f] = (__bf16)xt[p.idx];
        }
        __syncthreads();

        // ---- 1. h1 = GELU(x W1 + e_t) -> bf16 in LDS, row = token
        {
            const float* et = d.temb + (size_t)t * H;
#pragma unroll
            for (int hb = 0; hb < 4; ++hb) {
                const int n0 = w * 128 + hb * 32;
                const bf16x8 a = *reinterpret_cast<const bf16x8*>(d.w1t + (size_t)(n0 + l32) * kFeat + g * 8);
                float4 ev[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) ev[q] = *reinterpret_cast<const float4*>(et + n0 + q * 8 + g * 4);
#pragma unroll
                for (int tb2 = 0; tb2 < 2; ++tb2) {
                    const int tok = tb2 * 32 + l32;
                    const bf16x8 b = *reinterpret_cast<const bf16x8*>(xs + tok * kXRow + g * 8);
                    const f32x16 acc = mfma32(a, b, zero16);
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        bf16x4 v;
                        v[0] = (__bf16)gelu_erf(acc[q * 4 + 0] + ev[q].x);
                        v[1] = (__bf16)gelu_erf(acc[q * 4 + 1] + ev[q].y);
                        v[2] = (__bf16)gelu_erf(acc[q * 4 + 2] + ev[q].z);
                        v[3] = (__bf16)gelu_erf(acc[q * 4 + 3] + ev[q].w);
                        *reinterpret_cast<bf16x4*>(h1s + tok * HRow + n0 + q * 8 + g * 4) = v;
                    }
                }
            }
        }
        __syncthreads();

        // ---- 2. h2^T = W2^T h1^T, k-block of 32: lane group g takes k = 32kb + 16g + [0,16)
        f32x16 acc2[4][2];
#pragma unroll
        for (int hb = 0; hb < 4; ++hb)
#pragma unroll
            for (int tb2 = 0; tb2 < 2; ++tb2) acc2[hb][tb2] = zero16;
        const __bf16* wrow = d.w2t + (size_t)(w * 128 + l32) * H + g * 16;
        bf16x8 A[4][2];
#pragma unroll
        for (int hb = 0; hb < 4; ++hb)
#pragma unroll
            for (int j = 0; j < 2; ++j)
                A[hb][j] = *reinterpret_cast<const bf16x8*>(wrow + (size_t)hb * 32 * H + j * 8);
        for (int kb = 0; kb < KB; ++kb) {
            bf16x8 An[4][2];
            const int kn = (kb + 1 < KB) ? kb + 1 : kb;
#pragma unroll
            for (int hb = 0; hb < 4; ++hb)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    An[hb][j] = *reinterpret_cast<const bf16x8*>(wrow + (size_t)hb * 32 * H + kn * 32 + j * 8);
            bf16x8 B[2][2];
#pragma unroll
            for (int tb2 = 0; tb2 < 2; ++tb2)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    B[tb2][j] = *reinterpret_cast<const bf16x8*>(h1s + (tb2 * 32 + l32) * HRow + kb * 32 + g * 16 + j * 8);
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int hb = 0; hb < 4; ++hb)
#pragma unroll
                    for (int tb2 = 0; tb2 < 2; ++tb2)
                        acc2[hb][tb2] = mfma32(A[hb][j], B[tb2][j], acc2[hb][tb2]);
#pragma unroll
            for (int hb = 0; hb < 4; ++hb)
#pragma unroll
                for (int j = 0; j < 2; ++j) A[hb][j] = An[hb][j];
        }

        // ---- 3. eps^T += W3p h2^T straight from the accumulators (slot jj*8+i <-> reg jj*8+i)
        f32x16 acc3[2] = {zero16, zero16};
#pragma unroll
        for (int hb = 0; hb < 4; ++hb) {
#pragma unroll
            for (int jj = 0; jj < 2; ++jj) {
                const bf16x8 a3 = *reinterpret_cast<const bf16x8*>(
                    d.w3p + (((size_t)(w * 4 + hb) * 2 + jj) * 64 + lane) * 8);
#pragma unroll
                for (int tb2 = 0; tb2 < 2; ++tb2) {
                    bf16x8 b3;
#pragma unroll
                    for (int i = 0; i < 8; ++i) b3[i] = (__bf16)gelu_erf(acc2[hb][tb2][jj * 8 + i]);
                    acc3[tb2] = mfma32(a3, b3, acc3[tb2]);
                }
            }
        }
        __syncthreads();                 // every wave is done reading h1s
        // valid rows of acc3: regs 0..7 -> feature (r/4)*8 + g*4 + r%4, token tb2*32 + l32
#pragma unroll
        for (int tb2 = 0; tb2 < 2; ++tb2) {
            float* dst = red + ((size_t)w * kTok + tb2 * 32 + l32) * kFeat;
            *reinterpret_cast<float4*>(dst + g * 4) =
                make_float4(acc3[tb2][0], acc3[tb2][1], acc3[tb2][2], acc3[tb2][3]);
            *reinterpret_cast<float4*>(dst + 8 + g * 4) =
                make_float4(acc3[tb2][4], acc3[tb2][5], acc3[tb2][6], acc3[tb2][7]);
        }
        __syncthreads();

        // ---- 4. fixed-order sum over waves, unpatchify, store the fresh output
        float* out = d.Eh + (size_t)t * d.D;
        for (int e = tid; e < kTok * kFeat; e += NT) {
            const TokPos p = tok_pos(e, tb, d.Himg, d.Wimg);
            float sum = 0.f;
#pragma unroll
            for (int ww = 0; ww < NW; ++ww) sum += red[((size_t)ww * kTok + p.tl) * kFeat + p.f];
            out[p.idx] = sum;
        }
        __syncthreads();                 // LDS is reused by the next item
    }
}

int mlp_supported(int hidden) { return hidden == 512 || hidden == 1024; }

int mlp_grid_size(int device_cus) { return device_cus > 0 ? device_cus : 256; }

hipError_t launch_eps_mlp(const Dev& d, hipStream_t st) {
    switch (d.hidden) {
        case 512:
            hipLaunchKernelGGL(k_eps_mlp<512>, dim3(d.mlp_grid), dim3(256), 0, st, d);
            break;
        case 1024:
            hipLaunchKernelGGL(k_eps_mlp<1024>, dim3(d.mlp_grid), dim3(512), 0, st, d);
            break;
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace pa
