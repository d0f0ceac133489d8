// One level of Parallel Cyclic Reduction for block-bidiagonal systems
// (Sec. 3, Alg. 1; Eqs. 4-6), with the sub-diagonal operators taken as +J
// (Eq. 4), so a level with stride s reads the previous level's values and does
//   r_l <- r_l + A_l r_{l-s}   for rows l >= s
//   A_l <- A_l A_{l-s}         for rows l >= 2s
// Rows s <= l < 2s need no operator update: their new operator would multiply
// a row index below zero, whose unknown is identically zero.
//
// Generic path: any width 1 <= w <= 128, one workgroup per (system, row),
// float32 FMA on the vector ALUs, operands staged through LDS in k-chunks.
#include "internal.h"

namespace deeppcr {
namespace {

constexpr int kThreads = 256;
constexpr int kKC = 16;                                   // k-chunk of the block product
constexpr int kAccPerThread = kMaxWidth * kMaxWidth / kThreads;  // 64

__device__ inline float block_elem(const float* blk, int i, int k, int w, int trans) {
    return trans ? blk[(long long)k * w + i] : blk[(long long)i * w + k];
}

__device__ inline float wave_sum(float v) {
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__global__ __launch_bounds__(kThreads) void pcr_level_generic(
    BlockSrc Ain, VecSrc rin, float* __restrict__ Aout, VecDst rout, int L, int w, int s) {
    const long long row = blockIdx.x;
    const int l = (int)(row % L);
    const int b = (int)(row / L);
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = t >> 6;

    const float* rl = rin.base + b * rin.bstride + (long long)l * rin.rstride;
    float* xo = rout.base + b * rout.bstride + (long long)l * rout.rstride;
    if (l < s) {
        for (int i = t; i < w; i += kThreads) xo[i] = rl[i];
        return;
    }

    __shared__ float rprev[kMaxWidth];
    __shared__ float Atile[kMaxWidth][kKC + 1];
    __shared__ float Ptile[kKC][kMaxWidth];

    const float* rp = rin.base + b * rin.bstride + (long long)(l - s) * rin.rstride;
    for (int i = t; i < w; i += kThreads) rprev[i] = rp[i];
    __syncthreads();

    const float* Al = Ain.base + b * Ain.bstride + (long long)l * Ain.rstride;

    // r_l + A_l r_{l-s}: one wave per output row, lanes stride over columns.
    for (int i = wave; i < w; i += kThreads / 64) {
        float acc = 0.f;
        for (int j = lane; j < w; j += 64) acc = fmaf(block_elem(Al, i, j, w, Ain.trans), rprev[j], acc);
        acc = wave_sum(acc);
        if (lane == 0) xo[i] = rl[i] + acc;
    }

    if (l < 2 * s) return;

    // A_l A_{l-s}
    const float* Pl = Ain.base + b * Ain.bstride + (long long)(l - s) * Ain.rstride;
    const int nout = w * w;
    float acc[kAccPerThread];
#pragma unroll
    for (int q = 0; q < kAccPerThread; ++q) acc[q] = 0.f;

    for (int kc = 0; kc < w; kc += kKC) {
        const int kw = min(kKC, w - kc);
        for (int idx = t; idx < w * kw; idx += kThreads) {
            const int i = idx / kw, kk = idx - (idx / kw) * kw;
            Atile[i][kk] = block_elem(Al, i, kc + kk, w, Ain.trans);
        }
        for (int idx = t; idx < kw * w; idx += kThreads) {
            const int kk = idx / w, j = idx - (idx / w) * w;
            Ptile[kk][j] = block_elem(Pl, kc + kk, j, w, Ain.trans);
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < kAccPerThread; ++q) {
            const int idx = t + q * kThreads;
            if (idx < nout) {
                const int i = idx / w, j = idx - (idx / w) * w;
                float a = acc[q];
                for (int kk = 0; kk < kw; ++kk) a = fmaf(Atile[i][kk], Ptile[kk][j], a);
                acc[q] = a;
            }
        }
        __syncthreads();
    }
    float* Ao = Aout + ((long long)b * L + l) * nout;
#pragma unroll
    for (int q = 0; q < kAccPerThread; ++q) {
        const int idx = t + q * kThreads;
        if (idx < nout) Ao[idx] = acc[q];
    }
}

}  // namespace

hipError_t launch_pcr_level(const BlockSrc& Ain, const VecSrc& rin, float* Aout,
                            const VecDst& rout, int B, int L, int w, int s,
                            hipStream_t stream) {
    const long long rows = (long long)B * L;
    hipLaunchKernelGGL(pcr_level_generic, dim3((unsigned)rows), dim3(kThreads), 0, stream,
                       Ain, rin, Aout, rout, L, w, s);
    return hipGetLastError();
}

}  // namespace deeppcr
