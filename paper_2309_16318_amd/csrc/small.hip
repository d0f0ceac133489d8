// Small widths (w <= 8): one PCR level (Sec. 3, Alg. 1) with w x w blocks
// handled by groups of WP*WP lanes (WP = w rounded up to a power of two), so a
// wave reduces 64 / WP^2 rows at once; lane (i, j) of a group owns element
// (i, j) of its row's block.  Block products and mat-vecs use lane shuffles
// inside the group.  Rows are independent within a level, so no chain walk is
// needed: A_{l-s} is read again for row l (blocks are at most 256 bytes).
// Also the layer / Jacobian evaluation for small widths with one thread per
// state element.
#include "internal.h"

namespace deeppcr {
namespace {

constexpr int kThreads = 256;

template <int WP>
__global__ __launch_bounds__(kThreads) void pcr_level_small(BlockSrc Ain, VecSrc rin,
                                                            float* __restrict__ Aout, VecDst rout,
                                                            int B, int L, int w, int s) {
    constexpr int GL = WP * WP;         // lanes per row group
    constexpr int GPW = 64 / GL;        // row groups per wave
    const int lane = threadIdx.x & 63;
    const int grp = lane / GL, gl = lane % GL;
    const int i = gl / WP, j = gl % WP;
    const int base = lane - gl;
    const bool valid = i < w && j < w;
    const long long wave = ((long long)blockIdx.x * kThreads + threadIdx.x) / 64;
    const long long row = wave * GPW + grp;  // b * L + l
    const long long nrows = (long long)B * L;
    // whole groups beyond the last row still take part in the shuffles
    const bool live = row < nrows;
    const int l = live ? (int)(row % L) : 0;
    const int b = live ? (int)(row / L) : 0;
    const float* rl = rin.base + b * rin.bstride + (long long)l * rin.rstride;
    float* xo = rout.base + b * rout.bstride + (long long)l * rout.rstride;
    const bool reduce = live && l >= s;
    const bool prod = live && l >= 2 * s;

    float a = 0.f, p = 0.f, rp = 0.f;
    if (reduce && valid) {
        const float* Al = Ain.base + b * Ain.bstride + (long long)l * Ain.rstride;
        a = Ain.trans ? Al[j * w + i] : Al[i * w + j];
        rp = rin.base[b * rin.bstride + (long long)(l - s) * rin.rstride + j];
    }
    if (prod && valid) {
        const float* Pl = Ain.base + b * Ain.bstride + (long long)(l - s) * Ain.rstride;
        p = Ain.trans ? Pl[j * w + i] : Pl[i * w + j];
    }
    // r_l + A_l r_{l-s}: row i of the group sums a * rp over j
    float y = a * rp;
#pragma unroll
    for (int off = 1; off < WP; off <<= 1) y += __shfl_xor(y, off, 64);
    if (live && j == 0 && i < w) xo[i] = rl[i] + (reduce ? y : 0.f);
    // A_l A_{l-s}: element (i, j) = sum_k A[i][k] P[k][j]
    float c = 0.f;
#pragma unroll
    for (int k = 0; k < WP; ++k) {
        const float ak = __shfl(a, base + i * WP + k, 64);
        const float pk = __shfl(p, base + k * WP + j, 64);
        c = fmaf(ak, pk, c);
    }
    if (prod && valid) Aout[((long long)b * L + l) * w * w + i * w + j] = c;
}

// One thread per state element (b, l, i): the layer at Z_{l-1}, the residual
// (forward) or the scaled derivative and reversed right-hand side
// (backward), and row i of J_l (forward: at row l; backward: J_l itself at
// reversed row L - l, read transposed by the first level).
template <bool BWD>
__global__ __launch_bounds__(kThreads) void eval_small(
    const float* __restrict__ W, const float* __restrict__ bias, const float* __restrict__ z0,
    const float* __restrict__ Z, const float* __restrict__ G, float* __restrict__ A,
    float* __restrict__ r, float* __restrict__ dscale, unsigned* __restrict__ red, int B, int L,
    int w, int layer, float alpha) {
    const long long idx = (long long)blockIdx.x * kThreads + threadIdx.x;
    if (!BWD && blockIdx.x == 0)
        for (int k = threadIdx.x; k < 2 * kRedShards; k += kThreads) red[k] = 0u;
    unsigned mr = 0u;  // forward: max |r| bits
    if (idx < (long long)B * L * w) {
        const int i = (int)(idx % w);
        const long long row = idx / w;
        const int l = (int)(row % L);
        const int b = (int)(row / L);
        const float* zp = (l == 0) ? z0 + (long long)b * w : Z + (row - 1) * w;
        const float* Wr = W + ((long long)l * w + i) * w;
        float acc = 0.f;
        for (int k = 0; k < w; ++k) acc = fmaf(Wr[k], zp[k], acc);
        float d;
        const float y = activate(layer, acc + bias[(long long)l * w + i], &d);
        const bool res = layer_residual(layer);
        const float dsc = res ? alpha * d : d;
        if (!BWD) {
            const float rv = (res ? fmaf(alpha, y, zp[i]) : y) - Z[idx];
            r[idx] = rv;
            mr = __float_as_uint(fabsf(rv));
        } else {
            dscale[idx] = dsc;
            const int mr_row = L - 1 - l;
            r[((long long)b * L + mr_row) * w + i] = (mr_row == 0) ? G[(long long)b * w + i] : 0.f;
        }
        if (l >= 1) {
            float* Ar = A + ((long long)b * L + (BWD ? L - l : l)) * w * w + (long long)i * w;
            for (int k = 0; k < w; ++k) Ar[k] = dsc * Wr[k] + ((res && k == i) ? 1.f : 0.f);
        }
    }
    if (!BWD) {
        for (int off = 32; off > 0; off >>= 1) mr = max(mr, (unsigned)__shfl_xor((int)mr, off, 64));
        if ((threadIdx.x & 63) == 0) atomicMax(red + kRedF + (int)(blockIdx.x % kRedShards), mr);
    }
}

}  // namespace

bool small_width(int w) { return w <= 8; }

hipError_t launch_pcr_level_small(const BlockSrc& Ain, const VecSrc& rin, float* Aout,
                                  const VecDst& rout, int B, int L, int w, int s,
                                  hipStream_t stream) {
    const long long rows = (long long)B * L;
    const int wp = w <= 1 ? 1 : w <= 2 ? 2 : w <= 4 ? 4 : 8;
    const long long rows_per_wg = (kThreads / 64) * (64 / (wp * wp));
    const dim3 grid((unsigned)((rows + rows_per_wg - 1) / rows_per_wg)), block(kThreads);
    switch (wp) {
        case 1: hipLaunchKernelGGL(pcr_level_small<1>, grid, block, 0, stream, Ain, rin, Aout, rout, B, L, w, s); break;
        case 2: hipLaunchKernelGGL(pcr_level_small<2>, grid, block, 0, stream, Ain, rin, Aout, rout, B, L, w, s); break;
        case 4: hipLaunchKernelGGL(pcr_level_small<4>, grid, block, 0, stream, Ain, rin, Aout, rout, B, L, w, s); break;
        default: hipLaunchKernelGGL(pcr_level_small<8>, grid, block, 0, stream, Ain, rin, Aout, rout, B, L, w, s); break;
    }
    return hipGetLastError();
}

hipError_t launch_eval_small(bool bwd, const float* W, const float* bias, const float* z0,
                             const float* Z, const float* G, float* A, float* r, float* dscale,
                             unsigned* red, int B, int L, int w, int layer, float alpha,
                             hipStream_t stream) {
    const long long n = (long long)B * L * w;
    const dim3 grid((unsigned)((n + kThreads - 1) / kThreads)), block(kThreads);
    if (bwd)
        hipLaunchKernelGGL(eval_small<true>, grid, block, 0, stream, W, bias, z0, Z, G, A, r,
                           dscale, red, B, L, w, layer, alpha);
    else
        hipLaunchKernelGGL(eval_small<false>, grid, block, 0, stream, W, bias, z0, Z, G, A, r,
                           dscale, red, B, L, w, layer, alpha);
    return hipGetLastError();
}

}  // namespace deeppcr
