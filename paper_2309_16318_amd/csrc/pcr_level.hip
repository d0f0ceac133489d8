// One level of Parallel Cyclic Reduction for block-bidiagonal systems
// (Sec. 3, Alg. 1; Eqs. 4-6), with the sub-diagonal operators taken as +J
// (Eq. 4), so a level with stride s reads the previous level's values and does
//   r_l <- r_l + A_l r_{l-s}   for rows l >= s
//   A_l <- A_l A_{l-s}         for rows l >= 2s
// Rows s <= l < 2s need no operator update: their new operator would multiply
// a row index below zero, whose unknown is identically zero.
//
// Three implementations, chosen by width:
//   w = 16, 32   one wave walks a chain of rows l, l+s, l+2s, ... of one
//                residue class: each operator block is read from HBM once per
//                level, the block product runs on fp32 MFMA
//                (16x16x4 / 32x32x2) and the previous block is kept, transposed
//                through LDS, as the next row's right operand.
//   w = 64, 128  the same chain walk with a 4-wave workgroup per chain
//                segment: the current and previous blocks are staged in LDS
//                (double buffered), each wave owns 32x32 output tiles, and the
//                next block is prefetched into registers during the MFMAs.
//   other w      generic path: one workgroup per (system, row), float32 FMA on
//                the vector ALUs, operands staged through LDS in k-chunks.
// Block products are formed as C^T = P^T A^T so that the MFMA output of each
// lane is a contiguous run of a row of C (float4 stores) and the current block
// is consumed in the layout it is loaded in.
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

// ------------------------------------------------------------------------
// Chain-walking kernels.  A level with stride s partitions the rows l >= s
// into s chains (residue classes c = l mod s): c + s, c + 2s, ..., c + s*count_c
// with count_c = (L-1-c)/s.  Each chain is cut into segments of at most n rows
// and one segment is one work item; the segment with index j = 0 also copies
// row c (< s, already final).  Row c + s*m updates its operator iff m >= 2.
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));

struct Seg {
    int b, c, j, count, m0, m1;
};

__device__ inline Seg decode_segment(long long item, const LevelPlan& p, int L) {
    Seg g;
    const long long per_b = (long long)p.s * p.segs_per_class;
    g.b = (int)(item / per_b);
    const long long rem = item - (long long)g.b * per_b;
    g.c = (int)(rem / p.segs_per_class);
    g.j = (int)(rem - (long long)g.c * p.segs_per_class);
    g.count = (L - 1 - g.c) / p.s;
    g.m0 = 1 + g.j * p.n;
    g.m1 = min(g.count, g.m0 + p.n - 1);
    return g;
}

__device__ inline void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ---- one wave per segment, w = 16 or 32 -----------------------------------
// Lane layout "R": lane (i = lane % W, g = lane / W) holds row i of a block at
// the NV columns col(v) = 4*NG*(v/4) + 4*g + v%4 (NG = 64 / W lane groups).
// Layout "T" holds the same positions of the transposed block.  With MFMA v
// consuming k = col(v) on every lane, X = P^T (T layout of P) and Y = A^T
// (R layout of A) give D = (A P)^T, whose lane values are again layout R.
template <int W>
struct WaveShape {
    static constexpr int NG = 64 / W;
    static constexpr int NV = W * W / 64;
    static constexpr int PITCH = W + 4;
    __device__ static int col(int v, int g) { return 4 * NG * (v / 4) + 4 * g + (v % 4); }
};

template <int W>
__device__ inline void load_R(const float* blk, int trans, int i, int g, float* out) {
    using S = WaveShape<W>;
    if (!trans) {
#pragma unroll
        for (int q = 0; q < S::NV / 4; ++q) {
            const v4f x = *reinterpret_cast<const v4f*>(blk + i * W + S::col(4 * q, g));
            out[4 * q + 0] = x[0];
            out[4 * q + 1] = x[1];
            out[4 * q + 2] = x[2];
            out[4 * q + 3] = x[3];
        }
    } else {
#pragma unroll
        for (int v = 0; v < S::NV; ++v) out[v] = blk[S::col(v, g) * W + i];
    }
}

template <int W>
__device__ inline void lds_transpose(float* lds, const float* aR, int i, int g, float* pT) {
    using S = WaveShape<W>;
    wave_sync();
#pragma unroll
    for (int q = 0; q < S::NV / 4; ++q) {
        v4f x = {aR[4 * q], aR[4 * q + 1], aR[4 * q + 2], aR[4 * q + 3]};
        *reinterpret_cast<v4f*>(lds + i * S::PITCH + S::col(4 * q, g)) = x;
    }
    wave_sync();
#pragma unroll
    for (int v = 0; v < S::NV; ++v) pT[v] = lds[S::col(v, g) * S::PITCH + i];
}

template <int W>
__global__ __launch_bounds__(256) void pcr_level_wave(
    BlockSrc Ain, VecSrc rin, float* __restrict__ Aout, VecDst rout, int L, LevelPlan plan) {
    using S = WaveShape<W>;
    __shared__ float lds_all[4][W * S::PITCH];
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const long long item = (long long)blockIdx.x * 4 + wv;
    if (item >= plan.total) return;
    const Seg sg = decode_segment(item, plan, L);
    const int s = plan.s;
    const float* rb = rin.base + sg.b * rin.bstride;
    float* ob = rout.base + sg.b * rout.bstride;
    if (sg.j == 0 && lane < W) ob[sg.c * rout.rstride + lane] = rb[sg.c * rin.rstride + lane];
    if (sg.m0 > sg.count) return;

    float* lds = lds_all[wv];
    const int i = lane % W;
    const int g = lane / W;
    const float* ab = Ain.base + sg.b * Ain.bstride;
    float* Ob = Aout + (long long)sg.b * L * W * W;

    float aR[S::NV], pT[S::NV], rp[S::NV];
    int l = sg.c + s * sg.m0;
    {
        const int lp = l - s;
        const float* rrow = rb + (long long)lp * rin.rstride;
#pragma unroll
        for (int v = 0; v < S::NV; ++v) rp[v] = rrow[S::col(v, g)];
        if (sg.m0 >= 2) {
            load_R<W>(ab + (long long)lp * Ain.rstride, Ain.trans, i, g, aR);
            lds_transpose<W>(lds, aR, i, g, pT);
        }
    }
    for (int m = sg.m0; m <= sg.m1; ++m, l += s) {
        load_R<W>(ab + (long long)l * Ain.rstride, Ain.trans, i, g, aR);
        const float* rrow = rb + (long long)l * rin.rstride;
        const float ri = rrow[i];
        float rn[S::NV];
#pragma unroll
        for (int v = 0; v < S::NV; ++v) rn[v] = rrow[S::col(v, g)];
        // r_l + A_l r_{l-s}
        float part = 0.f;
#pragma unroll
        for (int v = 0; v < S::NV; ++v) part = fmaf(aR[v], rp[v], part);
#pragma unroll
        for (int off = W; off < 64; off <<= 1) part += __shfl_xor(part, off, 64);
        if (g == 0) ob[(long long)l * rout.rstride + i] = ri + part;
        // A_l A_{l-s}
        if (m >= 2) {
            float* cb = Ob + (long long)l * W * W + i * W;
            if constexpr (W == 16) {
                v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(pT[v], aR[v], acc, 0, 0, 0);
                *reinterpret_cast<v4f*>(cb + S::col(0, g)) = acc;
            } else {
                v16f acc = {};
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(pT[v], aR[v], acc, 0, 0, 0);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    v4f x = {acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]};
                    *reinterpret_cast<v4f*>(cb + S::col(4 * q, g)) = x;
                }
            }
        }
        if (m < sg.m1) lds_transpose<W>(lds, aR, i, g, pT);
#pragma unroll
        for (int v = 0; v < S::NV; ++v) rp[v] = rn[v];
    }
}

// ---- 4-wave workgroup per segment, w = 64 or 128 --------------------------
template <int W>
struct TileShape {
    static constexpr int PITCH = W + 4;
    static constexpr int NL = W * W / 4 / 256;    // float4 loads per thread per block
    static constexpr int TW = W / 64;             // 32x32 tiles per wave along each axis... (1 or 2)
    static constexpr int RPT = 256 / W;           // threads per row in the mat-vec (4 or 2)
    static constexpr int KPT = W / RPT;           // columns per thread in the mat-vec
};

template <int W>
__device__ inline void load_block_regs(const float* blk, v4f* pre) {
    using S = TileShape<W>;
#pragma unroll
    for (int p = 0; p < S::NL; ++p)
        pre[p] = *reinterpret_cast<const v4f*>(blk + 4 * (threadIdx.x + 256 * p));
}

template <int W>
__device__ inline void regs_to_lds(const v4f* pre, float* buf, int trans) {
    using S = TileShape<W>;
#pragma unroll
    for (int p = 0; p < S::NL; ++p) {
        const int f = 4 * (threadIdx.x + 256 * p);
        const int row = f / W, col = f % W;
        if (!trans) {
            *reinterpret_cast<v4f*>(buf + row * S::PITCH + col) = pre[p];
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) buf[(col + e) * S::PITCH + row] = pre[p][e];
        }
    }
}

template <int W>
__global__ __launch_bounds__(256) void pcr_level_tile(
    BlockSrc Ain, VecSrc rin, float* __restrict__ Aout, VecDst rout, int L, LevelPlan plan) {
    using S = TileShape<W>;
    __shared__ float bufs[2][W * S::PITCH];
    __shared__ float rpv[2][W];
    const int t = threadIdx.x;
    const long long item = blockIdx.x;
    const Seg sg = decode_segment(item, plan, L);
    const int s = plan.s;
    const float* rb = rin.base + sg.b * rin.bstride;
    float* ob = rout.base + sg.b * rout.bstride;
    if (sg.j == 0 && t < W) ob[sg.c * rout.rstride + t] = rb[sg.c * rin.rstride + t];
    if (sg.m0 > sg.count) return;  // uniform over the workgroup

    const float* ab = Ain.base + sg.b * Ain.bstride;
    float* Ob = Aout + (long long)sg.b * L * W * W;
    const int lane = t & 63, wv = t >> 6;
    const int i = lane & 31, h = lane >> 5;
    // output tiles of this wave: rows (TW*(wv>>1) + a)*32, cols (TW*(wv&1) + bb)*32
    const int tr0 = S::TW * (wv >> 1), tc0 = S::TW * (wv & 1);

    v4f pre[S::NL];
    float rl_pre = 0.f;
    int l = sg.c + s * sg.m0;
    {
        const int lp = l - s;
        if (t < W) rpv[1][t] = rb[(long long)lp * rin.rstride + t];
        if (sg.m0 >= 2) {
            load_block_regs<W>(ab + (long long)lp * Ain.rstride, pre);
            regs_to_lds<W>(pre, bufs[1], Ain.trans);
        }
    }
    load_block_regs<W>(ab + (long long)l * Ain.rstride, pre);
    if (t < W) rl_pre = rb[(long long)l * rin.rstride + t];

    for (int m = sg.m0, u = 0; m <= sg.m1; ++m, ++u, l += s) {
        float* cur = bufs[u & 1];
        const float* prv = bufs[(u + 1) & 1];
        const float* rprev = rpv[(u + 1) & 1];
        regs_to_lds<W>(pre, cur, Ain.trans);
        if (t < W) rpv[u & 1][t] = rl_pre;
        __syncthreads();
        if (m < sg.m1) {
            load_block_regs<W>(ab + (long long)(l + s) * Ain.rstride, pre);
            if (t < W) rl_pre = rb[(long long)(l + s) * rin.rstride + t];
        }
        // r_l + A_l r_{l-s}: RPT threads per row, KPT columns each.
        {
            const int row = t / S::RPT, k0 = (t % S::RPT) * S::KPT;
            float part = 0.f;
#pragma unroll
            for (int k = 0; k < S::KPT; k += 4) {
                const v4f a = *reinterpret_cast<const v4f*>(cur + row * S::PITCH + k0 + k);
                part = fmaf(a[0], rprev[k0 + k], part);
                part = fmaf(a[1], rprev[k0 + k + 1], part);
                part = fmaf(a[2], rprev[k0 + k + 2], part);
                part = fmaf(a[3], rprev[k0 + k + 3], part);
            }
#pragma unroll
            for (int off = 1; off < S::RPT; off <<= 1) part += __shfl_xor(part, off, 64);
            if (t % S::RPT == 0) ob[(long long)l * rout.rstride + row] = rpv[u & 1][row] + part;
        }
        // A_l A_{l-s} on MFMA: D = (A P)^T tiles.
        if (m >= 2) {
            v16f acc[S::TW][S::TW];
#pragma unroll
            for (int a = 0; a < S::TW; ++a)
#pragma unroll
                for (int bb = 0; bb < S::TW; ++bb) acc[a][bb] = v16f{};
#pragma unroll 2
            for (int q = 0; q < W / 8; ++q) {
                const int k = 8 * q + 4 * h;
                v4f av[S::TW];
                float pv[S::TW][4];
#pragma unroll
                for (int a = 0; a < S::TW; ++a)
                    av[a] = *reinterpret_cast<const v4f*>(cur + ((tr0 + a) * 32 + i) * S::PITCH + k);
#pragma unroll
                for (int bb = 0; bb < S::TW; ++bb)
#pragma unroll
                    for (int e = 0; e < 4; ++e) pv[bb][e] = prv[(k + e) * S::PITCH + (tc0 + bb) * 32 + i];
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int a = 0; a < S::TW; ++a)
#pragma unroll
                        for (int bb = 0; bb < S::TW; ++bb)
                            acc[a][bb] = __builtin_amdgcn_mfma_f32_32x32x2f32(pv[bb][e], av[a][e],
                                                                              acc[a][bb], 0, 0, 0);
            }
            float* cb = Ob + (long long)l * W * W;
#pragma unroll
            for (int a = 0; a < S::TW; ++a)
#pragma unroll
                for (int bb = 0; bb < S::TW; ++bb)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const v16f& x = acc[a][bb];
                        v4f y = {x[4 * q], x[4 * q + 1], x[4 * q + 2], x[4 * q + 3]};
                        *reinterpret_cast<v4f*>(cb + ((tr0 + a) * 32 + i) * W + (tc0 + bb) * 32 +
                                                8 * q + 4 * h) = y;
                    }
        }
        __syncthreads();
    }
}

}  // namespace

LevelPlan plan_level(int B, int L, int s, long long target_items, int n_max) {
    LevelPlan p;
    p.s = s;
    const int Q = (L - 1) / s;
    const long long rows = (long long)B * s * Q;
    long long n = (rows + target_items - 1) / target_items;
    if (n < 1) n = 1;
    if (n > n_max) n = n_max;
    p.n = (int)n;
    p.segs_per_class = (Q + p.n - 1) / p.n;
    if (p.segs_per_class < 1) p.segs_per_class = 1;
    p.total = (long long)B * s * p.segs_per_class;
    return p;
}

hipError_t launch_pcr_level(const BlockSrc& Ain, const VecSrc& rin, float* Aout,
                            const VecDst& rout, int B, int L, int w, int s,
                            hipStream_t stream) {
    if (w == 16 || w == 32) {
        const LevelPlan p = plan_level(B, L, s, 8192, 64);
        const unsigned grid = (unsigned)((p.total + 3) / 4);
        if (w == 16)
            hipLaunchKernelGGL(pcr_level_wave<16>, dim3(grid), dim3(256), 0, stream, Ain, rin,
                               Aout, rout, L, p);
        else
            hipLaunchKernelGGL(pcr_level_wave<32>, dim3(grid), dim3(256), 0, stream, Ain, rin,
                               Aout, rout, L, p);
        return hipGetLastError();
    }
    if (w == 64 || w == 128) {
        const LevelPlan p = plan_level(B, L, s, w == 64 ? 4096 : 1024, 64);
        if (w == 64)
            hipLaunchKernelGGL(pcr_level_tile<64>, dim3((unsigned)p.total), dim3(256), 0, stream,
                               Ain, rin, Aout, rout, L, p);
        else
            hipLaunchKernelGGL(pcr_level_tile<128>, dim3((unsigned)p.total), dim3(256), 0, stream,
                               Ain, rin, Aout, rout, L, p);
        return hipGetLastError();
    }
    const long long rows = (long long)B * L;
    hipLaunchKernelGGL(pcr_level_generic, dim3((unsigned)rows), dim3(kThreads), 0, stream,
                       Ain, rin, Aout, rout, L, w, s);
    return hipGetLastError();
}

}  // namespace deeppcr
