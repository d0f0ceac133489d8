// One level of Parallel Cyclic Reduction for block-bidiagonal systems
// (Sec. 3, Alg. 1; Eqs. 4-6), with the sub-diagonal operators taken as +J
// (Eq. 4), so a level with stride s reads the previous level's values and does
//   r_l <- r_l + A_l r_{l-s}   for rows l >= s
//   A_l <- A_l A_{l-s}         for rows l >= 2s
// Rows s <= l < 2s need no operator update: their new operator would multiply
// a row index below zero, whose unknown is identically zero.
//
// Implementations, chosen by width:
//   w = 16, 32   one wave walks a chain of rows l, l+s, l+2s, ... of one
//                residue class: each operator block is read from HBM once per
//                level, the block product runs on fp32 MFMA
//                (16x16x4 / 32x32x2) and the previous block is kept, transposed
//                through LDS, as the next row's right operand; two levels per
//                pass where the chains allow.
//   w = 64, 128  the same chain walk with one workgroup per chain segment,
//                one wave per 32-row strip of the blocks (left MFMA operand in
//                registers, right operands in LDS), two levels per pass; the
//                strip kernels also serve w = 32 for the first two levels of
//                a Newton iteration or backward solve.
//   last levels  at w = 32, 64, 128 the last 3-6 levels are not run here:
//                the chains they act on are solved by substitution
//                (chain.hip; tail_levels below says how many).
//   w <= 8       lane groups of a wave per row (small.hip).
//   other w      generic path: one workgroup per (system, row), float32 FMA on
//                the vector ALUs, operands staged through LDS in k-chunks.
// Block products are formed as C^T = P^T A^T so that the MFMA output of each
// lane is a contiguous run of a row of C (float4 stores) and the current block
// is consumed in the layout it is loaded in.
#include "internal.h"
#include "strip.h"


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

template <int W, bool TRANS>
__device__ inline void load_R(const float* blk, int i, int g, float* out) {
    using S = WaveShape<W>;
    if constexpr (!TRANS) {
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

// Per-wave LDS: the transpose buffer, a two-row ring of right-hand-side rows
// (the current row's r and the previous row's r, both of the previous level),
// and, for the fused first level, a two-row ring of iterate rows Z.
template <int W>
struct WaveLds {
    float tr[W * WaveShape<W>::PITCH];
    float r[2][W];
    float z[2][W];
};

enum { SRC_MEM = 0, SRC_LAYER = 1 };

// Layer l evaluated at zprev (a row in LDS) for lane (i, g):
//   a_i = W_l[i, :] zprev + b_i, y = sigma(a_i), d = sigma'(a_i),
//   J_l row i = c d_i W_l[i, :] (+ e_i for the residual layer), c = 1 or alpha,
//   r_i = f_i - zcur_i with f_i = y (plain) or zprev_i + alpha y (residual).
// w_in holds W_l[i, col(v)] (layer R) and is turned into J_l[i, col(v)].
template <int W>
__device__ inline float eval_layer_row(const NewtonArgs& na, int l, const float* zprev,
                                       float zcur_i, int i, int g, float* w_in) {
    using S = WaveShape<W>;
    float part = 0.f;
#pragma unroll
    for (int q = 0; q < S::NV / 4; ++q) {
        const v4f z4 = *reinterpret_cast<const v4f*>(zprev + S::col(4 * q, g));
#pragma unroll
        for (int e = 0; e < 4; ++e) part = fmaf(w_in[4 * q + e], z4[e], part);
    }
    part = group_sum<W>(part);
    const float a = part + na.bias[(long long)l * W + i];
    float d;
    const float y = activate(na.layer, a, &d);
    const bool resid = layer_residual(na.layer);
    const float dsc = resid ? na.alpha * d : d;
    const float f = resid ? fmaf(na.alpha, y, zprev[i]) : y;
#pragma unroll
    for (int v = 0; v < S::NV; ++v) {
        float j = dsc * w_in[v];
        if (resid && S::col(v, g) == i) j += 1.f;
        w_in[v] = j;
    }
    return f - zcur_i;
}

template <int W>
__device__ inline void wave_umax2(unsigned& a, unsigned& b) {
    for (int off = 32; off > 0; off >>= 1) {
        a = max(a, (unsigned)__shfl_xor((int)a, off, 64));
        b = max(b, (unsigned)__shfl_xor((int)b, off, 64));
    }
}

// The chain walk of one wave.  SRC_MEM reads the previous level's blocks and
// vectors (Ain, rin); SRC_LAYER (first level, s = 1) evaluates them from the
// layers at the iterate.  UPD (last level) adds the solution rows to the
// iterate and reduces max|dZ|, max|Z| instead of storing them.
template <int W, bool TRANS, int SRC, bool UPD>
__global__ __launch_bounds__(256) void pcr_level_wave(
    BlockSrc Ain, VecSrc rin, float* __restrict__ Aout, VecDst rout, int L, LevelPlan plan,
    NewtonArgs na) {
    using S = WaveShape<W>;
    __shared__ WaveLds<W> lds_all[4];
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const long long item = (long long)blockIdx.x * 4 + wv;
    if (SRC == SRC_LAYER && blockIdx.x == 0)
        for (int k = threadIdx.x; k < 2 * kRedShards; k += 256) na.red[k] = 0u;
    if (item >= plan.total) return;
    const Seg sg = decode_segment(item, plan, L);
    const int s = plan.s;
    WaveLds<W>& lds = lds_all[wv];
    const int i = lane % W;
    const int g = lane / W;
    const float* rb = rin.base + sg.b * rin.bstride;
    float* ob = rout.base + sg.b * rout.bstride;
    const float* zb = na.Z + (long long)sg.b * L * W;      // SRC_LAYER / UPD
    float* zw = na.Z + (long long)sg.b * L * W;
    const float* z0b = na.z0 + (long long)sg.b * W;
    unsigned mx = 0u, mz = 0u;  // UPD reductions
    unsigned mr = 0u;           // SRC_LAYER: max |r| of the evaluated rows

    // Writes solution / next-level row l (lanes with g == 0 hold element i).
    auto emit = [&](int l, float x) {
        if (g != 0) return;
        if constexpr (UPD) {
            const long long o = (long long)l * W + i;
            const float z = zw[o] + x;
            zw[o] = z;
            mx = max(mx, __float_as_uint(fabsf(x)));
            mz = max(mz, __float_as_uint(fabsf(z)));
        } else {
            ob[(long long)l * rout.rstride + i] = x;
        }
    };
    // row c (< s) is final: copied, or for the fused first level evaluated.
    if (sg.j == 0) {
        if constexpr (SRC == SRC_LAYER) {
            // r_0 = f_0(z0) - Z_0
            if (lane < W) lds.z[0][lane] = z0b[lane];
            wave_sync();
            float w_in[S::NV];
            load_R<W, false>(na.W, i, g, w_in);
            const float r0 = eval_layer_row<W>(na, 0, lds.z[0], zb[i], i, g, w_in);
            mr = __float_as_uint(fabsf(r0));
            emit(0, r0);
        } else {
            emit(sg.c, rb[sg.c * rin.rstride + i]);
        }
    }
    // With DEEP the next block (row l+s) is already in registers (aF) when
    // row l starts and the block of row l+2s is requested: two blocks in
    // flight per wave.
    constexpr bool DEEP = (W == 32) && (SRC == SRC_MEM);
    float aR[S::NV], pT[S::NV], aF[DEEP ? S::NV : 1];
    if (sg.m0 <= sg.count) {
        int l = sg.c + s * sg.m0;
        if constexpr (SRC == SRC_LAYER) {
            // rows l-1 and l of the iterate, and r_{l-1} / J_{l-1} from row l-1's layer
            wave_sync();
            if (lane < W) {
                lds.z[0][lane] = zb[(long long)l * W + lane];              // Z_l
                lds.z[1][lane] = zb[(long long)(l - 1) * W + lane];        // Z_{l-1}
                lds.r[0][lane] = (l >= 2) ? zb[(long long)(l - 2) * W + lane] : z0b[lane];
            }
            wave_sync();
            // evaluate layer l-1 at Z_{l-2} (parked in lds.r[0] for the moment)
            float w_in[S::NV];
            load_R<W, false>(na.W + (long long)(l - 1) * W * W, i, g, w_in);
            const float rp = eval_layer_row<W>(na, l - 1, lds.r[0], lds.z[1][i], i, g, w_in);
            if (sg.m0 >= 2) lds_transpose<W>(lds.tr, w_in, i, g, pT);
            wave_sync();
            if (g == 0) lds.r[1][i] = rp;  // r_{l-1}
            wave_sync();
            load_R<W, false>(na.W + (long long)l * W * W, i, g, aR);
        } else {
            if (lane < W) {
                lds.r[1][lane] = rb[(long long)(l - s) * rin.rstride + lane];
                lds.r[0][lane] = rb[(long long)l * rin.rstride + lane];
            }
            if (sg.m0 >= 2) {
                load_R<W, TRANS>(Ain.base + sg.b * Ain.bstride + (long long)(l - s) * Ain.rstride, i, g, aR);
                lds_transpose<W>(lds.tr, aR, i, g, pT);
            }
            load_R<W, TRANS>(Ain.base + sg.b * Ain.bstride + (long long)l * Ain.rstride, i, g, aR);
            if (DEEP && sg.m0 < sg.m1)
                load_R<W, TRANS>(Ain.base + sg.b * Ain.bstride + (long long)(l + s) * Ain.rstride,
                                 i, g, aF);
            wave_sync();
        }
        const float* ab = Ain.base + sg.b * Ain.bstride;
        float* Ob = Aout + (long long)sg.b * L * W * W;
        for (int m = sg.m0, u = 0; m <= sg.m1; ++m, ++u, l += s) {
            const bool more = m < sg.m1;
            float* rcur = lds.r[u & 1];
            float* rprev = lds.r[(u + 1) & 1];
            float aN[S::NV];
            float rnext = 0.f;
            float ri;
            if constexpr (SRC == SRC_LAYER) {
                // this row's layer: A_l = J_l from W_l at Z_{l-1}, r_l
                const float* zcur = lds.z[u & 1];
                const float* zprv = lds.z[(u + 1) & 1];
                if (more) {
                    load_R<W, false>(na.W + (long long)(l + 1) * W * W, i, g, aN);
                    if (lane < W) rnext = zb[(long long)(l + 1) * W + lane];  // Z_{l+1}
                }
                ri = eval_layer_row<W>(na, l, zprv, zcur[i], i, g, aR);
                mr = max(mr, __float_as_uint(fabsf(ri)));
            } else {
                if constexpr (DEEP) {
                    if (m + 1 < sg.m1) load_R<W, TRANS>(ab + (long long)(l + 2 * s) * Ain.rstride, i, g, aN);
                } else {
                    if (more) load_R<W, TRANS>(ab + (long long)(l + s) * Ain.rstride, i, g, aN);
                }
                if (more && lane < W) rnext = rb[(long long)(l + s) * rin.rstride + lane];
                ri = rcur[i];
            }
            // r_l + A_l r_{l-s}
            float part = 0.f;
#pragma unroll
            for (int q = 0; q < S::NV / 4; ++q) {
                const v4f rp = *reinterpret_cast<const v4f*>(rprev + S::col(4 * q, g));
#pragma unroll
                for (int e = 0; e < 4; ++e) part = fmaf(aR[4 * q + e], rp[e], part);
            }
            part = group_sum<W>(part);
            emit(l, ri + part);
            // A_l A_{l-s}
            if (m >= 2) {
                if constexpr (W == 16) {
                    float* cb = Ob + (long long)l * W * W + i * W;
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
                    // Each lane holds 32-byte pieces of 16 rows; stage the block in LDS
                    // so the global stores are contiguous 1 KiB per instruction.
                    wave_sync();
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        v4f x = {acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]};
                        *reinterpret_cast<v4f*>(lds.tr + i * S::PITCH + S::col(4 * q, g)) = x;
                    }
                    wave_sync();
                    float* blk = Ob + (long long)l * W * W;
#pragma unroll
                    for (int p = 0; p < 4; ++p) {
                        const int e = 4 * (lane + 64 * p);
                        *reinterpret_cast<v4f*>(blk + e) =
                            *reinterpret_cast<const v4f*>(lds.tr + (e / W) * S::PITCH + e % W);
                    }
                }
            }
            if (more) {
                lds_transpose<W>(lds.tr, aR, i, g, pT);  // begins with a wave sync
                if constexpr (SRC == SRC_LAYER) {
                    if (g == 0) rcur[i] = ri;                        // r_l replaces r_{l-1}...
                    if (lane < W) lds.z[(u + 1) & 1][lane] = rnext;  // Z_{l+1} replaces Z_{l-1}
                } else {
                    if (lane < W) rprev[lane] = rnext;  // the ring slot of r_{l-s}
                }
                wave_sync();
#pragma unroll
                for (int v = 0; v < S::NV; ++v) {
                    if constexpr (DEEP) {
                        aR[v] = aF[v];
                        aF[v] = aN[v];
                    } else {
                        aR[v] = aN[v];
                    }
                }
            }
        }
    }
    if constexpr (UPD) {
        wave_umax2<W>(mx, mz);
        if (lane == 0) {
            const int slot = blockIdx.x % kRedShards;
            atomicMax(na.red + kRedDZ + slot, mx);
            atomicMax(na.red + kRedZ + slot, mz);
        }
    }
    if constexpr (SRC == SRC_LAYER) {
        for (int off = 32; off > 0; off >>= 1) mr = max(mr, (unsigned)__shfl_xor((int)mr, off, 64));
        if (lane == 0) atomicMax(na.red + kRedF + (int)(blockIdx.x % kRedShards), mr);
    }
}

// ---- one workgroup per segment, w = 64 or 128 ----------------------------
// The waves form a WGR x WGC grid over the product; each owns TW_R x TW_C
// 32x32 tiles.  w = 64: 4 waves, one tile each.  w = 128: 16 waves, one tile
// each (4 waves per SIMD); 8 waves of 64x32 or 32x64 tiles and 4 waves of
// 64x64 tiles measured within 3% of it.
template <int W>
struct TileShape {
    static constexpr int NT = (W == 128) ? 1024 : 256;  // threads per workgroup
    static constexpr int NWV = NT / 64;                        // waves
    static constexpr int PITCH = W + 4;
    static constexpr int NL = W * W / 4 / NT;  // float4 loads per thread per block
    static constexpr int T = W / 32;           // 32x32 tiles per side
    static constexpr int TW_R = 1;  // row tiles per wave
    static constexpr int TW_C = 1;  // column tiles per wave
    static constexpr int WGR = T / TW_R;                       // waves along the rows
    static constexpr int WGC = T / TW_C;                       // waves along the columns
    static constexpr int NQ = W / 8;             // k-steps of 8 (4 per lane half)
    static constexpr int NST = 4 * TW_R * TW_C;  // float4 stores per lane per product
    static_assert(WGR * WGC == NWV, "the wave grid covers the product");
    static_assert(NL <= NQ && NST <= NQ, "prefetch/stores are spread over the k-steps");
};

template <int W>
__device__ inline void load_block_regs(const float* blk, v4f* pre) {
    using S = TileShape<W>;
#pragma unroll
    for (int p = 0; p < S::NL; ++p)
        pre[p] = *reinterpret_cast<const v4f*>(blk + 4 * (threadIdx.x + S::NT * p));
}

template <int W>
__device__ inline void regs_to_lds(const v4f* pre, float* buf, bool trans) {
    using S = TileShape<W>;
#pragma unroll
    for (int p = 0; p < S::NL; ++p) {
        const int f = 4 * (threadIdx.x + S::NT * p);
        const int row = f / W, col = f % W;
        if (!trans) {
            *reinterpret_cast<v4f*>(buf + row * S::PITCH + col) = pre[p];
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) buf[(col + e) * S::PITCH + row] = pre[p][e];
        }
    }
}

// One row of a tile segment.  The wave owns row tile tr and column tiles
// tc0 + bb of the product and, through the same A operands, the matching
// rows of the mat-vec A_l r_{l-s}.  Interleaved with the MFMAs of k-step q:
// the LDS operands of step q+1 and float4 number q of the previous row's
// product (acc_old, when STORE); the prefetch of the next block is issued
// at step 0.  The memory traffic of a row thus overlaps its matrix work.  PROD and
// STORE are compile-time so that the unrolled k-loop is one basic block.
// A 32x32 product tile in the MFMA output layout (lane (i, h) holds row i at
// columns 8q + 4h .. +3) is written to the wave's LDS staging area with its
// 16-byte chunks XOR-swizzled by row, and read back so that lane t holds row
// 8p + t/8, columns 4(t%8) .. +3: each global store then covers 8 whole
// 128-byte rows of the tile instead of 32-byte pieces of 32 rows.
// stage_tile in two parts (so that other work can run between them): the
// tile into the staging area, then back out as whole rows.
__device__ inline void stage_tile_in(float* stg, const v16f& acc, int i, int h) {
    wave_sync();
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        v4f x = {acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]};
        *reinterpret_cast<v4f*>(stg + i * 32 + 4 * ((2 * q + h) ^ (i & 7))) = x;
    }
}
__device__ inline void stage_tile_out(const float* stg, v4f (&cst)[4]) {
    wave_sync();
    const int t = threadIdx.x & 63;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const int r = 8 * p + t / 8;
        cst[p] = *reinterpret_cast<const v4f*>(stg + r * 32 + 4 * ((t % 8) ^ (r & 7)));
    }
}
__device__ inline void stage_tile(float* stg, const v16f& acc, int i, int h, v4f (&cst)[4]) {
    stage_tile_in(stg, acc, i, h);
    stage_tile_out(stg, cst);
}

template <int W>
using TileAcc = v16f[TileShape<W>::TW_R][TileShape<W>::TW_C];

template <int W, bool PROD, bool STORE>
__device__ __forceinline__ void tile_row(const float* cur, const float* prv, const float* rprv,
                                         const float* next_blk, v4f (&pre)[TileShape<W>::NL],
                                         TileAcc<W>& acc, const TileAcc<W>& acc_old,
                                         float* old_dst, int tr0, int tc0, int i, int h,
                                         float (&part)[TileShape<W>::TW_R], float* stg) {
    using S = TileShape<W>;
    // w = 64: the previous row's product goes out through the staging area
    // (old_dst is then the tile's first element in the product block).
    constexpr bool STAGED = (W == 64);
    v4f cst[4];
    if constexpr (STORE && STAGED) stage_tile(stg, acc_old[0][0], i, h, cst);
#pragma unroll
    for (int a = 0; a < S::TW_R; ++a) {
        part[a] = 0.f;
#pragma unroll
        for (int bb = 0; bb < S::TW_C; ++bb) acc[a][bb] = v16f{};
    }
    v4f av[2][S::TW_R], rv[2];
    float pv[2][S::TW_C][4];
#pragma unroll
    for (int q = 0; q <= S::NQ; ++q) {
        if (q < S::NQ) {
            const int k = 8 * q + 4 * h;
#pragma unroll
            for (int a = 0; a < S::TW_R; ++a)
                av[q & 1][a] =
                    *reinterpret_cast<const v4f*>(cur + ((tr0 + a) * 32 + i) * S::PITCH + k);
            rv[q & 1] = *reinterpret_cast<const v4f*>(rprv + k);
            if (PROD) {
#pragma unroll
                for (int bb = 0; bb < S::TW_C; ++bb)
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        pv[q & 1][bb][e] = prv[(k + e) * S::PITCH + (tc0 + bb) * 32 + i];
            }
        }
        if (q == 0) {
#pragma unroll
            for (int p = 0; p < S::NL; ++p)
                pre[p] = *reinterpret_cast<const v4f*>(next_blk + 4 * (threadIdx.x + S::NT * p));
        }
        if (STORE && q < S::NST) {
            if constexpr (STAGED) {
                const int t = threadIdx.x & 63;
                *reinterpret_cast<v4f*>(old_dst + (8 * q + t / 8) * W + 4 * (t % 8)) = cst[q];
            } else {
                const int a = q / (4 * S::TW_C), bb = (q / 4) % S::TW_C, qq = q % 4;
                const v16f& x = acc_old[a][bb];
                v4f y = {x[4 * qq], x[4 * qq + 1], x[4 * qq + 2], x[4 * qq + 3]};
                *reinterpret_cast<v4f*>(old_dst + a * 32 * W + (tc0 + bb) * 32 + 8 * qq) = y;
            }
        }
        __builtin_amdgcn_sched_barrier(0);
        if (q > 0) {
            const int qb = (q - 1) & 1;
            if (PROD) {
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int a = 0; a < S::TW_R; ++a)
#pragma unroll
                        for (int bb = 0; bb < S::TW_C; ++bb)
                            acc[a][bb] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                                pv[qb][bb][e], av[qb][a][e], acc[a][bb], 0, 0, 0);
            }
#pragma unroll
            for (int a = 0; a < S::TW_R; ++a)
#pragma unroll
                for (int e = 0; e < 4; ++e) part[a] = fmaf(av[qb][a][e], rv[qb][e], part[a]);
        }
    }
#pragma unroll
    for (int a = 0; a < S::TW_R; ++a) part[a] += __shfl_xor(part[a], 32, 64);
}

// Chain walk with a double-buffered LDS block pair per workgroup: at the u-th
// row of the segment cur = bufs[u&1] holds A_l and prv = bufs[(u+1)&1] holds
// A_{l-s}; after the row, the prefetched A_{l+s} replaces prv.  Products are
// kept in one of two accumulator sets and stored during the next row.
template <int W, bool TRANS>
__global__ __launch_bounds__(TileShape<W>::NT)
__attribute__((amdgpu_waves_per_eu(TileShape<W>::NT / 256))) void pcr_level_tile(
    BlockSrc Ain, VecSrc rin, float* __restrict__ Aout, VecDst rout, int L, LevelPlan plan) {
    using S = TileShape<W>;
    __shared__ float bufs[2][W * S::PITCH];
    __shared__ float rpv[2][W];
    constexpr bool STAGED = (W == 64);
    __shared__ float stg_all[STAGED ? S::NWV : 1][STAGED ? 32 * 32 : 1];
    const int t = threadIdx.x;
    const long long item = blockIdx.x;
    const Seg sg = decode_segment(item, plan, L);
    const int s = plan.s;
    const float* rb = rin.base + sg.b * rin.bstride;
    float* ob = rout.base + sg.b * rout.bstride;
    if (sg.j == 0 && t < W) ob[sg.c * rout.rstride + t] = rb[sg.c * rin.rstride + t];
    if (sg.m0 > sg.count) return;  // uniform over the workgroup
    float* stg = stg_all[STAGED ? (t >> 6) : 0];

    const float* ab = Ain.base + sg.b * Ain.bstride;
    float* Ob = Aout + (long long)sg.b * L * W * W;
    const int lane = t & 63, wv = t >> 6;
    const int i = lane & 31, h = lane >> 5;
    const int tr0 = (wv / S::WGC) * S::TW_R, tc0 = (wv % S::WGC) * S::TW_C;
    const bool writes_r = (wv % S::WGC) == 0 && h == 0;
    // this lane's place in a product block (staged: the wave's tile origin)
    const int orow_off = STAGED ? tr0 * 32 * W + tc0 * 32 : (tr0 * 32 + i) * W + 4 * h;

    int l = sg.c + s * sg.m0;
    {
        const int lp = l - s;
        v4f pre[S::NL];
        if (t < W) rpv[1][t] = rb[(long long)lp * rin.rstride + t];
        if (sg.m0 >= 2) {
            load_block_regs<W>(ab + (long long)lp * Ain.rstride, pre);
            regs_to_lds<W>(pre, bufs[1], TRANS);
        }
        load_block_regs<W>(ab + (long long)l * Ain.rstride, pre);
        regs_to_lds<W>(pre, bufs[0], TRANS);
        if (t < W) rpv[0][t] = rb[(long long)l * rin.rstride + t];
    }

    TileAcc<W> accA, accB;
    float* pending = nullptr;  // destination of the product held in the "old" set
    int m = sg.m0, u = 0;
    auto row = [&](TileAcc<W>& an, TileAcc<W>& ao) -> bool {
        const float* cur = bufs[u & 1];
        float* prv = bufs[(u + 1) & 1];
        const float* rcur = rpv[u & 1];
        float* rprv = rpv[(u + 1) & 1];
        const bool more = m < sg.m1;
        const bool prod = m >= 2;
        __syncthreads();
        float rl_next = 0.f;
        if (more && t < W) rl_next = rb[(long long)(l + s) * rin.rstride + t];
        v4f pre[S::NL];
        float part[S::TW_R];
        // without a next row the prefetch rereads the current block (unused)
        const float* nb = ab + (long long)(more ? l + s : l) * Ain.rstride;
        if (prod && pending)
            tile_row<W, true, true>(cur, prv, rprv, nb, pre, an, ao, pending, tr0, tc0, i, h, part, stg);
        else if (prod)
            tile_row<W, true, false>(cur, prv, rprv, nb, pre, an, ao, pending, tr0, tc0, i, h, part, stg);
        else
            tile_row<W, false, false>(cur, prv, rprv, nb, pre, an, ao, pending, tr0, tc0, i, h, part, stg);
        if (writes_r) {
#pragma unroll
            for (int a = 0; a < S::TW_R; ++a) {
                const int rr = (tr0 + a) * 32 + i;
                ob[(long long)l * rout.rstride + rr] = rcur[rr] + part[a];
            }
        }
        pending = prod ? Ob + (long long)l * W * W + orow_off : nullptr;
        __syncthreads();  // every wave is done with prv and rprv
        if (more) {
            regs_to_lds<W>(pre, prv, TRANS);
            if (t < W) rprv[t] = rl_next;
        }
        ++m;
        ++u;
        l += s;
        return more;
    };
    bool last_in_A = true;
    for (;;) {
        if (!row(accA, accB)) { last_in_A = true; break; }
        if (!row(accB, accA)) { last_in_A = false; break; }
    }
    if (pending) {
        auto flush = [&](const TileAcc<W>& acc) {
            if constexpr (STAGED) {
                v4f cst[4];
                stage_tile(stg, acc[0][0], i, h, cst);
                const int tl = t & 63;
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    *reinterpret_cast<v4f*>(pending + (8 * q + tl / 8) * W + 4 * (tl % 8)) = cst[q];
            } else {
#pragma unroll
                for (int q = 0; q < S::NST; ++q) {
                    const int a = q / (4 * S::TW_C), bb = (q / 4) % S::TW_C, qq = q % 4;
                    const v16f& x = acc[a][bb];
                    v4f y = {x[4 * qq], x[4 * qq + 1], x[4 * qq + 2], x[4 * qq + 3]};
                    *reinterpret_cast<v4f*>(pending + a * 32 * W + (tc0 + bb) * 32 + 8 * qq) = y;
                }
            }
        };
        if (last_in_A)
            flush(accA);
        else
            flush(accB);
    }
}

// ---- first Newton level with the layers, w = 64 or 128 ---------------------
// The first PCR level (s = 1) of a Newton iteration for the MLP layer kinds,
// with the Jacobian blocks and residuals formed on the fly from the raw
// weights: J_l = D_l W_l (+ I), D_l = c diag(sigma'(W_l Z_{l-1} + b_l)).  At
// row l the current LDS block is the raw W_l (the weights are shared by every
// system, so they mostly come from L2) and the previous one J_{l-1}; the
// k-loop forms P = W_l J_{l-1} and W_l r_{l-1}, and then
//   r_l   = f_l(Z_{l-1}) - Z_l,
//   r'_l  = r_l + J_l r_{l-1}     = r_l + D_l (W_l r_{l-1}) (+ r_{l-1}),
//   A'_l  = J_l J_{l-1}           = D_l P (+ J_{l-1}).
// The pre-activation W_l Z_{l-1} of row l is summed from the prefetched raw
// block while it is still in registers (during row l-1).  After the row, W_l
// becomes J_l in place: the right operand of the next row.  A segment starting
// at row l first evaluates layer l-1 for r_{l-1} and J_{l-1}.  Also clears
// the max|dZ|, max|Z| slots and reduces max|r| into the kRedF slots.
template <int W>
__device__ inline float layer_out(const NewtonArgs& na, float a, float zin, float* dsc) {
    float d;
    const float y = activate(na.layer, a, &d);
    const bool res = layer_residual(na.layer);
    *dsc = res ? na.alpha * d : d;
    return res ? fmaf(na.alpha, y, zin) : y;
}

// blk (in registers as load_block_regs holds it) times the vector x in LDS,
// into y (LDS); W/4 consecutive threads share a row of the block.
template <int W>
__device__ inline void regs_matvec(const v4f* blk, const float* x, float* y) {
    using S = TileShape<W>;
    constexpr int LPR = W / 4;
    const int t = threadIdx.x;
    const v4f x4 = *reinterpret_cast<const v4f*>(x + (4 * t) % W);
#pragma unroll
    for (int p = 0; p < S::NL; ++p) {
        float d = blk[p][0] * x4[0];
#pragma unroll
        for (int e = 1; e < 4; ++e) d = fmaf(blk[p][e], x4[e], d);
#pragma unroll
        for (int off = 1; off < LPR; off <<= 1) d += __shfl_xor(d, off, 64);
        if (t % LPR == 0) y[(4 * (t + S::NT * p)) / W] = d;
    }
}

// buf (a raw W_l in LDS) becomes diag(dsc) buf (+ I).
template <int W>
__device__ inline void lds_to_jacobian(float* buf, const float* dsc, bool res) {
    using S = TileShape<W>;
#pragma unroll
    for (int p = 0; p < S::NL; ++p) {
        const int f = 4 * (threadIdx.x + S::NT * p);
        const int row = f / W, col = f % W;
        v4f x = *reinterpret_cast<v4f*>(buf + row * S::PITCH + col);
        x *= dsc[row];
        if (res && row >= col && row < col + 4) x[row - col] += 1.f;
        *reinterpret_cast<v4f*>(buf + row * S::PITCH + col) = x;
    }
}

template <int W>
__global__ __launch_bounds__(TileShape<W>::NT)
__attribute__((amdgpu_waves_per_eu(TileShape<W>::NT / 256))) void pcr_level_tile_layer(
    float* __restrict__ Aout, VecDst rout, int L, LevelPlan plan, NewtonArgs na) {
    using S = TileShape<W>;
    __shared__ float bufs[2][W * S::PITCH];
    __shared__ float rpv[2][W];  // r_{l-1} / r_l
    __shared__ float zv[2][W];   // Z_{l-1} / Z_l
    __shared__ float zt[W];      // Z_{l-2} of the segment's first row
    __shared__ float pz[W];      // W_l Z_{l-1} of the coming row
    __shared__ float pzp[W];     // W_{l-1} Z_{l-2} of the segment's first row
    __shared__ float dv[W];      // D_l of the row just done
    constexpr bool STAGED = (W == 64);
    __shared__ float stg_all[STAGED ? S::NWV : 1][STAGED ? 32 * 32 : 1];
    const int t = threadIdx.x;
    if (blockIdx.x == 0)
        for (int k = t; k < 2 * kRedShards; k += S::NT) na.red[k] = 0u;
    const Seg sg = decode_segment(blockIdx.x, plan, L);  // s = 1: one chain (c = 0)
    const bool res = layer_residual(na.layer);
    const float* Zb = na.Z + (long long)sg.b * L * W;
    const float* z0b = na.z0 + (long long)sg.b * W;
    float* ob = rout.base + sg.b * rout.bstride;
    float* Ob = Aout + (long long)sg.b * L * W * W;
    const int lane = t & 63, wv = t >> 6;
    unsigned mr = 0u;
    auto finish = [&]() {
        for (int off = 32; off > 0; off >>= 1)
            mr = max(mr, (unsigned)__shfl_xor((int)mr, off, 64));
        if (lane == 0) atomicMax(na.red + kRedF + (int)(blockIdx.x % kRedShards), mr);
    };
    if (sg.m0 > sg.count) {  // uniform over the workgroup; only L = 1 gets here
        if (sg.j == 0 && t < W) {
            float a = na.bias[t];
            for (int k = 0; k < W; ++k) a = fmaf(na.W[t * W + k], z0b[k], a);
            float dsc;
            const float r = layer_out<W>(na, a, z0b[t], &dsc) - Zb[t];
            ob[t] = r;
            mr = __float_as_uint(fabsf(r));
        }
        finish();
        return;
    }
    float* stg = stg_all[STAGED ? (t >> 6) : 0];
    const int i = lane & 31, h = lane >> 5;
    const int tr0 = (wv / S::WGC) * S::TW_R, tc0 = (wv % S::WGC) * S::TW_C;
    const bool writes_r = (wv % S::WGC) == 0 && h == 0;
    const int orow_off = STAGED ? tr0 * 32 * W + tc0 * 32 : (tr0 * 32 + i) * W + 4 * h;

    int l = sg.m0;
    {
        // layer l-1 at Z_{l-2} from the raw W_{l-1} (bufs[1]); W_l to bufs[0]
        if (t < W) {
            zt[t] = (l >= 2) ? Zb[(long long)(l - 2) * W + t] : z0b[t];
            zv[1][t] = Zb[(long long)(l - 1) * W + t];
            zv[0][t] = Zb[(long long)l * W + t];
        }
        v4f pre[S::NL];
        load_block_regs<W>(na.W + (long long)(l - 1) * W * W, pre);
        regs_to_lds<W>(pre, bufs[1], false);
        __syncthreads();
        regs_matvec<W>(pre, zt, pzp);
        load_block_regs<W>(na.W + (long long)l * W * W, pre);
        regs_to_lds<W>(pre, bufs[0], false);
        regs_matvec<W>(pre, zv[1], pz);
        __syncthreads();
        if (t < W) {
            float dsc;
            const float f =
                layer_out<W>(na, pzp[t] + na.bias[(long long)(l - 1) * W + t], zt[t], &dsc);
            const float r = f - zv[1][t];
            rpv[1][t] = r;
            dv[t] = dsc;
            mr = __float_as_uint(fabsf(r));
            if (sg.j == 0) ob[t] = r;  // row 0 (< s) is final
        }
        __syncthreads();
        if (sg.m0 >= 2) lds_to_jacobian<W>(bufs[1], dv, res);
    }

    TileAcc<W> accA, accB;
    float* pending = nullptr;  // destination of the product held in the "old" set
    int m = sg.m0, u = 0;
    auto row = [&](TileAcc<W>& an, TileAcc<W>& ao) -> bool {
        float* cur = bufs[u & 1];        // raw W_l
        float* prv = bufs[(u + 1) & 1];  // J_{l-1}
        const float* rprv = rpv[(u + 1) & 1];
        const float* zp = zv[(u + 1) & 1];
        const float* zc = zv[u & 1];
        const bool more = m < sg.m1;
        const bool prod = m >= 2;
        __syncthreads();
        float z_next = 0.f;
        if (more && t < W) z_next = Zb[(long long)(l + 1) * W + t];
        v4f pre[S::NL];
        float part[S::TW_R];
        const float* nb = na.W + (long long)(more ? l + 1 : l) * W * W;
        if (prod && pending)
            tile_row<W, true, true>(cur, prv, rprv, nb, pre, an, ao, pending, tr0, tc0, i, h,
                                    part, stg);
        else if (prod)
            tile_row<W, true, false>(cur, prv, rprv, nb, pre, an, ao, pending, tr0, tc0, i, h,
                                     part, stg);
        else
            tile_row<W, false, false>(cur, prv, rprv, nb, pre, an, ao, pending, tr0, tc0, i, h,
                                      part, stg);
#pragma unroll
        for (int a = 0; a < S::TW_R; ++a) {
            const int R = (tr0 + a) * 32 + i;
            float dsc;
            const float f = layer_out<W>(na, pz[R] + na.bias[(long long)l * W + R], zp[R], &dsc);
            if (writes_r) {
                const float r = f - zc[R];
                ob[(long long)l * rout.rstride + R] = r + fmaf(dsc, part[a], res ? rprv[R] : 0.f);
                rpv[u & 1][R] = r;
                dv[R] = dsc;
                mr = max(mr, __float_as_uint(fabsf(r)));
            }
            if (prod) {
                // lane row R, columns (tc0 + bb) * 32 + 8 qq + 4 h + e
#pragma unroll
                for (int bb = 0; bb < S::TW_C; ++bb)
#pragma unroll
                    for (int qq = 0; qq < 4; ++qq) {
                        const int col = (tc0 + bb) * 32 + 8 * qq + 4 * h;
                        v4f jp = {0.f, 0.f, 0.f, 0.f};
                        if (res) jp = *reinterpret_cast<const v4f*>(prv + R * S::PITCH + col);
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            an[a][bb][4 * qq + e] = fmaf(dsc, an[a][bb][4 * qq + e], jp[e]);
                    }
            }
        }
        pending = prod ? Ob + (long long)l * W * W + orow_off : nullptr;
        __syncthreads();  // cur, prv, rprv, pz are read; dv is complete
        if (more) {
            regs_to_lds<W>(pre, prv, false);   // raw W_{l+1}
            regs_matvec<W>(pre, zc, pz);       // W_{l+1} Z_l
            lds_to_jacobian<W>(cur, dv, res);  // J_l
            if (t < W) zv[(u + 1) & 1][t] = z_next;
        }
        ++m;
        ++u;
        ++l;
        return more;
    };
    bool last_in_A = true;
    for (;;) {
        if (!row(accA, accB)) { last_in_A = true; break; }
        if (!row(accB, accA)) { last_in_A = false; break; }
    }
    if (pending) {
        auto flush = [&](const TileAcc<W>& acc) {
            if constexpr (STAGED) {
                v4f cst[4];
                stage_tile(stg, acc[0][0], i, h, cst);
                const int tl = t & 63;
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    *reinterpret_cast<v4f*>(pending + (8 * q + tl / 8) * W + 4 * (tl % 8)) = cst[q];
            } else {
#pragma unroll
                for (int q = 0; q < S::NST; ++q) {
                    const int a = q / (4 * S::TW_C), bb = (q / 4) % S::TW_C, qq = q % 4;
                    const v16f& x = acc[a][bb];
                    v4f y = {x[4 * qq], x[4 * qq + 1], x[4 * qq + 2], x[4 * qq + 3]};
                    *reinterpret_cast<v4f*>(pending + a * 32 * W + (tc0 + bb) * 32 + 8 * qq) = y;
                }
            }
        };
        if (last_in_A)
            flush(accA);
        else
            flush(accB);
    }
    finish();
}

// ---- two levels per pass, w = 16 or 32 ------------------------------------
// Levels with strides s and 2s fused: the chains of stride 2s are the even and
// odd elements of the chains of stride s, so one wave walking a chain of
// stride s (elements m = 0, 1, 2, ... at rows l = c + m s) applies level s to
// element m,  r'_m = r_m + A_m r_{m-1},  A'_m = A_m A_{m-1}  (m >= 1 / m >= 2),
// and then level 2s,  r''_m = r'_m + A'_m r'_{m-2},  A''_m = A'_m A'_{m-2}
// (m >= 2 / m >= 4), with A'_{m-1}, A'_{m-2} and r'_{m-1}, r'_{m-2} kept in
// the wave's LDS.  Every read of level 2s sees level s's result, as Alg. 1
// requires, and the arithmetic per row is that of two separate levels; but
// each operator block is read from HBM and each product written once per
// two levels.  A segment starting at element m0 > 0 first walks elements
// m0-3 .. m0-1 again to rebuild that state; element 0 (row c < s) is final
// and its block is never read.
template <int W>
struct Wave2Lds {
    float tr[W * WaveShape<W>::PITCH];  // transposes and product staging
    float r[2][W];                      // raw r_m in slot m & 1
    float rp[2][W];                     // r'_m in slot m & 1
};

// acc = (A P)^T in layout R from pT (T layout of P) and aR (R layout of A).
template <int W>
__device__ inline void wave_product(const float* pT, const float* aR, float* out) {
    if constexpr (W == 16) {
        v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int v = 0; v < 4; ++v) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(pT[v], aR[v], acc, 0, 0, 0);
#pragma unroll
        for (int v = 0; v < 4; ++v) out[v] = acc[v];
    } else {
        v16f acc = {};
#pragma unroll
        for (int v = 0; v < 16; ++v)
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(pT[v], aR[v], acc, 0, 0, 0);
#pragma unroll
        for (int v = 0; v < 16; ++v) out[v] = acc[v];
    }
}

// sum over the row of a layout-R block times a vector in LDS; every lane of
// row i receives the full sum.
template <int W>
__device__ inline float wave_matvec(const float* aR, const float* x, int g) {
    using S = WaveShape<W>;
    float part = 0.f;
#pragma unroll
    for (int q = 0; q < S::NV / 4; ++q) {
        const v4f xv = *reinterpret_cast<const v4f*>(x + S::col(4 * q, g));
#pragma unroll
        for (int e = 0; e < 4; ++e) part = fmaf(aR[4 * q + e], xv[e], part);
    }
    part = group_sum<W>(part);
    return part;
}

// Writes a layout-R block row-major at dst (pitch PITCH, LDS).
template <int W>
__device__ inline void lds_put_R(float* dst, const float* aR, int i, int g) {
    using S = WaveShape<W>;
#pragma unroll
    for (int q = 0; q < S::NV / 4; ++q) {
        v4f x = {aR[4 * q], aR[4 * q + 1], aR[4 * q + 2], aR[4 * q + 3]};
        *reinterpret_cast<v4f*>(dst + i * S::PITCH + S::col(4 * q, g)) = x;
    }
}

// Stores a layout-R block to global memory (w = 32 through the staging area
// so that each store instruction writes 1 KiB contiguously).
template <int W>
__device__ inline void store_R(float* blk, const float* cR, float* stg, int i, int g, int lane) {
    using S = WaveShape<W>;
    if constexpr (W == 16) {
        v4f x = {cR[0], cR[1], cR[2], cR[3]};
        *reinterpret_cast<v4f*>(blk + i * W + S::col(0, g)) = x;
    } else {
        wave_sync();
        lds_put_R<W>(stg, cR, i, g);
        wave_sync();
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const int e = 4 * (lane + 64 * p);
            *reinterpret_cast<v4f*>(blk + e) =
                *reinterpret_cast<const v4f*>(stg + (e / W) * S::PITCH + e % W);
        }
    }
}

template <int W, bool TRANS>
__global__ __launch_bounds__(256) void pcr_level2_wave(BlockSrc Ain, VecSrc rin,
                                                       float* __restrict__ Aout, VecDst rout,
                                                       int L, LevelPlan plan) {
    using S = WaveShape<W>;
    constexpr int NV = S::NV;
    __shared__ Wave2Lds<W> lds_all[4];
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const long long item = (long long)blockIdx.x * 4 + wv;
    if (item >= plan.total) return;
    const int s = plan.s;
    const long long per_b = (long long)s * plan.segs_per_class;
    const int b = (int)(item / per_b);
    const long long rem = item - (long long)b * per_b;
    const int c = (int)(rem / plan.segs_per_class);
    const int j = (int)(rem - (long long)c * plan.segs_per_class);
    const int count = (L - 1 - c) / s;  // elements m = 0 .. count
    const int m0 = j * plan.n;
    if (m0 > count) return;  // whole wave
    const int m1 = min(count, m0 + plan.n - 1);
    const int mw = max(0, m0 - 3);
    Wave2Lds<W>& lds = lds_all[wv];
    const int i = lane % W;
    const int g = lane / W;
    const float* ab = Ain.base + b * Ain.bstride;
    const float* rb = rin.base + b * rin.bstride;
    float* ob = rout.base + b * rout.bstride;
    float* Ob = Aout + (long long)b * L * W * W;

    // aR: raw A_m (layout R); pT: raw A_{m-1} transposed; ringE / ringO: the
    // level-s products A'_m of even / odd elements, transposed (T layout)
    float aR[NV], pT[NV], aN[NV], ap[NV], app[NV], ringE[NV], ringO[NV];
    int l = c + s * mw;
    if (lane < W) lds.r[mw & 1][lane] = rb[(long long)l * rin.rstride + lane];
    if (mw >= 1) load_R<W, TRANS>(ab + (long long)l * Ain.rstride, i, g, aR);
    // one element of the walk; `ring` holds A'_{m-2} on entry and A'_m on exit
    auto element = [&](int m, float (&ring)[NV]) {
        const bool more = m < m1;
        const bool have_prev = m > mw;  // state of element m-1 is valid
        const bool out_row = m >= m0;
        float rnext = 0.f;
        if (more) {
            load_R<W, TRANS>(ab + (long long)(l + s) * Ain.rstride, i, g, aN);
            if (lane < W) rnext = rb[(long long)(l + s) * rin.rstride + lane];
        }
        wave_sync();
        // level s: r'_m and A'_m
        float rp = lds.r[m & 1][i];
        if (m >= 1 && have_prev) rp += wave_matvec<W>(aR, lds.r[(m + 1) & 1], g);
        const bool prod1 = m >= 2 && have_prev;
        if (prod1) wave_product<W>(pT, aR, ap);
        // level 2s: r''_m and A''_m (A'_{m-2} in ring, r'_{m-2} in slot m & 1)
        float rpp = rp;
        if (m >= 2 && out_row) rpp += wave_matvec<W>(ap, lds.rp[m & 1], g);
        const bool prod2 = m >= 4 && out_row;
        if (prod2) wave_product<W>(ring, ap, app);
        if (out_row && g == 0) ob[(long long)l * rout.rstride + i] = rpp;
        if (prod2) store_R<W>(Ob + (long long)l * W * W, app, lds.tr, i, g, lane);
        // state for elements m+1 and m+2
        wave_sync();
        if (g == 0) lds.rp[m & 1][i] = rp;
        if (prod1) lds_transpose<W>(lds.tr, ap, i, g, ring);  // begins with a wave sync
        if (more) {
            if (m >= 1) lds_transpose<W>(lds.tr, aR, i, g, pT);
            if (lane < W) lds.r[(m + 1) & 1][lane] = rnext;
#pragma unroll
            for (int v = 0; v < NV; ++v) aR[v] = aN[v];
        }
        l += s;
    };
    for (int m = mw; m <= m1; ++m) {
        if (m & 1)
            element(m, ringO);
        else
            element(m, ringE);
    }
}

// ---- two levels per pass, w = 32 (first levels only), 64, 128 ------------
// The chain walk of pcr_level2_wave with one workgroup per segment and one
// wave per 32-row strip of the blocks.  A lane (i, h) of wave v holds row
// R = 32 v + i of a block at the columns 8q + 4h .. +3 (q = 0 .. W/8-1): the
// left MFMA operand, read straight from HBM into registers, and also the
// layout in which the MFMA leaves a strip of the product (tile tc, float4
// qq at q = 4 tc + qq).  So A'_m = A_m A_{m-1} stays in registers as the left
// operand of A''_m = A'_m A'_{m-2}; only the right operands A_{m-1} and
// A'_{m-2} go through LDS (two blocks), and each element costs one block
// read and one block write for two levels.
// Column tiles TC0 .. TC0+NTC-1 of a product strip to global memory through
// the wave's 4 KiB LDS buffer stg: each tile goes in in the MFMA layout and
// comes back as 8 rows of 32 columns per store (whole 128-byte lines instead
// of 32-byte pieces of 32 rows).  Measured at w = 128 (one box): pair kernel
// 1177 -> 1160 us on the B 16, L 1024 solve; at w = 32 (one wave per
// workgroup) the extra 4 KiB and registers cost occupancy and it was slower.
// Column tile tc of a product strip, read back from the staging area as in
// tiles_store_staged, to global memory.
template <int W>
__device__ __forceinline__ void tile_rows_store(float* dst, const v4f (&cst)[4], int R, int tc) {
    const int lane = threadIdx.x & 63;
    float* d = dst + (R - (R & 31) + lane / 8) * W + 4 * (lane % 8);
#pragma unroll
    for (int p = 0; p < 4; ++p) *reinterpret_cast<v4f*>(d + 8 * p * W + 32 * tc) = cst[p];
}

template <int W, int TC0, int NTC>
__device__ __forceinline__ void tiles_store_staged(float* dst, const v16f (&acc)[NTC], int R,
                                                   int h, float* stg) {
#pragma unroll
    for (int tc = 0; tc < NTC; ++tc) {
        v4f cst[4];
        stage_tile(stg, acc[tc], R & 31, h, cst);
        tile_rows_store<W>(dst, cst, R, TC0 + tc);
    }
}

// Level-2s product of an element, A''_m = A'_m A'_{m-2} (A'_{m-2} in YT),
// two column tiles at a time (so no whole product strip is held); returns
// A'_m r'_{m-2} (r'_{m-2} in LDS).  side(q) runs at k-step q of the first
// pair of column tiles (see strip_product).  At w = 128 the tiles go out
// through stg, the first pair's beside the second pair's products (separate
// accumulators; per tile, at three k-steps: into stg, back as whole rows,
// to memory), the second pair's after them.  Measured on one box: pair
// kernel 1123 -> 1112 us on the B 16, L 1024 solve against the first pair
// stored between the two; the second pair's stores moved beside the next
// element's level-s product in the same way gained nothing more.
template <int W, class F = NoSide>
__device__ __forceinline__ float second_product(const float* YT, const StripC<W>& pC,
                                                const float* rpp, float* dst, int i, int h,
                                                int R, float* stg, F side = F{}) {
    constexpr int T = Tile2Shape<W>::T;
    constexpr int N0 = T < 2 ? T : 2;
    v16f acc[N0];
    const float part = strip_matvec<W>(pC, rpp, h);
    strip_product<W, 0, N0, false>(YT, pC, acc, i, h, nullptr, side);
    if constexpr (T == 4) {
        v16f acc2[2];
        v4f cst[4];
        auto out = [&](int q) {
            if (q == 1 || q == 5) stage_tile_in(stg, acc[q / 4], i, h);
            if (q == 2 || q == 6) stage_tile_out(stg, cst);
            if (q == 3 || q == 7) tile_rows_store<W>(dst, cst, R, q / 4);
        };
        strip_product<W, 2, 2, false>(YT, pC, acc2, i, h, nullptr, out);
        tiles_store_staged<W, 2, 2>(dst, acc2, R, h, stg);
    } else {
        tiles_store<W, 0, N0>(dst, acc, R, h);
    }
    return part;
}

// Quad q of the strip of strip_load_bwd below.
template <int W>
__device__ __forceinline__ void strip_load_bwd_quad(const BwdArgs& bw, int b, int L, int m,
                                                    StripA<W>& a, int R, int h, int q) {
    const int lay = L - max(m, 1);
    const float* Wl = bw.W + (long long)lay * W * W;
    const float* dl = bw.dscale + ((long long)b * L + lay) * W;
    const int dk = bw.residual ? R - 4 * h : -1;
    const v4f d4 = *reinterpret_cast<const v4f*>(dl + 8 * q + 4 * h);
#pragma unroll
    for (int e = 0; e < 4; ++e)
        a[q][e] = fmaf(d4[e], Wl[(8 * q + 4 * h + e) * W + R], dk == 8 * q + e ? 1.f : 0.f);
}

// The strip of row m of the backward's reversed transposed system, formed
// from the weights: J_{L-m}^T[R][k] = dscale_k W_{L-m}[k][R] (+ 1 if k = R);
// rows m < 1 (never read) are formed as row 1.
template <int W>
__device__ __forceinline__ void strip_load_bwd(const BwdArgs& bw, int b, int L, int m,
                                               StripA<W>& a, int R, int h) {
    const int lay = L - max(m, 1);
    const float* Wl = bw.W + (long long)lay * W * W;
    const float* dl = bw.dscale + ((long long)b * L + lay) * W;
    // the diagonal is column k = R, at 8q + e = R - 4h (opaque, so that the
    // compiler forms the selects here instead of holding them all)
    int dk = bw.residual ? R - 4 * h : -1;
    asm volatile("" : "+v"(dk));
#pragma unroll
    for (int q = 0; q < Tile2Shape<W>::NQ; ++q) {
        const v4f d4 = *reinterpret_cast<const v4f*>(dl + 8 * q + 4 * h);
#pragma unroll
        for (int e = 0; e < 4; ++e)
            a[q][e] = fmaf(d4[e], Wl[(8 * q + 4 * h + e) * W + R], dk == 8 * q + e ? 1.f : 0.f);
    }
}

// SRCB: the blocks are the backward's, formed from the weights (bw; Ain is
// unused; s = 1).
// (w = 64: two waves per SIMD; for the blocks from memory the register
// budget allows that without spilling, the backward's source spills a few
// registers and is still faster: 3% on a w = 64 backward in all)
template <int W, bool TRANS, bool SRCB = false>
__global__ __launch_bounds__(Tile2Shape<W>::NT)
__attribute__((amdgpu_waves_per_eu(W == 32 ? 3 : W == 64 ? 2 : 1))) void pcr_level2_tile(BlockSrc Ain, VecSrc rin,
                                                                     float* __restrict__ Aout,
                                                                     VecDst rout, int L,
                                                                     LevelPlan plan,
                                                                     BwdArgs bw = {}) {
    using S = Tile2Shape<W>;
    __shared__ float X[W * S::PITCH];  // A_{m-1}, transposed
    __shared__ float Y[W * S::PITCH];  // A'_{m-2}, transposed
    __shared__ float rv[2][W];         // r_m in slot m & 1, r_{m-1} in the other
    __shared__ float rp[2][W];         // r'_{m-2} in slot m & 1, r'_{m-1} in the other
    // w = 128: per-wave staging of the level-2s product's stores
    __shared__ float STG[W == 128 ? S::NWV * 1024 : 1];
    const int t = threadIdx.x;
    const int lane = t & 63, i = lane & 31, h = lane >> 5;
    const int R = 32 * (t >> 6) + i;
    float* stg = STG + (W == 128 ? (t >> 6) * 1024 : 0);
    const int s = plan.s;
    const long long item = blockIdx.x;
    const long long per_b = (long long)s * plan.segs_per_class;
    const int b = (int)(item / per_b);
    const long long rem = item - (long long)b * per_b;
    const int c = (int)(rem / plan.segs_per_class);
    const int j = (int)(rem - (long long)c * plan.segs_per_class);
    const int count = (L - 1 - c) / s;  // elements m = 0 .. count
    const int m0 = j * plan.n;
    if (m0 > count) return;  // uniform over the workgroup
    const int m1 = min(count, m0 + plan.n - 1);
    const int mw = max(0, m0 - 3);
    const float* ab = Ain.base + b * Ain.bstride;
    const float* rb = rin.base + b * rin.bstride;
    float* ob = rout.base + b * rout.bstride;
    float* Ob = Aout + (long long)b * L * W * W;

    StripA<W> a;             // A_m, then A_{m+1}
    StripC<W> pE, pO;        // A'_m of even / odd elements (w >= 64: of m % 3 = 0, 1)
    auto load = [&](int row) {
        if constexpr (SRCB)
            strip_load_bwd<W>(bw, b, L, row, a, R, h);
        else
            strip_load<W, TRANS>(ab + (long long)row * Ain.rstride, a, R, h);
    };
    auto load_quad = [&](int row, int q) {
        if constexpr (SRCB)
            strip_load_bwd_quad<W>(bw, b, L, row, a, R, h, q);
        else
            strip_load_quad<W, TRANS>(ab + (long long)row * Ain.rstride, a, R, h, q);
    };
    int l = c + s * mw;
    if (t < W) rv[mw & 1][t] = rb[(long long)l * rin.rstride + t];
    if (mw >= 1) load(l);
    __syncthreads();
    // element m: a = A_m on entry and A_{m+1} on exit, pC <- A'_m.  A_m
    // replaces A_{m-1} in X as soon as the first product is done, and only
    // then is A_{m+1} requested into the same registers.  Two barriers per
    // element: B0 after the reads of X and rv, B1 after those of Y and rp.
    // X and rv are rewritten between B0 and B1 (read again after B1), Y and
    // rp after B1 (read again after the next B0).
    // YD (w = 64, 128): A'_{m-2} (pY) goes to Y beside the level-s product
    // of element m, which reads neither Y nor pY, so three product strips
    // are held (A'_{m-2}, A'_{m-1}, A'_m).  Otherwise (w = 32, whose three
    // waves per SIMD leave no registers for a third strip) A'_{m-1} (pY)
    // goes to Y after B1 of element m and two strips are held.  Measured on
    // one box: w = 128 pair 1159 -> 1145 us on the B 16, L 1024 solve
    // (B 16, L 1024 residual forward + backward 19.99 -> 19.67 ms); w = 64
    // backward (B 64, L 1024) 1.66 -> 1.63 ms.
    constexpr bool YD = W >= 64;
    auto element = [&](int m, StripC<W>& pC, StripC<W>& pY) {
        const bool more = m < m1;
        const bool have_prev = m > mw;  // state of element m-1 is valid
        const bool out_row = m >= m0;
        float rnext = 0.f;
        if (more && t < W) rnext = rb[(long long)(l + s) * rin.rstride + t];
        // level s: r'_m and A'_m (the strips are set on every path, so that no
        // old value of a register set stays live across elements)
        float r1 = rv[m & 1][R];
        const bool prod1 = m >= 2 && have_prev;
        const bool puty = YD && m >= 4 && m - 2 > mw;
        auto yside = [&](int q) {
            if (puty) strip_put_T_quad<W>(Y, pY, R, h, q);
        };
        if (prod1) {
            r1 += strip_product<W, 0, S::T, true>(X, a, pC, i, h, rv[(m + 1) & 1], yside);
        } else {
            if (puty) strip_put_T<W>(Y, pY, R, h);
            if (m >= 1 && have_prev) r1 += strip_matvec<W>(a, rv[(m + 1) & 1], h);
            strip_zero<W>(pC);
        }
        __syncthreads();  // B0: X and rv are read
        if (more && t < W) rv[(m + 1) & 1][t] = rnext;
        // A_m to X and the strip of the next element into a (without a next
        // element the load rereads the current block, unused).  At w = 128
        // from memory: quad by quad beside the level-2s product, which reads
        // neither (the matrix cores are otherwise idle while a lone
        // workgroup per CU writes and loads); else before it (w = 64 measured
        // no faster, and the quad form of the backward's strips spills).
        constexpr bool SIDE = W == 128 && !SRCB;
        const bool putx = more && m >= 1;
        const int nrow = more ? l + s : l;
        auto side = [&](int q) {
            if (putx) strip_put_T_quad<W>(X, a, R, h, q);
            load_quad(nrow, q);
        };
        if constexpr (!SIDE) {
            if (putx) strip_put_T<W>(X, a, R, h);
            load(nrow);
        }
        // level 2s: r''_m and A''_m
        float r2 = r1;
        const bool prod2 = m >= 4 && out_row;
        if (prod2) {
            if constexpr (SIDE)
                r2 += second_product<W>(Y, pC, rp[m & 1], Ob + (long long)l * W * W, i, h, R,
                                        stg, side);
            else
                r2 += second_product<W>(Y, pC, rp[m & 1], Ob + (long long)l * W * W, i, h, R,
                                        stg);
        } else {
            if constexpr (SIDE) {
#pragma unroll
                for (int q = 0; q < S::NQ; ++q) side(q);
            }
            if (m >= 2 && out_row) r2 += strip_matvec<W>(pC, rp[m & 1], h);
        }
        if (out_row && h == 0) ob[(long long)l * rout.rstride + R] = r2;
        __syncthreads();  // B1: Y and rp are read
        if (h == 0) rp[m & 1][R] = r1;
        if constexpr (!YD)
            if (more && m >= 3 && m - 1 > mw) strip_put_T<W>(Y, pY, R, h);  // A'_{m-1}
        l += s;
    };
    if constexpr (YD) {
        // three elements per loop step, so that every register set keeps its
        // role (set m % 3 receives A'_m, p3 for m % 3 = 2); elements before
        // mw are skipped
        StripC<W> p3;
        for (int m = mw - mw % 3; m <= m1; m += 3) {
            if (m >= mw) element(m, pE, pO);
            if (m + 1 >= mw && m + 1 <= m1) element(m + 1, pO, p3);
            if (m + 2 >= mw && m + 2 <= m1) element(m + 2, p3, pE);
        }
    } else {
        // an even and an odd element per loop step, so that every register
        // set keeps its role through the loop (no parity branch to merge);
        // an odd first element starts the loop with its even slot skipped
        for (int m = mw & ~1; m <= m1; m += 2) {
            if (m >= mw) element(m, pE, pO);
            if (m + 1 <= m1) element(m + 1, pO, pE);
        }
    }
}

// The last two levels of a solve (strides s and 2s, 4s >= L): no operator
// is written, and the one product the walk would form, A'_m = A_m A_{m-1},
// only ever meets the vector r'_{m-2}, so A'_m r'_{m-2} is taken as
// A_m (A_{m-1} r'_{m-2}) = A_m t_{m-1}, with t_m = A_m r'_{m-1} formed by the
// element before: three mat-vecs per element and no MFMA work.  The strips
// are double-buffered in registers (the next one is requested before the
// mat-vecs of the current one).
template <int W, bool TRANS>
__global__ __launch_bounds__(Tile2Shape<W>::NT) void pcr_level2_tile_last(BlockSrc Ain,
                                                                          VecSrc rin,
                                                                          VecDst rout, int L,
                                                                          LevelPlan plan) {
    using S = Tile2Shape<W>;
    __shared__ float rv[2][W];  // r_m in slot m & 1, r_{m-1} in the other
    __shared__ float rp[2][W];  // r'_{m-1} in slot (m+1) & 1
    __shared__ float tv[2][W];  // t_{m-1} = A_{m-1} r'_{m-2} in slot (m+1) & 1
    const int t = threadIdx.x;
    const int lane = t & 63, h = lane >> 5;
    const int R = 32 * (t >> 6) + (lane & 31);
    const int s = plan.s;
    const long long item = blockIdx.x;
    const long long per_b = (long long)s * plan.segs_per_class;
    const int b = (int)(item / per_b);
    const long long rem = item - (long long)b * per_b;
    const int c = (int)(rem / plan.segs_per_class);
    const int j = (int)(rem - (long long)c * plan.segs_per_class);
    const int count = (L - 1 - c) / s;  // elements m = 0 .. count
    const int m0 = j * plan.n;
    if (m0 > count) return;  // uniform over the workgroup
    const int m1 = min(count, m0 + plan.n - 1);
    const int mw = max(0, m0 - 3);
    const float* ab = Ain.base + b * Ain.bstride;
    const float* rb = rin.base + b * rin.bstride;
    float* ob = rout.base + b * rout.bstride;

    StripA<W> aE, aO;  // A_m of even / odd elements (A_0 is never read)
    int l = c + s * mw;
    if (t < W) rv[mw & 1][t] = rb[(long long)l * rin.rstride + t];
    if (mw >= 1) {
        if (mw & 1)
            strip_load<W, TRANS>(ab + (long long)l * Ain.rstride, aO, R, h);
        else
            strip_load<W, TRANS>(ab + (long long)l * Ain.rstride, aE, R, h);
    } else {
#pragma unroll
        for (int q = 0; q < S::NQ; ++q) aE[q] = v4f{0.f, 0.f, 0.f, 0.f};
    }
    __syncthreads();
    auto element = [&](int m, StripA<W>& aC, StripA<W>& aN) {
        const bool more = m < m1;
        const bool have_prev = m > mw;
        const bool out_row = m >= m0;
        // the next strip; with chains of a few elements, as here, the
        // segments are short, so no block is read that is not used
        if (more) strip_load<W, TRANS>(ab + (long long)(l + s) * Ain.rstride, aN, R, h);
        float rnext = 0.f;
        if (more && t < W) rnext = rb[(long long)(l + s) * rin.rstride + t];
        const float* rm1 = rv[(m + 1) & 1];
        const float* rpm1 = rp[(m + 1) & 1];
        const float* tm1 = tv[(m + 1) & 1];
        float u1 = 0.f, u2 = 0.f, u3 = 0.f;  // A_m r_{m-1}, A_m r'_{m-1}, A_m t_{m-1}
#pragma unroll
        for (int q = 0; q < S::NQ; ++q) {
            const int k = 8 * q + 4 * h;
            const v4f x1 = *reinterpret_cast<const v4f*>(rm1 + k);
            const v4f x2 = *reinterpret_cast<const v4f*>(rpm1 + k);
            const v4f x3 = *reinterpret_cast<const v4f*>(tm1 + k);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                u1 = fmaf(aC[q][e], x1[e], u1);
                u2 = fmaf(aC[q][e], x2[e], u2);
                u3 = fmaf(aC[q][e], x3[e], u3);
            }
        }
        u1 += __shfl_xor(u1, 32, 64);
        u2 += __shfl_xor(u2, 32, 64);
        u3 += __shfl_xor(u3, 32, 64);
        float r1 = rv[m & 1][R];
        if (m >= 1 && have_prev) r1 += u1;
        const float r2 = (m >= 2 && out_row) ? r1 + u3 : r1;
        if (out_row && h == 0) ob[(long long)l * rout.rstride + R] = r2;
        __syncthreads();  // rv, rp and tv are read
        if (h == 0) {
            rp[m & 1][R] = r1;
            tv[m & 1][R] = u2;
        }
        if (more && t < W) rv[(m + 1) & 1][t] = rnext;
        __syncthreads();
        l += s;
    };
    for (int m = mw; m <= m1; ++m) {
        if (m & 1)
            element(m, aO, aE);
        else
            element(m, aE, aO);
    }
}

// The first two levels (s = 1, 2) of a Newton iteration as one pass of the
// walk above, with the layers evaluated on the fly: element m loads the raw
// W_m strip, forms the pre-activation W_m Z_{m-1} from it, then
// r_m = f_m(Z_{m-1}) - Z_m and, scaling its own row, the strip of
// J_m = D_m W_m (+ I); the walk goes on with A_m = J_m.  Also clears the
// max|dZ|, max|Z| slots and reduces max|r| into the kRedF slots.
// w = 32: four one-wave workgroups per SIMD (128 registers, 9.75 KiB of LDS
// each: the CU's 160 KiB hold all sixteen); with 4096 segments that is one
// round over the chip (measured on one box: PCR level time of the B 256,
// L 256 forward 0.91 -> 0.85-0.89 ms against three per SIMD and 6144).
template <int W>
__global__ __launch_bounds__(Tile2Shape<W>::NT)
__attribute__((amdgpu_waves_per_eu(W == 32 ? 4 : 1))) void pcr_level2_tile_layer(
    float* __restrict__ Aout, VecDst rout, int L, LevelPlan plan, NewtonArgs na) {
    using S = Tile2Shape<W>;
    __shared__ float X[W * S::PITCH];  // J_{m-1}, transposed
    __shared__ float Y[W * S::PITCH];  // A'_{m-2}, transposed
    __shared__ float rv[2][W];         // r_{m-1} in slot (m+1) & 1
    __shared__ float rp[2][W];         // r'_{m-2} in slot m & 1
    __shared__ float zv[2][W];         // Z_m in slot m & 1, Z_{m-1} in the other
    __shared__ float STG[W == 128 ? S::NWV * 1024 : 1];  // as in pcr_level2_tile
    const int t = threadIdx.x;
    float* stg = STG + (W == 128 ? (t >> 6) * 1024 : 0);
    if (blockIdx.x == 0)
        for (int k = t; k < 2 * kRedShards; k += S::NT) na.red[k] = 0u;
    const int lane = t & 63, i0 = lane & 31, h0 = lane >> 5;
    const int R0 = 32 * (t >> 6) + i0;
    const int b = (int)(blockIdx.x / plan.segs_per_class);  // s = 1: one chain per system
    const int j = (int)(blockIdx.x - (long long)b * plan.segs_per_class);
    const int count = L - 1;
    const int m0 = j * plan.n;
    unsigned mr = 0u;
    if (m0 <= count) {  // uniform over the workgroup
        const int m1 = min(count, m0 + plan.n - 1);
        const int mw = max(0, m0 - 3);
        const bool res = layer_residual(na.layer);
        // w = 128 (registers to spare): the residual layers' identity as a
        // per-lane pattern held through the walk, one FMA per strip element
        float dg[S::NQ][4];
        if constexpr (W == 128) {
            const int dk = res ? R0 - 4 * h0 : -1;
#pragma unroll
            for (int q = 0; q < S::NQ; ++q)
#pragma unroll
                for (int e = 0; e < 4; ++e) dg[q][e] = dk == 8 * q + e ? 1.f : 0.f;
        }
        const float* Zb = na.Z + (long long)b * L * W;
        float* ob = rout.base + b * rout.bstride;
        float* Ob = Aout + (long long)b * L * W * W;
        // PF (w = 32, where an element's products are short): the weight
        // strip, iterate row and bias of later elements are requested at the
        // start of an element, into the other slot of a two-slot ring (by
        // element parity), and every request is issued on every element
        // (clamped to the chain's last row), so no branch makes the compiler
        // wait for all of them.  Otherwise (w = 64, 128, no registers to
        // spare) one strip buffer is refilled after J_m has gone to LDS.
        constexpr bool PF = W == 32;
        StripA<W> aE, aO;       // W_m, then J_m (PF: by element parity)
        StripC<W> pE, pO;       // A'_m of even / odd elements
        float zq0 = 0.f, zq1 = 0.f, bq0 = 0.f, bq1 = 0.f;  // PF: Z and bias ring
        const int tw = t & (W - 1);
        if (t < W) {
            zv[(mw + 1) & 1][t] =
                mw >= 1 ? Zb[(long long)(mw - 1) * W + t] : na.z0[(long long)b * W + t];
            zv[mw & 1][t] = Zb[(long long)mw * W + t];
        }
        strip_load<W, false>(na.W + (long long)mw * W * W, (PF && (mw & 1)) ? aO : aE, R0, h0);
        if constexpr (PF) {
            const float zn = Zb[(long long)min(mw + 1, count) * W + tw];  // Z_{mw+1}
            const float bn = na.bias[(long long)mw * W + R0];
            if (mw & 1) {
                zq0 = zn;
                bq1 = bn;
            } else {
                zq1 = zn;
                bq0 = bn;
            }
        }
        __syncthreads();
        // Two barriers per element as in pcr_level2_tile; zv and rv are
        // rewritten before B1, rp and Y after it.  aC holds the strip of
        // element m; with PF, aN receives that of m+1, zS (slot m & 1)
        // Z_{m+2} and bO the bias of m+1, while zO holds Z_{m+1} and bS the
        // bias of m.
        auto element = [&](int m, StripC<W>& pC, StripC<W>& pP, StripA<W>& aC, StripA<W>& aN,
                           float& zS, float& zO, float& bS, float& bO) {
            const bool more = m < m1;
            const bool have_prev = m > mw;
            const bool out_row = m >= m0;
            float znext = 0.f, bm;
            if constexpr (PF) {
                strip_load<W, false>(na.W + (long long)min(m + 1, count) * W * W, aN, R0, h0);
                zS = Zb[(long long)min(m + 2, count) * W + tw];
                bO = na.bias[(long long)min(m + 1, count) * W + R0];
                bm = bS;
            } else {
                if (more && t < W) znext = Zb[(long long)(m + 1) * W + t];
                bm = na.bias[(long long)m * W + R0];
            }
            // The lane's row and half as opaque values: the LDS and global
            // addresses derived from them are formed per element instead of
            // being held (or spilled) across the whole walk.
            int R = R0, h = h0, i = i0;
            asm volatile("" : "+v"(R), "+v"(h), "+v"(i));
            // layer m at Z_{m-1}: r_m and the strip of J_m
            const float* zp = zv[(m + 1) & 1];
            float dsc;
            const float f = layer_out<W>(na, strip_matvec<W>(aC, zp, h) + bm, zp[R], &dsc);
            const float rm = f - zv[m & 1][R];
            mr = max(mr, __float_as_uint(fabsf(rm)));
            if (W == 128 && res) {
#pragma unroll
                for (int q = 0; q < S::NQ; ++q)
#pragma unroll
                    for (int e = 0; e < 4; ++e) aC[q][e] = fmaf(dsc, aC[q][e], dg[q][e]);
            } else if (res) {
                // the diagonal is column k = R, at 8q + e = R - 4h (the empty
                // asm keeps the compiler from holding 64 precomputed selects)
                int dk = R - 4 * h;
                asm volatile("" : "+v"(dk));
#pragma unroll
                for (int q = 0; q < S::NQ; ++q)
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        aC[q][e] = fmaf(dsc, aC[q][e], dk == 8 * q + e ? 1.f : 0.f);
            } else {
#pragma unroll
                for (int q = 0; q < S::NQ; ++q)
#pragma unroll
                    for (int e = 0; e < 4; ++e) aC[q][e] *= dsc;
            }
            // level 1: r'_m and A'_m
            float r1 = rm;
            const bool prod1 = m >= 2 && have_prev;
            if (prod1) {
                r1 += strip_product<W, 0, S::T, true>(X, aC, pC, i, h, rv[(m + 1) & 1]);
            } else {
                if (m >= 1 && have_prev) r1 += strip_matvec<W>(aC, rv[(m + 1) & 1], h);
                // pC is read only where a product has set it (m >= 2 after
                // the walk's first element); at w = 32 its zeroing, which
                // the compiler hoists onto every element, is left out
                if constexpr (W != 32) strip_zero<W>(pC);
            }
            __syncthreads();  // B0: X, rv and zv are read
            if (h == 0) rv[m & 1][R] = rm;
            // J_m to X and (without PF) the weight strip of the next element
            // into aC (without a next element this rereads the current one,
            // unused): at w = 128 quad by quad beside the level-2 product,
            // which reads neither, else before it
            constexpr bool SIDE = W == 128 && !PF;
            const bool putx = more && m >= 1;
            const float* wn = na.W + (long long)(more ? m + 1 : m) * W * W;
            auto side = [&](int q) {
                if (putx) strip_put_T_quad<W>(X, aC, R, h, q);
                strip_load_quad<W, false>(wn, aC, R, h, q);
            };
            if constexpr (!SIDE)
                if (putx) strip_put_T<W>(X, aC, R, h);  // J_m
            if constexpr (PF) {
                if (more && t < W) zv[(m + 1) & 1][t] = zO;
            } else {
                if (more && t < W) zv[(m + 1) & 1][t] = znext;
                if constexpr (!SIDE) strip_load<W, false>(wn, aC, R, h);
            }
            // level 2: r''_m and A''_m
            float r2 = r1;
            const bool prod2 = m >= 4 && out_row;
            if (prod2) {
                if constexpr (SIDE)
                    r2 += second_product<W>(Y, pC, rp[m & 1], Ob + (long long)m * W * W, i, h, R,
                                            stg, side);
                else
                    r2 += second_product<W>(Y, pC, rp[m & 1], Ob + (long long)m * W * W, i, h, R,
                                            stg);
            } else {
                if constexpr (SIDE) {
#pragma unroll
                    for (int q = 0; q < S::NQ; ++q) side(q);
                }
                if (m >= 2 && out_row) r2 += strip_matvec<W>(pC, rp[m & 1], h);
            }
            if (out_row && h == 0) ob[(long long)m * rout.rstride + R] = r2;
            __syncthreads();  // B1: Y and rp are read
            if (h == 0) rp[m & 1][R] = r1;
            if (more && m >= 3 && m - 1 > mw) strip_put_T<W>(Y, pP, R, h);  // A'_{m-1}
        };
        // an even and an odd element per loop step, so that every register
        // set keeps its role through the loop (no parity branch to merge);
        // an odd first element starts the loop with its even slot skipped
        for (int m = mw & ~1; m <= m1; m += 2) {
            if (m >= mw) {
                if constexpr (PF)
                    element(m, pE, pO, aE, aO, zq0, zq1, bq0, bq1);
                else
                    element(m, pE, pO, aE, aE, zq0, zq1, bq0, bq1);
            }
            if (m + 1 <= m1) {
                if constexpr (PF)
                    element(m + 1, pO, pE, aO, aE, zq1, zq0, bq1, bq0);
                else
                    element(m + 1, pO, pE, aE, aE, zq1, zq0, bq1, bq0);
            }
        }
    }
    for (int off = 32; off > 0; off >>= 1) mr = max(mr, (unsigned)__shfl_xor((int)mr, off, 64));
    if (lane == 0) atomicMax(na.red + kRedF + (int)(blockIdx.x % kRedShards), mr);
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
        const dim3 g3((unsigned)((p.total + 3) / 4)), block(256);
        const NewtonArgs na{};
        if (w == 16) {
            if (Ain.trans)
                hipLaunchKernelGGL((pcr_level_wave<16, true, SRC_MEM, false>), g3, block, 0,
                                   stream, Ain, rin, Aout, rout, L, p, na);
            else
                hipLaunchKernelGGL((pcr_level_wave<16, false, SRC_MEM, false>), g3, block, 0,
                                   stream, Ain, rin, Aout, rout, L, p, na);
        } else {
            if (Ain.trans)
                hipLaunchKernelGGL((pcr_level_wave<32, true, SRC_MEM, false>), g3, block, 0,
                                   stream, Ain, rin, Aout, rout, L, p, na);
            else
                hipLaunchKernelGGL((pcr_level_wave<32, false, SRC_MEM, false>), g3, block, 0,
                                   stream, Ain, rin, Aout, rout, L, p, na);
        }
        return hipGetLastError();
    }
    if (w == 64 || w == 128) {
        const LevelPlan p = plan_level(B, L, s, w == 64 ? 4096 : 1024, 64);
        const dim3 grid((unsigned)p.total),
            block(w == 64 ? TileShape<64>::NT : TileShape<128>::NT);
        if (w == 64) {
            if (Ain.trans)
                hipLaunchKernelGGL((pcr_level_tile<64, true>), grid, block, 0, stream, Ain, rin,
                                   Aout, rout, L, p);
            else
                hipLaunchKernelGGL((pcr_level_tile<64, false>), grid, block, 0, stream, Ain, rin,
                                   Aout, rout, L, p);
        } else {
            if (Ain.trans)
                hipLaunchKernelGGL((pcr_level_tile<128, true>), grid, block, 0, stream, Ain, rin,
                                   Aout, rout, L, p);
            else
                hipLaunchKernelGGL((pcr_level_tile<128, false>), grid, block, 0, stream, Ain, rin,
                                   Aout, rout, L, p);
        }
        return hipGetLastError();
    }
    if (small_width(w)) return launch_pcr_level_small(Ain, rin, Aout, rout, B, L, w, s, stream);
    const long long rows = (long long)B * L;
    hipLaunchKernelGGL(pcr_level_generic, dim3((unsigned)rows), dim3(kThreads), 0, stream,
                       Ain, rin, Aout, rout, L, w, s);
    return hipGetLastError();
}

// Tile widths pair their levels only for B L >= 2048 chain elements: the
// pair kernels walk segments of at least 8 elements, so below that they
// would run fewer workgroups than the chip has CUs, where single levels
// (segments of one row) keep it busy.
bool two_level(int B, int L, int w) {
    if (w == 16 || w == 32) return true;
    return (w == 64 || w == 128) && (long long)B * L >= 2048;
}

// Segments of the fused pair cover elements m = 0 .. (L-1-c)/s of each chain;
// n rows each, at least 8 so that the 3-row warm-up stays a small share.
// Tile pairs: about target_wgs workgroups (one segment each), segments of at
// least 8 elements where the chains allow (a segment re-walks up to 3
// elements before its first).
LevelPlan plan_level2_tile(int B, int L, int s, long long target_wgs) {
    LevelPlan p;
    p.s = s;
    const int E = (L - 1) / s + 1;
    const long long chains = (long long)B * s;
    long long segs = target_wgs / chains;
    if (segs < 1) segs = 1;
    long long n = (E + segs - 1) / segs;
    if (n < 8) n = 8;
    p.n = (int)n;
    p.segs_per_class = (int)((E + n - 1) / n);
    p.total = chains * p.segs_per_class;
    return p;
}

// Workgroups per tile pass: w = 128 and 64 fill the CUs with one or two
// workgroups of 4 or 2 waves each; a w = 32 workgroup is one wave: 4096 for
// the first pair with the layers (four per SIMD, one round; segments of 16
// elements for the B 256, L 256 forward), 6144 for the backward's first
// pair (three per SIMD; with three per SIMD the forward measured 3% faster
// at 6144 than at 8192 and 1.4% than at 4096, on one box); 512 workgroups
// at w = 128 and 2048 at w = 64 were 3% and 13% slower.
long long pair_tile_target(int w, bool layer = false) {
    return w == 32 ? (layer ? 4096 : 6144) : w == 64 ? 1024 : 256;
}

LevelPlan plan_level2(int B, int L, int s, long long target_items) {
    LevelPlan p;
    p.s = s;
    const int E = (L - 1) / s + 1;  // elements of the longest chain
    const long long rows = (long long)B * s * E;
    long long n = (rows + target_items - 1) / target_items;
    if (n < 8) n = 8;
    if (n > 64) n = 64;
    p.n = (int)n;
    p.segs_per_class = (E + p.n - 1) / p.n;
    p.total = (long long)B * s * p.segs_per_class;
    return p;
}

hipError_t launch_pcr_level2(const BlockSrc& Ain, const VecSrc& rin, float* Aout,
                             const VecDst& rout, int B, int L, int w, int s,
                             hipStream_t stream) {
    const LevelPlan p = plan_level2(B, L, s, w == 16 ? 8192 : 4096);
    const dim3 g3((unsigned)((p.total + 3) / 4)), block(256);
    if (w == 16) {
        if (Ain.trans)
            hipLaunchKernelGGL((pcr_level2_wave<16, true>), g3, block, 0, stream, Ain, rin, Aout,
                               rout, L, p);
        else
            hipLaunchKernelGGL((pcr_level2_wave<16, false>), g3, block, 0, stream, Ain, rin, Aout,
                               rout, L, p);
    } else if (w == 32) {
        if (Ain.trans)
            hipLaunchKernelGGL((pcr_level2_wave<32, true>), g3, block, 0, stream, Ain, rin, Aout,
                               rout, L, p);
        else
            hipLaunchKernelGGL((pcr_level2_wave<32, false>), g3, block, 0, stream, Ain, rin, Aout,
                               rout, L, p);
    } else if (w == 64 || w == 128) {
        const LevelPlan q = plan_level2_tile(B, L, s, pair_tile_target(w));
        const dim3 grid((unsigned)q.total);
        if (w == 64) {
            const dim3 blk(Tile2Shape<64>::NT);
            if (Ain.trans)
                hipLaunchKernelGGL((pcr_level2_tile<64, true>), grid, blk, 0, stream, Ain, rin,
                                   Aout, rout, L, q);
            else
                hipLaunchKernelGGL((pcr_level2_tile<64, false>), grid, blk, 0, stream, Ain, rin,
                                   Aout, rout, L, q);
        } else {
            const dim3 blk(Tile2Shape<128>::NT);
            if (Ain.trans)
                hipLaunchKernelGGL((pcr_level2_tile<128, true>), grid, blk, 0, stream, Ain, rin,
                                   Aout, rout, L, q);
            else
                hipLaunchKernelGGL((pcr_level2_tile<128, false>), grid, blk, 0, stream, Ain, rin,
                                   Aout, rout, L, q);
        }
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_pcr_level2_bwd(const BwdArgs& bw, const VecSrc& rin, float* Aout,
                                 const VecDst& rout, int B, int L, int w, hipStream_t stream) {
    const LevelPlan q = plan_level2_tile(B, L, 1, pair_tile_target(w));
    const dim3 grid((unsigned)q.total);
    const BlockSrc none{nullptr, 0, 0, 0};
    if (w == 32)
        hipLaunchKernelGGL((pcr_level2_tile<32, false, true>), grid, dim3(Tile2Shape<32>::NT), 0,
                           stream, none, rin, Aout, rout, L, q, bw);
    else if (w == 64)
        hipLaunchKernelGGL((pcr_level2_tile<64, false, true>), grid, dim3(Tile2Shape<64>::NT), 0,
                           stream, none, rin, Aout, rout, L, q, bw);
    else if (w == 128)
        hipLaunchKernelGGL((pcr_level2_tile<128, false, true>), grid, dim3(Tile2Shape<128>::NT),
                           0, stream, none, rin, Aout, rout, L, q, bw);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_pcr_level2_last(const BlockSrc& Ain, const VecSrc& rin, const VecDst& rout,
                                  int B, int L, int w, int s, hipStream_t stream) {
    const LevelPlan q = plan_level2_tile(B, L, s, w == 64 ? 4096 : 2048);
    const dim3 grid((unsigned)q.total);
    if (w == 64) {
        const dim3 blk(Tile2Shape<64>::NT);
        if (Ain.trans)
            hipLaunchKernelGGL((pcr_level2_tile_last<64, true>), grid, blk, 0, stream, Ain, rin,
                               rout, L, q);
        else
            hipLaunchKernelGGL((pcr_level2_tile_last<64, false>), grid, blk, 0, stream, Ain, rin,
                               rout, L, q);
    } else if (w == 128) {
        const dim3 blk(Tile2Shape<128>::NT);
        if (Ain.trans)
            hipLaunchKernelGGL((pcr_level2_tile_last<128, true>), grid, blk, 0, stream, Ain, rin,
                               rout, L, q);
        else
            hipLaunchKernelGGL((pcr_level2_tile_last<128, false>), grid, blk, 0, stream, Ain, rin,
                               rout, L, q);
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

bool last_pair_width(int w) { return w == 64 || w == 128; }

namespace {
int num_levels_of(int L) {
    int k = 0;
    for (long long s = 1; s < L; s *= 2) ++k;
    return k;
}
}  // namespace

int tail_levels(int B, int L, int w, int first) {
    if (!(w == 16 || w == 32 || w == 64 || w == 128) || !two_level(B, L, w)) return 0;
    const int K = num_levels_of(L);
    // the most levels (6 down to 3) such that the levels before the tail are
    // the first pass plus pairs, the tail reads operators written by this
    // solve (not the caller's possibly transposed blocks), and B s >= 256
    // chains keep every CU walking one (chains of at most 64 elements)
    const int kmin = first == 1 ? 1 : 2;
    for (int kt = 6; kt >= 3; --kt) {
        const int k0 = K - kt;
        if (k0 < kmin || k0 < first || ((k0 - first) & 1)) continue;
        if (((long long)B << k0) < 256) continue;
        return kt;
    }
    return 0;
}

bool fused_newton_levels(int w) { return w == 16 || w == 32; }

// The first two levels in one tile pass with the layers: w = 64, 128 where
// two_level pairs them; w = 32 from B L >= 2048 chain elements (below, the
// one-row segments of the wave kernel's first level keep more CUs busy: the
// batch-1 sweep measured the pair 4-20% slower up to L = 1024 and 10-15%
// faster from L = 2048).
int first_level_count(int B, int L, int w) {
    if (L <= 2 || !two_level(B, L, w)) return 1;
    if (w == 64 || w == 128) return 2;
    return w == 32 && (long long)B * L >= 2048 ? 2 : 1;
}
bool layer_first_level(int w) { return w == 16 || w == 32 || w == 64 || w == 128; }

hipError_t launch_first_level_fwd(const NewtonArgs& na, float* Aout, const VecDst& rout, int B,
                                  int L, int w, hipStream_t stream) {
    if (first_level_count(B, L, w) == 2) {
        const LevelPlan q = plan_level2_tile(B, L, 1, pair_tile_target(w, true));
        const dim3 grid((unsigned)q.total);
        if (w == 32)
            hipLaunchKernelGGL((pcr_level2_tile_layer<32>), grid, dim3(Tile2Shape<32>::NT), 0,
                               stream, Aout, rout, L, q, na);
        else if (w == 64)
            hipLaunchKernelGGL((pcr_level2_tile_layer<64>), grid, dim3(Tile2Shape<64>::NT), 0,
                               stream, Aout, rout, L, q, na);
        else
            hipLaunchKernelGGL((pcr_level2_tile_layer<128>), grid, dim3(Tile2Shape<128>::NT), 0,
                               stream, Aout, rout, L, q, na);
        return hipGetLastError();
    }
    if (w == 64 || w == 128) {
        const LevelPlan p = plan_level(B, L, 1, w == 64 ? 4096 : 1024, 64);
        const dim3 grid((unsigned)p.total),
            block(w == 64 ? TileShape<64>::NT : TileShape<128>::NT);
        if (w == 64)
            hipLaunchKernelGGL((pcr_level_tile_layer<64>), grid, block, 0, stream, Aout, rout, L,
                               p, na);
        else
            hipLaunchKernelGGL((pcr_level_tile_layer<128>), grid, block, 0, stream, Aout, rout, L,
                               p, na);
        return hipGetLastError();
    }
    const LevelPlan p = plan_level(B, L, 1, 8192, 64);
    const dim3 g3((unsigned)((p.total + 3) / 4)), block(256);
    const BlockSrc noA{nullptr, 0, 0, 0};
    const VecSrc nor{nullptr, 0, 0};
    if (w == 16)
        hipLaunchKernelGGL((pcr_level_wave<16, false, SRC_LAYER, false>), g3, block, 0, stream,
                           noA, nor, Aout, rout, L, p, na);
    else if (w == 32)
        hipLaunchKernelGGL((pcr_level_wave<32, false, SRC_LAYER, false>), g3, block, 0, stream,
                           noA, nor, Aout, rout, L, p, na);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_last_level_update(const BlockSrc& Ain, const VecSrc& rin, const NewtonArgs& na,
                                    int B, int L, int w, int s, hipStream_t stream) {
    const LevelPlan p = plan_level(B, L, s, 8192, 64);
    const dim3 g3((unsigned)((p.total + 3) / 4)), block(256);
    const VecDst noout{nullptr, 0, 0};
    if (Ain.trans) return hipErrorInvalidValue;
    if (w == 16)
        hipLaunchKernelGGL((pcr_level_wave<16, false, SRC_MEM, true>), g3, block, 0, stream, Ain,
                           rin, nullptr, noout, L, p, na);
    else if (w == 32)
        hipLaunchKernelGGL((pcr_level_wave<32, false, SRC_MEM, true>), g3, block, 0, stream, Ain,
                           rin, nullptr, noout, L, p, na);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace deeppcr
