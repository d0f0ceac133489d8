// The block-bidiagonal solve of Eq. 3 with its rows cut into consecutive
// chunks, the layout of a solve whose rows are spread over several devices
// (the memory and communication remarks of Sec. 3.1).  Three phases:
//
//   chunk-local PCR  Alg. 1 run inside every chunk independently, except that
//                    the chunk's first row keeps its coupling to the unknown
//                    x_in just outside the chunk: its operator is the block
//                    itself instead of zero.  A level with stride s reads the
//                    previous level and, for rows j >= s of the chunk (j the
//                    index inside the chunk),
//                      r_j <- r_j + A_j r_{j-s},   A_j <- A_j A_{j-s};
//                    rows j < s are final and copied.  After ceil(log2 Lc)
//                    levels every row holds x_l = P_l x_in + q_l
//                    (A_j = P_j, r_j = q_j).  The chunk holding row 0 has
//                    x_in = 0: it is ordinary PCR (operators only where
//                    later levels read them, i.e. rows j >= 2s).
//   carry            one pass over the chunk ends in order: x_in of the
//                    next chunk = P x_in + q at the current chunk's last row.
//   apply            x_l = q_l + P_l x_in of the row's chunk.
//
// Rows are in the solve's internal order m (the transposed system runs in
// reversed row order with the transposed blocks, as in the full solve), and
// chunks are defined on the natural rows: chunk g holds rows
// g Lc .. min(L, (g+1) Lc) - 1.
#include "internal.h"
#include "strip.h"

namespace deeppcr {
namespace {

constexpr int kThreads = 256;
constexpr int kKC = 16;
constexpr int kAccPerThread = kMaxWidth * kMaxWidth / kThreads;

// Chunk of internal row m: its index k in internal order and its first row ms.
struct ChunkPos {
    int k, ms;
};

__host__ __device__ inline int num_chunks(int L, int Lc) { return (L + Lc - 1) / Lc; }

// First internal row of the chunk with internal index k.
__host__ __device__ inline int chunk_start(int k, int L, int Lc, int rev) {
    if (!rev) return k * Lc;
    const int nch = num_chunks(L, Lc);
    const int hi = (nch - k) * Lc;  // natural end of natural chunk nch-1-k
    return L - (hi < L ? hi : L);
}

__device__ inline ChunkPos chunk_of(int m, int L, int Lc, int rev) {
    ChunkPos p;
    if (!rev) {
        p.k = m / Lc;
    } else {
        const int g = (L - 1 - m) / Lc;  // natural chunk
        p.k = num_chunks(L, Lc) - 1 - g;
    }
    p.ms = chunk_start(p.k, L, Lc, rev);
    return p;
}

__device__ inline float block_elem(const float* blk, int i, int k, int w, int trans) {
    return trans ? blk[(long long)k * w + i] : blk[(long long)i * w + k];
}

__device__ inline float wave_sum(float v) {
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// One chunk-local level, any w <= kMaxWidth: one workgroup per (system, row),
// float32 FMA on the vector ALUs with the product's operands staged through
// LDS in k-chunks.  Aout and rout are contiguous [B, L, w, w] / [B, L, w] in
// internal row order.
__global__ __launch_bounds__(kThreads) void chunk_level_generic(BlockSrc Ain, VecSrc rin,
                                                                float* __restrict__ Aout,
                                                                float* __restrict__ rout, int L,
                                                                int Lc, int rev, int w, int s) {
    const long long row = blockIdx.x;
    const int m = (int)(row % L);
    const int b = (int)(row / L);
    const int t = threadIdx.x;
    const ChunkPos cp = chunk_of(m, L, Lc, rev);
    const int j = m - cp.ms;
    const bool coupled = cp.k >= 1;
    const float* rl = rin.base + b * rin.bstride + (long long)m * rin.rstride;
    float* xo = rout + row * w;
    const float* Al = Ain.base + b * Ain.bstride + (long long)m * Ain.rstride;
    float* Ao = Aout + row * w * w;
    if (j < s) {  // final row: carried to the next level
        for (int i = t; i < w; i += kThreads) xo[i] = rl[i];
        if (coupled)
            for (int idx = t; idx < w * w; idx += kThreads) {
                const int i = idx / w, k = idx - (idx / w) * w;
                Ao[idx] = block_elem(Al, i, k, w, Ain.trans);
            }
        return;
    }

    __shared__ float rprev[kMaxWidth];
    __shared__ float Atile[kMaxWidth][kKC + 1];
    __shared__ float Ptile[kKC][kMaxWidth];
    const int lane = t & 63, wave = t >> 6;
    const float* rp = rin.base + b * rin.bstride + (long long)(m - s) * rin.rstride;
    for (int i = t; i < w; i += kThreads) rprev[i] = rp[i];
    __syncthreads();
    for (int i = wave; i < w; i += kThreads / 64) {
        float acc = 0.f;
        for (int k = lane; k < w; k += 64) acc = fmaf(block_elem(Al, i, k, w, Ain.trans), rprev[k], acc);
        acc = wave_sum(acc);
        if (lane == 0) xo[i] = rl[i] + acc;
    }
    if (!coupled && j < 2 * s) return;

    const float* Pl = Ain.base + b * Ain.bstride + (long long)(m - s) * Ain.rstride;
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
            const int kk = idx / w, jj = idx - (idx / w) * w;
            Ptile[kk][jj] = block_elem(Pl, kc + kk, jj, w, Ain.trans);
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < kAccPerThread; ++q) {
            const int idx = t + q * kThreads;
            if (idx < nout) {
                const int i = idx / w, jj = idx - (idx / w) * w;
                float a = acc[q];
                for (int kk = 0; kk < kw; ++kk) a = fmaf(Atile[i][kk], Ptile[kk][jj], a);
                acc[q] = a;
            }
        }
        __syncthreads();
    }
#pragma unroll
    for (int q = 0; q < kAccPerThread; ++q) {
        const int idx = t + q * kThreads;
        if (idx < nout) Ao[idx] = acc[q];
    }
}

// One chunk-local level at w <= 16: one wave per (system, row), four rows
// per workgroup, both blocks staged in the wave's own LDS area.
constexpr int kSmallW = 16;
constexpr int kSmallRows = kThreads / 64;

// WT > 0: the width as a compile-time constant (index arithmetic in shifts,
// inner loops unrolled); WT = 0 reads it at run time.
template <int WT>
__global__ __launch_bounds__(kThreads) void chunk_level_small(BlockSrc Ain, VecSrc rin,
                                                              float* __restrict__ Aout,
                                                              float* __restrict__ rout, int B,
                                                              int L, int Lc, int rev, int w_rt,
                                                              int s) {
    const int w = WT > 0 ? WT : w_rt;
    __shared__ float Am_all[kSmallRows][kSmallW][kSmallW + 1];
    __shared__ float Ap_all[kSmallRows][kSmallW][kSmallW + 1];
    __shared__ float rp_all[kSmallRows][kSmallW];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const long long row = (long long)blockIdx.x * kSmallRows + wave;
    if (row >= (long long)B * L) return;  // uniform over the wave
    const int m = (int)(row % L);
    const int b = (int)(row / L);
    const ChunkPos cp = chunk_of(m, L, Lc, rev);
    const int j = m - cp.ms;
    const bool coupled = cp.k >= 1;
    const float* rl = rin.base + b * rin.bstride + (long long)m * rin.rstride;
    float* xo = rout + row * w;
    const float* Al = Ain.base + b * Ain.bstride + (long long)m * Ain.rstride;
    float* Ao = Aout + row * w * w;
    const int n2 = w * w;
    if (j < s) {  // final row: carried to the next level
        if (lane < w) xo[lane] = rl[lane];
        if (coupled)
            for (int idx = lane; idx < n2; idx += 64) {
                const int u = idx / w, v = idx - (idx / w) * w;
                Ao[Ain.trans ? v * w + u : idx] = Al[idx];
            }
        return;
    }
    float (*Am)[kSmallW + 1] = Am_all[wave];
    float (*Ap)[kSmallW + 1] = Ap_all[wave];
    float* rp = rp_all[wave];
    const bool prod = coupled || j >= 2 * s;
    const float* Pl = Ain.base + b * Ain.bstride + (long long)(m - s) * Ain.rstride;
    // the blocks read in memory order (contiguous across the wave), each
    // entry placed at its (row, column) of the stored or transposed block
    for (int idx = lane; idx < n2; idx += 64) {
        const int u = idx / w, v = idx - (idx / w) * w;
        const int i = Ain.trans ? v : u, k = Ain.trans ? u : v;
        Am[i][k] = Al[idx];
        if (prod) Ap[i][k] = Pl[idx];
    }
    if (lane < w) rp[lane] = rin.base[b * rin.bstride + (long long)(m - s) * rin.rstride + lane];
    wave_sync();
    if (lane < w) {
        float acc = rl[lane];
        for (int k = 0; k < w; ++k) acc = fmaf(Am[lane][k], rp[k], acc);
        xo[lane] = acc;
    }
    if (!prod) return;
    for (int idx = lane; idx < n2; idx += 64) {
        const int i = idx / w, jj = idx - (idx / w) * w;
        float acc = 0.f;
        for (int k = 0; k < w; ++k) acc = fmaf(Am[i][k], Ap[k][jj], acc);
        Ao[idx] = acc;
    }
}

// One chunk-local level at w = 32, 64, 128 on fp32 MFMA: one workgroup per
// (system, row), one wave per 32-row strip.  The row's block A_j is the left
// operand in registers (read straight from memory); A_{j-s} goes through LDS
// transposed; the mat-vec A_j r_{j-s} rides on the product's operand reads.
template <int W, bool TRANS>
__global__ __launch_bounds__(Tile2Shape<W>::NT) void chunk_level_strip(BlockSrc Ain, VecSrc rin,
                                                                       float* __restrict__ Aout,
                                                                       float* __restrict__ rout,
                                                                       int L, int Lc, int rev,
                                                                       int s) {
    using S = Tile2Shape<W>;
    __shared__ float XT[W * S::PITCH];  // A_{j-s}, transposed
    __shared__ float rp[W];             // r_{j-s}
    const long long row = blockIdx.x;
    const int m = (int)(row % L);
    const int b = (int)(row / L);
    const int t = threadIdx.x;
    const int lane = t & 63, i = lane & 31, h = lane >> 5;
    const int R = 32 * (t >> 6) + i;
    const ChunkPos cp = chunk_of(m, L, Lc, rev);
    const int j = m - cp.ms;
    const bool coupled = cp.k >= 1;
    const float* ab = Ain.base + b * Ain.bstride;
    const float* rl = rin.base + b * rin.bstride + (long long)m * rin.rstride;
    float* xo = rout + row * W;
    float* Ao = Aout + row * W * W;
    StripA<W> a;
    if (j < s) {  // final row: carried to the next level
        if (t < W) xo[t] = rl[t];
        if (coupled) {
            strip_load<W, TRANS>(ab + (long long)m * Ain.rstride, a, R, h);
            strip_store<W>(Ao, a, R, h);
        }
        return;
    }
    const bool prod = coupled || j >= 2 * s;
    if (t < W) rp[t] = rin.base[b * rin.bstride + (long long)(m - s) * rin.rstride + t];
    if (prod) {
        StripA<W> x;
        strip_load<W, TRANS>(ab + (long long)(m - s) * Ain.rstride, x, R, h);
        strip_put_T<W>(XT, x, R, h);
    }
    strip_load<W, TRANS>(ab + (long long)m * Ain.rstride, a, R, h);
    __syncthreads();
    float part;
    if (prod) {
        StripC<W> acc;
        part = strip_product<W, 0, S::T, true>(XT, a, acc, i, h, rp);
        tiles_store<W, 0, S::T>(Ao, acc, R, h);
    } else {
        part = strip_matvec<W>(a, rp, h);
    }
    if (h == 0) xo[R] = rl[R] + part;
}

// ---- the chains of the last chunk-local levels, by substitution ---------
// After the chunk-local levels with strides below s, every row j >= s of a
// chunk satisfies x_j = A_j x_{j-s} + r_j, and rows j < s are final: maps
// x_j = P_j x_in + q_j of the chunk's carry-in in a coupled chunk, plain
// values in the chunk holding internal row 0.  Each chunk is then s
// independent chains (rows c, c + s, ... of the chunk, c < s), and walking a
// chain in order gives every row's map: P_j = A_j P_{j-s},
// q_j = A_j q_{j-s} + r_j (q only in the first chunk, whose carry-in is
// zero and whose P is never read).  The walk replaces the chunk's remaining
// levels the way the full solve's substitution pass replaces its last ones.
// (b, k, c) of a chain from its index, chunk k's first internal row ms, its
// length n; false for an empty chain (c beyond a short chunk).
struct ChainPos {
    int b, k, c, ms, n;
};

__device__ inline bool chain_of(long long chain, int L, int Lc, int rev, int s, ChainPos* p) {
    const int nch = num_chunks(L, Lc);
    p->c = (int)(chain % s);
    const long long bk = chain / s;
    p->k = (int)(bk % nch);
    p->b = (int)(bk / nch);
    p->ms = chunk_start(p->k, L, Lc, rev);
    p->n = (p->k + 1 < nch ? chunk_start(p->k + 1, L, Lc, rev) : L) - p->ms;
    return p->c < p->n;
}

// w <= 16: one wave per chain; the chain's previous map and the current
// block in the wave's LDS, the next block and right-hand side requested
// into registers while the current row is formed.
constexpr int kSmallPer = kSmallW * kSmallW / 64;  // block entries per lane
constexpr int kSmallAhead = 4;                       // rows requested ahead

template <int WT>
__global__ __launch_bounds__(kThreads) void chunk_chain_small(const float* __restrict__ Ain,
                                                              const float* __restrict__ rin,
                                                              float* __restrict__ Pout,
                                                              float* __restrict__ qout, int B,
                                                              int L, int Lc, int rev, int w_rt,
                                                              int s) {
    const int w = WT > 0 ? WT : w_rt;
    __shared__ float As_all[kSmallRows][kSmallW][kSmallW + 1];
    __shared__ float Pp_all[kSmallRows][kSmallW][kSmallW + 1];
    __shared__ float qp_all[kSmallRows][kSmallW];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const long long chain = (long long)blockIdx.x * kSmallRows + wave;
    if (chain >= (long long)B * num_chunks(L, Lc) * s) return;  // uniform over the wave
    ChainPos cp;
    if (!chain_of(chain, L, Lc, rev, s, &cp)) return;
    const bool coupled = cp.k >= 1;
    const int n2 = w * w;
    const int count = (cp.n - 1 - cp.c) / s;
    float (*As)[kSmallW + 1] = As_all[wave];
    float (*Pp)[kSmallW + 1] = Pp_all[wave];
    float* qp = qp_all[wave];
    long long row = (long long)cp.b * L + cp.ms + cp.c;
    // element 0: final; its map is the chain's first
    if (lane < w) {
        const float v = rin[row * w + lane];
        qout[row * w + lane] = v;
        qp[lane] = v;
    }
    if (coupled)
        for (int idx = lane; idx < n2; idx += 64) {
            const float v = Ain[row * n2 + idx];
            Pout[row * n2 + idx] = v;
            Pp[idx / w][idx - (idx / w) * w] = v;
        }
    // a ring of kSmallAhead rows in flight: element t uses slot (t - 1) % D
    constexpr int D = kSmallAhead;
    float an[D][kSmallPer], rn[D];
    auto request = [&](int slot, long long rw) {
#pragma unroll
        for (int p = 0; p < kSmallPer; ++p) {
            const int idx = lane + 64 * p;
            an[slot][p] = idx < n2 ? Ain[rw * n2 + idx] : 0.f;
        }
        rn[slot] = lane < w ? rin[rw * w + lane] : 0.f;
    };
#pragma unroll
    for (int j = 0; j < D; ++j)
        if (1 + j <= count) request(j, row + (long long)(1 + j) * s);
    for (int t0 = 1; t0 <= count; t0 += D) {
#pragma unroll
    for (int j = 0; j < D; ++j) {
        const int t = t0 + j;
        if (t > count) break;  // uniform over the wave
        row += s;
#pragma unroll
        for (int p = 0; p < kSmallPer; ++p) {
            const int idx = lane + 64 * p;
            if (idx < n2) As[idx / w][idx - (idx / w) * w] = an[j][p];
        }
        const float rc = rn[j];
        if (t + D <= count) request(j, row + (long long)D * s);
        wave_sync();
        float qn = 0.f;
        if (lane < w) {
            qn = rc;
            for (int kk = 0; kk < w; ++kk) qn = fmaf(As[lane][kk], qp[kk], qn);
        }
        float pn[kSmallPer];
        if (coupled) {
#pragma unroll
            for (int p = 0; p < kSmallPer; ++p) {
                const int idx = lane + 64 * p;
                float acc = 0.f;
                if (idx < n2) {
                    const int i = idx / w, jj = idx - (idx / w) * w;
                    for (int kk = 0; kk < w; ++kk) acc = fmaf(As[i][kk], Pp[kk][jj], acc);
                }
                pn[p] = acc;
            }
        }
        wave_sync();  // every lane has read As, Pp and qp
        if (lane < w) {
            qp[lane] = qn;
            qout[row * w + lane] = qn;
        }
        if (coupled) {
#pragma unroll
            for (int p = 0; p < kSmallPer; ++p) {
                const int idx = lane + 64 * p;
                if (idx < n2) {
                    Pp[idx / w][idx - (idx / w) * w] = pn[p];
                    Pout[row * n2 + idx] = pn[p];
                }
            }
        }
        wave_sync();
    }
    }
}

// w = 32, 64, 128: one workgroup per chain, one wave per 32-row strip.  The
// row's block is the left MFMA operand in registers (the next one requested
// before the current product), the chain's previous map goes through LDS
// transposed, and q_{j-s} rides on the product's operand reads.
template <int W>
__global__ __launch_bounds__(Tile2Shape<W>::NT) void chunk_chain_strip(
    const float* __restrict__ Ain, const float* __restrict__ rin, float* __restrict__ Pout,
    float* __restrict__ qout, int L, int Lc, int rev, int s) {
    using S = Tile2Shape<W>;
    __shared__ float XT[W * S::PITCH];  // P of the chain's previous row, transposed
    __shared__ float qp[W];
    const int t = threadIdx.x;
    const int lane = t & 63, i = lane & 31, h = lane >> 5;
    const int R = 32 * (t >> 6) + i;
    ChainPos cp;
    if (!chain_of(blockIdx.x, L, Lc, rev, s, &cp)) return;  // uniform over the workgroup
    const bool coupled = cp.k >= 1;
    const long long w2 = (long long)W * W;
    const int count = (cp.n - 1 - cp.c) / s;
    long long row = (long long)cp.b * L + cp.ms + cp.c;
    // a ring of D rows in flight: element tt uses slot (tt - 1) % D
    constexpr int D = W == 128 ? 1 : W == 64 ? 2 : 4;
    StripA<W> a, an[D];
    float rn[D];
    if (t < W) {
        const float v = rin[row * W + t];
        qout[row * W + t] = v;
        qp[t] = v;
    }
    if (coupled) {
        strip_load<W, false>(Ain + row * w2, a, R, h);
        strip_store<W>(Pout + row * w2, a, R, h);
        strip_put_T<W>(XT, a, R, h);
    }
    auto request = [&](int slot, long long rw) {
        strip_load<W, false>(Ain + rw * w2, an[slot], R, h);
        rn[slot] = rin[rw * W + R];
    };
#pragma unroll
    for (int j = 0; j < D; ++j)
        if (1 + j <= count) request(j, row + (long long)(1 + j) * s);
    __syncthreads();
    for (int t0 = 1; t0 <= count; t0 += D) {
#pragma unroll
    for (int j = 0; j < D; ++j) {
        const int tt = t0 + j;
        if (tt > count) break;  // uniform over the workgroup
        row += s;
#pragma unroll
        for (int q = 0; q < S::NQ; ++q) a[q] = an[j][q];
        const float rc = rn[j];
        if (tt + D <= count) request(j, row + (long long)D * s);
        StripC<W> acc;
        float part;
        if (coupled)
            part = strip_product<W, 0, S::T, true>(XT, a, acc, i, h, qp);
        else
            part = strip_matvec<W>(a, qp, h);
        const float qn = rc + part;
        __syncthreads();  // XT and qp are read
        if (h == 0) {
            qp[R] = qn;
            qout[row * W + R] = qn;
        }
        if (coupled) {
            tiles_store<W, 0, S::T>(Pout + row * w2, acc, R, h);
            strip_put_T<W>(XT, acc, R, h);
        }
        __syncthreads();
    }
    }
}

// Carry pass, one workgroup per system: in internal chunk order,
// xin[b, k] = carry; carry <- P_e carry + q_e at the chunk's last row e
// (P_e of the first chunk is not read: its carry-in is zero).  At w <= 16
// the next chunk's P_e and q_e (one entry per thread) are requested into
// registers before the current chunk's product and staged in LDS after it.
__device__ inline int chunk_end(int k, int nch, int L, int Lc, int rev) {
    return (k + 1 < nch ? chunk_start(k + 1, L, Lc, rev) : L) - 1;
}

__global__ __launch_bounds__(kThreads) void chunk_carry_kernel(const float* __restrict__ P,
                                                               const float* __restrict__ q,
                                                               float* __restrict__ xin, int L,
                                                               int Lc, int rev, int w) {
    const int b = blockIdx.x;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int nch = num_chunks(L, Lc);
    __shared__ float c[kMaxWidth], cn[kMaxWidth];
    for (int i = t; i < w; i += kThreads) c[i] = 0.f;
    if (w <= kSmallW) {
        __shared__ float Ps[kSmallW * kSmallW], qs[kSmallW];
        const int n2 = w * w;
        float pv = 0.f, qv = 0.f;
        auto request = [&](int k) {
            const long long e = (long long)b * L + chunk_end(k, nch, L, Lc, rev);
            pv = (k >= 1 && t < n2) ? P[e * n2 + t] : 0.f;
            qv = t < w ? q[e * w + t] : 0.f;
        };
        request(0);
        for (int k = 0; k < nch; ++k) {
            if (t < n2) Ps[t] = pv;
            if (t < w) qs[t] = qv;
            if (k + 1 < nch) request(k + 1);
            __syncthreads();
            if (t < w) {
                xin[((long long)b * nch + k) * w + t] = c[t];
                float acc = qs[t];
                for (int j = 0; j < w; ++j) acc = fmaf(Ps[t * w + j], c[j], acc);
                cn[t] = acc;
            }
            __syncthreads();
            if (t < w) c[t] = cn[t];
        }
        return;
    }
    __syncthreads();
    for (int k = 0; k < nch; ++k) {
        for (int i = t; i < w; i += kThreads) xin[((long long)b * nch + k) * w + i] = c[i];
        const long long e = (long long)b * L + chunk_end(k, nch, L, Lc, rev);
        const float* Pe = P + e * w * w;
        const float* qe = q + e * w;
        for (int ii = wave; ii < w; ii += kThreads / 64) {
            float acc = 0.f;
            if (k >= 1)
                for (int jj = lane; jj < w; jj += 64) acc = fmaf(Pe[(long long)ii * w + jj], c[jj], acc);
            acc = wave_sum(acc);
            if (lane == 0) cn[ii] = acc + qe[ii];
        }
        __syncthreads();
        for (int i = t; i < w; i += kThreads) c[i] = cn[i];
        __syncthreads();
    }
}

// Carry and apply at w = 32, 64, 128: thread t takes row t / TPR of a block
// and TPR-th of its columns (float4 reads along the row), partial dot
// products summed over the row's TPR lanes by DPP.
template <int W>
struct RowSplit {
    static constexpr int TPR = kThreads / W;  // threads per block row
    static constexpr int CPT = W / TPR;       // columns per thread
    static constexpr int NV = CPT / 4;        // float4 per thread
};

template <int W>
__device__ __forceinline__ float row_dot(const float* prow, const float* v) {
    float acc = 0.f;
#pragma unroll
    for (int u = 0; u < RowSplit<W>::NV; ++u) {
        const v4f a = *reinterpret_cast<const v4f*>(prow + 4 * u);
        const v4f c = *reinterpret_cast<const v4f*>(v + 4 * u);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc = fmaf(a[e], c[e], acc);
    }
    return acc;
}

// The carry at w = 32, 64, 128, one workgroup per system; the next
// chunk's P_e entries of a thread are requested before the current product.
template <int W>
__global__ __launch_bounds__(kThreads) void chunk_carry_rows(const float* __restrict__ P,
                                                             const float* __restrict__ q,
                                                             float* __restrict__ xin, int L,
                                                             int Lc, int rev) {
    using S = RowSplit<W>;
    const int b = blockIdx.x;
    const int t = threadIdx.x, i = t / S::TPR, p = t % S::TPR;
    const int nch = num_chunks(L, Lc);
    __shared__ float c[2][W];
    if (t < W) c[0][t] = 0.f;
    v4f pe[S::NV];
    float qe = 0.f;
    auto request = [&](int k) {
        const long long e = (long long)b * L + chunk_end(k, nch, L, Lc, rev);
        const float* pr = P + (e * W + i) * W + p * S::CPT;
#pragma unroll
        for (int u = 0; u < S::NV; ++u)
            pe[u] = k >= 1 ? *reinterpret_cast<const v4f*>(pr + 4 * u) : v4f{0.f, 0.f, 0.f, 0.f};
        qe = q[e * W + i];
    };
    request(0);
    __syncthreads();
    for (int k = 0; k < nch; ++k) {
        const float* cc = c[k & 1];
        if (t < W) xin[((long long)b * nch + k) * W + t] = cc[t];
        v4f pc[S::NV];
#pragma unroll
        for (int u = 0; u < S::NV; ++u) pc[u] = pe[u];
        const float qc = qe;
        if (k + 1 < nch) request(k + 1);
        float acc = 0.f;
#pragma unroll
        for (int u = 0; u < S::NV; ++u) {
            const v4f cv = *reinterpret_cast<const v4f*>(cc + p * S::CPT + 4 * u);
#pragma unroll
            for (int e = 0; e < 4; ++e) acc = fmaf(pc[u][e], cv[e], acc);
        }
        acc = row_sum<S::TPR>(acc);
        if (p == 0) c[(k + 1) & 1][i] = qc + acc;
        __syncthreads();
    }
}

// The apply at w = 32, 64, 128: one workgroup per row of the system.
template <int W>
__global__ __launch_bounds__(kThreads) void chunk_apply_rows(const float* __restrict__ P,
                                                             const float* __restrict__ q,
                                                             const float* __restrict__ xin,
                                                             VecDst x, int L, int Lc, int rev) {
    using S = RowSplit<W>;
    const long long row = blockIdx.x;
    const int m = (int)(row % L);
    const int b = (int)(row / L);
    const int t = threadIdx.x, i = t / S::TPR, p = t % S::TPR;
    const ChunkPos cp = chunk_of(m, L, Lc, rev);
    float* xo = x.base + b * x.bstride + (long long)m * x.rstride;
    if (cp.k == 0) {  // uniform over the workgroup
        if (t < W) xo[t] = q[row * W + t];
        return;
    }
    const float* c = xin + ((long long)b * num_chunks(L, Lc) + cp.k) * W + p * S::CPT;
    const float acc = row_sum<S::TPR>(row_dot<W>(P + (row * W + i) * W + p * S::CPT, c));
    if (p == 0) xo[i] = q[row * W + i] + acc;
}

// x at internal row m: q_m + P_m xin[chunk of m] (just q_m in the first
// chunk), written through the natural-order destination.
__global__ __launch_bounds__(kThreads) void chunk_apply_kernel(const float* __restrict__ P,
                                                               const float* __restrict__ q,
                                                               const float* __restrict__ xin,
                                                               VecDst x, int L, int Lc, int rev,
                                                               int w) {
    const long long row = blockIdx.x;
    const int m = (int)(row % L);
    const int b = (int)(row / L);
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const ChunkPos cp = chunk_of(m, L, Lc, rev);
    const float* qm = q + row * w;
    float* xo = x.base + b * x.bstride + (long long)m * x.rstride;
    if (cp.k == 0) {
        for (int i = t; i < w; i += kThreads) xo[i] = qm[i];
        return;
    }
    __shared__ float c[kMaxWidth];
    const int nch = num_chunks(L, Lc);
    for (int i = t; i < w; i += kThreads) c[i] = xin[((long long)b * nch + cp.k) * w + i];
    __syncthreads();
    const float* Pm = P + row * w * w;
    for (int ii = wave; ii < w; ii += kThreads / 64) {
        float acc = 0.f;
        for (int jj = lane; jj < w; jj += 64) acc = fmaf(Pm[(long long)ii * w + jj], c[jj], acc);
        acc = wave_sum(acc);
        if (lane == 0) xo[ii] = qm[ii] + acc;
    }
}

// The apply at w <= 16: sixteen lanes per row (four rows per wave), lane i
// forms output i from row i of P_m.
template <int WT>
__global__ __launch_bounds__(kThreads) void chunk_apply_small(const float* __restrict__ P,
                                                              const float* __restrict__ q,
                                                              const float* __restrict__ xin,
                                                              VecDst x, int B, int L, int Lc,
                                                              int rev, int w_rt) {
    const int w = WT > 0 ? WT : w_rt;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const long long row = ((long long)blockIdx.x * kSmallRows + wave) * 4 + lane / 16;
    const int i = lane & 15;
    if (row >= (long long)B * L || i >= w) return;
    const int m = (int)(row % L);
    const int b = (int)(row / L);
    const ChunkPos cp = chunk_of(m, L, Lc, rev);
    float acc = q[row * w + i];
    if (cp.k >= 1) {
        const float* c = xin + ((long long)b * num_chunks(L, Lc) + cp.k) * w;
        const float* Pm = P + row * w * w + (long long)i * w;
        for (int k = 0; k < w; ++k) acc = fmaf(Pm[k], c[k], acc);
    }
    x.base[b * x.bstride + (long long)m * x.rstride + i] = acc;
}

}  // namespace

int chunk_count(int L, int Lc) { return num_chunks(L, Lc); }

void chunk_level_work(int B, int L, int w, int Lc, int rev, int s, double* bytes,
                      double* flops) {
    double nmv = 0, npr = 0, ncp = 0;
    const int nch = num_chunks(L, Lc);
    for (int k = 0; k < nch; ++k) {
        const int n = (k + 1 < nch ? chunk_start(k + 1, L, Lc, rev) : L) - chunk_start(k, L, Lc, rev);
        const int lag = k >= 1 ? s : 2 * s;  // rows from which operators are formed
        nmv += n > s ? n - s : 0;
        npr += n > lag ? n - lag : 0;
        if (k >= 1) ncp += n < s ? n : s;
    }
    const double w2 = (double)w * w;
    *bytes = 4.0 * B * (nmv * w2 + npr * w2 + 2.0 * ncp * w2 + 2.0 * L * w);
    *flops = (double)B * (nmv * 2.0 * w2 + npr * 2.0 * w2 * w);
}

hipError_t launch_chunk_level(const BlockSrc& Ain, const VecSrc& rin, float* Aout, float* rout,
                              int B, int L, int w, int Lc, int rev, int s, hipStream_t stream) {
    const dim3 grid((unsigned)((long long)B * L));
    const bool trans = Ain.trans != 0;
#define DEEPPCR_CHUNK_STRIP(WW)                                                                \
    if (w == WW) {                                                                             \
        if (trans)                                                                             \
            chunk_level_strip<WW, true><<<grid, Tile2Shape<WW>::NT, 0, stream>>>(              \
                Ain, rin, Aout, rout, L, Lc, rev, s);                                          \
        else                                                                                   \
            chunk_level_strip<WW, false><<<grid, Tile2Shape<WW>::NT, 0, stream>>>(             \
                Ain, rin, Aout, rout, L, Lc, rev, s);                                          \
        return hipGetLastError();                                                              \
    }
    DEEPPCR_CHUNK_STRIP(32)
    DEEPPCR_CHUNK_STRIP(64)
    DEEPPCR_CHUNK_STRIP(128)
#undef DEEPPCR_CHUNK_STRIP
    if (w <= kSmallW) {
        const long long nwg = ((long long)B * L + kSmallRows - 1) / kSmallRows;
#define DEEPPCR_LEVEL_SMALL(WT)                                                           \
    chunk_level_small<WT><<<dim3((unsigned)nwg), kThreads, 0, stream>>>(Ain, rin, Aout, rout, \
                                                                       B, L, Lc, rev, w, s)
        switch (w) {
            case 4: DEEPPCR_LEVEL_SMALL(4); break;
            case 8: DEEPPCR_LEVEL_SMALL(8); break;
            case 16: DEEPPCR_LEVEL_SMALL(16); break;
            default: DEEPPCR_LEVEL_SMALL(0); break;
        }
#undef DEEPPCR_LEVEL_SMALL
        return hipGetLastError();
    }
    chunk_level_generic<<<grid, kThreads, 0, stream>>>(Ain, rin, Aout, rout, L, Lc, rev, w, s);
    return hipGetLastError();
}

bool chunk_chain_width(int w) { return w <= kSmallW || w == 32 || w == 64 || w == 128; }

void chunk_chain_work(int B, int L, int w, int Lc, int rev, int s, double* bytes,
                      double* flops) {
    // every row's block and right-hand side read, its map written; the rows
    // past the chains' first (rows j >= s) form one product and one mat-vec
    double rows_c = 0, rows_u = 0, fin_c = 0;
    const int nch = num_chunks(L, Lc);
    for (int k = 0; k < nch; ++k) {
        const int n = (k + 1 < nch ? chunk_start(k + 1, L, Lc, rev) : L) - chunk_start(k, L, Lc, rev);
        const int past = n > s ? n - s : 0;
        if (k >= 1) {
            rows_c += past;
            fin_c += n - past;
        } else {
            rows_u += past;
        }
    }
    const double w2 = (double)w * w;
    *bytes = 4.0 * B * (2.0 * (rows_c + fin_c) * w2 + rows_u * w2 + 2.0 * L * w);
    *flops = (double)B * (rows_c * (2.0 * w2 * w + 2.0 * w2) + rows_u * 2.0 * w2);
}

hipError_t launch_chunk_chain(const float* Ain, const float* rin, float* Pout, float* qout,
                              int B, int L, int w, int Lc, int rev, int s, hipStream_t stream) {
    const long long chains = (long long)B * num_chunks(L, Lc) * s;
#define DEEPPCR_CHUNK_CHAIN(WW)                                                              \
    if (w == WW) {                                                                           \
        chunk_chain_strip<WW><<<dim3((unsigned)chains), Tile2Shape<WW>::NT, 0, stream>>>(    \
            Ain, rin, Pout, qout, L, Lc, rev, s);                                            \
        return hipGetLastError();                                                            \
    }
    DEEPPCR_CHUNK_CHAIN(32)
    DEEPPCR_CHUNK_CHAIN(64)
    DEEPPCR_CHUNK_CHAIN(128)
#undef DEEPPCR_CHUNK_CHAIN
    if (w > kSmallW) return hipErrorInvalidValue;
    const long long nwg = (chains + kSmallRows - 1) / kSmallRows;
#define DEEPPCR_CHAIN_SMALL(WT)                                                             \
    chunk_chain_small<WT><<<dim3((unsigned)nwg), kThreads, 0, stream>>>(Ain, rin, Pout, qout, B, \
                                                                       L, Lc, rev, w, s)
    switch (w) {
        case 4: DEEPPCR_CHAIN_SMALL(4); break;
        case 8: DEEPPCR_CHAIN_SMALL(8); break;
        case 16: DEEPPCR_CHAIN_SMALL(16); break;
        default: DEEPPCR_CHAIN_SMALL(0); break;
    }
#undef DEEPPCR_CHAIN_SMALL
    return hipGetLastError();
}

hipError_t launch_chunk_carry(const float* P, const float* q, float* xin, int B, int L, int w,
                              int Lc, int rev, hipStream_t stream) {
#define DEEPPCR_CARRY_ROWS(WW)                                                                 \
    if (w == WW) {                                                                             \
        chunk_carry_rows<WW><<<B, kThreads, 0, stream>>>(P, q, xin, L, Lc, rev);               \
        return hipGetLastError();                                                              \
    }
    DEEPPCR_CARRY_ROWS(32)
    DEEPPCR_CARRY_ROWS(64)
    DEEPPCR_CARRY_ROWS(128)
#undef DEEPPCR_CARRY_ROWS
    chunk_carry_kernel<<<B, kThreads, 0, stream>>>(P, q, xin, L, Lc, rev, w);
    return hipGetLastError();
}

hipError_t launch_chunk_apply(const float* P, const float* q, const float* xin, const VecDst& x,
                              int B, int L, int w, int Lc, int rev, hipStream_t stream) {
    if (w <= kSmallW) {
        const long long rows_per_wg = 4LL * kSmallRows;
        const long long nwg = ((long long)B * L + rows_per_wg - 1) / rows_per_wg;
        if (w == 16)
            chunk_apply_small<16><<<dim3((unsigned)nwg), kThreads, 0, stream>>>(P, q, xin, x, B, L,
                                                                               Lc, rev, w);
        else
            chunk_apply_small<0><<<dim3((unsigned)nwg), kThreads, 0, stream>>>(P, q, xin, x, B, L,
                                                                              Lc, rev, w);
        return hipGetLastError();
    }
    const dim3 grid((unsigned)((long long)B * L));
#define DEEPPCR_APPLY_ROWS(WW)                                                                 \
    if (w == WW) {                                                                             \
        chunk_apply_rows<WW><<<grid, kThreads, 0, stream>>>(P, q, xin, x, L, Lc, rev);         \
        return hipGetLastError();                                                              \
    }
    DEEPPCR_APPLY_ROWS(32)
    DEEPPCR_APPLY_ROWS(64)
    DEEPPCR_APPLY_ROWS(128)
#undef DEEPPCR_APPLY_ROWS
    chunk_apply_kernel<<<grid, kThreads, 0, stream>>>(P, q, xin, x, L, Lc, rev, w);
    return hipGetLastError();
}

}  // namespace deeppcr
