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

__global__ __launch_bounds__(kThreads) void chunk_level_small(BlockSrc Ain, VecSrc rin,
                                                              float* __restrict__ Aout,
                                                              float* __restrict__ rout, int B,
                                                              int L, int Lc, int rev, int w,
                                                              int s) {
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
                const int i = idx / w, k = idx - (idx / w) * w;
                Ao[idx] = block_elem(Al, i, k, w, Ain.trans);
            }
        return;
    }
    float (*Am)[kSmallW + 1] = Am_all[wave];
    float (*Ap)[kSmallW + 1] = Ap_all[wave];
    float* rp = rp_all[wave];
    const bool prod = coupled || j >= 2 * s;
    const float* Pl = Ain.base + b * Ain.bstride + (long long)(m - s) * Ain.rstride;
    for (int idx = lane; idx < n2; idx += 64) {
        const int i = idx / w, k = idx - (idx / w) * w;
        Am[i][k] = block_elem(Al, i, k, w, Ain.trans);
        if (prod) Ap[i][k] = block_elem(Pl, i, k, w, Ain.trans);
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

// Carry pass, one workgroup per system: in internal chunk order,
// xin[b, k] = carry; carry <- P_e carry + q_e at the chunk's last row e
// (P_e of the first chunk is not read: its carry-in is zero).
__global__ __launch_bounds__(kThreads) void chunk_carry_kernel(const float* __restrict__ P,
                                                               const float* __restrict__ q,
                                                               float* __restrict__ xin, int L,
                                                               int Lc, int rev, int w) {
    const int b = blockIdx.x;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int nch = num_chunks(L, Lc);
    __shared__ float c[kMaxWidth], cn[kMaxWidth];
    for (int i = t; i < w; i += kThreads) c[i] = 0.f;
    __syncthreads();
    for (int k = 0; k < nch; ++k) {
        for (int i = t; i < w; i += kThreads) xin[((long long)b * nch + k) * w + i] = c[i];
        const int e = (k + 1 < nch ? chunk_start(k + 1, L, Lc, rev) : L) - 1;
        const float* Pe = P + ((long long)b * L + e) * w * w;
        const float* qe = q + ((long long)b * L + e) * w;
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

// The apply at w <= 16: one wave per row, lane i forms output i.
__global__ __launch_bounds__(kThreads) void chunk_apply_small(const float* __restrict__ P,
                                                              const float* __restrict__ q,
                                                              const float* __restrict__ xin,
                                                              VecDst x, int B, int L, int Lc,
                                                              int rev, int w) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const long long row = (long long)blockIdx.x * kSmallRows + wave;
    if (row >= (long long)B * L || lane >= w) return;
    const int m = (int)(row % L);
    const int b = (int)(row / L);
    const ChunkPos cp = chunk_of(m, L, Lc, rev);
    float acc = q[row * w + lane];
    if (cp.k >= 1) {
        const float* c = xin + ((long long)b * num_chunks(L, Lc) + cp.k) * w;
        const float* Pm = P + row * w * w + (long long)lane * w;
        for (int k = 0; k < w; ++k) acc = fmaf(Pm[k], c[k], acc);
    }
    x.base[b * x.bstride + (long long)m * x.rstride + lane] = acc;
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
        chunk_level_small<<<dim3((unsigned)nwg), kThreads, 0, stream>>>(Ain, rin, Aout, rout, B,
                                                                       L, Lc, rev, w, s);
        return hipGetLastError();
    }
    chunk_level_generic<<<grid, kThreads, 0, stream>>>(Ain, rin, Aout, rout, L, Lc, rev, w, s);
    return hipGetLastError();
}

hipError_t launch_chunk_carry(const float* P, const float* q, float* xin, int B, int L, int w,
                              int Lc, int rev, hipStream_t stream) {
    chunk_carry_kernel<<<B, kThreads, 0, stream>>>(P, q, xin, L, Lc, rev, w);
    return hipGetLastError();
}

hipError_t launch_chunk_apply(const float* P, const float* q, const float* xin, const VecDst& x,
                              int B, int L, int w, int Lc, int rev, hipStream_t stream) {
    if (w <= kSmallW) {
        const long long nwg = ((long long)B * L + kSmallRows - 1) / kSmallRows;
        chunk_apply_small<<<dim3((unsigned)nwg), kThreads, 0, stream>>>(P, q, xin, x, B, L, Lc,
                                                                       rev, w);
        return hipGetLastError();
    }
    const dim3 grid((unsigned)((long long)B * L));
    chunk_apply_kernel<<<grid, kThreads, 0, stream>>>(P, q, xin, x, L, Lc, rev, w);
    return hipGetLastError();
}

}  // namespace deeppcr
