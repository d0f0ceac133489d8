// Widths 129 .. 1024: the PCR level, the layer and Jacobian evaluation of
// the forward and backward passes, the parameter gradients and the
// sequential passes, for blocks too large for the one-workgroup-per-block
// kernels of the smaller widths.
//
// PCR level (Sec. 3, Alg. 1, with A = +J as in Eq. 4), stride s:
//   rows l <  s : r_l copied                          (pcr_wide_rows)
//   rows l >= s : r_l <- r_l + A_l r_{l-s}           (pcr_wide_rows for
//                 l < 2s, the product kernel's first column tiles for l >= 2s)
//   rows l >= 2s: A_l <- A_l A_{l-s}                 (pcr_wide_prod)
// At these widths the block product is a real matrix product (2 w^3 flops on
// 12 w^2 bytes: 43 flop/B at w = 256, above the fp32 MFMA ridge), so each
// product is tiled into 128 x 128 output tiles, one workgroup per tile, k in
// chunks of 16 double-buffered through LDS (the next chunk stored part by part
// beside the current chunk's products), three workgroups per CU, on
// v_mfma_f32_32x32x2_f32.
// Workgroups are dispatched round-robin over the 8 XCDs; the tile index is
// remapped so that the tiles of one product run on one XCD (its L2 then
// serves the row and column panels the tiles share).
#include "internal.h"

namespace deeppcr {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kWide = kMaxWideWidth;  // 1024
constexpr int kTile = 128;            // output tile of the block product
constexpr int kKC = 16;               // k chunk
constexpr int kFpr = kKC / 4;         // float4 per row of a k chunk
constexpr int kNp = kTile * kKC / (4 * 256);  // float4 per thread per tile chunk
constexpr int kPitch = kKC + 4;       // LDS row pitch (conflict-free 16-byte reads)
constexpr int kXcds = 8;

__device__ inline float wave_sum(float v) {
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__device__ inline unsigned wave_umax(unsigned v) {
    for (int off = 32; off > 0; off >>= 1) v = max(v, (unsigned)__shfl_xor((int)v, off, 64));
    return v;
}

// ------------------------------------------------------------ row helpers
// A row of w <= 1024 floats held by one wave, 16 values per lane.
// VEC (w % 4 == 0): lane holds columns 4 lane + 256 p .. +3, p = 0..3;
// otherwise columns lane + 64 p, p = 0..15.
template <bool VEC>
__device__ inline int row_col(int lane, int idx) {
    return VEC ? 4 * lane + 256 * (idx >> 2) + (idx & 3) : lane + 64 * idx;
}

template <bool VEC>
__device__ inline void row_load(const float* __restrict__ row, int w, float (&v)[16], int lane) {
    if constexpr (VEC) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const int c = 4 * lane + 256 * p;
            v4f x = c < w ? *reinterpret_cast<const v4f*>(row + c) : v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int e = 0; e < 4; ++e) v[4 * p + e] = x[e];
        }
    } else {
#pragma unroll
        for (int p = 0; p < 16; ++p) {
            const int c = lane + 64 * p;
            v[p] = c < w ? row[c] : 0.f;
        }
    }
}

// sum over the row of v * z (z in LDS, zero beyond w); every lane gets it
template <bool VEC>
__device__ inline float row_dot(const float (&v)[16], const float* z, int lane) {
    float acc = 0.f;
#pragma unroll
    for (int idx = 0; idx < 16; ++idx) acc = fmaf(v[idx], z[row_col<VEC>(lane, idx)], acc);
    return wave_sum(acc);
}

// dst[col] = c * v[col] (+ 1 at column diag, if diag >= 0)
template <bool VEC>
__device__ inline void row_store_scaled(float* __restrict__ dst, int w, const float (&v)[16],
                                        float c, int diag, int lane) {
    if constexpr (VEC) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const int c0 = 4 * lane + 256 * p;
            if (c0 < w) {
                v4f x;
#pragma unroll
                for (int e = 0; e < 4; ++e) x[e] = c * v[4 * p + e] + (c0 + e == diag ? 1.f : 0.f);
                *reinterpret_cast<v4f*>(dst + c0) = x;
            }
        }
    } else {
#pragma unroll
        for (int p = 0; p < 16; ++p) {
            const int col = lane + 64 * p;
            if (col < w) dst[col] = c * v[p] + (col == diag ? 1.f : 0.f);
        }
    }
}

// z[0 .. kWide) = src[0 .. w), zero beyond
__device__ inline void stage_vec(float* z, const float* __restrict__ src, int w) {
    for (int i = threadIdx.x; i < kWide; i += kThreads) z[i] = i < w ? src[i] : 0.f;
}

// ---------------------------------------------------------- PCR level
// A kTile x kKC tile of a logical w x w block into registers: element (r, c)
// is L(r0 + r, c0 + c) with L(i, k) = blk[i w + k], or blk[k w + i] when TR.
// Zero outside the block.  256 threads, four float4 each.
template <bool VEC, bool TR>
__device__ inline void tile_load(const float* __restrict__ blk, int w, int r0, int c0,
                                 v4f (&reg)[kNp]) {
    const int t = threadIdx.x;
#pragma unroll
    for (int p = 0; p < kNp; ++p) {
        const int f = t + kThreads * p;
        if constexpr (!TR) {
            const int r = r0 + f / kFpr, c = c0 + 4 * (f % kFpr);
            if constexpr (VEC) {
                reg[p] = (r < w && c < w) ? *reinterpret_cast<const v4f*>(blk + (long long)r * w + c)
                                          : v4f{0.f, 0.f, 0.f, 0.f};
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    reg[p][e] = (r < w && c + e < w) ? blk[(long long)r * w + c + e] : 0.f;
            }
        } else {
            const int c = c0 + (f >> 5), r = r0 + 4 * (f & 31);
            if constexpr (VEC) {
                reg[p] = (r < w && c < w) ? *reinterpret_cast<const v4f*>(blk + (long long)c * w + r)
                                          : v4f{0.f, 0.f, 0.f, 0.f};
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    reg[p][e] = (r + e < w && c < w) ? blk[(long long)c * w + r + e] : 0.f;
            }
        }
    }
}

// Part p of tile_store below.
template <bool TR>
__device__ inline void tile_store_part(float* T, const v4f (&reg)[kNp], int p) {
    const int f = threadIdx.x + kThreads * p;
    if constexpr (!TR) {
        *reinterpret_cast<v4f*>(T + (f / kFpr) * kPitch + 4 * (f % kFpr)) = reg[p];
    } else {
        const int c = f >> 5, r = 4 * (f & 31);
#pragma unroll
        for (int e = 0; e < 4; ++e) T[(r + e) * kPitch + c] = reg[p][e];
    }
}

// The registers of tile_load into T[r][c] (pitch kPitch).
template <bool TR>
__device__ inline void tile_store(float* T, const v4f (&reg)[kNp]) {
    const int t = threadIdx.x;
#pragma unroll
    for (int p = 0; p < kNp; ++p) {
        const int f = t + kThreads * p;
        if constexpr (!TR) {
            *reinterpret_cast<v4f*>(T + (f / kFpr) * kPitch + 4 * (f % kFpr)) = reg[p];
        } else {
            const int c = f >> 5, r = 4 * (f & 31);
#pragma unroll
            for (int e = 0; e < 4; ++e) T[(r + e) * kPitch + c] = reg[p][e];
        }
    }
}

// Product tiles of one level: item = (b, l >= 2s, tile ti, tile tj) computes
// the 128 x 128 tile (ti, tj) of A_l A_{l-s}; the tiles with tj = 0 also form
// rows 128 ti .. of r_l + A_l r_{l-s} from the A_l chunks as they pass.
// Wave (wr, wc) of the 2 x 2 wave grid owns a 64 x 64 quarter: 2 x 2 MFMA
// 32 x 32 tiles.  The k order inside a chunk: lane half h supplies
// k = 8q + 4h + e to the MFMA of step (q, e), for both operands.
template <bool VEC, bool TRANS>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3))) void
pcr_wide_prod(BlockSrc Ain, VecSrc rin, float* __restrict__ Aout, VecDst rout, int L, int w,
              int s, int nt, long long items, long long per_xcd) {
    __shared__ float TA[2][kTile * kPitch];  // A_l tile, [i][k]
    __shared__ float TB[2][kTile * kPitch];  // A_{l-s} tile transposed, [j][k]
    __shared__ float rp[kWide + kKC];        // r_{l-s}, zero beyond w
    const long long id = (long long)(blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    if (id >= items) return;  // uniform over the workgroup
    const int nt2 = nt * nt;
    const long long prod = id / nt2;
    const int tt = (int)(id - prod * nt2);
    const int ti = tt / nt, tj = tt - (tt / nt) * nt;
    const long long np = L - 2 * s;
    const int b = (int)(prod / np);
    const int l = 2 * s + (int)(prod - (long long)b * np);
    const float* Al = Ain.base + b * Ain.bstride + (long long)l * Ain.rstride;
    const float* Ap = Ain.base + b * Ain.bstride + (long long)(l - s) * Ain.rstride;
    const int i0 = kTile * ti, j0 = kTile * tj;
    const bool mv = tj == 0;
    const int t = threadIdx.x;
    if (mv) {
        const float* rq = rin.base + b * rin.bstride + (long long)(l - s) * rin.rstride;
        for (int i = t; i < kWide + kKC; i += kThreads) rp[i] = i < w ? rq[i] : 0.f;
    }
    const int lane = t & 63, wave = t >> 6;
    const int wr = wave >> 1, wc = wave & 1;
    const int li = lane & 31, h = lane >> 5;
    v16f acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int c = 0; c < 2; ++c) acc[a][c] = v16f{};
    float mva = 0.f;
    const int nk = (w + kKC - 1) / kKC;
    v4f ra[kNp], rb[kNp];
    tile_load<VEC, TRANS>(Al, w, i0, 0, ra);
    tile_load<VEC, !TRANS>(Ap, w, j0, 0, rb);
    tile_store<TRANS>(TA[0], ra);
    tile_store<!TRANS>(TB[0], rb);
    __syncthreads();
    for (int kc = 0; kc < nk; ++kc) {
        const int buf = kc & 1;
        const bool more = kc + 1 < nk;
        if (more) {
            tile_load<VEC, TRANS>(Al, w, i0, (kc + 1) * kKC, ra);
            tile_load<VEC, !TRANS>(Ap, w, j0, (kc + 1) * kKC, rb);
        }
        const float* ta = TA[buf] + (64 * wr + li) * kPitch + 4 * h;
        const float* tb = TB[buf] + (64 * wc + li) * kPitch + 4 * h;
#pragma unroll
        for (int q = 0; q < kKC / 8; ++q) {
            const v4f a0 = *reinterpret_cast<const v4f*>(ta + 8 * q);
            const v4f a1 = *reinterpret_cast<const v4f*>(ta + 32 * kPitch + 8 * q);
            const v4f b0 = *reinterpret_cast<const v4f*>(tb + 8 * q);
            const v4f b1 = *reinterpret_cast<const v4f*>(tb + 32 * kPitch + 8 * q);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[e], b0[e], acc[0][0], 0, 0, 0);
                acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[e], b1[e], acc[0][1], 0, 0, 0);
                acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[e], b0[e], acc[1][0], 0, 0, 0);
                acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[e], b1[e], acc[1][1], 0, 0, 0);
            }
            // the next chunk's part q into the other buffer, beside this
            // step's products (that buffer is not read before the barrier)
            if (more && q < kNp) {
                tile_store_part<TRANS>(TA[buf ^ 1], ra, q);
                tile_store_part<!TRANS>(TB[buf ^ 1], rb, q);
            }
        }
        if (mv) {
            // thread t: row t / 2 of the tile, half t % 2 of the chunk's columns
            const float* arow = TA[buf] + (t >> 1) * kPitch + (kKC / 2) * (t & 1);
            const float* rv = rp + kc * kKC + (kKC / 2) * (t & 1);
#pragma unroll
            for (int c = 0; c < kKC / 2; ++c) mva = fmaf(arow[c], rv[c], mva);
        }
        __syncthreads();
    }
    // lane (li, h) holds column li of each 32 x 32 tile, rows 8 (v/4) + 4 h + v%4
    float* Ao = Aout + ((long long)b * L + l) * w * w;
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int col = j0 + 64 * wc + 32 * c + li;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = i0 + 64 * wr + 32 * a + 8 * (v >> 2) + 4 * h + (v & 3);
                if (row < w && col < w) Ao[(long long)row * w + col] = acc[a][c][v];
            }
        }
    if (mv) {
        mva += __shfl_xor(mva, 1, 64);
        const int row = i0 + (t >> 1);
        if ((t & 1) == 0 && row < w) {
            const float* rl = rin.base + b * rin.bstride + (long long)l * rin.rstride;
            rout.base[b * rout.bstride + (long long)l * rout.rstride + row] = rl[row] + mva;
        }
    }
}

// Rows l < min(2s, L) of a level: copy (l < s) or r_l + A_l r_{l-s}
// (s <= l < 2s).  Workgroup (system and row, 32 output rows): a wave per
// output row (four waves, eight rows each), or (TRANS, A_l(i, k) =
// blk[k w + i]) eight groups of 32 threads over k, one output row per
// thread, meeting in LDS.
constexpr int kRowsPerWg = 32;

template <bool VEC, bool TRANS>
__global__ __launch_bounds__(kThreads) void pcr_wide_rows(BlockSrc Ain, VecSrc rin, VecDst rout,
                                                          int L, int w, int s, int nrows) {
    __shared__ float rp[kWide];
    __shared__ float part[kThreads / kRowsPerWg][kRowsPerWg];
    const int b = blockIdx.x / nrows;
    const int l = blockIdx.x - b * nrows;
    const int i0 = kRowsPerWg * blockIdx.y;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const float* rl = rin.base + b * rin.bstride + (long long)l * rin.rstride;
    float* xo = rout.base + b * rout.bstride + (long long)l * rout.rstride;
    if (l < s) {
        if (t < kRowsPerWg && i0 + t < w) xo[i0 + t] = rl[i0 + t];
        return;
    }
    stage_vec(rp, rin.base + b * rin.bstride + (long long)(l - s) * rin.rstride, w);
    __syncthreads();
    const float* Al = Ain.base + b * Ain.bstride + (long long)l * Ain.rstride;
    if constexpr (!TRANS) {
        for (int i = i0 + wave; i < min(w, i0 + kRowsPerWg); i += kWaves) {
            float v[16];
            row_load<VEC>(Al + (long long)i * w, w, v, lane);
            const float d = row_dot<VEC>(v, rp, lane);
            if (lane == 0) xo[i] = rl[i] + d;
        }
    } else {
        const int ii = t % kRowsPerWg, kg = t / kRowsPerWg;
        const int i = i0 + ii;
        float acc = 0.f;
        if (i < w)
            for (int k = kg; k < w; k += kThreads / kRowsPerWg)
                acc = fmaf(Al[(long long)k * w + i], rp[k], acc);
        part[kg][ii] = acc;
        __syncthreads();
        if (kg == 0 && i < w) {
            float sum = part[0][ii];
            for (int q = 1; q < kThreads / kRowsPerWg; ++q) sum += part[q][ii];
            xo[i] = rl[i] + sum;
        }
    }
}

// ------------------------------------------------------- layer kernels
// Forward Newton evaluation at the iterate, one workgroup per (b, l): each
// wave takes rows i of W_l, holds the row in registers for the
// pre-activation a_i = W_l[i] . Z[b, l-1] + b_l[i] and writes row i of
// J_l = diag(c) W_l (+ I) from the same registers (W_l is read once).
template <bool VEC>
__global__ __launch_bounds__(kThreads) void forward_eval_wide(
    const float* __restrict__ W, const float* __restrict__ bias, const float* __restrict__ z0,
    const float* __restrict__ Z, float* __restrict__ A, float* __restrict__ r,
    unsigned* __restrict__ red, int L, int w, int layer, float alpha) {
    __shared__ float zp[kWide];
    const long long row = blockIdx.x;
    const int l = (int)(row % L);
    const int b = (int)(row / L);
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    if (row == 0)
        for (int k = t; k < 2 * kRedShards; k += kThreads) red[k] = 0u;
    stage_vec(zp, (l == 0) ? z0 + (long long)b * w : Z + (row - 1) * w, w);
    __syncthreads();
    const bool res = layer_residual(layer);
    const float* Wl = W + (long long)l * w * w;
    unsigned mr = 0u;
    for (int i = wave; i < w; i += kWaves) {
        float v[16];
        row_load<VEC>(Wl + (long long)i * w, w, v, lane);
        const float a = row_dot<VEC>(v, zp, lane) + bias[(long long)l * w + i];
        float d;
        const float y = activate(layer, a, &d);
        const float f = res ? fmaf(alpha, y, zp[i]) : y;
        const float rv = f - Z[row * w + i];
        if (lane == 0) r[row * w + i] = rv;
        mr = max(mr, __float_as_uint(fabsf(rv)));
        if (l >= 1)
            row_store_scaled<VEC>(A + row * w * w + (long long)i * w, w, v, res ? alpha * d : d,
                                  res ? i : -1, lane);
    }
    if (lane == 0) atomicMax(red + kRedF + (int)(row % kRedShards), mr);
}

// Z[b, l] = Z[b, 0] for l >= 1.
__global__ __launch_bounds__(kThreads) void broadcast_row0(float* __restrict__ Z, int L, int w,
                                                           int rows_per_block) {
    const int chunks = (L + rows_per_block - 1) / rows_per_block;
    const int b = blockIdx.x / chunks;
    const int l0 = max(1, (blockIdx.x % chunks) * rows_per_block);
    const int l1 = min(L, (blockIdx.x % chunks + 1) * rows_per_block);
    float* zb = Z + (long long)b * L * w;
    for (long long idx = threadIdx.x; idx < (long long)(l1 - l0) * w; idx += kThreads)
        zb[(long long)l0 * w + idx] = zb[idx % w];
}

// Backward assembly, one workgroup per (b, l): c d_l (dscale), the reversed
// right-hand side (G at m = 0), and block m = L - l = J_l (to be read
// transposed), each row of J_l from the W_l row held for its pre-activation.
template <bool VEC>
__global__ __launch_bounds__(kThreads) void backward_assemble_wide(
    const float* __restrict__ W, const float* __restrict__ bias, const float* __restrict__ z0,
    const float* __restrict__ Z, const float* __restrict__ G, float* __restrict__ A,
    float* __restrict__ rrev, float* __restrict__ dscale, int L, int w, int layer, float alpha) {
    __shared__ float zp[kWide];
    const long long row = blockIdx.x;
    const int l = (int)(row % L);
    const int b = (int)(row / L);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    stage_vec(zp, (l == 0) ? z0 + (long long)b * w : Z + (row - 1) * w, w);
    __syncthreads();
    const bool res = layer_residual(layer);
    const int m = L - 1 - l;
    const float* Wl = W + (long long)l * w * w;
    float* Ab = A ? A + ((long long)b * L + (L - l)) * w * w : nullptr;
    for (int k = wave; k < w; k += kWaves) {
        float v[16];
        row_load<VEC>(Wl + (long long)k * w, w, v, lane);
        const float a = row_dot<VEC>(v, zp, lane) + bias[(long long)l * w + k];
        float d;
        activate(layer, a, &d);
        const float c = res ? alpha * d : d;
        if (lane == 0) {
            dscale[row * w + k] = c;
            rrev[((long long)b * L + m) * w + k] = (m == 0) ? G[(long long)b * w + k] : 0.f;
        }
        if (l >= 1 && Ab) row_store_scaled<VEC>(Ab + (long long)k * w, w, v, c, res ? k : -1, lane);
    }
}

// out[b][k] = sum_i W[i][k] g_b[i] (+ add[b][k]) with g_b = g1_b (* g2_b).
// Grid (chunks of 64 k, B), 1024 threads: thread (k = k0 + t % 64, group
// t / 64) sums over i = group, group + 16, ... (eight loads in flight per
// thread); the sixteen groups meet in LDS in a fixed order.
// single = 1: one workgroup per system covers every chunk after g_b is in
// LDS (out may then be the memory g1 points to).
constexpr int kMvtThreads = 1024;
constexpr int kMvtGroups = kMvtThreads / 64;

__global__ __launch_bounds__(kMvtThreads) void matvec_t_wide(
    const float* __restrict__ W, const float* g1, long long g1_bstride, const float* g2,
    long long g2_bstride, const float* add, long long add_bstride, float* out,
    long long out_bstride, int w, int single) {
    __shared__ float g[kWide];
    __shared__ float part[kMvtGroups][64];
    const int b = blockIdx.y;
    const int t = threadIdx.x, kk = t & 63, grp = t >> 6;
    for (int i = t; i < w; i += kMvtThreads) {
        float x = g1[b * g1_bstride + i];
        if (g2) x *= g2[b * g2_bstride + i];
        g[i] = x;
    }
    __syncthreads();
    const int nchunk = (w + 63) / 64;
    const int c0 = single ? 0 : blockIdx.x, c1 = single ? nchunk : blockIdx.x + 1;
    for (int c = c0; c < c1; ++c) {
        const int k = 64 * c + kk;
        float acc = 0.f;
        if (k < w) {
            const float* col = W + k;
            int i = grp;
            for (; i + 7 * kMvtGroups < w; i += 8 * kMvtGroups) {
                float v[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) v[u] = col[(long long)(i + u * kMvtGroups) * w];
#pragma unroll
                for (int u = 0; u < 8; ++u) acc = fmaf(v[u], g[i + u * kMvtGroups], acc);
            }
            for (; i < w; i += kMvtGroups) acc = fmaf(col[(long long)i * w], g[i], acc);
        }
        part[grp][kk] = acc;
        __syncthreads();
        if (grp == 0 && k < w) {
            float sum = part[0][kk];
            for (int q = 1; q < kMvtGroups; ++q) sum += part[q][kk];
            if (add) sum += add[b * add_bstride + k];
            out[b * out_bstride + k] = sum;
        }
        __syncthreads();
    }
}

// Parameter gradients, one workgroup per (layer, 8 rows of dW[l]):
// dW[l][i][j] = sum_b g[b][i] zin[b][j], db[l][i] = sum_b g[b][i],
// g = dscale * Lambda at (b, l), zin = Z[b, l-1] (z0 at l = 0); the batch in
// chunks of 8, summed in a fixed order.
constexpr int kWgRows = 8;
constexpr int kWgBC = 8;

__global__ __launch_bounds__(kThreads) void wgrad_wide(
    const float* __restrict__ z0, const float* __restrict__ Z, const float* __restrict__ dscale,
    const float* __restrict__ Lambda, float* __restrict__ dW, float* __restrict__ db, int B,
    int L, int w) {
    __shared__ float zs[kWgBC][kWide];
    __shared__ float gs[kWgBC][kWgRows];
    const int l = blockIdx.x;
    const int i0 = kWgRows * blockIdx.y;
    const int t = threadIdx.x;
    float acc[kWgRows][4];
#pragma unroll
    for (int r = 0; r < kWgRows; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = 0.f;
    float dbacc = 0.f;
    for (int b0 = 0; b0 < B; b0 += kWgBC) {
        const int nb = min(kWgBC, B - b0);
        for (int idx = t; idx < nb * w; idx += kThreads) {
            const int bb = idx / w, j = idx - (idx / w) * w;
            const long long rowj = ((long long)(b0 + bb) * L + l) * w;
            zs[bb][j] = (l == 0) ? z0[(long long)(b0 + bb) * w + j] : Z[rowj - w + j];
        }
        if (t < nb * kWgRows) {
            const int bb = t / kWgRows, r = t - (t / kWgRows) * kWgRows;
            const long long idx = ((long long)(b0 + bb) * L + l) * w + i0 + r;
            gs[bb][r] = (i0 + r < w) ? dscale[idx] * Lambda[idx] : 0.f;
        }
        __syncthreads();
        for (int bb = 0; bb < nb; ++bb) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int j = t + kThreads * c;
                const float z = j < w ? zs[bb][j] : 0.f;
#pragma unroll
                for (int r = 0; r < kWgRows; ++r) acc[r][c] = fmaf(gs[bb][r], z, acc[r][c]);
            }
            if (t < kWgRows) dbacc += gs[bb][t];
        }
        __syncthreads();
    }
#pragma unroll
    for (int r = 0; r < kWgRows; ++r) {
        if (i0 + r >= w) break;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int j = t + kThreads * c;
            if (j < w) dW[((long long)l * w + i0 + r) * w + j] = acc[r][c];
        }
    }
    if (t < kWgRows && i0 + t < w) db[(long long)l * w + i0 + t] = dbacc;
}

// ------------------------------------------------------ sequential passes
// One layer l of the sequential passes for a tile of up to 8 systems:
// workgroup (row group, system tile), a wave per row i of W_l, the row held
// in registers for every system of the tile.
// BWD = false: Z[b, l] = f_l(Z[b, l-1]).
// BWD = true:  g[b][i] = c d_i Lambda[b, l][i] (Lambda[b, L-1] := G, which
//              is also written), the first half of the adjoint step.
constexpr int kSeqBC = 8;

template <bool VEC, bool BWD>
__global__ __launch_bounds__(kThreads) void seq_layer_wide(
    const float* __restrict__ W, const float* __restrict__ bias, const float* __restrict__ z0,
    const float* Zin, float* __restrict__ Zout, const float* __restrict__ G,
    float* __restrict__ Lambda, float* __restrict__ g, int B, int L, int w, int layer,
    float alpha, int l) {
    __shared__ float zs[kSeqBC][kWide];
    const int b0 = kSeqBC * blockIdx.y;
    const int nb = min(kSeqBC, B - b0);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int bb = 0; bb < nb; ++bb) {
        const int b = b0 + bb;
        stage_vec(zs[bb], (l == 0) ? z0 + (long long)b * w : Zin + ((long long)b * L + l - 1) * w, w);
    }
    __syncthreads();
    const int i = kWaves * blockIdx.x + wave;
    if (i >= w) return;
    float v[16];
    row_load<VEC>(W + ((long long)l * w + i) * w, w, v, lane);
    const float bi = bias[(long long)l * w + i];
    const bool res = layer_residual(layer);
    for (int bb = 0; bb < nb; ++bb) {
        const int b = b0 + bb;
        const float a = row_dot<VEC>(v, zs[bb], lane) + bi;
        float d;
        const float y = activate(layer, a, &d);
        if (lane != 0) continue;
        const long long o = ((long long)b * L + l) * w + i;
        if constexpr (!BWD) {
            Zout[o] = res ? fmaf(alpha, y, zs[bb][i]) : y;
        } else {
            float lam;
            if (l == L - 1) {
                lam = G[(long long)b * w + i];
                Lambda[o] = lam;
            } else {
                lam = Lambda[o];
            }
            g[(long long)b * w + i] = (res ? alpha * d : d) * lam;
        }
    }
}

}  // namespace

bool wide_width(int w) { return w > kMaxWidth && w <= kMaxWideWidth; }

hipError_t launch_pcr_level_wide(const BlockSrc& Ain, const VecSrc& rin, float* Aout,
                                 const VecDst& rout, int B, int L, int w, int s,
                                 hipStream_t stream) {
    const bool vec = (w % 4) == 0;
    const bool tr = Ain.trans != 0;
    const int nrows = L < 2 * s ? L : 2 * s;
    const dim3 g1((unsigned)((long long)B * nrows), (unsigned)((w + kRowsPerWg - 1) / kRowsPerWg));
#define DEEPPCR_WIDE_ROWS(V, T) \
    hipLaunchKernelGGL((pcr_wide_rows<V, T>), g1, dim3(kThreads), 0, stream, Ain, rin, rout, L, w, s, nrows)
    if (vec && tr) DEEPPCR_WIDE_ROWS(true, true);
    else if (vec) DEEPPCR_WIDE_ROWS(true, false);
    else if (tr) DEEPPCR_WIDE_ROWS(false, true);
    else DEEPPCR_WIDE_ROWS(false, false);
#undef DEEPPCR_WIDE_ROWS
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || L <= 2 * s) return e;
    const int nt = (w + kTile - 1) / kTile;
    const long long items = (long long)B * (L - 2 * s) * nt * nt;
    const long long per_xcd = (items + kXcds - 1) / kXcds;
    const dim3 g2((unsigned)(per_xcd * kXcds));
#define DEEPPCR_WIDE_PROD(V, T)                                                                 \
    hipLaunchKernelGGL((pcr_wide_prod<V, T>), g2, dim3(kThreads), 0, stream, Ain, rin, Aout,   \
                       rout, L, w, s, nt, items, per_xcd)
    if (vec && tr) DEEPPCR_WIDE_PROD(true, true);
    else if (vec) DEEPPCR_WIDE_PROD(true, false);
    else if (tr) DEEPPCR_WIDE_PROD(false, true);
    else DEEPPCR_WIDE_PROD(false, false);
#undef DEEPPCR_WIDE_PROD
    return hipGetLastError();
}

hipError_t launch_forward_eval_wide(const float* W, const float* bias, const float* z0,
                                    const float* Z, float* A, float* r, unsigned* red, int B,
                                    int L, int w, int layer, float alpha, hipStream_t stream) {
    const dim3 grid((unsigned)((long long)B * L));
    if (w % 4 == 0)
        hipLaunchKernelGGL((forward_eval_wide<true>), grid, dim3(kThreads), 0, stream, W, bias, z0,
                           Z, A, r, red, L, w, layer, alpha);
    else
        hipLaunchKernelGGL((forward_eval_wide<false>), grid, dim3(kThreads), 0, stream, W, bias,
                           z0, Z, A, r, red, L, w, layer, alpha);
    return hipGetLastError();
}

hipError_t launch_initial_guess_wide(const float* W, const float* bias, const float* z0, float* Z,
                                     int B, int L, int w, int layer, float alpha,
                                     hipStream_t stream) {
    // Z[:, 0] = f_0(z0) (the sequential kernel's layer 0), then the broadcast
    hipError_t e = launch_seq_forward_wide(W, bias, z0, Z, B, L, w, layer, alpha, 0, stream);
    if (e != hipSuccess || L == 1) return e;
    const int rows_per_block = 16;
    const int chunks = (L + rows_per_block - 1) / rows_per_block;
    hipLaunchKernelGGL(broadcast_row0, dim3((unsigned)((long long)B * chunks)), dim3(kThreads), 0,
                       stream, Z, L, w, rows_per_block);
    return hipGetLastError();
}

hipError_t launch_backward_assemble_wide(const float* W, const float* bias, const float* z0,
                                         const float* Z, const float* G, float* A, float* rrev,
                                         float* dscale, int B, int L, int w, int layer,
                                         float alpha, hipStream_t stream) {
    const dim3 grid((unsigned)((long long)B * L));
    if (w % 4 == 0)
        hipLaunchKernelGGL((backward_assemble_wide<true>), grid, dim3(kThreads), 0, stream, W, bias,
                           z0, Z, G, A, rrev, dscale, L, w, layer, alpha);
    else
        hipLaunchKernelGGL((backward_assemble_wide<false>), grid, dim3(kThreads), 0, stream, W,
                           bias, z0, Z, G, A, rrev, dscale, L, w, layer, alpha);
    return hipGetLastError();
}

hipError_t launch_dz0_wide(const float* W, const float* dscale, const float* Lambda, float* dz0,
                           int B, int L, int w, int layer, hipStream_t stream) {
    // dz0[b] = W_0^T (dscale_0 * Lambda_0) (+ Lambda_0 for residual layers)
    const long long ld = (long long)L * w;
    const dim3 grid((unsigned)((w + 63) / 64), (unsigned)B);
    hipLaunchKernelGGL(matvec_t_wide, grid, dim3(kMvtThreads), 0, stream, W, dscale, ld, Lambda, ld,
                       layer_residual(layer) ? Lambda : nullptr, ld, dz0, (long long)w, w, 0);
    return hipGetLastError();
}

hipError_t launch_wgrad_wide(const float* z0, const float* Z, const float* dscale,
                             const float* Lambda, float* dW, float* db, int B, int L, int w,
                             hipStream_t stream) {
    const dim3 grid((unsigned)L, (unsigned)((w + kWgRows - 1) / kWgRows));
    hipLaunchKernelGGL(wgrad_wide, grid, dim3(kThreads), 0, stream, z0, Z, dscale, Lambda, dW, db,
                       B, L, w);
    return hipGetLastError();
}

hipError_t launch_seq_forward_wide(const float* W, const float* bias, const float* z0, float* Z,
                                   int B, int L, int w, int layer, float alpha, int l,
                                   hipStream_t stream) {
    const dim3 grid((unsigned)((w + kWaves - 1) / kWaves), (unsigned)((B + kSeqBC - 1) / kSeqBC));
    if (w % 4 == 0)
        hipLaunchKernelGGL((seq_layer_wide<true, false>), grid, dim3(kThreads), 0, stream, W, bias,
                           z0, Z, Z, nullptr, nullptr, nullptr, B, L, w, layer, alpha, l);
    else
        hipLaunchKernelGGL((seq_layer_wide<false, false>), grid, dim3(kThreads), 0, stream, W,
                           bias, z0, Z, Z, nullptr, nullptr, nullptr, B, L, w, layer, alpha, l);
    return hipGetLastError();
}

hipError_t launch_seq_backward_wide(const float* W, const float* bias, const float* z0,
                                    const float* Z, const float* G, float* Lambda, float* dz0,
                                    int B, int L, int w, int layer, float alpha, int l,
                                    hipStream_t stream) {
    // g = c d_l Lambda_l into dz0 (free until the last step), then
    // Lambda_{l-1} = W_l^T g (+ Lambda_l), or dz0 = W_0^T g (+ Lambda_0) at l = 0
    const dim3 grid((unsigned)((w + kWaves - 1) / kWaves), (unsigned)((B + kSeqBC - 1) / kSeqBC));
    if (w % 4 == 0)
        hipLaunchKernelGGL((seq_layer_wide<true, true>), grid, dim3(kThreads), 0, stream, W, bias,
                           z0, Z, nullptr, G, Lambda, dz0, B, L, w, layer, alpha, l);
    else
        hipLaunchKernelGGL((seq_layer_wide<false, true>), grid, dim3(kThreads), 0, stream, W,
                           bias, z0, Z, nullptr, G, Lambda, dz0, B, L, w, layer, alpha, l);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const long long ld = (long long)L * w;
    const float* Wl = W + (long long)l * w * w;
    const float* add = layer_residual(layer) ? Lambda + (long long)l * w : nullptr;
    if (l >= 1) {
        const dim3 g2((unsigned)((w + 63) / 64), (unsigned)B);
        hipLaunchKernelGGL(matvec_t_wide, g2, dim3(kMvtThreads), 0, stream, Wl, dz0, (long long)w,
                           nullptr, 0LL, add, ld, Lambda + (long long)(l - 1) * w, ld, w, 0);
    } else {
        hipLaunchKernelGGL(matvec_t_wide, dim3(1u, (unsigned)B), dim3(kMvtThreads), 0, stream, Wl, dz0,
                           (long long)w, nullptr, 0LL, add, ld, dz0, (long long)w, w, 1);
    }
    return hipGetLastError();
}

}  // namespace deeppcr
