// Layer evaluation, Jacobian assembly, Newton update and gradient kernels of
// the DeepPCR hot path.
//
// Layers (App. A.1, Eqs. 7-9, post-activation form; App. A.3 with a skip of
// length one), sigma in {tanh, logistic sigmoid, ReLU}:
//   plain    : f_l(z) = sigma(W_l z + b_l),          J_l = diag(sigma') W_l
//   residual : f_l(z) = z + alpha sigma(W_l z + b_l), J_l = I + alpha diag(sigma') W_l
#include "internal.h"

namespace deeppcr {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

__device__ inline float wave_sum(float v) {
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__device__ inline unsigned wave_umax(unsigned v) {
    for (int off = 32; off > 0; off >>= 1) v = max(v, (unsigned)__shfl_xor((int)v, off, 64));
    return v;
}

// a_i = sum_j W[i][j] z[j] + b[i] for all rows i < w; one wave per row,
// lanes stride over j.  z lives in LDS.  Results go to out[i] in LDS.
__device__ inline void preactivations(const float* __restrict__ Wl, const float* __restrict__ bl,
                                      const float* z, float* out, int w) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int i = wave; i < w; i += kWaves) {
        float acc = 0.f;
        for (int j = lane; j < w; j += 64) acc = fmaf(Wl[(long long)i * w + j], z[j], acc);
        acc = wave_sum(acc);
        if (lane == 0) out[i] = acc + bl[i];
    }
}

// ---------------------------------------------------------------- forward
__global__ __launch_bounds__(kThreads) void forward_eval_kernel(
    const float* __restrict__ W, const float* __restrict__ bias, const float* __restrict__ z0,
    const float* __restrict__ Z, float* __restrict__ A, float* __restrict__ r,
    unsigned* __restrict__ red, int L, int w, int layer, float alpha) {
    const long long row = blockIdx.x;
    const int l = (int)(row % L);
    const int b = (int)(row / L);
    const int t = threadIdx.x;
    if (row == 0)
        for (int k = t; k < 2 * kRedShards; k += kThreads) red[k] = 0u;

    __shared__ float zp[kMaxWidth];
    __shared__ float a[kMaxWidth];
    __shared__ float dsc[kMaxWidth];
    const float* zprev = (l == 0) ? z0 + (long long)b * w : Z + (row - 1) * w;
    for (int i = t; i < w; i += kThreads) zp[i] = zprev[i];
    __syncthreads();
    const float* Wl = W + (long long)l * w * w;
    preactivations(Wl, bias + (long long)l * w, zp, a, w);
    __syncthreads();
    const bool res = layer_residual(layer);
    unsigned mr = 0u;  // max |r| bits
    for (int i = t; i < w; i += kThreads) {
        float d;
        const float y = activate(layer, a[i], &d);
        const float f = res ? fmaf(alpha, y, zp[i]) : y;
        const float rv = f - Z[row * w + i];
        r[row * w + i] = rv;
        mr = max(mr, __float_as_uint(fabsf(rv)));
        dsc[i] = res ? alpha * d : d;
    }
    if ((t >> 6) * 64 < w) {  // waves holding residual elements
        mr = wave_umax(mr);
        if ((t & 63) == 0) atomicMax(red + kRedF + (int)(row % kRedShards), mr);
    }
    __syncthreads();
    if (l == 0) return;
    float* Ab = A + row * w * w;
    for (int idx = t; idx < w * w; idx += kThreads) {
        const int i = idx / w, j = idx - (idx / w) * w;
        float v = dsc[i] * Wl[idx];
        if (res && i == j) v += 1.f;
        Ab[idx] = v;
    }
}

__global__ __launch_bounds__(kThreads) void initial_guess_kernel(
    const float* __restrict__ W, const float* __restrict__ bias, const float* __restrict__ z0,
    float* __restrict__ Z, int L, int w, int layer, float alpha, int rows_per_block) {
    const int chunks = (L + rows_per_block - 1) / rows_per_block;
    const int b = blockIdx.x / chunks;
    const int l0 = (blockIdx.x % chunks) * rows_per_block;
    const int t = threadIdx.x;
    __shared__ float zp[kMaxWidth];
    __shared__ float a[kMaxWidth];
    __shared__ float f0[kMaxWidth];
    for (int i = t; i < w; i += kThreads) zp[i] = z0[(long long)b * w + i];
    __syncthreads();
    preactivations(W, bias, zp, a, w);
    __syncthreads();
    for (int i = t; i < w; i += kThreads) {
        float d;
        const float y = activate(layer, a[i], &d);
        f0[i] = layer_residual(layer) ? fmaf(alpha, y, zp[i]) : y;
    }
    __syncthreads();
    const int l1 = min(L, l0 + rows_per_block);
    for (long long idx = t; idx < (long long)(l1 - l0) * w; idx += kThreads) {
        const int i = (int)(idx % w);
        Z[((long long)b * L + l0) * w + idx] = f0[i];
    }
}

__global__ __launch_bounds__(kThreads) void update_reduce_kernel(
    float* __restrict__ Z, const float* __restrict__ x, long long n, unsigned* __restrict__ red) {
    unsigned mx = 0u, mz = 0u;
    for (long long i = (long long)blockIdx.x * kThreads + threadIdx.x; i < n;
         i += (long long)gridDim.x * kThreads) {
        const float dx = x[i];
        const float z = Z[i] + dx;
        Z[i] = z;
        mx = max(mx, __float_as_uint(fabsf(dx)));
        mz = max(mz, __float_as_uint(fabsf(z)));
    }
    mx = wave_umax(mx);
    mz = wave_umax(mz);
    __shared__ unsigned sx[kWaves], sz[kWaves];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) {
        sx[wave] = mx;
        sz[wave] = mz;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned a = sx[0], c = sz[0];
        for (int i = 1; i < kWaves; ++i) {
            a = max(a, sx[i]);
            c = max(c, sz[i]);
        }
        const int slot = blockIdx.x % kRedShards;
        atomicMax(red + kRedDZ + slot, a);
        atomicMax(red + kRedZ + slot, c);
    }
}

// --------------------------------------------------------------- backward
__global__ __launch_bounds__(kThreads) void backward_assemble_kernel(
    const float* __restrict__ W, const float* __restrict__ bias, const float* __restrict__ z0,
    const float* __restrict__ Z, const float* __restrict__ G, float* __restrict__ A,
    float* __restrict__ rrev, float* __restrict__ dscale, int L, int w, int layer, float alpha) {
    const long long row = blockIdx.x;  // natural (b, l)
    const int l = (int)(row % L);
    const int b = (int)(row / L);
    const int t = threadIdx.x;
    __shared__ float zp[kMaxWidth];
    __shared__ float a[kMaxWidth];
    __shared__ float dsc[kMaxWidth];
    const float* zprev = (l == 0) ? z0 + (long long)b * w : Z + (row - 1) * w;
    for (int i = t; i < w; i += kThreads) zp[i] = zprev[i];
    __syncthreads();
    const float* Wl = W + (long long)l * w * w;
    preactivations(Wl, bias + (long long)l * w, zp, a, w);
    __syncthreads();
    const int m = L - 1 - l;  // reversed row of this layer's adjoint
    const bool res = layer_residual(layer);
    for (int i = t; i < w; i += kThreads) {
        float d;
        activate(layer, a[i], &d);
        const float c = res ? alpha * d : d;
        dsc[i] = c;
        dscale[row * w + i] = c;
        rrev[((long long)b * L + m) * w + i] = (m == 0) ? G[(long long)b * w + i] : 0.f;
    }
    __syncthreads();
    if (l == 0) return;
    // Reversed row L - l holds J_l^T: element (i, k) = J_l[k][i] = dsc[k] W_l[k][i] (+ delta).
    float* Ab = A + ((long long)b * L + (L - l)) * w * w;
    for (int idx = t; idx < w * w; idx += kThreads) {
        const int i = idx / w, k = idx - (idx / w) * w;
        float v = dsc[k] * Wl[(long long)k * w + i];
        if (res && i == k) v += 1.f;
        Ab[idx] = v;
    }
}

__global__ __launch_bounds__(kThreads) void dz0_kernel(
    const float* __restrict__ W, const float* __restrict__ dscale, const float* __restrict__ Lambda,
    float* __restrict__ dz0, int L, int w, int layer) {
    const int b = blockIdx.x;
    const int t = threadIdx.x;
    __shared__ float g[kMaxWidth];
    const float* lam = Lambda + (long long)b * L * w;  // row l = 0
    const float* dsc = dscale + (long long)b * L * w;
    for (int k = t; k < w; k += kThreads) g[k] = dsc[k] * lam[k];
    __syncthreads();
    for (int i = t; i < w; i += kThreads) {
        float acc = 0.f;
        for (int k = 0; k < w; ++k) acc = fmaf(W[(long long)k * w + i], g[k], acc);
        dz0[(long long)b * w + i] = layer_residual(layer) ? lam[i] + acc : acc;
    }
}

constexpr int kWgradBC = 32;  // batch rows staged per LDS chunk

// PRE = false: g = dscale * Lambda and the layer inputs as they are (the
// post-activation MLP of Eq. 10).  PRE = true: g = Lambda and sigma(layer
// input) with activation act (the pre-activation layers of the ResNet).
template <bool PRE>
__global__ __launch_bounds__(kThreads) void wgrad_kernel(
    const float* __restrict__ z0, const float* __restrict__ Z, const float* __restrict__ dscale,
    const float* __restrict__ Lambda, float* __restrict__ dW, float* __restrict__ db, int B, int L,
    int w, int act) {
    const int l = blockIdx.x;
    const int t = threadIdx.x;
    __shared__ float g[kWgradBC][kMaxWidth];
    __shared__ float zp[kWgradBC][kMaxWidth];
    constexpr int kAcc = kMaxWidth * kMaxWidth / kThreads;
    float acc[kAcc];
#pragma unroll
    for (int q = 0; q < kAcc; ++q) acc[q] = 0.f;
    float dbacc = 0.f;
    const int nout = w * w;
    for (int b0 = 0; b0 < B; b0 += kWgradBC) {
        const int nb = min(kWgradBC, B - b0);
        for (int idx = t; idx < nb * w; idx += kThreads) {
            const int bb = idx / w, i = idx - (idx / w) * w;
            const long long rowi = ((long long)(b0 + bb) * L + l) * w + i;
            const float zin = (l == 0) ? z0[(long long)(b0 + bb) * w + i] : Z[rowi - w];
            if constexpr (PRE) {
                float d;
                g[bb][i] = Lambda[rowi];
                zp[bb][i] = activate(2 * act, zin, &d);
            } else {
                g[bb][i] = dscale[rowi] * Lambda[rowi];
                zp[bb][i] = zin;
            }
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < kAcc; ++q) {
            const int idx = t + q * kThreads;
            if (idx < nout) {
                const int i = idx / w, j = idx - (idx / w) * w;
                float a = acc[q];
                for (int bb = 0; bb < nb; ++bb) a = fmaf(g[bb][i], zp[bb][j], a);
                acc[q] = a;
            }
        }
        if (t < w) {
            for (int bb = 0; bb < nb; ++bb) dbacc += g[bb][t];
        }
        __syncthreads();
    }
#pragma unroll
    for (int q = 0; q < kAcc; ++q) {
        const int idx = t + q * kThreads;
        if (idx < nout) dW[(long long)l * nout + idx] = acc[q];
    }
    if (t < w) db[(long long)l * w + t] = dbacc;
}

// The same sums for w = 16, 32, 64, 128, one workgroup per layer: thread
// (ti, tj) of a 16 x 16 grid owns the (w/16) x (w/16) tile of dW_l at rows
// ti w/16.. and columns tj w/16..; per staged batch row it reads its rows of
// g and columns of the layer input from LDS once and forms their outer
// product in registers (the index arithmetic is done once, outside the
// batch loop).
template <int W, bool PRE>
__global__ __launch_bounds__(kThreads) void wgrad_tile_kernel(
    const float* __restrict__ z0, const float* __restrict__ Z, const float* __restrict__ dscale,
    const float* __restrict__ Lambda, float* __restrict__ dW, float* __restrict__ db, int B, int L,
    int act) {
    constexpr int RT = W / 16;  // rows and columns of the tile of a thread
    const int l = blockIdx.x;
    const int t = threadIdx.x;
    const int i0 = (t >> 4) * RT, j0 = (t & 15) * RT;
    __shared__ float g[kWgradBC][W];
    __shared__ float zp[kWgradBC][W];
    float acc[RT][RT];
#pragma unroll
    for (int a = 0; a < RT; ++a)
#pragma unroll
        for (int c = 0; c < RT; ++c) acc[a][c] = 0.f;
    float dbacc = 0.f;
    for (int b0 = 0; b0 < B; b0 += kWgradBC) {
        const int nb = min(kWgradBC, B - b0);
        for (int idx = t; idx < nb * W; idx += kThreads) {
            const int bb = idx / W, i = idx % W;
            const long long rowi = ((long long)(b0 + bb) * L + l) * W + i;
            const float zin = (l == 0) ? z0[(long long)(b0 + bb) * W + i] : Z[rowi - W];
            if constexpr (PRE) {
                float d;
                g[bb][i] = Lambda[rowi];
                zp[bb][i] = activate(2 * act, zin, &d);
            } else {
                g[bb][i] = dscale[rowi] * Lambda[rowi];
                zp[bb][i] = zin;
            }
        }
        __syncthreads();
        for (int bb = 0; bb < nb; ++bb) {
            float gi[RT], zj[RT];
#pragma unroll
            for (int a = 0; a < RT; ++a) {
                gi[a] = g[bb][i0 + a];
                zj[a] = zp[bb][j0 + a];
            }
#pragma unroll
            for (int a = 0; a < RT; ++a)
#pragma unroll
                for (int c = 0; c < RT; ++c) acc[a][c] = fmaf(gi[a], zj[c], acc[a][c]);
        }
        if (t < W)
            for (int bb = 0; bb < nb; ++bb) dbacc += g[bb][t];
        __syncthreads();
    }
    float* dWl = dW + (long long)l * W * W;
#pragma unroll
    for (int a = 0; a < RT; ++a)
#pragma unroll
        for (int c = 0; c < RT; ++c) dWl[(i0 + a) * W + j0 + c] = acc[a][c];
    if (t < W) db[(long long)l * W + t] = dbacc;
}

// The same sums for w <= 8: one thread per element (l, i, j) of dW (and of db
// for j = 0), the batch summed in the same order, so the results equal
// wgrad_kernel's.
template <bool PRE>
__global__ __launch_bounds__(kThreads) void wgrad_small_kernel(
    const float* __restrict__ z0, const float* __restrict__ Z, const float* __restrict__ dscale,
    const float* __restrict__ Lambda, float* __restrict__ dW, float* __restrict__ db, int B, int L,
    int w, int act) {
    const long long o = (long long)blockIdx.x * kThreads + threadIdx.x;  // (l w + i) w + j
    if (o >= (long long)L * w * w) return;
    const int j = (int)(o % w);
    const long long li = o / w;
    const int i = (int)(li % w);
    const long long l = li / w;
    float acc = 0.f, dbacc = 0.f;
    for (int b = 0; b < B; ++b) {
        const long long row = ((long long)b * L + l) * w;
        const float gi = PRE ? Lambda[row + i] : dscale[row + i] * Lambda[row + i];
        const float zin = (l == 0) ? z0[(long long)b * w + j] : Z[row - w + j];
        float zpj = zin;
        if constexpr (PRE) {
            float d;
            zpj = activate(2 * act, zin, &d);
        }
        acc = fmaf(gi, zpj, acc);
        dbacc += gi;
    }
    dW[o] = acc;
    if (j == 0) db[l * w + i] = dbacc;
}

// Backward assembly without the blocks (the first PCR pass forms them from
// the weights): per (b, l) the scale c d_l (d = sigma'(W_l Z_{l-1} + b_l))
// and the reversed right-hand side, as layer_eval_vec<W, true> writes them.
// One workgroup per layer, so that W_l is read once for all systems: thread
// t holds row i = t % w of W_l in registers and forms that row's sum for
// batch rows t / w, t / w + 256 / w, ... of each staged chunk (the chunk's
// state rows are read from LDS as broadcasts, and each wave's results are
// consecutive rows, so the stores are contiguous).
template <int W>
__global__ __launch_bounds__(kThreads) void bwd_scale_kernel(
    const float* __restrict__ W_, const float* __restrict__ bias, const float* __restrict__ z0,
    const float* __restrict__ Z, const float* __restrict__ G, float* __restrict__ r,
    float* __restrict__ dscale, int B, int L, int layer, float alpha) {
    constexpr int NG = kThreads / W;  // batch rows formed at once
    const int l = blockIdx.x;
    const int t = threadIdx.x;
    const int i = t % W, grp = t / W;
    __shared__ __align__(16) float zs[kWgradBC][W];
    float wr[W];
    const float* Wrow = W_ + ((long long)l * W + i) * W;
#pragma unroll
    for (int q = 0; q < W / 4; ++q) {
        const v4f x = *reinterpret_cast<const v4f*>(Wrow + 4 * q);
#pragma unroll
        for (int e = 0; e < 4; ++e) wr[4 * q + e] = x[e];
    }
    const float bi = bias[(long long)l * W + i];
    const bool res = layer_residual(layer);
    const int mr = L - 1 - l;  // reversed row of layer l
    for (int b0 = 0; b0 < B; b0 += kWgradBC) {
        const int nb = min(kWgradBC, B - b0);
        for (int idx = t; idx < nb * W; idx += kThreads) {
            const int bb = idx / W, k = idx % W;
            const long long b = b0 + bb;
            zs[bb][k] = (l == 0) ? z0[b * W + k] : Z[(b * L + l - 1) * W + k];
        }
        __syncthreads();
        for (int bb = grp; bb < nb; bb += NG) {
            // four partial sums (columns k = 4q + e), added pairwise
            float p[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < W / 4; ++q) {
                const v4f z4 = *reinterpret_cast<const v4f*>(&zs[bb][4 * q]);
#pragma unroll
                for (int e = 0; e < 4; ++e) p[e] = fmaf(wr[4 * q + e], z4[e], p[e]);
            }
            float d;
            activate(layer, ((p[0] + p[1]) + (p[2] + p[3])) + bi, &d);
            const long long b = b0 + bb;
            dscale[(b * L + l) * W + i] = res ? alpha * d : d;
            r[(b * L + mr) * W + i] = (mr == 0) ? G[b * W + i] : 0.f;
        }
        __syncthreads();
    }
}

// r = F - Z over n floats, max |r| bits into the kRedF slots of red.
__global__ __launch_bounds__(kThreads) void residual_kernel(const float* __restrict__ F,
                                                           const float* __restrict__ Z,
                                                           float* __restrict__ r, long long n,
                                                           unsigned* __restrict__ red) {
    unsigned mr = 0u;
    for (long long k = (long long)blockIdx.x * kThreads + threadIdx.x; k < n;
         k += (long long)gridDim.x * kThreads) {
        const float v = F[k] - Z[k];
        r[k] = v;
        mr = max(mr, __float_as_uint(fabsf(v)));
    }
    mr = wave_umax(mr);
    if ((threadIdx.x & 63) == 0) atomicMax(red + kRedF + (int)(blockIdx.x % kRedShards), mr);
}

__global__ __launch_bounds__(kThreads) void zero_words_kernel(unsigned* __restrict__ p, int n) {
    const int i = blockIdx.x * kThreads + threadIdx.x;
    if (i < n) p[i] = 0u;
}

// The Newton stopping measures for the host: max |dZ|, max |Z| and max |F|,
// each the max over its kRedShards slots, go to out[0..2], then seq to
// out[3] after a system-scope fence, so that a host that reads seq in out[3]
// (host-mapped memory) also reads the maxima.  One workgroup of kRedShards
// threads, one slot of each measure per thread.
__global__ __launch_bounds__(kRedShards) void measures_kernel(const unsigned* __restrict__ red,
                                                              unsigned* out, unsigned seq) {
    __shared__ unsigned part[3][kRedShards / 64];
    const int t = threadIdx.x;
    unsigned v[3] = {red[kRedDZ + t], red[kRedZ + t], red[kRedF + t]};
#pragma unroll
    for (int j = 0; j < 3; ++j)
        for (int off = 32; off > 0; off >>= 1) v[j] = max(v[j], (unsigned)__shfl_xor((int)v[j], off, 64));
    if ((t & 63) == 0)
        for (int j = 0; j < 3; ++j) part[j][t >> 6] = v[j];
    __syncthreads();
    if (t == 0) {
        for (int j = 0; j < 3; ++j) {
            unsigned m = part[j][0];
            for (int q = 1; q < kRedShards / 64; ++q) m = max(m, part[j][q]);
            out[j] = m;
        }
        __threadfence_system();
        __hip_atomic_store(out + 3, seq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
}

__global__ __launch_bounds__(kThreads) void copy_rows_kernel(VecSrc src, VecDst dst, int L, int w) {
    const long long row = blockIdx.x;
    const int l = (int)(row % L);
    const int b = (int)(row / L);
    const float* s = src.base + b * src.bstride + (long long)l * src.rstride;
    float* d = dst.base + b * dst.bstride + (long long)l * dst.rstride;
    for (int i = threadIdx.x; i < w; i += kThreads) d[i] = s[i];
}

// ---------------------------------------------------------------------------
// Vectorized layer + Jacobian evaluation for w in {16, 32, 64, 128}.
// Every thread owns float4 chunks of W_l (row i, columns 4c..4c+3); the W/4
// threads of a row form a contiguous lane group, so the pre-activation
// a_i = W_l[i,:] z + b_i is reduced by lane shuffles inside the group and
// every lane of the group then holds a_i.  The Jacobian rows are written with
// float4 stores.  Mode FWD writes J_l at row l and the residual; mode BWD
// writes J_l (not transposed) at reversed row L - l (unless A is null),
// c * d_l and the reversed right-hand side (G at reversed row 0).

template <int W>
struct EvalShape {
    static constexpr int ROWS_PER_WG = (W * W >= 1024) ? 1 : 1024 / (W * W);  // (b, l) rows
    static constexpr int NCH = W * W / 4;                                      // chunks per block
    static constexpr int TPB = NCH < 256 ? NCH : 256;                          // threads per block
    static constexpr int CPT = NCH / TPB;                                      // chunks per thread
    static constexpr int GROUP = W / 4;                                        // lanes per row
};

template <int W, bool BWD>
__global__ __launch_bounds__(256) void layer_eval_vec(
    const float* __restrict__ W_, const float* __restrict__ bias, const float* __restrict__ z0,
    const float* __restrict__ Z, const float* __restrict__ G, float* __restrict__ A,
    float* __restrict__ r, float* __restrict__ dscale, unsigned* __restrict__ red, int B, int L,
    int layer, float alpha) {
    using S = EvalShape<W>;
    const int t = threadIdx.x;
    const long long row = (long long)blockIdx.x * S::ROWS_PER_WG + t / S::TPB;  // b*L + l
    if (!BWD && blockIdx.x == 0)
        for (int k = t; k < 2 * kRedShards; k += 256) red[k] = 0u;
    if (row >= (long long)B * L) return;
    const int l = (int)(row % L);
    const int b = (int)(row / L);
    const int tt = t % S::TPB;
    unsigned mr = 0u;  // forward: max |r| bits
    const float* zprev = (l == 0) ? z0 + (long long)b * W : Z + (row - 1) * W;
    const float* Wl = W_ + (long long)l * W * W;
    const int m_rev = L - l;  // reversed row of J_l (backward)
    float* Ab = BWD ? A + ((long long)b * L + m_rev) * W * W : A + row * W * W;
#pragma unroll
    for (int p = 0; p < S::CPT; ++p) {
        const int f = tt + S::TPB * p;
        const int i = f / S::GROUP;
        const int c4 = 4 * (f % S::GROUP);
        const v4f w4 = *reinterpret_cast<const v4f*>(Wl + i * W + c4);
        const v4f z4 = *reinterpret_cast<const v4f*>(zprev + c4);
        float part = w4[0] * z4[0];
        part = fmaf(w4[1], z4[1], part);
        part = fmaf(w4[2], z4[2], part);
        part = fmaf(w4[3], z4[3], part);
#pragma unroll
        for (int off = 1; off < S::GROUP; off <<= 1) part += __shfl_xor(part, off, 64);
        const float a = part + bias[(long long)l * W + i];
        float d;
        const float y = activate(layer, a, &d);
        const bool res = layer_residual(layer);
        const float dsc = res ? alpha * d : d;
        const bool lead = (f % S::GROUP) == 0;
        if (!BWD) {
            if (lead) {
                const float zi = zprev[i];
                const float fv = res ? fmaf(alpha, y, zi) : y;
                const float rv = fv - Z[row * W + i];
                r[row * W + i] = rv;
                mr = max(mr, __float_as_uint(fabsf(rv)));
            }
        } else if (lead) {
            dscale[row * W + i] = dsc;
            const int mr = L - 1 - l;
            r[((long long)b * L + mr) * W + i] = (mr == 0) ? G[(long long)b * W + i] : 0.f;
        }
        if (l >= 1 && A != nullptr) {
            v4f j4 = w4 * dsc;
            if (res && i >= c4 && i < c4 + 4) j4[i - c4] += 1.f;
            *reinterpret_cast<v4f*>(Ab + i * W + c4) = j4;
        }
    }
    if (!BWD) {
        // rows beyond B * L returned above with their whole wave (TPB >= 64)
        mr = wave_umax(mr);
        if ((t & 63) == 0) atomicMax(red + kRedF + (int)(row % kRedShards), mr);
    }
}

}  // namespace

template <int W, bool BWD>
hipError_t launch_eval_vec(const float* W_, const float* bias, const float* z0, const float* Z,
                           const float* G, float* A, float* r, float* dscale, unsigned* red, int B,
                           int L, int layer, float alpha, hipStream_t stream) {
    using S = EvalShape<W>;
    const long long rows = (long long)B * L;
    const long long grid = (rows + S::ROWS_PER_WG - 1) / S::ROWS_PER_WG;
    hipLaunchKernelGGL((layer_eval_vec<W, BWD>), dim3((unsigned)grid), dim3(256), 0, stream, W_,
                       bias, z0, Z, G, A, r, dscale, red, B, L, layer, alpha);
    return hipGetLastError();
}

hipError_t launch_forward_eval(const float* W, const float* bias, const float* z0,
                               const float* Z, float* A, float* r, unsigned* red,
                               int B, int L, int w, int layer, float alpha,
                               hipStream_t stream) {
    if (small_width(w))
        return launch_eval_small(false, W, bias, z0, Z, nullptr, A, r, nullptr, red, B, L, w,
                                 layer, alpha, stream);
    if (wide_width(w))
        return launch_forward_eval_wide(W, bias, z0, Z, A, r, red, B, L, w, layer, alpha, stream);
    switch (w) {
        case 16: return launch_eval_vec<16, false>(W, bias, z0, Z, nullptr, A, r, nullptr, red, B, L, layer, alpha, stream);
        case 32: return launch_eval_vec<32, false>(W, bias, z0, Z, nullptr, A, r, nullptr, red, B, L, layer, alpha, stream);
        case 64: return launch_eval_vec<64, false>(W, bias, z0, Z, nullptr, A, r, nullptr, red, B, L, layer, alpha, stream);
        case 128: return launch_eval_vec<128, false>(W, bias, z0, Z, nullptr, A, r, nullptr, red, B, L, layer, alpha, stream);
        default: break;
    }
    hipLaunchKernelGGL(forward_eval_kernel, dim3((unsigned)((long long)B * L)), dim3(kThreads), 0,
                       stream, W, bias, z0, Z, A, r, red, L, w, layer, alpha);
    return hipGetLastError();
}

bool backward_blocks_transposed(int w) {
    return small_width(w) || w == 16 || w == 32 || w == 64 || w == 128 || wide_width(w);
}

hipError_t launch_initial_guess(const float* W, const float* bias, const float* z0, float* Z,
                                int B, int L, int w, int layer, float alpha,
                                hipStream_t stream) {
    if (wide_width(w))
        return launch_initial_guess_wide(W, bias, z0, Z, B, L, w, layer, alpha, stream);
    const int rows_per_block = 64;
    const int chunks = (L + rows_per_block - 1) / rows_per_block;
    hipLaunchKernelGGL(initial_guess_kernel, dim3((unsigned)((long long)B * chunks)),
                       dim3(kThreads), 0, stream, W, bias, z0, Z, L, w, layer, alpha,
                       rows_per_block);
    return hipGetLastError();
}

hipError_t launch_update_reduce(float* Z, const float* x, long long n, unsigned* red,
                                hipStream_t stream) {
    long long blocks = (n + kThreads * 8 - 1) / (kThreads * 8);
    if (blocks > 4096) blocks = 4096;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(update_reduce_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, stream, Z,
                       x, n, red);
    return hipGetLastError();
}

hipError_t launch_backward_assemble(const float* W, const float* bias, const float* z0,
                                    const float* Z, const float* G, float* A, float* rrev,
                                    float* dscale, int B, int L, int w, int layer,
                                    float alpha, hipStream_t stream) {
    if (small_width(w))
        return launch_eval_small(true, W, bias, z0, Z, G, A, rrev, dscale, nullptr, B, L, w,
                                 layer, alpha, stream);
    if (wide_width(w))
        return launch_backward_assemble_wide(W, bias, z0, Z, G, A, rrev, dscale, B, L, w, layer,
                                             alpha, stream);
    if (A == nullptr && (w == 32 || w == 64 || w == 128)) {
        // no blocks to write: one workgroup per layer
        switch (w) {
            case 32: hipLaunchKernelGGL((bwd_scale_kernel<32>), dim3((unsigned)L), dim3(kThreads), 0, stream, W, bias, z0, Z, G, rrev, dscale, B, L, layer, alpha); break;
            case 64: hipLaunchKernelGGL((bwd_scale_kernel<64>), dim3((unsigned)L), dim3(kThreads), 0, stream, W, bias, z0, Z, G, rrev, dscale, B, L, layer, alpha); break;
            default: hipLaunchKernelGGL((bwd_scale_kernel<128>), dim3((unsigned)L), dim3(kThreads), 0, stream, W, bias, z0, Z, G, rrev, dscale, B, L, layer, alpha); break;
        }
        return hipGetLastError();
    }
    switch (w) {
        case 16: return launch_eval_vec<16, true>(W, bias, z0, Z, G, A, rrev, dscale, nullptr, B, L, layer, alpha, stream);
        case 32: return launch_eval_vec<32, true>(W, bias, z0, Z, G, A, rrev, dscale, nullptr, B, L, layer, alpha, stream);
        case 64: return launch_eval_vec<64, true>(W, bias, z0, Z, G, A, rrev, dscale, nullptr, B, L, layer, alpha, stream);
        case 128: return launch_eval_vec<128, true>(W, bias, z0, Z, G, A, rrev, dscale, nullptr, B, L, layer, alpha, stream);
        default: break;
    }
    hipLaunchKernelGGL(backward_assemble_kernel, dim3((unsigned)((long long)B * L)),
                       dim3(kThreads), 0, stream, W, bias, z0, Z, G, A, rrev, dscale, L, w,
                       layer, alpha);
    return hipGetLastError();
}

hipError_t launch_dz0(const float* W, const float* dscale, const float* Lambda, float* dz0,
                      int B, int L, int w, int layer, hipStream_t stream) {
    if (wide_width(w)) return launch_dz0_wide(W, dscale, Lambda, dz0, B, L, w, layer, stream);
    hipLaunchKernelGGL(dz0_kernel, dim3((unsigned)B), dim3(kThreads), 0, stream, W, dscale,
                       Lambda, dz0, L, w, layer);
    return hipGetLastError();
}

template <bool PRE>
hipError_t launch_wgrad_any(const float* z0, const float* Z, const float* dscale,
                            const float* Lambda, float* dW, float* db, int B, int L, int w,
                            int act, hipStream_t stream) {
    const dim3 grid((unsigned)L), blk(kThreads);
    switch (w) {
        case 16: hipLaunchKernelGGL((wgrad_tile_kernel<16, PRE>), grid, blk, 0, stream, z0, Z, dscale, Lambda, dW, db, B, L, act); break;
        case 32: hipLaunchKernelGGL((wgrad_tile_kernel<32, PRE>), grid, blk, 0, stream, z0, Z, dscale, Lambda, dW, db, B, L, act); break;
        case 64: hipLaunchKernelGGL((wgrad_tile_kernel<64, PRE>), grid, blk, 0, stream, z0, Z, dscale, Lambda, dW, db, B, L, act); break;
        case 128: hipLaunchKernelGGL((wgrad_tile_kernel<128, PRE>), grid, blk, 0, stream, z0, Z, dscale, Lambda, dW, db, B, L, act); break;
        default:
            if (w <= 8) {
                const long long n = (long long)L * w * w;
                hipLaunchKernelGGL((wgrad_small_kernel<PRE>), dim3((unsigned)((n + kThreads - 1) / kThreads)), blk, 0, stream, z0, Z, dscale, Lambda, dW, db, B, L, w, act);
            } else {
                hipLaunchKernelGGL((wgrad_kernel<PRE>), grid, blk, 0, stream, z0, Z, dscale, Lambda, dW, db, B, L, w, act);
            }
            break;
    }
    return hipGetLastError();
}

hipError_t launch_wgrad(const float* z0, const float* Z, const float* dscale,
                        const float* Lambda, float* dW, float* db, int B, int L, int w,
                        hipStream_t stream) {
    if (wide_width(w)) return launch_wgrad_wide(z0, Z, dscale, Lambda, dW, db, B, L, w, stream);
    return launch_wgrad_any<false>(z0, Z, dscale, Lambda, dW, db, B, L, w, 0, stream);
}

hipError_t launch_wgrad_pre(const float* z0, const float* Z, const float* Lambda, float* dW,
                            float* db, int B, int L, int w, int act, hipStream_t stream) {
    return launch_wgrad_any<true>(z0, Z, nullptr, Lambda, dW, db, B, L, w, act, stream);
}

hipError_t launch_residual(const float* F, const float* Z, float* r, long long n, unsigned* red,
                           hipStream_t stream) {
    long long blocks = (n + kThreads - 1) / kThreads;
    if (blocks > 4096) blocks = 4096;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(residual_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, stream, F, Z, r,
                       n, red);
    return hipGetLastError();
}

hipError_t launch_zero_words(unsigned* p, int n, hipStream_t stream) {
    hipLaunchKernelGGL(zero_words_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, stream, p, n);
    return hipGetLastError();
}

hipError_t launch_measures(const unsigned* red, unsigned* out, unsigned seq, hipStream_t stream) {
    hipLaunchKernelGGL(measures_kernel, dim3(1), dim3(kRedShards), 0, stream, red, out, seq);
    return hipGetLastError();
}

hipError_t launch_copy_rows(const VecSrc& src, const VecDst& dst, int B, int L, int w,
                            hipStream_t stream) {
    hipLaunchKernelGGL(copy_rows_kernel, dim3((unsigned)((long long)B * L)), dim3(kThreads), 0,
                       stream, src, dst, L, w);
    return hipGetLastError();
}

}  // namespace deeppcr
