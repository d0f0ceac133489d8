// Sequential layer-by-layer passes on the GPU: the baseline DeepPCR is
// compared against (Sec. 4.1: the forward pass applied one layer after the
// other, and the backward pass as back substitution of Eq. 11).  Each system
// of the batch is walked by one workgroup, layer after layer; the layers of a
// system are inherently sequential, so only the batch is parallel.  Two launch
// shapes: all layers in one launch (no per-layer launch cost), or one launch
// per layer (the shape of an eager framework's layer loop).
#include "internal.h"

#include <type_traits>

namespace deeppcr {
namespace {

constexpr int kThreads = 256;

// Thread layout for w-wide mat-vecs: TPR threads share one row (a power of
// two <= 64, so a row's partial sums reduce inside a wave).
struct RowMap {
    int tpr, rows_per_pass, cols;
};

__device__ inline RowMap row_map(int w) {
    int tpr = 1;
    while (tpr * 2 * w <= kThreads && tpr * 2 <= 64) tpr *= 2;
    RowMap m;
    m.tpr = tpr;
    m.rows_per_pass = kThreads / tpr;
    m.cols = (w + tpr - 1) / tpr;
    return m;
}

// out[i] = sum_j M[i][j] v[j] (+ add[i]) for rows i < w, M row-major; v in LDS.
// Every lane of a row group ends with the full sum; returns through `out`.
__device__ inline void rows_dot(const float* __restrict__ M, const float* v, float* out, int w,
                                const RowMap& m) {
    const int t = threadIdx.x;
    const int sub = t % m.tpr;
    for (int i0 = 0; i0 < w; i0 += m.rows_per_pass) {
        const int i = i0 + t / m.tpr;
        float acc = 0.f;
        if (i < w)
            for (int c = 0; c < m.cols; ++c) {
                const int j = sub + c * m.tpr;
                if (j < w) acc = fmaf(M[(long long)i * w + j], v[j], acc);
            }
        for (int off = 1; off < m.tpr; off <<= 1) acc += __shfl_xor(acc, off, 64);
        if (i < w && sub == 0) out[i] = acc;
    }
}

// out[j] = sum_i M[i][j] g[i] for columns j < w (the transposed mat-vec).
__device__ inline void cols_dot(const float* __restrict__ M, const float* g, float* out, int w,
                                const RowMap& m) {
    const int t = threadIdx.x;
    const int sub = t % m.tpr;
    for (int j0 = 0; j0 < w; j0 += m.rows_per_pass) {
        const int j = j0 + t / m.tpr;
        float acc = 0.f;
        if (j < w)
            for (int c = 0; c < m.cols; ++c) {
                const int i = sub + c * m.tpr;
                if (i < w) acc = fmaf(M[(long long)i * w + j], g[i], acc);
            }
        for (int off = 1; off < m.tpr; off <<= 1) acc += __shfl_xor(acc, off, 64);
        if (j < w && sub == 0) out[j] = acc;
    }
}

__global__ __launch_bounds__(kThreads) void seq_forward_kernel(
    const float* __restrict__ W, const float* __restrict__ bias, const float* __restrict__ z0,
    float* __restrict__ Z, int L, int w, int layer, float alpha, int l0, int l1) {
    const int b = blockIdx.x;
    __shared__ float z[kMaxWidth], a[kMaxWidth];
    const RowMap m = row_map(w);
    const bool res = layer_residual(layer);
    for (int i = threadIdx.x; i < w; i += kThreads)
        z[i] = (l0 == 0) ? z0[(long long)b * w + i] : Z[((long long)b * L + l0 - 1) * w + i];
    __syncthreads();
    for (int l = l0; l < l1; ++l) {
        rows_dot(W + (long long)l * w * w, z, a, w, m);
        __syncthreads();
        for (int i = threadIdx.x; i < w; i += kThreads) {
            float d;
            const float y = activate(layer, a[i] + bias[(long long)l * w + i], &d);
            const float f = res ? fmaf(alpha, y, z[i]) : y;
            z[i] = f;
            Z[((long long)b * L + l) * w + i] = f;
        }
        __syncthreads();
    }
}

// Adjoints lambda_{l-1} = J_l^T lambda_l for l = l1-1 down to l0, starting from
// lambda_{l1-1} (G when l1 = L, else Lambda[:, l1-1]); writes Lambda[:, l-1]
// and, at l = 0, dz0.
__global__ __launch_bounds__(kThreads) void seq_backward_kernel(
    const float* __restrict__ W, const float* __restrict__ bias, const float* __restrict__ z0,
    const float* __restrict__ Z, const float* __restrict__ G, float* __restrict__ Lambda,
    float* __restrict__ dz0, int L, int w, int layer, float alpha, int l0, int l1) {
    const int b = blockIdx.x;
    __shared__ float lam[kMaxWidth], zp[kMaxWidth], a[kMaxWidth], g[kMaxWidth], nl[kMaxWidth];
    const RowMap m = row_map(w);
    const bool res = layer_residual(layer);
    for (int i = threadIdx.x; i < w; i += kThreads) {
        const float v = (l1 == L) ? G[(long long)b * w + i] : Lambda[((long long)b * L + l1 - 1) * w + i];
        lam[i] = v;
        if (l1 == L) Lambda[((long long)b * L + L - 1) * w + i] = v;
    }
    for (int l = l1 - 1; l >= l0; --l) {
        for (int i = threadIdx.x; i < w; i += kThreads)
            zp[i] = (l == 0) ? z0[(long long)b * w + i] : Z[((long long)b * L + l - 1) * w + i];
        __syncthreads();
        const float* Wl = W + (long long)l * w * w;
        rows_dot(Wl, zp, a, w, m);
        __syncthreads();
        for (int i = threadIdx.x; i < w; i += kThreads) {
            float d;
            activate(layer, a[i] + bias[(long long)l * w + i], &d);
            g[i] = (res ? alpha * d : d) * lam[i];
        }
        __syncthreads();
        cols_dot(Wl, g, nl, w, m);
        __syncthreads();
        for (int i = threadIdx.x; i < w; i += kThreads) {
            const float v = res ? lam[i] + nl[i] : nl[i];
            lam[i] = v;
            if (l >= 1)
                Lambda[((long long)b * L + l - 1) * w + i] = v;
            else
                dz0[(long long)b * w + i] = v;
        }
        __syncthreads();
    }
}

// Collapsed-skip ResNet, sequentially: Z_j = W_j sigma(Z_{j-1}) + b_j, plus
// Z_{j-s} when (j+1) % s == 0, for layers l0 .. l1-1 (reading Z[:, l0-1] and
// the block input Z[:, s*(l0/s) - 1], or z0).  The skip source (the last
// block output) stays in LDS between layers.
__global__ __launch_bounds__(kThreads) void resnet_seq_forward_kernel(
    const float* __restrict__ W, const float* __restrict__ bias, const float* __restrict__ z0,
    float* __restrict__ Z, int L, int w, int skip, int act, int l0, int l1) {
    const int b = blockIdx.x;
    __shared__ float z[kMaxWidth], xs[kMaxWidth], sg[kMaxWidth], a[kMaxWidth];
    const RowMap m = row_map(w);
    const int src = (l0 / skip) * skip - 1;  // the current block's input row
    for (int i = threadIdx.x; i < w; i += kThreads) {
        z[i] = (l0 == 0) ? z0[(long long)b * w + i] : Z[((long long)b * L + l0 - 1) * w + i];
        xs[i] = (src < 0) ? z0[(long long)b * w + i] : Z[((long long)b * L + src) * w + i];
    }
    for (int l = l0; l < l1; ++l) {
        __syncthreads();
        for (int i = threadIdx.x; i < w; i += kThreads) {
            float d;
            sg[i] = activate(2 * act, z[i], &d);
        }
        __syncthreads();
        rows_dot(W + (long long)l * w * w, sg, a, w, m);
        __syncthreads();
        const bool sk = (l + 1) % skip == 0;
        for (int i = threadIdx.x; i < w; i += kThreads) {
            const float v = a[i] + bias[(long long)l * w + i] + (sk ? xs[i] : 0.f);
            z[i] = v;
            Z[((long long)b * L + l) * w + i] = v;
            if (sk) xs[i] = v;
        }
    }
}

// Its reverse-mode pass over layers l1-1 down to l0, starting from
// lambda_{l1-1} (G when l1 = L, else Lambda[:, l1-1]): Lambda[:, j] =
// dLoss/dZ_j; layer j sends diag(sigma'(Z_{j-1})) W_j^T lambda_j to Z_{j-1},
// and the first layer of a block adds to it the adjoint the block's skip
// layer (row j+s-1, already final) sends to the block input; dz0 at l = 0.
__global__ __launch_bounds__(kThreads) void resnet_seq_backward_kernel(
    const float* __restrict__ W, const float* __restrict__ z0, const float* __restrict__ Z,
    const float* __restrict__ G, float* __restrict__ Lambda, float* __restrict__ dz0, int L, int w,
    int skip, int act, int l0, int l1) {
    const int b = blockIdx.x;
    __shared__ float lam[kMaxWidth], ds[kMaxWidth], nl[kMaxWidth];
    const RowMap m = row_map(w);
    float* Lb = Lambda + (long long)b * L * w;
    for (int i = threadIdx.x; i < w; i += kThreads) {
        const float v = (l1 == L) ? G[(long long)b * w + i] : Lb[(long long)(l1 - 1) * w + i];
        lam[i] = v;
        if (l1 == L) Lb[(long long)(L - 1) * w + i] = v;
    }
    for (int l = l1 - 1; l >= l0; --l) {
        __syncthreads();
        for (int i = threadIdx.x; i < w; i += kThreads) {
            const float zin = (l == 0) ? z0[(long long)b * w + i] : Z[((long long)b * L + l - 1) * w + i];
            float d;
            activate(2 * act, zin, &d);
            ds[i] = d;
        }
        __syncthreads();
        cols_dot(W + (long long)l * w * w, lam, nl, w, m);
        __syncthreads();
        const bool first = l % skip == 0;  // first layer of a block: its input took the skip
        for (int i = threadIdx.x; i < w; i += kThreads) {
            // the same thread wrote row l + skip - 1 of Lambda earlier
            const float v = nl[i] * ds[i] + (first ? Lb[(long long)(l + skip - 1) * w + i] : 0.f);
            if (l >= 1) {
                lam[i] = v;
                Lb[(long long)(l - 1) * w + i] = v;
            } else {
                dz0[(long long)b * w + i] = v;
            }
        }
    }
}

// ---- w = 16, 32, 64, 128: the weights streamed ahead of the walk -----------
// The layers' weights do not depend on the state, so each w x w block is
// requested NB - 1 layers before its layer into a ring of register slots
// (every thread a w^2/256 share, slot k % NB for the walk's k-th layer) and
// moved into one of two LDS buffers at the end of the layer before its own;
// a layer's mat-vecs then read LDS only.  The state rows a layer reads
// (backward: Z_{l-1}) come through the same ring.  Requests past the walk's
// end are clamped to its last layer and never used, so that every thread
// issues the same loads on every layer.

template <int I, int N, class F>
__device__ __forceinline__ void each_slot(F& f) {
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        each_slot<I + 1, N>(f);
    }
}

template <int W>
struct Stream {
    static constexpr int PER = W * W / kThreads;  // floats of a block per thread
    static constexpr int NB = W <= 32 ? 8 : W == 64 ? 4 : 2;
};

// step(k, U) for k = 0 .. count-1, U = integral_constant<k % NB>.  Whole
// trips of NB steps run unguarded, so that the compiler sees every step's
// loads issued and can wait for just the one it needs; only the last partial
// trip is guarded.
template <int NB, class F>
__device__ __forceinline__ void walk(int count, F& step) {
    int k0 = 0;
    for (; k0 + NB <= count; k0 += NB) {
        auto trip = [&](auto U) { step(k0 + decltype(U)::value, U); };
        each_slot<0, NB>(trip);
    }
    auto rest = [&](auto U) {
        const int k = k0 + decltype(U)::value;
        if (k < count) step(k, U);
    };
    each_slot<0, NB>(rest);
}

template <int W>
__device__ __forceinline__ void block_to_regs(const float* __restrict__ blk,
                                              float (&r)[Stream<W>::PER]) {
#pragma unroll
    for (int p = 0; p < Stream<W>::PER; ++p) r[p] = blk[threadIdx.x + kThreads * p];
}

// The LDS copy has rows of pitch w + 1, so that the lanes of a row-wise dot
// product (rows i, i + 1, ... at the same column) fall into different banks.
template <int W>
__device__ __forceinline__ void regs_to_lds(const float (&r)[Stream<W>::PER], float* lds) {
#pragma unroll
    for (int p = 0; p < Stream<W>::PER; ++p) {
        const int idx = threadIdx.x + kThreads * p;
        lds[(idx / W) * (W + 1) + idx % W] = r[p];
    }
}

// rows_dot / cols_dot on the padded LDS copy, four partial sums per lane.
template <int W>
__device__ __forceinline__ void rows_dot_p(const float* M, const float* v, float* out) {
    const RowMap m = row_map(W);
    const int t = threadIdx.x;
    const int sub = t % m.tpr;
    for (int i0 = 0; i0 < W; i0 += m.rows_per_pass) {
        const int i = i0 + t / m.tpr;
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
        if (i < W)
            for (int c = 0; c < m.cols; ++c) {
                const int j = sub + c * m.tpr;
                if (j < W) acc[c & 3] = fmaf(M[i * (W + 1) + j], v[j], acc[c & 3]);
            }
        float sum = (acc[0] + acc[1]) + (acc[2] + acc[3]);
        for (int off = 1; off < m.tpr; off <<= 1) sum += __shfl_xor(sum, off, 64);
        if (i < W && sub == 0) out[i] = sum;
    }
}

template <int W>
__device__ __forceinline__ void cols_dot_p(const float* M, const float* g, float* out) {
    const RowMap m = row_map(W);
    const int t = threadIdx.x;
    const int sub = t % m.tpr;
    for (int j0 = 0; j0 < W; j0 += m.rows_per_pass) {
        const int j = j0 + t / m.tpr;
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
        if (j < W)
            for (int c = 0; c < m.cols; ++c) {
                const int i = sub + c * m.tpr;
                if (i < W) acc[c & 3] = fmaf(M[i * (W + 1) + j], g[i], acc[c & 3]);
            }
        float sum = (acc[0] + acc[1]) + (acc[2] + acc[3]);
        for (int off = 1; off < m.tpr; off <<= 1) sum += __shfl_xor(sum, off, 64);
        if (j < W && sub == 0) out[j] = sum;
    }
}

// As seq_forward_kernel (MLP layers), layers l0 .. l1-1.
template <int W>
__global__ __launch_bounds__(kThreads) void seq_forward_stream(
    const float* __restrict__ Wt, const float* __restrict__ bias, const float* __restrict__ z0,
    float* __restrict__ Z, int L, int layer, float alpha, int l0, int l1) {
    using SS = Stream<W>;
    constexpr int NB = SS::NB;
    __shared__ float Ws[2][W * (W + 1)];
    __shared__ float z[W], a[W];
    const int b = blockIdx.x, t = threadIdx.x;
    const bool res = layer_residual(layer);
    const int count = l1 - l0;
    if (count <= 0) return;  // uniform over the workgroup
    const int tw = t & (W - 1);
    float rg[NB][SS::PER], bq[NB];  // blocks and bias rows, slot k % NB
    auto lay = [&](int k) { return l0 + min(k, count - 1); };
    auto blk = [&](int k) { return Wt + (long long)lay(k) * W * W; };
    auto bia = [&](int k) { return bias[(long long)lay(k) * W + tw]; };
    block_to_regs<W>(blk(0), rg[0]);
    regs_to_lds<W>(rg[0], Ws[0]);
    auto pro = [&](auto J) {
        constexpr int j = decltype(J)::value;
        if constexpr (j >= 1) block_to_regs<W>(blk(j), rg[j]);
        bq[j] = bia(j);
    };
    each_slot<0, NB>(pro);
    for (int i = t; i < W; i += kThreads)
        z[i] = (l0 == 0) ? z0[(long long)b * W + i] : Z[((long long)b * L + l0 - 1) * W + i];
    __syncthreads();
    auto step = [&](int k, auto U) {
        constexpr int u = decltype(U)::value;
        const int l = l0 + k;
        const float bl = bq[u];
        block_to_regs<W>(blk(k + NB), rg[u]);
        bq[u] = bia(k + NB);
        rows_dot_p<W>(Ws[k & 1], z, a);
        __syncthreads();
        if (t < W) {
            float d;
            const float y = activate(layer, a[t] + bl, &d);
            const float f = res ? fmaf(alpha, y, z[t]) : y;
            z[t] = f;
            Z[((long long)b * L + l) * W + t] = f;
        }
        regs_to_lds<W>(rg[(u + 1) % NB], Ws[(k + 1) & 1]);
        __syncthreads();
    };
    walk<NB>(count, step);
}

// As seq_backward_kernel, layers l1-1 down to l0.
template <int W>
__global__ __launch_bounds__(kThreads) void seq_backward_stream(
    const float* __restrict__ Wt, const float* __restrict__ bias, const float* __restrict__ z0,
    const float* __restrict__ Z, const float* __restrict__ G, float* __restrict__ Lambda,
    float* __restrict__ dz0, int L, int layer, float alpha, int l0, int l1) {
    using SS = Stream<W>;
    constexpr int NB = SS::NB;
    __shared__ float Ws[2][W * (W + 1)];
    __shared__ float lam[W], zp[W], a[W], g[W], nl[W];
    const int b = blockIdx.x, t = threadIdx.x;
    const bool res = layer_residual(layer);
    const int count = l1 - l0;
    if (count <= 0) return;  // uniform over the workgroup
    const int tw = t & (W - 1);
    float rg[NB][SS::PER], zq[NB], bq[NB];
    // the k-th layer of the walk is l1-1-k; its block, bias and input row Z_{l-1}
    auto lay = [&](int k) { return l1 - 1 - min(k, count - 1); };
    auto blk = [&](int k) { return Wt + (long long)lay(k) * W * W; };
    auto bia = [&](int k) { return bias[(long long)lay(k) * W + tw]; };
    auto zin = [&](int k) {
        const int l = lay(k);
        return (l == 0) ? z0[(long long)b * W + tw] : Z[((long long)b * L + l - 1) * W + tw];
    };
    block_to_regs<W>(blk(0), rg[0]);
    regs_to_lds<W>(rg[0], Ws[0]);
    auto pro = [&](auto J) {
        constexpr int j = decltype(J)::value;
        if constexpr (j >= 1) block_to_regs<W>(blk(j), rg[j]);
        zq[j] = zin(j);
        bq[j] = bia(j);
    };
    each_slot<0, NB>(pro);
    for (int i = t; i < W; i += kThreads) {
        const float v = (l1 == L) ? G[(long long)b * W + i] : Lambda[((long long)b * L + l1 - 1) * W + i];
        lam[i] = v;
        if (l1 == L) Lambda[((long long)b * L + L - 1) * W + i] = v;
    }
    auto step = [&](int k, auto U) {
        constexpr int u = decltype(U)::value;
        const int l = l1 - 1 - k;
        if (t < W) zp[t] = zq[u];
        const float bl = bq[u];
        block_to_regs<W>(blk(k + NB), rg[u]);
        zq[u] = zin(k + NB);
        bq[u] = bia(k + NB);
        __syncthreads();
        const float* Wl = Ws[k & 1];
        rows_dot_p<W>(Wl, zp, a);
        __syncthreads();
        if (t < W) {
            float d;
            activate(layer, a[t] + bl, &d);
            g[t] = (res ? alpha * d : d) * lam[t];
        }
        __syncthreads();
        cols_dot_p<W>(Wl, g, nl);
        __syncthreads();
        if (t < W) {
            const float v = res ? lam[t] + nl[t] : nl[t];
            lam[t] = v;
            if (l >= 1)
                Lambda[((long long)b * L + l - 1) * W + t] = v;
            else
                dz0[(long long)b * W + t] = v;
        }
        regs_to_lds<W>(rg[(u + 1) % NB], Ws[(k + 1) & 1]);
        __syncthreads();
    };
    walk<NB>(count, step);
}

// As resnet_seq_forward_kernel, layers l0 .. l1-1.
template <int W>
__global__ __launch_bounds__(kThreads) void resnet_seq_forward_stream(
    const float* __restrict__ Wt, const float* __restrict__ bias, const float* __restrict__ z0,
    float* __restrict__ Z, int L, int skip, int act, int l0, int l1) {
    using SS = Stream<W>;
    constexpr int NB = SS::NB;
    __shared__ float Ws[2][W * (W + 1)];
    __shared__ float z[W], xs[W], sg[W], a[W];
    const int b = blockIdx.x, t = threadIdx.x;
    const int count = l1 - l0;
    if (count <= 0) return;  // uniform over the workgroup
    const int src = (l0 / skip) * skip - 1;  // the current block's input row
    const int tw = t & (W - 1);
    float rg[NB][SS::PER], bq[NB];
    auto lay = [&](int k) { return l0 + min(k, count - 1); };
    auto blk = [&](int k) { return Wt + (long long)lay(k) * W * W; };
    auto bia = [&](int k) { return bias[(long long)lay(k) * W + tw]; };
    block_to_regs<W>(blk(0), rg[0]);
    regs_to_lds<W>(rg[0], Ws[0]);
    auto pro = [&](auto J) {
        constexpr int j = decltype(J)::value;
        if constexpr (j >= 1) block_to_regs<W>(blk(j), rg[j]);
        bq[j] = bia(j);
    };
    each_slot<0, NB>(pro);
    for (int i = t; i < W; i += kThreads) {
        z[i] = (l0 == 0) ? z0[(long long)b * W + i] : Z[((long long)b * L + l0 - 1) * W + i];
        xs[i] = (src < 0) ? z0[(long long)b * W + i] : Z[((long long)b * L + src) * W + i];
    }
    auto step = [&](int k, auto U) {
        constexpr int u = decltype(U)::value;
        const int l = l0 + k;
        const float bl = bq[u];
        block_to_regs<W>(blk(k + NB), rg[u]);
        bq[u] = bia(k + NB);
        __syncthreads();
        if (t < W) {
            float d;
            sg[t] = activate(2 * act, z[t], &d);
        }
        __syncthreads();
        rows_dot_p<W>(Ws[k & 1], sg, a);
        __syncthreads();
        const bool sk = (l + 1) % skip == 0;
        if (t < W) {
            const float v = a[t] + bl + (sk ? xs[t] : 0.f);
            z[t] = v;
            Z[((long long)b * L + l) * W + t] = v;
            if (sk) xs[t] = v;
        }
        regs_to_lds<W>(rg[(u + 1) % NB], Ws[(k + 1) & 1]);
    };
    walk<NB>(count, step);
}

// As resnet_seq_backward_kernel, layers l1-1 down to l0.
template <int W>
__global__ __launch_bounds__(kThreads) void resnet_seq_backward_stream(
    const float* __restrict__ Wt, const float* __restrict__ z0, const float* __restrict__ Z,
    const float* __restrict__ G, float* __restrict__ Lambda, float* __restrict__ dz0, int L,
    int skip, int act, int l0, int l1) {
    using SS = Stream<W>;
    constexpr int NB = SS::NB;
    __shared__ float Ws[2][W * (W + 1)];
    __shared__ float lam[W], ds[W], nl[W];
    const int b = blockIdx.x, t = threadIdx.x;
    const int count = l1 - l0;
    if (count <= 0) return;  // uniform over the workgroup
    const int tw = t & (W - 1);
    float* Lb = Lambda + (long long)b * L * W;
    float rg[NB][SS::PER], zq[NB];
    auto lay = [&](int k) { return l1 - 1 - min(k, count - 1); };
    auto blk = [&](int k) { return Wt + (long long)lay(k) * W * W; };
    auto zin = [&](int k) {
        const int l = lay(k);
        return (l == 0) ? z0[(long long)b * W + tw] : Z[((long long)b * L + l - 1) * W + tw];
    };
    block_to_regs<W>(blk(0), rg[0]);
    regs_to_lds<W>(rg[0], Ws[0]);
    zq[0] = zin(0);
    auto pro = [&](auto J) {
        constexpr int j = decltype(J)::value;
        if constexpr (j >= 1) {
            block_to_regs<W>(blk(j), rg[j]);
            zq[j] = zin(j);
        }
    };
    each_slot<0, NB>(pro);
    // xsk: the adjoint of the current block's last row (its skip source),
    // which the block's first layer adds; kept from when it was written
    float xsk = 0.f;
    if (t < W) {
        const float v = (l1 == L) ? G[(long long)b * W + t] : Lb[(long long)(l1 - 1) * W + t];
        lam[t] = v;
        xsk = v;
        if (l1 == L) Lb[(long long)(L - 1) * W + t] = v;
    }
    auto step = [&](int k, auto U) {
        constexpr int u = decltype(U)::value;
        const int l = l1 - 1 - k;
        const float zv = zq[u];
        block_to_regs<W>(blk(k + NB), rg[u]);
        zq[u] = zin(k + NB);
        __syncthreads();
        if (t < W) {
            float d;
            activate(2 * act, zv, &d);
            ds[t] = d;
        }
        __syncthreads();
        cols_dot_p<W>(Ws[k & 1], lam, nl);
        __syncthreads();
        const bool first = l % skip == 0;  // first layer of a block: its input took the skip
        if (t < W) {
            // the first layer of a block adds the adjoint of the block's last
            // row l + skip - 1 (<= L - 1 only for a first layer): written by
            // this thread in this launch (then xsk holds it), or, in a launch
            // that starts below it, earlier
            float sa = 0.f;
            if (first)
                sa = l + skip - 1 <= l1 - 1 ? xsk : Lb[(long long)min(l + skip - 1, L - 1) * W + t];
            const float v = nl[t] * ds[t] + sa;
            if (l >= 1) {
                lam[t] = v;
                Lb[(long long)(l - 1) * W + t] = v;
                if (l % skip == 0) xsk = v;  // row l - 1 ends the block below
            } else {
                dz0[(long long)b * W + t] = v;
            }
        }
        regs_to_lds<W>(rg[(u + 1) % NB], Ws[(k + 1) & 1]);
    };
    walk<NB>(count, step);
}

// ---- w = 2 .. 64: one wave per system -------------------------------------
// (forward at w = 2 .. 64, backward at w = 2 .. 32: at w = 64 the
// backward's transposed product, one column per lane over all rows, made the
// one-wave version slower than the workgroup one, 29 against 22 ms at
// L = 16384)
// Lane group i (64/w lanes) holds row i of each layer's block, w^2/64
// columns per lane, in a ring of register slots requested NB - 1 layers
// ahead (with the bias); the state lives in the wave's LDS, so a layer costs
// one wave-level barrier.  The backward also puts each block into LDS for the
// transposed product.
template <int W>
struct WaveSeq {
    static constexpr int LPR = W >= 16 ? 64 / W : W;  // lanes per row
    static constexpr int CPL = W / LPR;               // columns per lane
    static constexpr int RL = W * LPR;                // lanes that hold a row (64 from w = 8)
    static constexpr int NB = W <= 16 ? 16 : W == 32 ? 8 : 4;
};


template <int W>
__device__ __forceinline__ void row_to_regs(const float* __restrict__ blk, int i, int c0,
                                            float (&r)[WaveSeq<W>::CPL]) {
    const float* src = blk + i * W + c0;
    if constexpr (WaveSeq<W>::CPL % 4 == 0) {
#pragma unroll
        for (int c = 0; c < WaveSeq<W>::CPL; c += 4) {
            const float4 x = *reinterpret_cast<const float4*>(src + c);
            r[c] = x.x;
            r[c + 1] = x.y;
            r[c + 2] = x.z;
            r[c + 3] = x.w;
        }
    } else {
#pragma unroll
        for (int c = 0; c < WaveSeq<W>::CPL; ++c) r[c] = src[c];
    }
}

// sum over the row of (registers) x (vector in LDS); every lane of the row
// group receives it
template <int W>
__device__ __forceinline__ float wave_row_dot(const float (&r)[WaveSeq<W>::CPL], const float* v,
                                              int c0) {
    constexpr int CPL = WaveSeq<W>::CPL;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < CPL; ++c) acc[c & 3] = fmaf(r[c], v[c0 + c], acc[c & 3]);
    float sum = (acc[0] + acc[1]) + (acc[2] + acc[3]);
#pragma unroll
    for (int off = 1; off < WaveSeq<W>::LPR; off <<= 1) sum += __shfl_xor(sum, off, 64);
    return sum;
}

// As seq_forward_kernel, one wave per system.
template <int W>
__global__ __launch_bounds__(64) void seq_forward_wave(
    const float* __restrict__ Wt, const float* __restrict__ bias, const float* __restrict__ z0,
    float* __restrict__ Z, int L, int layer, float alpha, int l0, int l1) {
    using SQ = WaveSeq<W>;
    constexpr int NB = SQ::NB;
    __shared__ float z[2][W];
    const int b = blockIdx.x, lane = threadIdx.x;
    // lanes past the rows (w < 8) read the last row again and write nothing
    const int i = min(lane / SQ::LPR, W - 1), c0 = (lane % SQ::LPR) * SQ::CPL;
    const bool lead = lane % SQ::LPR == 0 && lane < SQ::RL;
    const bool res = layer_residual(layer);
    const int count = l1 - l0;
    if (count <= 0) return;
    float wr[NB][SQ::CPL], bq[NB];
    auto lay = [&](int k) { return l0 + min(k, count - 1); };
    auto load = [&](int k, float (&r)[SQ::CPL], float& bb) {
        const int l = lay(k);
        row_to_regs<W>(Wt + (long long)l * W * W, i, c0, r);
        bb = bias[(long long)l * W + i];
    };
    auto pro = [&](auto J) {
        constexpr int j = decltype(J)::value;
        load(j, wr[j], bq[j]);
    };
    each_slot<0, NB>(pro);
    if (lane < W)
        z[0][lane] = (l0 == 0) ? z0[(long long)b * W + lane] : Z[((long long)b * L + l0 - 1) * W + lane];
    auto step = [&](int k, auto U) {
        constexpr int u = decltype(U)::value;
        const int l = l0 + k;
        const float* zc = z[k & 1];
        wave_sync();
        const float a = wave_row_dot<W>(wr[u], zc, c0) + bq[u];
        load(k + NB, wr[u], bq[u]);
        float d;
        const float y = activate(layer, a, &d);
        const float f = res ? fmaf(alpha, y, zc[i]) : y;
        if (lead) {
            z[(k + 1) & 1][i] = f;
            Z[((long long)b * L + l) * W + i] = f;
        }
    };
    walk<NB>(count, step);
}

// As seq_backward_kernel, one wave per system.
template <int W>
__global__ __launch_bounds__(64) void seq_backward_wave(
    const float* __restrict__ Wt, const float* __restrict__ bias, const float* __restrict__ z0,
    const float* __restrict__ Z, const float* __restrict__ G, float* __restrict__ Lambda,
    float* __restrict__ dz0, int L, int layer, float alpha, int l0, int l1) {
    using SQ = WaveSeq<W>;
    constexpr int NB = SQ::NB;
    __shared__ float Wl[W * (W + 1)];  // the current block, rows of pitch w + 1
    __shared__ float zp[W], g[W], lam[W];
    const int b = blockIdx.x, lane = threadIdx.x;
    // lanes past the rows (w < 8) read the last row again and write nothing
    const int i = min(lane / SQ::LPR, W - 1), c0 = (lane % SQ::LPR) * SQ::CPL;
    const bool lead = lane % SQ::LPR == 0 && lane < SQ::RL;
    const bool res = layer_residual(layer);
    const int count = l1 - l0;
    if (count <= 0) return;
    const int tw = lane & (W - 1);
    float wr[NB][SQ::CPL], bq[NB], zq[NB];
    auto lay = [&](int k) { return l1 - 1 - min(k, count - 1); };
    auto load = [&](int k, float (&r)[SQ::CPL], float& bb, float& zz) {
        const int l = lay(k);
        row_to_regs<W>(Wt + (long long)l * W * W, i, c0, r);
        bb = bias[(long long)l * W + i];
        zz = (l == 0) ? z0[(long long)b * W + tw] : Z[((long long)b * L + l - 1) * W + tw];
    };
    auto pro = [&](auto J) {
        constexpr int j = decltype(J)::value;
        load(j, wr[j], bq[j], zq[j]);
    };
    each_slot<0, NB>(pro);
    if (lane < W) {
        const float v = (l1 == L) ? G[(long long)b * W + lane] : Lambda[((long long)b * L + l1 - 1) * W + lane];
        lam[lane] = v;
        if (l1 == L) Lambda[((long long)b * L + L - 1) * W + lane] = v;
    }
    auto step = [&](int k, auto U) {
        constexpr int u = decltype(U)::value;
        const int l = l1 - 1 - k;
        wave_sync();  // the previous layer's reads of Wl, zp, g and lam are done
        if (lane < W) zp[lane] = zq[u];
        if (lane < SQ::RL) {
#pragma unroll
            for (int c = 0; c < SQ::CPL; ++c) Wl[i * (W + 1) + c0 + c] = wr[u][c];
        }
        wave_sync();
        const float a = wave_row_dot<W>(wr[u], zp, c0) + bq[u];
        load(k + NB, wr[u], bq[u], zq[u]);
        float d;
        activate(layer, a, &d);
        if (lead) g[i] = (res ? alpha * d : d) * lam[i];
        wave_sync();
        // column j = lane (w <= 64 lanes): sum over the rows of Wl[r][j] g[r]
        if (lane < W) {
            float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int r = 0; r < W; ++r) acc[r & 3] = fmaf(Wl[r * (W + 1) + lane], g[r], acc[r & 3]);
            const float nl = (acc[0] + acc[1]) + (acc[2] + acc[3]);
            const float v = res ? lam[lane] + nl : nl;
            if (l >= 1)
                Lambda[((long long)b * L + l - 1) * W + lane] = v;
            else
                dz0[(long long)b * W + lane] = v;
            lam[lane] = v;  // this lane alone read lam[lane] above
        }
    };
    walk<NB>(count, step);
}

// As resnet_seq_forward_kernel, one wave per system (w = 16, 32).
template <int W>
__global__ __launch_bounds__(64) void resnet_seq_forward_wave(
    const float* __restrict__ Wt, const float* __restrict__ bias, const float* __restrict__ z0,
    float* __restrict__ Z, int L, int skip, int act, int l0, int l1) {
    using SQ = WaveSeq<W>;
    constexpr int NB = SQ::NB;
    __shared__ float sg[W];
    const int b = blockIdx.x, lane = threadIdx.x;
    const int i = min(lane / SQ::LPR, W - 1), c0 = (lane % SQ::LPR) * SQ::CPL;
    const int count = l1 - l0;
    if (count <= 0) return;
    const int tw = lane & (W - 1);
    const int src = (l0 / skip) * skip - 1;  // the current block's input row
    float wr[NB][SQ::CPL], bq[NB];
    auto lay = [&](int k) { return l0 + min(k, count - 1); };
    auto load = [&](int k, float (&r)[SQ::CPL], float& bb) {
        const int l = lay(k);
        row_to_regs<W>(Wt + (long long)l * W * W, i, c0, r);
        bb = bias[(long long)l * W + i];
    };
    auto pro = [&](auto J) {
        constexpr int j = decltype(J)::value;
        load(j, wr[j], bq[j]);
    };
    each_slot<0, NB>(pro);
    // every lane holds element tw of the state and of the skip source
    float z = (l0 == 0) ? z0[(long long)b * W + tw] : Z[((long long)b * L + l0 - 1) * W + tw];
    float xs = (src < 0) ? z0[(long long)b * W + tw] : Z[((long long)b * L + src) * W + tw];
    auto step = [&](int k, auto U) {
        constexpr int u = decltype(U)::value;
        const int l = l0 + k;
        wave_sync();  // the previous layer's reads of sg are done
        if (lane < W) {
            float d;
            sg[lane] = activate(2 * act, z, &d);
        }
        wave_sync();
        const float a = wave_row_dot<W>(wr[u], sg, c0) + bq[u];
        load(k + NB, wr[u], bq[u]);
        const bool sk = (l + 1) % skip == 0;
        // row i's value to every lane holding element i (lane tw == i)
        const float v = __shfl(a, (tw) * SQ::LPR, 64) + (sk ? xs : 0.f);
        z = v;
        if (sk) xs = v;
        if (lane < W) Z[((long long)b * L + l) * W + lane] = v;
    };
    walk<NB>(count, step);
}

// As resnet_seq_backward_kernel, one wave per system (w = 16, 32).
template <int W>
__global__ __launch_bounds__(64) void resnet_seq_backward_wave(
    const float* __restrict__ Wt, const float* __restrict__ z0, const float* __restrict__ Z,
    const float* __restrict__ G, float* __restrict__ Lambda, float* __restrict__ dz0, int L,
    int skip, int act, int l0, int l1) {
    using SQ = WaveSeq<W>;
    constexpr int NB = SQ::NB;
    __shared__ float Wl[W * (W + 1)];  // the current block, rows of pitch w + 1
    __shared__ float lam[W];
    const int b = blockIdx.x, lane = threadIdx.x;
    const int i = min(lane / SQ::LPR, W - 1), c0 = (lane % SQ::LPR) * SQ::CPL;
    const int count = l1 - l0;
    if (count <= 0) return;
    const int tw = lane & (W - 1);
    float* Lb = Lambda + (long long)b * L * W;
    float wr[NB][SQ::CPL], zq[NB];
    auto lay = [&](int k) { return l1 - 1 - min(k, count - 1); };
    auto load = [&](int k, float (&r)[SQ::CPL], float& zz) {
        const int l = lay(k);
        row_to_regs<W>(Wt + (long long)l * W * W, i, c0, r);
        zz = (l == 0) ? z0[(long long)b * W + tw] : Z[((long long)b * L + l - 1) * W + tw];
    };
    auto pro = [&](auto J) {
        constexpr int j = decltype(J)::value;
        load(j, wr[j], zq[j]);
    };
    each_slot<0, NB>(pro);
    // xsk: the adjoint of the current block's last row (its skip source)
    float xsk = (l1 == L) ? G[(long long)b * W + tw] : Lb[(long long)(l1 - 1) * W + tw];
    if (lane < W) {
        lam[lane] = xsk;
        if (l1 == L) Lb[(long long)(L - 1) * W + lane] = xsk;
    }
    auto step = [&](int k, auto U) {
        constexpr int u = decltype(U)::value;
        const int l = l1 - 1 - k;
        wave_sync();  // the previous layer's reads of Wl and lam are done
#pragma unroll
        for (int c = 0; c < SQ::CPL; ++c) Wl[i * (W + 1) + c0 + c] = wr[u][c];
        float d;
        activate(2 * act, zq[u], &d);
        load(k + NB, wr[u], zq[u]);
        wave_sync();
        // element tw: sum over the rows of Wl[r][tw] lam[r]
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int r = 0; r < W; ++r) acc[r & 3] = fmaf(Wl[r * (W + 1) + tw], lam[r], acc[r & 3]);
        const float nl = (acc[0] + acc[1]) + (acc[2] + acc[3]);
        const bool first = l % skip == 0;  // first layer of a block: its input took the skip
        // the block's last row l + skip - 1 is <= L - 1 only for a first layer
        float sa = 0.f;
        if (first)
            sa = l + skip - 1 <= l1 - 1 ? xsk : Lb[(long long)min(l + skip - 1, L - 1) * W + tw];
        const float v = nl * d + sa;
        wave_sync();  // every lane's reads of lam are done
        if (l >= 1) {
            if (lane < W) {
                lam[lane] = v;
                Lb[(long long)(l - 1) * W + lane] = v;
            }
            if (l % skip == 0) xsk = v;  // row l - 1 ends the block below
        } else if (lane < W) {
            dz0[(long long)b * W + lane] = v;
        }
    };
    walk<NB>(count, step);
}

}  // namespace

hipError_t launch_resnet_seq_forward(const float* W, const float* bias, const float* z0, float* Z,
                                     int B, int L, int w, int skip, int act, int l0, int l1,
                                     hipStream_t stream) {
    switch (w) {
        case 16: hipLaunchKernelGGL((resnet_seq_forward_wave<16>), dim3((unsigned)B), dim3(64), 0, stream, W, bias, z0, Z, L, skip, act, l0, l1); return hipGetLastError();
        case 32: hipLaunchKernelGGL((resnet_seq_forward_wave<32>), dim3((unsigned)B), dim3(64), 0, stream, W, bias, z0, Z, L, skip, act, l0, l1); return hipGetLastError();
        default: break;
    }
    switch (w) {
        case 16: hipLaunchKernelGGL((resnet_seq_forward_stream<16>), dim3((unsigned)B), dim3(kThreads), 0, stream, W, bias, z0, Z, L, skip, act, l0, l1); return hipGetLastError();
        case 32: hipLaunchKernelGGL((resnet_seq_forward_stream<32>), dim3((unsigned)B), dim3(kThreads), 0, stream, W, bias, z0, Z, L, skip, act, l0, l1); return hipGetLastError();
        case 64: hipLaunchKernelGGL((resnet_seq_forward_stream<64>), dim3((unsigned)B), dim3(kThreads), 0, stream, W, bias, z0, Z, L, skip, act, l0, l1); return hipGetLastError();
        case 128: hipLaunchKernelGGL((resnet_seq_forward_stream<128>), dim3((unsigned)B), dim3(kThreads), 0, stream, W, bias, z0, Z, L, skip, act, l0, l1); return hipGetLastError();
        default: break;
    }
    hipLaunchKernelGGL(resnet_seq_forward_kernel, dim3((unsigned)B), dim3(kThreads), 0, stream, W,
                       bias, z0, Z, L, w, skip, act, l0, l1);
    return hipGetLastError();
}

hipError_t launch_resnet_seq_backward(const float* W, const float* z0, const float* Z,
                                      const float* G, float* Lambda, float* dz0, int B, int L,
                                      int w, int skip, int act, int l0, int l1,
                                      hipStream_t stream) {
    switch (w) {
        case 16: hipLaunchKernelGGL((resnet_seq_backward_wave<16>), dim3((unsigned)B), dim3(64), 0, stream, W, z0, Z, G, Lambda, dz0, L, skip, act, l0, l1); return hipGetLastError();
        case 32: hipLaunchKernelGGL((resnet_seq_backward_wave<32>), dim3((unsigned)B), dim3(64), 0, stream, W, z0, Z, G, Lambda, dz0, L, skip, act, l0, l1); return hipGetLastError();
        default: break;
    }
    switch (w) {
        case 16: hipLaunchKernelGGL((resnet_seq_backward_stream<16>), dim3((unsigned)B), dim3(kThreads), 0, stream, W, z0, Z, G, Lambda, dz0, L, skip, act, l0, l1); return hipGetLastError();
        case 32: hipLaunchKernelGGL((resnet_seq_backward_stream<32>), dim3((unsigned)B), dim3(kThreads), 0, stream, W, z0, Z, G, Lambda, dz0, L, skip, act, l0, l1); return hipGetLastError();
        case 64: hipLaunchKernelGGL((resnet_seq_backward_stream<64>), dim3((unsigned)B), dim3(kThreads), 0, stream, W, z0, Z, G, Lambda, dz0, L, skip, act, l0, l1); return hipGetLastError();
        case 128: hipLaunchKernelGGL((resnet_seq_backward_stream<128>), dim3((unsigned)B), dim3(kThreads), 0, stream, W, z0, Z, G, Lambda, dz0, L, skip, act, l0, l1); return hipGetLastError();
        default: break;
    }
    hipLaunchKernelGGL(resnet_seq_backward_kernel, dim3((unsigned)B), dim3(kThreads), 0, stream,
                       W, z0, Z, G, Lambda, dz0, L, w, skip, act, l0, l1);
    return hipGetLastError();
}

hipError_t launch_seq_forward(const float* W, const float* bias, const float* z0, float* Z, int B,
                              int L, int w, int layer, float alpha, int l0, int l1,
                              hipStream_t stream) {
    switch (w) {
        case 2: hipLaunchKernelGGL((seq_forward_wave<2>), dim3((unsigned)B), dim3(64), 0, stream, W, bias, z0, Z, L, layer, alpha, l0, l1); return hipGetLastError();
        case 4: hipLaunchKernelGGL((seq_forward_wave<4>), dim3((unsigned)B), dim3(64), 0, stream, W, bias, z0, Z, L, layer, alpha, l0, l1); return hipGetLastError();
        case 8: hipLaunchKernelGGL((seq_forward_wave<8>), dim3((unsigned)B), dim3(64), 0, stream, W, bias, z0, Z, L, layer, alpha, l0, l1); return hipGetLastError();
        case 16: hipLaunchKernelGGL((seq_forward_wave<16>), dim3((unsigned)B), dim3(64), 0, stream, W, bias, z0, Z, L, layer, alpha, l0, l1); return hipGetLastError();
        case 32: hipLaunchKernelGGL((seq_forward_wave<32>), dim3((unsigned)B), dim3(64), 0, stream, W, bias, z0, Z, L, layer, alpha, l0, l1); return hipGetLastError();
        case 64: hipLaunchKernelGGL((seq_forward_wave<64>), dim3((unsigned)B), dim3(64), 0, stream, W, bias, z0, Z, L, layer, alpha, l0, l1); return hipGetLastError();
        default: break;
    }
    switch (w) {
        case 16: hipLaunchKernelGGL((seq_forward_stream<16>), dim3((unsigned)B), dim3(kThreads), 0, stream, W, bias, z0, Z, L, layer, alpha, l0, l1); return hipGetLastError();
        case 32: hipLaunchKernelGGL((seq_forward_stream<32>), dim3((unsigned)B), dim3(kThreads), 0, stream, W, bias, z0, Z, L, layer, alpha, l0, l1); return hipGetLastError();
        case 64: hipLaunchKernelGGL((seq_forward_stream<64>), dim3((unsigned)B), dim3(kThreads), 0, stream, W, bias, z0, Z, L, layer, alpha, l0, l1); return hipGetLastError();
        case 128: hipLaunchKernelGGL((seq_forward_stream<128>), dim3((unsigned)B), dim3(kThreads), 0, stream, W, bias, z0, Z, L, layer, alpha, l0, l1); return hipGetLastError();
        default: break;
    }
    hipLaunchKernelGGL(seq_forward_kernel, dim3((unsigned)B), dim3(kThreads), 0, stream, W, bias,
                       z0, Z, L, w, layer, alpha, l0, l1);
    return hipGetLastError();
}

hipError_t launch_seq_backward(const float* W, const float* bias, const float* z0, const float* Z,
                               const float* G, float* Lambda, float* dz0, int B, int L, int w,
                               int layer, float alpha, int l0, int l1, hipStream_t stream) {
    switch (w) {
        case 2: hipLaunchKernelGGL((seq_backward_wave<2>), dim3((unsigned)B), dim3(64), 0, stream, W, bias, z0, Z, G, Lambda, dz0, L, layer, alpha, l0, l1); return hipGetLastError();
        case 4: hipLaunchKernelGGL((seq_backward_wave<4>), dim3((unsigned)B), dim3(64), 0, stream, W, bias, z0, Z, G, Lambda, dz0, L, layer, alpha, l0, l1); return hipGetLastError();
        case 8: hipLaunchKernelGGL((seq_backward_wave<8>), dim3((unsigned)B), dim3(64), 0, stream, W, bias, z0, Z, G, Lambda, dz0, L, layer, alpha, l0, l1); return hipGetLastError();
        case 16: hipLaunchKernelGGL((seq_backward_wave<16>), dim3((unsigned)B), dim3(64), 0, stream, W, bias, z0, Z, G, Lambda, dz0, L, layer, alpha, l0, l1); return hipGetLastError();
        case 32: hipLaunchKernelGGL((seq_backward_wave<32>), dim3((unsigned)B), dim3(64), 0, stream, W, bias, z0, Z, G, Lambda, dz0, L, layer, alpha, l0, l1); return hipGetLastError();
        default: break;
    }
    switch (w) {
        case 16: hipLaunchKernelGGL((seq_backward_stream<16>), dim3((unsigned)B), dim3(kThreads), 0, stream, W, bias, z0, Z, G, Lambda, dz0, L, layer, alpha, l0, l1); return hipGetLastError();
        case 32: hipLaunchKernelGGL((seq_backward_stream<32>), dim3((unsigned)B), dim3(kThreads), 0, stream, W, bias, z0, Z, G, Lambda, dz0, L, layer, alpha, l0, l1); return hipGetLastError();
        case 64: hipLaunchKernelGGL((seq_backward_stream<64>), dim3((unsigned)B), dim3(kThreads), 0, stream, W, bias, z0, Z, G, Lambda, dz0, L, layer, alpha, l0, l1); return hipGetLastError();
        case 128: hipLaunchKernelGGL((seq_backward_stream<128>), dim3((unsigned)B), dim3(kThreads), 0, stream, W, bias, z0, Z, G, Lambda, dz0, L, layer, alpha, l0, l1); return hipGetLastError();
        default: break;
    }
    hipLaunchKernelGGL(seq_backward_kernel, dim3((unsigned)B), dim3(kThreads), 0, stream, W, bias,
                       z0, Z, G, Lambda, dz0, L, w, layer, alpha, l0, l1);
    return hipGetLastError();
}

}  // namespace deeppcr
