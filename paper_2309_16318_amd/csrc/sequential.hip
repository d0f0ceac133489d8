// Sequential layer-by-layer passes on the GPU: the baseline DeepPCR is
// compared against (Sec. 4.1: the forward pass applied one layer after the
// other, and the backward pass as back substitution of Eq. 11).  Each system
// of the batch is walked by one workgroup, layer after layer; the layers of a
// system are inherently sequential, so only the batch is parallel.  Two launch
// shapes: all layers in one launch (no per-layer launch cost), or one launch
// per layer (the shape of an eager framework's layer loop).
#include "internal.h"

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

}  // namespace

hipError_t launch_resnet_seq_forward(const float* W, const float* bias, const float* z0, float* Z,
                                     int B, int L, int w, int skip, int act, int l0, int l1,
                                     hipStream_t stream) {
    hipLaunchKernelGGL(resnet_seq_forward_kernel, dim3((unsigned)B), dim3(kThreads), 0, stream, W,
                       bias, z0, Z, L, w, skip, act, l0, l1);
    return hipGetLastError();
}

hipError_t launch_resnet_seq_backward(const float* W, const float* z0, const float* Z,
                                      const float* G, float* Lambda, float* dz0, int B, int L,
                                      int w, int skip, int act, int l0, int l1,
                                      hipStream_t stream) {
    hipLaunchKernelGGL(resnet_seq_backward_kernel, dim3((unsigned)B), dim3(kThreads), 0, stream,
                       W, z0, Z, G, Lambda, dz0, L, w, skip, act, l0, l1);
    return hipGetLastError();
}

hipError_t launch_seq_forward(const float* W, const float* bias, const float* z0, float* Z, int B,
                              int L, int w, int layer, float alpha, int l0, int l1,
                              hipStream_t stream) {
    hipLaunchKernelGGL(seq_forward_kernel, dim3((unsigned)B), dim3(kThreads), 0, stream, W, bias,
                       z0, Z, L, w, layer, alpha, l0, l1);
    return hipGetLastError();
}

hipError_t launch_seq_backward(const float* W, const float* bias, const float* z0, const float* Z,
                               const float* G, float* Lambda, float* dz0, int B, int L, int w,
                               int layer, float alpha, int l0, int l1, hipStream_t stream) {
    hipLaunchKernelGGL(seq_backward_kernel, dim3((unsigned)B), dim3(kThreads), 0, stream, W, bias,
                       z0, Z, G, Lambda, dz0, L, w, layer, alpha, l0, l1);
    return hipGetLastError();
}

}  // namespace deeppcr
