// Collapsed-skip ResNet (App. A.3).  Layer j maps Z_{j-1} to
//   Z_j = W_j sigma(Z_{j-1}) + b_j            (+ Z_{j-s} when (j+1) % s == 0),
// Z_{-1} = z0 (the pre-activation MLP layer and residual addition of the
// appendix).  Collapsing the s layers of a block gives a Markov chain over the
// block outputs X_g = Z_{gs+s-1}:
//   X_g = F_g(X_{g-1}) = h_{gs+s-1}(... h_{gs}(X_{g-1}) ...) + X_{g-1},
//   dF_g/dX = I + J_{gs+s-1} ... J_{gs},   J_j = W_j diag(sigma'(Z_{j-1})),
// which Newton + PCR solves with L/s unknowns; the backward pass solves the
// transposed block system for the block-output adjoints and recovers the
// adjoints inside each block by back-propagating through its s layers.
//
// The kernels here work on whole blocks, one workgroup per (system, block),
// with the state vectors and the w x w running Jacobian product in LDS
// (dynamic, sized by w).  The PCR levels, the Newton update and its
// reductions are those of the MLP path.
#include "internal.h"
#include "strip.h"

namespace deeppcr {
namespace {

constexpr int kThreads = 256;

// sigma(z) and sigma'(z) for activation act (0 tanh, 1 sigmoid, 2 ReLU with
// derivative 0 at 0): the MLP layer codes with the residual bit clear.
__device__ inline float act_fn(int act, float z, float* d) { return activate(2 * act, z, d); }

// One layer on the state z (LDS, length w): z <- W_j sigma(z) + b_j.
// sg receives sigma(z) of the input.  Starts and ends with a barrier.
__device__ inline void layer_forward(const float* __restrict__ Wj, const float* __restrict__ bj,
                                     float* z, float* sg, int w, int act) {
    const int t = threadIdx.x;
    __syncthreads();
    if (t < w) {
        float d;
        sg[t] = act_fn(act, z[t], &d);
    }
    __syncthreads();
    float a = 0.f;
    if (t < w) {
        for (int k = 0; k < w; ++k) a = fmaf(Wj[(long long)t * w + k], sg[k], a);
        a += bj[t];
    }
    __syncthreads();
    if (t < w) z[t] = a;
    __syncthreads();
}

// Jacobian product of block g, P = J_{gs+s-1} ... J_{gs}, built in two LDS
// buffers of w x w floats (P and Q, swapped after each layer; the returned
// pointer holds the product).  J_j P = W_j (diag(sigma'(z)) P) is formed with
// W_j read from global memory (L2-resident, shared by every system), so no
// third buffer is needed.  The layer inputs are either recomputed from the
// block input (FROM_STATES = false: z holds X_{g-1} on entry and the block's
// last pre-skip output on exit) or read from the stored layer outputs Zb
// (FROM_STATES = true; Zb = Z + b*L*w).  jac = false skips the product.
template <bool FROM_STATES>
__device__ float* block_product(const float* __restrict__ W, const float* __restrict__ bias,
                                const float* __restrict__ Zb, const float* xin, float* z,
                                float* sg, float* ds, float* P, float* Q, int g, int w, int skip,
                                int act, bool jac) {
    const int t = threadIdx.x;
    const int ww = w * w;
    for (int tt = 0; tt < skip; ++tt) {
        const long long j = (long long)g * skip + tt;
        const float* Wj = W + j * ww;
        // the layer input and its activation
        if (t < w) {
            const float zin = FROM_STATES ? (tt == 0 ? xin[t] : Zb[(j - 1) * w + t]) : z[t];
            float d;
            sg[t] = act_fn(act, zin, &d);
            ds[t] = d;
        }
        __syncthreads();
        if (jac) {
            if (tt == 0) {
                for (int idx = t; idx < ww; idx += kThreads)
                    P[idx] = Wj[idx] * ds[idx - (idx / w) * w];
            } else {
                for (int idx = t; idx < ww; idx += kThreads) {
                    const int i = idx / w, k = idx - (idx / w) * w;
                    const float* wr = Wj + (long long)i * w;
                    float acc = 0.f;
                    for (int m = 0; m < w; ++m) acc = fmaf(wr[m] * ds[m], P[m * w + k], acc);
                    Q[idx] = acc;
                }
            }
        }
        float a = 0.f;
        if (!FROM_STATES && t < w) {
            for (int k = 0; k < w; ++k) a = fmaf(Wj[(long long)t * w + k], sg[k], a);
            a += bias[j * w + t];
        }
        __syncthreads();
        if (jac && tt > 0) {
            float* tmp = P;
            P = Q;
            Q = tmp;
        }
        if (!FROM_STATES && t < w) z[t] = a;
        __syncthreads();
    }
    return P;
}

// Forward Newton step on the block chain: for row (b, g) evaluate the block
// at the iterate's X_{g-1} (z0 for g = 0): r = F_g(X_{g-1}) - X_g and, for
// g >= 1, the block A_g = I + P in forward order.  Clears the max|dZ|, max|Z|
// reduction slots.
__global__ __launch_bounds__(kThreads) void resnet_block_eval_kernel(
    const float* __restrict__ W, const float* __restrict__ bias, const float* __restrict__ z0,
    const float* __restrict__ X, float* __restrict__ A, float* __restrict__ r,
    unsigned* __restrict__ red, int G, int w, int skip, int act) {
    extern __shared__ float smem[];
    float* xin = smem;
    float* z = xin + w;
    float* sg = z + w;
    float* ds = sg + w;
    float* P = ds + w;
    float* Q = P + w * w;
    const long long row = blockIdx.x;  // b * G + g
    const int g = (int)(row % G);
    const int b = (int)(row / G);
    const int t = threadIdx.x;
    if (row == 0)
        for (int k = t; k < 2 * kRedShards; k += kThreads) red[k] = 0u;
    const float* xp = (g == 0) ? z0 + (long long)b * w : X + (row - 1) * w;
    if (t < w) {
        xin[t] = xp[t];
        z[t] = xp[t];
    }
    __syncthreads();
    const bool jac = g > 0;  // the block of row 0 couples to z0 and is never read
    const float* Pf = block_product<false>(W, bias, nullptr, xin, z, sg, ds, P, Q, g, w, skip, act,
                                           jac);
    if (t < w) r[row * w + t] = (z[t] + xin[t]) - X[row * w + t];
    if (jac) {
        float* Ab = A + row * w * w;
        for (int idx = t; idx < w * w; idx += kThreads)
            Ab[idx] = Pf[idx] + ((idx / w == idx - (idx / w) * w) ? 1.f : 0.f);
    }
}

// X[b, g] = F_0(z0[b]) for every block g (App. F.2 applied to the blocks).
__global__ __launch_bounds__(kThreads) void resnet_initial_guess_kernel(
    const float* __restrict__ W, const float* __restrict__ bias, const float* __restrict__ z0,
    float* __restrict__ X, int G, int w, int skip, int act) {
    __shared__ float xin[kMaxWidth], z[kMaxWidth], sg[kMaxWidth];
    const int b = blockIdx.x;
    const int t = threadIdx.x;
    if (t < w) {
        xin[t] = z0[(long long)b * w + t];
        z[t] = xin[t];
    }
    for (int tt = 0; tt < skip; ++tt)
        layer_forward(W + (long long)tt * w * w, bias + (long long)tt * w, z, sg, w, act);
    for (long long idx = t; idx < (long long)G * w; idx += kThreads) {
        const int i = (int)(idx % w);
        X[(long long)b * G * w + idx] = z[i] + xin[i];
    }
}

// All layer outputs from the block outputs: in block g the first s-1 layers
// run from X_{g-1} (z0 for g = 0), and row gs+s-1 is X_g itself.
__global__ __launch_bounds__(kThreads) void resnet_expand_kernel(
    const float* __restrict__ W, const float* __restrict__ bias, const float* __restrict__ z0,
    const float* __restrict__ X, float* __restrict__ Z, int G, int w, int skip, int act) {
    __shared__ float z[kMaxWidth], sg[kMaxWidth];
    const long long row = blockIdx.x;  // b * G + g
    const int g = (int)(row % G);
    const int b = (int)(row / G);
    const int t = threadIdx.x;
    const long long L = (long long)G * skip;
    const float* xp = (g == 0) ? z0 + (long long)b * w : X + (row - 1) * w;
    if (t < w) z[t] = xp[t];
    float* Zb = Z + (long long)b * L * w;
    for (int tt = 0; tt + 1 < skip; ++tt) {
        const long long j = (long long)g * skip + tt;
        layer_forward(W + j * w * w, bias + j * w, z, sg, w, act);
        if (t < w) Zb[j * w + t] = z[t];
    }
    if (t < w) Zb[((long long)g * skip + skip - 1) * w + t] = X[row * w + t];
}

// Backward: blocks of the transposed block system in reversed row order.
// Reversed row m = G - g holds A_g = I + P_g (g >= 1) with P_g evaluated at
// the stored layer inputs, stored untransposed (the first PCR level reads it
// transposed); the right-hand side is G at reversed row 0 and 0 elsewhere.
__global__ __launch_bounds__(kThreads) void resnet_block_jac_kernel(
    const float* __restrict__ W, const float* __restrict__ z0, const float* __restrict__ Z,
    const float* __restrict__ Gv, float* __restrict__ A, float* __restrict__ rrev, int G, int w,
    int skip, int act) {
    extern __shared__ float smem[];
    float* xin = smem;
    float* z = xin + w;
    float* sg = z + w;
    float* ds = sg + w;
    float* P = ds + w;
    float* Q = P + w * w;
    const long long row = blockIdx.x;  // b * G + g
    const int g = (int)(row % G);
    const int b = (int)(row / G);
    const int t = threadIdx.x;
    const long long L = (long long)G * skip;
    const float* Zb = Z + (long long)b * L * w;
    const int m = G - 1 - g;
    if (t < w) rrev[((long long)b * G + m) * w + t] = (m == 0) ? Gv[(long long)b * w + t] : 0.f;
    if (g == 0) return;  // uniform over the workgroup
    if (t < w) xin[t] = Zb[((long long)g * skip - 1) * w + t];
    __syncthreads();
    const float* Pf = block_product<true>(W, nullptr, Zb, xin, z, sg, ds, P, Q, g, w, skip, act,
                                          true);
    float* Ab = A + ((long long)b * G + (G - g)) * w * w;
    for (int idx = t; idx < w * w; idx += kThreads)
        Ab[idx] = Pf[idx] + ((idx / w == idx - (idx / w) * w) ? 1.f : 0.f);
}

// Adjoints inside block g from the block-output adjoint mu_g (natural order
// [B, G, w]): Lambda[gs+s-1] = mu_g and, going down the block,
// lambda_{j-1} = diag(sigma'(Z_{j-1})) W_j^T lambda_j.  Block 0 also gives
// dz0 = diag(sigma'(z0)) W_0^T lambda_0 + mu_0 (the skip from z0).
__global__ __launch_bounds__(kThreads) void resnet_intra_adjoint_kernel(
    const float* __restrict__ W, const float* __restrict__ z0, const float* __restrict__ Z,
    const float* __restrict__ mu, float* __restrict__ Lambda, float* __restrict__ dz0, int G,
    int w, int skip, int act) {
    __shared__ float lam[kMaxWidth];
    const long long row = blockIdx.x;  // b * G + g
    const int g = (int)(row % G);
    const int b = (int)(row / G);
    const int t = threadIdx.x;
    const long long L = (long long)G * skip;
    const float* Zb = Z + (long long)b * L * w;
    float* Lb = Lambda + (long long)b * L * w;
    const long long jl = (long long)g * skip + skip - 1;
    float mu_t = 0.f;
    if (t < w) {
        mu_t = mu[row * w + t];
        lam[t] = mu_t;
        Lb[jl * w + t] = mu_t;
    }
    __syncthreads();
    const int lo = (g == 0) ? 0 : 1;  // block 0 also goes through layer 0 into z0
    for (int tt = skip - 1; tt >= lo; --tt) {
        const long long j = (long long)g * skip + tt;
        const float* Wj = W + j * w * w;
        float v = 0.f;
        if (t < w) {
            const float zin = (j == 0) ? z0[(long long)b * w + t] : Zb[(j - 1) * w + t];
            float d;
            act_fn(act, zin, &d);
            float s = 0.f;
            for (int k = 0; k < w; ++k) s = fmaf(Wj[(long long)k * w + t], lam[k], s);
            v = d * s;
        }
        __syncthreads();
        if (t < w) {
            if (j >= 1) {
                lam[t] = v;
                Lb[(j - 1) * w + t] = v;
            } else {
                dz0[(long long)b * w + t] = v + mu_t;
            }
        }
        __syncthreads();
    }
}

size_t block_lds_bytes(int w) { return (4 * (size_t)w + 2 * (size_t)w * w) * sizeof(float); }

// ---- one wave per (system, block), w = 16 or 32 ----------------------------
// Lane l owns row i = l / LPR of the running product P and its NC columns
// c0 = (l % LPR) * NC ..; the next factor's row, W_j[i, :] scaled by
// sigma'(z), comes from global memory (L2-resident, shared by every system)
// and the previous product's rows from the wave's LDS copy.  Only wave-level
// barriers; four independent waves per workgroup.
template <int W>
struct BlockWaveShape {
    static constexpr int LPR = 64 / W;     // lanes per product row
    static constexpr int NC = W / LPR;     // columns per lane (4 for w = 16, 16 for w = 32)
};

template <int W>
struct alignas(16) BlockWaveLds {
    float P[W * W];
    float xin[W], z[W], sg[W], ds[W];
};

// BWD = false: the forward block evaluation at the iterate (as
// resnet_block_eval_kernel).  BWD = true: the backward blocks at the stored
// states and the reversed right-hand side (as resnet_block_jac_kernel).
template <int W, bool BWD>
__global__ __launch_bounds__(256) void resnet_block_wave(
    const float* __restrict__ Wt, const float* __restrict__ bias, const float* __restrict__ z0,
    const float* __restrict__ S, const float* __restrict__ Gv, float* __restrict__ A,
    float* __restrict__ r, unsigned* __restrict__ red, int B, int G, int skip, int act) {
    using SH = BlockWaveShape<W>;
    constexpr int NC = SH::NC;
    __shared__ BlockWaveLds<W> lds_all[4];
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    if (!BWD && blockIdx.x == 0)
        for (int k = threadIdx.x; k < 2 * kRedShards; k += 256) red[k] = 0u;
    const long long item = (long long)blockIdx.x * 4 + wv;  // b * G + g
    if (item >= (long long)B * G) return;  // whole wave
    BlockWaveLds<W>& lds = lds_all[wv];
    const int g = (int)(item % G);
    const int b = (int)(item / G);
    const long long L = (long long)G * skip;
    const int i = lane / SH::LPR;
    const int c0 = (lane % SH::LPR) * NC;
    // S: forward, the iterate X [B, G, W]; backward, the stored states Z [B, L, W]
    const float* Zb = S + (long long)b * L * W;
    if (BWD) {
        const int m = G - 1 - g;
        if (lane < W) r[((long long)b * G + m) * W + lane] = (m == 0) ? Gv[(long long)b * W + lane] : 0.f;
        if (g == 0) return;
    }
    if (lane < W) {
        const float x = BWD ? Zb[((long long)g * skip - 1) * W + lane]
                            : (g == 0 ? z0[(long long)b * W + lane] : S[(item - 1) * W + lane]);
        lds.xin[lane] = x;
        lds.z[lane] = x;
    }
    const bool jac = g > 0;
    float pr[NC];
    for (int tt = 0; tt < skip; ++tt) {
        const long long j = (long long)g * skip + tt;
        wave_sync();
        if (lane < W) {
            const float zin = BWD ? (tt == 0 ? lds.xin[lane] : Zb[(j - 1) * W + lane]) : lds.z[lane];
            float d;
            lds.sg[lane] = act_fn(act, zin, &d);
            lds.ds[lane] = d;
        }
        wave_sync();
        float wr[W];
        const float* wrow = Wt + (j * W + i) * W;
#pragma unroll
        for (int q = 0; q < W / 4; ++q) {
            const v4f x = *reinterpret_cast<const v4f*>(wrow + 4 * q);
            wr[4 * q] = x[0];
            wr[4 * q + 1] = x[1];
            wr[4 * q + 2] = x[2];
            wr[4 * q + 3] = x[3];
        }
        if (jac) {
            if (tt == 0) {
#pragma unroll
                for (int c = 0; c < NC; ++c) pr[c] = wr[c0 + c] * lds.ds[c0 + c];
            } else {
                float pn[NC];
#pragma unroll
                for (int c = 0; c < NC; ++c) pn[c] = 0.f;
#pragma unroll
                for (int m = 0; m < W; ++m) {
                    const float f = wr[m] * lds.ds[m];
#pragma unroll
                    for (int q = 0; q < NC / 4; ++q) {
                        const v4f p4 = *reinterpret_cast<const v4f*>(lds.P + m * W + c0 + 4 * q);
                        pn[4 * q] = fmaf(f, p4[0], pn[4 * q]);
                        pn[4 * q + 1] = fmaf(f, p4[1], pn[4 * q + 1]);
                        pn[4 * q + 2] = fmaf(f, p4[2], pn[4 * q + 2]);
                        pn[4 * q + 3] = fmaf(f, p4[3], pn[4 * q + 3]);
                    }
                }
#pragma unroll
                for (int c = 0; c < NC; ++c) pr[c] = pn[c];
            }
        }
        float a = 0.f;
        if (!BWD) {
#pragma unroll
            for (int k = 0; k < W; ++k) a = fmaf(wr[k], lds.sg[k], a);
            a += bias[j * W + i];
        }
        wave_sync();  // every read of P, sg, ds, z of this layer is done
        if (jac) {
#pragma unroll
            for (int q = 0; q < NC / 4; ++q) {
                v4f x = {pr[4 * q], pr[4 * q + 1], pr[4 * q + 2], pr[4 * q + 3]};
                *reinterpret_cast<v4f*>(lds.P + i * W + c0 + 4 * q) = x;
            }
        }
        if (!BWD && (lane % SH::LPR) == 0) lds.z[i] = a;
    }
    wave_sync();
    if (!BWD && lane < W) r[item * W + lane] = (lds.z[lane] + lds.xin[lane]) - S[item * W + lane];
    if (jac) {
        float* Ab = A + (BWD ? ((long long)b * G + (G - g)) : item) * W * W + i * W + c0;
#pragma unroll
        for (int q = 0; q < NC / 4; ++q) {
            v4f x = {pr[4 * q], pr[4 * q + 1], pr[4 * q + 2], pr[4 * q + 3]};
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (c0 + 4 * q + e == i) x[e] += 1.f;
            *reinterpret_cast<v4f*>(Ab + 4 * q) = x;
        }
    }
}

// ---- one workgroup per (system, block), w = 64 or 128 ----------------------
// The running product on fp32 MFMA: one wave per 32-row strip (the register
// strips of the PCR kernels).  Layer j of the block multiplies the product
// from the left by J_j = W_j diag(sigma'(z_{j-1})): the lane's strip of W_j
// comes from global memory (L2-resident, shared by every system), first
// serves the state update W_j sigma(z) + b_j (forward), then has its columns
// scaled by sigma' and is multiplied with the previous product, held
// transposed in LDS (two buffers, one per layer parity).  The last product
// strip, plus I, is stored as the block's operator.  Same roles of BWD and
// the arguments as resnet_block_wave.
template <int W, bool BWD>
__global__ __launch_bounds__(Tile2Shape<W>::NT) void resnet_block_tile(
    const float* __restrict__ Wt, const float* __restrict__ bias, const float* __restrict__ z0,
    const float* __restrict__ S, const float* __restrict__ Gv, float* __restrict__ A,
    float* __restrict__ r, unsigned* __restrict__ red, int B, int G, int skip, int act) {
    using SH = Tile2Shape<W>;
    __shared__ float PT[2][W * SH::PITCH];  // the product so far, transposed
    __shared__ float xin[W], z[W], sg[W], ds[W];
    const int t = threadIdx.x;
    const int lane = t & 63, i = lane & 31, h = lane >> 5;
    const int R = 32 * (t >> 6) + i;
    if (!BWD && blockIdx.x == 0)
        for (int k = t; k < 2 * kRedShards; k += SH::NT) red[k] = 0u;
    const long long item = blockIdx.x;  // b * G + g
    const int g = (int)(item % G);
    const int b = (int)(item / G);
    const long long L = (long long)G * skip;
    // S: forward, the iterate X [B, G, W]; backward, the stored states Z [B, L, W]
    const float* Zb = S + (long long)b * L * W;
    if (BWD) {
        const int m = G - 1 - g;
        if (t < W) r[((long long)b * G + m) * W + t] = (m == 0) ? Gv[(long long)b * W + t] : 0.f;
        if (g == 0) return;  // uniform over the workgroup
    }
    if (t < W) {
        const float x = BWD ? Zb[((long long)g * skip - 1) * W + t]
                            : (g == 0 ? z0[(long long)b * W + t] : S[(item - 1) * W + t]);
        xin[t] = x;
        z[t] = x;
    }
    const bool jac = g > 0;  // the block of row 0 couples to z0 and is never read
    StripA<W> a;             // rows R of W_j, then of W_j diag(sigma')
    StripC<W> c;             // rows R of the product after layer j (j >= 1)
    strip_zero<W>(c);
    for (int tt = 0; tt < skip; ++tt) {
        const long long j = (long long)g * skip + tt;
        strip_load<W, false>(Wt + j * W * W, a, R, h);
        __syncthreads();  // z of the previous layer is in place
        if (t < W) {
            const float zin = BWD ? (tt == 0 ? xin[t] : Zb[(j - 1) * W + t]) : z[t];
            float d;
            sg[t] = act_fn(act, zin, &d);
            ds[t] = d;
        }
        __syncthreads();  // sg and ds are in place; every read of z is done
        if (!BWD) {
            const float zr = strip_matvec<W>(a, sg, h) + bias[j * W + R];
            if (h == 0) z[R] = zr;
        }
        if (jac) {
#pragma unroll
            for (int q = 0; q < SH::NQ; ++q) {
                const v4f d4 = *reinterpret_cast<const v4f*>(ds + 8 * q + 4 * h);
                a[q] *= d4;
            }
            const bool last = tt + 1 == skip;
            if (tt == 0) {
                if (!last) strip_put_T<W>(PT[0], a, R, h);
            } else {
                strip_product<W, 0, SH::T, false>(PT[(tt + 1) & 1], a, c, i, h);
                if (!last) strip_put_T<W>(PT[tt & 1], c, R, h);
            }
        }
    }
    __syncthreads();  // the block's output state is in place
    if (!BWD && t < W) r[item * W + t] = (z[t] + xin[t]) - S[item * W + t];
    if (jac) {
        float* Ab = A + (BWD ? ((long long)b * G + (G - g)) : item) * W * W;
        // the diagonal element R is column 8q + 4h + e with 8q + e = R - 4h
        const int dk = R - 4 * h;
#pragma unroll
        for (int q = 0; q < SH::NQ; ++q) {
            v4f x = skip == 1 ? a[q] : strip_quad<W>(c, q);
#pragma unroll
            for (int e = 0; e < 4; ++e) x[e] += dk == 8 * q + e ? 1.f : 0.f;
            *reinterpret_cast<v4f*>(Ab + R * W + 8 * q + 4 * h) = x;
        }
    }
}

template <int W, bool BWD>
hipError_t launch_block_tile(const float* Wt, const float* bias, const float* z0, const float* S,
                             const float* Gv, float* A, float* r, unsigned* red, int B, int G,
                             int skip, int act, hipStream_t stream) {
    hipLaunchKernelGGL((resnet_block_tile<W, BWD>), dim3((unsigned)((long long)B * G)),
                       dim3(Tile2Shape<W>::NT), 0, stream, Wt, bias, z0, S, Gv, A, r, red, B, G,
                       skip, act);
    return hipGetLastError();
}

// ---- one wave per (system, block) for the state expansion and the in-block
// adjoints, w = 16, 32, 64: lane t < w owns element t, four blocks per
// workgroup, wave-level barriers only.  Same work as resnet_expand_kernel
// and resnet_intra_adjoint_kernel.
template <int W>
__global__ __launch_bounds__(256) void resnet_expand_wave(
    const float* __restrict__ Wt, const float* __restrict__ bias, const float* __restrict__ z0,
    const float* __restrict__ X, float* __restrict__ Z, int B, int G, int skip, int act) {
    __shared__ float z_all[4][W], sg_all[4][W];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const long long item = (long long)blockIdx.x * 4 + wv;  // b * G + g
    if (item >= (long long)B * G) return;                   // whole wave
    const int g = (int)(item % G);
    const int b = (int)(item / G);
    float* z = z_all[wv];
    float* sg = sg_all[wv];
    const long long L = (long long)G * skip;
    float* Zb = Z + (long long)b * L * W;
    const float* xp = (g == 0) ? z0 + (long long)b * W : X + (item - 1) * W;
    if (lane < W) z[lane] = xp[lane];
    for (int tt = 0; tt + 1 < skip; ++tt) {
        const long long j = (long long)g * skip + tt;
        wave_sync();
        if (lane < W) {
            float d;
            sg[lane] = act_fn(act, z[lane], &d);
        }
        wave_sync();
        if (lane < W) {
            const float* wr = Wt + (j * W + lane) * W;
            float a = 0.f;
#pragma unroll
            for (int k = 0; k < W; ++k) a = fmaf(wr[k], sg[k], a);
            a += bias[j * W + lane];
            z[lane] = a;  // only lane t reads z[t] before the next barrier
            Zb[j * W + lane] = a;
        }
    }
    if (lane < W) Zb[((long long)g * skip + skip - 1) * W + lane] = X[item * W + lane];
}

template <int W>
__global__ __launch_bounds__(256) void resnet_intra_adjoint_wave(
    const float* __restrict__ Wt, const float* __restrict__ z0, const float* __restrict__ Z,
    const float* __restrict__ mu, float* __restrict__ Lambda, float* __restrict__ dz0, int B,
    int G, int skip, int act) {
    __shared__ float lam_all[4][W];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const long long item = (long long)blockIdx.x * 4 + wv;  // b * G + g
    if (item >= (long long)B * G) return;                   // whole wave
    const int g = (int)(item % G);
    const int b = (int)(item / G);
    float* lam = lam_all[wv];
    const long long L = (long long)G * skip;
    const float* Zb = Z + (long long)b * L * W;
    float* Lb = Lambda + (long long)b * L * W;
    const long long jl = (long long)g * skip + skip - 1;
    float mu_t = 0.f;
    if (lane < W) {
        mu_t = mu[item * W + lane];
        lam[lane] = mu_t;
        Lb[jl * W + lane] = mu_t;
    }
    const int lo = (g == 0) ? 0 : 1;  // block 0 also goes through layer 0 into z0
    for (int tt = skip - 1; tt >= lo; --tt) {
        const long long j = (long long)g * skip + tt;
        const float* Wj = Wt + j * W * W;
        wave_sync();
        float v = 0.f;
        if (lane < W) {
            const float zin = (j == 0) ? z0[(long long)b * W + lane] : Zb[(j - 1) * W + lane];
            float d;
            act_fn(act, zin, &d);
            float sum = 0.f;
#pragma unroll
            for (int k = 0; k < W; ++k) sum = fmaf(Wj[k * W + lane], lam[k], sum);
            v = d * sum;
        }
        wave_sync();
        if (lane < W) {
            if (j >= 1) {
                lam[lane] = v;
                Lb[(j - 1) * W + lane] = v;
            } else {
                dz0[(long long)b * W + lane] = v + mu_t;
            }
        }
    }
}

template <int W, bool BWD>
hipError_t launch_block_wave(const float* Wt, const float* bias, const float* z0, const float* S,
                             const float* Gv, float* A, float* r, unsigned* red, int B, int G,
                             int skip, int act, hipStream_t stream) {
    const long long items = (long long)B * G;
    hipLaunchKernelGGL((resnet_block_wave<W, BWD>), dim3((unsigned)((items + 3) / 4)), dim3(256), 0,
                       stream, Wt, bias, z0, S, Gv, A, r, red, B, G, skip, act);
    return hipGetLastError();
}

}  // namespace

// Dynamic LDS beyond 64 KiB (w > 90) must be allowed per kernel first.
template <class K>
hipError_t allow_lds(K kernel, size_t bytes) {
    if (bytes <= 65536) return hipSuccess;
    return hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)bytes);
}

hipError_t launch_resnet_block_eval(const float* W, const float* bias, const float* z0,
                                    const float* X, float* A, float* r, unsigned* red, int B,
                                    int G, int w, int skip, int act, hipStream_t stream) {
    if (w == 16)
        return launch_block_wave<16, false>(W, bias, z0, X, nullptr, A, r, red, B, G, skip, act,
                                            stream);
    if (w == 32)
        return launch_block_wave<32, false>(W, bias, z0, X, nullptr, A, r, red, B, G, skip, act,
                                            stream);
    if (w == 64)
        return launch_block_tile<64, false>(W, bias, z0, X, nullptr, A, r, red, B, G, skip, act,
                                            stream);
    if (w == 128)
        return launch_block_tile<128, false>(W, bias, z0, X, nullptr, A, r, red, B, G, skip, act,
                                             stream);
    const hipError_t e = allow_lds(resnet_block_eval_kernel, block_lds_bytes(w));
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(resnet_block_eval_kernel, dim3((unsigned)((long long)B * G)),
                       dim3(kThreads), block_lds_bytes(w), stream, W, bias, z0, X, A, r, red, G,
                       w, skip, act);
    return hipGetLastError();
}

hipError_t launch_resnet_initial_guess(const float* W, const float* bias, const float* z0,
                                       float* X, int B, int G, int w, int skip, int act,
                                       hipStream_t stream) {
    hipLaunchKernelGGL(resnet_initial_guess_kernel, dim3((unsigned)B), dim3(kThreads), 0, stream,
                       W, bias, z0, X, G, w, skip, act);
    return hipGetLastError();
}

hipError_t launch_resnet_expand(const float* W, const float* bias, const float* z0,
                                const float* X, float* Z, int B, int G, int w, int skip, int act,
                                hipStream_t stream) {
    const dim3 g4((unsigned)(((long long)B * G + 3) / 4)), b4(256);
    switch (w) {
        case 16: hipLaunchKernelGGL((resnet_expand_wave<16>), g4, b4, 0, stream, W, bias, z0, X, Z, B, G, skip, act); return hipGetLastError();
        case 32: hipLaunchKernelGGL((resnet_expand_wave<32>), g4, b4, 0, stream, W, bias, z0, X, Z, B, G, skip, act); return hipGetLastError();
        case 64: hipLaunchKernelGGL((resnet_expand_wave<64>), g4, b4, 0, stream, W, bias, z0, X, Z, B, G, skip, act); return hipGetLastError();
        default: break;
    }
    hipLaunchKernelGGL(resnet_expand_kernel, dim3((unsigned)((long long)B * G)), dim3(kThreads),
                       0, stream, W, bias, z0, X, Z, G, w, skip, act);
    return hipGetLastError();
}

hipError_t launch_resnet_block_jac(const float* W, const float* z0, const float* Z,
                                   const float* Gv, float* A, float* rrev, int B, int G, int w,
                                   int skip, int act, hipStream_t stream) {
    if (w == 16)
        return launch_block_wave<16, true>(W, nullptr, z0, Z, Gv, A, rrev, nullptr, B, G, skip,
                                           act, stream);
    if (w == 32)
        return launch_block_wave<32, true>(W, nullptr, z0, Z, Gv, A, rrev, nullptr, B, G, skip,
                                           act, stream);
    if (w == 64)
        return launch_block_tile<64, true>(W, nullptr, z0, Z, Gv, A, rrev, nullptr, B, G, skip,
                                           act, stream);
    if (w == 128)
        return launch_block_tile<128, true>(W, nullptr, z0, Z, Gv, A, rrev, nullptr, B, G, skip,
                                            act, stream);
    const hipError_t e = allow_lds(resnet_block_jac_kernel, block_lds_bytes(w));
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(resnet_block_jac_kernel, dim3((unsigned)((long long)B * G)),
                       dim3(kThreads), block_lds_bytes(w), stream, W, z0, Z, Gv, A, rrev, G, w,
                       skip, act);
    return hipGetLastError();
}

hipError_t launch_resnet_intra_adjoint(const float* W, const float* z0, const float* Z,
                                       const float* mu, float* Lambda, float* dz0, int B, int G,
                                       int w, int skip, int act, hipStream_t stream) {
    const dim3 g4((unsigned)(((long long)B * G + 3) / 4)), b4(256);
    switch (w) {
        case 16: hipLaunchKernelGGL((resnet_intra_adjoint_wave<16>), g4, b4, 0, stream, W, z0, Z, mu, Lambda, dz0, B, G, skip, act); return hipGetLastError();
        case 32: hipLaunchKernelGGL((resnet_intra_adjoint_wave<32>), g4, b4, 0, stream, W, z0, Z, mu, Lambda, dz0, B, G, skip, act); return hipGetLastError();
        case 64: hipLaunchKernelGGL((resnet_intra_adjoint_wave<64>), g4, b4, 0, stream, W, z0, Z, mu, Lambda, dz0, B, G, skip, act); return hipGetLastError();
        default: break;
    }
    hipLaunchKernelGGL(resnet_intra_adjoint_kernel, dim3((unsigned)((long long)B * G)),
                       dim3(kThreads), 0, stream, W, z0, Z, mu, Lambda, dz0, G, w, skip, act);
    return hipGetLastError();
}

}  // namespace deeppcr
