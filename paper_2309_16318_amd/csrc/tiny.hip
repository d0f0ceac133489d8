// Newton + PCR forward pass for small problems in a single workgroup
// (Sec. 2, Eqs. 1-3; Sec. 3, Alg. 1): the weights (copied once), the iterate,
// the Jacobian blocks and the right-hand sides live in LDS, every Newton
// iteration (layer and Jacobian evaluation, all PCR levels, update,
// convergence test) runs inside one launch, and the host reads back one
// status record.  Both stopping rules
// of the library are evaluated inside the kernel.  Used when the whole batch
// fits in 64 KiB of LDS, where a multi-kernel solve would be dominated by
// launch and synchronisation latency.
#include "internal.h"

namespace deeppcr {
namespace {

constexpr int kThreads = 256;

// The width as a compile-time constant (WT > 0) for the small widths this
// solver serves most, so that the index arithmetic is shifts and the inner
// loops unroll; WT = 0 reads it at run time.
template <int WT>
struct Width {
    int rt;
    __device__ int operator()() const { return WT > 0 ? WT : rt; }
};

struct TinyLds {
    float* Z;      // [B, L, w]
    float* A[2];   // [B, L, w, w] ping-pong
    float* r[2];   // [B, L, w] ping-pong
    float* dsc;    // [B, L, w]
    float* W;      // [L, w, w], copied once
    float* bias;   // [L, w]
    unsigned* red; // [2 * kThreads / 64]
};

__device__ inline unsigned wave_umax(unsigned v) {
    for (int off = 32; off > 0; off >>= 1) v = max(v, (unsigned)__shfl_xor((int)v, off, 64));
    return v;
}

// f_l and its Jacobian at the current iterate: r = f_l(Z_{l-1}) - Z_l into r,
// J_l into A (rows l >= 1).
template <int WT>
__device__ void tiny_eval(Width<WT> wd, const float* __restrict__ z0, const TinyLds& s, float* A,
                          float* r, int B, int L, int layer, float alpha) {
    const int w = wd();
    const int n = B * L * w;
    for (int idx = threadIdx.x; idx < n; idx += kThreads) {
        const int i = idx % w;
        const int bl = idx / w;
        const int l = bl % L, b = bl / L;
        const float* zp = (l == 0) ? z0 + b * w : s.Z + (bl - 1) * w;
        const float* Wr = s.W + (l * w + i) * w;
        float a = 0.f;
        for (int j = 0; j < w; ++j) a = fmaf(Wr[j], zp[j], a);
        a += s.bias[l * w + i];
        float d;
        const float y = activate(layer, a, &d);
        const bool res = layer_residual(layer);
        const float f = res ? fmaf(alpha, y, zp[i]) : y;
        r[idx] = f - s.Z[idx];
        s.dsc[idx] = res ? alpha * d : d;
    }
    __syncthreads();
    const int na = n * w;
    for (int idx = threadIdx.x; idx < na; idx += kThreads) {
        const int bli = idx / w;  // (b, l) * w + i
        const int i = bli % w;
        const int l = (bli / w) % L;
        const int j = idx % w;
        float v = s.dsc[bli] * s.W[(l * w + i) * w + j];
        if (layer_residual(layer) && i == j) v += 1.f;
        A[idx] = v;
    }
    __syncthreads();
}

// Max over the workgroup of two values per thread (bit patterns of
// non-negative floats); every thread receives both results.
__device__ inline void block_umax2(unsigned& a, unsigned& b, unsigned* red) {
    a = wave_umax(a);
    b = wave_umax(b);
    constexpr int NW = kThreads / 64;
    if ((threadIdx.x & 63) == 0) {
        red[threadIdx.x >> 6] = a;
        red[NW + (threadIdx.x >> 6)] = b;
    }
    __syncthreads();
    unsigned ma = 0u, mb = 0u;
    for (int q = 0; q < NW; ++q) {
        ma = max(ma, red[q]);
        mb = max(mb, red[NW + q]);
    }
    __syncthreads();
    a = ma;
    b = mb;
}

template <int WT>
__global__ __launch_bounds__(kThreads) void newton_tiny_kernel(
    const float* __restrict__ Wg, const float* __restrict__ bg, const float* __restrict__ z0,
    float* __restrict__ Zout, const float* __restrict__ Z_init, int B, int L, int w_rt, int layer,
    float alpha, StopRule rule, unsigned* __restrict__ result) {
    extern __shared__ float smem[];
    const Width<WT> wd{w_rt};
    const int w = wd();
    const int nz = B * L * w, na = nz * w;
    TinyLds s;
    s.Z = smem;
    s.A[0] = s.Z + nz;
    s.A[1] = s.A[0] + na;
    s.r[0] = s.A[1] + na;
    s.r[1] = s.r[0] + nz;
    s.dsc = s.r[1] + nz;
    s.W = s.dsc + nz;
    s.bias = s.W + L * w * w;
    s.red = reinterpret_cast<unsigned*>(s.bias + L * w);
    const int t = threadIdx.x;
    for (int idx = t; idx < L * w * w; idx += kThreads) s.W[idx] = Wg[idx];
    for (int idx = t; idx < L * w; idx += kThreads) s.bias[idx] = bg[idx];
    __syncthreads();

    // initial guess: Z_init, or f_0(z0) in every row (App. F.2)
    for (int idx = t; idx < nz; idx += kThreads) {
        if (Z_init) {
            s.Z[idx] = Z_init[idx];
        } else {
            const int i = idx % w, b = idx / (L * w);
            const float* zp = z0 + b * w;
            float a = 0.f;
            for (int j = 0; j < w; ++j) a = fmaf(s.W[i * w + j], zp[j], a);
            float d;
            const float y = activate(layer, a + s.bias[i], &d);
            s.Z[idx] = layer_residual(layer) ? fmaf(alpha, y, zp[i]) : y;
        }
    }
    __syncthreads();

    // Update rule: k counts solves 1..max_iter, tested after each update.
    // Residual rule: iterates k = 0..max_iter, tested before each solve.
    unsigned status = 2u;  // no convergence unless stated otherwise
    unsigned meas = 0u, iters = 0u;
    float res0 = 0.f;
    for (int k = 0; k <= rule.max_iter; ++k) {
        if (!rule.residual && k == rule.max_iter) break;
        tiny_eval<WT>(wd, z0, s, s.A[0], s.r[0], B, L, layer, alpha);
        if (rule.residual) {
            unsigned lr = 0u, none = 0u;
            for (int idx = t; idx < nz; idx += kThreads)
                lr = max(lr, __float_as_uint(fabsf(s.r[0][idx])));
            block_umax2(lr, none, s.red);
            iters = (unsigned)k;
            meas = lr;
            if (lr >= 0x7f800000u) {
                status = 3u;
                break;
            }
            const float res = __uint_as_float(lr);
            if (k == 0) res0 = res;
            if (res <= rule.atol || res <= rule.rtol * res0) {
                status = 0u;
                break;
            }
            if (k == rule.max_iter) break;
        }
        // PCR levels (Alg. 1): read level k-1 buffers, write level k buffers
        int cur = 0;
        for (int st = 1; st < L; st *= 2) {
            const float* Ai = s.A[cur];
            const float* ri = s.r[cur];
            float* Ao = s.A[cur ^ 1];
            float* ro = s.r[cur ^ 1];
            for (int idx = t; idx < nz; idx += kThreads) {
                const int i = idx % w, bl = idx / w, l = bl % L;
                float v = ri[idx];
                if (l >= st) {
                    const float* Ar = Ai + (bl * w + i) * w;
                    const float* rp = ri + (bl - st) * w;
                    float acc = 0.f;
                    for (int j = 0; j < w; ++j) acc = fmaf(Ar[j], rp[j], acc);
                    v += acc;
                }
                ro[idx] = v;
            }
            for (int idx = t; idx < na; idx += kThreads) {
                const int j = idx % w, bli = idx / w, i = bli % w, bl = bli / w, l = bl % L;
                if (l < 2 * st) continue;
                const float* Ar = Ai + (bl * w + i) * w;
                const float* Pb = Ai + (bl - st) * w * w;
                float acc = 0.f;
                for (int q = 0; q < w; ++q) acc = fmaf(Ar[q], Pb[q * w + j], acc);
                Ao[idx] = acc;
            }
            __syncthreads();
            cur ^= 1;
        }
        // update and convergence measures
        const float* x = s.r[cur];
        unsigned lmx = 0u, lmz = 0u;
        for (int idx = t; idx < nz; idx += kThreads) {
            const float z = s.Z[idx] + x[idx];
            s.Z[idx] = z;
            lmx = max(lmx, __float_as_uint(fabsf(x[idx])));
            lmz = max(lmz, __float_as_uint(fabsf(z)));
        }
        if (rule.residual) {
            __syncthreads();  // the next evaluation reads the whole iterate
            continue;
        }
        block_umax2(lmx, lmz, s.red);
        meas = lmx;
        iters = (unsigned)(k + 1);
        if (lmx >= 0x7f800000u || lmz >= 0x7f800000u) {
            status = 3u;
            break;
        }
        const float m = __uint_as_float(lmx), zmax = __uint_as_float(lmz);
        if (rule.tol > 0.f && m < rule.tol * fmaxf(1.f, zmax)) {
            status = 0u;
            break;
        }
    }
    if (!rule.residual && rule.tol == 0.f && status == 2u) status = 0u;
    for (int idx = t; idx < nz; idx += kThreads) Zout[idx] = s.Z[idx];
    if (t == 0) {
        result[0] = status;
        result[1] = iters;
        result[2] = meas;
    }
}

}  // namespace

size_t tiny_lds_bytes(int B, int L, int w) {
    const size_t nz = (size_t)B * L * w, na = nz * w;
    const size_t nw = (size_t)L * w * w + (size_t)L * w;  // the cached weights and biases
    return (3 * nz + 2 * na + nz + nw) * sizeof(float) + 2 * (kThreads / 64) * sizeof(unsigned);
}

bool tiny_eligible(int B, int L, int w) {
    return (double)B * L * w * (w + 4.0) * 4.0 <= 60000.0 && tiny_lds_bytes(B, L, w) <= 65536;
}

hipError_t launch_newton_tiny(const float* W, const float* bias, const float* z0, float* Z,
                              const float* Z_init, int B, int L, int w, int layer, float alpha,
                              const StopRule& rule, unsigned* result, hipStream_t stream) {
    const size_t lds = tiny_lds_bytes(B, L, w);
#define DEEPPCR_TINY(WT)                                                                     \
    hipLaunchKernelGGL((newton_tiny_kernel<WT>), dim3(1), dim3(kThreads), lds, stream, W, bias, \
                       z0, Z, Z_init, B, L, w, layer, alpha, rule, result)
    switch (w) {
        case 1: DEEPPCR_TINY(1); break;
        case 2: DEEPPCR_TINY(2); break;
        case 4: DEEPPCR_TINY(4); break;
        case 8: DEEPPCR_TINY(8); break;
        default: DEEPPCR_TINY(0); break;
    }
#undef DEEPPCR_TINY
    return hipGetLastError();
}

}  // namespace deeppcr
