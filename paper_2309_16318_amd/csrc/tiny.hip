// Newton + PCR forward pass for small problems in a single workgroup
// (Sec. 2, Eqs. 1-3; Sec. 3, Alg. 1): the iterate, the Jacobian blocks and
// the right-hand sides live in LDS, every Newton iteration (layer and
// Jacobian evaluation, all PCR levels, update, convergence test) runs inside
// one launch, and the host reads back one status record.  Both stopping rules
// of the library are evaluated inside the kernel.  Used when the whole batch
// fits in 64 KiB of LDS, where a multi-kernel solve would be dominated by
// launch and synchronisation latency.
#include "internal.h"

namespace deeppcr {
namespace {

constexpr int kThreads = 256;

struct TinyLds {
    float* Z;      // [B, L, w]
    float* A[2];   // [B, L, w, w] ping-pong
    float* r[2];   // [B, L, w] ping-pong
    float* dsc;    // [B, L, w]
    unsigned* red; // [kThreads / 64]
};

__device__ inline unsigned wave_umax(unsigned v) {
    for (int off = 32; off > 0; off >>= 1) v = max(v, (unsigned)__shfl_xor((int)v, off, 64));
    return v;
}

// f_l and its Jacobian at the current iterate: r = f_l(Z_{l-1}) - Z_l into r,
// J_l into A (rows l >= 1).
__device__ void tiny_eval(const float* __restrict__ W, const float* __restrict__ bias,
                          const float* __restrict__ z0, const TinyLds& s, float* A, float* r,
                          int B, int L, int w, int layer, float alpha) {
    const int n = B * L * w;
    for (int idx = threadIdx.x; idx < n; idx += kThreads) {
        const int i = idx % w;
        const int bl = idx / w;
        const int l = bl % L, b = bl / L;
        const float* zp = (l == 0) ? z0 + b * w : s.Z + (bl - 1) * w;
        const float* Wr = W + ((long long)l * w + i) * w;
        float a = 0.f;
        for (int j = 0; j < w; ++j) a = fmaf(Wr[j], zp[j], a);
        a += bias[l * w + i];
        float d;
        const float y = activate(layer, a, &d);
        const bool res = layer_residual(layer);
        const float f = res ? fmaf(alpha, y, zp[i]) : y;
        r[idx] = f - s.Z[idx];
        s.dsc[idx] = res ? alpha * d : d;
    }
    __syncthreads();
    const int na = B * L * w * w;
    for (int idx = threadIdx.x; idx < na; idx += kThreads) {
        const int j = idx % w;
        const int i = (idx / w) % w;
        const int bl = idx / (w * w);
        const int l = bl % L;
        float v = s.dsc[bl * w + i] * W[((long long)l * w + i) * w + j];
        if (layer_residual(layer) && i == j) v += 1.f;
        A[idx] = v;
    }
    __syncthreads();
}

// Max over the workgroup of one value per thread (bit patterns of
// non-negative floats); every thread receives the result.
__device__ inline unsigned block_umax(unsigned v, unsigned* red) {
    v = wave_umax(v);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    unsigned m = 0u;
    for (int q = 0; q < kThreads / 64; ++q) m = max(m, red[q]);
    __syncthreads();
    return m;
}

__global__ __launch_bounds__(kThreads) void newton_tiny_kernel(
    const float* __restrict__ W, const float* __restrict__ bias, const float* __restrict__ z0,
    float* __restrict__ Zout, const float* __restrict__ Z_init, int B, int L, int w, int layer,
    float alpha, StopRule rule, unsigned* __restrict__ result) {
    extern __shared__ float smem[];
    const int nz = B * L * w, na = nz * w;
    TinyLds s;
    s.Z = smem;
    s.A[0] = s.Z + nz;
    s.A[1] = s.A[0] + na;
    s.r[0] = s.A[1] + na;
    s.r[1] = s.r[0] + nz;
    s.dsc = s.r[1] + nz;
    s.red = reinterpret_cast<unsigned*>(s.dsc + nz);
    const int t = threadIdx.x;

    // initial guess: Z_init, or f_0(z0) in every row (App. F.2)
    for (int idx = t; idx < nz; idx += kThreads) {
        if (Z_init) {
            s.Z[idx] = Z_init[idx];
        } else {
            const int i = idx % w, b = idx / (L * w);
            const float* zp = z0 + b * w;
            float a = 0.f;
            for (int j = 0; j < w; ++j) a = fmaf(W[i * w + j], zp[j], a);
            float d;
            const float y = activate(layer, a + bias[i], &d);
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
        tiny_eval(W, bias, z0, s, s.A[0], s.r[0], B, L, w, layer, alpha);
        if (rule.residual) {
            unsigned lr = 0u;
            for (int idx = t; idx < nz; idx += kThreads)
                lr = max(lr, __float_as_uint(fabsf(s.r[0][idx])));
            const unsigned gr = block_umax(lr, s.red);
            iters = (unsigned)k;
            meas = gr;
            if (gr >= 0x7f800000u) {
                status = 3u;
                break;
            }
            const float res = __uint_as_float(gr);
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
                    const float* Ar = Ai + ((long long)bl * w + i) * w;
                    const float* rp = ri + (bl - st) * w;
                    float acc = 0.f;
                    for (int j = 0; j < w; ++j) acc = fmaf(Ar[j], rp[j], acc);
                    v += acc;
                }
                ro[idx] = v;
            }
            for (int idx = t; idx < na; idx += kThreads) {
                const int j = idx % w, i = (idx / w) % w, bl = idx / (w * w), l = bl % L;
                if (l < 2 * st) continue;
                const float* Ar = Ai + ((long long)bl * w + i) * w;
                const float* Pb = Ai + (long long)(bl - st) * w * w;
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
        const unsigned gmx = block_umax(lmx, s.red);
        const unsigned gmz = block_umax(lmz, s.red);
        meas = gmx;
        iters = (unsigned)(k + 1);
        if (gmx >= 0x7f800000u || gmz >= 0x7f800000u) {
            status = 3u;
            break;
        }
        const float m = __uint_as_float(gmx), zmax = __uint_as_float(gmz);
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
    return (3 * nz + 2 * na + nz) * sizeof(float) + (kThreads / 64) * sizeof(unsigned);
}

bool tiny_eligible(int B, int L, int w) {
    return (double)B * L * w * (w + 4.0) * 4.0 <= 60000.0 && tiny_lds_bytes(B, L, w) <= 65536;
}

hipError_t launch_newton_tiny(const float* W, const float* bias, const float* z0, float* Z,
                              const float* Z_init, int B, int L, int w, int layer, float alpha,
                              const StopRule& rule, unsigned* result, hipStream_t stream) {
    const size_t lds = tiny_lds_bytes(B, L, w);
    hipLaunchKernelGGL(newton_tiny_kernel, dim3(1), dim3(kThreads), lds, stream, W, bias, z0, Z,
                       Z_init, B, L, w, layer, alpha, rule, result);
    return hipGetLastError();
}

}  // namespace deeppcr
