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
        // then the completion word the host may watch instead of waiting for
        // the stream: visible only after the record
        __threadfence_system();
        __hip_atomic_store(result + 3, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
}

template <int CTRL>
__device__ __forceinline__ unsigned dpp_u(unsigned v) {
    return (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

// Max over the wave in every lane, from register-to-register exchanges:
// DPP quad permutations and row mirrors within each 16-lane row, then the
// row swaps of v_permlane16_swap and v_permlane32_swap (each returns, in
// every lane, its own value and its partner row's).
__device__ __forceinline__ unsigned wave_umax_dpp(unsigned v) {
    v = max(v, dpp_u<0xB1>(v));   // quad_perm [1,0,3,2]
    v = max(v, dpp_u<0x4E>(v));   // quad_perm [2,3,0,1]
    v = max(v, dpp_u<0x141>(v));  // row_half_mirror
    v = max(v, dpp_u<0x140>(v));  // row_mirror
    const auto a = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    v = max(a[0], a[1]);
    const auto c = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return max(c[0], c[1]);
}

// The same solve held in one wave's registers, for problems whose iterate has
// at most 64 entries and w in {1, 2, 4, 8}: lane t owns entry t of Z
// (system b, layer l, row i), the row i of W_l, A_l and r_l that goes with it,
// and every value from another row (the previous layer's state, row l - s of
// a PCR level) arrives by a lane shuffle; no LDS and no barriers.  Each PCR
// level computes the new values from the old ones of all lanes before any
// lane keeps them, as the two buffers of a level do in the workgroup form;
// rows l < 2s keep their operator (never read again).  Same steps, stopping
// rules and status record as newton_tiny_kernel.
template <int W>
__global__ __launch_bounds__(64) void newton_wave_kernel(
    const float* __restrict__ Wg, const float* __restrict__ bg, const float* __restrict__ z0,
    float* __restrict__ Zout, const float* __restrict__ Z_init, int B, int L, int layer,
    float alpha, StopRule rule, unsigned* __restrict__ result) {
    const int t = threadIdx.x;
    const int n = B * L * W;
    const bool on = t < n;
    const int i = t % W, bl = t / W;
    const int l = on ? bl % L : -1, b = bl / L;
    const bool res = layer_residual(layer);
    // lane of entry (b, l, 0): rows of the same system are W lanes apart
    const int row0 = t - i;
    float Wr[W], W0[W], zin[W];
    float bias = 0.f, bias0 = 0.f, zini = 0.f;  // zini: z0[b][i]
#pragma unroll
    for (int j = 0; j < W; ++j) Wr[j] = W0[j] = zin[j] = 0.f;
    if (on) {
#pragma unroll
        for (int j = 0; j < W; ++j) {
            Wr[j] = Wg[((long long)l * W + i) * W + j];
            W0[j] = Wg[i * W + j];
            zin[j] = z0[b * W + j];
        }
        bias = bg[l * W + i];
        bias0 = bg[i];
        zini = z0[b * W + i];
    }
    // initial guess: Z_init, or f_0(z0) in every row (App. F.2)
    float Z = 0.f;
    if (on) {
        if (Z_init) {
            Z = Z_init[t];
        } else {
            float a = 0.f;
#pragma unroll
            for (int j = 0; j < W; ++j) a = fmaf(W0[j], zin[j], a);
            float d;
            const float y = activate(layer, a + bias0, &d);
            Z = res ? fmaf(alpha, y, zini) : y;
        }
    }
    unsigned status = 2u;
    unsigned meas = 0u, iters = 0u;
    float res0 = 0.f;
    for (int k = 0; k <= rule.max_iter; ++k) {
        if (!rule.residual && k == rule.max_iter) break;
        // layer l at Z_{l-1} (z0 for l = 0): r and row i of J_l
        float zp[W];
#pragma unroll
        for (int j = 0; j < W; ++j) {
            const float zj = __shfl(Z, l >= 1 ? row0 - W + j : t, 64);
            zp[j] = l >= 1 ? zj : zin[j];
        }
        float a = 0.f;
#pragma unroll
        for (int j = 0; j < W; ++j) a = fmaf(Wr[j], zp[j], a);
        a += bias;
        float d;
        const float y = activate(layer, a, &d);
        // the lane's own entry of the previous state
        const float zpi = __shfl(Z, l >= 1 ? t - W : t, 64);
        const float f = res ? fmaf(alpha, y, l >= 1 ? zpi : zini) : y;
        float r = on ? f - Z : 0.f;
        const float dsc = res ? alpha * d : d;
        float A[W];
#pragma unroll
        for (int j = 0; j < W; ++j) {
            float v = dsc * Wr[j];
            if (res && i == j) v += 1.f;
            A[j] = v;
        }
        if (rule.residual) {
            const unsigned lr = wave_umax_dpp(__float_as_uint(fabsf(r)));
            iters = (unsigned)k;
            meas = lr;
            if (lr >= 0x7f800000u) {
                status = 3u;
                break;
            }
            const float rv = __uint_as_float(lr);
            if (k == 0) res0 = rv;
            if (rv <= rule.atol || rv <= rule.rtol * res0) {
                status = 0u;
                break;
            }
            if (k == rule.max_iter) break;
        }
        // PCR levels (Alg. 1): every lane reads the old values of row l - s
        // before it replaces its own
        for (int st = 1; st < L; st *= 2) {
            const bool has = l >= st;
            const int src = has ? row0 - st * W : t;
            float acc = 0.f;
#pragma unroll
            for (int j = 0; j < W; ++j) acc = fmaf(A[j], __shfl(r, src + (has ? j : 0), 64), acc);
            float An[W];
#pragma unroll
            for (int j = 0; j < W; ++j) An[j] = 0.f;
#pragma unroll
            for (int q = 0; q < W; ++q)
#pragma unroll
                for (int j = 0; j < W; ++j)
                    An[j] = fmaf(A[q], __shfl(A[j], src + (has ? q : 0), 64), An[j]);
            if (has) r += acc;
            if (l >= 2 * st) {
#pragma unroll
                for (int j = 0; j < W; ++j) A[j] = An[j];
            }
        }
        // update and convergence measures
        const float z = Z + r;
        if (on) Z = z;
        const unsigned lmx = wave_umax_dpp(on ? __float_as_uint(fabsf(r)) : 0u);
        const unsigned lmz = wave_umax_dpp(on ? __float_as_uint(fabsf(z)) : 0u);
        if (rule.residual) continue;
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
    if (on) Zout[t] = Z;
    if (t == 0) {
        result[0] = status;
        result[1] = iters;
        result[2] = meas;
        // then the completion word the host may watch instead of waiting for
        // the stream: visible only after the record
        __threadfence_system();
        __hip_atomic_store(result + 3, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
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
    if ((long long)B * L * w <= 64 && (w == 1 || w == 2 || w == 4 || w == 8)) {
#define DEEPPCR_WAVE(WT)                                                                    \
    hipLaunchKernelGGL((newton_wave_kernel<WT>), dim3(1), dim3(64), 0, stream, W, bias, z0, Z, \
                       Z_init, B, L, layer, alpha, rule, result)
        switch (w) {
            case 1: DEEPPCR_WAVE(1); break;
            case 2: DEEPPCR_WAVE(2); break;
            case 4: DEEPPCR_WAVE(4); break;
            default: DEEPPCR_WAVE(8); break;
        }
#undef DEEPPCR_WAVE
        return hipGetLastError();
    }
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
