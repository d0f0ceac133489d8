// The last levels of a solve by substitution along the chains that the
// levels before them leave.  After the PCR levels with strides below s
// (Sec. 3, Alg. 1), rows l < s are final and every row l >= s satisfies
//   x_l = A_l x_{l-s} + r_l,
// so the system is B s independent block-bidiagonal chains (rows c, c + s,
// c + 2s, ...), each at most 2^KT rows long.  The remaining KT levels of
// Alg. 1 solve each chain in KT doubling steps whose operator products are
// only ever applied to vectors; here each chain is instead solved by
// substitution (the sequential solve of Sec. 3 on the reduced system): one
// mat-vec per row, walking the chain, each operator block read once.
//
// One workgroup per chain.  Thread t takes row t / TPR of the block and
// TPR-th of its columns; the blocks and right-hand sides of the next D rows
// are requested into a register ring before the current row's mat-vec (the
// loads do not depend on the chain's solution), the partial dot products
// meet through DPP lane permutations, and the new x goes to LDS for the next row
// (double-buffered, one barrier per row).
// UPD (the last pass of a Newton iteration): rout is the iterate; each
// solution row is added to it and max |x|, max |Z + x| are reduced into the
// kRedDZ, kRedZ slots of red.
#include "internal.h"
#include "strip.h"

#include <type_traits>

namespace deeppcr {
namespace {

// Measured (bench.py, one MI355X, same box): at w = 128, 1024 threads and
// one row ahead 206 us per pass against 217 with 512 threads and 246 with
// two rows ahead (more rows in flight make the pass slower, not faster: its
// limit is the per-row chain of mat-vec, reduction and barrier, not the
// bytes in flight); w = 32: 4 rows ahead 49 us, 8 rows 59 us; w = 64: 1-3
// rows ahead 224-227 us, 4 rows 235 us.  w = 16: one wave per chain (a
// 1 KiB block is one float4 per lane), 8 rows ahead.
template <int W>
struct ChainShape {
    // threads per workgroup
    static constexpr int NT = W == 128 ? 1024 : W == 16 ? 64 : 256;
    static constexpr int TPR = NT / W;   // threads per block row
    static constexpr int CPT = W / TPR;  // columns per thread
    static constexpr int NV = CPT / 4;   // float4 per thread per block
    // rows requested ahead
    static constexpr int D = W == 16 ? 8 : W == 32 ? 4 : W == 64 ? 2 : 1;
    static constexpr int NB = D + 1;  // ring slots
    static_assert(CPT % 4 == 0 && TPR >= 2 && TPR <= 16 && (TPR & (TPR - 1)) == 0, "row split");
};

template <int I, int N, class F>
__device__ __forceinline__ void each_slot(F& f) {
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        each_slot<I + 1, N>(f);
    }
}

template <int W, bool UPD>
__global__ __launch_bounds__(ChainShape<W>::NT) void pcr_chain_subst(BlockSrc Ain, VecSrc rin,
                                                                      VecDst rout, unsigned* red,
                                                                      int L, int s) {
    using S = ChainShape<W>;
    __shared__ float xs[2][W];
    __shared__ unsigned wmax[2][S::NT / 64];
    const int t = threadIdx.x;
    const int i = t / S::TPR, p = t % S::TPR;
    const int b = blockIdx.x / s;
    const int c = blockIdx.x - b * s;
    const int count = (L - 1 - c) / s;  // rows c + s m, m = 0 .. count
    const float* ab = Ain.base + b * Ain.bstride;
    const float* rb = rin.base + b * rin.bstride;
    float* ob = rout.base + b * rout.bstride;
    const int col0 = p * S::CPT;

    v4f blk[S::NB][S::NV];
    float rr[S::NB], zz[S::NB];
    // Rows are requested in chain order, m = 1, 2, ...: the row bases (the
    // same in every lane) advance by one chain step per request and stop at
    // the chain's last row, which rows past the end re-read (their results
    // are never used); the lane's offsets are added at the access.
    const long long sa = (long long)s * Ain.rstride, sr = (long long)s * rin.rstride,
                    so = (long long)s * rout.rstride;
    const float* qa = ab + (long long)(c + s) * Ain.rstride;
    const float* qr = rb + (long long)(c + s) * rin.rstride;
    const float* qz = ob + (long long)(c + s) * rout.rstride;
    int mq = 1;
    const int offa = i * W + col0;
    // element mq into ring slot mq % NB; with UPD also the iterate's row,
    // which the solution row is added to
    auto request = [&](auto slot) {
#pragma unroll
        for (int v = 0; v < S::NV; ++v)
            blk[slot][v] = *reinterpret_cast<const v4f*>(qa + offa + 4 * v);
        rr[slot] = qr[i];
        if constexpr (UPD) zz[slot] = qz[i];
        if (mq < count) {
            qa += sa;
            qr += sr;
            qz += so;
        }
        ++mq;
    };
    // element 0: row c is final.  Maxima as bit patterns of non-negative
    // floats, which order like the floats (NaN above Inf).
    unsigned mx = 0u, mz = 0u;
    {
        const float x0 = rb[(long long)c * rin.rstride + i];
        if (p == 0) {
            float* o = ob + (long long)c * rout.rstride + i;
            if constexpr (UPD) {
                const float z = *o + x0;
                *o = z;
                mz = __float_as_uint(fabsf(z));
            } else {
                *o = x0;
            }
            mx = __float_as_uint(fabsf(x0));
            xs[0][i] = x0;
        }
    }
    auto prefetch = [&](auto slot) {
        if constexpr (decltype(slot)::value >= 1)
            if (decltype(slot)::value <= S::D) request(slot);
    };
    each_slot<0, S::NB>(prefetch);
    __syncthreads();
    // elements 1 .. count, NB per round so that ring slots are compile-time;
    // po: the row base of element m
    float* po = ob + (long long)(c + s) * rout.rstride;
    for (int m0 = 0; m0 <= count; m0 += S::NB) {
        auto element = [&](auto jc) {
            constexpr int j = decltype(jc)::value;
            const int m = m0 + j;
            if (m < 1 || m > count) return;  // uniform over the workgroup
            // the block D rows ahead into the slot freed by row m - 1
            constexpr int ahead = (j + S::D) % S::NB;
            request(std::integral_constant<int, ahead>{});
            const float* xp = xs[(m - 1) & 1] + col0;
            float acc = 0.f;
#pragma unroll
            for (int v = 0; v < S::NV; ++v) {
                const v4f xv = *reinterpret_cast<const v4f*>(xp + 4 * v);
#pragma unroll
                for (int e = 0; e < 4; ++e) acc = fmaf(blk[j][v][e], xv[e], acc);
            }
            const float x = rr[j] + row_sum<S::TPR>(acc);
            if (p == 0) {
                float* o = po + i;
                if constexpr (UPD) {
                    const float z = zz[j] + x;
                    *o = z;
                    mz = max(mz, __float_as_uint(fabsf(z)));
                } else {
                    *o = x;
                }
                mx = max(mx, __float_as_uint(fabsf(x)));
                xs[m & 1][i] = x;
            }
            // one wave (w = 16): its LDS operations complete in issue order,
            // so the next row's reads see this write without a barrier
            if constexpr (S::NT > 64)
                __syncthreads();
            else
                __builtin_amdgcn_wave_barrier();
            po += so;
        };
        each_slot<0, S::NB>(element);
    }
    if constexpr (UPD) {
        unsigned ux = mx, uz = mz;
        for (int off = 32; off > 0; off >>= 1) {
            ux = max(ux, (unsigned)__shfl_xor((int)ux, off, 64));
            uz = max(uz, (unsigned)__shfl_xor((int)uz, off, 64));
        }
        if ((t & 63) == 0) {
            wmax[0][t >> 6] = ux;
            wmax[1][t >> 6] = uz;
        }
        __syncthreads();
        if (t == 0) {
            for (int q = 1; q < S::NT / 64; ++q) {
                ux = max(ux, wmax[0][q]);
                uz = max(uz, wmax[1][q]);
            }
            const int slot = blockIdx.x % kRedShards;
            atomicMax(red + kRedDZ + slot, ux);
            atomicMax(red + kRedZ + slot, uz);
        }
    }
}

}  // namespace

hipError_t launch_pcr_chain_subst(const BlockSrc& Ain, const VecSrc& rin, const VecDst& rout,
                                  int B, int L, int w, int s, hipStream_t stream, unsigned* red) {
    if (Ain.trans) return hipErrorInvalidValue;
    const dim3 grid((unsigned)((long long)B * s));
#define DEEPPCR_CHAIN(WW)                                                                      \
    do {                                                                                       \
        if (red)                                                                               \
            hipLaunchKernelGGL((pcr_chain_subst<WW, true>), grid, dim3(ChainShape<WW>::NT), 0, \
                               stream, Ain, rin, rout, red, L, s);                             \
        else                                                                                   \
            hipLaunchKernelGGL((pcr_chain_subst<WW, false>), grid, dim3(ChainShape<WW>::NT), 0,\
                               stream, Ain, rin, rout, red, L, s);                             \
    } while (0)
    switch (w) {
        case 16: DEEPPCR_CHAIN(16); break;
        case 32: DEEPPCR_CHAIN(32); break;
        case 64: DEEPPCR_CHAIN(64); break;
        case 128: DEEPPCR_CHAIN(128); break;
        default: return hipErrorInvalidValue;
    }
#undef DEEPPCR_CHAIN
    return hipGetLastError();
}

}  // namespace deeppcr
