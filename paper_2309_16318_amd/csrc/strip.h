// Register strips of w x w blocks for the fp32 MFMA kernels (w = 32, 64,
// 128): one wave per 32-row strip of a block.  A lane (i, h) of wave v holds
// row R = 32 v + i at the columns 8q + 4h .. +3 (q = 0 .. W/8-1).  That is
// the left operand of v_mfma_f32_32x32x2_f32 (k-step q, element e: column
// 8q + 4h + e), read straight from memory, and also the layout in which the
// MFMA leaves a strip of the product (tile tc, float4 qq at q = 4 tc + qq):
// a product strip can be the left operand of the next product as it is.
// Right operands sit in LDS transposed (XT[col][k], pitch W + 4), so that a
// k-step of a 32-column tile is one 16-byte read per lane.
#pragma once

#include <hip/hip_runtime.h>

namespace deeppcr {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));

template <int W>
struct Tile2Shape {
    static constexpr int NWV = W / 32;  // waves, one 32-row strip each
    static constexpr int NT = 64 * NWV;
    static constexpr int PITCH = W + 4;
    static constexpr int NQ = W / 8;  // k-steps of 8 (4 per lane half)
    static constexpr int T = W / 32;  // 32-column tiles of a strip
};

template <int W>
using StripA = v4f[Tile2Shape<W>::NQ];
template <int W>
using StripC = v16f[Tile2Shape<W>::T];

template <int W, bool TRANS>
__device__ __forceinline__ void strip_load(const float* blk, StripA<W>& a, int R, int h) {
#pragma unroll
    for (int q = 0; q < Tile2Shape<W>::NQ; ++q) {
        if constexpr (!TRANS) {
            a[q] = *reinterpret_cast<const v4f*>(blk + R * W + 8 * q + 4 * h);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) a[q][e] = blk[(8 * q + 4 * h + e) * W + R];
        }
    }
}

template <int W>
__device__ __forceinline__ v4f strip_quad(const StripA<W>& a, int q) {
    return a[q];
}
template <int W>
__device__ __forceinline__ v4f strip_quad(const StripC<W>& c, int q) {
    const v16f& x = c[q / 4];
    const int o = 4 * (q % 4);
    return v4f{x[o], x[o + 1], x[o + 2], x[o + 3]};
}

template <int W>
__device__ __forceinline__ void strip_zero(StripC<W>& c) {
#pragma unroll
    for (int tc = 0; tc < Tile2Shape<W>::T; ++tc) c[tc] = v16f{};
}

// x + (x of lane l ^ 32): one v_permlane32_swap exchanges the two halves of
// the wave (no LDS round trip); its two results hold, in every lane, the
// lane's own value and its partner's.
__device__ __forceinline__ float half_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Sum over the lanes l, l ^ W, l ^ 2W, ... of the wave (W = 16 or 32) in
// every lane: the row swap of v_permlane16_swap (16-lane rows 2r and 2r + 1)
// and then that of v_permlane32_swap, no LDS round trip.
template <int W>
__device__ __forceinline__ float group_sum(float v) {
    static_assert(W == 16 || W == 32, "lane groups of 16 or 32");
    if constexpr (W == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v),
                                                        false, false);
        v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    }
    return half_sum(v);
}

// (strip of M) x for x in LDS; every lane of the row gets the sum.
template <int W, class M>
__device__ __forceinline__ float strip_matvec(const M& a, const float* x, int h) {
    float part = 0.f;
#pragma unroll
    for (int q = 0; q < Tile2Shape<W>::NQ; ++q) {
        const v4f xv = *reinterpret_cast<const v4f*>(x + 8 * q + 4 * h);
        const v4f av = strip_quad<W>(a, q);
#pragma unroll
        for (int e = 0; e < 4; ++e) part = fmaf(av[e], xv[e], part);
    }
    return half_sum(part);
}

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over the TPR consecutive lanes of a block row (TPR = 2 .. 16, inside
// one 16-lane DPP row), in every lane of the row: butterfly steps whose
// partner lanes come from DPP permutations (quad_perm [1,0,3,2] and
// [2,3,0,1], then the half-row and row mirrors, which pair each lane with one
// of the other group of 4 or 8 lanes), VALU operations with no LDS round trip.
template <int TPR>
__device__ __forceinline__ float row_sum(float v) {
    v += dpp<0xB1>(v);
    if constexpr (TPR >= 4) v += dpp<0x4E>(v);
    if constexpr (TPR >= 8) v += dpp<0x141>(v);
    if constexpr (TPR >= 16) v += dpp<0x140>(v);
    return v;
}

// No side work in a product's k-loop.
struct NoSide {
    __device__ __forceinline__ void operator()(int) const {}
};

// acc[0 .. NTC-1] = column tiles TC0 .. TC0+NTC-1 of (strip of M) X, X in
// LDS transposed (XT[col][k], pitch PITCH): the right operand of k-step q for
// one column tile is one 16-byte read, and all offsets fit the immediate
// field of one base address.  With MV also returns (strip of M) x for the
// vector x in LDS (every lane of the row gets the sum), from the left
// operands as they pass (for accumulator strips this avoids copying the
// whole strip out of the accumulation registers at once).  side(q) runs at
// k-step q beside the MFMAs of step q-1: work that touches neither XT, a,
// acc nor x (a block going to another LDS buffer, the next strip's loads).
template <int W, int TC0, int NTC, bool MV, class M, class F = NoSide>
__device__ __forceinline__ float strip_product(const float* XT, const M& a, v16f (&acc)[NTC],
                                               int i, int h, const float* x = nullptr,
                                               F side = F{}) {
    using S = Tile2Shape<W>;
#pragma unroll
    for (int tc = 0; tc < NTC; ++tc) acc[tc] = v16f{};
    const float* xb = XT + (32 * TC0 + i) * S::PITCH + 4 * h;
    v4f pv[2][NTC], xv[2];
    float part = 0.f;
#pragma unroll
    for (int q = 0; q <= S::NQ; ++q) {
        if (q < S::NQ) {
#pragma unroll
            for (int tc = 0; tc < NTC; ++tc)
                pv[q & 1][tc] = *reinterpret_cast<const v4f*>(xb + 32 * tc * S::PITCH + 8 * q);
            if constexpr (MV) xv[q & 1] = *reinterpret_cast<const v4f*>(x + 8 * q + 4 * h);
            side(q);
        }
        // keeps the operand reads of step q beside the MFMAs of step q-1
        __builtin_amdgcn_sched_barrier(0);
        if (q > 0) {
            const int qb = (q - 1) & 1;
            const v4f av = strip_quad<W>(a, q - 1);
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int tc = 0; tc < NTC; ++tc)
                    acc[tc] = __builtin_amdgcn_mfma_f32_32x32x2f32(pv[qb][tc][e], av[e], acc[tc],
                                                                   0, 0, 0);
            if constexpr (MV) {
#pragma unroll
                for (int e = 0; e < 4; ++e) part = fmaf(av[e], xv[qb][e], part);
            }
        }
    }
    if constexpr (MV) return half_sum(part);
    return 0.f;
}

// Stores column tiles TC0 .. TC0+NTC-1 of a product strip (row-major block
// in global memory).
template <int W, int TC0, int NTC>
__device__ __forceinline__ void tiles_store(float* dst, const v16f (&acc)[NTC], int R, int h) {
#pragma unroll
    for (int tc = 0; tc < NTC; ++tc)
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
            const v16f& x = acc[tc];
            *reinterpret_cast<v4f*>(dst + R * W + 32 * (TC0 + tc) + 8 * qq + 4 * h) =
                v4f{x[4 * qq], x[4 * qq + 1], x[4 * qq + 2], x[4 * qq + 3]};
        }
}

// A strip to a row-major block in global memory.
template <int W, class M>
__device__ __forceinline__ void strip_store(float* dst, const M& a, int R, int h) {
#pragma unroll
    for (int q = 0; q < Tile2Shape<W>::NQ; ++q)
        *reinterpret_cast<v4f*>(dst + R * W + 8 * q + 4 * h) = strip_quad<W>(a, q);
}

// Quad q (columns 8q + 4h .. +3) of a strip from a block in global memory.
template <int W, bool TRANS>
__device__ __forceinline__ void strip_load_quad(const float* blk, StripA<W>& a, int R, int h,
                                                int q) {
    if constexpr (!TRANS) {
        a[q] = *reinterpret_cast<const v4f*>(blk + R * W + 8 * q + 4 * h);
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) a[q][e] = blk[(8 * q + 4 * h + e) * W + R];
    }
}

// Quad q of a strip to a transposed block in LDS (see strip_put_T).
template <int W, class M>
__device__ __forceinline__ void strip_put_T_quad(float* XT, const M& a, int R, int h, int q) {
    using S = Tile2Shape<W>;
    float* xb = XT + 4 * h * S::PITCH + R;
    const v4f x = strip_quad<W>(a, q);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        xb[(8 * q + e) * S::PITCH] = x[e];
        asm volatile("" ::: "memory");
    }
}

// A strip to a transposed block in LDS (XT[col][row], pitch PITCH).  The
// empty asm statements keep the writes single (not paired into two-offset
// writes, whose short offsets would need a base register per pair of rows):
// every offset then fits the immediate field of one base address.
template <int W, class M>
__device__ __forceinline__ void strip_put_T(float* XT, const M& a, int R, int h) {
    using S = Tile2Shape<W>;
    float* xb = XT + 4 * h * S::PITCH + R;
#pragma unroll
    for (int q = 0; q < S::NQ; ++q) {
        const v4f x = strip_quad<W>(a, q);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            xb[(8 * q + e) * S::PITCH] = x[e];
            asm volatile("" ::: "memory");
        }
    }
}

}  // namespace
}  // namespace deeppcr
