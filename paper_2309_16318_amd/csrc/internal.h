// Internal interface between the host driver (api.hip) and the kernel files.
// Not installed; the public interface is include/deeppcr.h.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace deeppcr {

// Widths up to kMaxWidth use the per-width kernels (one workgroup or wave
// holds a whole block); kMaxWidth < w <= kMaxWideWidth use the tiled kernels
// of wide.hip.
constexpr int kMaxWidth = 128;
constexpr int kMaxWideWidth = 1024;

// The Newton convergence maxima are reduced into kRedShards slots each
// (slot = workgroup index mod kRedShards) to keep atomic contention low; the
// host takes the max over the slots after its one read-back per iteration.
// Reduction area: max|dZ| slots, then max|Z| slots (both cleared by the
// forward layer evaluation), then max|F| slots (the residual of the iterate,
// written by the forward layer evaluation; cleared by launch_zero_words).
constexpr int kRedShards = 256;
constexpr int kRedDZ = 0, kRedZ = kRedShards, kRedF = 2 * kRedShards;
constexpr int kRedWords = 3 * kRedShards;

// Layer kinds: code = 2 * activation + residual, activation 0 = tanh,
// 1 = logistic sigmoid, 2 = ReLU (derivative 0 at 0; a NaN input gives NaN).  The residual form is
// f(z) = z + alpha * sigma(W z + b), the plain form f(z) = sigma(W z + b).
constexpr int kNumLayerKinds = 6;
__host__ __device__ inline bool layer_residual(int layer) { return (layer & 1) != 0; }

// sigma(a) for the layer's activation; *d receives sigma'(a).
__device__ inline float activate(int layer, float a, float* d) {
    const int act = layer >> 1;
    if (act == 0) {
        const float t = tanhf(a);
        *d = 1.f - t * t;
        return t;
    }
    if (act == 1) {
        const float s = 1.f / (1.f + expf(-a));
        *d = s * (1.f - s);
        return s;
    }
    // NaN passes through (as max(a, 0) does in the usual frameworks)
    *d = a > 0.f ? 1.f : 0.f;
    return (a > 0.f || __builtin_isnan(a)) ? a : 0.f;
}

// Orders the LDS accesses of one wave (a barrier for the wave only).
__device__ inline void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// A batch of w x w blocks addressed as base + b*bstride + m*rstride (floats).
// Row strides may be negative (the transposed system is stored reversed).
// trans = 1: element (i, k) of block m is stored at [k*w + i].
struct BlockSrc {
    const float* base;
    long long bstride;
    long long rstride;
    int trans;
};

// A batch of length-w vectors, addressed like BlockSrc.
struct VecSrc {
    const float* base;
    long long bstride;
    long long rstride;
};

struct VecDst {
    float* base;
    long long bstride;
    long long rstride;
};

// ---------------------------------------------------------------- PCR level
// Work decomposition of one level with stride s: the rows l >= s form s
// chains (l mod s); each chain is cut into segments of at most n rows;
// segs_per_class segments per chain, total = B * s * segs_per_class items.
struct LevelPlan {
    int s;
    int n;
    int segs_per_class;
    long long total;
};
LevelPlan plan_level(int B, int L, int s, long long target_items, int n_max);

// The blocks of the backward's reversed transposed system formed from the
// weights instead of read from memory: row m >= 1 holds J_{L-m}^T with
// J_l = diag(dscale_l) W_l (+ I for residual layers), dscale [B, L, w].
struct BwdArgs {
    const float* W;       // [L, w, w]
    const float* dscale;  // [B, L, w]
    int residual;
};

// Inputs of the layer evaluation fused into the first PCR level of a Newton
// iteration, and of the Newton update fused into the last level.
struct NewtonArgs {
    const float* W;      // [L, w, w]
    const float* bias;   // [L, w]
    const float* z0;     // [B, w]
    float* Z;            // [B, L, w] current iterate (read by the first level,
                         // updated by the last level)
    unsigned* red;       // reduction area (kRedDZ, kRedZ and kRedF slots)
    int layer;
    float alpha;
};

// Whether the first level with the layer evaluation (layer_first_level) and
// the last level with the update (fused_newton_levels) exist for width w.
bool fused_newton_levels(int w);
bool layer_first_level(int w);

// Number of PCR levels launch_first_level_fwd runs (1, or 2 for w = 64, 128
// when the solve has two levels or more and two_level accepts the shape, and
// for w = 32 from B L >= 2048 chain elements).
int first_level_count(int B, int L, int w);

// First level (s = 1) of the Newton linear solve with the layers, Jacobian
// blocks and residuals evaluated on the fly (never stored):
//   r_l = f_l(Z_{l-1}) - Z_l, J_l = df_l at Z_{l-1};
//   rout[l] = r_l + J_l r_{l-1} (rout[0] = r_0), Aout[l] = J_l J_{l-1} (l >= 2);
// or, when first_level_count says 2, the first two levels: rout and Aout
// then hold what the level s = 2 writes.
// Also clears the max|dZ| and max|Z| slots and reduces max|r| into the
// kRedF slots.
hipError_t launch_first_level_fwd(const NewtonArgs& na, float* Aout, const VecDst& rout, int B,
                                  int L, int w, hipStream_t stream);

// Last level of the Newton linear solve (stride s, reading the previous
// level's blocks and vectors) fused with the update: Z[l] += x_l for every
// row, and atomic max of |x| and |Z| into na.red.
hipError_t launch_last_level_update(const BlockSrc& Ain, const VecSrc& rin, const NewtonArgs& na,
                                    int B, int L, int w, int s, hipStream_t stream);

// One level (stride s) of Parallel Cyclic Reduction over B systems of L rows:
//   rows l <  s : rout[l] = rin[l]                     (already final)
//   rows l >= s : rout[l] = rin[l] + Ain[l] rin[l-s]
//   rows l >= 2s: Aout[l] = Ain[l] Ain[l-s]
// Aout is contiguous [B, L, w, w] in internal row order.
hipError_t launch_pcr_level(const BlockSrc& Ain, const VecSrc& rin, float* Aout,
                            const VecDst& rout, int B, int L, int w, int s,
                            hipStream_t stream);

// Two levels (strides s and 2s) in one pass, where two_level accepts the
// shape: rout[l] and Aout[l] hold what level 2s would have written
// (operators for rows l >= 4s).  Aout must not be the buffer Ain reads.
bool two_level(int B, int L, int w);

// The first two levels (s = 1, 2) of the backward solve with the blocks
// formed from the weights (w = 32, 64, 128, L > 2); rout and Aout as for
// launch_pcr_level2.
hipError_t launch_pcr_level2_bwd(const BwdArgs& bw, const VecSrc& rin, float* Aout,
                                 const VecDst& rout, int B, int L, int w, hipStream_t stream);

// The number of last levels (0: none) solved instead by substitution along
// the chains they act on (launch_pcr_chain_subst), for the problem shape and
// the number of levels `first` the solve's first pass does (then pairs up to
// them): 3 to 6 levels at w = 32, 64, 128.
int tail_levels(int B, int L, int w, int first);
// After the levels with strides below s = 2^(levels - kt) every row l >= s
// satisfies x_l = A_l x_{l-s} + r_l: B s independent chains
// (l = c, c + s, ...), each solved by substitution, one mat-vec per row.
// Ain holds the operators of the level before (rows l >= s), not
// transposed; the solution goes to rout.  With red, rout is the Newton
// iterate instead: the solution is added to it and max |x|, max |Z + x| are
// reduced into the kRedDZ, kRedZ slots of red.
hipError_t launch_pcr_chain_subst(const BlockSrc& Ain, const VecSrc& rin, const VecDst& rout,
                                  int B, int L, int w, int s, hipStream_t stream,
                                  unsigned* red = nullptr);

// The last two levels of a solve (strides s, 2s with 4s >= L) in one pass
// without operator products (mat-vecs only), for the widths last_pair_width
// accepts; rout gets the solution.
bool last_pair_width(int w);
hipError_t launch_pcr_level2_last(const BlockSrc& Ain, const VecSrc& rin, const VecDst& rout,
                                  int B, int L, int w, int s, hipStream_t stream);
hipError_t launch_pcr_level2(const BlockSrc& Ain, const VecSrc& rin, float* Aout,
                             const VecDst& rout, int B, int L, int w, int s,
                             hipStream_t stream);

// ------------------------------------------------------------ layer kernels
// Forward Newton step: for every (b, l) evaluate the layer at Zprev = Z[b,l-1]
// (z0[b] for l = 0), write r[b,l] = f_l(Zprev) - Z[b,l] and, for l >= 1,
// the Jacobian block J_l into A ([B, L, w, w], forward row order).  The grid
// also clears the max|dZ| and max|Z| slots of `red` and reduces max|r| into
// its kRedF slots.
hipError_t launch_forward_eval(const float* W, const float* bias, const float* z0,
                               const float* Z, float* A, float* r, unsigned* red,
                               int B, int L, int w, int layer, float alpha,
                               hipStream_t stream);

// Z[b, l] = f_0(z0[b]) for every l.
hipError_t launch_initial_guess(const float* W, const float* bias, const float* z0,
                                float* Z, int B, int L, int w, int layer, float alpha,
                                hipStream_t stream);

// Z += x over n floats; red[kRedDZ + slot] = max bits of |x|,
// red[kRedZ + slot] = max bits of |Z| (atomic max on the IEEE bit patterns of
// non-negative floats, which orders NaN above Inf).
hipError_t launch_update_reduce(float* Z, const float* x, long long n, unsigned* red,
                                hipStream_t stream);

// Backward: Jacobian blocks of the transposed system in reversed row order,
// blocks[m = L-l] = J_l^T for l >= 1 (stored as J_l itself, i.e. to be read
// transposed, when backward_blocks_transposed(w)), right-hand side
// rrev[m] = G if m == 0 else 0, and dscale[b, l] = c * (1 - tanh(a_l)^2) in
// natural order.  For w = 16, 32, 64, 128 a null `blocks` skips the blocks.
bool backward_blocks_transposed(int w);
hipError_t launch_backward_assemble(const float* W, const float* bias, const float* z0,
                                    const float* Z, const float* G, float* A, float* rrev,
                                    float* dscale, int B, int L, int w, int layer,
                                    float alpha, hipStream_t stream);

// dz0[b] = J_0^T Lambda[b, 0].
hipError_t launch_dz0(const float* W, const float* dscale, const float* Lambda, float* dz0,
                      int B, int L, int w, int layer, hipStream_t stream);

// dW[l] = sum_b (dscale*Lambda)[b,l] Zprev[b,l]^T, db[l] = sum_b (dscale*Lambda)[b,l].
hipError_t launch_wgrad(const float* z0, const float* Z, const float* dscale,
                        const float* Lambda, float* dW, float* db, int B, int L, int w,
                        hipStream_t stream);

// r = F - Z over n floats; max |r| bits into the kRedF slots of red.
hipError_t launch_residual(const float* F, const float* Z, float* r, long long n, unsigned* red,
                           hipStream_t stream);

// p[0 .. n) = 0 (a kernel, so that the call can sit in a captured graph).
hipError_t launch_zero_words(unsigned* p, int n, hipStream_t stream);
// out (host-mapped): out[0..2] = max over the kRedDZ, kRedZ, kRedF slots of
// red, then out[3] = seq.
hipError_t launch_measures(const unsigned* red, unsigned* out, unsigned seq, hipStream_t stream);

// dW[l] = sum_b Lambda[b,l] sigma(Zprev[b,l])^T, db[l] = sum_b Lambda[b,l]
// (pre-activation layers W sigma(z) + b; activation act: 0 tanh, 1 sigmoid,
// 2 ReLU).
hipError_t launch_wgrad_pre(const float* z0, const float* Z, const float* Lambda, float* dW,
                            float* db, int B, int L, int w, int act, hipStream_t stream);

// dst[b, l] = src[b, l] for every (b, l) (used when L = 1).
hipError_t launch_copy_rows(const VecSrc& src, const VecDst& dst, int B, int L, int w,
                            hipStream_t stream);

// ----------------------------------------------------------- small widths
// w <= 8: one PCR level with a lane group per row, and the layer evaluation
// with one thread per state element (forward and backward layouts as in
// launch_forward_eval / launch_backward_assemble).
bool small_width(int w);
hipError_t launch_pcr_level_small(const BlockSrc& Ain, const VecSrc& rin, float* Aout,
                                  const VecDst& rout, int B, int L, int w, int s,
                                  hipStream_t stream);
hipError_t launch_eval_small(bool bwd, const float* W, const float* bias, const float* z0,
                             const float* Z, const float* G, float* A, float* r, float* dscale,
                             unsigned* red, int B, int L, int w, int layer, float alpha,
                             hipStream_t stream);

// ------------------------------------------------------- sequential passes
// Layers l0 .. l1-1 of the sequential forward pass (one workgroup per system;
// reads Z[:, l0-1], or z0 when l0 = 0), and the sequential adjoint pass over
// layers l1-1 down to l0 (starting from G when l1 = L, else Lambda[:, l1-1]).
hipError_t launch_seq_forward(const float* W, const float* bias, const float* z0, float* Z, int B,
                              int L, int w, int layer, float alpha, int l0, int l1,
                              hipStream_t stream);
hipError_t launch_seq_backward(const float* W, const float* bias, const float* z0, const float* Z,
                               const float* G, float* Lambda, float* dz0, int B, int L, int w,
                               int layer, float alpha, int l0, int l1, hipStream_t stream);

// ------------------------------------------------- collapsed-skip ResNet
// Blocks of s layers, G = L / s blocks per system, X [B, G, w] the block
// outputs; act: 0 tanh, 1 sigmoid, 2 ReLU.
// Block evaluation at the iterate: r[b,g] = F_g(X[b,g-1]) - X[b,g] and, for
// g >= 1, A[b,g] = I + P_g (forward order); clears the max|dZ|, max|Z| slots.
hipError_t launch_resnet_block_eval(const float* W, const float* bias, const float* z0,
                                    const float* X, float* A, float* r, unsigned* red, int B,
                                    int G, int w, int skip, int act, hipStream_t stream);
// X[b, g] = F_0(z0[b]) for every g.
hipError_t launch_resnet_initial_guess(const float* W, const float* bias, const float* z0,
                                       float* X, int B, int G, int w, int skip, int act,
                                       hipStream_t stream);
// Z [B, L, w]: the layers inside each block run from X[b, g-1]; row gs+s-1 = X[b, g].
hipError_t launch_resnet_expand(const float* W, const float* bias, const float* z0,
                                const float* X, float* Z, int B, int G, int w, int skip, int act,
                                hipStream_t stream);
// Backward blocks at the stored states Z: A[b, G-g] = I + P_g (g >= 1, to be
// read transposed), rrev[b, m] = G[b] if m == 0 else 0.
hipError_t launch_resnet_block_jac(const float* W, const float* z0, const float* Z,
                                   const float* Gv, float* A, float* rrev, int B, int G, int w,
                                   int skip, int act, hipStream_t stream);
// Lambda [B, L, w] inside every block from mu [B, G, w] (block-output
// adjoints, natural order), and dz0.
hipError_t launch_resnet_intra_adjoint(const float* W, const float* z0, const float* Z,
                                       const float* mu, float* Lambda, float* dz0, int B, int G,
                                       int w, int skip, int act, hipStream_t stream);

// The collapsed-skip ResNet's sequential passes (one workgroup per system):
// forward layers l0 .. l1-1, and the reverse-mode adjoints over layers l1-1
// down to l0 (Lambda, and dz0 when l0 = 0).
hipError_t launch_resnet_seq_forward(const float* W, const float* bias, const float* z0, float* Z,
                                     int B, int L, int w, int skip, int act, int l0, int l1,
                                     hipStream_t stream);
hipError_t launch_resnet_seq_backward(const float* W, const float* z0, const float* Z,
                                      const float* G, float* Lambda, float* dz0, int B, int L,
                                      int w, int skip, int act, int l0, int l1,
                                      hipStream_t stream);

// ----------------------------------------------------- row-chunked solve
// The rows of each system cut into chunks of Lc rows (natural order; the
// last chunk may be shorter); rev = 1 runs the transposed system in reversed
// internal row order.  Chunk-local PCR level with stride s keeping every
// chunk's coupling to the row outside it (except the chunk holding internal
// row 0): Aout [B, L, w, w] and rout [B, L, w] contiguous, internal order.
int chunk_count(int L, int Lc);
void chunk_level_work(int B, int L, int w, int Lc, int rev, int s, double* bytes,
                      double* flops);
hipError_t launch_chunk_level(const BlockSrc& Ain, const VecSrc& rin, float* Aout, float* rout,
                              int B, int L, int w, int Lc, int rev, int s, hipStream_t stream);
// The chains left after the chunk-local levels with strides below s, solved
// by substitution into every row's map (P_j, q_j; q only in the chunk
// holding internal row 0), for the widths chunk_chain_width accepts; Ain and
// rin are the level buffers (contiguous, internal order), Pout and qout the
// same layout.
bool chunk_chain_width(int w);
void chunk_chain_work(int B, int L, int w, int Lc, int rev, int s, double* bytes,
                      double* flops);
hipError_t launch_chunk_chain(const float* Ain, const float* rin, float* Pout, float* qout,
                              int B, int L, int w, int Lc, int rev, int s, hipStream_t stream);
// xin [B, chunk_count, w]: the carry-in of every chunk (internal chunk order)
// from the chunk-end rows of P (the final operators) and q (final vectors).
hipError_t launch_chunk_carry(const float* P, const float* q, float* xin, int B, int L, int w,
                              int Lc, int rev, hipStream_t stream);
// x (natural-order destination) = q + P xin of each row's chunk.
hipError_t launch_chunk_apply(const float* P, const float* q, const float* xin, const VecDst& x,
                              int B, int L, int w, int Lc, int rev, hipStream_t stream);

// ------------------------------------------------------------ wide widths
// kMaxWidth < w <= kMaxWideWidth: the same operations as launch_pcr_level,
// launch_forward_eval, launch_initial_guess, launch_backward_assemble (blocks
// stored as J_l, read transposed), launch_dz0 and launch_wgrad, and one
// layer l of the sequential passes (the backward uses dz0 as its scratch for
// the scaled adjoint until the last step).
bool wide_width(int w);
hipError_t launch_pcr_level_wide(const BlockSrc& Ain, const VecSrc& rin, float* Aout,
                                 const VecDst& rout, int B, int L, int w, int s,
                                 hipStream_t stream);
hipError_t launch_forward_eval_wide(const float* W, const float* bias, const float* z0,
                                    const float* Z, float* A, float* r, unsigned* red, int B,
                                    int L, int w, int layer, float alpha, hipStream_t stream);
hipError_t launch_initial_guess_wide(const float* W, const float* bias, const float* z0, float* Z,
                                     int B, int L, int w, int layer, float alpha,
                                     hipStream_t stream);
hipError_t launch_backward_assemble_wide(const float* W, const float* bias, const float* z0,
                                         const float* Z, const float* G, float* A, float* rrev,
                                         float* dscale, int B, int L, int w, int layer,
                                         float alpha, hipStream_t stream);
hipError_t launch_dz0_wide(const float* W, const float* dscale, const float* Lambda, float* dz0,
                           int B, int L, int w, int layer, hipStream_t stream);
hipError_t launch_wgrad_wide(const float* z0, const float* Z, const float* dscale,
                             const float* Lambda, float* dW, float* db, int B, int L, int w,
                             hipStream_t stream);
hipError_t launch_seq_forward_wide(const float* W, const float* bias, const float* z0, float* Z,
                                   int B, int L, int w, int layer, float alpha, int l,
                                   hipStream_t stream);
hipError_t launch_seq_backward_wide(const float* W, const float* bias, const float* z0,
                                    const float* Z, const float* G, float* Lambda, float* dz0,
                                    int B, int L, int w, int layer, float alpha, int l,
                                    hipStream_t stream);

// ------------------------------------------------------------- tiny path
// Whole Newton + PCR forward solve in one workgroup with everything in LDS,
// for batches that fit in 64 KiB.  result[0] = status (0 ok, 2 no
// convergence, 3 non-finite), result[1] = solves, result[2] = bits of the
// last max|dZ| (update rule) or of the last residual norm (residual rule).
// Z_init may be null or alias Z.
struct StopRule {
    int residual;  // 0: max|dZ| < tol * max(1, max|Z|) after each update;
                   // 1: max|F| <= atol or <= rtol * max|F_0| before each solve
    float tol, atol, rtol;
    int max_iter;
};
bool tiny_eligible(int B, int L, int w);
size_t tiny_lds_bytes(int B, int L, int w);
hipError_t launch_newton_tiny(const float* W, const float* bias, const float* z0, float* Z,
                              const float* Z_init, int B, int L, int w, int layer, float alpha,
                              const StopRule& rule, unsigned* result, hipStream_t stream);

}  // namespace deeppcr
