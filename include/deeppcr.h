/*
 * deeppcr.h -- C ABI of the DeepPCR hot path for AMD Instinct MI355X (gfx950).
 *
 * DeepPCR (Danieli et al., "DeepPCR: Parallelizing Sequential Operations in
 * Neural Networks", NeurIPS 2023) writes an L-step recurrence
 * z_l = f_l(z_{l-1}) as one system F(z) = 0 (Sec. 2, Eq. 1), solves it with
 * Newton's method (Eq. 2) whose linear systems are block bidiagonal (Eq. 3),
 * and solves those with Parallel Cyclic Reduction in ceil(log2 L) levels
 * (Sec. 3, Alg. 1).  The backward pass is the transposed block-bidiagonal
 * system, solved by one PCR pass without Newton (App. A.2, Eq. 12).
 *
 * Conventions for every entry point
 *   - Indices are 0-based.  Layer l = 0..L-1 maps Z[:, l-1] to Z[:, l] with
 *     Z[:, -1] := z0 (an input).  J_l = dZ[:, l] / dZ[:, l-1].
 *   - Every array pointer is a DEVICE pointer to contiguous, row-major float32
 *     memory owned by the caller, starting on a 16-byte boundary (the kernels
 *     load rows as 16-byte vectors; a misaligned pointer returns
 *     DEEPPCR_EINVAL).  The library never allocates device memory; all
 *     scratch lives in the caller's `workspace` (size from
 *     deeppcr_workspace_bytes, also 16-byte aligned), which must not overlap
 *     any other argument.  One workspace must not be used by two calls that
 *     run concurrently.
 *   - Host-side state.  The first Newton call (the forward entry points and
 *     deeppcr_newton_step) of a host thread allocates one pinned, mapped host
 *     buffer of 32 bytes for that thread's per-iteration read-back of the
 *     convergence measures; it is reused by the thread's later calls and
 *     freed by deeppcr_release_thread_state().  The text of the last error
 *     and the instrumentation state are also per host thread.  Nothing else
 *     persists between calls, so calls from different host threads on
 *     different workspaces are independent.
 *   - All GPU work is enqueued on `stream` (a hipStream_t passed as void*;
 *     NULL is the default stream).  pcr_solve_block_bidiag and
 *     deeppcr_mlp_backward return without waiting for the GPU;
 *     the Newton entry points wait once per Newton iteration to read their
 *     convergence measures: a one-workgroup kernel at the end of the
 *     iteration reduces them and writes them, then a sequence word, into the
 *     thread's mapped host buffer, and the call watches that word, falling
 *     back to a stream wait after 5 ms (a problem small enough for the
 *     one-launch solver waits once, the same way, for the kernel's status
 *     record and completion word).  The last kernel may still be retiring
 *     when the call returns; later work on `stream` is ordered after it.
 *   - Host out-parameters are plain host pointers.
 *   - Arguments are validated before any HIP call: an invalid argument returns
 *     DEEPPCR_EINVAL (or DEEPPCR_EWORKSPACE for a short workspace) and
 *     launches nothing.  A HIP runtime error returns DEEPPCR_EHIP; its text is
 *     available from deeppcr_last_error().
 *   - Arithmetic is float32 with float32 accumulation (no reduced-precision
 *     matrix instructions).  Results are deterministic run to run.
 */
#ifndef DEEPPCR_H
#define DEEPPCR_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    DEEPPCR_OK = 0,
    DEEPPCR_EINVAL = 1,      /* bad pointer, size, flag or overlap            */
    DEEPPCR_ENOCONV = 2,     /* Newton hit max_iter before the tolerance      */
    DEEPPCR_ENONFINITE = 3,  /* a NaN/Inf appeared in the Newton iterate      */
    DEEPPCR_EHIP = 4,        /* HIP runtime error                             */
    DEEPPCR_EWORKSPACE = 5   /* workspace_bytes below deeppcr_workspace_bytes */
};

/* Layer kinds: code = 2 * activation + residual.  The plain kinds are the
 * MLP layer of App. A.1 (Eq. 7) written on post-activation states; the
 * residual kinds are residual blocks with a skip of length one (App. A.3).
 * The activations are those of the paper's MLP experiments (Sec. 4.1,
 * App. C): tanh, logistic sigmoid and ReLU (whose derivative is taken as 0
 * at 0). */
enum {
    DEEPPCR_TANH_MLP = 0,         /* Z_l = tanh(W_l Z_{l-1} + b_l)                    */
    DEEPPCR_TANH_RESIDUAL = 1,    /* Z_l = Z_{l-1} + alpha*tanh(W_l Z_{l-1} + b_l)    */
    DEEPPCR_SIGMOID_MLP = 2,      /* Z_l = sigmoid(W_l Z_{l-1} + b_l)                 */
    DEEPPCR_SIGMOID_RESIDUAL = 3, /* Z_l = Z_{l-1} + alpha*sigmoid(W_l Z_{l-1} + b_l) */
    DEEPPCR_RELU_MLP = 4,         /* Z_l = max(W_l Z_{l-1} + b_l, 0)                  */
    DEEPPCR_RELU_RESIDUAL = 5     /* Z_l = Z_{l-1} + alpha*max(W_l Z_{l-1} + b_l, 0)  */
};

enum { DEEPPCR_OP_PCR = 0, DEEPPCR_OP_FWD = 1, DEEPPCR_OP_BWD = 2 };

/* Largest supported state width w. */
#define DEEPPCR_MAX_WIDTH 1024
/* Largest width of the collapsed-skip ResNet entry points and of
 * pcr_solve_block_bidiag_chunked. */
#define DEEPPCR_MAX_BLOCK_WIDTH 128

/* Bytes of device workspace that operation `op` (DEEPPCR_OP_*) needs for a
 * batch of B systems of L rows of width w: two ping-pong copies of the
 * operators A_l ([B, L, w, w] each; the extra memory the paper attributes to
 * the stored A_l, Sec. 3.1) plus vectors and a small reduction area.
 * Returns 0 for invalid sizes. */
size_t deeppcr_workspace_bytes(int op, int B, int L, int w);

/* Static text for a DEEPPCR_* status code. */
const char* deeppcr_status_string(int status);

/* Text of the last DEEPPCR_EHIP error raised on the calling thread. */
const char* deeppcr_last_error(void);

/* Frees what the library holds for the calling host thread: its pinned
 * read-back buffer and its instrumentation events (after waiting for the
 * recorded ones).  Call it before a thread that used the library ends, or
 * before the process unloads the library; later calls allocate again. */
void deeppcr_release_thread_state(void);

/*
 * Standalone block-bidiagonal solve by Parallel Cyclic Reduction
 * (Sec. 3, Alg. 1 and Eqs. 4-6; the transposed form is the system of
 * App. A.2, Eq. 12).  B independent systems:
 *   transpose = 0:  x[b,l] = J[b,l] x[b,l-1] + r[b,l],        l = 0..L-1, x[b,-1] = 0
 *   transpose = 1:  x[b,l] = J[b,l+1]^T x[b,l+1] + r[b,l],    l = L-1..0, x[b,L]  = 0
 * i.e. M x = r (or M^T x = r) with M = identity blocks on the diagonal and
 * -J[b,l] in block (l, l-1).  J[b,0] is never read.
 *   J  [B, L, w, w]  input, read only
 *   r  [B, L, w]     input
 *   x  [B, L, w]     output; may alias r, must not overlap J
 * 1 <= w <= DEEPPCR_MAX_WIDTH, B >= 1, L >= 1, transpose in {0, 1};
 * workspace_bytes >= deeppcr_workspace_bytes(DEEPPCR_OP_PCR, B, L, w).
 */
int pcr_solve_block_bidiag(const float* J, const float* r, float* x,
                           int B, int L, int w, int transpose,
                           void* workspace, size_t workspace_bytes, void* stream);

/*
 * The standalone solve of pcr_solve_block_bidiag computed the way a solve
 * whose rows are spread over G devices would compute it (the memory and
 * communication setting of Sec. 3.1), all on this one GPU: the rows of each
 * system are cut into consecutive chunks of Lc = ceil(L / G) rows (natural
 * row order; the last chunk may be shorter, so there are ceil(L / Lc) <= G
 * chunks).
 *   1. Chunk-local PCR (Alg. 1 inside every chunk, all chunks at once) that
 *      keeps each chunk's coupling to the one unknown outside it, x_in (row
 *      a-1 of chunk [a, e) for transpose = 0, row e for transpose = 1), so
 *      that every row ends as x_l = P_l x_in + q_l.  For w <= 16 and
 *      w = 32, 64, 128 the chunk's last levels (all but the first
 *      max(1, ceil(log2 Lc) - 6)) are replaced by substitution along the
 *      chains of at most 64 rows they act on: P_j = A_j P_{j-s},
 *      q_j = A_j q_{j-s} + r_j, the way the full solve ends.
 *   2. A pass over the chunk ends in solve order: the carry-in of the next
 *      chunk is P x_in + q at the current chunk's last row (the first
 *      chunk's carry-in is zero).
 *   3. x_l = q_l + P_l x_in for every row.
 * On G devices step 1 runs on each device's rows, step 2 needs the G
 * chunk-end maps (P, q) of one row each from every device, and step 3 is
 * local again.  The result is the solution of pcr_solve_block_bidiag (the
 * summation order differs).
 *   J, r, x, B, L, w, transpose  as for pcr_solve_block_bidiag (x may alias r)
 *   G  >= 1: the number of chunks asked for (G >= L gives one row per chunk)
 * workspace_bytes >= deeppcr_chunked_workspace_bytes(B, L, w, G): two copies
 * of the operators [B, L, w, w], two of the vectors [B, L, w] and the
 * carry-ins [B, chunks, w].  Returns without waiting for the GPU.
 */
size_t deeppcr_chunked_workspace_bytes(int B, int L, int w, int G);
int pcr_solve_block_bidiag_chunked(const float* J, const float* r, float* x,
                                   int B, int L, int w, int transpose, int G,
                                   void* workspace, size_t workspace_bytes, void* stream);

/*
 * pcr_solve_block_bidiag without a workspace argument and without any
 * allocation, for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).
 * The solve, its kernels and its results are those of
 * pcr_solve_block_bidiag (bit for bit); its scratch is a fixed device array
 * of DEEPPCR_NOALLOC_SCRATCH_BYTES inside the library, one per GPU, held
 * from the library's first use on that GPU until the process ends.  The
 * call allocates nothing (no hipMalloc, no host allocation, no new events, even
 * with instrumentation enabled) and enqueues only kernels on `stream`.
 *   J, r, x, B, L, w, transpose as for pcr_solve_block_bidiag.
 * Returns DEEPPCR_EWORKSPACE when the problem needs more scratch than that
 * (deeppcr_workspace_bytes(DEEPPCR_OP_PCR, B, L, w) >
 * DEEPPCR_NOALLOC_SCRATCH_BYTES; e.g. B L w (w + 1) <= about 8.3 million at
 * 64 MiB), before any HIP call.
 * All calls on one GPU share its scratch array: two calls that overlap in
 * time on one GPU (on different streams, or from different host threads)
 * race and give wrong results; serialise them.  The solve needs no part of
 * the scratch to start at zero.
 */
#define DEEPPCR_NOALLOC_SCRATCH_BYTES (64u << 20)
int pcr_solve_block_bidiag_noalloc(const float* J, const float* r, float* x,
                                   int B, int L, int w, int transpose, void* stream);
/* The size of that scratch array, DEEPPCR_NOALLOC_SCRATCH_BYTES. */
size_t deeppcr_noalloc_scratch_bytes(void);

/*
 * One Newton iteration for a step function the caller evaluates (Sec. 2,
 * Eqs. 1-3; the paper's general setting of z_l = f_l(z_{l-1}), e.g. the
 * denoising steps of App. A.4 whose Jacobians come from autograd).  At the
 * current iterate Z the caller supplies, for every step in parallel, the step
 * values F[b, l] = f_l(Z[b, l-1]) (Z[b, -1] being the fixed start) and the
 * Jacobians J[b, l] = df_l/dz at Z[b, l-1]; the library forms the residual
 * r = F - Z, solves the block-bidiagonal system of Eq. 3 for dZ by PCR,
 * applies Z += dZ and tests the update with the rule of
 * deeppcr_mlp_forward: max|dZ| < tol * max(1, max|Z|).  J[b, 0] is never read.
 *   J [B, L, w, w], F [B, L, w]  inputs;  Z [B, L, w] input and output
 *   tol            >= 0 and finite; 0 never reports convergence (a caller
 *                  running a fixed number of iterations ignores ENOCONV)
 *   residual_out   (host, may be NULL) max |F - Z| before the update
 *   max_update_out (host, may be NULL) max |dZ|;  max_abs_out: max |Z| after it
 * Returns DEEPPCR_OK when the update met the tolerance (the iteration has
 * converged), DEEPPCR_ENOCONV when it did not (the caller iterates again),
 * DEEPPCR_ENONFINITE if any of the three measures is NaN/Inf.  Waits for the
 * GPU once.  workspace_bytes >= deeppcr_workspace_bytes(DEEPPCR_OP_PCR, B, L, w).
 */
int deeppcr_newton_step(const float* J, const float* F, float* Z, int B, int L, int w,
                        float tol, void* workspace, size_t workspace_bytes, float* residual_out,
                        float* max_update_out, float* max_abs_out, void* stream);

/*
 * Forward pass of a depth-L network by Newton + PCR (Sec. 2, Eqs. 1-3).
 * Each Newton iteration evaluates every layer and its Jacobian at the current
 * iterate in parallel (App. A.1, Eq. 8), forms the residual
 * r_l = f_l(Z_{l-1}) - Z_l, solves the block-bidiagonal system for the
 * update by PCR and applies it.
 *   W     [L, w, w]  weights (row-major, W[l] acts on column vectors)
 *   bias  [L, w]
 *   z0    [B, w]     network input (the fixed state before layer 0)
 *   Z     [B, L, w]  output: Z[:, l] = output of layer l
 *   layer one of the DEEPPCR_*_MLP / DEEPPCR_*_RESIDUAL kinds; alpha is the
 *         residual branch scale (ignored for the plain kinds)
 *   Z_init NULL: every row starts at the first layer's output f_0(z0)
 *         (App. F.2); else [B, L, w] warm start (App. F.2).  May alias Z.
 *   tol   stop once max|dZ| < tol * max(1, max|Z|) after an update; tol = 0
 *         runs exactly max_iter iterations (fixed-count Newton, App. F.1)
 *   max_iter >= 1: at most this many PCR solves
 *   iters_out       (host, may be NULL) number of PCR solves performed
 *   last_update_out (host, may be NULL) max|dZ| of the last iteration
 * Returns DEEPPCR_ENOCONV if tol > 0 and max_iter iterations did not reach it
 * (Z then holds the last iterate), DEEPPCR_ENONFINITE if the iterate became
 * NaN/Inf (Z holds that iterate).
 */
int deeppcr_mlp_forward(const float* W, const float* bias, const float* z0, float* Z,
                        int B, int L, int w, int layer, float alpha,
                        float tol, int max_iter, const float* Z_init,
                        void* workspace, size_t workspace_bytes,
                        int* iters_out, float* last_update_out, void* stream);

/*
 * Forward pass by Newton + PCR with the residual stopping rule of the
 * paper's Newton-solver parameter table (App. F.1): the infinity norm of the
 * residual F(z^k) = [f_l(Z_{l-1}) - Z_l]_l of Eq. 1 at iterate z^k is tested
 * against an absolute threshold and against a threshold relative to the
 * first iterate's residual norm.  For k = 0, 1, ...: the layers are
 * evaluated at z^k and res_k = max|F(z^k)| is reduced on the fly; the
 * iteration stops with Z = z^k when res_k <= atol or res_k <= rtol * res_0
 * (either one suffices), stops with DEEPPCR_ENOCONV when k = max_iter, and
 * otherwise solves Eq. 3 by PCR and sets z^{k+1} = z^k + dz^k.  (The paper's
 * defaults for forward passes: atol = rtol = 1e-4, max_iter = 15.)
 *   W, bias, z0, Z, layer, alpha, Z_init, workspace  as for deeppcr_mlp_forward
 *   atol, rtol  >= 0 and finite (0 disables the criterion)
 *   max_iter    >= 0: at most this many PCR solves (0 only tests the start)
 *   iters_out    (host, may be NULL) number of PCR solves performed
 *   residual_out (host, may be NULL) res_k of the returned iterate
 * Returns DEEPPCR_ENONFINITE if the residual is NaN/Inf (Z holds that
 * iterate).  Waits for the GPU once per iteration, after the evaluation.
 */
int deeppcr_mlp_forward_residual(const float* W, const float* bias, const float* z0, float* Z,
                                 int B, int L, int w, int layer, float alpha,
                                 float atol, float rtol, int max_iter, const float* Z_init,
                                 void* workspace, size_t workspace_bytes,
                                 int* iters_out, float* residual_out, void* stream);

/*
 * Backward pass by one transposed PCR solve (App. A.2, Eqs. 10-12) for
 * Loss = sum_b <G[b], Z[b, L-1]>.  The layer Jacobians are evaluated at the
 * stored layer inputs Z[:, l-1] (Eq. 11).  With
 * d_l = sigma'(W_l Z_{l-1} + b_l) and c = 1 (plain layers) or alpha
 * (residual layers), the parameter gradients of Eq. 10 read
 *   dW[l] = c * sum_b (d_l * Lambda[b,l]) Z[b,l-1]^T,  db[l] = c * sum_b d_l * Lambda[b,l].
 *   W, bias, z0  as for deeppcr_mlp_forward;  Z [B, L, w] forward states
 *   G      [B, w]     dLoss/dZ[:, L-1]
 *   Lambda [B, L, w]  output: dLoss/dZ[:, l]
 *   dz0    [B, w]     output: dLoss/dz0
 *   dW     [L, w, w]  output (overwritten; summed over the batch)
 *   db     [L, w]     output (overwritten; summed over the batch)
 * workspace_bytes >= deeppcr_workspace_bytes(DEEPPCR_OP_BWD, B, L, w).
 */
int deeppcr_mlp_backward(const float* W, const float* bias, const float* z0, const float* Z,
                         const float* G, float* Lambda, float* dz0, float* dW, float* db,
                         int B, int L, int w, int layer, float alpha,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * Collapsed-skip ResNet (App. A.3).  Fully connected layers in the
 * pre-activation form of the appendix with a skip connection of length
 * `skip`: for layer j = 0..L-1 (Z[:, -1] := z0)
 *   Z[:, j] = W_j sigma(Z[:, j-1]) + b_j                 if (j + 1) % skip != 0
 *   Z[:, j] = W_j sigma(Z[:, j-1]) + b_j + Z[:, j-skip]   if (j + 1) % skip == 0
 * with sigma one of the DEEPPCR_ACT_* activations and L a multiple of skip.
 * Collapsing the layers between two skips turns the network into a Markov
 * chain over the block outputs X_g = Z[:, g*skip + skip - 1],
 * g = 0..L/skip-1, X_{-1} = z0, with steps
 *   X_g = F_g(X_{g-1}) = h_{g*skip+skip-1}(... h_{g*skip}(X_{g-1})) + X_{g-1},
 *   dF_g/dX = I + J_{g*skip+skip-1} ... J_{g*skip},  J_j = W_j diag(sigma'(Z[:, j-1])),
 * (h_j(z) = W_j sigma(z) + b_j), and DeepPCR runs on that chain: L/skip
 * unknowns, each Newton step evaluating every block (its skip layers and the
 * product of their Jacobians) in parallel.
 */
enum { DEEPPCR_ACT_TANH = 0, DEEPPCR_ACT_SIGMOID = 1, DEEPPCR_ACT_RELU = 2 };

/* Workspace bytes of deeppcr_resnet_forward (op = DEEPPCR_OP_FWD) or
 * deeppcr_resnet_backward (DEEPPCR_OP_BWD); 0 for an invalid op or shape. */
size_t deeppcr_resnet_workspace_bytes(int op, int B, int L, int w, int skip);

/*
 * Forward pass by Newton + PCR on the block chain (App. A.3; Sec. 2,
 * Eqs. 1-3).  Each iteration evaluates every block and its Jacobian at the
 * iterate, solves the block-bidiagonal system of Eq. 3 for the block-output
 * update by PCR and applies it; stops once max|dX| < tol * max(1, max|X|)
 * (tol = 0: exactly max_iter iterations).  Start: every X_g = F_0(z0) (the
 * rule of App. F.2 applied to the blocks), or X_g = Z_init[:, g*skip+skip-1].
 * After the last iteration the rows inside each block are recomputed from the
 * block's input X_{g-1}; row g*skip+skip-1 of Z is X_g itself.
 *   W [L, w, w], bias [L, w], z0 [B, w]; Z [B, L, w] output (every layer)
 *   skip >= 1 with L % skip == 0; act a DEEPPCR_ACT_* value
 *   Z_init NULL or [B, L, w] (only its block-output rows are read); may alias Z
 *   iters_out, last_update_out (host, may be NULL): solves, last max|dX|
 * Status as for deeppcr_mlp_forward.  Waits for the GPU once per iteration.
 * workspace_bytes >= deeppcr_resnet_workspace_bytes(DEEPPCR_OP_FWD, B, L, w, skip).
 */
int deeppcr_resnet_forward(const float* W, const float* bias, const float* z0, float* Z,
                           int B, int L, int w, int skip, int act, float tol, int max_iter,
                           const float* Z_init, void* workspace, size_t workspace_bytes,
                           int* iters_out, float* last_update_out, void* stream);

/*
 * Backward pass for Loss = sum_b <G[b], Z[b, L-1]> (App. A.3, "a similar
 * reasoning" for the backward; App. A.2, Eqs. 10-12).  The block-output
 * adjoints mu_g = dLoss/dX_g solve the transposed block system
 * mu_{G-1} = G, mu_{g-1} = (dF_g/dX)^T mu_g by one transposed PCR pass with
 * the block Jacobians evaluated at the stored states Z; the adjoints inside
 * each block follow by back-propagation through its layers,
 * Lambda[:, j-1] = diag(sigma'(Z[:, j-1])) W_j^T Lambda[:, j], and
 *   dW[j] = sum_b Lambda[b, j] sigma(Z[b, j-1])^T,   db[j] = sum_b Lambda[b, j]
 * (Eq. 10 in the pre-activation form), dz0 = dLoss/dz0.
 *   W, z0 as for the forward; Z [B, L, w] forward states; G [B, w]
 *   Lambda [B, L, w], dz0 [B, w], dW [L, w, w], db [L, w]: outputs (overwritten)
 * Returns without waiting for the GPU.
 * workspace_bytes >= deeppcr_resnet_workspace_bytes(DEEPPCR_OP_BWD, B, L, w, skip).
 */
int deeppcr_resnet_backward(const float* W, const float* z0, const float* Z, const float* G,
                            float* Lambda, float* dz0, float* dW, float* db,
                            int B, int L, int w, int skip, int act,
                            void* workspace, size_t workspace_bytes, void* stream);

/*
 * The collapsed-skip ResNet's sequential passes on the GPU (the baseline of
 * the paper's ResNet timings, Sec. 4.2): the network of deeppcr_resnet_forward
 * applied layer after layer, and its reverse-mode adjoints (Lambda, dz0; no
 * parameter gradients).  One workgroup walks the layers of one system;
 * launch_per_layer = 0 runs all layers in one launch, 1 launches once per
 * layer.  No workspace.
 */
int deeppcr_resnet_seq_forward(const float* W, const float* bias, const float* z0, float* Z,
                               int B, int L, int w, int skip, int act, int launch_per_layer,
                               void* stream);
int deeppcr_resnet_seq_backward(const float* W, const float* z0, const float* Z, const float* G,
                                float* Lambda, float* dz0, int B, int L, int w, int skip, int act,
                                int launch_per_layer, void* stream);

/*
 * Sequential passes: the layer-by-layer baseline the paper measures DeepPCR
 * against (Sec. 4.1), on the same GPU.  Forward: Z[:, l] = f_l(Z[:, l-1]) for
 * l = 0..L-1 (Eq. 1 applied one step at a time).  Backward: the adjoints of
 * Eq. 11 by back substitution, Lambda[:, L-1] = G, Lambda[:, l-1] =
 * J_l^T Lambda[:, l], dz0 = J_0^T Lambda[:, 0] (no parameter gradients).
 * One workgroup walks the layers of one system; launch_per_layer = 0 runs all
 * layers in one launch, 1 launches once per layer (as an eager framework's
 * layer loop does).  Arguments as for deeppcr_mlp_forward / _backward; no
 * workspace.
 */
int deeppcr_seq_forward(const float* W, const float* bias, const float* z0, float* Z,
                        int B, int L, int w, int layer, float alpha, int launch_per_layer,
                        void* stream);
int deeppcr_seq_backward(const float* W, const float* bias, const float* z0, const float* Z,
                         const float* G, float* Lambda, float* dz0, int B, int L, int w,
                         int layer, float alpha, int launch_per_layer, void* stream);

/*
 * Instrumentation (not part of the numerical path).  While enabled, the
 * library brackets its kernel launches with HIP events on the launch's own
 * stream and records, per kernel class, the launch count, the summed device
 * time and the algorithmic bytes and flops of each launch.  Consecutive
 * launches of one class on one stream (no host wait or other class between
 * them, e.g. the levels of one PCR sweep) share one event pair, so the time
 * of such a run includes the gaps between its kernels but no event overhead
 * per kernel; where a run of one class follows a run of another, one event
 * ends the first and starts the second.  The state is per host thread: a
 * thread's enable, select, reset and read see only that thread's launches.
 */
enum {
    DEEPPCR_KCLASS_PCR_LEVEL = 0,  /* one PCR level (Alg. 1 inner parfor)      */
    DEEPPCR_KCLASS_LAYER = 1,      /* layers + Jacobian blocks + residual      */
    DEEPPCR_KCLASS_UPDATE = 2,     /* Newton update and convergence reduction  */
    DEEPPCR_KCLASS_WGRAD = 3,      /* parameter gradients                      */
    DEEPPCR_KCLASS_OTHER = 4,      /* initial guess, copies, dz0               */
    DEEPPCR_KCLASS_SEQUENTIAL = 5, /* sequential baseline passes               */
    DEEPPCR_KCLASS_PCR_TAIL = 6,   /* last levels: substitution along the chains */
    DEEPPCR_KCLASS_COUNT = 7
};
int deeppcr_profile_enable(int on);
/* Times only the classes whose bit (1 << class) is set in `class_mask` (all
 * by default); a launch of another class ends the open span without events
 * of its own.  Fewer classes mean fewer events between kernels. */
int deeppcr_profile_select(unsigned class_mask);
void deeppcr_profile_reset(void);
/* Waits for the recorded events, then reports class `kclass`. */
int deeppcr_profile_read(int kclass, long long* launches, double* total_ms,
                         double* alg_bytes, double* alg_flops);

#ifdef __cplusplus
}
#endif

#endif /* DEEPPCR_H */
